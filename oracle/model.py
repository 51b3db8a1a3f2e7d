"""Oracle: target forward and the one-layer decoupled draft head (float64).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Target (Sec. 3.1): the interleaved embedding sequence e_x (text rows from the
embedding table E_t, visual rows given) runs through the decoder; the feature
h_x is the output of the final RMSNorm, and the projection head (LM head)
turns it into next-token logits.

Draft (Sec. 3.2, Eq. concat; Sec. 4.1, Eq. decouple): the draft input row for
position i is
    text i:    f_i = f_down(Concat(h_i, e_{i+1}))   (f_down: Linear 2d -> d)
    visual i:  f_i = e_i                             (the visual embedding)
One decoder layer maps f to the predicted feature, which goes straight into
the target's LM head (no extra norm).
"""
import numpy as np

from . import lib


def _p(a):
    return a.ctypes.data


def widen(bits):
    """bfloat16 bit patterns -> float64 (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def linear(x, w):
    """y = x @ w.T with x [M, K] float64, w [N, K] bf16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    M, K = x.shape
    N = w.shape[0]
    assert w.shape[1] == K and w.dtype == np.uint16 and w.flags.c_contiguous
    y = np.empty((M, N), dtype=np.float64)
    if M:
        lib().orc_linear(M, K, N, _p(x), _p(w), _p(y))
    return y


def rmsnorm(x, g, eps):
    x = np.ascontiguousarray(x, dtype=np.float64)
    y = np.empty_like(x)
    if x.shape[0]:
        lib().orc_rmsnorm(x.shape[0], x.shape[1], _p(x), _p(np.ascontiguousarray(g)), eps, _p(y))
    return y


def rope(x, pos, n_heads, head_dim, theta):
    """Rotate-half RoPE in place on x [M, n_heads*head_dim]."""
    assert x.dtype == np.float64 and x.flags.c_contiguous
    pos = np.ascontiguousarray(pos, dtype=np.int32)
    if x.shape[0]:
        lib().orc_rope(x.shape[0], n_heads, head_dim, _p(x), _p(pos), theta)
    return x


def silu_mul(g, u):
    g = np.ascontiguousarray(g, dtype=np.float64)
    u = np.ascontiguousarray(u, dtype=np.float64)
    y = np.empty_like(g)
    lib().orc_silu_mul(g.size, _p(g), _p(u), _p(y))
    return y


def attention(q, kc, vc, L, R, anc, n_heads, n_kv, head_dim):
    """q [M, H*hd]; kc, vc [S, KV, hd] (one layer); see orc_attention."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    M = q.shape[0]
    o = np.empty_like(q)
    if M == 0:
        return o
    assert kc.flags.c_contiguous and vc.flags.c_contiguous and kc.shape[0] >= L + R
    a = None
    if anc is not None:
        a = np.ascontiguousarray(anc, dtype=np.uint64)
        assert a.shape == (M,) and R <= 64
    else:
        assert R == M
    lib().orc_attention(M, n_heads, n_kv, head_dim, _p(q), _p(kc), _p(vc), L, R,
                        _p(a) if a is not None else None, _p(o))
    return o


class KVCache:
    """float64 K and V, [layers][slots][kv_heads][head_dim]."""

    def __init__(self, n_layers, max_slots, n_kv, head_dim):
        self.k = np.zeros((n_layers, max_slots, n_kv, head_dim), dtype=np.float64)
        self.v = np.zeros_like(self.k)

    def copy(self):
        c = KVCache.__new__(KVCache)
        c.k, c.v = self.k.copy(), self.v.copy()
        return c


def layer_forward(dims, lw, kc, vc, x, pos, slots, L, R, anc):
    """One pre-norm decoder layer on rows x [M, d] (returns the new residual).

    The rows' keys/values are written to `slots` of this layer's cache before
    attention; each row attends to [0, L) plus the region [L, L+R) under the
    causal (anc None) or ancestor-bitmask rule.
    """
    H, KV, hd = dims.n_heads, dims.n_kv_heads, dims.head_dim
    M = x.shape[0]
    a = rmsnorm(x, lw["attn_norm"], dims.norm_eps)
    q = rope(linear(a, lw["wq"]), pos, H, hd, dims.rope_theta)
    k = rope(linear(a, lw["wk"]), pos, KV, hd, dims.rope_theta)
    v = linear(a, lw["wv"])
    kc[slots] = k.reshape(M, KV, hd)
    vc[slots] = v.reshape(M, KV, hd)
    o = attention(q, kc, vc, L, R, anc, H, KV, hd)
    x = x + linear(o, lw["wo"])
    a = rmsnorm(x, lw["ffn_norm"], dims.norm_eps)
    m = silu_mul(linear(a, lw["wg"]), linear(a, lw["wu"]))
    return x + linear(m, lw["wd"])


def embed_rows(weights, tokens, visual_rows=None):
    """Input rows: E_t[token] for text, the given visual embedding otherwise.

    visual_rows: None, or a sequence (one entry per row) of bf16 rows / None.
    """
    x = widen(weights["embed"][np.asarray(tokens, dtype=np.int64)])
    if visual_rows is not None:
        for i, r in enumerate(visual_rows):
            if r is not None:
                x[i] = widen(r)
    return x


def target_forward(dims, weights, kv, x, pos, slots, L, R, anc, want_logits=True):
    """Target decoder over input rows x; returns (h, logits).

    h is the final-RMSNorm feature (what the LM head reads); logits = h Wlm^T.
    """
    for l, lw in enumerate(weights["layers"]):
        x = layer_forward(dims, lw, kv.k[l], kv.v[l], x, pos, slots, L, R, anc)
    h = rmsnorm(x, weights["final_norm"], dims.norm_eps)
    logits = linear(h, weights["lm_head"]) if want_logits else None
    return h, logits


def draft_input(draft, h, e_next, is_visual, e_visual):
    """Decoupled draft input (Eq. decouple), row by row.

    Text rows: f_down(Concat(h_i, e_{i+1})) with h first; visual rows: e_i.
    h, e_next: [M, d] float64 (e_next unused on visual rows);
    e_visual: [M, d] float64 visual embeddings (unused on text rows).
    """
    is_visual = np.asarray(is_visual, dtype=bool)
    f = np.empty_like(h)
    txt = ~is_visual
    if txt.any():
        f[txt] = linear(np.concatenate([h[txt], e_next[txt]], axis=1), draft["fc"])
    if is_visual.any():
        f[is_visual] = e_visual[is_visual]
    return f


def draft_forward(dims, draft, dkv, f, pos, slots, L, R, anc):
    """The draft's decoder layer on input rows f; returns the predicted features."""
    return layer_forward(dims, draft["layer"], dkv.k[0], dkv.v[0], f, pos, slots, L, R, anc)
