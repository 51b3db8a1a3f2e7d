"""Oracle for the draft-head training step -- TEST INFRASTRUCTURE ONLY.

Float64 PyTorch on the CPU: the draft's forward written out plainly and its
gradients from autograd.  It shares nothing with the HIP library.

Sec. 4.2 trains the one-layer draft head against the frozen target in two
stages, first on text-only data, then on a mix whose visual share grows
linearly over the epochs (Eq. progressive_data):
    D_mix^t = D_text (T - t) / T + D_visual t / T,
with the optimiser settings of the experimental set-up (learning rate 5e-5,
cosine schedule, 20 epochs, batch 4).  The paper leaves the loss and the
optimiser to the feature-level draft it builds on; the readings used here:

  * teacher forcing: on a training sequence of n positions the target's
    features h_0 .. h_{n-1} (final-norm outputs, the LM head's input) are
    computed once; the draft's input rows i = 0 .. n-2 follow the decoupled
    rule (Eq. decouple): text rows f_down(Concat(h_i, e_{i+1})), visual rows
    e_i; the draft layer runs causally over them at positions i;
  * the draft output d_i predicts the target feature h_{i+1}:
        loss_i = mean_k SmoothL1(d_i - h_{i+1})_k          (beta = 1)
               + 0.1 * CE(softmax(W_lm h_{i+1}), softmax(W_lm d_i)),
    the cross-entropy taken against the target's full next-token
    distribution at that position;
  * a batch's loss is the mean of loss_i over all rows of its sequences;
  * AdamW (beta1 0.9, beta2 0.999, eps 1e-8, no weight decay) over the draft
    parameters f_down, the layer's seven matrices and its two norm gains; the
    embedding table and LM head are the target's and stay frozen.

Pinned by tests/test_oracle_train.py (finite differences, closed forms,
special cases); parity of everything else is unpinned beyond those.
"""
import math

import numpy as np
import torch

from . import model as M

PARAM_KEYS = ("fc", "wq", "wk", "wv", "wo", "wg", "wu", "wd", "attn_norm", "ffn_norm")
CLS_WEIGHT = 0.1
ADAM_B1, ADAM_B2, ADAM_EPS = 0.9, 0.999, 1e-8


def draft_params(draft):
    """Float64 leaf tensors of the draft's trainable parameters (bf16 bits in)."""
    p = {"fc": draft["fc"]}
    p.update({k: draft["layer"][k] for k in PARAM_KEYS[1:]})
    return {k: torch.tensor(M.widen(v), dtype=torch.float64, requires_grad=True)
            for k, v in p.items()}


def rmsnorm_t(x, g, eps):
    return x * torch.rsqrt((x * x).mean(-1, keepdim=True) + eps) * g


def rope_t(x, pos, n_heads, hd, theta):
    """Rotate-half RoPE of x [M, n_heads*hd] at positions pos (Sec. 3.1 target layer)."""
    half = hd // 2
    inv = theta ** (-2.0 * torch.arange(half, dtype=torch.float64) / hd)
    ang = pos.to(torch.float64)[:, None] * inv[None, :]
    c, s = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]
    x = x.reshape(x.shape[0], n_heads, hd)
    a, b = x[..., :half], x[..., half:]
    return torch.cat([a * c - b * s, b * c + a * s], dim=-1).reshape(x.shape[0], -1)


def causal_attention_t(q, k, v, H, KV, hd):
    """Each row attends to rows 0..itself; query head h reads kv head h // (H/KV)."""
    R = q.shape[0]
    g = H // KV
    q = q.reshape(R, H, hd).transpose(0, 1)                         # [H, R, hd]
    k = k.reshape(R, KV, hd).transpose(0, 1).repeat_interleave(g, 0)
    v = v.reshape(R, KV, hd).transpose(0, 1).repeat_interleave(g, 0)
    s = q @ k.transpose(1, 2) / math.sqrt(hd)
    mask = torch.ones(R, R, dtype=torch.bool).tril()
    s = s.masked_fill(~mask, float("-inf"))
    o = torch.softmax(s, dim=-1) @ v                                 # [H, R, hd]
    return o.transpose(0, 1).reshape(R, H * hd)


def layer_forward_t(dims, p, x, pos):
    """The draft's pre-norm decoder layer, causal over the rows of x."""
    H, KV, hd, eps = dims.n_heads, dims.n_kv_heads, dims.head_dim, dims.norm_eps
    a = rmsnorm_t(x, p["attn_norm"], eps)
    q = rope_t(a @ p["wq"].T, pos, H, hd, dims.rope_theta)
    k = rope_t(a @ p["wk"].T, pos, KV, hd, dims.rope_theta)
    v = a @ p["wv"].T
    x = x + causal_attention_t(q, k, v, H, KV, hd) @ p["wo"].T
    a = rmsnorm_t(x, p["ffn_norm"], eps)
    gt = a @ p["wg"].T
    return x + (gt * torch.sigmoid(gt) * (a @ p["wu"].T)) @ p["wd"].T


def sequence_inputs(m, tokens, is_visual, visual):
    """The frozen target's side of one training sequence (float64 numpy):
    features h [n, d], input embeddings e [n, d] (token rows from the
    embedding table, visual rows given) and its next-token distributions
    softmax(W_lm h) [n, V]."""
    dims = m.dims
    n = len(tokens)
    is_visual = np.asarray(is_visual, dtype=bool)
    rows, vi = [None] * n, 0
    for i in range(n):
        if is_visual[i]:
            rows[i] = visual[vi]
            vi += 1
    e = M.embed_rows(m.w, tokens, rows)
    kv = M.KVCache(dims.n_layers, n, dims.n_kv_heads, dims.head_dim)
    pos = np.arange(n, dtype=np.int32)
    h, logits = M.target_forward(dims, m.w, kv, e.copy(), pos, pos, 0, n, None)
    z = logits - logits.max(axis=1, keepdims=True)
    pt = np.exp(z)
    pt /= pt.sum(axis=1, keepdims=True)
    return h, e, pt


def draft_inputs(p, h, e, is_visual, visual_input="embedding"):
    """Input rows i = 0..n-2 of the draft (Eq. decouple): text rows
    f_down(Concat(h_i, e_{i+1})), visual rows e_i, or h_i in the Visual
    Feature variant of the input-decoupling ablation (Sec. 5.3)."""
    R = h.shape[0] - 1
    vis = torch.as_tensor(np.asarray(is_visual, dtype=bool)[:R])
    cat = torch.cat([h[:R], e[1:]], dim=1)
    src = e[:R] if visual_input == "embedding" else h[:R]
    return torch.where(vis[:, None], src, cat @ p["fc"].T)


def row_losses(d, h, pt, lm_head):
    """Sums over rows i of the regression and cross-entropy terms of loss_i
    for draft outputs d [n-1, d] against target features h [n, d] and the
    target's next-token distributions pt [n, V] (row i against row i + 1)."""
    diff = d - h[1:]
    ad = diff.abs()
    sl1 = torch.where(ad < 1.0, 0.5 * diff * diff, ad - 0.5)
    reg = sl1.mean(dim=1).sum()
    logp = torch.log_softmax(d @ lm_head.T, dim=1)
    cls = -(torch.as_tensor(pt[1:], dtype=torch.float64) * logp).sum()
    return reg, cls


def sequence_loss_sum(dims, p, lm_head, h, e, is_visual, pt, visual_input="embedding"):
    """Sum over rows i = 0..n-2 of loss_i for one sequence, with its parts
    (sum of the regression terms, sum of the cross-entropy terms)."""
    h = torch.as_tensor(h, dtype=torch.float64)
    e = torch.as_tensor(e, dtype=torch.float64)
    R = h.shape[0] - 1
    d = layer_forward_t(dims, p, draft_inputs(p, h, e, is_visual, visual_input),
                        torch.arange(R))
    reg, cls = row_losses(d, h, pt, lm_head)
    return reg + CLS_WEIGHT * cls, reg, cls


def batch_loss(m, params, seqs, visual_input="embedding"):
    """The batch loss alone (no gradients)."""
    lm = torch.as_tensor(M.widen(m.w["lm_head"]), dtype=torch.float64)
    rows = sum(s[0].shape[0] - 1 for s in seqs)
    with torch.no_grad():
        tot = sum(sequence_loss_sum(m.dims, params, lm, h, e, vis, pt, visual_input)[0]
                  for h, e, vis, pt in seqs)
    return float(tot) / rows


def batch_grads(m, params, seqs, visual_input="embedding"):
    """Loss (mean over every row of the batch's sequences) and its gradients.

    seqs: list of (h, e, is_visual, pt) from sequence_inputs.  Returns
    (loss, reg, cls, {key: grad ndarray}) with reg and cls the row means.
    visual_input: the draft input rule of visual rows ("embedding", the
    method, or "feature", the Visual Feature variant).
    """
    lm = torch.as_tensor(M.widen(m.w["lm_head"]), dtype=torch.float64)
    for t in params.values():
        t.grad = None
    rows = sum(s[0].shape[0] - 1 for s in seqs)
    tot = reg = cls = 0.0
    for h, e, vis, pt in seqs:
        l, r, c = sequence_loss_sum(m.dims, params, lm, h, e, vis, pt, visual_input)
        tot = tot + l
        reg += r.item()
        cls += c.item()
    loss = tot / rows
    loss.backward()
    return (loss.item(), reg / rows, cls / rows,
            {k: t.grad.detach().numpy().copy() for k, t in params.items()})


class AdamW:
    """AdamW without weight decay; step t counts from 1 (bias correction)."""

    def __init__(self, params):
        self.m = {k: np.zeros(v.shape) for k, v in params.items()}
        self.v = {k: np.zeros(v.shape) for k, v in params.items()}
        self.t = 0

    def step(self, values, grads, lr):
        """values: {key: float64 ndarray}, updated in place."""
        self.t += 1
        c1 = 1.0 - ADAM_B1 ** self.t
        c2 = 1.0 - ADAM_B2 ** self.t
        for k in values:
            g = grads[k]
            self.m[k] = ADAM_B1 * self.m[k] + (1.0 - ADAM_B1) * g
            self.v[k] = ADAM_B2 * self.v[k] + (1.0 - ADAM_B2) * g * g
            values[k] -= lr * (self.m[k] / c1) / (np.sqrt(self.v[k] / c2) + ADAM_EPS)


def cosine_lr(step, total_steps, lr_max):
    """Cosine learning-rate schedule from lr_max at step 0 to 0 at total_steps."""
    return 0.5 * lr_max * (1.0 + math.cos(math.pi * step / total_steps))


def progressive_counts(epoch, n_epochs, n_per_epoch):
    """Eq. progressive_data: the text-only and visual sample counts of epoch t
    (0-based) of stage 2, the visual share t / T of n_per_epoch samples,
    rounded to the nearest integer (ties to even)."""
    n_vis = int(round(n_per_epoch * epoch / n_epochs))
    return n_per_epoch - n_vis, n_vis
