"""Seeded synthetic inputs shared by the CPU oracle and the HIP path.

Holds no arithmetic of the decoding method: it only draws numbers (see
synth.c for the generator's definition) and lays them out as weight tensors,
prompts and test fixtures.  Weights are returned as bfloat16 bit patterns in
numpy uint16 arrays, row-major [out_features, in_features].
"""
import ctypes
import os
import subprocess

import numpy as np

from .configs import WORKLOADS, Workload, ModelDims, TreeShape  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

# tensor ids (see synth.c for how (seed, tid, i) picks a number)
TID_EMBED, TID_LM_HEAD = 1, 2
TID_TEST = 16            # 16..63: free for test fixtures
TID_LAYER0 = 64          # layer l, matrix j -> 64 + 8*l + j
TID_DRAFT = 1024         # draft-only random tensors
TID_VISUAL = 2048        # + sequence index
TID_TEXT = 2560          # + sequence index
BF16_ONE = 0x3F80


def build():
    subprocess.check_call([os.path.join(_HERE, "build.sh")])


def _lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "libsynth.so")
        if not os.path.exists(path):
            build()
        lib = ctypes.CDLL(path)
        u64, u32, dbl, p = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_double, ctypes.c_void_p
        lib.synth_normal_bf16.argtypes = [p, u64, u64, u32, u32, dbl]
        lib.synth_normal_f32.argtypes = [p, u64, u64, u32, u32, dbl]
        lib.synth_ids.argtypes = [p, u64, u64, u32, u32, u32]
        lib.synth_fill_bf16.argtypes = [p, u64, ctypes.c_uint16]
        _LIB = lib
    return _LIB


def normal_bf16(shape, seed, tid, sigma, out=None):
    n = int(np.prod(shape))
    a = np.empty(shape, dtype=np.uint16) if out is None else out
    assert a.dtype == np.uint16 and a.flags.c_contiguous and a.size == n
    _lib().synth_normal_bf16(a.ctypes.data, n, 0, seed, tid, float(sigma))
    return a


def normal_f32(shape, seed, tid, sigma):
    n = int(np.prod(shape))
    a = np.empty(shape, dtype=np.float32)
    _lib().synth_normal_f32(a.ctypes.data, n, 0, seed, tid, float(sigma))
    return a


def ids(n, seed, tid, vocab):
    a = np.empty(n, dtype=np.int32)
    _lib().synth_ids(a.ctypes.data, n, 0, seed, tid, vocab)
    return a


def ones_bf16(n):
    a = np.empty(n, dtype=np.uint16)
    _lib().synth_fill_bf16(a.ctypes.data, n, BF16_ONE)
    return a


def bf16_to_f32(a):
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.asarray(a, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def f32_to_bf16(a):
    """Round-to-nearest-even narrowing of float32 values to bfloat16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


LAYER_KEYS = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")


def layer_shapes(dims: ModelDims):
    d, hd, F = dims.d_model, dims.head_dim, dims.ffn_dim
    return {
        "wq": (dims.n_heads * hd, d), "wk": (dims.n_kv_heads * hd, d),
        "wv": (dims.n_kv_heads * hd, d), "wo": (d, dims.n_heads * hd),
        "wg": (F, d), "wu": (F, d), "wd": (d, F),
    }


def make_target_weights(dims: ModelDims, seed: int, sigma: float = 0.02):
    """Random-init target: every matrix ~ N(0, sigma^2) in bf16, norm gains 1."""
    shapes = layer_shapes(dims)
    w = {
        "embed": normal_bf16((dims.vocab, dims.d_model), seed, TID_EMBED, sigma),
        "lm_head": normal_bf16((dims.vocab, dims.d_model), seed, TID_LM_HEAD, sigma),
        "final_norm": ones_bf16(dims.d_model),
        "layers": [],
    }
    for l in range(dims.n_layers):
        lw = {k: normal_bf16(shapes[k], seed, TID_LAYER0 + 8 * l + j, sigma)
              for j, k in enumerate(LAYER_KEYS)}
        lw["attn_norm"] = ones_bf16(dims.d_model)
        lw["ffn_norm"] = ones_bf16(dims.d_model)
        w["layers"].append(lw)
    return w


def make_draft_weights(dims: ModelDims, target, seed: int, mode: str = "hidden",
                       sigma: float = 0.02):
    """One-layer draft head.

    The decoder layer is a copy (own buffers) of the target's last layer so
    that a random-init draft agrees with the target often enough to accept.
    The down-projection fc: [d, 2d] acting on concat(hidden, embedding):
      "hidden"    -> [I | 0]   (passes the target feature through)
      "embedding" -> [0 | I]   (passes the next-token embedding through)
      "mean"      -> [I/2 | I/2]
      "random"    -> N(0, sigma^2)
    """
    d = dims.d_model
    if mode == "random":
        fc = normal_bf16((d, 2 * d), seed, TID_DRAFT, sigma)
    else:
        fc = np.zeros((d, 2 * d), dtype=np.uint16)
        eye = np.arange(d)
        if mode == "hidden":
            fc[eye, eye] = BF16_ONE
        elif mode == "embedding":
            fc[eye, d + eye] = BF16_ONE
        elif mode == "mean":
            half = 0x3F00  # 0.5
            fc[eye, eye] = half
            fc[eye, d + eye] = half
        else:
            raise ValueError(mode)
    last = target["layers"][-1]
    layer = {k: np.array(v, copy=True) for k, v in last.items()}
    return {"fc": fc, "layer": layer}


def make_prompt(wl: Workload, seq: int = 0):
    """Visual rows first, then text ids (no system tokens before the image).

    Returns (tokens int32[n], is_visual uint8[n], visual bf16 bits [n_vis, d]);
    token ids at visual positions are 0 and unused.
    """
    d = wl.dims.d_model
    n = wl.prompt_len
    tokens = np.zeros(n, dtype=np.int32)
    tokens[wl.n_visual:] = ids(wl.n_text, wl.seed, TID_TEXT + seq, wl.dims.vocab)
    is_visual = np.zeros(n, dtype=np.uint8)
    is_visual[:wl.n_visual] = 1
    visual = normal_bf16((wl.n_visual, d), wl.seed, TID_VISUAL + seq, wl.visual_scale)
    return tokens, is_visual, visual


def static_tree_arrays(paths):
    """Rank paths -> (parent, rank, depth) for nodes 0..N; node 0 is the root.

    Nodes are numbered in canonical order: depth ascending, then rank path
    lexicographically, so every parent precedes its children.
    """
    index = {"": 0}
    parent, rank, depth = [-1], [0], [0]
    for i, p in enumerate(sorted(paths, key=lambda q: (len(q), q)), start=1):
        if p[:-1] not in index:
            raise ValueError(f"parent of {p!r} missing")
        index[p] = i
        parent.append(index[p[:-1]])
        rank.append(int(p[-1]))
        depth.append(len(p))
    return (np.array(parent, dtype=np.int32), np.array(rank, dtype=np.int32),
            np.array(depth, dtype=np.int32))
