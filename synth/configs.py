"""Workload definitions (model shapes, prompts, tree shapes, seeds).

Pure data: nothing in this module computes any part of the decoding method.
Each entry describes a Llama-style target (pre-norm RMSNorm, rotate-half RoPE,
SwiGLU FFN, no biases, untied embedding / LM head), its one-layer draft head,
the multimodal prompt layout (visual rows first, then text) and the draft-tree
shape used by each decode cycle.
"""
from dataclasses import dataclass, field
from typing import Optional, Tuple

# Static 26-node, depth-5 tree: rank paths per depth ("01" = the root's
# best child's second-best child).
STATIC_26 = [
    "0", "1", "2", "3",
    "00", "01", "02", "10", "11", "20", "30",
    "000", "001", "010", "020", "100", "200",
    "0000", "0001", "0010", "0100", "1000",
    "00000", "00001", "00010", "00100",
]


def full_tree_paths(depth: int, branch: int):
    """Rank paths of the full `branch`-ary tree of the given depth."""
    out, level = [], [""]
    for _ in range(depth):
        level = [p + str(r) for p in level for r in range(branch)]
        out.extend(level)
    return out


def chain_paths(depth: int):
    return ["0" * (i + 1) for i in range(depth)]


@dataclass(frozen=True)
class ModelDims:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rope_theta: float
    norm_eps: float


@dataclass(frozen=True)
class TreeShape:
    kind: str                      # "static" | "dynamic"
    depth: int
    paths: Tuple[str, ...] = ()    # static: rank paths in canonical order
    topk: int = 0                  # dynamic: children per expanded node
    n_nodes: int = 0               # dynamic: drafted nodes kept (root excluded)

    @property
    def n_draft(self) -> int:
        return len(self.paths) if self.kind == "static" else self.n_nodes


@dataclass(frozen=True)
class Workload:
    name: str
    dims: ModelDims
    n_visual: int
    n_text: int
    visual_scale: float            # visual rows ~ N(0,1) * visual_scale
    tree: TreeShape
    new_tokens: int
    batch: int = 1
    seed: int = 1000
    weight_sigma: float = 0.02
    draft_fc_mode: str = "hidden"  # see synth.make_draft_weights

    @property
    def prompt_len(self) -> int:
        return self.n_visual + self.n_text


TINY = Workload(
    name="tiny-llama-4L-d256",
    dims=ModelDims(4, 256, 4, 4, 64, 688, 4096, 1e4, 1e-5),
    n_visual=64, n_text=32, visual_scale=1.0 / 16,
    tree=TreeShape("static", 3, tuple(full_tree_paths(3, 2))),
    new_tokens=64, seed=1000,
)

LLAVA7B = Workload(
    name="llava-1.5-7b-shaped",
    dims=ModelDims(32, 4096, 32, 32, 128, 11008, 32000, 1e4, 1e-5),
    n_visual=576, n_text=64, visual_scale=1.0 / 64,
    tree=TreeShape("static", 5, tuple(STATIC_26)),
    new_tokens=512, seed=1001,
)

LLAVA13B = Workload(
    name="llava-1.5-13b-shaped",
    dims=ModelDims(40, 5120, 40, 40, 128, 13824, 32000, 1e4, 1e-5),
    n_visual=576, n_text=128, visual_scale=1.0 / 64,
    tree=TreeShape("static", 5, tuple(STATIC_26)),
    new_tokens=512, seed=1002,
)

LLAVA7B_LONG = Workload(
    name="llava-1.5-7b-shaped-long-visual",
    dims=LLAVA7B.dims,
    n_visual=2880, n_text=256, visual_scale=1.0 / 64,
    tree=TreeShape("dynamic", 6, topk=10, n_nodes=60),
    new_tokens=1024, seed=1003,
)

QWEN7B = Workload(
    name="qwen2.5-vl-7b-shaped",
    dims=ModelDims(28, 3584, 28, 4, 128, 18944, 152064, 1e6, 1e-6),
    n_visual=1024, n_text=128, visual_scale=1.0 / 64,
    tree=TreeShape("dynamic", 6, topk=10, n_nodes=60),
    new_tokens=512, batch=4, seed=1004,
)

# Small grouped-query model for CPU invariant tests.
MINI_GQA = Workload(
    name="mini-gqa-2L-d128",
    dims=ModelDims(2, 128, 4, 2, 32, 256, 512, 1e4, 1e-5),
    n_visual=12, n_text=8, visual_scale=1.0 / 16,
    tree=TreeShape("static", 3, tuple(full_tree_paths(3, 2))),
    new_tokens=24, seed=1010,
)

# Wider small model with a 320-row prompt for the many-row GEMM: an odd
# number of 64-row FFN tiles, a partial last 128-column block and K splits.
WIDE = Workload(
    name="wide-gqa-2L-d1024",
    dims=ModelDims(2, 1024, 8, 2, 128, 2880, 4096, 1e4, 1e-5),
    n_visual=256, n_text=64, visual_scale=1.0 / 32,
    tree=TreeShape("static", 3, tuple(full_tree_paths(3, 2))),
    new_tokens=16, seed=1011,
)

# The widest model the library accepts (d_model 8192, 8-way GQA), one layer,
# with a small FFN and vocabulary so that the oracle stays quick.
MAXW = Workload(
    name="max-width-1L-d8192",
    dims=ModelDims(1, 8192, 64, 8, 128, 2048, 4096, 1e4, 1e-5),
    n_visual=40, n_text=24, visual_scale=1.0 / 64,
    tree=TreeShape("static", 3, tuple(full_tree_paths(3, 2))),
    new_tokens=12, seed=1012,
)

WORKLOADS = {w.name: w for w in (TINY, LLAVA7B, LLAVA13B, LLAVA7B_LONG, QWEN7B, MINI_GQA, WIDE,
                                 MAXW)}
