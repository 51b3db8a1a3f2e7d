"""MI355X (gfx950) implementation of the multimodal speculative decoding
(MSD, arXiv 2505.14260) decode path: draft tree, tree-masked verification,
greedy acceptance with KV compaction, behind the C ABI of include/msd.h.
"""
from . import msd  # noqa: F401
