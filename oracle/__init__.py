"""CPU oracle for the MSD decode path -- TEST INFRASTRUCTURE ONLY.

Only tests/, __graft_entry__.smoke() and the CPU-baseline leg of bench.py may
import this package.  It shares no code with the HIP library and never calls
it; its only common dependency is the seeded input generator (`synth`).

Everything is float64.  Weights are bfloat16 bit patterns (numpy uint16),
widened exactly.  The heavy loops live in orc.c (see its header for the
fixed summation order); the steps of the method are composed here in the
order the paper gives them:

  model.py  target forward (Sec. 3.1) and the one-layer draft head with the
            decoupled draft input (Sec. 4.1, the case split of the draft input
            between text and visual tokens; Sec. 3.2 for the concat form).
  msd.py    draft-tree construction (Sec. 3.2, tree-structured drafting),
            greedy verification / longest accepted path with the bonus token
            (Sec. 3.2 verification, temperature 0), KV compaction, the full
            speculative decode loop and the plain greedy decode it must equal.
  sampling.py speculative sampling on the tree at temperature > 0 (Sec. 3.2
            acceptance rule and adjusted distribution) with its counter-based
            SplitMix64 draws.
  metrics.py the expected-tokens closed form omega(gamma, alpha) and the
            speedup model of Sec. 5.1.3.
  train.py  the draft-head training step of Sec. 4.2 (teacher-forced draft
            forward, feature-regression + token loss, AdamW, cosine schedule,
            the progressive data mix of Eq. progressive_data), in float64
            PyTorch on the CPU with autograd gradients.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None


def build():
    subprocess.check_call([os.path.join(_HERE, "build.sh")])


def lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "liborc.so")
        if not os.path.exists(path):
            build()
        L = ctypes.CDLL(path)
        i, d, p, sz = ctypes.c_int, ctypes.c_double, ctypes.c_void_p, ctypes.c_size_t
        L.orc_linear.argtypes = [i, i, i, p, p, p]
        L.orc_rmsnorm.argtypes = [i, i, p, p, d, p]
        L.orc_rope.argtypes = [i, i, i, p, p, d]
        L.orc_silu_mul.argtypes = [sz, p, p, p]
        L.orc_attention.argtypes = [i, i, i, i, p, p, p, i, i, p, p]
        for f in (L.orc_linear, L.orc_rmsnorm, L.orc_rope, L.orc_silu_mul, L.orc_attention):
            f.restype = None
        _LIB = L
    return _LIB
