"""The C ABI library loads and exports every entry point of include/msd.h
(no compute: runs without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "msd.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(msd_[a-z_]+)\s*\(", src)))


def test_header_declares_the_four_calls():
    names = declared_functions()
    for n in ("msd_prefill", "msd_draft_tree", "msd_verify", "msd_accept_compact"):
        assert n in names


def test_library_exports_every_declared_symbol():
    from paper_2505_14260_amd import msd
    if not os.path.exists(msd.LIB_PATH):
        pytest.skip("libmsd.so not built")
    lib = ctypes.CDLL(msd.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_struct_sizes_match_header_layout():
    from paper_2505_14260_amd import msd
    # msd_tree: int32 + 3*64 int32 + 64 float, padded to 8, + 64 uint64
    assert ctypes.sizeof(msd.Tree) == 4 + 3 * 256 + 256 + 4 + 512
    assert ctypes.sizeof(msd.ModelDesc) == 9 * 4


def test_buffer_sizes_and_errors_without_gpu():
    from paper_2505_14260_amd import msd
    if not os.path.exists(msd.LIB_PATH):
        pytest.skip("libmsd.so not built")
    d = msd.ModelDesc(2, 128, 4, 2, 64, 256, 512, 1e4, 1e-5)
    lim = msd.Limits(1, 256, 16, 64)
    tkv, dkv, ws, pw = msd.msd_buffer_sizes(d, lim)
    assert tkv == 2 * 1 * 2 * 256 * 64 * 2 and dkv == tkv // 2 and ws > 0

    def packed(n, k):  # 64-row x 128-column bf16 blocks, zero-padded
        return -(-n // 64) * -(-k // 128) * 64 * 128 * 2
    dm, hd, H, KV, F, V = 128, 64, 4, 2, 256, 512
    layer = (packed(H * hd, dm) + 2 * packed(KV * hd, dm) + packed(dm, H * hd)
             + 2 * packed(F, dm) + packed(dm, F))
    assert pw == 3 * layer + packed(dm, 2 * dm) + packed(V, dm)
    bad = msd.ModelDesc(2, 128, 4, 3, 64, 256, 512, 1e4, 1e-5)
    with pytest.raises(msd.MSDError) as e:
        msd.msd_buffer_sizes(bad, lim)
    assert e.value.code == msd.MSD_ERR_INVALID_ARG
    with pytest.raises(msd.MSDError):
        msd.msd_buffer_sizes(msd.ModelDesc(2, 128, 4, 2, 96, 256, 512, 1e4, 1e-5), lim)
    with pytest.raises(msd.MSDError):
        msd.msd_buffer_sizes(d, msd.Limits(1, 256, 65, 64))
    # a packed matrix of 2 GiB or more is refused (the weight stream's 32-bit
    # byte offsets): the LM head 131072 x 8192 is exactly 2^31 bytes, one
    # 64-row tile fewer fits
    with pytest.raises(msd.MSDError) as e:
        msd.msd_buffer_sizes(msd.ModelDesc(1, 8192, 64, 8, 128, 8192, 131072, 1e4, 1e-5), lim)
    assert e.value.code == msd.MSD_ERR_INVALID_ARG
    assert packed(131072, 8192) == 1 << 31 and packed(131008, 8192) < 1 << 31
    msd.msd_buffer_sizes(msd.ModelDesc(1, 8192, 64, 8, 128, 8192, 131008, 1e4, 1e-5), lim)


def test_training_schedule_and_mix_match_oracle():
    # host-side arithmetic of the training calls (no GPU): the cosine
    # schedule and the progressive mix of Eq. progressive_data
    from paper_2505_14260_amd import msd
    from oracle import train as TR
    if not os.path.exists(msd.LIB_PATH):
        pytest.skip("libmsd.so not built")
    for total in (1, 7, 100):
        for step in range(total + 1):
            assert abs(msd.msd_train_lr(step, total, 5e-5) - TR.cosine_lr(step, total, 5e-5)) \
                <= 1e-20
    for T in (1, 4, 5, 20):
        for t in range(T + 1):
            for n in (0, 3, 40, 68000):
                assert msd.msd_train_mix(t, T, n) == TR.progressive_counts(t, T, n)
    with pytest.raises(msd.MSDError):
        msd.msd_train_lr(5, 4, 1.0)
    with pytest.raises(msd.MSDError):
        msd.msd_train_mix(6, 5, 10)


def test_context_calls_reject_a_null_context_without_gpu():
    from paper_2505_14260_amd import msd
    if not os.path.exists(msd.LIB_PATH):
        pytest.skip("libmsd.so not built")
    for call in (lambda: msd.msd_use_caller_weights(None, 1),
                 lambda: msd.msd_set_draft_input(None, 0)):
        with pytest.raises(msd.MSDError) as e:
            call()
        assert e.value.code == msd.MSD_ERR_INVALID_ARG
