"""Pins for the oracle's numerical primitives.

Each check compares against something other than the oracle's own formula:
a library routine (numpy matmul, scipy expit, torch SDPA), an algebraic
identity, or a special case with a known answer.
"""
import numpy as np
import pytest
import torch
from scipy.special import expit

import synth
from oracle import model as M


def rng(seed=0):
    return np.random.default_rng(seed)


def bf16_matrix(shape, seed):
    return synth.f32_to_bf16(rng(seed).standard_normal(shape).astype(np.float32) * 0.1)


def test_widen_exact():
    vals = np.array([0.0, 1.0, -2.5, 3.140625, 1e-3, -65504.0], dtype=np.float32)
    bits = synth.f32_to_bf16(vals)
    back = M.widen(bits)
    # bf16 keeps the top 16 bits: widening must reproduce them exactly
    assert np.array_equal(synth.f32_to_bf16(back.astype(np.float32)), bits)
    assert back[1] == 1.0 and back[2] == -2.5 and back[3] == 3.140625


@pytest.mark.parametrize("M_,K,N", [(1, 8, 3), (5, 64, 17), (33, 200, 9)])
def test_linear_matches_numpy(M_, K, N):
    x = rng(1).standard_normal((M_, K))
    w = bf16_matrix((N, K), 2)
    y = M.linear(x, w)
    ref = x @ M.widen(w).T
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_linear_row_independent_of_batch():
    x = rng(3).standard_normal((7, 96))
    w = bf16_matrix((11, 96), 4)
    full = M.linear(x, w)
    for i in range(7):
        assert np.array_equal(M.linear(x[i:i + 1], w)[0], full[i])


def test_rmsnorm_properties():
    x = rng(5).standard_normal((4, 64)) * 3.0
    ones = synth.ones_bf16(64)
    y = M.rmsnorm(x, ones, 0.0)
    assert np.allclose(np.mean(y * y, axis=1), 1.0, atol=1e-12)
    # scale invariance (eps = 0) and direction preserved
    assert np.allclose(M.rmsnorm(7.5 * x, ones, 0.0), y, atol=1e-12)
    assert np.allclose(y / np.linalg.norm(y, axis=1, keepdims=True),
                       x / np.linalg.norm(x, axis=1, keepdims=True), atol=1e-12)
    # the gain multiplies feature-wise
    g = synth.f32_to_bf16(np.linspace(0.5, 2.0, 64).astype(np.float32))
    assert np.allclose(M.rmsnorm(x, g, 0.0), y * M.widen(g), atol=1e-12)
    # eps enters as mean(x^2) + eps
    eps = 0.25
    z = np.full((1, 64), 0.5)
    assert np.allclose(M.rmsnorm(z, ones, eps), 0.5 / np.sqrt(0.25 + eps))


def test_rope_is_complex_rotation():
    H, hd, theta = 3, 16, 1e4
    x = rng(6).standard_normal((5, H * hd))
    pos = np.array([0, 1, 7, 100, 4097], dtype=np.int32)
    y = M.rope(x.copy(), pos, H, hd, theta)
    half = hd // 2
    # rotate-half pairs (i, i+half) as complex numbers times exp(i * pos * f_i)
    f = theta ** (-np.arange(half) * 2.0 / hd)
    for m in range(5):
        for h in range(H):
            seg = x[m, h * hd:(h + 1) * hd]
            z = (seg[:half] + 1j * seg[half:]) * np.exp(1j * pos[m] * f)
            out = y[m, h * hd:(h + 1) * hd]
            assert np.allclose(out[:half], z.real, atol=1e-12)
            assert np.allclose(out[half:], z.imag, atol=1e-12)
    assert np.array_equal(y[0], x[0])  # position 0 is the identity


def test_rope_relative_positions():
    hd = 32
    q = rng(7).standard_normal((1, hd))
    k = rng(8).standard_normal((1, hd))

    def dot(pq, pk):
        a = M.rope(q.copy(), np.array([pq], dtype=np.int32), 1, hd, 1e4)
        b = M.rope(k.copy(), np.array([pk], dtype=np.int32), 1, hd, 1e4)
        return (a @ b.T).item()
    assert np.isclose(dot(10, 3), dot(110, 103), atol=1e-10)
    assert np.isclose(dot(5, 5), (q @ k.T).item(), atol=1e-10)


def test_silu_mul_matches_scipy():
    g = rng(9).standard_normal(1000) * 4
    u = rng(10).standard_normal(1000)
    assert np.allclose(M.silu_mul(g, u), g * expit(g) * u, rtol=1e-13, atol=1e-15)


def _sdpa(q, kc, vc, mask, H, KV, hd):
    """torch scaled_dot_product_attention with a boolean visibility mask."""
    Mq = q.shape[0]
    S = mask.shape[1]
    tq = torch.from_numpy(q.reshape(Mq, H, hd).transpose(1, 0, 2).copy())
    tk = torch.from_numpy(kc[:S].transpose(1, 0, 2).copy()).repeat_interleave(H // KV, 0)
    tv = torch.from_numpy(vc[:S].transpose(1, 0, 2).copy()).repeat_interleave(H // KV, 0)
    o = torch.nn.functional.scaled_dot_product_attention(
        tq, tk, tv, attn_mask=torch.from_numpy(mask)[None])
    return o.numpy().transpose(1, 0, 2).reshape(Mq, H * hd)


@pytest.mark.parametrize("H,KV", [(4, 4), (4, 2), (6, 1)])
def test_attention_causal_matches_sdpa(H, KV):
    hd, L, R = 16, 9, 6
    S = L + R + 3
    kc = rng(11).standard_normal((S, KV, hd))
    vc = rng(12).standard_normal((S, KV, hd))
    kc[L + R:] = np.nan  # slack never read
    vc[L + R:] = np.nan
    q = rng(13).standard_normal((R, H * hd))
    o = M.attention(q, kc, vc, L, R, None, H, KV, hd)
    mask = np.zeros((R, L + R), dtype=bool)
    mask[:, :L] = True
    for i in range(R):
        mask[i, L:L + i + 1] = True
    assert np.allclose(o, _sdpa(q, kc, vc, mask, H, KV, hd), atol=1e-12)


def test_attention_tree_mask_matches_sdpa():
    H, KV, hd, L, R = 4, 2, 8, 5, 7
    kc = rng(14).standard_normal((L + R, KV, hd))
    vc = rng(15).standard_normal((L + R, KV, hd))
    q = rng(16).standard_normal((3, H * hd))
    anc = np.array([0b1, 0b1000101, 0b0110011], dtype=np.uint64)
    o = M.attention(q, kc, vc, L, R, anc, H, KV, hd)
    mask = np.zeros((3, L + R), dtype=bool)
    mask[:, :L] = True
    for i in range(3):
        for j in range(R):
            mask[i, L + j] = bool((int(anc[i]) >> j) & 1)
    assert np.allclose(o, _sdpa(q, kc, vc, mask, H, KV, hd), atol=1e-12)


def test_attention_special_cases():
    H = KV = 1
    hd, L = 4, 6
    vc = rng(17).standard_normal((L, 1, hd))
    # identical keys -> uniform average of the values
    kc = np.tile(rng(18).standard_normal((1, 1, hd)), (L, 1, 1))
    q = rng(19).standard_normal((1, hd))
    o = M.attention(q, kc, vc, L - 1, 1, None, H, KV, hd)
    assert np.allclose(o[0], vc[:, 0].mean(axis=0), atol=1e-12)
    # one dominant key -> its value
    kc = np.zeros((L, 1, hd))
    kc[3, 0, 0] = 1000.0
    q = np.zeros((1, hd)); q[0, 0] = 1.0
    o = M.attention(q, kc, vc, L - 1, 1, None, H, KV, hd)
    assert np.allclose(o[0], vc[3, 0], atol=1e-12)
