"""Pins for the draft-head training oracle (CPU only).

Each is checked against something other than the oracle's own code path:
  * its torch decoder layer equals the numpy/C oracle layer used for
    inference (causal rows from slot 0), so the trained draft is the draft
    that decodes;
  * autograd against central finite differences of the loss;
  * the loss assembly (row i against target row i + 1, SmoothL1 with
    beta = 1, the 0.1 cross-entropy weight against the target's full
    distribution, means over features and rows) against a numpy closed form
    on a known draft output;
  * the decoupled input rule (Eq. decouple) against the inference oracle's
    draft_input;
  * AdamW's first step (a step of lr * g / (|g| + eps)), the cosine schedule's
    end points and the progressive mix of Eq. progressive_data.
"""
import dataclasses
import math

import numpy as np
import pytest
from scipy.special import log_softmax as sp_log_softmax

torch = pytest.importorskip("torch")

import synth
from synth.configs import MINI_GQA
from oracle import model as M
from oracle import msd as O
from oracle import train as TR


def setup(mode="random"):
    wl = MINI_GQA
    w = synth.make_target_weights(wl.dims, wl.seed)
    dr = synth.make_draft_weights(wl.dims, w, wl.seed, mode)
    return wl, O.Models(wl.dims, w, dr), synth.make_prompt(wl)


def test_torch_layer_equals_inference_layer():
    wl, m, (tokens, vis, visual) = setup()
    dims = wl.dims
    x = np.random.default_rng(3).standard_normal((17, dims.d_model)) * 0.5
    p = TR.draft_params(m.draft)
    got = TR.layer_forward_t(dims, p, torch.tensor(x), torch.arange(17)).detach().numpy()
    kv = M.KVCache(1, 17, dims.n_kv_heads, dims.head_dim)
    pos = np.arange(17, dtype=np.int32)
    want = M.layer_forward(dims, m.draft["layer"], kv.k[0], kv.v[0], x, pos, pos, 0, 17, None)
    assert np.allclose(got, want, rtol=1e-11, atol=1e-12)


def test_gradients_match_finite_differences():
    wl, m, prompt = setup()
    seq = TR.sequence_inputs(m, *prompt)
    params = TR.draft_params(m.draft)
    loss, _, _, g = TR.batch_grads(m, params, [seq[:2] + (prompt[1], seq[2])])
    rng = np.random.default_rng(7)
    for k in TR.PARAM_KEYS:
        t = params[k]
        for _ in range(3):
            idx = tuple(int(rng.integers(0, s)) for s in t.shape)
            eps = 1e-6
            batch = [seq[:2] + (prompt[1], seq[2])]
            with torch.no_grad():
                old = t[idx].item()
                t[idx] = old + eps
                lp = TR.batch_loss(m, params, batch)
                t[idx] = old - eps
                lm = TR.batch_loss(m, params, batch)
                t[idx] = old
            fd = (lp - lm) / (2 * eps)
            assert abs(fd - g[k][idx]) <= 1e-6 * max(1.0, abs(fd)) + 1e-9, (k, idx, fd, g[k][idx])


def test_loss_assembly_closed_form():
    wl, m, (tokens, vis, visual) = setup()
    h, e, pt = TR.sequence_inputs(m, tokens, vis, visual)
    n, d = h.shape
    rng = np.random.default_rng(11)
    D = h[1:] + rng.standard_normal((n - 1, d)) * rng.choice([0.1, 3.0], size=(n - 1, d))
    lm = torch.tensor(M.widen(m.w["lm_head"]))
    reg, cls = TR.row_losses(torch.tensor(D), torch.tensor(h), pt, lm)
    delta = D - h[1:]
    sl1 = np.where(np.abs(delta) < 1, 0.5 * delta ** 2, np.abs(delta) - 0.5)
    reg_want = sl1.mean(axis=1).sum()
    logits = D @ M.widen(m.w["lm_head"]).T
    cls_want = -(pt[1:] * sp_log_softmax(logits, axis=1)).sum()
    assert abs(float(reg) - reg_want) <= 1e-10 * reg_want
    assert abs(float(cls) - cls_want) <= 1e-10 * cls_want
    # a one-hot target distribution reduces the token term to -log p(label)
    lab = rng.integers(0, wl.dims.vocab, size=n)
    onehot = np.zeros_like(pt)
    onehot[np.arange(n), lab] = 1.0
    _, c1 = TR.row_losses(torch.tensor(D), torch.tensor(h), onehot, lm)
    want = -sp_log_softmax(logits, axis=1)[np.arange(n - 1), lab[1:]].sum()
    assert abs(float(c1) - want) <= 1e-10 * want
    # the draft exactly on the targets leaves only the token term
    r0, _ = TR.row_losses(torch.tensor(h[1:]), torch.tensor(h), pt, lm)
    assert float(r0) == 0.0


def test_batch_loss_weights_and_means():
    # loss = mean over every row of the batch of (reg_i + 0.1 cls_i)
    wl, m, prompt = setup()
    seq = TR.sequence_inputs(m, *prompt)
    p2 = synth.make_prompt(wl, seq=1)
    cut = wl.n_visual + 5
    p2 = (p2[0][:cut], p2[1][:cut], p2[2])
    seq2 = TR.sequence_inputs(m, *p2)
    params = TR.draft_params(m.draft)
    lm = torch.tensor(M.widen(m.w["lm_head"]))
    batch = [seq[:2] + (prompt[1], seq[2]), seq2[:2] + (p2[1], seq2[2])]
    want, rows = 0.0, 0
    for h, e, vis, pt in batch:
        hh, ee = torch.tensor(h), torch.tensor(e)
        d = TR.layer_forward_t(wl.dims, params, TR.draft_inputs(params, hh, ee, vis),
                               torch.arange(len(h) - 1))
        r, c = TR.row_losses(d, hh, pt, lm)
        want += float(r) + 0.1 * float(c)
        rows += len(h) - 1
    got = TR.batch_loss(m, params, batch)
    assert rows == len(prompt[0]) - 1 + cut - 1
    assert abs(got - want / rows) <= 1e-12 * abs(got)


@pytest.mark.parametrize("visual_input", ["embedding", "feature"])
def test_draft_inputs_follow_decoupled_rule(visual_input):
    wl, m, (tokens, vis, visual) = setup()
    h, e, pt = TR.sequence_inputs(m, tokens, vis, visual)
    x = TR.draft_inputs(TR.draft_params(m.draft), torch.tensor(h), torch.tensor(e), vis,
                        visual_input)
    n = len(tokens)
    v = np.asarray(vis, dtype=bool)[:n - 1]
    src = e[:n - 1] if visual_input == "embedding" else h[:n - 1]
    want = M.draft_input(m.draft, h[:n - 1], e[1:], v, src)
    assert np.allclose(x.detach().numpy(), want, rtol=1e-12, atol=1e-14)
    assert v.any() and (~v).any()


def test_adamw_first_step_and_schedule():
    rng = np.random.default_rng(5)
    vals = {"a": rng.standard_normal((4, 3)), "b": rng.standard_normal(6)}
    g = {k: rng.standard_normal(v.shape) for k, v in vals.items()}
    before = {k: v.copy() for k, v in vals.items()}
    opt = TR.AdamW(vals)
    opt.step(vals, g, 1e-3)
    for k in vals:
        want = before[k] - 1e-3 * g[k] / (np.abs(g[k]) + TR.ADAM_EPS)
        assert np.allclose(vals[k], want, rtol=1e-12, atol=1e-15)
    assert TR.cosine_lr(0, 100, 5e-5) == 5e-5
    assert abs(TR.cosine_lr(50, 100, 5e-5) - 2.5e-5) < 1e-18
    assert abs(TR.cosine_lr(100, 100, 5e-5)) < 1e-18


@pytest.mark.parametrize("T", [4, 5, 20])
def test_progressive_mix_counts(T):
    # Eq. progressive_data: epoch t holds (T - t)/T text and t/T visual samples
    assert TR.progressive_counts(0, T, 40) == (40, 0)
    assert TR.progressive_counts(T, T, 40) == (0, 40)
    for t in range(T + 1):
        nt, nv = TR.progressive_counts(t, T, 40)
        assert nt + nv == 40 and abs(nv - 40 * t / T) <= 0.5
        if t:
            assert nv >= TR.progressive_counts(t - 1, T, 40)[1]


def test_training_lowers_the_loss():
    wl, m, prompt = setup()
    seq = TR.sequence_inputs(m, *prompt)
    batch = [seq[:2] + (prompt[1], seq[2])]
    params = TR.draft_params(m.draft)
    vals = {k: t.detach().numpy().copy() for k, t in params.items()}
    opt = TR.AdamW(vals)
    first = None
    for step in range(6):
        for k, t in params.items():
            with torch.no_grad():
                t.copy_(torch.tensor(vals[k]))
        loss, _, _, g = TR.batch_grads(m, params, batch)
        first = loss if first is None else first
        opt.step(vals, g, 1e-3)
    assert loss < first
