"""GPU parity of the draft-head training step (Sec. 4.2) through the C ABI,
against the float64 training oracle (oracle/train.py) on the same seeded
weights and sequences.

Tolerances: the loss within 1e-2 relative; every parameter's gradient within
2e-2 of that parameter's largest oracle gradient (the target features the
GPU trains on come from its bf16-weight target forward, as in every other
parity test); the AdamW update against its closed form from the GPU's own
gradients within float32 rounding; after an update the decoder drafts with
the new weights (its draft tree against the oracle's on the bf16-rounded
master weights).
"""
import dataclasses

import numpy as np
import pytest

import synth
from synth.configs import TINY, WIDE
from oracle import model as M
from oracle import msd as O
from oracle import train as TR
from parity import compare_static_tree, oracle_draft_static

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

WIDE_SHORT = dataclasses.replace(WIDE, n_visual=24, n_text=16)


def f32_to_bf16_bits(x):
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def make(wl, max_batch=1):
    from paper_2505_14260_amd.msd import Engine
    dims = wl.dims
    w = synth.make_target_weights(dims, wl.seed)
    dr = synth.make_draft_weights(dims, w, wl.seed, "random")
    eng = Engine(dims, w, dr, max_batch=max_batch, max_seq=256, max_tree=64,
                 max_prompt=max(wl.prompt_len, 64))
    return eng, O.Models(dims, w, dr), w, dr


def oracle_batch(m, prompts):
    seqs = []
    for tokens, vis, visual in prompts:
        h, e, pt = TR.sequence_inputs(m, tokens, vis, visual)
        seqs.append((h, e, vis, pt))
    return seqs


@pytest.mark.parametrize("wl,visual_input", [(TINY, "embedding"), (WIDE_SHORT, "embedding"),
                                             (TINY, "feature")],
                         ids=["tiny", "wide-gqa", "tiny-visual-feature"])
def test_gradients_match_oracle(wl, visual_input):
    print(f"case: training gradients {wl.name} ({visual_input} input), two sequences", flush=True)
    eng, m, w, dr = make(wl)
    try:
        eng.set_draft_input(visual_input)
        p0 = synth.make_prompt(wl, seq=0)
        p1 = synth.make_prompt(wl, seq=1)
        cut = wl.n_visual + 7
        p1 = (p1[0][:cut], p1[1][:cut], p1[2])
        l0 = eng.train_accumulate(0, *p0)
        l1 = eng.train_accumulate(0, *p1)
        g = eng.train_read(0)
        rows = len(p0[0]) - 1 + len(p1[0]) - 1
        params = TR.draft_params(m.draft)
        loss, reg, cls, gref = TR.batch_grads(m, params, oracle_batch(m, [p0, p1]), visual_input)
        got = (l0[0] + l1[0]) / rows
        print(f"loss {got:.6f} oracle {loss:.6f} (reg {reg:.5f}, token {cls:.5f})")
        assert abs(got - loss) <= 1e-2 * abs(loss)
        assert abs((l0[1] + l1[1]) / rows - reg) <= 1e-2 * abs(reg)
        assert abs((l0[2] + l1[2]) / rows - cls) <= 1e-2 * abs(cls)
        worst = 0.0
        for k in TR.PARAM_KEYS:
            ref = gref[k]
            gg = g[k].astype(np.float64) / rows
            err = np.abs(gg - ref).max() / np.abs(ref).max()
            worst = max(worst, err)
            assert err <= 2e-2, (k, err)
        print(f"gradients: max error {worst:.2e} of each parameter's largest")
    finally:
        eng.close()


def test_update_and_decoder_use_the_trained_draft():
    wl = TINY
    print("case: training update tiny, AdamW closed form, draft tree after the update",
          flush=True)
    eng, m, w, dr = make(wl)
    try:
        prompt = synth.make_prompt(wl)
        eng.train_accumulate(0, *prompt)
        g = eng.train_read(0)
        w0 = eng.train_read(1)
        rows = len(prompt[0]) - 1
        lr = 2e-3
        eng.train_apply(lr)
        w1 = eng.train_read(1)
        for k in TR.PARAM_KEYS:
            gm = g[k].astype(np.float64) / rows
            want = w0[k] - lr * gm / (np.abs(gm) + TR.ADAM_EPS)
            assert np.allclose(w1[k], want, rtol=2e-6, atol=2e-7 * lr / 1e-3), k
        assert all(not np.any(eng.train_read(0)[k]) for k in TR.PARAM_KEYS)  # sums cleared
        # the decoder's draft is the updated one
        dr2 = {"fc": f32_to_bf16_bits(w1["fc"]),
               "layer": dict(dr["layer"], **{k: f32_to_bf16_bits(w1[k])
                                             for k in TR.PARAM_KEYS[1:]})}
        m2 = O.Models(wl.dims, w, dr2)
        from paper_2505_14260_amd.msd import make_static_spec
        parent, rank, _ = synth.static_tree_arrays(wl.tree.paths)
        spec = make_static_spec(parent[1:], rank[1:])
        eng.prefill(0, *prompt)
        trees = eng.new_trees(1)
        eng.draft_tree([0], spec, trees)
        g0 = eng.trees_to_host(trees, 1)[0]
        st, _, _, _ = O.prefill(m2, *prompt, max_slots=256)
        ref, logs, rank_ = oracle_draft_static(m2, st, wl.tree.paths)
        same = compare_static_tree(g0, ref, logs, rank_)
        print(f"draft tree after the update: {same}/{len(ref.token) - 1} tokens equal")
    finally:
        eng.close()


def test_training_lowers_the_loss_on_gpu():
    wl = TINY
    print("case: six training steps tiny", flush=True)
    eng, m, w, dr = make(wl)
    try:
        prompt = synth.make_prompt(wl)
        losses = []
        for step in range(6):
            losses.append(eng.train_accumulate(0, *prompt)[0])
            eng.train_apply(1e-3)
        print("losses", ["%.4f" % x for x in losses])
        assert losses[-1] < losses[0]
    finally:
        eng.close()


def test_training_argument_checks():
    from paper_2505_14260_amd.msd import MSDError
    wl = TINY
    eng, m, w, dr = make(wl)
    try:
        with pytest.raises(MSDError):
            eng.train_apply(1e-3)  # nothing accumulated
        tokens, vis, visual = synth.make_prompt(wl)
        with pytest.raises(MSDError):
            eng.train_accumulate(0, tokens[:1], vis[:1], visual)  # one row: nothing to predict
        bad = tokens.copy()
        bad[-1] = wl.dims.vocab
        with pytest.raises(MSDError):
            eng.train_accumulate(0, bad, vis, visual)
    finally:
        eng.close()
