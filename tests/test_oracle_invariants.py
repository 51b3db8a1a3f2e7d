"""Invariants the paper's method fixes, checked on the oracle (CPU).

* Tree-structured attention (Sec. 3.2): every tree node sees exactly its
  ancestors, so the tree-masked verification equals a plain causal forward
  of each root-to-node branch.
* Speculative decoding is lossless: at temperature 0 MSD emits exactly the
  target's plain greedy sequence, whatever the draft proposes.
* Decoupled draft input (Eq. decouple): text rows use f_down(Concat(h, e_next))
  (the feature-level form of Eq. concat); visual rows use the visual
  embedding itself and never touch f_down.  In the Visual Feature variant
  of the input-decoupling ablation (Sec. 5.3) they use the target's feature
  of the row instead, still without f_down.
"""
import numpy as np
import pytest

import synth
from synth.configs import MINI_GQA, TINY, TreeShape, chain_paths
from oracle import model as M
from oracle import msd as O


def setup(wl, mode="hidden"):
    dims = wl.dims
    w = synth.make_target_weights(dims, wl.seed)
    dr = synth.make_draft_weights(dims, w, wl.seed, mode)
    return O.Models(dims, w, dr), synth.make_prompt(wl)


SHAPES = {
    "static": lambda wl: wl.tree,
    "dynamic": lambda wl: TreeShape("dynamic", 4, topk=3, n_nodes=12),
    "chain": lambda wl: TreeShape("static", 4, tuple(chain_paths(4))),
}


def arrays(shape):
    return synth.static_tree_arrays(shape.paths) if shape.kind == "static" else None


@pytest.mark.parametrize("wl", [MINI_GQA, TINY], ids=lambda w: w.name)
@pytest.mark.parametrize("kind", ["static", "dynamic"])
def test_tree_forward_equals_branch_forwards(wl, kind):
    m, prompt = setup(wl)
    shape = SHAPES[kind](wl)
    st, first, _, _ = O.prefill(m, *prompt, max_slots=wl.prompt_len + 80)
    for cycle in range(3):
        tree = O.draft_tree(m, st, shape, arrays(shape))
        kv0 = st.kv.copy()
        h, logits = O.verify(m, st, tree)
        for leaf in range(tree.n):
            path = []
            u = leaf
            while u >= 0:
                path.append(u)
                u = int(tree.parent[u])
            path.reverse()
            kv = kv0.copy()
            x = M.embed_rows(m.w, tree.token[path])
            pos = np.arange(st.L, st.L + len(path), dtype=np.int32)
            hb, lb = M.target_forward(m.dims, m.w, kv, x, pos, pos, st.L, len(path), None)
            assert np.array_equal(hb, h[path]), (cycle, leaf)
            assert np.array_equal(lb, logits[path]), (cycle, leaf)
        amax = np.argmax(logits, axis=1)
        O.accept_and_compact(m, st, tree, h, amax)


@pytest.mark.parametrize("wl", [MINI_GQA, TINY], ids=lambda w: w.name)
@pytest.mark.parametrize("kind", ["static", "dynamic", "chain"])
@pytest.mark.parametrize("mode", ["hidden", "embedding", "random"])
def test_speculative_equals_greedy(wl, kind, mode):
    m, prompt = setup(wl, mode)
    shape = SHAPES[kind](wl)
    ref = O.greedy_generate(m, prompt, wl.new_tokens)
    out, cycles = O.msd_generate(m, prompt, shape, wl.new_tokens, arrays(shape))
    assert out == ref
    assert len(out) == wl.new_tokens
    assert all(1 <= len(c["emitted"]) <= shape.depth + 1 for c in cycles)


@pytest.mark.parametrize("kind", ["static", "dynamic"])
def test_speculative_equals_greedy_visual_feature_input(kind):
    # the draft's input rule changes what it proposes, never what is emitted
    wl = TINY
    m, prompt = setup(wl, "hidden")
    shape = SHAPES[kind](wl)
    ref = O.greedy_generate(m, prompt, wl.new_tokens)
    out, cycles = O.msd_generate(m, prompt, shape, wl.new_tokens, arrays(shape),
                                 visual_input="feature")
    assert out == ref
    assert len(out) == wl.new_tokens
    assert all(1 <= len(c["emitted"]) <= shape.depth + 1 for c in cycles)


def test_speculative_accepts_something():
    # with the pass-through draft init, acceptance on the tiny model is nonzero,
    # so compaction with k > 0 is exercised by the losslessness test above
    m, prompt = setup(TINY, "hidden")
    _, cycles = O.msd_generate(m, prompt, TINY.tree, TINY.new_tokens, arrays(TINY.tree))
    assert max(c["n_accepted"] for c in cycles) >= 2


def test_all_text_prompt_matches_feature_level_baseline():
    wl = TINY
    m, _ = setup(wl, "random")
    tokens = synth.ids(20, wl.seed, synth.TID_TEST, wl.dims.vocab)
    st, first, h, _ = O.prefill(m, tokens, np.zeros(20, np.uint8), None, 64)
    # Eq. concat: f_i = f_down(Concat(h_i, e_{i+1})) for every row
    e = M.widen(m.w["embed"][np.append(tokens[1:], first)])
    ref = np.concatenate([h, e], axis=1) @ M.widen(m.draft["fc"]).T
    hh = np.stack([p.h for p in st.pending])
    en = np.stack([p.e_next for p in st.pending])
    f = M.draft_input(m.draft, hh, en, np.zeros(20, bool), None)
    assert np.allclose(f, ref, rtol=1e-12, atol=1e-14)


def test_visual_rows_bypass_fdown():
    wl = TINY
    m, prompt = setup(wl, "random")
    st, _, _, _ = O.prefill(m, *prompt, max_slots=wl.prompt_len + 8)
    rows = st.pending
    assert [p.is_visual for p in rows] == [bool(v) for v in prompt[1]]
    poisoned = dict(m.draft)
    poisoned["fc"] = np.full_like(m.draft["fc"], 0x7FC0)  # NaN everywhere
    d = wl.dims.d_model
    vis = np.array([p.is_visual for p in rows])
    hh = np.stack([p.h if p.h is not None else np.zeros(d) for p in rows])
    en = np.stack([p.e_next if p.e_next is not None else np.zeros(d) for p in rows])
    ev = np.stack([p.e_visual if p.e_visual is not None else np.zeros(d) for p in rows])
    f = M.draft_input(poisoned, hh, en, vis, ev)
    assert np.array_equal(f[vis], M.widen(prompt[2]))     # bit-exact e_v
    assert np.isnan(f[~vis]).all()                        # text rows went through f_down
    # the text row just before the first text token's successor: e_{i+1} of the
    # last visual row's predecessor is not needed; the last text row's next
    # embedding is the first generated token's
    assert not rows[-1].is_visual


def test_visual_feature_rows_are_target_features():
    wl = TINY
    m, prompt = setup(wl, "random")
    st, _, h, _ = O.prefill(m, *prompt, max_slots=wl.prompt_len + 8, visual_input="feature")
    emb, _, _, _ = O.prefill(m, *prompt, max_slots=wl.prompt_len + 8)
    vis = np.array([p.is_visual for p in st.pending])
    assert vis.any() and (~vis).any()
    ev = np.stack([p.e_visual for p in np.array(st.pending)[vis]])
    assert np.array_equal(ev, h[vis])                     # bit-exact h_v
    assert not np.array_equal(ev, M.widen(prompt[2]))     # not the embedding
    for a, b in zip(st.pending, emb.pending):             # text rows unchanged
        if not a.is_visual:
            assert np.array_equal(a.h, b.h) and np.array_equal(a.e_next, b.e_next)
    with pytest.raises(ValueError):
        O.prefill(m, *prompt, max_slots=wl.prompt_len + 8, visual_input="concat")


def test_prompt_must_end_in_text():
    m, (tokens, is_visual, visual) = setup(MINI_GQA)
    with pytest.raises(ValueError):
        O.prefill(m, tokens[:MINI_GQA.n_visual], is_visual[:MINI_GQA.n_visual], visual, 64)
