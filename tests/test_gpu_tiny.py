"""GPU parity on the tiny Llama-style workload (4 layers, d=256, vocab 4096):
the HIP path through the C ABI against the float64 oracle on the same seeded
weights and prompt.

Tolerances (see tests/parity.py): logits and KV within 2e-2 of the row's
max magnitude; tokens identical wherever the oracle's margin exceeds that;
tree structure, accepted paths and slot maps bit-exact.
"""
import ctypes

import numpy as np
import pytest

import synth
from synth.configs import MAXW, TINY, WIDE, TreeShape, chain_paths
from oracle import model as M
from oracle import msd as O
from parity import (argmax_ok, compare_dynamic_tree, compare_static_tree,
                    oracle_draft_dynamic, oracle_draft_static, row_close, sampling_agrees)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def bits_to_f64(t):
    """int16 tensor of bf16 bits -> float64 numpy."""
    a = t.cpu().numpy().astype(np.int16).view(np.uint16)
    return M.widen(a)


@pytest.fixture(scope="module")
def setup():
    from paper_2505_14260_amd.msd import Engine
    wl = TINY
    dims = wl.dims
    w = synth.make_target_weights(dims, wl.seed)
    dr = synth.make_draft_weights(dims, w, wl.seed, wl.draft_fc_mode)
    prompt = synth.make_prompt(wl)
    eng = Engine(dims, w, dr, max_batch=2, max_seq=256, max_tree=64, max_prompt=128)
    m = O.Models(dims, w, dr)
    yield wl, eng, m, prompt
    eng.close()


def static_spec(paths):
    from paper_2505_14260_amd.msd import make_static_spec
    parent, rank, depth = synth.static_tree_arrays(paths)
    return make_static_spec(parent[1:], rank[1:]), (parent, rank, depth)


def upload_tree(eng, tree: O.Tree):
    from paper_2505_14260_amd.msd import Tree
    t = Tree()
    t.n_nodes = tree.n
    anc = tree.anc
    for i in range(tree.n):
        t.token[i] = int(tree.token[i])
        t.parent[i] = int(tree.parent[i])
        t.depth[i] = int(tree.depth[i])
        t.anc[i] = int(anc[i])
    raw = bytes(t)
    dev = eng.new_trees(1)
    dev.copy_(torch.frombuffer(bytearray(raw), dtype=torch.uint8))
    return dev


def test_prefill_kv_and_first_token(setup):
    wl, eng, m, prompt = setup
    print(f"case: prefill tiny seq 0 n={wl.prompt_len}", flush=True)
    first = eng.prefill(0, *prompt)
    st, f_ref, _, logits = O.prefill(m, *prompt, max_slots=256)
    assert argmax_ok(first, logits[-1]), (first, f_ref)
    n = wl.prompt_len
    tk, tv, dk, dv = eng.kv_views()
    torch.cuda.synchronize()
    for l in range(wl.dims.n_layers):
        kg = bits_to_f64(tk[l, 0, :, :n, :].permute(1, 0, 2).reshape(n, -1))
        vg = bits_to_f64(tv[l, 0, :, :, :n].permute(2, 0, 1).reshape(n, -1))
        ok, err = row_close(kg, st.kv.k[l, :n].reshape(n, -1))
        assert ok, (l, "K", err)
        ok, err = row_close(vg, st.kv.v[l, :n].reshape(n, -1))
        assert ok, (l, "V", err)
    # draft cache after the draft has consumed the prompt (Eq. decouple inputs)
    O.draft_catch_up(m, st)
    kg = bits_to_f64(dk[0, 0, :, :n, :].permute(1, 0, 2).reshape(n, -1))
    ok, err = row_close(kg, st.dkv.k[0, :n].reshape(n, -1))
    assert ok, ("draft K", err)


@pytest.mark.parametrize("n_visual", [136, 256, 480, 1036])
def test_prefill_many_rows_wide(n_visual):
    """200-, 320-, 544- and 1100-row prompts through the rocBLAS path (single
    hi+lo products of 400, 640 and 1088 rows; 1100 rows = one 1024-row
    launch of two products plus a 76-row one; an odd FFN tile count and a
    partial last K block of the packed layout): every layer's K/V, the first
    token and the draft cache against the oracle."""
    import dataclasses
    from paper_2505_14260_amd.msd import Engine
    wl = dataclasses.replace(WIDE, n_visual=n_visual)
    dims = wl.dims
    print(f"case: prefill {wl.name} n={wl.prompt_len}", flush=True)
    w = synth.make_target_weights(dims, wl.seed)
    dr = synth.make_draft_weights(dims, w, wl.seed, wl.draft_fc_mode)
    prompt = synth.make_prompt(wl)
    m = O.Models(dims, w, dr)
    max_seq = (wl.prompt_len + 64 + 255) // 256 * 256
    eng = Engine(dims, w, dr, max_batch=1, max_seq=max_seq, max_tree=64, max_prompt=wl.prompt_len)
    try:
        first = eng.prefill(0, *prompt)
        st, f_ref, _, logits = O.prefill(m, *prompt, max_slots=max_seq)
        assert argmax_ok(first, logits[-1]), (first, f_ref)
        n = wl.prompt_len
        tk, tv, dk, dv = eng.kv_views()
        torch.cuda.synchronize()
        worst = 0.0
        for l in range(dims.n_layers):
            kg = bits_to_f64(tk[l, 0, :, :n, :].permute(1, 0, 2).reshape(n, -1))
            vg = bits_to_f64(tv[l, 0, :, :, :n].permute(2, 0, 1).reshape(n, -1))
            ok, err = row_close(kg, st.kv.k[l, :n].reshape(n, -1))
            assert ok, (l, "K", err)
            ok2, err2 = row_close(vg, st.kv.v[l, :n].reshape(n, -1))
            assert ok2, (l, "V", err2)
            worst = max(worst, err, err2)
        O.draft_catch_up(m, st)
        kg = bits_to_f64(dk[0, 0, :, :n, :].permute(1, 0, 2).reshape(n, -1))
        ok, err = row_close(kg, st.dkv.k[0, :n].reshape(n, -1))
        assert ok, ("draft K", err)
        print(f"target K/V max rel err {worst:.2e}, draft K {err:.2e}")
    finally:
        eng.close()


def test_prefill_caller_row_major_weights():
    """msd_use_caller_weights: a 1100-row prompt (one 1024-row rocBLAS pass
    plus a 76-row one) whose output, gate, up and down products read the
    uploaded row-major matrices: every layer's K/V, the first token and the
    draft cache against the oracle, and the K/V bit for bit against the
    default (unpacking) engine's, before and after switching back."""
    import dataclasses
    from paper_2505_14260_amd.msd import Engine
    wl = dataclasses.replace(WIDE, n_visual=1036)
    dims = wl.dims
    print(f"case: prefill on caller weights {wl.name} n={wl.prompt_len}", flush=True)
    w = synth.make_target_weights(dims, wl.seed)
    dr = synth.make_draft_weights(dims, w, wl.seed, wl.draft_fc_mode)
    prompt = synth.make_prompt(wl)
    m = O.Models(dims, w, dr)
    n = wl.prompt_len
    max_seq = (n + 64 + 255) // 256 * 256
    st, f_ref, _, logits = O.prefill(m, *prompt, max_slots=max_seq)
    O.draft_catch_up(m, st)
    engines = [Engine(dims, w, dr, max_batch=1, max_seq=max_seq, max_tree=64, max_prompt=n)
               for _ in range(2)]
    try:
        engines[1].use_caller_weights(True)
        firsts = [e.prefill(0, *prompt) for e in engines]
        torch.cuda.synchronize()
        assert argmax_ok(firsts[1], logits[-1]), (firsts, f_ref)
        assert firsts[1] == firsts[0]
        views = [e.kv_views() for e in engines]
        worst = 0.0
        for l in range(dims.n_layers):
            for which in ("K", "V"):
                got = []
                for tk, tv, _, _ in views:
                    if which == "K":
                        got.append(bits_to_f64(tk[l, 0, :, :n, :].permute(1, 0, 2).reshape(n, -1)))
                    else:
                        got.append(bits_to_f64(tv[l, 0, :, :, :n].permute(2, 0, 1).reshape(n, -1)))
                ref = (st.kv.k if which == "K" else st.kv.v)[l, :n].reshape(n, -1)
                ok, err = row_close(got[1], ref)
                assert ok, (l, which, err)
                assert np.array_equal(got[1], got[0]), (l, which, "differs from the unpacking path")
                worst = max(worst, err)
        dk = views[1][2]
        kg = bits_to_f64(dk[0, 0, :, :n, :].permute(1, 0, 2).reshape(n, -1))
        ok, err = row_close(kg, st.dkv.k[0, :n].reshape(n, -1))
        assert ok, ("draft K", err)
        print(f"caller weights: target K/V max rel err {worst:.2e}, draft K {err:.2e}")
        # back to unpacking: the same prompt again gives the default engine's
        # cache bit for bit
        engines[1].use_caller_weights(False)
        assert engines[1].prefill(0, *prompt) == firsts[0]
        torch.cuda.synchronize()
        tk0, tk1 = views[0][0], views[1][0]
        assert torch.equal(tk0[:, 0, :, :n, :], tk1[:, 0, :, :n, :])
    finally:
        for e in engines:
            e.close()


def test_wide_vocab_lm_head_full_k():
    """A 152,064-word vocabulary at d_model 1024: three sequences' 15-node
    trees make a 45-row verify whose LM head takes the full-K GEMM (ten
    tiles per workgroup, X restaged for each of two K chunks, one partial per
    tile); its logits and argmax against the oracle on the GPU's trees."""
    import dataclasses
    from paper_2505_14260_amd.msd import Engine
    from parity import oracle_tree_of
    wl = dataclasses.replace(WIDE, dims=dataclasses.replace(WIDE.dims, vocab=152064),
                             n_visual=24, n_text=12)
    dims = wl.dims
    print(f"case: verify {wl.name} vocab {dims.vocab}, batch 3", flush=True)
    w = synth.make_target_weights(dims, wl.seed)
    dr = synth.make_draft_weights(dims, w, wl.seed, wl.draft_fc_mode)
    prompts = [synth.make_prompt(wl, seq=b) for b in range(3)]
    m = O.Models(dims, w, dr)
    spec, _ = static_spec(wl.tree.paths)
    T = spec.n_nodes + 1
    max_seq = 256
    eng = Engine(dims, w, dr, max_batch=3, max_seq=max_seq, max_tree=64,
                 max_prompt=wl.prompt_len)
    try:
        for b in range(3):
            eng.prefill(b, *prompts[b])
        trees = eng.new_trees(3)
        eng.draft_tree([0, 1, 2], spec, trees)
        amax, logits = eng.verify([0, 1, 2], trees, T, want_logits=True)
        torch.cuda.synchronize()
        lg = logits.cpu().numpy().reshape(3, T, -1)
        am = amax.cpu().numpy().reshape(3, T)
        gts = eng.trees_to_host(trees, 3)
        worst = 0.0
        for b in range(3):
            st, _, _, _ = O.prefill(m, *prompts[b], max_slots=max_seq)
            _, lg_ref = O.verify(m, st, oracle_tree_of(gts[b]))
            ok, err = row_close(lg[b], lg_ref)
            assert ok, (b, err)
            for i in range(T):
                assert argmax_ok(am[b, i], lg_ref[i]), (b, i)
            worst = max(worst, err)
        print(f"logits max rel err {worst:.2e}")
    finally:
        eng.close()


@pytest.mark.timeout(240)
def test_prefill_k_sliced_products_max_width():
    """A 224-row prompt at d_model 8192 (one layer, FFN 2048): its rocBLAS
    products take one GEMM over the 448 hi and lo rows, split along K into
    strided batches (the gate+up pair into eight slices, q|k|v and down into
    two, the output into four), on the uploaded row-major weights.  Layer
    0's K/V, the first token and the draft cache (whose text rows carry the
    whole target layer) against the oracle, and bit for bit against an
    engine that unpacks the weights instead."""
    import dataclasses
    from paper_2505_14260_amd.msd import Engine
    wl = dataclasses.replace(MAXW, n_visual=200)
    dims = wl.dims
    n = wl.prompt_len
    print(f"case: {wl.name} prefill of {n} rows, K-sliced rocBLAS products", flush=True)
    w = synth.make_target_weights(dims, wl.seed)
    dr = synth.make_draft_weights(dims, w, wl.seed, wl.draft_fc_mode)
    prompt = synth.make_prompt(wl)
    m = O.Models(dims, w, dr)
    max_seq = 512
    st, f_ref, _, logits = O.prefill(m, *prompt, max_slots=max_seq)
    O.draft_catch_up(m, st)
    engines = [Engine(dims, w, dr, max_batch=1, max_seq=max_seq, max_tree=64, max_prompt=n)
               for _ in range(2)]
    try:
        engines[1].use_caller_weights(True)
        firsts = [e.prefill(0, *prompt) for e in engines]
        torch.cuda.synchronize()
        assert argmax_ok(firsts[1], logits[-1]), (firsts, f_ref)
        assert firsts[0] == firsts[1]
        views = [e.kv_views() for e in engines]
        tk, tv, dk, _ = views[1]
        kg = bits_to_f64(tk[0, 0, :, :n, :].permute(1, 0, 2).reshape(n, -1))
        vg = bits_to_f64(tv[0, 0, :, :, :n].permute(2, 0, 1).reshape(n, -1))
        ok, ek = row_close(kg, st.kv.k[0, :n].reshape(n, -1))
        ok2, ev = row_close(vg, st.kv.v[0, :n].reshape(n, -1))
        assert ok and ok2, (ek, ev)
        dkg = bits_to_f64(dk[0, 0, :, :n, :].permute(1, 0, 2).reshape(n, -1))
        ok3, ed = row_close(dkg, st.dkv.k[0, :n].reshape(n, -1))
        assert ok3, ed
        for a_, b_ in zip(views[0], views[1]):
            assert torch.equal(a_, b_)
        print(f"K-sliced prefill: K/V rel err {ek:.2e} / {ev:.2e}, draft K {ed:.2e}")
    finally:
        for e in engines:
            e.close()


def test_max_width_model():
    """d_model 8192, the library's limit (whole-row kernels at two 16-byte
    units per thread), with 8-way GQA: the prompt forward's K/V, first token
    and draft cache, verification logits on a fixed tree, and a short
    speculative decode against the plain greedy one."""
    from paper_2505_14260_amd.msd import Engine
    wl = MAXW
    dims = wl.dims
    print(f"case: {wl.name} prefill, verify and decode", flush=True)
    w = synth.make_target_weights(dims, wl.seed)
    dr = synth.make_draft_weights(dims, w, wl.seed, wl.draft_fc_mode)
    prompt = synth.make_prompt(wl)
    m = O.Models(dims, w, dr)
    n = wl.prompt_len
    max_seq = 256
    eng = Engine(dims, w, dr, max_batch=1, max_seq=max_seq, max_tree=64, max_prompt=n)
    try:
        first = eng.prefill(0, *prompt)
        st, f_ref, _, logits = O.prefill(m, *prompt, max_slots=max_seq)
        assert argmax_ok(first, logits[-1]), (first, f_ref)
        tk, tv, dk, dv = eng.kv_views()
        torch.cuda.synchronize()
        kg = bits_to_f64(tk[0, 0, :, :n, :].permute(1, 0, 2).reshape(n, -1))
        vg = bits_to_f64(tv[0, 0, :, :, :n].permute(2, 0, 1).reshape(n, -1))
        ok, ek = row_close(kg, st.kv.k[0, :n].reshape(n, -1))
        ok2, ev = row_close(vg, st.kv.v[0, :n].reshape(n, -1))
        assert ok and ok2, (ek, ev)
        O.draft_catch_up(m, st)
        dkg = bits_to_f64(dk[0, 0, :, :n, :].permute(1, 0, 2).reshape(n, -1))
        ok3, ed = row_close(dkg, st.dkv.k[0, :n].reshape(n, -1))
        assert ok3, ed
        parent, rank, depth = synth.static_tree_arrays(wl.tree.paths)
        toks = synth.ids(len(parent), wl.seed, synth.TID_TEST, dims.vocab)
        toks[0] = first
        tree = O.Tree(toks.astype(np.int32), parent, depth, np.zeros(len(parent)))
        dev = upload_tree(eng, tree)
        amax, lg = eng.verify([0], dev, tree.n, want_logits=True)
        _, lg_ref = O.verify(m, st, tree)
        ok4, el = row_close(lg.cpu().numpy(), lg_ref)
        assert ok4, el
        am = amax.cpu().numpy()
        for i in range(tree.n):
            assert argmax_ok(am[i], lg_ref[i]), i
        print(f"K/V max rel err {max(ek, ev):.2e}, draft K {ed:.2e}, logits {el:.2e}")
    finally:
        eng.close()
    eng = Engine(dims, w, dr, max_batch=1, max_seq=max_seq, max_tree=64, max_prompt=n)
    try:
        spec, _ = static_spec(wl.tree.paths)
        out, cycles = eng.generate(0, prompt, spec, wl.new_tokens)
        ref, rows = O.greedy_generate(m, prompt, wl.new_tokens, return_logits=True)
        bad = next((i for i in range(len(ref)) if out[i] != ref[i]), None)
        print(f"decode: {bad if bad is not None else len(ref)}/{len(ref)} tokens equal, "
              f"tau={np.mean(cycles):.2f}")
        if bad is not None:
            assert argmax_ok(out[bad], rows[bad]), (bad, out[bad], ref[bad])
    finally:
        eng.close()


def test_bitwise_deterministic(setup):
    """Two identical runs give bitwise-equal caches, trees and logits (every
    reduction has a fixed order; a race would show here)."""
    import dataclasses
    from paper_2505_14260_amd.msd import Engine
    wl, eng, m, prompt = setup
    print("case: determinism, tiny cycle twice and a 544-row wide prefill twice", flush=True)
    spec, _ = static_spec(wl.tree.paths)
    T = spec.n_nodes + 1
    n = wl.prompt_len
    tk, tv, dk, dv = eng.kv_views()
    trees = eng.new_trees(1)
    runs = []
    for _ in range(2):
        eng.prefill(0, *prompt)
        eng.draft_tree([0], spec, trees)
        amax, logits = eng.verify([0], trees, T, want_logits=True)
        torch.cuda.synchronize()
        runs.append([tk[:, 0, :, :n + T].clone(), tv[:, 0, :, :, :n + T].clone(),
                     dk[:, 0, :, :n].clone(), dv[:, 0, :, :, :n].clone(), trees.clone(),
                     amax.clone(), logits.clone()])
    for a, b in zip(*runs):
        assert torch.equal(a, b)
    wide = dataclasses.replace(WIDE, n_visual=480)
    w = synth.make_target_weights(wide.dims, wide.seed)
    dr = synth.make_draft_weights(wide.dims, w, wide.seed, wide.draft_fc_mode)
    wp = synth.make_prompt(wide)
    e2 = Engine(wide.dims, w, dr, max_batch=1, max_seq=1024, max_tree=64,
                max_prompt=wide.prompt_len)
    try:
        kvs = []
        for _ in range(2):
            first = e2.prefill(0, *wp)
            k2, v2, d2, _ = e2.kv_views()
            torch.cuda.synchronize()
            kvs.append((first, k2[:, 0, :, :wide.prompt_len].clone(),
                        v2[:, 0, :, :, :wide.prompt_len].clone(),
                        d2[:, 0, :, :wide.prompt_len].clone()))
        assert kvs[0][0] == kvs[1][0]
        for a, b in zip(kvs[0][1:], kvs[1][1:]):
            assert torch.equal(a, b)
    finally:
        e2.close()


def test_verify_logits_on_fixed_tree(setup):
    wl, eng, m, prompt = setup
    print("case: verify tiny fixed tree", flush=True)
    eng.prefill(0, *prompt)
    st, first, _, _ = O.prefill(m, *prompt, max_slots=256)
    parent, rank, depth = synth.static_tree_arrays(wl.tree.paths)
    toks = synth.ids(len(parent), wl.seed, synth.TID_TEST, wl.dims.vocab)
    toks[0] = first
    tree = O.Tree(toks.astype(np.int32), parent, depth, np.zeros(len(parent)))
    dev = upload_tree(eng, tree)
    amax, logits = eng.verify([0], dev, tree.n, want_logits=True)
    h_ref, lg_ref = O.verify(m, st, tree)
    lg = logits.cpu().numpy()
    ok, err = row_close(lg, lg_ref)
    print(f"verify logits max rel err {err:.2e}")
    assert ok, err
    am = amax.cpu().numpy()
    for i in range(tree.n):
        assert argmax_ok(am[i], lg_ref[i]), i


def test_accept_compact_bit_exact(setup):
    wl, eng, m, prompt = setup
    print("case: accept/compact tiny synthetic", flush=True)
    eng.prefill(1, *prompt)
    L = wl.prompt_len
    parent, rank, depth = synth.static_tree_arrays(wl.tree.paths)
    T = len(parent)
    rng = np.random.default_rng(7)
    for trial in range(4):
        toks = np.zeros(T, dtype=np.int32)
        for c in range(1, T):
            toks[c] = 100 + c  # siblings distinct
        toks[0] = 5
        tree = O.Tree(toks, parent, depth, np.zeros(T))
        dev = upload_tree(eng, tree)
        eng.verify([1], dev, T)
        # argmax chosen so a random branch is accepted to a random depth
        amax = rng.integers(0, 50, T).astype(np.int32)
        leaf = int(rng.integers(1, T))
        path = []
        u = leaf
        while u > 0:
            path.append(u)
            u = int(parent[u])
        path.reverse()
        stop = int(rng.integers(0, len(path) + 1))
        prev = 0
        for u in path[:stop]:
            amax[prev] = toks[u]
            prev = u
        tk, tv, _, _ = eng.kv_views()
        Lc = eng_len = __import__("paper_2505_14260_amd.msd", fromlist=["x"]).msd_seq_len(eng.ctx, 1)
        kv_bits = torch.from_numpy(rng.integers(-30000, 30000, size=tk[:, 1, :, Lc:Lc + T, :].shape,
                                                dtype=np.int16)).cuda()
        vv_bits = torch.from_numpy(rng.integers(-30000, 30000, size=tv[:, 1, :, :, Lc:Lc + T].shape,
                                                dtype=np.int16)).cuda()
        tk[:, 1, :, Lc:Lc + T, :] = kv_bits
        tv[:, 1, :, :, Lc:Lc + T] = vv_bits
        before_k = tk[:, 1].clone()
        am_dev = torch.from_numpy(amax).cuda()
        em, slots = eng.accept([1], dev, T, am_dev, want_slots=True)
        ref_path, ref_emit = O.greedy_accept(tree, amax)
        assert em[0] == ref_emit
        sl = slots.cpu().numpy()[:len(ref_path)]
        assert list(sl) == [Lc + j for j in ref_path]
        # compaction against an out-of-place copy of the same bits
        k_after = tk[:, 1].cpu().numpy()
        k_before = before_k.cpu().numpy()
        for j, u in enumerate(ref_path):
            assert np.array_equal(k_after[:, :, Lc + j, :], k_before[:, :, Lc + u, :])
        assert np.array_equal(k_after[:, :, :Lc, :], k_before[:, :, :Lc, :])
        v_after = tv[:, 1].cpu().numpy()
        vb = vv_bits.cpu().numpy()
        for j, u in enumerate(ref_path):
            assert np.array_equal(v_after[:, :, :, Lc + j], vb[:, :, :, u])
        assert eng_len + len(ref_path) == __import__(
            "paper_2505_14260_amd.msd", fromlist=["x"]).msd_seq_len(eng.ctx, 1)


@pytest.mark.parametrize("paths", [TINY.tree.paths, tuple(chain_paths(4))], ids=["binary3", "chain4"])
def test_static_draft_tree_matches_oracle(setup, paths):
    wl, eng, m, prompt = setup
    print(f"case: static draft tree tiny {len(paths)} nodes", flush=True)
    eng.prefill(0, *prompt)
    st, first, _, _ = O.prefill(m, *prompt, max_slots=256)
    spec, _ = static_spec(paths)
    dev = eng.new_trees(1)
    eng.draft_tree([0], spec, dev)
    g = eng.trees_to_host(dev, 1)[0]
    ref, logs, rank = oracle_draft_static(m, st, paths)
    checked = compare_static_tree(g, ref, logs, rank)
    print(f"draft tree: {checked}/{ref.n - 1} nodes compared equal")
    assert checked >= (ref.n - 1) // 2


def test_speculative_decode_matches_greedy(setup):
    wl, eng, m, prompt = setup
    print("case: e2e tiny static tree", flush=True)
    spec, _ = static_spec(wl.tree.paths)
    toks, cycles = eng.generate(0, prompt, spec, wl.new_tokens)
    ref, rows = O.greedy_generate(m, prompt, wl.new_tokens, return_logits=True)
    first_bad = next((i for i in range(len(ref)) if toks[i] != ref[i]), None)
    print(f"e2e: {first_bad if first_bad is not None else len(ref)}/{len(ref)} tokens equal; "
          f"tau={np.mean(cycles):.2f}")
    if first_bad is not None:
        assert argmax_ok(toks[first_bad], rows[first_bad]), (first_bad, toks[first_bad],
                                                              ref[first_bad])


def test_visual_feature_draft_input_matches_oracle(setup):
    # the Visual Feature variant of the draft input (Sec. 5.3): visual prompt
    # rows enter the draft as the target's features h_v instead of e_v
    wl, eng, m, prompt = setup
    print("case: visual-feature draft input, tiny", flush=True)
    n = wl.prompt_len
    vis = np.asarray(prompt[1], dtype=bool)
    eng.set_draft_input("feature")
    try:
        eng.prefill(0, *prompt)
        st, _, _, _ = O.prefill(m, *prompt, max_slots=256, visual_input="feature")
        tk, tv, dk, dv = eng.kv_views()
        torch.cuda.synchronize()
        kg = bits_to_f64(dk[0, 0, :, :n, :].permute(1, 0, 2).reshape(n, -1))
        vg = bits_to_f64(dv[0, 0, :, :, :n].permute(2, 0, 1).reshape(n, -1))
        emb, _, _, _ = O.prefill(m, *prompt, max_slots=256)
        O.draft_catch_up(m, emb)
        spec, _ = static_spec(wl.tree.paths)
        ref, logs, rank = oracle_draft_static(m, st, wl.tree.paths)  # catch-up + tree
        ok, err = row_close(kg, st.dkv.k[0, :n].reshape(n, -1))
        assert ok, ("draft K", err)
        ok, err = row_close(vg, st.dkv.v[0, :n].reshape(n, -1))
        assert ok, ("draft V", err)
        # the embedding-input cache differs at the visual rows: the mode took effect
        ok_emb, _ = row_close(kg[vis], emb.dkv.k[0, :n][vis].reshape(int(vis.sum()), -1))
        assert not ok_emb
        dev = eng.new_trees(1)
        eng.draft_tree([0], spec, dev)
        g = eng.trees_to_host(dev, 1)[0]
        checked = compare_static_tree(g, ref, logs, rank)
        print(f"visual-feature draft tree: {checked}/{ref.n - 1} nodes compared equal")
        assert checked >= (ref.n - 1) // 2
        # the emitted tokens are still the target's greedy decode
        toks, cycles = eng.generate(0, prompt, spec, wl.new_tokens)
        want, rows = O.greedy_generate(m, prompt, wl.new_tokens, return_logits=True)
        bad = next((i for i in range(len(want)) if toks[i] != want[i]), None)
        print(f"visual-feature e2e: {bad if bad is not None else len(want)}/{len(want)} "
              f"tokens equal; tau={np.mean(cycles):.2f}")
        if bad is not None:
            assert argmax_ok(toks[bad], rows[bad]), (bad, toks[bad], want[bad])
    finally:
        eng.set_draft_input("embedding")
    from paper_2505_14260_amd import msd as B
    with pytest.raises(B.MSDError):
        B.msd_set_draft_input(eng.ctx, 2)


def test_chain_n_alpha_matches_oracle(setup):
    """Chain drafts (one token per draft forward): the per-cycle accepted
    counts, and so the n-alpha acceptance rates, equal the oracle's MSD loop
    on the same prompt."""
    from oracle import metrics
    wl, eng, m, prompt = setup
    gamma, n_new = 5, 40
    print(f"case: tiny chain drafts, gamma={gamma}, {n_new} tokens", flush=True)
    paths = tuple(chain_paths(gamma))
    spec, arrays = static_spec(paths)
    toks, cycles = eng.generate(0, prompt, spec, n_new)
    ref, recs = O.msd_generate(m, prompt, TreeShape("static", gamma, paths), n_new,
                               static_arrays=arrays, max_slots=256)
    acc_gpu = [c - 1 for c in cycles]
    acc_ref = [r["n_accepted"] for r in recs]
    a_gpu, a_ref = metrics.n_alpha(acc_gpu, gamma), metrics.n_alpha(acc_ref, gamma)
    print("n-alpha gpu   ", [None if a is None else round(a, 3) for a in a_gpu])
    print("n-alpha oracle", [None if a is None else round(a, 3) for a in a_ref])
    assert toks == ref
    assert acc_gpu == acc_ref


def test_dynamic_tree_decode(setup):
    wl, eng, m, prompt = setup
    print("case: e2e tiny dynamic tree", flush=True)
    from paper_2505_14260_amd.msd import make_dynamic_spec
    shape = TreeShape("dynamic", 4, topk=3, n_nodes=12)
    spec = make_dynamic_spec(shape.topk, shape.depth, shape.n_nodes)
    eng.prefill(0, *prompt)
    dev = eng.new_trees(1)
    eng.draft_tree([0], spec, dev)
    g = eng.trees_to_host(dev, 1)[0]
    assert g.n_nodes == 13
    st, _, _, _ = O.prefill(m, *prompt, max_slots=256)
    ref, pool, rows, root_logits = oracle_draft_dynamic(m, st, shape.topk, shape.depth,
                                                        shape.n_nodes)
    same, scored = compare_dynamic_tree(g, pool, rows, root_logits, shape.topk, shape.n_nodes,
                                        ref=ref)
    print(f"dynamic draft tree: {same}/{shape.n_nodes} nodes as the oracle's, {scored} scored, "
          f"{compare_dynamic_tree.exact} compared bit for bit so far")
    for c in range(1, 13):
        assert 0 <= g.parent[c] < c
        assert g.depth[c] == g.depth[g.parent[c]] + 1
        assert g.score[c] <= g.score[g.parent[c]] + 1e-6
        assert int(g.anc[c]) == int(g.anc[g.parent[c]]) | (1 << c)
    for p in range(13):
        kids = [g.token[c] for c in range(1, 13) if g.parent[c] == p]
        assert len(kids) == len(set(kids))
    toks, cycles = eng.generate(0, prompt, spec, wl.new_tokens)
    ref, rows = O.greedy_generate(m, prompt, wl.new_tokens, return_logits=True)
    first_bad = next((i for i in range(len(ref)) if toks[i] != ref[i]), None)
    print(f"e2e dynamic: {first_bad if first_bad is not None else len(ref)}/{len(ref)} equal")
    if first_bad is not None:
        assert argmax_ok(toks[first_bad], rows[first_bad])


def test_errors_and_capacity(setup):
    wl, eng, m, prompt = setup
    from paper_2505_14260_amd import msd as B
    tokens, is_visual, visual = prompt
    with pytest.raises(B.MSDError) as e:
        eng.prefill(0, tokens[:10], is_visual[:10], visual)  # ends in a visual row
    assert e.value.code == B.MSD_ERR_INVALID_ARG
    with pytest.raises(B.MSDError) as e:
        eng.prefill(0, np.zeros(200, np.int32), np.zeros(200, np.uint8), None)
    assert e.value.code == B.MSD_ERR_INVALID_ARG  # beyond max_prompt
    spec, _ = static_spec(wl.tree.paths)
    dev = eng.new_trees(1)
    with pytest.raises(B.MSDError) as e:
        B.msd_accept_compact(eng.ctx, [0], dev.data_ptr(), 15, dev.data_ptr())
    assert e.value.code == B.MSD_ERR_STATE


def test_empty_and_malformed_calls(setup):
    """Empty inputs and malformed argument lists are rejected on the host
    with MSD_ERR_INVALID_ARG before any kernel runs, and the context keeps
    working afterwards (a root-only verify against the oracle)."""
    wl, _, m, prompt = setup
    from paper_2505_14260_amd import msd as B
    print("case: tiny empty and malformed calls", flush=True)
    eng = B.Engine(wl.dims, m.w, m.draft, max_batch=2, max_seq=256, max_tree=64, max_prompt=128)
    try:
        _empty_and_malformed(wl, eng, m, prompt, B)
    finally:
        eng.close()


def _empty_and_malformed(wl, eng, m, prompt, B):
    first = eng.prefill(0, *prompt)
    empty = np.zeros(0, np.int32)
    with pytest.raises(B.MSDError) as e:                       # empty prompt
        eng.prefill(1, empty, np.zeros(0, np.uint8), None)
    assert e.value.code == B.MSD_ERR_INVALID_ARG
    tokens, is_visual, _ = prompt
    bad = tokens.copy()
    bad[-1] = wl.dims.vocab                                     # token id out of range
    with pytest.raises(B.MSDError) as e:
        eng.prefill(1, bad, is_visual, None)
    assert e.value.code == B.MSD_ERR_INVALID_ARG
    with pytest.raises(B.MSDError) as e:                       # visual rows without embeddings
        eng.prefill(1, tokens, is_visual, None)
    assert e.value.code == B.MSD_ERR_INVALID_ARG
    spec, _ = static_spec(wl.tree.paths)
    dev = eng.new_trees(2)
    amax = torch.zeros(2 * 64, dtype=torch.int32, device="cuda")
    for seqs in ([], [0, 0], [5], [-1]):                        # empty, duplicate, out of range
        with pytest.raises(B.MSDError) as e:
            B.msd_draft_tree(eng.ctx, seqs, spec, dev.data_ptr())
        assert e.value.code == B.MSD_ERR_INVALID_ARG, seqs
        with pytest.raises(B.MSDError) as e:
            B.msd_verify(eng.ctx, seqs, dev.data_ptr(), 4, amax.data_ptr())
        assert e.value.code == B.MSD_ERR_INVALID_ARG, seqs
    with pytest.raises(B.MSDError) as e:                       # sequence without a prompt
        B.msd_verify(eng.ctx, [1], dev.data_ptr(), 4, amax.data_ptr())
    assert e.value.code == B.MSD_ERR_STATE
    for T in (0, 65):                                           # tree sizes outside [1, 64]
        with pytest.raises(B.MSDError) as e:
            B.msd_verify(eng.ctx, [0], dev.data_ptr(), T, amax.data_ptr())
        assert e.value.code == B.MSD_ERR_INVALID_ARG, T
    with pytest.raises(B.MSDError) as e:                       # a static tree of no nodes
        B.msd_draft_tree(eng.ctx, [0], B.make_static_spec(np.zeros(0, np.int32),
                                                          np.zeros(0, np.int32)), dev.data_ptr())
    assert e.value.code == B.MSD_ERR_INVALID_ARG
    st, _, _, _ = O.prefill(m, *prompt, max_slots=256)
    tree = O.Tree(np.array([first], np.int32), np.array([-1], np.int32), np.zeros(1, np.int32),
                  np.zeros(1))
    one = upload_tree(eng, tree)
    am, lg = eng.verify([0], one, 1, want_logits=True)
    _, lg_ref = O.verify(m, st, tree)
    ok, err = row_close(lg.cpu().numpy(), lg_ref)
    assert ok, err


def _tree_bytes(tok, par, dep, anc, n_nodes=None):
    from paper_2505_14260_amd.msd import Tree
    t = Tree()
    t.n_nodes = len(tok) if n_nodes is None else n_nodes
    for i in range(len(tok)):
        t.token[i], t.parent[i], t.depth[i], t.anc[i] = int(tok[i]), int(par[i]), int(dep[i]), \
            int(anc[i])
    return bytes(t)


def test_accept_state_and_malformed_trees(setup):
    """Acceptance must follow a verify of the same sequences with nothing in
    between (MSD_ERR_STATE otherwise), and a malformed caller tree makes the
    acceptance return MSD_ERR_INVALID_ARG with no effect on any sequence of
    the call; the decode then continues as the plain greedy decode."""
    wl, _, m, prompt = setup
    from paper_2505_14260_amd import msd as B
    print("case: tiny acceptance state checks and malformed trees", flush=True)
    eng = B.Engine(wl.dims, m.w, m.draft, max_batch=2, max_seq=256, max_tree=64, max_prompt=128)
    try:
        spec, _ = static_spec(wl.tree.paths)
        T = spec.n_nodes + 1
        out = [eng.prefill(0, *prompt)]
        eng.prefill(1, *prompt)
        trees, other = eng.new_trees(1), eng.new_trees(1)

        def expect(code, fn):
            with pytest.raises(B.MSDError) as e:
                fn()
            assert e.value.code == code, (e.value.code, str(e.value))

        eng.draft_tree([0], spec, trees)
        amax, _ = eng.verify([0], trees, T)
        expect(B.MSD_ERR_STATE, lambda: eng.accept([1], trees, T, amax))   # other sequence
        eng.prefill(1, *prompt)                                            # prompt in between
        expect(B.MSD_ERR_STATE, lambda: eng.accept([0], trees, T, amax))
        amax, _ = eng.verify([0], trees, T)
        eng.draft_tree([1], spec, other)                                   # draft in between
        expect(B.MSD_ERR_STATE, lambda: eng.accept([0], trees, T, amax))
        amax, _ = eng.verify([0], trees, T)
        em, _ = eng.accept([0], trees, T, amax)
        out.extend(int(t) for t in em[0])
        expect(B.MSD_ERR_STATE, lambda: eng.accept([0], trees, T, amax))   # accepted twice
        # malformed trees, built from a well-formed one
        par, rank, dep = synth.static_tree_arrays(wl.tree.paths)
        tok = np.arange(100, 100 + T, dtype=np.int32)
        anc = [int(a) for a in O.ancestor_masks(par)]
        bad = []
        p2 = par.copy(); p2[3] = 5                                         # parent after child
        bad.append(("parent order", _tree_bytes(tok, p2, dep, anc)))
        d2 = dep.copy(); d2[4] += 1                                        # depth off by one
        bad.append(("depth", _tree_bytes(tok, par, d2, anc)))
        a2 = list(anc); a2[5] ^= 1 << 2                                    # stray ancestor bit
        bad.append(("ancestor mask", _tree_bytes(tok, par, dep, a2)))
        t2 = tok.copy(); t2[2] = t2[1]                                     # duplicate siblings
        bad.append(("duplicate sibling", _tree_bytes(t2, par, dep, anc)))
        t3 = tok.copy(); t3[6] = wl.dims.vocab                             # id out of range
        bad.append(("token id", _tree_bytes(t3, par, dep, anc)))
        bad.append(("node count", _tree_bytes(tok, par, dep, anc, n_nodes=T - 1)))
        good = _tree_bytes(tok, par, dep, anc)
        for name, raw in bad:
            L0, L1 = B.msd_seq_len(eng.ctx, 0), B.msd_seq_len(eng.ctx, 1)
            dev = eng.new_trees(1)
            dev.copy_(torch.frombuffer(bytearray(raw), dtype=torch.uint8))
            a, _ = eng.verify([0], dev, T)
            expect(B.MSD_ERR_INVALID_ARG, lambda: eng.accept([0], dev, T, a))
            assert B.msd_seq_len(eng.ctx, 0) == L0, name
            # in a batch with a well-formed tree: neither sequence moves
            pair = eng.new_trees(2)
            pair.copy_(torch.frombuffer(bytearray(good + raw), dtype=torch.uint8))
            a, _ = eng.verify([1, 0], pair, T)
            expect(B.MSD_ERR_INVALID_ARG, lambda: eng.accept([1, 0], pair, T, a))
            assert (B.msd_seq_len(eng.ctx, 0), B.msd_seq_len(eng.ctx, 1)) == (L0, L1), name
            print(f"malformed tree ({name}): rejected, lengths unchanged", flush=True)
        # the context keeps decoding sequence 0 as the target's greedy decode
        n_new = 24
        while len(out) < n_new:
            eng.draft_tree([0], spec, trees)
            amax, _ = eng.verify([0], trees, T)
            em, _ = eng.accept([0], trees, T, amax)
            out.extend(int(t) for t in em[0])
        ref, rows = O.greedy_generate(m, prompt, n_new, return_logits=True)
        out = out[:n_new]
        bad_i = next((i for i in range(n_new) if out[i] != ref[i]), None)
        print(f"decode after rejected calls: {bad_i if bad_i is not None else n_new}/{n_new} "
              f"equal", flush=True)
        if bad_i is not None:
            assert argmax_ok(out[bad_i], rows[bad_i]), bad_i
    finally:
        eng.close()


def test_root_only_tree(setup):
    """T = 1: the verify step degenerates to one plain decode step."""
    wl, eng, m, prompt = setup
    print("case: tiny verify with a root-only tree", flush=True)
    first = eng.prefill(0, *prompt)
    st, f_ref, _, _ = O.prefill(m, *prompt, max_slots=256)
    tree = O.Tree(np.array([first], np.int32), np.array([-1], np.int32), np.zeros(1, np.int32),
                  np.zeros(1))
    dev = upload_tree(eng, tree)
    amax, logits = eng.verify([0], dev, 1, want_logits=True)
    _, lg_ref = O.verify(m, st, tree)
    ok, err = row_close(logits.cpu().numpy(), lg_ref)
    assert ok, err
    em, slots = eng.accept([0], dev, 1, amax, want_slots=True)
    assert em[0] == [int(amax.cpu().numpy()[0])]
    assert slots.cpu().numpy()[0] == wl.prompt_len
    assert argmax_ok(em[0][0], lg_ref[0])


def test_max_tree_dynamic_64_nodes(setup):
    """The largest tree (64 nodes incl. the root): draft tree against the
    oracle's selection, verification logits on it, then a short decode."""
    wl, eng, m, prompt = setup
    print("case: tiny dynamic tree K=8 D=4 N=63", flush=True)
    from paper_2505_14260_amd.msd import make_dynamic_spec
    K, D, N = 8, 4, 63
    spec = make_dynamic_spec(K, D, N)
    eng.prefill(0, *prompt)
    st, _, _, _ = O.prefill(m, *prompt, max_slots=256)
    dev = eng.new_trees(1)
    eng.draft_tree([0], spec, dev)
    g = eng.trees_to_host(dev, 1)[0]
    assert g.n_nodes == 64
    ref, pool, rows, root_logits = oracle_draft_dynamic(m, st, K, D, N)
    same, scored = compare_dynamic_tree(g, pool, rows, root_logits, K, N, ref=ref)
    print(f"64-node tree: {same}/{N} nodes as the oracle's, {scored} scored, "
          f"{compare_dynamic_tree.exact} compared bit for bit so far")
    from parity import oracle_tree_of
    tree = oracle_tree_of(g)
    amax, logits = eng.verify([0], dev, 64, want_logits=True)
    _, lg_ref = O.verify(m, st, tree)
    ok, err = row_close(logits.cpu().numpy(), lg_ref)
    assert ok, err
    am = amax.cpu().numpy()
    for i in range(64):
        assert argmax_ok(am[i], lg_ref[i]), i
    eng.accept([0], dev, 64, amax)
    toks, _ = eng.generate(0, prompt, spec, 24)
    ref, rows_g = O.greedy_generate(m, prompt, 24, return_logits=True)
    bad = next((i for i in range(24) if toks[i] != ref[i]), None)
    if bad is not None:
        assert argmax_ok(toks[bad], rows_g[bad]), bad


def test_batch2_ragged_decode(setup):
    """Two sequences of different prompt lengths decoded together, each
    against its own plain greedy decode."""
    wl, eng, m, prompt = setup
    print("case: tiny batch of 2 ragged prompts, static tree", flush=True)
    tokens, is_visual, visual = prompt
    cut = wl.n_visual + 17
    p1 = (tokens[:cut], is_visual[:cut], visual)
    spec, _ = static_spec(wl.tree.paths)
    T = spec.n_nodes + 1
    outs = [[eng.prefill(0, *prompt)], [eng.prefill(1, *p1)]]
    trees = eng.new_trees(2)
    n_new = 40
    while min(len(o) for o in outs) < n_new:
        eng.draft_tree([0, 1], spec, trees)
        amax, _ = eng.verify([0, 1], trees, T)
        em, _ = eng.accept([0, 1], trees, T, amax)
        for b in range(2):
            outs[b].extend(int(t) for t in em[b])
    for b, p in enumerate((prompt, p1)):
        ref, rows = O.greedy_generate(m, p, n_new, return_logits=True)
        got = outs[b][:n_new]
        bad = next((i for i in range(n_new) if got[i] != ref[i]), None)
        print(f"seq {b}: {bad if bad is not None else n_new}/{n_new} equal")
        if bad is not None:
            assert argmax_ok(got[bad], rows[bad]), (b, bad)


def test_sequence_joins_running_batch(setup):
    """A sequence prefilled while another already has pending draft rows: the
    catch-up batch pads the new sequence (which has none), and both decode as
    their plain greedy decodes."""
    wl, eng, m, prompt = setup
    print("case: tiny batch, second sequence joins after two cycles", flush=True)
    tokens, is_visual, visual = prompt
    cut = wl.n_visual + 13
    p1 = (tokens[:cut], is_visual[:cut], visual)
    spec, _ = static_spec(wl.tree.paths)
    T = spec.n_nodes + 1
    outs = [[eng.prefill(0, *prompt)], []]
    one = eng.new_trees(1)
    for _ in range(2):
        eng.draft_tree([0], spec, one)
        amax, _ = eng.verify([0], one, T)
        em, _ = eng.accept([0], one, T, amax)
        outs[0].extend(int(t) for t in em[0])
    outs[1].append(eng.prefill(1, *p1))
    trees = eng.new_trees(2)
    n_new = 24
    while min(len(o) for o in outs) < n_new:
        eng.draft_tree([0, 1], spec, trees)
        amax, _ = eng.verify([0, 1], trees, T)
        em, _ = eng.accept([0, 1], trees, T, amax)
        for b in range(2):
            outs[b].extend(int(t) for t in em[b])
    for b, p in enumerate((prompt, p1)):
        ref, rows = O.greedy_generate(m, p, n_new, return_logits=True)
        got = outs[b][:n_new]
        bad = next((i for i in range(n_new) if got[i] != ref[i]), None)
        print(f"seq {b}: {bad if bad is not None else n_new}/{n_new} equal")
        if bad is not None:
            assert argmax_ok(got[bad], rows[bad]), (b, bad)


def oracle_tree_from(g, T):
    return O.Tree(np.array(g.token[:T], dtype=np.int32), np.array(g.parent[:T], dtype=np.int32),
                  np.array(g.depth[:T], dtype=np.int32), np.zeros(T))


def test_sample_accept_matches_oracle(setup):
    """Speculative sampling at temperature > 0: path, slots and emitted tokens
    equal the oracle's on the GPU's own float32 logits and the same draws
    (a decision may differ only within float32 rounding of its threshold);
    the accepted rows are compacted like the greedy rule's.  Low temperatures
    concentrate the target on its argmax, so drafted children get accepted
    and the walk goes down the tree."""
    from oracle import sampling as S
    from paper_2505_14260_amd.msd import MAX_TREE, msd_seq_len
    wl, eng, m, prompt = setup
    # near-greedy cycles follow the sequence on which the draft agrees with
    # the target (deep accepts), warm ones make the decisions fractional
    temps = (0.005, 0.005, 0.05, 0.005, 0.02, 0.005) * 2 + (1.0, 0.7, 1.0, 0.7)
    n_cyc = len(temps)
    print(f"case: tiny sampling acceptance, {n_cyc} cycles at temperatures {temps}", flush=True)
    spec, _ = static_spec(wl.tree.paths)
    T = spec.n_nodes + 1
    eng.prefill(0, *prompt)
    trees = eng.new_trees(1)
    tk, tv, _, _ = eng.kv_views()
    deep = 0
    for cyc in range(n_cyc):
        temp = temps[cyc % len(temps)]
        eng.draft_tree([0], spec, trees)
        amax, logits = eng.verify([0], trees, T, want_logits=True)
        L = msd_seq_len(eng.ctx, 0)
        tree = oracle_tree_from(eng.trees_to_host(trees, 1)[0], T)
        lg = logits.cpu().numpy().reshape(T, -1)
        before_k = tk[:, 0, :, L:L + T, :].clone()
        em, slots = eng.accept_sample([0], trees, T, logits, temp, 4242, want_slots=True)
        torch.cuda.synchronize()
        sl = slots.cpu().numpy()[:MAX_TREE]
        n = len(em[0])
        path = [int(x) - L for x in sl[:n]]
        assert all(x == -1 for x in sl[n:])
        r_path, r_emit, dec = S.sample_accept(tree, lg, temp, 4242, 0, L)
        same = path == r_path and [int(x) for x in em[0]] == r_emit
        print(f"cycle {cyc} T={temp}: path {path} emitted {list(em[0])} "
              f"{'equal' if same else 'gated'}")
        assert sampling_agrees(path, em[0], r_path, r_emit, dec), (cyc, path, r_path, em, r_emit)
        assert msd_seq_len(eng.ctx, 0) == L + n
        for j, u in enumerate(path):
            assert torch.equal(tk[:, 0, :, L + j, :], before_k[:, :, u, :]), (cyc, j)
        deep += n > 1
    print(f"{deep}/{n_cyc} cycles accepted at least one drafted token")
    assert deep > 0


def test_sampling_is_lossless_on_gpu(setup):
    """Over many cycles the first emitted token follows the target
    distribution at the root: its randomised probability integral transform
    under that distribution is uniform (Kolmogorov-Smirnov)."""
    from scipy import stats
    from oracle import sampling as S
    from paper_2505_14260_amd.msd import msd_seq_len
    wl, eng, m, prompt = setup
    n_cycles = 240
    print(f"case: tiny sampling distribution, {n_cycles} cycles at temperature 1", flush=True)
    spec, _ = static_spec(wl.tree.paths)
    T = spec.n_nodes + 1
    trees = eng.new_trees(1)
    rng = np.random.default_rng(0)
    pit, epoch = [], 0
    eng.prefill(0, *prompt)
    for _ in range(n_cycles):
        if msd_seq_len(eng.ctx, 0) + 2 * T > 256:
            eng.prefill(0, *prompt)
            epoch += 1  # a fresh seed: the same lengths come round again
        eng.draft_tree([0], spec, trees)
        amax, logits = eng.verify([0], trees, T, want_logits=True)
        p = S.target_probs(logits[0].cpu().numpy(), 1.0)
        em, _ = eng.accept_sample([0], trees, T, logits, 1.0, 1000 + epoch)
        y = int(em[0][0])
        lo = p[:y].sum()
        pit.append(lo + rng.random() * p[y])
    res = stats.kstest(pit, "uniform")
    print(f"KS statistic {res.statistic:.3f}, p-value {res.pvalue:.3g} over {n_cycles} cycles")
    assert res.pvalue > 1e-3


def test_sample_accept_argument_checks(setup):
    from paper_2505_14260_amd.msd import MSDError
    wl, eng, m, prompt = setup
    print("case: tiny sampling acceptance error paths", flush=True)
    spec, _ = static_spec(wl.tree.paths)
    T = spec.n_nodes + 1
    eng.prefill(0, *prompt)
    trees = eng.new_trees(1)
    eng.draft_tree([0], spec, trees)
    amax, logits = eng.verify([0], trees, T, want_logits=True)
    for bad in (0.0, -1.0, float("nan"), float("inf")):
        with pytest.raises(MSDError):
            eng.accept_sample([0], trees, T, logits, bad, 1)
    eng.accept_sample([0], trees, T, logits, 1.0, 1)
    with pytest.raises(MSDError):  # a second acceptance of the same verify
        eng.accept_sample([0], trees, T, logits, 1.0, 1)


def test_stale_cache_slots_never_read(setup):
    """KV slots at or past a sequence's committed length may hold any bits
    (never written, rejected tree nodes, or whatever the caller left there).
    Every such slot of both caches is filled with NaN and infinity patterns
    before each cycle of a ragged batch-of-2 decode; the tokens must still
    be the plain greedy decode's.  Catch-up padding of the shorter sequence
    and the last partial key block of every attention pass are covered."""
    from paper_2505_14260_amd.msd import msd_seq_len
    wl, eng, m, prompt = setup
    print("case: tiny batch of 2 with NaN/inf bits past every length", flush=True)
    tokens, is_visual, visual = prompt
    cut = wl.n_visual + 9
    p1 = (tokens[:cut], is_visual[:cut], visual)
    spec, _ = static_spec(wl.tree.paths)
    T = spec.n_nodes + 1
    tk, tv, dk, dv = eng.kv_views()
    bits = (-1, 0x7F80, -128)       # NaN, +inf, -inf as bf16 bit patterns

    def poison(b, t_from, d_from, pat):
        for a, lo in ((tk, t_from), (dk, d_from)):
            a[:, b, :, lo:, :] = pat
        for a, lo in ((tv, t_from), (dv, d_from)):
            a[:, b, :, :, lo:] = pat
        torch.cuda.synchronize()        # the library runs on its own stream

    outs = [[eng.prefill(0, *prompt)], [eng.prefill(1, *p1)]]
    for b in range(2):
        L = msd_seq_len(eng.ctx, b)
        poison(b, L, L, bits[b])
    trees = eng.new_trees(2)
    n_new = 24
    cycle = 0
    while min(len(o) for o in outs) < n_new:
        eng.draft_tree([0, 1], spec, trees)
        amax, _ = eng.verify([0, 1], trees, T)
        em, _ = eng.accept([0, 1], trees, T, amax)
        cycle += 1
        for b in range(2):
            outs[b].extend(int(t) for t in em[b])
            L = msd_seq_len(eng.ctx, b)
            # target slots past L and draft slots past the catch-up start
            poison(b, L, L - len(em[b]), bits[(b + cycle) % 3])
    torch.cuda.synchronize()
    for b, p in enumerate((prompt, p1)):
        ref, rows = O.greedy_generate(m, p, n_new, return_logits=True)
        got = outs[b][:n_new]
        bad = next((i for i in range(n_new) if got[i] != ref[i]), None)
        print(f"seq {b}: {bad if bad is not None else n_new}/{n_new} equal")
        if bad is not None:
            assert argmax_ok(got[bad], rows[bad]), (b, bad)


def test_capacity_limits(setup):
    wl, eng, m, prompt = setup
    from paper_2505_14260_amd import msd as B
    spec, _ = static_spec(wl.tree.paths)
    eng.prefill(0, *prompt)
    h = torch.zeros(wl.dims.d_model, dtype=torch.int16, device="cuda")
    with pytest.raises(B.MSDError) as e:
        B.msd_set_state(eng.ctx, 0, 256 - 63, h.data_ptr(), 1)   # L + max_tree > max_seq
    assert e.value.code == B.MSD_ERR_CAPACITY
    B.msd_set_state(eng.ctx, 0, 256 - 64, h.data_ptr(), 1)
    dev = eng.new_trees(1)
    B.msd_set_state(eng.ctx, 0, 256 - 64, h.data_ptr(), 1)
    eng.draft_tree([0], spec, dev)
    amax, _ = eng.verify([0], dev, spec.n_nodes + 1)
    eng.accept([0], dev, spec.n_nodes + 1, amax)
    with pytest.raises(B.MSDError) as e:       # the next tree no longer fits
        for _ in range(64):
            eng.draft_tree([0], spec, dev)
            amax, _ = eng.verify([0], dev, spec.n_nodes + 1)
            eng.accept([0], dev, spec.n_nodes + 1, amax)
    assert e.value.code == B.MSD_ERR_CAPACITY
