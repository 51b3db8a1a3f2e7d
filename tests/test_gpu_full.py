"""GPU parity at the full model shapes, in the launch configuration of the
decode benchmark: one MSD cycle (draft tree, tree verification, greedy
acceptance and compaction) from a seeded synthetic cache state, through the C
ABI, against the float64 oracle on the same bf16 weights and cache values.

A full-size prompt forward costs the oracle minutes, so each case starts from
an imported state (msd_set_state): target cache slots [0, L) and draft slots
[0, L-1) hold the same seeded bf16 values on both sides, the pending draft
row is one text row (a seeded target feature h and the root token).  The
prompt forward itself is checked at full size on what the oracle can compute
row by row: layer 0 of the target cache and the draft cache of visual rows
(both depend on their own row only).

Checks per cycle (tolerances in tests/parity.py):
  * draft tree: structure bit-exact; tokens equal wherever the oracle's
    ranking is decided (static), or every divergence sits at a near tie of
    the oracle's scores (dynamic);
  * verification on the GPU's tree (teacher forced): logits within 2e-2 of
    each row's max, argmax equal where the top-2 margin is decided, the K/V
    rows written at the tree slots within the same tolerance;
  * acceptance with a forced argmax (so that a path of chosen depth is
    accepted): emitted tokens, slot map and the compacted cache bit-exact;
    the oracle then adopts the same path and a second cycle checks the draft
    catch-up over the accepted rows.
"""
import dataclasses
import time

import numpy as np
import pytest

import synth
from synth.configs import LLAVA7B, LLAVA13B, LLAVA7B_LONG, QWEN7B
from oracle import model as M
from oracle import msd as O
from parity import (RTOL, argmax_ok, compare_dynamic_tree, compare_static_tree, decided,
                    gpu_tree_arrays, oracle_draft_dynamic, oracle_draft_static,
                    oracle_tree_of, row_close, sampling_agrees)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TID_STATE = synth.TID_TEST + 8     # + 4*seq + {0: K, 1: V, 2: draft K, 3: draft V}
TID_FEAT = synth.TID_TEST + 40     # + seq: pending target feature
TID_ROOT = synth.TID_TEST + 48     # + seq: root token


def log(msg):
    print(msg, flush=True)


def i16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16))


def bits64(t):
    return M.widen(t.cpu().numpy().view(np.uint16))


class Case:
    """Engine + oracle models + per-sequence synthetic states of one workload."""

    def __init__(self, wl, lengths, cycles=2, caller_weights=False):
        from paper_2505_14260_amd.msd import Engine, msd_set_state, make_static_spec, \
            make_dynamic_spec
        t0 = time.perf_counter()
        self.wl, self.dims = wl, wl.dims
        dims = wl.dims
        self.w = synth.make_target_weights(dims, wl.seed, wl.weight_sigma)
        self.dr = synth.make_draft_weights(dims, self.w, wl.seed, wl.draft_fc_mode)
        T = wl.tree.n_draft + 1
        self.T = T
        self.max_seq = (max(lengths) + cycles * T + 255) // 256 * 256
        self.eng = Engine(dims, self.w, self.dr, max_batch=len(lengths), max_seq=self.max_seq,
                          max_tree=64, max_prompt=wl.prompt_len)
        if caller_weights:
            self.eng.use_caller_weights(True)
        self.m = O.Models(dims, self.w, self.dr)
        if wl.tree.kind == "static":
            self.arrays = synth.static_tree_arrays(wl.tree.paths)
            self.spec = make_static_spec(self.arrays[0][1:], self.arrays[1][1:])
        else:
            self.arrays = None
            self.spec = make_dynamic_spec(wl.tree.topk, wl.tree.depth, wl.tree.n_nodes)
        tk, tv, dk, dv = self.eng.kv_views()
        nl, KV, hd, d = dims.n_layers, dims.n_kv_heads, dims.head_dim, dims.d_model
        self.states, self.prefix_k = [], []
        for b, L in enumerate(lengths):
            k = synth.normal_bf16((nl, L, KV, hd), wl.seed, TID_STATE + 4 * b, 1.0)
            v = synth.normal_bf16((nl, L, KV, hd), wl.seed, TID_STATE + 4 * b + 1, 1.0)
            dkb = synth.normal_bf16((1, L - 1, KV, hd), wl.seed, TID_STATE + 4 * b + 2, 1.0)
            dvb = synth.normal_bf16((1, L - 1, KV, hd), wl.seed, TID_STATE + 4 * b + 3, 1.0)
            tk[:, b, :, :L, :].copy_(i16(k.transpose(0, 2, 1, 3)).cuda())
            tv[:, b, :, :, :L].copy_(i16(v.transpose(0, 2, 3, 1)).cuda())
            dk[:, b, :, :L - 1, :].copy_(i16(dkb.transpose(0, 2, 1, 3)).cuda())
            dv[:, b, :, :, :L - 1].copy_(i16(dvb.transpose(0, 2, 3, 1)).cuda())
            h = synth.normal_bf16((d,), wl.seed, TID_FEAT + b, 1.0)
            root = int(synth.ids(1, wl.seed, TID_ROOT + b, dims.vocab)[0])
            h_dev = i16(h).cuda()
            torch.cuda.synchronize()
            msd_set_state(self.eng.ctx, b, L, h_dev.data_ptr(), root)
            kv = M.KVCache(nl, self.max_seq, KV, hd)
            kv.k[:, :L] = M.widen(k)
            kv.v[:, :L] = M.widen(v)
            dkv = M.KVCache(1, self.max_seq, KV, hd)
            dkv.k[:, :L - 1] = M.widen(dkb)
            dkv.v[:, :L - 1] = M.widen(dvb)
            st = O.SeqState(kv=kv, dkv=dkv, L=L, root=root,
                            pending=[O.PendingRow(False, h=M.widen(h), e_next=self.m.embed(root))])
            self.states.append(st)
            self.prefix_k.append(tk[:, b, :, :L, :].clone())
            del k, v, dkb, dvb
        torch.cuda.synchronize()
        log(f"[{wl.name}] set up in {time.perf_counter() - t0:.1f}s: L={lengths}, T={T}, "
            f"max_seq={self.max_seq}")

    def close(self):
        self.eng.close()
        del self.eng
        torch.cuda.empty_cache()

    # --- one cycle ------------------------------------------------------------------
    def cycle(self, accept_depths, label):
        from paper_2505_14260_amd.msd import MAX_TREE, msd_seq_len
        wl, eng, m, T = self.wl, self.eng, self.m, self.T
        n = len(self.states)
        seqs = list(range(n))
        t0 = time.perf_counter()
        trees = eng.new_trees(n)
        eng.draft_tree(seqs, self.spec, trees)
        gts = eng.trees_to_host(trees, n)
        for b, (g, st) in enumerate(zip(gts, self.states)):
            assert g.token[0] == st.root
            if wl.tree.kind == "static":
                ref, logs, rank = oracle_draft_static(m, st, wl.tree.paths)
                c = compare_static_tree(g, ref, logs, rank)
                log(f"[{label} seq {b}] static draft tree: {c}/{T - 1} tokens compared equal")
            else:
                K, N = wl.tree.topk, wl.tree.n_nodes
                ref, pool, rows, root_logits = oracle_draft_dynamic(m, st, K, wl.tree.depth, N)
                same, scored = compare_dynamic_tree(g, pool, rows, root_logits, K, N, ref=ref)
                log(f"[{label} seq {b}] dynamic draft tree: {same}/{N} nodes as the oracle's, "
                    f"{scored} scores compared, {compare_dynamic_tree.exact} trees compared "
                    f"bit for bit so far")
        amax, logits = eng.verify(seqs, trees, T, want_logits=True)
        torch.cuda.synchronize()
        lg = logits.cpu().numpy().reshape(n, T, -1)
        am = amax.cpu().numpy().reshape(n, T)
        tk, tv, _, _ = eng.kv_views()
        refs = []
        for b, (g, st) in enumerate(zip(gts, self.states)):
            tree = oracle_tree_of(g)
            h_ref, lg_ref = O.verify(m, st, tree)
            ok, err = row_close(lg[b], lg_ref)
            n_dec = 0
            for i in range(T):
                assert argmax_ok(am[b, i], lg_ref[i]), (b, i)
                n_dec += decided(lg_ref[i])
            L = st.L
            kerr = 0.0
            for l in range(self.dims.n_layers):
                kg = bits64(tk[l, b, :, L:L + T, :].permute(1, 0, 2).reshape(T, -1))
                vg = bits64(tv[l, b, :, :, L:L + T].permute(2, 0, 1).reshape(T, -1))
                okk, ek = row_close(kg, st.kv.k[l, L:L + T].reshape(T, -1))
                okv, ev = row_close(vg, st.kv.v[l, L:L + T].reshape(T, -1))
                assert okk and okv, (b, l, ek, ev)
                kerr = max(kerr, ek, ev)
            log(f"[{label} seq {b}] verify L={L}: logits max rel err {err:.2e}, "
                f"{n_dec}/{T} argmax decided and equal (the rest in the near-tie band), "
                f"tree K/V max rel err {kerr:.2e}")
            assert ok, err
            refs.append((tree, h_ref))
        # acceptance along a chosen chain of first children, forced through argmax
        forced = am.copy()
        paths = []
        for b, (tree, _) in enumerate(refs):
            u, path = 0, [0]
            for _ in range(accept_depths[b]):
                kids = [c for c in range(1, T) if tree.parent[c] == u]
                if not kids:
                    break
                forced[b, u] = tree.token[kids[0]]
                u = kids[0]
                path.append(u)
            paths.append(path)
        before_k = [tk[:, b, :, self.states[b].L:self.states[b].L + T, :].clone() for b in seqs]
        before_v = [tv[:, b, :, :, self.states[b].L:self.states[b].L + T].clone() for b in seqs]
        forced_dev = torch.from_numpy(forced.reshape(-1).astype(np.int32)).cuda()
        em, slots = eng.accept(seqs, trees, T, forced_dev, want_slots=True)
        torch.cuda.synchronize()
        sl = slots.cpu().numpy().reshape(n, MAX_TREE)
        for b, ((tree, h_ref), st) in enumerate(zip(refs, self.states)):
            L = st.L
            path, emitted = O.greedy_accept(tree, forced[b])
            assert path[:len(paths[b])] == paths[b]
            assert em[b] == emitted, (b, em[b], emitted)
            assert list(sl[b, :len(path)]) == [L + j for j in path]
            assert all(x == -1 for x in sl[b, len(path):])
            for j, u in enumerate(path):
                assert torch.equal(tk[:, b, :, L + j, :], before_k[b][:, :, u, :]), (b, j)
                assert torch.equal(tv[:, b, :, :, L + j], before_v[b][:, :, :, u]), (b, j)
            assert torch.equal(tk[:, b, :, :self.prefix_k[b].shape[2], :], self.prefix_k[b])
            O.accept_and_compact(m, st, tree, h_ref, forced[b])
            assert msd_seq_len(eng.ctx, b) == st.L
            log(f"[{label} seq {b}] accepted path {path}, emitted {emitted}")
        log(f"[{label}] cycle checked in {time.perf_counter() - t0:.1f}s")

    def natural_cycle(self, n_chain, label):
        """One cycle whose tree holds the target's own greedy continuation.

        The oracle decodes n_chain tokens greedily from the committed state;
        they replace the tokens of the first-ranked chain of the GPU's draft
        tree (siblings kept distinct), so the verify's own argmax accepts them
        without any forcing.  Everything the GPU emits must equal the oracle's
        acceptance on the oracle's logits wherever those are decided, and the
        accepted path must reach the chain's depth when every step is decided.
        """
        from paper_2505_14260_amd.msd import MAX_TREE, Tree, msd_seq_len
        wl, eng, m, T, dims = self.wl, self.eng, self.m, self.T, self.dims
        assert len(self.states) == 1 and wl.tree.kind == "static"
        st = self.states[0]
        t0 = time.perf_counter()
        trees = eng.new_trees(1)
        eng.draft_tree([0], self.spec, trees)
        g = eng.trees_to_host(trees, 1)[0]
        # the target's greedy continuation of the root, one row at a time
        kv = st.kv.copy()
        cur, chain, margins = st.root, [], []
        for j in range(n_chain):
            x = M.embed_rows(m.w, [cur])
            pos = np.array([st.L + j], dtype=np.int32)
            _, lg1 = M.target_forward(dims, m.w, kv, x, pos, pos, st.L + j, 1, None)
            cur = int(np.argmax(lg1[0]))
            chain.append(cur)
            margins.append(decided(lg1[0]))
        # the first-ranked chain of the static shape: node 0 -> ... by rank 0
        par = list(g.parent[:T])
        rank = list(self.arrays[1])
        u, nodes = 0, []
        for _ in range(n_chain):
            kids = [c for c in range(1, T) if par[c] == u and rank[c] == 0]
            if not kids:
                break
            u = kids[0]
            nodes.append(u)
        tok = list(g.token[:T])
        for u, t in zip(nodes, chain):
            tok[u] = t
        for u in nodes:  # a sibling holding the same token gets another one
            for c in range(1, T):
                if c != u and par[c] == par[u] and tok[c] == tok[u]:
                    while tok[c] in [tok[x] for x in range(1, T) if par[x] == par[u] and x != c]:
                        tok[c] = (tok[c] + 1) % dims.vocab
        t = Tree()
        t.n_nodes = T
        for i in range(T):
            t.token[i], t.parent[i], t.depth[i], t.anc[i] = tok[i], g.parent[i], g.depth[i], \
                g.anc[i]
        trees.copy_(torch.frombuffer(bytearray(bytes(t)), dtype=torch.uint8).cuda())
        tree = oracle_tree_of(t)
        amax, logits = eng.verify([0], trees, T, want_logits=True)
        torch.cuda.synchronize()
        lg = logits.cpu().numpy().reshape(T, -1)
        am = amax.cpu().numpy().reshape(T)
        h_ref, lg_ref = O.verify(m, st, tree)
        ok, err = row_close(lg, lg_ref)
        assert ok, err
        for i in range(T):
            assert argmax_ok(am[i], lg_ref[i]), i
        em, slots = eng.accept([0], trees, T, amax, want_slots=True)
        torch.cuda.synchronize()
        sl = slots.cpu().numpy().reshape(1, MAX_TREE)[0]
        L = st.L
        ref_am = np.argmax(lg_ref, axis=1)
        r_path, r_emit = O.greedy_accept(tree, ref_am)
        g_path, g_emit = O.greedy_accept(tree, am)
        assert em[0] == g_emit and list(sl[:len(g_path)]) == [L + j for j in g_path]
        # the chain is accepted as far as the oracle's own decisions are decided
        n_dec = next((j for j, d in enumerate(margins) if not d), n_chain)
        assert len(g_path) - 1 >= min(n_dec, len(nodes)), (g_path, margins)
        assert g_emit[:min(n_dec, len(nodes))] == chain[:min(n_dec, len(nodes))]
        if all(decided(lg_ref[u]) for u in [0] + g_path[1:]):
            assert g_path == r_path and g_emit == r_emit
        O.accept_and_compact(m, st, tree, h_ref, am)
        assert msd_seq_len(eng.ctx, 0) == st.L
        log(f"[{label}] greedy chain {chain} (decided {margins}); accepted path {g_path}, "
            f"emitted {g_emit}; logits max rel err {err:.2e}; "
            f"checked in {time.perf_counter() - t0:.1f}s")
        return len(g_path) - 1

    def sample_cycle(self, temperature, seed, label):
        """One cycle with speculative-sampling acceptance, checked against the
        oracle's rule on the GPU's own logits and draws (the state is not
        tracked further)."""
        from oracle import sampling as S
        from paper_2505_14260_amd.msd import MAX_TREE, msd_seq_len
        eng, T = self.eng, self.T
        n = len(self.states)
        seqs = list(range(n))
        trees = eng.new_trees(n)
        eng.draft_tree(seqs, self.spec, trees)
        gts = eng.trees_to_host(trees, n)
        _, logits = eng.verify(seqs, trees, T, want_logits=True)
        torch.cuda.synchronize()
        lg = logits.cpu().numpy().reshape(n, T, -1)
        Ls = [msd_seq_len(eng.ctx, b) for b in seqs]
        tk, tv, _, _ = eng.kv_views()
        before_k = [tk[:, b, :, Ls[b]:Ls[b] + T, :].clone() for b in seqs]
        before_v = [tv[:, b, :, :, Ls[b]:Ls[b] + T].clone() for b in seqs]
        em, slots = eng.accept_sample(seqs, trees, T, logits, temperature, seed, want_slots=True)
        torch.cuda.synchronize()
        sl = slots.cpu().numpy().reshape(n, MAX_TREE)
        for b in seqs:
            L, k = Ls[b], len(em[b])
            path = [int(x) - L for x in sl[b, :k]]
            r_path, r_emit, dec = S.sample_accept(oracle_tree_of(gts[b]), lg[b], temperature,
                                                  seed, b, L)
            assert sampling_agrees(path, em[b], r_path, r_emit, dec), (b, path, r_path)
            for j, u in enumerate(path):
                assert torch.equal(tk[:, b, :, L + j, :], before_k[b][:, :, u, :]), (b, j)
                assert torch.equal(tv[:, b, :, :, L + j], before_v[b][:, :, :, u]), (b, j)
            assert msd_seq_len(eng.ctx, b) == L + k
            log(f"[{label} seq {b}] sampled at T={temperature}: path {path}, emitted {em[b]} "
                f"({'as the oracle' if path == r_path else 'gated'})")


@pytest.mark.timeout(240)
def test_llava7b_two_cycles():
    """7B-shaped, static 26-node tree at the benchmark's prompt length."""
    log("case: full llava-1.5-7b-shaped, L=640, two cycles")
    c = Case(LLAVA7B, [LLAVA7B.prompt_len])
    try:
        c.cycle([3], "7b c1")
        c.cycle([0], "7b c2")
        c.sample_cycle(1.0, 2024, "7b c3")
    finally:
        c.close()


@pytest.mark.timeout(300)
def test_llava7b_natural_acceptance():
    """7B-shaped: a tree carrying the target's greedy continuation is accepted
    by the verify's own argmax (no forcing), then the draft catches up over
    the accepted rows in the next cycle."""
    log("case: full llava-1.5-7b-shaped, natural multi-token acceptance")
    c = Case(LLAVA7B, [LLAVA7B.prompt_len])
    try:
        k = c.natural_cycle(LLAVA7B.tree.depth, "7b natural")
        assert k >= 1
        c.cycle([0], "7b after natural")
    finally:
        c.close()


@pytest.mark.timeout(240)
def test_llava13b_cycle():
    log("case: full llava-1.5-13b-shaped, L=704, one cycle")
    c = Case(LLAVA13B, [LLAVA13B.prompt_len], cycles=1)
    try:
        c.cycle([2], "13b")
    finally:
        c.close()


@pytest.mark.timeout(240)
def test_llava7b_long_prefix_dynamic_cycle():
    log("case: full 7b long visual prefix, L=3136, dynamic 60-node tree")
    c = Case(LLAVA7B_LONG, [LLAVA7B_LONG.prompt_len], cycles=1)
    try:
        c.cycle([4], "7b-long")
    finally:
        c.close()


@pytest.mark.timeout(300)
@pytest.mark.parametrize("caller_weights", [False, True])
def test_qwen7b_gqa_batch4_ragged(caller_weights):
    """Qwen-shaped GQA (28 query / 4 KV heads, vocab 152064), four sequences
    at different lengths, dynamic 60-node trees, different accepted depths.
    The 244-row verify runs as 64-row weight-streaming launches, or with
    msd_use_caller_weights as rocBLAS products on the row-major weights."""
    n = QWEN7B.prompt_len
    lengths = [n, n - 37, n + 5, n - 100]
    log(f"case: full qwen2.5-vl-7b-shaped, batch 4, L={lengths}, caller weights {caller_weights}")
    c = Case(QWEN7B, lengths, cycles=2, caller_weights=caller_weights)
    try:
        c.cycle([0, 1, 3, 6], "qwen")
        c.sample_cycle(0.8, 99, "qwen sampled")
    finally:
        c.close()


@pytest.mark.timeout(240)
def test_llava7b_prefill_rows():
    """The prompt forward at full size, on what depends on one row only:
    layer 0 of the target cache (all 640 rows) and the draft cache of the
    576 visual rows (their draft input is the visual embedding itself)."""
    from paper_2505_14260_amd.msd import Engine
    wl = LLAVA7B
    dims = wl.dims
    log("case: full llava-1.5-7b-shaped prefill, layer-0 and visual draft rows")
    w = synth.make_target_weights(dims, wl.seed, wl.weight_sigma)
    dr = synth.make_draft_weights(dims, w, wl.seed, wl.draft_fc_mode)
    prompt = synth.make_prompt(wl)
    eng = Engine(dims, w, dr, max_batch=1, max_seq=1024, max_tree=64, max_prompt=wl.prompt_len)
    try:
        eng.prefill(0, *prompt)
        torch.cuda.synchronize()
        tokens, is_visual, visual = prompt
        n = len(tokens)
        vis_rows = [None] * n
        vi = 0
        for i in range(n):
            if is_visual[i]:
                vis_rows[i] = visual[vi]
                vi += 1
        x = M.embed_rows(w, tokens, vis_rows)
        one = dataclasses.replace(dims, n_layers=1)
        kv = M.KVCache(1, n, dims.n_kv_heads, dims.head_dim)
        pos = np.arange(n, dtype=np.int32)
        w1 = dict(w)
        w1["layers"] = w["layers"][:1]
        M.target_forward(one, w1, kv, x, pos, pos, 0, n, None, want_logits=False)
        tk, tv, dk, dv = eng.kv_views()
        kg = bits64(tk[0, 0, :, :n, :].permute(1, 0, 2).reshape(n, -1))
        vg = bits64(tv[0, 0, :, :, :n].permute(2, 0, 1).reshape(n, -1))
        ok_k, ek = row_close(kg, kv.k[0, :n].reshape(n, -1))
        ok_v, ev = row_close(vg, kv.v[0, :n].reshape(n, -1))
        log(f"prefill layer-0 K/V max rel err {ek:.2e} / {ev:.2e}")
        assert ok_k and ok_v
        vis = np.where(np.asarray(is_visual, dtype=bool))[0]
        f = x[vis]
        dkv = M.KVCache(1, n, dims.n_kv_heads, dims.head_dim)
        M.draft_forward(dims, dr, dkv, f, vis.astype(np.int32), vis, 0, len(vis), None)
        kg = bits64(dk[0, 0, :, :n, :].permute(1, 0, 2).reshape(n, -1))[vis]
        vg = bits64(dv[0, 0, :, :, :n].permute(2, 0, 1).reshape(n, -1))[vis]
        ok_k, ek = row_close(kg, dkv.k[0, vis].reshape(len(vis), -1))
        ok_v, ev = row_close(vg, dkv.v[0, vis].reshape(len(vis), -1))
        log(f"prefill draft visual-row K/V max rel err {ek:.2e} / {ev:.2e}")
        assert ok_k and ok_v
    finally:
        eng.close()
        torch.cuda.empty_cache()
