"""msd_verify_noalloc (scratch in the library's static device array) against
msd_verify through the C ABI, on two calls in a row: a batch of two full
draft trees, then a smaller call (one sequence, the first nodes of its tree).
Both entry points run the same kernels with the same attention chunking, so
argmax and logits must agree bit for bit (well inside the float tolerance);
the acceptance that follows the no-allocation verify must behave as after
msd_verify.  A call larger than the stated maximum is rejected."""
import numpy as np
import pytest

import synth
from synth.configs import TINY, WIDE
from oracle import msd as O
from parity import argmax_ok, row_close

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def models(wl):
    w = synth.make_target_weights(wl.dims, wl.seed)
    dr = synth.make_draft_weights(wl.dims, w, wl.seed, wl.draft_fc_mode)
    return O.Models(wl.dims, w, dr)


def sub_tree_bytes(g, n):
    """The first n nodes of a tree (parents precede children, so they form
    a tree) as msd_tree bytes."""
    from paper_2505_14260_amd.msd import Tree
    t = Tree()
    t.n_nodes = n
    for i in range(n):
        t.token[i], t.parent[i], t.depth[i], t.anc[i] = g.token[i], g.parent[i], g.depth[i], \
            g.anc[i]
    return bytes(t)


def both(eng, B, seqs, trees, T):
    V = eng.dims.vocab
    am1 = torch.full((len(seqs) * T,), -7, dtype=torch.int32, device="cuda")
    am2 = torch.full_like(am1, -7)
    lg1 = torch.full((len(seqs) * T, V), float("nan"), dtype=torch.float32, device="cuda")
    lg2 = torch.full_like(lg1, float("nan"))
    B.msd_verify(eng.ctx, seqs, trees.data_ptr(), T, am1.data_ptr(), lg1.data_ptr())
    torch.cuda.synchronize()
    B.msd_verify_noalloc(eng.ctx, seqs, trees.data_ptr(), T, am2.data_ptr(), lg2.data_ptr())
    torch.cuda.synchronize()
    return am1, lg1, am2, lg2


@pytest.mark.parametrize("wl", [TINY, WIDE], ids=lambda w: w.name)
def test_verify_noalloc_matches_verify(wl):
    from paper_2505_14260_amd import msd as B
    from paper_2505_14260_amd.msd import Engine, make_static_spec
    print(f"case: verify_noalloc vs verify, {wl.name}", flush=True)
    m = models(wl)
    prompt = synth.make_prompt(wl)
    eng = Engine(wl.dims, m.w, m.draft, max_batch=2, max_seq=wl.prompt_len + 128, max_tree=64,
                 max_prompt=wl.prompt_len)
    try:
        parent, rank, _ = synth.static_tree_arrays(wl.tree.paths)
        spec = make_static_spec(parent[1:], rank[1:])
        T = spec.n_nodes + 1
        tokens, is_visual, visual = prompt
        cut = wl.n_visual + wl.n_text // 2
        eng.prefill(0, *prompt)
        eng.prefill(1, tokens[:cut], is_visual[:cut], visual)
        trees = eng.new_trees(2)
        eng.draft_tree([0, 1], spec, trees)
        # call 1: both sequences, full trees
        am1, lg1, am2, lg2 = both(eng, B, [0, 1], trees, T)
        assert torch.equal(am1, am2)
        assert torch.equal(lg1, lg2)
        ok, err = row_close(lg2.cpu().numpy(), lg1.cpu().numpy())
        assert ok, err
        # the acceptance after the no-allocation verify
        gts = eng.trees_to_host(trees, 2)
        L0 = [B.msd_seq_len(eng.ctx, b) for b in (0, 1)]
        em, _ = eng.accept([0, 1], trees, T, am2)
        a = am2.cpu().numpy().reshape(2, T)
        for b in range(2):
            tree = O.Tree(np.array(gts[b].token[:T]), np.array(gts[b].parent[:T]),
                          np.array(gts[b].depth[:T]), np.zeros(T))
            _, want = O.greedy_accept(tree, a[b])
            assert em[b] == want, (b, em[b], want)
            assert B.msd_seq_len(eng.ctx, b) == L0[b] + len(want)
        # call 2: one sequence, a smaller tree (the first 7 nodes of a new one)
        one = eng.new_trees(1)
        eng.draft_tree([1], spec, one)
        g = eng.trees_to_host(one, 1)[0]
        n = 7
        small = eng.new_trees(1)
        small.copy_(torch.frombuffer(bytearray(sub_tree_bytes(g, n)), dtype=torch.uint8))
        am1, lg1, am2, lg2 = both(eng, B, [1], small, n)
        assert torch.equal(am1, am2)
        assert torch.equal(lg1, lg2)
        l1 = lg1.cpu().numpy()
        for i, x in enumerate(am2.cpu().numpy()):
            assert argmax_ok(x, l1[i]), i
        em, _ = eng.accept([1], small, n, am2)
        assert 1 <= len(em[0]) <= n
        print(f"{wl.name}: no-allocation verify equal to msd_verify on 2x{T} and 1x{n} nodes",
              flush=True)
    finally:
        eng.close()


def test_verify_noalloc_rejects_oversized_calls():
    from paper_2505_14260_amd import msd as B
    from paper_2505_14260_amd.msd import Engine, make_dynamic_spec
    wl = TINY
    print("case: verify_noalloc beyond its maximum", flush=True)
    m = models(wl)
    prompt = synth.make_prompt(wl)
    eng = Engine(wl.dims, m.w, m.draft, max_batch=5, max_seq=256, max_tree=64, max_prompt=128)
    try:
        for b in range(5):
            eng.prefill(b, *prompt)
        spec = make_dynamic_spec(8, 4, 63)
        trees = eng.new_trees(5)
        eng.draft_tree(list(range(5)), spec, trees)
        am = torch.empty(5 * 64, dtype=torch.int32, device="cuda")
        with pytest.raises(B.MSDError) as e:  # 320 tree rows > 256
            B.msd_verify_noalloc(eng.ctx, list(range(5)), trees.data_ptr(), 64, am.data_ptr())
        assert e.value.code == B.MSD_ERR_INVALID_ARG
        # the context still verifies (the regular entry point takes any size)
        B.msd_verify(eng.ctx, list(range(5)), trees.data_ptr(), 64, am.data_ptr())
        torch.cuda.synchronize()
    finally:
        eng.close()
