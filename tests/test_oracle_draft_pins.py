"""Pins for the oracle's draft path and dynamic tree beam (CPU only).

Each is checked against a formulation written here from the paper's
definitions, not against the oracle's own code path:

* Tree-structured drafting (Sec. 3.2): a drafted node sees the committed
  draft cache plus exactly its own ancestors, so the draft feature the tree
  expansion computes for a node must equal a plain one-token-at-a-time causal
  decode of the draft head along that node's root-to-node branch, each step
  at the next position.  Float64 sums in the same key order, so the match is
  bit-exact.
* Draft catch-up (Eq. decouple): after any number of cycles, the committed
  draft cache and the root feature must equal one causal draft forward over
  the whole committed sequence, with each row's input assembled here from a
  fresh target forward: text row i takes f_down(Concat(h_i, e_{i+1})),
  visual row i takes e_i, or h_i in the Visual Feature variant of the
  input-decoupling ablation (Sec. 5.3).
* Dynamic tree: the beam is defined breadth-wise by sets (each depth's
  frontier is the best K of its candidates by cumulative log-probability;
  the tree keeps the best N of the whole pool), and the canonical node order
  is depth, then the lexicographic order of rank paths.  A brute force over
  every path of a small vocabulary, with log-probabilities from scipy, must
  reproduce the oracle's tree exactly.
* log-softmax against scipy.special.log_softmax.
"""
import itertools

import numpy as np
import pytest
from scipy.special import log_softmax as sp_log_softmax

import synth
from synth.configs import MINI_GQA, TINY, TreeShape, chain_paths
from oracle import model as M
from oracle import msd as O


def setup(wl):
    dims = wl.dims
    w = synth.make_target_weights(dims, wl.seed)
    dr = synth.make_draft_weights(dims, w, wl.seed, wl.draft_fc_mode)
    return O.Models(dims, w, dr), synth.make_prompt(wl)


SHAPES = {
    "static": lambda wl: wl.tree,
    "dynamic": lambda wl: TreeShape("dynamic", 4, topk=3, n_nodes=12),
    "chain": lambda wl: TreeShape("static", 4, tuple(chain_paths(4))),
}


def arrays(shape):
    return synth.static_tree_arrays(shape.paths) if shape.kind == "static" else None


def sequential_branch_decode(m, dkv, L, root_feat, tokens):
    """Plain causal decode of the draft head along one branch.

    Step j (1-based) feeds f_down(Concat(feature from step j-1, e(t_j))) at
    position and slot L + j - 1, attending to every earlier slot (the
    committed cache [0, L) and the branch's earlier steps) and itself.
    Returns the feature after the last step.
    """
    lw = m.draft["layer"]
    fc = m.draft["fc"]
    feat = root_feat
    for j, t in enumerate(tokens, start=1):
        x = np.concatenate([feat, M.widen(m.w["embed"][int(t)])])[None, :]
        f = M.linear(x, fc)
        p = np.array([L + j - 1], dtype=np.int32)
        feat = M.layer_forward(m.dims, lw, dkv.k[0], dkv.v[0], f, p, p, L + j - 1, 1, None)[0]
    return feat


@pytest.mark.parametrize("wl", [MINI_GQA, TINY], ids=lambda w: w.name)
@pytest.mark.parametrize("kind", ["static", "dynamic", "chain"])
def test_draft_nodes_equal_sequential_branch_decode(wl, kind):
    m, prompt = setup(wl)
    shape = SHAPES[kind](wl)
    st, _, _, _ = O.prefill(m, *prompt, max_slots=wl.prompt_len + 96)
    checked = 0
    for cycle in range(3):
        trace = {}
        tree = O.draft_tree(m, st, shape, arrays(shape), trace)
        L = trace["L"]
        assert L == st.L
        base = st.dkv.copy()  # slots [0, L) are committed; later slots get overwritten
        for path, feat in trace["feat"].items():
            want = sequential_branch_decode(m, base.copy(), L, trace["root_feat"], path)
            assert np.array_equal(feat, want), (cycle, path)
            checked += 1
        # every drafted node's token is one of its parent's draft top choices
        # computed from the sequential features
        for u in range(1, tree.n):
            p, x = [], u
            while x > 0:
                p.append(int(tree.token[x]))
                x = int(tree.parent[x])
            p = tuple(reversed(p))
            pf = trace["root_feat"] if len(p) == 1 else trace["feat"][p[:-1]]
            lg = M.linear(pf[None, :], m.w["lm_head"])[0]
            rank = int(np.sum(lg > lg[p[-1]]) + np.sum((lg == lg[p[-1]]) &
                                                       (np.arange(len(lg)) < p[-1])))
            bound = shape.topk if shape.kind == "dynamic" else 1 + max(
                int(c) for c in "".join(shape.paths))
            assert rank < bound, (cycle, p, rank)
        h, logits = O.verify(m, st, tree)
        O.accept_and_compact(m, st, tree, h, np.argmax(logits, axis=1))
    assert checked >= 3 * (shape.depth - 1)


def decoupled_inputs(m, rows_x, is_visual, h, root, visual_input="embedding"):
    """Draft input rows of Eq. decouple, assembled independently (visual rows:
    the embedding, or the target feature for visual_input="feature")."""
    L = len(rows_x)
    f = np.empty_like(rows_x)
    e_root = M.widen(m.w["embed"][int(root)])
    for i in range(L):
        if is_visual[i]:
            f[i] = rows_x[i] if visual_input == "embedding" else h[i]
        else:
            e_next = rows_x[i + 1] if i + 1 < L else e_root
            f[i] = M.linear(np.concatenate([h[i], e_next])[None, :], m.draft["fc"])[0]
    return f


@pytest.mark.parametrize("wl", [MINI_GQA, TINY], ids=lambda w: w.name)
@pytest.mark.parametrize("kind,visual_input", [("static", "embedding"), ("chain", "embedding"),
                                               ("static", "feature")])
def test_draft_cache_equals_one_causal_draft_forward(wl, kind, visual_input):
    m, prompt = setup(wl)
    tokens, vis_flags, visual = prompt
    shape = SHAPES[kind](wl)
    n = len(tokens)
    st, first, _, _ = O.prefill(m, *prompt, max_slots=n + 96, visual_input=visual_input)
    out = [first]
    for cycle in range(4):
        trace = {}
        tree = O.draft_tree(m, st, shape, arrays(shape), trace)
        L = trace["L"]
        # committed rows: the prompt, then every emitted token but the last
        # (the root, not yet in the cache)
        assert L == n + len(out) - 1
        seq_tok = np.concatenate([np.asarray(tokens, dtype=np.int64),
                                  np.asarray(out[:-1], dtype=np.int64)])
        is_vis = np.concatenate([np.asarray(vis_flags, dtype=bool),
                                 np.zeros(len(out) - 1, dtype=bool)])
        vrows = [None] * L
        vi = 0
        for i in range(n):
            if is_vis[i]:
                vrows[i] = visual[vi]
                vi += 1
        x = M.embed_rows(m.w, seq_tok, vrows)
        kv = M.KVCache(m.dims.n_layers, L, m.dims.n_kv_heads, m.dims.head_dim)
        pos = np.arange(L, dtype=np.int32)
        h, _ = M.target_forward(m.dims, m.w, kv, x, pos, pos, 0, L, None, want_logits=False)
        f = decoupled_inputs(m, x, is_vis, h, out[-1], visual_input)
        dkv = M.KVCache(1, L, m.dims.n_kv_heads, m.dims.head_dim)
        feats = M.layer_forward(m.dims, m.draft["layer"], dkv.k[0], dkv.v[0], f, pos, pos,
                                0, L, None)
        assert np.array_equal(trace["root_feat"], feats[-1]), cycle
        assert np.array_equal(st.dkv.k[:, :L], dkv.k), cycle
        assert np.array_equal(st.dkv.v[:, :L], dkv.v), cycle
        assert np.array_equal(st.kv.k[:, :L], kv.k), cycle
        h_t, logits = O.verify(m, st, tree)
        _, emitted, _ = O.accept_and_compact(m, st, tree, h_t, np.argmax(logits, axis=1))
        out.extend(emitted)


# ---- dynamic beam against a brute force over all paths ---------------------

def path_logits(path, V, seed):
    """Deterministic draft logits for the node reached by `path` (tie-free)."""
    h = hash((seed, V) + tuple(int(t) for t in path)) & 0xFFFFFFFF
    return np.random.default_rng(h).standard_normal(V) * 2.0


def brute_beam(V, K, D, N, seed):
    """The beam of the dynamic tree, by its set definition.

    Returns the kept paths in canonical order (depth, then rank path
    lexicographic) with their cumulative log-probabilities.
    """
    lq = {}      # path -> log-prob of its last token under its parent's draft
    rank = {}    # path -> rank of its last token among the parent's children
    for d in range(1, D + 1):
        for p in itertools.product(range(V), repeat=d):
            row = sp_log_softmax(path_logits(p[:-1], V, seed))
            lq[p] = row[p[-1]]
            order = np.lexsort((np.arange(V), -row))
            rank[p] = int(np.nonzero(order == p[-1])[0][0])
    score = {p: sum(lq[p[:i]] for i in range(1, len(p) + 1)) for p in lq}

    def children(p):
        return [c for c in lq if len(c) == len(p) + 1 and c[:-1] == p and rank[c] < K]

    def rank_path(p):
        return tuple(rank[p[:i]] for i in range(1, len(p) + 1))

    frontier = children(())
    pool = list(frontier)
    for d in range(2, D + 1):
        cand = [c for p in frontier for c in children(p)]
        pool += cand
        cand.sort(key=lambda c: (-score[c], rank_path(c)))
        frontier = cand[:K]
    pool.sort(key=lambda c: (-score[c], len(c), rank_path(c)))
    kept = pool[:N]
    kept.sort(key=lambda c: (len(c), rank_path(c)))
    return kept, score


@pytest.mark.parametrize("V,K,D,N", [(8, 3, 3, 5), (8, 3, 3, 21), (12, 3, 3, 9),
                                     (16, 3, 3, 12), (10, 2, 4, 8), (9, 3, 3, 1)])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_dynamic_tree_matches_brute_force_beam(V, K, D, N, seed):
    kept, score = brute_beam(V, K, D, N, seed)

    def expand(ids, parents, tokens, d):
        return [path_logits(paths[i], V, seed) for i in ids]

    paths = {}  # the oracle's pool index -> token path
    root_logits = path_logits((), V, seed)

    def expand_tracking(ids, parents, tokens, d):
        for i, p, t in zip(ids, parents, tokens):
            paths[i] = (paths[p] if p >= 0 else ()) + (int(t),)
        return expand(ids, parents, tokens, d)

    tree, pool = O.select_dynamic_tree(K, D, N, 99, root_logits, expand_tracking)
    got = []
    for u in range(tree.n):
        p, x = [], u
        while x > 0:
            p.append(int(tree.token[x]))
            x = int(tree.parent[x])
        got.append(tuple(reversed(p)))
    assert got[0] == () and tree.parent[0] == -1 and tree.token[0] == 99
    assert got[1:] == kept
    for u in range(1, tree.n):
        assert tree.depth[u] == len(got[u])
        assert got[tree.parent[u]] == got[u][:-1]
        assert abs(tree.score[u] - score[got[u]]) <= 1e-12 * max(1.0, abs(score[got[u]]))
    # the pool holds K nodes at depth 1 and K*K at each further depth
    depths = [d for (_, _, d, _) in pool]
    assert depths.count(1) == K and all(depths.count(d) == K * K for d in range(2, D + 1))


@pytest.mark.parametrize("scale", [1.0, 30.0, 800.0])
def test_log_softmax_matches_scipy(scale):
    rng = np.random.default_rng(int(scale))
    for n in (1, 2, 17, 4096):
        x = rng.standard_normal(n) * scale
        got = O.log_softmax(x)
        want = sp_log_softmax(x)
        assert np.allclose(got, want, rtol=1e-13, atol=1e-13 * max(1.0, scale))
        assert abs(np.sum(np.exp(got)) - 1.0) < 1e-12
