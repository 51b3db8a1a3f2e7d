"""Pins for tree selection, greedy acceptance, compaction and the metrics.

Checked against brute-force enumeration, the paper's general stochastic
acceptance rule specialised to a one-hot target, out-of-place copies and a
Monte-Carlo estimate -- never against the oracle's own formulation.
"""
import itertools

import numpy as np
import pytest

import synth
from synth.configs import STATIC_26, full_tree_paths
from oracle import metrics
from oracle import model as M
from oracle import msd as O


def hashed_logits(path, V, seed=0):
    """Deterministic pseudo-random draft logits for a token path."""
    h = hash((seed,) + tuple(int(t) for t in path)) & 0xFFFFFFFF
    return np.random.default_rng(h).standard_normal(V) * 2.0


def full_rank(values):
    # rank by value descending, ties by id ascending, via lexsort on (id, -value)
    return np.lexsort((np.arange(len(values)), -np.asarray(values)))


def node_paths(tree):
    out = []
    for u in range(tree.n):
        p, x = [], u
        while x > 0:
            p.append(int(tree.token[x]))
            x = int(tree.parent[x])
        out.append(tuple(reversed(p)))
    return out


@pytest.mark.parametrize("paths", [STATIC_26, full_tree_paths(3, 2), ["0", "00", "000"]],
                         ids=["static26", "binary3", "chain3"])
def test_static_tree_brute_force(paths):
    V, root = 50, 7
    parent, rank, depth = synth.static_tree_arrays(paths)
    calls = []

    def expand(nodes, tokens, d):
        calls.append((d, list(nodes)))
        return [hashed_logits(tree_paths[u], V) for u in nodes]

    # token paths for expanded nodes are known once their ancestors are assigned
    tree_paths = {}

    def expand_tracking(nodes, tokens, d):
        for u in nodes:
            p, x = [], u
            while x > 0:
                p.append(int(tok_now[x]))
                x = int(parent[x])
            tree_paths[u] = tuple(reversed(p))
        return expand(nodes, tokens, d)

    tok_now = np.zeros(len(parent), dtype=np.int64)

    def wrapped(nodes, tokens, d):
        for u, t in zip(nodes, tokens):
            tok_now[u] = t
        return expand_tracking(nodes, tokens, d)

    tree = O.select_static_tree(parent, rank, depth, root, hashed_logits((), V), wrapped)
    paths_tok = node_paths(tree)
    for c in range(1, tree.n):
        prefix = paths_tok[c][:-1]
        order = full_rank(hashed_logits(prefix, V))
        assert tree.token[c] == order[rank[c]]
    # siblings distinct, parents first, depth consistent
    for c in range(1, tree.n):
        assert tree.parent[c] < c and tree.depth[c] == tree.depth[tree.parent[c]] + 1
    for p in range(tree.n):
        kids = [int(tree.token[c]) for c in range(tree.n) if tree.parent[c] == p]
        assert len(kids) == len(set(kids))
    # only nodes with children are run through the draft, depth by depth
    assert [d for d, _ in calls] == sorted(d for d, _ in calls)


def test_topk_ties_prefer_lower_id():
    v = np.array([1.0, 3.0, 3.0, 2.0, 3.0])
    assert list(O.topk_desc(v, 4)) == [1, 2, 4, 3]


def brute_dynamic_depth2(V, N, root_lq, child_lq):
    """All paths of length <= 2 ranked by cumulative log-prob."""
    cands = [((a,), root_lq[a]) for a in range(V)]
    cands += [((a, b), root_lq[a] + child_lq[a][b]) for a in range(V) for b in range(V)]
    cands.sort(key=lambda c: -c[1])
    return set(p for p, _ in cands[:N])


@pytest.mark.parametrize("N", [1, 5, 17, 30])
def test_dynamic_tree_full_beam_is_global_topN(N):
    V, K, D = 5, 5, 2
    rl = np.random.default_rng(1).standard_normal(V) * 2
    root_lq = O.log_softmax(rl)
    child_raw = {a: np.random.default_rng(10 + a).standard_normal(V) * 2 for a in range(V)}
    child_lq = {a: O.log_softmax(child_raw[a]) for a in range(V)}
    pool_tok = {}

    def expand(ids, parents, tokens, d):
        assert d == 1
        return [child_raw[t] for t in tokens]
    tree, pool = O.select_dynamic_tree(K, D, N, 99, rl, expand)
    got = set(node_paths(tree)[1:])
    assert got == brute_dynamic_depth2(V, N, root_lq, child_lq)
    # scores are cumulative log-probs
    for u in range(1, tree.n):
        p = node_paths(tree)[u]
        want = root_lq[p[0]] + (child_lq[p[0]][p[1]] if len(p) == 2 else 0.0)
        assert np.isclose(tree.score[u], want, atol=1e-12)


def test_dynamic_tree_beam_properties():
    V, K, D, N = 12, 3, 4, 10
    rl = hashed_logits((), V, 5)

    def expand(ids, parents, tokens, d):
        return [hashed_logits((i,), V, 5) for i in ids]
    tree, pool = O.select_dynamic_tree(K, D, N, 0, rl, expand)
    assert tree.n == N + 1
    kept = sorted(tree.score[1:], reverse=True)
    dropped_best = max(s for (_, _, _, s) in pool if s not in set(tree.score[1:]))
    assert kept[-1] >= dropped_best
    for u in range(1, tree.n):
        assert tree.parent[u] < u
        assert tree.depth[u] == tree.depth[tree.parent[u]] + 1
        if u > 1:
            assert (tree.depth[u - 1], 0) <= (tree.depth[u], 0)
    # per depth at most K frontier nodes were expanded
    depths = [d for (_, _, d, _) in pool]
    for d in range(2, D + 1):
        assert depths.count(d) == K * K


def paper_chain_verify(tokens, p_rows, q_rows, u):
    """Sequential speculative sampling on one branch (Sec. 3.2 verification).

    Token n is accepted with probability min(1, p/q); on the first rejection
    the replacement is drawn from norm(max(0, p - q)); after a fully accepted
    branch one more token is drawn from p.  u: uniforms.
    """
    out = []
    for n, t in enumerate(tokens):
        p, q = p_rows[n], q_rows[n]
        if u[2 * n] < min(1.0, p[t] / q[t]):
            out.append(int(t))
            continue
        r = np.maximum(0.0, p - q)
        r = r / r.sum()
        out.append(int(np.searchsorted(np.cumsum(r), u[2 * n + 1])))
        return out, n
    p = p_rows[len(tokens)]
    out.append(int(np.searchsorted(np.cumsum(p), u[-1])))
    return out, len(tokens)


@pytest.mark.parametrize("seed", range(20))
def test_greedy_accept_matches_paper_rule_with_one_hot_target(seed):
    rng = np.random.default_rng(seed)
    V = 6
    parent, rank, depth = synth.static_tree_arrays(full_tree_paths(3, 2))
    T = len(parent)
    token = np.zeros(T, dtype=np.int32)
    for c in range(1, T):
        sib = [int(token[s]) for s in range(1, c) if parent[s] == parent[c]]
        token[c] = rng.choice([t for t in range(V) if t not in sib])
    tree = O.Tree(token, parent, depth, np.zeros(T))
    amax = rng.integers(0, V, T).astype(np.int32)
    # bias toward acceptance so long paths occur
    for c in range(1, T):
        if rng.random() < 0.6 and all(token[s] != amax[parent[c]] for s in range(1, T)
                                      if parent[s] == parent[c] and s != c):
            amax[parent[c]] = token[c]
    path, emitted = O.greedy_accept(tree, amax)
    onehot = np.eye(V)
    best = None
    for leaf in range(T):
        if any(parent[c] == leaf for c in range(T)):
            continue
        br = []
        x = leaf
        while x > 0:
            br.append(x)
            x = int(parent[x])
        br.reverse()
        q_rows = [rng.dirichlet(np.ones(V)) for _ in br]
        p_rows = [onehot[amax[0]]] + [onehot[amax[u]] for u in br]
        out, n_acc = paper_chain_verify(token[br], p_rows, q_rows, rng.random(2 * len(br) + 1))
        if best is None or n_acc > best[0]:
            best = (n_acc, out)
    assert len(path) - 1 == best[0]
    assert emitted == best[1]


def test_compaction_in_place_matches_out_of_place():
    L, T, S = 10, 8, 24
    kv = M.KVCache(3, S, 2, 4)
    rng = np.random.default_rng(0)
    kv.k[:, :L + T] = rng.standard_normal((3, L + T, 2, 4))
    kv.v[:, :L + T] = rng.standard_normal((3, L + T, 2, 4))
    kv.k[:, L + T:] = np.nan
    kv.v[:, L + T:] = np.nan
    for path in ([0], [0, 2, 3], [0, 1, 5, 7], [0, 3, 4, 6]):
        c = kv.copy()
        ref_k = kv.k[:, [L + j for j in path]].copy()
        ref_v = kv.v[:, [L + j for j in path]].copy()
        slot_map = O.compact_kv(c, L, path)
        assert list(slot_map) == [L + j for j in path]
        assert np.array_equal(c.k[:, L:L + len(path)], ref_k)
        assert np.array_equal(c.v[:, L:L + len(path)], ref_v)
        assert np.array_equal(c.k[:, :L], kv.k[:, :L])
        assert np.isnan(c.k[:, L + T:]).all()


@pytest.mark.parametrize("gamma,alpha", [(1, 0.5), (4, 0.8), (5, 0.3), (3, 1.0), (6, 0.0)])
def test_omega_matches_monte_carlo(gamma, alpha):
    rng = np.random.default_rng(gamma)
    n = 200000
    acc = rng.random((n, gamma)) < alpha
    # tokens per verification: accepted prefix + the one from the target
    first_rej = np.where(acc.all(axis=1), gamma, np.argmin(acc, axis=1))
    mc = (first_rej + 1).mean()
    assert abs(metrics.omega(gamma, alpha) - mc) < 0.02
    assert np.isclose(metrics.omega(gamma, alpha), sum(alpha ** i for i in range(gamma + 1)))


def test_speedup_ratio_limits():
    # no acceptance and free drafting: verification costs what a step costs
    assert np.isclose(metrics.speedup_ratio(100, 1.0, 0.0, 1.0, 4, 0.0, 0.0), 1.0)
    # perfect acceptance, free drafting, verify == one step -> gamma + 1
    assert np.isclose(metrics.speedup_ratio(100, 1.0, 0.0, 1.0, 4, 1.0, 0.0), 5.0)


def test_n_alpha_counts_and_iid_limit():
    # hand count: cycles accepting 0, 1, 3, 3 of a 3-token chain
    assert metrics.n_alpha([0, 1, 3, 3], 3) == [3 / 4, 2 / 3, 2 / 2]
    assert metrics.n_alpha([0, 0], 2) == [0.0, None]
    # independent acceptance with probability alpha at every position: each
    # n-alpha estimates alpha, and the mean emitted tokens is omega
    rng = np.random.default_rng(5)
    alpha, gamma = 0.6, 5
    acc = []
    for _ in range(40000):
        a = 0
        while a < gamma and rng.random() < alpha:
            a += 1
        acc.append(a)
    for v in metrics.n_alpha(acc, gamma):
        assert abs(v - alpha) < 0.02
    assert abs(np.mean(acc) + 1 - metrics.omega(gamma, alpha)) < 0.02

