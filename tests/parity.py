"""Shared tolerances for GPU-versus-oracle comparisons.

Float results: |gpu - oracle| <= RTOL * max|oracle row| per row (bf16 weights
and activations with float32 accumulation against a float64 oracle).
Integer decisions taken from floats (argmax, top-k) must agree wherever the
oracle's margin between the competing values exceeds the same tolerance.
"""
import numpy as np

RTOL = 2e-2


def row_close(gpu, ref, rtol=RTOL):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    scale = np.abs(ref).max(axis=-1, keepdims=True)
    err = np.abs(gpu - ref)
    ok = err <= rtol * scale
    return bool(ok.all()), float((err / np.maximum(scale, 1e-30)).max())


def decided(row, rtol=RTOL):
    """True when the top-2 margin of an oracle logits row exceeds the tolerance."""
    s = np.sort(np.asarray(row, dtype=np.float64))[::-1]
    return (s[0] - s[1]) > rtol * np.abs(row).max()


def argmax_ok(g, row, rtol=RTOL):
    """The GPU's greedy token g is valid for an oracle logits row: it is the
    oracle's argmax, or (at an undecided row) its oracle logit lies within the
    tolerance band below the row's maximum."""
    row = np.asarray(row, dtype=np.float64)
    return bool(0 <= int(g) < len(row) and row[int(g)] >= row.max() - rtol * np.abs(row).max())


def rank_decided(row, r, rtol=RTOL):
    """True when the r-th and (r+1)-th best values are separated (top-k boundary)."""
    s = np.sort(np.asarray(row, dtype=np.float64))[::-1]
    tol = rtol * np.abs(row).max()
    lo = (s[r - 1] - s[r]) > tol if r > 0 else True
    hi = (s[r] - s[r + 1]) > tol if r + 1 < len(s) else True
    return lo and hi


# --- trees: GPU results against the oracle's own selection -----------------------------

def log_softmax(row):
    row = np.asarray(row, dtype=np.float64)
    m = row.max()
    return row - (m + np.log(np.exp(row - m).sum()))


def gpu_tree_arrays(g):
    """(token, parent, depth, score) numpy arrays of a ctypes msd_tree."""
    n = g.n_nodes
    return (np.array(g.token[:n], dtype=np.int32), np.array(g.parent[:n], dtype=np.int32),
            np.array(g.depth[:n], dtype=np.int32), np.array(g.score[:n], dtype=np.float64))


def check_tree_invariants(g):
    """Canonical order, depth, ancestor masks, distinct siblings, monotone scores."""
    tok, par, dep, sc = gpu_tree_arrays(g)
    n = g.n_nodes
    assert par[0] == -1 and dep[0] == 0 and int(g.anc[0]) == 1
    for c in range(1, n):
        p = int(par[c])
        assert 0 <= p < c, (c, p)
        assert dep[c] == dep[p] + 1 and dep[c] >= dep[c - 1]
        assert int(g.anc[c]) == int(g.anc[p]) | (1 << c)
    for p in range(n):
        kids = [int(tok[c]) for c in range(1, n) if par[c] == p]
        assert len(kids) == len(set(kids)), ("duplicate siblings", p)


def compare_static_tree(g, ref, logs, rank, rtol=RTOL):
    """Static tree: structure bit-exact; node c's token equal to the oracle's
    wherever the oracle's rank boundary at c is decided (descendants of an
    undecided node are skipped).  Returns the number of nodes compared."""
    assert g.n_nodes == ref.n
    assert list(g.parent[:ref.n]) == list(ref.parent)
    assert list(g.depth[:ref.n]) == list(ref.depth)
    assert [int(x) for x in g.anc[:ref.n]] == [int(x) for x in ref.anc]
    assert g.token[0] == ref.token[0]
    skip, checked = set(), 0
    for c in range(1, ref.n):
        p = int(ref.parent[c])
        if p in skip:
            skip.add(c)
            continue
        if g.token[c] != ref.token[c]:
            assert not rank_decided(logs[p], int(rank[c]), rtol), (c, g.token[c], ref.token[c])
            # a gated node: the GPU's token must itself sit in the near-tie
            # band around the oracle's value at that rank
            row = np.asarray(logs[p], dtype=np.float64)
            s = np.sort(row)[::-1]
            gt = int(g.token[c])
            assert 0 <= gt < len(row)
            assert abs(row[gt] - s[int(rank[c])]) <= 2 * rtol * np.abs(row).max(), \
                (c, gt, row[gt], s[int(rank[c])])
            skip.add(c)
        else:
            checked += 1
    return checked


def dynamic_tree_gated(pool, rows, root_logits, K, N, rtol=RTOL):
    """True when any decision that shapes the oracle's dynamic tree lies
    within the tolerance: adjacent log-probabilities among the top K + 1 of
    an expanded row (membership and creation order), the K-th/(K+1)-th score
    of a depth's candidates (the frontier), or the N-th/(N+1)-th score of the
    pool (the kept nodes)."""
    def gaps(vals, k):
        s = np.sort(np.asarray(vals, dtype=np.float64))[::-1][:k + 1]
        return np.diff(-s)

    for r in [root_logits] + list(rows.values()):
        if (gaps(log_softmax(r), K) <= 2 * rtol * np.abs(r).max()).any():
            return True
    # cumulative tolerance along a path: one per-step tolerance per depth
    steps = [2 * rtol * np.abs(r).max() for r in [root_logits] + list(rows.values())]
    tol = max(steps) * max(p[2] for p in pool)
    scores = np.array([p[3] for p in pool])
    depths = np.array([p[2] for p in pool])
    for d in np.unique(depths):
        sd = np.sort(scores[depths == d])[::-1]
        if len(sd) > K and sd[K - 1] - sd[K] <= 2 * tol:
            return True
    sp = np.sort(scores)[::-1]
    return len(sp) > N and sp[N - 1] - sp[N] <= 2 * tol


def compare_dynamic_tree(g, pool, rows, root_logits, K, N, rtol=RTOL, ref=None):
    """Dynamic tree against the oracle's pool (select_dynamic_tree's output).

    Several trees are correct when draft scores tie within the tolerance, so:
    every GPU node that the oracle also generated carries the oracle's
    cumulative log-probability within the summed per-step tolerance
    (2*rtol*max|logits row| per step, the log-softmax of rows that agree
    within rtol*max|row|); a GPU node the oracle did not select must sit
    within that tolerance of the decision that excluded it (its parent's
    top-K boundary, the frontier boundary at its parent's depth, or the
    top-N boundary of the pool), and so must every oracle node the GPU did
    not select.  When `ref` (the oracle's tree) is given and no decision of
    the oracle lies within the tolerance, the token, parent, depth and
    ancestor arrays must equal the oracle's bit for bit.  Returns (nodes
    equal to the oracle's tree, nodes compared by score)."""
    check_tree_invariants(g)
    assert g.n_nodes == N + 1
    tok, par, dep, sc = gpu_tree_arrays(g)
    lq = {-1: log_softmax(root_logits)}
    rtol_row = {-1: 2 * rtol * np.abs(root_logits).max()}
    for i, r in rows.items():
        lq[i] = log_softmax(r)
        rtol_row[i] = 2 * rtol * np.abs(r).max()
    key_of, tol_of, index = [], [], {}
    for i, (p, t, d, s) in enumerate(pool):
        k = (key_of[p] if p >= 0 else ()) + (t,)
        key_of.append(k)
        tol_of.append((tol_of[p] if p >= 0 else 0.0) + rtol_row[p])
        index[k] = i
    scores = np.array([p[3] for p in pool])
    order = np.argsort(-scores, kind="stable")
    s_N = scores[order[N - 1]]
    s_N1 = scores[order[N]] if len(pool) > N else -np.inf
    depths = np.array([p[2] for p in pool])
    front = {}
    for d in np.unique(depths):
        ids = np.where(depths == d)[0]
        srt = np.sort(scores[ids])[::-1]
        front[int(d)] = (srt[K - 1] if len(srt) >= K else -np.inf,
                         srt[K] if len(srt) > K else -np.inf)
    expanded = set(rows.keys())
    kth = {i: np.sort(v)[::-1][K - 1] for i, v in lq.items()}
    kth1 = {i: np.sort(v)[::-1][K] for i, v in lq.items()}
    ref_keys = set(key_of[i] for i in order[:N])
    gkeys = []
    for c in range(1, g.n_nodes):
        k = (gkeys[par[c] - 1] if par[c] > 0 else ()) + (int(tok[c]),)
        gkeys.append(k)
    if ref is not None:
        # Bit-exact tree indices unless a near tie decided them: either no
        # decision of the oracle is near a tie, or the GPU kept the oracle's
        # nodes and no two kept siblings have log-probabilities within the
        # tolerance (their creation order, hence the node order, is decided).
        order_gated = False
        for k in ref_keys:
            i = index[k]
            p = pool[i][0]
            for k2 in ref_keys:
                i2 = index[k2]
                if i2 != i and pool[i2][0] == p and \
                        abs(lq[p][k[-1]] - lq[p][k2[-1]]) <= rtol_row[p]:
                    order_gated = True
        exact = not dynamic_tree_gated(pool, rows, root_logits, K, N, rtol) or \
            (set(gkeys) == ref_keys and not order_gated)
        if exact:
            assert list(tok) == [int(x) for x in ref.token], "tokens differ with no near tie"
            assert list(par) == [int(x) for x in ref.parent]
            assert list(dep) == [int(x) for x in ref.depth]
            assert [int(x) for x in g.anc[:g.n_nodes]] == [int(x) for x in ref.anc]
            compare_dynamic_tree.exact += 1
    same, scored = 0, 0
    for c, k in enumerate(gkeys, start=1):
        if k in ref_keys:
            same += 1
        i = index.get(k)
        if i is not None:
            assert abs(sc[c] - scores[i]) <= tol_of[i] + 1e-4, (k, sc[c], scores[i], tol_of[i])
            scored += 1
            if k not in ref_keys:       # generated by both, not kept by the oracle
                assert scores[i] >= s_N - 2 * tol_of[i], (k, scores[i], s_N)
            continue
        pk = k[:-1]
        pi = index.get(pk, -1) if pk else -1
        if pk and pi < 0:
            continue                    # the parent is itself a justified divergence
        if pi == -1 or pi in expanded:
            assert lq[pi][k[-1]] >= kth[pi] - rtol_row[pi], ("outside top-K", k)
        else:
            f_k, _ = front[int(pool[pi][2])]
            assert scores[pi] >= f_k - 2 * tol_of[pi] - rtol_row[pi], ("parent off frontier", k)
    gset = set(gkeys)
    for k in ref_keys - gset:
        i = index[k]
        p = pool[i][0]
        near = scores[i] <= s_N1 + 2 * tol_of[i]
        near |= lq[p][k[-1]] <= kth1[p] + rtol_row[p]
        if p >= 0:
            _, f_k1 = front[int(pool[p][2])]
            near |= scores[p] <= f_k1 + 2 * tol_of[p] + rtol_row[p]
        assert near, ("oracle node missing on the GPU without a near tie", k)
    return same, scored


compare_dynamic_tree.exact = 0  # trees compared bit for bit (no gate fired)


def oracle_draft_static(m, st, paths):
    """The oracle's static draft tree with every expanded node's logits row."""
    import synth
    from oracle import model as M
    from oracle import msd as O
    parent, rank, depth = synth.static_tree_arrays(paths)
    root_feat = O.draft_catch_up(m, st)
    root_logits = M.linear(root_feat[None, :], m.w["lm_head"])[0]
    ex = O._DraftExpander(m, st, root_feat)
    logs = {0: root_logits}

    def expand(nodes, tokens, d):
        pk = [None if parent[u] == 0 else int(parent[u]) for u in nodes]
        rows = ex(list(nodes), pk, tokens, d)
        for u, r in zip(nodes, rows):
            logs[u] = r
        return rows
    tree = O.select_static_tree(parent, rank, depth, st.root, root_logits, expand)
    return tree, logs, rank


def oracle_draft_dynamic(m, st, K, D, N):
    """The oracle's dynamic draft tree, its pool and the expanded rows."""
    from oracle import model as M
    from oracle import msd as O
    root_feat = O.draft_catch_up(m, st)
    root_logits = M.linear(root_feat[None, :], m.w["lm_head"])[0]
    ex = O._DraftExpander(m, st, root_feat)
    rows = {}

    def expand(ids, parents, tokens, d):
        out = ex(list(ids), [None if p < 0 else p for p in parents], tokens, d)
        for i, r in zip(ids, out):
            rows[i] = r
        return out
    tree, pool = O.select_dynamic_tree(K, D, N, st.root, root_logits, expand)
    return tree, pool, rows, root_logits


def oracle_tree_of(g):
    """The GPU's tree as an oracle Tree (teacher forcing)."""
    from oracle import msd as O
    tok, par, dep, sc = gpu_tree_arrays(g)
    return O.Tree(token=tok, parent=par, depth=dep, score=sc)


# Speculative sampling: a float32 decision may differ from the float64 one
# only when the oracle's draw lies this close to the threshold.
SAMPLE_GATE = 1e-4


def sampling_agrees(path, emitted, r_path, r_emit, decisions, gate=SAMPLE_GATE):
    """GPU sampling acceptance against the oracle's on the same logits and
    draws: identical, or the first difference follows a decision the oracle
    took within `gate` of its threshold at the last node both paths share."""
    path, emitted = [int(x) for x in path], [int(x) for x in emitted]
    if path == list(r_path) and emitted == list(r_emit):
        return True
    k = 0
    while k < min(len(path), len(r_path)) and path[k] == r_path[k]:
        k += 1
    node = r_path[k - 1]
    return any(d["at"] == node and d["margin"] < gate for d in decisions)

