"""Oracle: the MSD decode loop at temperature 0 (float64).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

One cycle (Sec. 3.2 and Sec. 4.1):
  1. draft catch-up: the pending rows (decoupled inputs, Eq. decouple) run
     through the draft layer; the last row's predicted feature gives the
     draft distribution for the first drafted token;
  2. draft tree: depth by depth, every node that gets children is fed back as
     f_down(Concat(predicted feature of its parent, embedding of its token)),
     with tree-structured attention over the draft cache and its ancestors;
     children are the parent's top-ranked tokens (static shape) or the best
     cumulative log-probabilities (dynamic shape);
  3. verification: the target runs once over [root, drafted nodes] with the
     ancestor mask; at temperature 0 the target distribution is one-hot at
     its argmax, so min(1, p/q) accepts a node exactly when its token is the
     parent's argmax, and the adjusted distribution norm(max(0, p - q)) after
     a rejection (Eq. padjusted) and the extra sample after full acceptance
     are both that argmax: the bonus token;
  4. the longest accepted root-to-node path is kept: its cache rows are moved
     to consecutive slots, and its target features become the next pending
     draft rows.
Ties: top-k ranks by value descending, then token id ascending; argmax takes
the lowest id among equal maxima.
"""
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from . import model as M


def topk_desc(values, k):
    """Indices of the k largest values, ties broken by the lower index."""
    return np.argsort(-np.asarray(values, dtype=np.float64), kind="stable")[:k]


def log_softmax(logits):
    m = np.max(logits)
    return logits - (m + np.log(np.sum(np.exp(logits - m))))


def ancestor_masks(parent):
    """anc[i] has bit j set iff node j is node i or one of its ancestors."""
    T = len(parent)
    assert T <= 64
    anc = np.zeros(T, dtype=np.uint64)
    for i in range(T):
        p = int(parent[i])
        assert p < i, "parents must precede children"
        anc[i] = (anc[p] if p >= 0 else np.uint64(0)) | np.uint64(1 << i)
    return anc


@dataclass
class Tree:
    token: np.ndarray      # int32 [T], node 0 = root
    parent: np.ndarray     # int32 [T], -1 for the root
    depth: np.ndarray      # int32 [T]
    score: np.ndarray      # float64 [T] (cumulative draft log-prob; 0 for static)

    @property
    def n(self):
        return len(self.token)

    @property
    def anc(self):
        return ancestor_masks(self.parent)


@dataclass
class PendingRow:
    is_visual: bool
    h: Optional[np.ndarray] = None         # target feature of the row (text)
    e_next: Optional[np.ndarray] = None    # embedding of the following token (text)
    # the draft input of a visual row: its own embedding (Eq. decouple), or
    # its target feature in the Visual Feature variant (Sec. 5.3)
    e_visual: Optional[np.ndarray] = None


@dataclass
class SeqState:
    kv: M.KVCache
    dkv: M.KVCache
    L: int                       # committed target (and draft) length
    root: int                    # last emitted token, not yet in the cache
    pending: List[PendingRow] = field(default_factory=list)


class Models:
    def __init__(self, dims, weights, draft=None):
        self.dims, self.w, self.draft = dims, weights, draft

    def embed(self, token):
        return M.widen(self.w["embed"][int(token)])


VISUAL_INPUTS = ("embedding", "feature")


def prefill(m: Models, tokens, is_visual, visual, max_slots, visual_input="embedding"):
    """Target forward over the prompt; returns (state, first generated token).

    visual_input selects the draft input of the visual rows.  "embedding" is
    the method's decoupled input (Eq. decouple): a visual row enters the draft
    as its own embedding e_v.  "feature" is the Visual Feature variant of the
    input-decoupling ablation (Sec. 5.3, Table decouple_input): a visual row
    enters as the target's feature h_v of that row (the final-norm output,
    the same feature the text rows concatenate), with no next-token
    concatenation and no f_down.
    """
    if visual_input not in VISUAL_INPUTS:
        raise ValueError(f"visual_input must be one of {VISUAL_INPUTS}")
    dims = m.dims
    n = len(tokens)
    is_visual = np.asarray(is_visual, dtype=bool)
    if n == 0 or is_visual[-1]:
        raise ValueError("prompt must be non-empty and end in a text token")
    vis_rows = [None] * n
    vi = 0
    for i in range(n):
        if is_visual[i]:
            vis_rows[i] = visual[vi]
            vi += 1
    x = M.embed_rows(m.w, tokens, vis_rows)
    kv = M.KVCache(dims.n_layers, max_slots, dims.n_kv_heads, dims.head_dim)
    dkv = M.KVCache(1, max_slots, dims.n_kv_heads, dims.head_dim)
    pos = np.arange(n, dtype=np.int32)
    h, logits = M.target_forward(dims, m.w, kv, x, pos, pos, 0, n, None)
    first = int(np.argmax(logits[n - 1]))
    st = SeqState(kv=kv, dkv=dkv, L=n, root=first)
    for i in range(n):
        if is_visual[i]:
            src = x[i] if visual_input == "embedding" else h[i]
            st.pending.append(PendingRow(True, e_visual=src.copy()))
        else:
            e_next = x[i + 1].copy() if i + 1 < n else m.embed(first)
            st.pending.append(PendingRow(False, h=h[i].copy(), e_next=e_next))
    return st, first, h, logits


def draft_catch_up(m: Models, st: SeqState):
    """Runs the pending rows through the draft; returns the last predicted feature."""
    dims, d = m.dims, m.dims.d_model
    r = len(st.pending)
    L0 = st.L - r
    hh = np.zeros((r, d)); en = np.zeros((r, d)); ev = np.zeros((r, d))
    vis = np.zeros(r, dtype=bool)
    for j, p in enumerate(st.pending):
        vis[j] = p.is_visual
        if p.is_visual:
            ev[j] = p.e_visual
        else:
            hh[j], en[j] = p.h, p.e_next
    f = M.draft_input(m.draft, hh, en, vis, ev)
    pos = np.arange(L0, L0 + r, dtype=np.int32)
    out = M.draft_forward(dims, m.draft, st.dkv, f, pos, pos, L0, r, None)
    st.pending = []
    return out[-1].copy()


def select_static_tree(parent, rank, depth, root_token, root_logits, expand):
    """Static shape: node c is the rank[c]-th best token of its parent's draft.

    expand(nodes, tokens_of_nodes, depth) -> draft logits rows for those nodes
    (called depth by depth, for the nodes that have children, in node order).
    """
    T = len(parent)
    token = np.zeros(T, dtype=np.int32)
    token[0] = root_token
    D = int(np.max(depth))
    has_kids = np.zeros(T, dtype=bool)
    has_kids[np.asarray(parent[1:], dtype=np.int64)] = True

    def assign(u, logits):
        kids = [c for c in range(T) if parent[c] == u]
        order = topk_desc(logits, max(int(rank[c]) for c in kids) + 1)
        for c in kids:
            token[c] = order[rank[c]]

    assign(0, root_logits)
    for d in range(1, D):
        nodes = [u for u in range(T) if depth[u] == d and has_kids[u]]
        if not nodes:
            continue
        rows = expand(nodes, [int(token[u]) for u in nodes], d)
        for j, u in enumerate(nodes):
            assign(u, rows[j])
    return Tree(token=token, parent=np.asarray(parent, dtype=np.int32),
                depth=np.asarray(depth, dtype=np.int32), score=np.zeros(T))


def select_dynamic_tree(K, D, N, root_token, root_logits, expand):
    """Dynamic shape: top-K per node, top-K frontier per depth, top-N overall.

    A candidate's score is its cumulative draft log-probability (sum of
    log-softmax values along its path).  Depth 1 holds the root's top-K; at
    each further depth every frontier node gets its top-K children, and the
    best K of those K*K candidates become the next frontier (expanded in
    creation order).  The tree keeps the best N candidates of the whole pool.
    Every ranking is by score descending, then creation index ascending.
    expand(pool_ids, parent_pool_ids, tokens, depth) -> draft logits rows.
    Returns (tree, pool) where pool lists (parent, token, depth, score).
    """
    pool = []  # (parent pool index or -1, token, depth, score)

    def add(par, tok, dep, sc):
        pool.append((par, int(tok), dep, float(sc)))
        return len(pool) - 1

    lq = log_softmax(np.asarray(root_logits, dtype=np.float64))
    frontier = [add(-1, t, 1, lq[t]) for t in topk_desc(lq, K)]
    for d in range(2, D + 1):
        frontier = sorted(frontier)
        rows = expand(frontier, [pool[u][0] for u in frontier],
                      [pool[u][1] for u in frontier], d - 1)
        new = []
        for j, u in enumerate(frontier):
            lq = log_softmax(np.asarray(rows[j], dtype=np.float64))
            for t in topk_desc(lq, K):
                new.append(add(u, t, d, pool[u][3] + lq[t]))
        sc = np.array([pool[i][3] for i in new])
        frontier = [new[i] for i in topk_desc(sc, K)]
    keep = topk_desc(np.array([p[3] for p in pool]), N)
    keep = sorted((int(i) for i in keep), key=lambda i: (pool[i][2], i))
    index = {-1: 0}
    for j, i in enumerate(keep, start=1):
        index[i] = j
    T = len(keep) + 1
    token = np.zeros(T, dtype=np.int32); token[0] = root_token
    parent = np.full(T, -1, dtype=np.int32)
    depth = np.zeros(T, dtype=np.int32)
    score = np.zeros(T)
    for i in keep:
        par, tok, dep, sc = pool[i]
        assert par in index, "selected node without its parent"
        j = index[i]
        token[j], parent[j], depth[j], score[j] = tok, index[par], dep, sc
    return Tree(token=token, parent=parent, depth=depth, score=score), pool


class _DraftExpander:
    """Runs tree nodes through the draft head (Sec. 3.2 tree drafting).

    Each expanded node gets the next free draft-cache slot L + e (e = order of
    expansion) and sees the committed draft cache plus its expanded ancestors.
    A node's input is f_down(Concat(parent's predicted feature, e(token))).
    """

    def __init__(self, m: Models, st: SeqState, root_feat):
        self.m, self.st = m, st
        self.feat = {None: root_feat}
        self.slot, self.mask = {}, {}
        self.path = {None: ()}   # token path from the root, for inspection only

    def __call__(self, keys, parent_keys, tokens, depth):
        m, st = self.m, self.st
        for k, pk, t in zip(keys, parent_keys, tokens):
            self.path[k] = self.path[pk] + (int(t),)
            self.slot[k] = len(self.slot)
            a = np.uint64(1 << self.slot[k])
            if pk is not None:
                a |= self.mask[pk]
            self.mask[k] = a
        pf = np.stack([self.feat[pk] for pk in parent_keys])
        e = np.stack([m.embed(t) for t in tokens])
        f = M.draft_input(m.draft, pf, e, np.zeros(len(keys), dtype=bool), None)
        pos = np.full(len(keys), st.L + depth - 1, dtype=np.int32)
        slots = st.L + np.array([self.slot[k] for k in keys], dtype=np.int64)
        R = max(self.slot[k] for k in keys) + 1
        out = M.draft_forward(m.dims, m.draft, st.dkv, f, pos, slots, st.L, R,
                              np.array([self.mask[k] for k in keys], dtype=np.uint64))
        for j, k in enumerate(keys):
            self.feat[k] = out[j]
        return M.linear(out, m.w["lm_head"])


def draft_tree(m: Models, st: SeqState, shape, static_arrays=None, trace=None):
    """Catch-up on the pending rows, then the draft tree for this cycle.

    trace: optional dict that receives, for inspection, the committed length
    L, the root feature (the catch-up's last predicted feature) and the
    predicted feature of every expanded node keyed by its token path from the
    root (a tuple of drafted tokens).
    """
    root_feat = draft_catch_up(m, st)
    root_logits = M.linear(root_feat[None, :], m.w["lm_head"])[0]
    ex = _DraftExpander(m, st, root_feat)
    if shape.kind == "static":
        parent, rank, depth = static_arrays

        def expand(nodes, tokens, d):
            pk = [None if parent[u] == 0 else int(parent[u]) for u in nodes]
            return ex(list(nodes), pk, tokens, d)
        tree = select_static_tree(parent, rank, depth, st.root, root_logits, expand)
    else:
        def expand_dyn(ids, parents, tokens, d):
            return ex(list(ids), [None if p < 0 else p for p in parents], tokens, d)
        tree, _ = select_dynamic_tree(shape.topk, shape.depth, shape.n_nodes, st.root,
                                      root_logits, expand_dyn)
    if trace is not None:
        trace["L"] = st.L
        trace["root_feat"] = root_feat
        trace["root_logits"] = root_logits
        trace["feat"] = {ex.path[k]: ex.feat[k] for k in ex.feat if k is not None}
    return tree


def verify(m: Models, st: SeqState, tree: Tree):
    """Target forward over the tree; node i at position L + depth[i], slot L + i."""
    T = tree.n
    x = M.embed_rows(m.w, tree.token)
    pos = (st.L + tree.depth).astype(np.int32)
    slots = st.L + np.arange(T)
    return M.target_forward(m.dims, m.w, st.kv, x, pos, slots, st.L, T, tree.anc)


def greedy_accept(tree: Tree, amax):
    """Longest root-to-node path whose every token is its parent's argmax.

    Returns (path of node indices starting at the root, emitted tokens =
    accepted drafted tokens followed by the bonus token amax[last]).
    """
    T = tree.n
    ok = np.zeros(T, dtype=bool)
    ok[0] = True
    for j in range(1, T):
        p = tree.parent[j]
        ok[j] = ok[p] and tree.token[j] == amax[p]
    best = 0
    for j in range(T):
        if ok[j] and tree.depth[j] > tree.depth[best]:
            best = j
    path = []
    u = best
    while u >= 0:
        path.append(int(u))
        u = int(tree.parent[u])
    path.reverse()
    emitted = [int(tree.token[u]) for u in path[1:]] + [int(amax[best])]
    return path, emitted


def compact_kv(kv: M.KVCache, L, path):
    """Moves cache rows L + path[j] to L + j (all reads before any write).

    Returns the slot map: slot_map[j] = L + path[j].
    """
    src = L + np.asarray(path, dtype=np.int64)
    kv.k[:, L:L + len(path)] = kv.k[:, src].copy()
    kv.v[:, L:L + len(path)] = kv.v[:, src].copy()
    return src.astype(np.int32)


def accept_and_compact(m: Models, st: SeqState, tree: Tree, h_tree, amax):
    path, emitted = greedy_accept(tree, amax)
    slot_map = compact_kv(st.kv, st.L, path)
    nxt = emitted  # token following path[j] is emitted[j]
    st.pending = [PendingRow(False, h=h_tree[u].copy(), e_next=m.embed(nxt[j]))
                  for j, u in enumerate(path)]
    st.L += len(path)
    st.root = emitted[-1]
    return path, emitted, slot_map


def msd_generate(m: Models, prompt, shape, n_new, static_arrays=None, max_slots=None,
                 record=False, visual_input="embedding"):
    """Speculative greedy decoding; returns (tokens[n_new], per-cycle records)."""
    tokens, is_visual, visual = prompt
    T = (shape.n_draft + 1)
    max_slots = max_slots or (len(tokens) + n_new + 2 * T + 8)
    st, first, _, _ = prefill(m, tokens, is_visual, visual, max_slots, visual_input)
    out = [first]
    cycles = []
    while len(out) < n_new:
        tree = draft_tree(m, st, shape, static_arrays)
        L = st.L
        h, logits = verify(m, st, tree)
        amax = np.argmax(logits, axis=1).astype(np.int32)
        path, emitted, slot_map = accept_and_compact(m, st, tree, h, amax)
        out.extend(emitted)
        rec = {"L": L, "n_accepted": len(path) - 1, "emitted": emitted}
        if record:
            rec.update(tree=tree, logits=logits, amax=amax, path=path, slot_map=slot_map)
        cycles.append(rec)
    return out[:n_new], cycles


def greedy_generate(m: Models, prompt, n_new, max_slots=None, return_logits=False):
    """Plain greedy decoding of the target: the sequence MSD must reproduce.

    With return_logits, also returns the logits row each token was chosen from.
    """
    tokens, is_visual, visual = prompt
    max_slots = max_slots or (len(tokens) + n_new + 8)
    st, first, _, lg = prefill(m, tokens, is_visual, visual, max_slots)
    out = [first]
    rows = [lg[-1]]
    while len(out) < n_new:
        x = M.embed_rows(m.w, [out[-1]])
        pos = np.array([st.L], dtype=np.int32)
        _, logits = M.target_forward(m.dims, m.w, st.kv, x, pos, pos, st.L, 1, None)
        st.L += 1
        out.append(int(np.argmax(logits[0])))
        rows.append(logits[0])
    return (out, np.stack(rows)) if return_logits else out
