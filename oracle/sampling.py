"""Oracle: speculative sampling on a draft tree at temperature > 0 (float64).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Sec. 3.2 (verification phase) accepts a drafted token x with probability
min(1, p(x)/q(x)) (Eq. for p_accept), where q is the distribution x was
proposed from; after a rejection the next token comes from the adjusted
distribution norm(max(0, p - q)) (Eq. padjusted); when every drafted token is
accepted one more token is drawn from p.

Tree reading.  The drafted children of a node are the draft's top-ranked
tokens (Sec. 3.2, tree-structured drafting), a deterministic choice, so the
proposal each child stands for is the point mass on its own token.  With
q = delta_x the acceptance probability is p(x) and the adjusted distribution
is p with x removed and renormalised.  Children are tried in node order (rank
order); each rejection removes its token from p before the next child is
tried, and after the last rejection the bonus token is drawn from what is
left.  Walking down from the root, an accepted child becomes the node whose
children are tried next, with the target distribution at that child.  The
emitted tokens are then distributed exactly as plain sampling from the target
(checked by the tests).

Random numbers.  Draw j of the cycle of sequence slot `seq` that starts at
committed length L is the n-th output of SplitMix64 (Steele, Lea and Flood,
2014) started at `seed`, with n = seq * 2^40 + L * 2^8 + j; its top 24 bits
give a uniform on [0, 1).  The GPU side implements the same published
generator on its own.
"""
import numpy as np

_M64 = (1 << 64) - 1
_GAMMA = 0x9E3779B97F4A7C15


def splitmix64(seed, n):
    """Output n (n >= 0) of the SplitMix64 sequence started at `seed`."""
    z = (int(seed) + (int(n) + 1) * _GAMMA) & _M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M64
    return z ^ (z >> 31)


def draw_index(seq, L, j):
    assert 0 <= j < 256 and 0 <= L < (1 << 32) and 0 <= seq < (1 << 24)
    return (int(seq) << 40) | (int(L) << 8) | int(j)


def draw_uniform(seed, seq, L, j):
    """Uniform on [0, 1), a multiple of 2^-24."""
    return (splitmix64(seed, draw_index(seq, L, j)) >> 40) / float(1 << 24)


def target_probs(logits_row, temperature):
    """softmax(logits / temperature), with the maximum subtracted."""
    z = np.asarray(logits_row, dtype=np.float64) / float(temperature)
    e = np.exp(z - z.max())
    return e / e.sum()


def sample_accept(tree, logits, temperature, seed, seq, L):
    """Speculative sampling over one verified tree.

    tree: token/parent arrays (node 0 = root, parents precede children);
    logits: [T][V] target logits of the tree's nodes.  Returns
    (path, emitted, decisions): the accepted root-to-node path, the emitted
    tokens (accepted drafted tokens, then the bonus token), and one record per
    random decision: the node it was taken at and its distance to the
    threshold (relative to the remaining mass for the bonus draw), for gating
    the comparison with a float32 implementation.
    """
    T = len(tree.token)
    children = [[] for _ in range(T)]
    for u in range(1, T):
        children[int(tree.parent[u])].append(u)
    cur, path, j = 0, [0], 0
    decisions = []
    while True:
        p = target_probs(logits[cur], temperature)
        removed = 0.0      # target mass of the rejected children
        rejected = []
        nxt = None
        for u in children[cur]:
            x = int(tree.token[u])
            r = draw_uniform(seed, seq, L, j)
            j += 1
            rem = 1.0 - removed
            ratio = p[x] / rem if rem > 0 else 0.0
            decisions.append({"kind": "child", "at": cur, "child": u, "r": r, "ratio": ratio,
                              "margin": abs(r - ratio)})
            if r < ratio:
                nxt = u
                break
            removed += p[x]
            rejected.append(x)
        if nxt is not None:
            path.append(nxt)
            cur = nxt
            continue
        r = draw_uniform(seed, seq, L, j)
        q = p.copy()
        q[rejected] = 0.0
        cdf = np.cumsum(q)
        total = cdf[-1]
        if total > 0:
            target = r * total
            y = int(np.searchsorted(cdf, target, side="right"))
            lo = cdf[y - 1] if y > 0 else 0.0
            margin = min(target - lo, cdf[y] - target) / total
        else:
            # every remaining token has zero mass: the best remaining logit
            masked = np.asarray(logits[cur], dtype=np.float64).copy()
            masked[rejected] = -np.inf
            y = int(np.argmax(masked))
            margin = 0.0
        decisions.append({"kind": "bonus", "at": cur, "r": r, "token": y, "margin": margin})
        emitted = [int(tree.token[u]) for u in path[1:]] + [y]
        return path, emitted, decisions
