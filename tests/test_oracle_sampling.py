"""Pins for the temperature-sampling oracle (oracle/sampling.py).

- The generator against the SplitMix64 reference implementation's published
  outputs and against uniformity.
- Losslessness: over many independent cycles the first emitted token follows
  the target distribution at the root, and the token after an accepted child
  follows the target distribution at that child (chi-square against the exact
  probabilities).  A dropped renormalisation, a rejected token left in the
  bonus distribution or a wrong sibling order fails these.
- The temperature -> 0 limit is the greedy rule (one-hot target).
"""
import os

import numpy as np
import pytest
from scipy import stats

import synth
from synth.configs import STATIC_26
from oracle import msd as O
from oracle import sampling as S


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_splitmix64_published_outputs():
    # published outputs of the reference generator (tests/golden, cited there)
    rows = [line.split() for line in open(os.path.join(GOLDEN, "splitmix64_test_vectors.txt"))
            if line.strip() and not line.startswith("#")]
    assert len(rows) == 7
    for seed, i, out in rows:
        assert S.splitmix64(int(seed), int(i)) == int(out, 0), (seed, i)


def test_uniform_draws():
    u = np.array([S.draw_uniform(7, s, L, j) for s in range(2) for L in range(500)
                  for j in range(40)])
    assert u.min() >= 0.0 and u.max() < 1.0
    assert np.all(u * (1 << 24) == np.floor(u * (1 << 24)))
    counts, _ = np.histogram(u, bins=64, range=(0.0, 1.0))
    assert stats.chisquare(counts).pvalue > 1e-3
    # neighbouring draws of a cycle are uncorrelated
    assert abs(np.corrcoef(u[:-1], u[1:])[0, 1]) < 0.02


def make_tree(parent, token):
    parent = np.asarray(parent, dtype=np.int32)
    depth = np.zeros(len(parent), dtype=np.int32)
    for i in range(1, len(parent)):
        depth[i] = depth[parent[i]] + 1
    return O.Tree(np.asarray(token, dtype=np.int32), parent, depth, np.zeros(len(parent)))


def chi2_pvalue(counts, probs, n):
    exp = probs * n
    big = exp >= 5
    obs = np.append(counts[big], counts[~big].sum())
    ex = np.append(exp[big], exp[~big].sum())
    if ex[-1] == 0:
        obs, ex = obs[:-1], ex[:-1]
    return stats.chisquare(obs, ex).pvalue


@pytest.mark.parametrize("temperature", [1.0, 0.6])
def test_emitted_tokens_follow_target_distribution(temperature):
    V = 10
    # root -> children tokens 3, 1, 7; node 1 (token 3) -> 5, 0; node 2 (token 1) -> 3
    parent = [-1, 0, 0, 0, 1, 1, 2]
    token = [9, 3, 1, 7, 5, 0, 3]
    rng = np.random.default_rng(11)
    logits = rng.standard_normal((len(parent), V)) * 1.5
    logits[0, 3] += 1.0  # make the first child likely enough to test its subtree
    n = 30000
    first = np.zeros(V, dtype=np.int64)
    second = {1: np.zeros(V, dtype=np.int64), 2: np.zeros(V, dtype=np.int64)}
    for L in range(n):
        path, emitted, _ = S.sample_accept(make_tree(parent, token), logits, temperature,
                                           seed=5, seq=1, L=L)
        first[emitted[0]] += 1
        if len(path) > 1 and path[1] in second:
            second[path[1]][emitted[1]] += 1
    p0 = S.target_probs(logits[0], temperature)
    assert chi2_pvalue(first, p0, n) > 1e-3
    for u, counts in second.items():
        m = counts.sum()
        assert m > 300
        assert chi2_pvalue(counts, S.target_probs(logits[u], temperature), m) > 1e-3


def test_chain_tree_follows_target_distribution():
    # the paper's chain case: one drafted token per depth
    V = 8
    parent = [-1, 0, 1, 2]
    token = [2, 4, 4, 1]
    rng = np.random.default_rng(3)
    logits = rng.standard_normal((4, V))
    logits[0, 4] += 1.5
    n = 20000
    first = np.zeros(V, dtype=np.int64)
    after = np.zeros(V, dtype=np.int64)
    for L in range(n):
        path, emitted, _ = S.sample_accept(make_tree(parent, token), logits, 1.0, seed=9,
                                           seq=0, L=L)
        first[emitted[0]] += 1
        if len(path) > 1:
            after[emitted[1]] += 1
    assert chi2_pvalue(first, S.target_probs(logits[0], 1.0), n) > 1e-3
    assert chi2_pvalue(after, S.target_probs(logits[1], 1.0), after.sum()) > 1e-3


@pytest.mark.parametrize("seed", range(4))
def test_low_temperature_is_greedy(seed):
    parent, rank, depth = synth.static_tree_arrays(STATIC_26)
    T, V = len(parent), 64
    rng = np.random.default_rng(seed)
    logits = rng.permuted(np.tile(np.arange(V, dtype=np.float64), (T, 1)), axis=1)
    amax = np.argmax(logits, axis=1).astype(np.int32)
    # tokens: the argmax child where it exists, so some paths go deep
    token = np.zeros(T, dtype=np.int32)
    for u in range(1, T):
        p = parent[u]
        token[u] = amax[p] if rank[u] == 0 and rng.random() < 0.7 else (amax[p] + 1 + rank[u]) % V
    tree = O.Tree(token, parent, depth, np.zeros(T))
    g_path, g_emit = O.greedy_accept(tree, amax)
    path, emitted, _ = S.sample_accept(tree, logits, 1e-3, seed=seed, seq=0, L=100)
    assert path == g_path
    assert emitted == g_emit
