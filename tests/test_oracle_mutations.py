"""Planted mistakes in the oracle must fail its pins (CPU only).

Each case plants one plausible mistake in the oracle (a wrong sign, a dropped
term, a swapped operand, an off-by-one index, a wrong loop order) and runs
the existing pins against it: at least one must fail with an assertion.
Python-level oracle functions are mutated in their source text; the
numerical primitives, which run in C, are wrapped so that they compute the
mistaken formula exactly.  Nothing here changes the oracle on disk.
"""
import inspect
import os
import sys
import textwrap

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))

import synth  # noqa: E402
from oracle import metrics as MET  # noqa: E402
from oracle import model as M  # noqa: E402
from oracle import msd as O  # noqa: E402
from oracle import sampling as S  # noqa: E402
from oracle import train as TR  # noqa: E402

import test_oracle_draft_pins as PD  # noqa: E402
import test_oracle_invariants as PI  # noqa: E402
import test_oracle_primitives as PP  # noqa: E402
import test_oracle_sampling as PS  # noqa: E402
import test_oracle_train as PTR  # noqa: E402
import test_oracle_trees as PT  # noqa: E402


def mutant(fn, old, new):
    """fn (a function or class) with the text `old` of its source replaced by
    `new` (exactly once)."""
    src = textwrap.dedent(inspect.getsource(fn))
    assert src.count(old) == 1, f"mutation site not found in {fn.__name__}: {old!r}"
    ns = dict(sys.modules[fn.__module__].__dict__)
    exec(compile(src.replace(old, new), f"<mutant of {fn.__name__}>", "exec"), ns)
    return ns[fn.__name__]


def caught(*runs):
    """True if at least one pin run fails with an assertion."""
    for run in runs:
        try:
            run()
        except AssertionError:
            return True
    return False


# ---- numerical primitives (C code, wrapped) -------------------------------

ORIG = {name: getattr(M, name) for name in ("rope", "rmsnorm", "silu_mul", "attention",
                                             "linear")}


def rope_wrong_direction(x, pos, n_heads, head_dim, theta):
    return ORIG["rope"](x, -np.asarray(pos, dtype=np.int32), n_heads, head_dim, theta)


def rope_interleaved_pairs(x, pos, n_heads, head_dim, theta):
    # rotates (2i, 2i+1) instead of (i, i + hd/2)
    half = head_dim // 2
    inter = np.concatenate([np.arange(0, head_dim, 2), np.arange(1, head_dim, 2)])
    idx = np.concatenate([h * head_dim + inter for h in range(n_heads)])
    y = np.ascontiguousarray(x[:, idx])
    ORIG["rope"](y, pos, n_heads, head_dim, theta)
    x[:, idx] = y
    assert half * 2 == head_dim
    return x


def rope_half_exponent(x, pos, n_heads, head_dim, theta):
    # inv_freq = theta^(-i/hd) instead of theta^(-2i/hd)
    return ORIG["rope"](x, pos, n_heads, head_dim, theta ** 0.5)


def rmsnorm_no_eps(x, g, eps):
    return ORIG["rmsnorm"](x, g, 0.0)


def rmsnorm_no_gain(x, g, eps):
    return ORIG["rmsnorm"](x, synth.ones_bf16(len(g)), eps)


def rmsnorm_sum_not_mean(x, g, eps):
    return ORIG["rmsnorm"](x, g, eps) / np.sqrt(np.asarray(x).shape[1])


def silu_on_up(g, u):
    return ORIG["silu_mul"](u, g)


def sigmoid_not_silu(g, u):
    return ORIG["silu_mul"](g, u) / np.asarray(g, dtype=np.float64)


def attention_no_scale(q, kc, vc, L, R, anc, n_heads, n_kv, head_dim):
    return ORIG["attention"](np.asarray(q) * np.sqrt(head_dim), kc, vc, L, R, anc, n_heads,
                             n_kv, head_dim)


def attention_gqa_modulo(q, kc, vc, L, R, anc, n_heads, n_kv, head_dim):
    # query head h reads kv head h % KV instead of h // (H / KV)
    G = n_heads // n_kv
    slots = {k: [h for h in range(n_heads) if h // G == k] for k in range(n_kv)}
    perm = np.empty(n_heads, dtype=np.int64)   # mutant head h computed as head perm[h]
    for h in range(n_heads):
        perm[h] = slots[h % n_kv].pop(0)
    q = np.asarray(q, dtype=np.float64)
    Mq = q.shape[0]
    qh = q.reshape(Mq, n_heads, head_dim)
    qp = np.empty_like(qh)
    qp[:, perm] = qh
    o = ORIG["attention"](qp.reshape(Mq, -1), kc, vc, L, R, anc, n_heads, n_kv, head_dim)
    return o.reshape(Mq, n_heads, head_dim)[:, perm].reshape(Mq, -1)


def attention_ignores_ancestors(q, kc, vc, L, R, anc, n_heads, n_kv, head_dim):
    if anc is not None:
        anc = np.full(len(anc), (1 << R) - 1, dtype=np.uint64)
    return ORIG["attention"](q, kc, vc, L, R, anc, n_heads, n_kv, head_dim)


def attention_mask_shifted(q, kc, vc, L, R, anc, n_heads, n_kv, head_dim):
    if anc is not None:
        anc = (np.asarray(anc, dtype=np.uint64) << np.uint64(1)) & np.uint64((1 << R) - 1)
    return ORIG["attention"](q, kc, vc, L, R, anc, n_heads, n_kv, head_dim)


def attention_causal_off_by_one(q, kc, vc, L, R, anc, n_heads, n_kv, head_dim):
    if anc is None:  # row i also sees row i + 1
        anc = np.array([(1 << min(i + 2, R)) - 1 for i in range(R)], dtype=np.uint64)
    return ORIG["attention"](q, kc, vc, L, R, anc, n_heads, n_kv, head_dim)


def linear_rounds_x(x, w):
    return ORIG["linear"](M.widen(synth.f32_to_bf16(np.asarray(x, dtype=np.float32))), w)


PRIMITIVE_CASES = [
    ("rope", rope_wrong_direction, [PP.test_rope_is_complex_rotation]),
    ("rope", rope_interleaved_pairs, [PP.test_rope_is_complex_rotation]),
    ("rope", rope_half_exponent, [PP.test_rope_is_complex_rotation]),
    ("rmsnorm", rmsnorm_no_eps, [PP.test_rmsnorm_properties]),
    ("rmsnorm", rmsnorm_no_gain, [PP.test_rmsnorm_properties]),
    ("rmsnorm", rmsnorm_sum_not_mean, [PP.test_rmsnorm_properties]),
    ("silu_mul", silu_on_up, [PP.test_silu_mul_matches_scipy]),
    ("silu_mul", sigmoid_not_silu, [PP.test_silu_mul_matches_scipy]),
    ("attention", attention_no_scale, [lambda: PP.test_attention_causal_matches_sdpa(4, 4)]),
    ("attention", attention_gqa_modulo, [lambda: PP.test_attention_causal_matches_sdpa(4, 2)]),
    ("attention", attention_ignores_ancestors, [PP.test_attention_tree_mask_matches_sdpa]),
    ("attention", attention_mask_shifted, [PP.test_attention_tree_mask_matches_sdpa]),
    ("attention", attention_causal_off_by_one,
     [lambda: PP.test_attention_causal_matches_sdpa(4, 4)]),
    ("linear", linear_rounds_x, [lambda: PP.test_linear_matches_numpy(5, 64, 17)]),
]


@pytest.mark.parametrize("name,fn,pins", PRIMITIVE_CASES,
                         ids=[c[1].__name__ for c in PRIMITIVE_CASES])
def test_primitive_mistake_is_caught(monkeypatch, name, fn, pins):
    for pin in pins:  # the pins pass on the real oracle ...
        pin()
    monkeypatch.setattr(M, name, fn)
    assert caught(*pins)  # ... and fail on the mutant


# ---- Python-level oracle code (mutated in its source) ---------------------

def greedy_pins():
    return [lambda s=s: PT.test_greedy_accept_matches_paper_rule_with_one_hot_target(s)
            for s in range(20)]


def draft_branch_pins():
    return [lambda k=k: PD.test_draft_nodes_equal_sequential_branch_decode(PI.TINY, k)
            for k in ("static", "dynamic")]


def beam_pins():
    return [lambda s=s: PD.test_dynamic_tree_matches_brute_force_beam(8, 3, 3, 5, s)
            for s in range(3)] + [lambda: PD.test_dynamic_tree_matches_brute_force_beam(
                12, 3, 3, 9, 0)]


SOURCE_CASES = [
    # acceptance compares with the node's own argmax instead of its parent's
    ("accept_own_argmax", O, "greedy_accept",
     "ok[j] = ok[p] and tree.token[j] == amax[p]", "ok[j] = ok[p] and tree.token[j] == amax[j]",
     greedy_pins),
    # acceptance ignores whether the parent was accepted
    ("accept_orphans", O, "greedy_accept",
     "ok[j] = ok[p] and tree.token[j] == amax[p]", "ok[j] = tree.token[j] == amax[p]",
     greedy_pins),
    # the bonus token is taken at the root instead of the deepest accepted node
    ("bonus_from_root", O, "greedy_accept",
     "+ [int(amax[best])]", "+ [int(amax[0])]", greedy_pins),
    # compaction moves rows in place in reverse order (a later read sees a write)
    ("compact_in_place_reverse", O, "compact_kv",
     "    kv.k[:, L:L + len(path)] = kv.k[:, src].copy()\n"
     "    kv.v[:, L:L + len(path)] = kv.v[:, src].copy()\n",
     "    for j in reversed(range(len(path))):\n"
     "        kv.k[:, L + j] = kv.k[:, src[j]]\n"
     "        kv.v[:, L + j] = kv.v[:, src[j]]\n",
     lambda: [PT.test_compaction_in_place_matches_out_of_place]),
    # a tree node does not see itself
    ("ancestor_mask_without_self", O, "ancestor_masks",
     "(anc[p] if p >= 0 else np.uint64(0)) | np.uint64(1 << i)",
     "(anc[p] | np.uint64(1 << p)) if p >= 0 else np.uint64(1)",
     lambda: [lambda: PI.test_tree_forward_equals_branch_forwards(PI.TINY, "static")]),
    # the draft input concatenates the embedding first
    ("concat_order", M, "draft_input",
     "np.concatenate([h[txt], e_next[txt]], axis=1)", "np.concatenate([e_next[txt], h[txt]], axis=1)",
     lambda: [PI.test_all_text_prompt_matches_feature_level_baseline]),
    # a sampled child is accepted with p(x) instead of p(x) / (1 - rejected mass)
    ("sampling_no_renormalisation", S, "sample_accept",
     "ratio = p[x] / rem if rem > 0 else 0.0", "ratio = p[x]",
     lambda: [lambda: PS.test_emitted_tokens_follow_target_distribution(1.0)]),
    # rejected tokens stay in the bonus distribution
    ("bonus_keeps_rejected", S, "sample_accept",
     "q[rejected] = 0.0", "pass",
     lambda: [lambda: PS.test_emitted_tokens_follow_target_distribution(1.0)]),
    # the geometric sum stops one term early
    ("omega_off_by_one", MET, "omega",
     "alpha ** (gamma + 1)", "alpha ** gamma",
     lambda: [lambda: PT.test_omega_matches_monte_carlo(4, 0.8)]),
    # a drafted node of depth d sits at position L + d instead of L + d - 1
    ("draft_node_position", O, "_DraftExpander",
     "np.full(len(keys), st.L + depth - 1, dtype=np.int32)",
     "np.full(len(keys), st.L + depth, dtype=np.int32)",
     draft_branch_pins),
    # a drafted node attends to the committed cache and itself, not its ancestors
    ("draft_node_without_ancestors", O, "_DraftExpander",
     "a |= self.mask[pk]", "pass",
     draft_branch_pins),
    # the draft catch-up rows are rotated one position too far
    ("catch_up_positions_shifted", O, "draft_catch_up",
     "np.arange(L0, L0 + r, dtype=np.int32)", "np.arange(L0 + 1, L0 + r + 1, dtype=np.int32)",
     lambda: [lambda: PD.test_draft_cache_equals_one_causal_draft_forward(PI.TINY, "static", "embedding")]),
    # the Visual Feature variant feeds the visual embedding after all
    ("visual_feature_input_ignored", O, "prefill",
     'src = x[i] if visual_input == "embedding" else h[i]', "src = x[i]",
     lambda: [lambda: PD.test_draft_cache_equals_one_causal_draft_forward(
         PI.TINY, "static", "feature")]),
    # log-softmax without the log-sum-exp term
    ("log_softmax_without_lse", O, "log_softmax",
     "return logits - (m + np.log(np.sum(np.exp(logits - m))))", "return logits - m",
     lambda: [lambda: PD.test_log_softmax_matches_scipy(1.0)] + beam_pins()),
    # the dynamic frontier keeps the first K candidates by creation order
    ("frontier_by_creation_order", O, "select_dynamic_tree",
     "frontier = [new[i] for i in topk_desc(sc, K)]", "frontier = new[:K]",
     beam_pins),
    # within a depth, the kept nodes are ordered by score instead of creation
    ("final_order_by_score", O, "select_dynamic_tree",
     "key=lambda i: (pool[i][2], i))", "key=lambda i: (pool[i][2], -pool[i][3]))",
     beam_pins),
    # training: the draft output is regressed on its own position's feature
    ("train_target_not_shifted", TR, "row_losses",
     "diff = d - h[1:]", "diff = d - h[:-1]",
     lambda: [PTR.test_loss_assembly_closed_form]),
    # training: the token term against the distribution of the wrong row
    ("train_labels_not_shifted", TR, "row_losses",
     "pt[1:]", "pt[:-1]", lambda: [PTR.test_loss_assembly_closed_form]),
    # training: SmoothL1 without its one-half in the quadratic zone
    ("train_smooth_l1_quadratic", TR, "row_losses",
     "0.5 * diff * diff", "diff * diff", lambda: [PTR.test_loss_assembly_closed_form]),
    # training: the token term at full weight
    ("train_token_weight", TR, "sequence_loss_sum",
     "reg + CLS_WEIGHT * cls", "reg + cls", lambda: [PTR.test_batch_loss_weights_and_means]),
    # training: text rows concatenate their own embedding, not the next one
    ("train_input_embedding", TR, "draft_inputs",
     "torch.cat([h[:R], e[1:]], dim=1)", "torch.cat([h[:R], e[:R]], dim=1)",
     lambda: [lambda: PTR.test_draft_inputs_follow_decoupled_rule("embedding")]),
    # training: the Visual Feature input ignored (visual rows keep e_i)
    ("train_visual_feature_ignored", TR, "draft_inputs",
     'src = e[:R] if visual_input == "embedding" else h[:R]', "src = e[:R]",
     lambda: [lambda: PTR.test_draft_inputs_follow_decoupled_rule("feature")]),
    # AdamW without bias correction
    ("adam_without_bias_correction", TR, "AdamW",
     "(self.m[k] / c1) / (np.sqrt(self.v[k] / c2) + ADAM_EPS)",
     "self.m[k] / (np.sqrt(self.v[k]) + ADAM_EPS)",
     lambda: [PTR.test_adamw_first_step_and_schedule]),
    # the progressive mix runs backwards (visual share (T - t) / T)
    ("mix_reversed", TR, "progressive_counts",
     "n_per_epoch * epoch / n_epochs", "n_per_epoch * (n_epochs - epoch) / n_epochs",
     lambda: [lambda: PTR.test_progressive_mix_counts(5)]),
]


@pytest.mark.parametrize("case", SOURCE_CASES, ids=[c[0] for c in SOURCE_CASES])
def test_source_mistake_is_caught(monkeypatch, case):
    _, module, fname, old, new, pins = case
    pins = pins()
    for pin in pins:
        pin()
    monkeypatch.setattr(module, fname, mutant(getattr(module, fname), old, new))
    assert caught(*pins)
