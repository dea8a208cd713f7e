"""Planted mistakes in the CPU oracle must be caught by its pins.

Each case swaps one oracle function for a plausible wrong version (a dropped
term, a wrong sign, a reversed order, an off-by-one, a transposed operand)
and runs the pins that cover it: at least one of them must fail.  The
mistakes are planted in the oracle only, on the CPU, for the duration of one
test.
"""
import numpy as np
import torch
import pytest

from oracle import dynaspec_oracle as O
from tests import test_oracle_pins as P

ORIG = {name: getattr(O, name) for name in dir(O) if callable(getattr(O, name))}


# ---------------------------------------------------------------- mutants
def layout_desc_within_cluster(cluster_of, M):
    sizes, offsets, perm, cap = ORIG["cluster_layout"](cluster_of, M)
    cluster_of = np.asarray(cluster_of)
    perm = np.lexsort((-np.arange(cluster_of.size), cluster_of))  # vocab ids descending inside a cluster
    return sizes, offsets, perm, cap


def layout_offsets_off_by_one(cluster_of, M):
    sizes, offsets, perm, cap = ORIG["cluster_layout"](cluster_of, M)
    offsets = offsets.copy()
    offsets[1:-1] += 1
    return sizes, offsets, perm, cap


def layout_cap_smallest(cluster_of, M):
    sizes, offsets, perm, cap = ORIG["cluster_layout"](cluster_of, M)
    cap = np.zeros_like(cap)
    cap[1:] = np.cumsum(np.sort(sizes))
    return sizes, offsets, perm, cap


def silu_wrong_sign(a, act):
    if act == "silu":
        return a / (1.0 + np.exp(a))
    return ORIG["activation"](a, act)


def router_transposed(x, W1, W2=None, b1=None, b2=None, act="silu"):
    x, W1 = O.as_f64(x), O.as_f64(W1)
    pre = (W1 @ x.T).T if W1.shape[1] == x.shape[1] else x @ W1
    pre = pre[:, ::-1]  # rows of W1 taken in the wrong order
    if b1 is not None:
        pre = pre + O.as_f64(b1)
    if W2 is None:
        return pre
    return ORIG["activation"](pre, act) @ O.as_f64(W2).T + (0 if b2 is None else O.as_f64(b2))


def router_drops_bias(x, W1, W2=None, b1=None, b2=None, act="silu"):
    return ORIG["router_scores"](x, W1, W2, None, b2, act)


def router_act_after_second_layer(x, W1, W2=None, b1=None, b2=None, act="silu"):
    if W2 is None:
        return ORIG["router_scores"](x, W1, None, b1, b2, act)
    pre = O.as_f64(x) @ O.as_f64(W1).T + (0 if b1 is None else O.as_f64(b1))
    s = pre @ O.as_f64(W2).T + (0 if b2 is None else O.as_f64(b2))
    return ORIG["activation"](s, act)


def rank_ties_to_higher_id(values, ids):
    v = ORIG["_canonical"](np.asarray(values, dtype=np.float64))
    return np.lexsort((-np.asarray(ids), -v))


def canonical_nan_high(values):
    v = np.where(np.isnan(values), np.inf, values)
    return v + 0.0


def shortlist_rank_order(cluster_ids, offsets, perm):
    sel = np.asarray(cluster_ids, dtype=np.int64)  # not sorted
    offsets = np.asarray(offsets, dtype=np.int64)
    sizes = offsets[sel + 1] - offsets[sel]
    rowoff = np.zeros(sel.size + 1, dtype=np.int64)
    rowoff[1:] = np.cumsum(sizes)
    rows = np.concatenate([np.arange(offsets[m], offsets[m + 1]) for m in sel])
    return sel, rowoff, rows, np.asarray(perm)[rows]


def shortlist_drops_last_row(cluster_ids, offsets, perm):
    sel, rowoff, rows, vids = ORIG["shortlist"](cluster_ids, offsets, perm)
    return sel, rowoff, rows[:-1], vids[:-1]


def logits_by_position(h, W_lm, vocab_ids):
    return ORIG["shortlist_logits"](h, W_lm, np.arange(len(vocab_ids)))


def log_softmax_no_temperature(z, temperature=1.0):
    return ORIG["log_softmax"](z, 1.0)


def log_softmax_drops_max(z, temperature=1.0):
    t = np.asarray(z, dtype=np.float64) / float(temperature)
    mx = np.max(t)
    return t - np.log(np.sum(np.exp(t - mx)))


def topk_ascending(z, vocab_ids, k_t):
    return ORIG["rank_order"](-np.asarray(z, dtype=np.float64), vocab_ids)[:k_t]


def sample_ge(z, u, temperature=1.0):
    F = ORIG["sample_cdf"](z, temperature)
    hit = np.nonzero(F >= u)[0]
    return int(hit[0]) if hit.size else len(F) - 1


def sample_reversed_cdf(z, u, temperature=1.0):
    z = np.asarray(z, dtype=np.float64)
    return len(z) - 1 - ORIG["sample_inverse_cdf"](z[::-1], u, temperature)


def select_logprobs_by_id(z, vocab_ids, k_t=1, temperature=1.0, u=None):
    r = ORIG["draft_select"](z, vocab_ids, k_t, temperature, u)
    lp = ORIG["log_softmax"](z, temperature)
    r["logprobs"] = lp[np.minimum(r["ids"], len(lp) - 1)]
    return r


def dense_static_suffix(h, W_lm, k_t=1, temperature=1.0, u=None, n_rows=None):
    if n_rows is None:
        return ORIG["dense_head"](h, W_lm, k_t, temperature, u)
    W = np.asarray(W_lm)[-n_rows:]
    return ORIG["dense_head"](h, W, k_t, temperature, u)


def schedule_eq_without_t(t, k0, k1, k_min=1):
    if t <= 1:
        return ORIG["k_schedule"](t, k0, k1, k_min)
    return max(k_min, k1 // (2 * t))


def kmeans_update_raw_rows(W, assign, M, prev):
    Wf = O.as_f64(W)
    mu = np.array(np.asarray(prev, dtype=np.float64), copy=True)
    assign = np.asarray(assign)
    for m in range(M):
        mem = np.nonzero(assign == m)[0]
        if len(mem):
            s = Wf[mem].sum(axis=0)  # rows not normalised first
            mu[m] = s / np.linalg.norm(s)
    return mu


def kmeans_ties_high(W, centroids):
    a, S = ORIG["kmeans_assign"](W, centroids)
    M = S.shape[1]
    return (M - 1 - np.argmax(O._canonical(S)[:, ::-1], axis=1)).astype(np.int64), S


def kmeans_empty_to_zero(W, assign, M, prev):
    mu = ORIG["kmeans_update"](W, assign, M, prev)
    counts = np.bincount(np.asarray(assign, dtype=np.int64), minlength=M)
    mu[counts == 0] = 0.0
    return mu


def kmeans_argmin(W, centroids):
    a, S = ORIG["kmeans_assign"](W, centroids)
    return np.argmin(S, axis=1).astype(np.int64), S


def kmeans_bf16_centroids(W, centroids):
    # the kernel's operand precision leaking into the definition
    c = torch.from_numpy(np.asarray(centroids, dtype=np.float32)).to(torch.bfloat16).double().numpy()
    return ORIG["kmeans_assign"](W, c)


def empty_shortlist_takes_complement_token(z, vocab_ids, k_t=1, temperature=1.0, u=None, beta=0.0,
                                           complement_ids=None):
    if len(vocab_ids) == 0:
        vocab_ids, z = np.array([0]), np.array([0.0])
    return ORIG["draft_select"](z, vocab_ids, k_t, temperature, u, beta, complement_ids)


def beam_ignores_parent_scores(logprobs, ids, last_scores, n_out):
    return ORIG["beam_expand"](logprobs, ids, None, n_out)


def beam_per_row_best(logprobs, ids, last_scores, n_out):
    # each parent keeps its own best candidates in turn instead of the global best
    sc, par, tok = ORIG["beam_expand"](logprobs, ids, last_scores, 10 ** 6)
    order = sorted(range(len(sc)), key=lambda i: (par[i], -sc[i]))[:n_out]
    return sc[order], par[order], tok[order]


def cycle_broadcasts_one_parent(x0, h0, next_inputs, *args, **kw):
    # h~[-1] taken for every row at every position, not only after position 0
    return ORIG["draft_cycle"](x0, h0, lambda hp, tok: next_inputs(np.repeat(hp[-1:], len(tok), axis=0), tok),
                               *args, **kw)


def cycle_fixed_budget(x0, h0, next_inputs, W1, W2, act, cluster_of, M, W_lm, k_first, k_second, k_t, gamma,
                       k_min=1, form="equation"):
    return ORIG["draft_cycle"](x0, h0, next_inputs, W1, W2, act, cluster_of, M, W_lm, k_first, k_first, k_t,
                               gamma, k_min=max(k_min, k_first), form=form)


MUTANTS = {
    "layout: descending ids inside a cluster": ("cluster_layout", layout_desc_within_cluster,
        [P.test_layout_hand_example, lambda: P.test_layout_is_disjoint_covering_and_contiguous(0)]),
    "layout: offsets off by one": ("cluster_layout", layout_offsets_off_by_one,
        [P.test_layout_hand_example, lambda: P.test_shortlist_is_exact_union(0)]),
    "layout: cap from the smallest clusters": ("cluster_layout", layout_cap_smallest,
        [P.test_layout_hand_example]),
    "router: SiLU with the wrong sign": ("activation", silu_wrong_sign,
        [P.test_silu_closed_form, lambda: P.test_router_matches_torch_modules("silu")]),
    "router: transposed / reordered first layer": ("router_scores", router_transposed,
        [P.test_router_relu_hand_example, lambda: P.test_router_matches_torch_modules("relu")]),
    "router: first-layer bias dropped": ("router_scores", router_drops_bias,
        [P.test_router_relu_hand_example, lambda: P.test_router_matches_torch_modules("relu")]),
    "router: activation after the second layer": ("router_scores", router_act_after_second_layer,
        [P.test_router_relu_hand_example, lambda: P.test_router_matches_torch_modules("silu")]),
    "order: ties to the higher id": ("rank_order", rank_ties_to_higher_id,
        [P.test_topk_hand_ties_nan, lambda: P.test_topk_matches_python_sorted_and_argmax(0),
         P.test_select_tie_goes_to_lower_vocab_id]),
    "order: NaN ranked highest": ("_canonical", canonical_nan_high,
        [P.test_topk_hand_ties_nan, P.test_topk_signed_zero_equal]),
    "shortlist: clusters in rank order": ("shortlist", shortlist_rank_order,
        [lambda: P.test_shortlist_is_exact_union(1)]),
    "shortlist: last row dropped": ("shortlist", shortlist_drops_last_row,
        [lambda: P.test_shortlist_is_exact_union(2), lambda: P.test_head_matches_masked_dense_head_every_k(0)]),
    "logits: rows by shortlist position": ("shortlist_logits", logits_by_position,
        [P.test_logits_one_hot_head_reads_back_h, P.test_logits_integer_exact]),
    "select: temperature ignored": ("log_softmax", log_softmax_no_temperature,
        [P.test_logprobs_normalised]),
    "select: max dropped from the log-sum": ("log_softmax", log_softmax_drops_max,
        [P.test_logprobs_normalised, P.test_select_hand_example]),
    "select: smallest logits first": ("topk_tokens", topk_ascending,
        [P.test_select_hand_example, P.test_select_tie_goes_to_lower_vocab_id]),
    "sampling: F_j >= u": ("sample_inverse_cdf", sample_ge,
        [P.test_sampling_boundary_uniform_goes_to_next_token, P.test_select_hand_example]),
    "sampling: CDF walked in reverse": ("sample_inverse_cdf", sample_reversed_cdf,
        [P.test_select_hand_example, lambda: P.test_head_matches_masked_dense_head_every_k(1)]),
    "select: log-probabilities indexed by vocabulary id": ("draft_select", select_logprobs_by_id,
        [lambda: P.test_head_matches_masked_dense_head_every_k(2), P.test_k_equals_M_is_the_dense_head]),
    "static head: suffix instead of prefix": ("dense_head", dense_static_suffix,
        [P.test_static_head_is_the_dense_head_on_a_prefix]),
    "schedule: floor(k1 / 2t)": ("k_schedule", schedule_eq_without_t,
        [P.test_k_schedule_closed_form]),
    "k-means: update sums the raw rows": ("kmeans_update", kmeans_update_raw_rows,
        [P.test_kmeans_mean_direction_hand_example, P.test_kmeans_is_invariant_to_positive_row_scales]),
    "k-means: ties to the higher cluster": ("kmeans_assign", kmeans_ties_high,
        [P.test_kmeans_ties_go_to_the_lower_cluster_and_empty_clusters_keep_their_centroid]),
    "k-means: empty cluster reset to zero": ("kmeans_update", kmeans_empty_to_zero,
        [P.test_kmeans_ties_go_to_the_lower_cluster_and_empty_clusters_keep_their_centroid]),
    "k-means: least similar centroid": ("kmeans_assign", kmeans_argmin,
        [P.test_kmeans_assignment_is_euclidean_argmin_on_the_sphere, P.test_kmeans_planted_directions_are_recovered]),
    "k-means: centroids rounded to bf16": ("kmeans_assign", kmeans_bf16_centroids,
        [P.test_kmeans_similarity_is_exact_below_bf16_resolution]),
    "select: an empty shortlist still proposes a token": ("draft_select", empty_shortlist_takes_complement_token,
        [P.test_empty_shortlist_proposes_nothing]),
    "beam: parent scores not added": ("beam_expand", beam_ignores_parent_scores,
        [P.test_beam_expand_hand_example, lambda: P.test_draft_cycle_on_the_full_vocabulary_is_a_brute_force_beam(0)]),
    "beam: best per parent instead of overall": ("beam_expand", beam_per_row_best,
        [P.test_beam_expand_hand_example, lambda: P.test_draft_cycle_on_the_full_vocabulary_is_a_brute_force_beam(1)]),
    "cycle: one parent row for every beam row": ("draft_cycle", cycle_broadcasts_one_parent,
        [lambda: P.test_draft_cycle_on_the_full_vocabulary_is_a_brute_force_beam(2),
         P.test_draft_cycle_budget_union_and_parent_rows]),
    "cycle: the first budget at every position": ("draft_cycle", cycle_fixed_budget,
        [P.test_draft_cycle_budget_union_and_parent_rows]),
}


@pytest.mark.parametrize("name", list(MUTANTS))
def test_planted_mistake_is_caught(name, monkeypatch):
    target, mutant, pins = MUTANTS[name]
    monkeypatch.setattr(O, target, mutant)
    caught = 0
    for pin in pins:
        try:
            pin()
        except Exception:  # an assertion, or the mutant breaking a shape
            caught += 1
    assert caught > 0, f"no pin caught: {name}"


def test_pins_pass_on_the_unmodified_oracle():
    for _, _, pins in MUTANTS.values():
        for pin in pins:
            pin()
