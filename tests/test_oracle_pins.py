"""Pins for the CPU oracle: each check ties it to something other than itself.

Sources of truth used here: hand-worked examples (tests/golden), closed forms,
invariants of the partition and the shortlist, special cases that reduce to a
different library routine (torch's Linear/SiLU, Python's sorted, numpy's
argmax, scipy's log_softmax), and brute force on tiny vocabularies by a
different route (masking the dense head instead of gathering rows).
"""
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import dynaspec_oracle as O

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))


def _num(v):
    return float("nan") if v == "nan" else float(v)


# ---------------------------------------------------------------- decoding
def test_bf16_decode_hand_values():
    bits = np.array([0x3F80, 0xC000, 0x3FC0, 0x0000, 0x8000, 0x7F80, 0x0001], dtype=np.uint16)
    got = O.as_f64(bits)
    assert got[0] == 1.0 and got[1] == -2.0 and got[2] == 1.5
    assert got[3] == 0.0 and np.signbit(got[4]) and got[5] == np.inf
    assert got[6] == 2.0 ** -133  # smallest bf16 subnormal: 2^-126 * 2^-7


def test_bf16_decode_matches_torch_conversion():
    rng = np.random.default_rng(1)
    bits = rng.integers(0, 1 << 16, size=4096, dtype=np.uint16)
    bits = bits[((bits >> 7) & 0xFF) != 0xFF]  # drop inf/nan patterns
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(O.as_f64(bits), ref)


# ---------------------------------------------------------------- partition
def test_layout_hand_example():
    g = GOLD["layout"]
    sizes, offsets, perm, cap = O.cluster_layout(np.array(g["cluster_of"]), g["M"])
    assert sizes.tolist() == g["sizes"]
    assert offsets.tolist() == g["offsets"]
    assert perm.tolist() == g["perm"]
    assert cap.tolist() == g["cap_by_k"]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_layout_is_disjoint_covering_and_contiguous(seed):
    rng = np.random.default_rng(seed)
    V, M = 997, 37
    cluster_of = rng.integers(0, M, size=V)
    cluster_of[cluster_of == 5] = 6  # force an empty cluster
    sizes, offsets, perm, cap = O.cluster_layout(cluster_of, M)
    assert sorted(perm.tolist()) == list(range(V))          # bijection
    assert offsets[0] == 0 and offsets[-1] == V
    assert np.all(np.diff(offsets) >= 0)
    assert sizes[5] == 0
    for m in range(M):                                      # each run is exactly C_m, ascending
        run = perm[offsets[m]:offsets[m + 1]].tolist()
        assert run == [v for v in range(V) if cluster_of[v] == m]
    # cap_by_k[k] is the best sum of k sizes (brute force over all k-subsets for small k)
    from itertools import combinations
    small = sizes[:9]
    _, _, _, cap9 = O.cluster_layout(np.repeat(np.arange(9), small), 9)
    for k in range(1, 4):
        assert cap9[k] == max(sum(c) for c in combinations(small.tolist(), k))


def test_layout_rejects_bad_ids():
    with pytest.raises(ValueError):
        O.cluster_layout(np.array([0, 3]), 3)
    with pytest.raises(ValueError):
        O.cluster_layout(np.array([0, -1]), 3)


# ---------------------------------------------------------------- router
def test_router_relu_hand_example():
    g = GOLD["router_relu"]
    x, W1, W2 = np.array(g["x"]), np.array(g["W1"], float), np.array(g["W2"], float)
    np.testing.assert_array_equal(O.router_scores(x, W1, W2, act="relu"), g["scores_no_bias"])
    np.testing.assert_array_equal(
        O.router_scores(x, W1, W2, b1=np.array(g["b1"]), b2=np.array(g["b2"]), act="relu"),
        g["scores_with_bias"])


def test_router_linear_hand_example():
    g = GOLD["router_linear"]
    got = O.router_scores(np.array(g["x"]), np.array(g["W1"], float), None, act="none")
    np.testing.assert_array_equal(got, g["scores"])


def test_silu_closed_form():
    g = GOLD["silu"]
    np.testing.assert_allclose(O.activation(np.array(g["a"]), "silu"), g["silu"], rtol=1e-15)
    a = np.linspace(-20, 20, 81)
    # silu(a) - silu(-a) = a  (sigmoid(a) + sigmoid(-a) = 1)
    np.testing.assert_allclose(O.activation(a, "silu") - O.activation(-a, "silu"), a, atol=1e-12)


@pytest.mark.parametrize("act", ["relu", "silu"])
def test_router_matches_torch_modules(act):
    rng = np.random.default_rng(3)
    d_r, H, M, B = 24, 16, 12, 5  # non-square everywhere: a transposed operand cannot fit
    x = rng.standard_normal((B, d_r))
    W1, b1 = rng.standard_normal((H, d_r)), rng.standard_normal(H)
    W2, b2 = rng.standard_normal((M, H)), rng.standard_normal(M)
    l1, l2 = torch.nn.Linear(d_r, H).double(), torch.nn.Linear(H, M).double()
    with torch.no_grad():
        l1.weight.copy_(torch.from_numpy(W1)); l1.bias.copy_(torch.from_numpy(b1))
        l2.weight.copy_(torch.from_numpy(W2)); l2.bias.copy_(torch.from_numpy(b2))
        mod = torch.nn.Sequential(l1, torch.nn.ReLU() if act == "relu" else torch.nn.SiLU(), l2)
        ref = mod(torch.from_numpy(x)).numpy()
    np.testing.assert_allclose(O.router_scores(x, W1, W2, b1, b2, act), ref, rtol=1e-12, atol=1e-12)


def test_router_bf16_inputs_decode_exactly():
    # a bf16 weight matrix must give the same scores as its exact fp64 values
    rng = np.random.default_rng(4)
    W = torch.from_numpy(rng.standard_normal((6, 8)).astype(np.float32)).to(torch.bfloat16)
    x = torch.from_numpy(rng.standard_normal((2, 8)).astype(np.float32)).to(torch.bfloat16)
    bits = lambda t: t.view(torch.int16).numpy().view(np.uint16)
    ref = x.double().numpy() @ W.double().numpy().T
    np.testing.assert_array_equal(O.router_scores(bits(x), bits(W), None, act="none"), ref)


# ---------------------------------------------------------------- top-k
def test_topk_hand_ties_nan():
    g = GOLD["topk_ties"]
    s = np.array([_num(v) for v in g["scores"]])
    for k in (3, 4, 6):
        assert O.topk_clusters(s, k)[0][0].tolist() == g[f"k{k}"]


def test_topk_signed_zero_equal():
    assert O.topk_clusters(np.array([-0.0, 0.0, -1.0]), 1)[0][0].tolist() == [0]
    assert O.topk_clusters(np.array([0.0, -0.0, -1.0]), 2)[0][0].tolist() == [0, 1]
    assert O.topk_clusters(np.array([np.nan, -np.inf]), 1)[0][0].tolist() == [0]


@pytest.mark.parametrize("seed", range(5))
def test_topk_matches_python_sorted_and_argmax(seed):
    rng = np.random.default_rng(seed)
    M = 23
    s = rng.integers(-3, 4, size=(6, M)).astype(float)  # many ties
    for k in (1, 5, M):
        ids, vals = O.topk_clusters(s, k)
        for b in range(s.shape[0]):
            ref = sorted(range(M), key=lambda i: (-s[b, i], i))[:k]
            assert ids[b].tolist() == ref
            assert vals[b].tolist() == [s[b, i] for i in ref]
    ids, _ = O.topk_clusters(s, 1)
    assert ids[:, 0].tolist() == np.argmax(s, axis=1).tolist()  # numpy: first maximum


# ---------------------------------------------------------------- shortlist
@pytest.mark.parametrize("seed", range(4))
def test_shortlist_is_exact_union(seed):
    rng = np.random.default_rng(seed)
    V, M, k = 300, 17, 5
    cluster_of = rng.integers(0, M, size=V)
    sizes, offsets, perm, cap = O.cluster_layout(cluster_of, M)
    K = rng.choice(M, size=k, replace=False)
    sel, rowoff, rows, vids = O.shortlist(K, offsets, perm)
    members = {v for v in range(V) if cluster_of[v] in set(K.tolist())}   # brute force
    assert set(vids.tolist()) == members and len(vids) == len(members)
    assert sel.tolist() == sorted(K.tolist())
    assert rowoff[-1] == len(members) <= cap[k]
    # ascending cluster id, then ascending vocabulary id inside a cluster
    key = [(cluster_of[v], v) for v in vids.tolist()]
    assert key == sorted(key)
    for i, m in enumerate(sel):
        assert rowoff[i + 1] - rowoff[i] == sizes[m]
        assert np.all(perm[rows[rowoff[i]:rowoff[i + 1]]] == vids[rowoff[i]:rowoff[i + 1]])


# ---------------------------------------------------------------- logits
def test_logits_one_hot_head_reads_back_h():
    # W_LM rows are unit vectors e_{v mod d}: z[j] must equal h[vocab_ids[j] mod d]
    V, d = 40, 16
    W = np.zeros((V, d)); W[np.arange(V), np.arange(V) % d] = 1.0
    h = np.arange(d, dtype=float) * 1.5 - 7.0
    vids = np.array([3, 17, 39, 0, 22])
    np.testing.assert_array_equal(O.shortlist_logits(h, W, vids), h[vids % d])


def test_logits_rank_one_head():
    # W_LM = a c^T  =>  z[j] = a[v_j] (c . h)
    rng = np.random.default_rng(5)
    a, c, h = rng.standard_normal(50), rng.standard_normal(12), rng.standard_normal(12)
    vids = rng.choice(50, size=9, replace=False)
    ch = sum(ci * hi for ci, hi in zip(c, h))
    np.testing.assert_allclose(O.shortlist_logits(h, np.outer(a, c), vids), a[vids] * ch, rtol=1e-12)


def test_logits_integer_exact():
    rng = np.random.default_rng(6)
    W = rng.integers(-8, 9, size=(30, 11)); h = rng.integers(-8, 9, size=11)
    vids = np.array([29, 0, 14])
    exact = [sum(int(W[v, i]) * int(h[i]) for i in range(11)) for v in vids]
    assert O.shortlist_logits(h.astype(float), W.astype(float), vids).tolist() == exact


# ---------------------------------------------------------------- select
def test_select_hand_example():
    g = GOLD["select"]
    p, vids = np.array(g["probs"]), np.array(g["vocab_ids"])
    z = np.log(p) + 3.0  # any shift gives the same q_S
    r = O.draft_select(z, vids, k_t=2)
    assert r["positions"].tolist() == g["top2_positions"] and r["ids"].tolist() == g["top2_ids"]
    np.testing.assert_allclose(np.exp(O.log_softmax(z)), p, rtol=1e-14)
    for u, pos in g["u_to_position"]:
        assert O.sample_inverse_cdf(z, u) == pos
        assert O.sample_inverse_cdf(2.0 * z, u, temperature=2.0) == pos  # z/T unchanged


def test_select_tie_goes_to_lower_vocab_id():
    g = GOLD["select_ties"]
    assert O.topk_tokens(np.array(g["z"]), np.array(g["vocab_ids"]), 3).tolist() == g["top3_positions"]


def test_sample_cdf_hand_example():
    g = GOLD["sample_cdf"]
    z = np.log(np.array(g["probs"])) - 1.5  # any shift gives the same q_S
    np.testing.assert_allclose(O.sample_cdf(z), g["cdf_T1"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(O.sample_cdf(z, temperature=0.5), np.array(g["cdf_T0.5_times_22"]) / 22.0,
                               rtol=0, atol=1e-15)
    # the inverse-CDF draw is the first position whose CDF exceeds u
    F = O.sample_cdf(z, temperature=0.5)
    for u in np.linspace(0.0, 0.999, 37):
        assert O.sample_inverse_cdf(z, u, temperature=0.5) == int(np.searchsorted(F, u, side="right"))


def test_empty_shortlist_proposes_nothing():
    # clusters may be empty (no balance is enforced); a router that picks only
    # empty clusters leaves an empty shortlist, which proposes no token
    cluster_of = np.array([0, 0, 2, 2, 2, 0])  # cluster 1 and 3 are empty
    W_lm = np.eye(6, 4, dtype=np.float32)
    x = np.ones((1, 4), dtype=np.float32)
    W1 = np.zeros((4, 4), dtype=np.float32)
    b1 = np.array([0.0, 5.0, 0.0, 4.0])  # scores from the bias alone: clusters 1, 3 on top
    r = O.draft_head(x, x, W1, None, "none", cluster_of, 4, W_lm, k=2, k_t=3, u=np.array([0.4]), b1=b1)[0]
    assert r["clusters"].tolist() == [1, 3]
    assert len(r["vocab_ids"]) == 0 and len(r["ids"]) == 0
    assert r["sample_id"] == -1 and r["sample_logprob"] == -np.inf
    # one more cluster brings in its tokens
    r = O.draft_head(x, x, W1, None, "none", cluster_of, 4, W_lm, k=3, k_t=3, u=np.array([0.4]), b1=b1)[0]
    assert sorted(r["vocab_ids"].tolist()) == [0, 1, 5]


def test_sampling_fallback_and_zero_mass():
    z = np.array([0.0, -np.inf])
    assert O.sample_inverse_cdf(z, 0.5) == 0
    assert O.sample_inverse_cdf(z, 1.0) == 0  # no F_j > u: last j with p_j > 0


def test_sampling_boundary_uniform_goes_to_next_token():
    # equal logits give exactly representable p_j = 1/4 and F = 1/4, 1/2, 3/4, 1:
    # a uniform equal to F_j picks token j + 1 (first F_j > u)
    z = np.zeros(4)
    assert [O.sample_inverse_cdf(z, u) for u in (0.0, 0.25, 0.5, 0.75, 0.99)] == [0, 1, 2, 3, 3]


def test_sampling_grid_frequencies_equal_probabilities():
    rng = np.random.default_rng(7)
    z = rng.standard_normal(9)
    p = np.exp(z - z.max()); p /= p.sum()
    N = 20000
    counts = np.bincount([O.sample_inverse_cdf(z, (i + 0.5) / N) for i in range(N)], minlength=9)
    assert np.all(np.abs(counts - p * N) <= 1.0)


def test_tail_mixture_hand_example():
    # S = two equal tokens, complement = two tokens, beta = 1/2 (Sec. 5):
    # q~ = 1/4 on every token; u in [0, 1/2) picks inside S by u / (1/2)
    z, vids, comp = np.zeros(2), np.array([7, 9]), np.array([3, 4])
    picks = [O.draft_select(z, vids, 1, u=u, beta=0.5, complement_ids=comp)["sample_id"]
             for u in (0.0, 0.2, 0.3, 0.5, 0.6, 0.75, 0.9)]
    assert picks == [7, 7, 9, 3, 3, 4, 4]
    r = O.draft_select(z, vids, 2, u=0.9, beta=0.5, complement_ids=comp)
    np.testing.assert_allclose(np.exp(r["logprobs"]), [0.25, 0.25], rtol=1e-15)
    assert abs(np.exp(r["sample_logprob"]) - 0.25) < 1e-15


def test_tail_mixture_is_a_full_support_distribution():
    # grid of u: every token's frequency is its q~ probability, and q~ sums to one
    rng = np.random.default_rng(13)
    z = rng.standard_normal(5)
    vids, comp, beta = np.arange(5), np.arange(5, 12), 0.3
    p = np.exp(z - z.max()); p /= p.sum()
    N = 70000
    ids = [O.draft_select(z, vids, 1, u=(i + 0.5) / N, beta=beta, complement_ids=comp)["sample_id"]
           for i in range(N)]
    freq = np.bincount(ids, minlength=12) / N
    q = np.concatenate([(1 - beta) * p, np.full(7, beta / 7)])
    assert np.all(np.abs(freq - q) <= 2.0 / N)
    r = O.draft_select(z, vids, 5, beta=beta, complement_ids=comp)
    assert abs(np.exp(r["logprobs"]).sum() + beta - 1.0) < 1e-12


def test_tail_mixture_reduces_to_the_shortlist_draft():
    rng = np.random.default_rng(14)
    z = rng.standard_normal(9)
    for u in (0.0, 0.31, 0.77, 0.999):
        a = O.draft_select(z, np.arange(9), 3, u=u)
        b = O.draft_select(z, np.arange(9), 3, u=u, beta=0.0, complement_ids=np.arange(9, 20))
        c = O.draft_select(z, np.arange(9), 3, u=u, beta=0.4, complement_ids=np.zeros(0, dtype=int))
        for x in (b, c):  # beta = 0, or an empty complement (k = M)
            assert x["ids"].tolist() == a["ids"].tolist() and x["sample_id"] == a["sample_id"]
            np.testing.assert_allclose(x["logprobs"], a["logprobs"], rtol=1e-15)


def test_complement_is_the_rest_of_the_vocabulary_in_layout_order():
    rng = np.random.default_rng(15)
    V, M = 200, 11
    cluster_of = rng.integers(0, M, size=V)
    sizes, offsets, perm, _ = O.cluster_layout(cluster_of, M)
    K = np.array([2, 5, 9])
    comp = O.complement(offsets, perm, K)
    assert set(comp.tolist()) == {v for v in range(V) if cluster_of[v] not in (2, 5, 9)}
    key = [(cluster_of[v], v) for v in comp.tolist()]
    assert key == sorted(key)


def test_logprobs_normalised():
    rng = np.random.default_rng(8)
    z = rng.standard_normal(1000) * 4
    lp = O.log_softmax(z, 0.7)
    assert np.all(lp <= 0)
    assert abs(np.exp(lp).sum() - 1.0) < 1e-12
    from scipy.special import log_softmax as ref
    np.testing.assert_allclose(lp, ref(z / 0.7), rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- whole head, brute force
def _tiny_problem(seed, V=16, M=4, d=6, B=3, H=5):
    rng = np.random.default_rng(seed)
    cluster_of = rng.permutation(np.arange(V) % M)
    W = rng.standard_normal((V, d)); h = rng.standard_normal((B, d))
    W1, W2 = rng.standard_normal((H, d)), rng.standard_normal((M, H))
    u = rng.random(B)
    return cluster_of, W, h, W1, W2, u


@pytest.mark.parametrize("seed", range(3))
def test_head_matches_masked_dense_head_every_k(seed):
    from scipy.special import log_softmax as ref_lsm
    V, M = 16, 4
    cluster_of, W, h, W1, W2, u = _tiny_problem(seed, V=V, M=M)
    s = O.router_scores(h, W1, W2, act="silu")
    for k in range(1, M + 1):
        out = O.draft_head(h, h, W1, W2, "silu", cluster_of, M, W, k, k_t=3, u=u)
        for b, r in enumerate(out):
            chosen = sorted(range(M), key=lambda m: (-s[b, m], m))[:k]      # brute force routing
            mask = np.isin(cluster_of, chosen)
            zfull = W @ h[b]
            zm = np.where(mask, zfull, -np.inf)
            top = sorted(np.nonzero(mask)[0].tolist(), key=lambda v: (-zfull[v], v))[:3]
            assert r["ids"].tolist() == top[:min(3, mask.sum())]
            lsm = ref_lsm(zm)
            np.testing.assert_allclose(r["logprobs"], lsm[r["ids"]], rtol=1e-12)
            np.testing.assert_allclose(r["logits"], zfull[r["vocab_ids"]], rtol=1e-12)
            # sampled token: walk the masked distribution in layout order
            order = sorted(np.nonzero(mask)[0].tolist(), key=lambda v: (cluster_of[v], v))
            p = np.exp(lsm[order]); F = np.cumsum(p)
            assert r["sample_id"] == order[int(np.nonzero(F > u[b])[0][0])]


def test_union_head_is_the_masked_dense_head_on_the_union():
    from scipy.special import log_softmax as ref_lsm
    V, M = 24, 6
    cluster_of, W, h, W1, W2, u = _tiny_problem(21, V=V, M=M, B=4)
    s = O.router_scores(h, W1, W2, act="silu")
    for k in (1, 2, 3):
        out = O.draft_head(h, h, W1, W2, "silu", cluster_of, M, W, k, k_t=3, union=True)
        chosen = {m for b in range(4) for m in sorted(range(M), key=lambda m: (-s[b, m], m))[:k]}
        mask = np.isin(cluster_of, sorted(chosen))                      # brute-force union
        for b, r in enumerate(out):
            assert set(r["vocab_ids"].tolist()) == set(np.nonzero(mask)[0].tolist())
            zfull = W @ h[b]
            top = sorted(np.nonzero(mask)[0].tolist(), key=lambda v: (-zfull[v], v))[:3]
            assert r["ids"].tolist() == top
            np.testing.assert_allclose(r["logprobs"], ref_lsm(np.where(mask, zfull, -np.inf))[top], rtol=1e-12)
    # one row: the union is that row's own shortlist
    a = O.draft_head(h[:1], h[:1], W1, W2, "silu", cluster_of, M, W, 2, k_t=3, union=True)[0]
    b = O.draft_head(h[:1], h[:1], W1, W2, "silu", cluster_of, M, W, 2, k_t=3)[0]
    assert a["vocab_ids"].tolist() == b["vocab_ids"].tolist() and a["ids"].tolist() == b["ids"].tolist()


def test_beam_expand_hand_example():
    # two beams, three candidates each: cumulative = row log-prob + parent score
    lp = np.log(np.array([[0.5, 0.3, 0.2], [0.6, 0.25, 0.15]]))
    ids = np.array([[10, 11, 12], [20, 21, 22]])
    last = np.log(np.array([0.4, 0.6]))
    scores, parent, tok = O.beam_expand(lp, ids, last, 3)
    # products: 0.2, 0.12, 0.08 | 0.36, 0.15, 0.09
    assert parent.tolist() == [1, 0, 1] and tok.tolist() == [20, 10, 21]
    np.testing.assert_allclose(np.exp(scores), [0.36, 0.2, 0.15], rtol=1e-14)
    # ties go to the lower parent row, then the lower rank
    s2, p2, t2 = O.beam_expand(np.zeros((2, 2)), np.array([[1, 2], [3, -1]]), None, 4)
    assert p2.tolist() == [0, 0, 1] and t2.tolist() == [1, 2, 3]  # the empty candidate is never chosen


# ---------------------------------------------------------------- Algorithm 1, one cycle
def _cycle_problem(seed, V, M, d, H=6):
    """A tiny cycle: router over [h_parent, emb(token)] (d_r = 2d, as in
    Algorithm 1) and a fixed map standing in for the draft layer."""
    rng = np.random.default_rng(seed)
    cluster_of = rng.permutation(np.arange(V) % M)
    W = rng.standard_normal((V, d))
    E = rng.standard_normal((V, d))
    A = rng.standard_normal((d, 2 * d)) / np.sqrt(2 * d)
    W1, W2 = rng.standard_normal((H, 2 * d)), rng.standard_normal((M, H))
    h0 = rng.standard_normal((1, d))
    x0 = np.concatenate([rng.standard_normal((1, d)), E[[3]]], axis=1)

    def next_inputs(hp, tok):
        xin = np.concatenate([hp, E[np.asarray(tok)]], axis=1)
        return xin, np.tanh(xin @ A.T) * 2.0
    return cluster_of, W, W1, W2, x0, h0, next_inputs


@pytest.mark.parametrize("seed", range(3))
def test_draft_cycle_on_the_full_vocabulary_is_a_brute_force_beam(seed):
    """Budget M at every position (k_min = M): the shortlist is the whole
    vocabulary, and each position's beam is the k_t best of ALL (parent,
    token) extensions by path log-probability (the best k_t overall always
    lie inside the parents' own k_t best, so the per-row cut loses nothing)."""
    from scipy.special import log_softmax as ref_lsm
    V, M, d, k_t, gamma = 12, 4, 5, 3, 3
    cluster_of, W, W1, W2, x0, h0, nxt = _cycle_problem(seed, V, M, d)
    pos, dl = O.draft_cycle(x0, h0, nxt, W1, W2, "silu", cluster_of, M, W, M, M, k_t, gamma, k_min=M)
    beam = [(0.0, h0[0], ())]  # (path log-prob, hidden row, tokens so far)
    listed = []
    for j in range(gamma + 1):
        assert pos[j]["k"] == M
        ext = []
        for b, (sc, hb, path) in enumerate(beam):
            lp = ref_lsm(W @ hb)
            for v in range(V):
                ext.append((sc + lp[v], b, v))
            listed += [sc + lp[v] for v in sorted(range(V), key=lambda v: (-lp[v], v))[:k_t]]
        ext.sort(key=lambda e: (-e[0], e[1], e[2]))
        best = ext[:k_t]
        np.testing.assert_allclose(pos[j]["scores"], [e[0] for e in best], rtol=1e-12)
        assert pos[j]["parents"].tolist() == [e[1] for e in best]
        assert pos[j]["tokens"].tolist() == [e[2] for e in best]
        hp = np.stack([beam[e[1]][1] for e in best])
        _, hn = nxt(hp, [e[2] for e in best])
        beam = [(e[0], hn[i], beam[e[1]][2] + (e[2],)) for i, e in enumerate(best)]
    # the draft list: every row's k_t candidates of every position, by path score
    np.testing.assert_allclose(dl["scores"], sorted(listed, reverse=True), rtol=1e-12)
    assert len(dl["ids"]) == k_t + gamma * k_t * k_t


def test_draft_cycle_budget_union_and_parent_rows():
    """Position j routes every row with k_c(j) clusters, all rows share the
    union of their clusters, and position j+1's router input row i is
    [h~_j[parent_i], emb(token_i)] (h~[-1] for every row after position 0)."""
    V, M, d, k_t, gamma = 40, 10, 4, 3, 4
    cluster_of, W, W1, W2, x0, h0, nxt = _cycle_problem(7, V, M, d)
    pos, dl = O.draft_cycle(x0, h0, nxt, W1, W2, "silu", cluster_of, M, W, 8, 6, k_t, gamma)
    assert [p["k"] for p in pos] == [8, 6, 2, 1, 1]    # eq. pos_schedule for k0 = 8, k1 = 6
    x, h = x0, h0
    for j, p in enumerate(pos):
        s = O.router_scores(x, W1, W2, act="silu")
        chosen = {m for b in range(len(x)) for m in sorted(range(M), key=lambda m: (-s[b, m], m))[:p["k"]]}
        union = set(np.nonzero(np.isin(cluster_of, sorted(chosen)))[0].tolist())
        for b, r in enumerate(p["heads"]):
            np.testing.assert_allclose(r["scores"], s[b], rtol=1e-12)
            assert set(r["vocab_ids"].tolist()) == union
            assert set(p["ids"][b][p["ids"][b] >= 0].tolist()) <= union
        np.testing.assert_allclose(p["cu_scores"], p["logprobs"] + (0 if j == 0 else pos[j - 1]["scores"][:, None]),
                                   rtol=1e-12)
        x, h = nxt(h[p["parents"]], p["tokens"])
        if j == 0:
            assert np.array_equal(x[:, :d], np.repeat(h0, k_t, axis=0))
    # draft list: sorted, every position's candidates once
    assert np.all(np.diff(dl["scores"]) <= 0)
    assert sorted(zip(dl["position"].tolist(), dl["row"].tolist(), dl["rank"].tolist())) == sorted(
        (j, b, r) for j, p in enumerate(pos) for b in range(p["ids"].shape[0]) for r in range(k_t)
        if p["ids"][b, r] >= 0)


def test_k_equals_M_is_the_dense_head():
    V, M = 64, 8
    cluster_of, W, h, W1, W2, u = _tiny_problem(11, V=V, M=M, d=10, B=4)
    dyn = O.draft_head(h, h, W1, W2, "silu", cluster_of, M, W, M, k_t=5)
    dense = O.dense_head(h, W, k_t=5)
    for i, (a, b) in enumerate(zip(dyn, dense)):
        assert sorted(a["vocab_ids"].tolist()) == list(range(V))
        assert a["ids"].tolist() == b["ids"].tolist()
        np.testing.assert_allclose(a["logprobs"], b["logprobs"], rtol=1e-12)
        np.testing.assert_allclose(a["logits"], b["logits"][a["vocab_ids"]], rtol=1e-12)
        assert a["ids"][0] == int(np.argmax(W @ h[i]))


def test_static_head_is_the_dense_head_on_a_prefix():
    rng = np.random.default_rng(12)
    W, h = rng.standard_normal((50, 7)), rng.standard_normal((2, 7))
    st = O.dense_head(h, W, k_t=4, n_rows=20)
    for b in range(2):
        z = W @ h[b]
        assert st[b]["ids"].tolist() == sorted(range(20), key=lambda v: (-z[v], v))[:4]


def test_k_schedule_closed_form():
    g = GOLD["k_schedule"]
    assert [O.k_schedule(t, g["k0"], g["k1"]) for t in range(10)] == g["t_0_to_9"]
    assert O.k_schedule(100, 64, 32) == 1  # clamped at k_min
    g = GOLD["k_schedule_algorithm1"]
    assert [O.k_schedule(t, g["k0"], g["k1"], form="algorithm1") for t in range(10)] == g["t_0_to_9"]


def test_k_schedule_is_non_increasing_after_the_first_two_positions():
    for k1 in (1, 7, 32, 64, 100):
        for form in ("equation", "algorithm1"):
            ks = [O.k_schedule(t, 200, k1, form=form) for t in range(1, 300)]
            assert all(a >= b for a, b in zip(ks[1:], ks[2:])) and min(ks) >= 1
    # the closed form is round-half-up of k1 / (2t): within 1/2 of it
    for t in range(2, 50):
        assert abs(O.k_schedule(t, 64, 32, k_min=0) - 32 / (2 * t)) <= 0.5 + 1e-12


def test_pa_fr_budget_hand_values():
    g = GOLD["pa_fr"]
    assert [O.pa_fr_budget(t, 32) for t in range(10)] == g["k_max_32"]
    assert [O.pa_fr_budget(t, 32768) for t in range(10)] == g["k_max_32768"]


# ---------------------------------------------------------------- spherical k-means (Sec. 4.2, "Vocabulary partition")
def test_kmeans_similarity_is_exact_below_bf16_resolution():
    # centroid 1 differs from centroid 0 = (1, 0) only below bf16 resolution in
    # its first coordinate: mu1 = (1, 2^-12) / |.|.  For the point (1, 2^-14),
    # exactly, x . mu1 = (1 + 2^-26) / sqrt(1 + 2^-24) < 1 = x . mu0 (times
    # 1/|x|), so cluster 0 wins; rounding mu1 to bf16 gives (1, 2^-12) and
    # would hand the point to cluster 1.
    W = np.array([[1.0, 2.0 ** -14]], dtype=np.float32)
    C = np.array([[1.0, 0.0], [1.0, 2.0 ** -12]])
    C[1] /= np.linalg.norm(C[1])
    assign, S = O.kmeans_assign(W, C)
    assert assign.tolist() == [0]
    assert S[0, 0] - S[0, 1] > 0


def test_kmeans_mean_direction_hand_example():
    # unit points at 0 and 90 degrees, and a long vector at 0 degrees: the
    # points are normalised first, so the resultant is (2, 1), not (6, 1)
    W = np.array([[1.0, 0.0], [0.0, 1.0], [5.0, 0.0]], dtype=np.float32)
    mu = O.kmeans_update(W, [0, 0, 0], 1, np.zeros((1, 2)))
    np.testing.assert_allclose(mu[0], np.array([2.0, 1.0]) / math.sqrt(5.0), rtol=0, atol=1e-15)


def test_kmeans_planted_directions_are_recovered():
    # points are positive multiples of four orthogonal directions (plus a
    # small orthogonal wobble); one point of each group seeds the centroids
    rng = np.random.default_rng(3)
    M, d, per = 4, 8, 25
    E = np.eye(d)[:M]
    rows, truth = [], []
    for m in range(M):
        for _ in range(per):
            wob = np.zeros(d)
            wob[M:] = rng.standard_normal(d - M) * 0.05
            rows.append(E[m] * rng.uniform(0.5, 4.0) + wob)
            truth.append(m)
    W = np.array(rows, dtype=np.float32)
    truth = np.array(truth)
    init = [m * per for m in range(M)]
    assign, mu = O.spherical_kmeans(W, M, init, iters=3)
    np.testing.assert_array_equal(assign, truth)
    for m in range(M):
        assert mu[m, m] > 0.99 and abs(np.linalg.norm(mu[m]) - 1.0) < 1e-12


def test_kmeans_assignment_is_euclidean_argmin_on_the_sphere():
    # with unit centroids, max cosine = min euclidean distance between unit
    # vectors; centroids are the rows of a normalised Hadamard matrix and of
    # its negation, plus random unit vectors
    from sklearn.metrics import pairwise_distances_argmin
    H = 0.5 * np.array([[1, 1, 1, 1], [1, -1, 1, -1], [1, 1, -1, -1], [1, -1, -1, 1]], dtype=np.float64)
    rng = np.random.default_rng(5)
    R = rng.standard_normal((5, 4))
    C = np.vstack([H, -H, R / np.linalg.norm(R, axis=1, keepdims=True)])
    W = rng.standard_normal((500, 4)).astype(np.float32)
    assign, _ = O.kmeans_assign(W, C)
    X = W.astype(np.float64) / np.linalg.norm(W.astype(np.float64), axis=1, keepdims=True)
    np.testing.assert_array_equal(assign, pairwise_distances_argmin(X, C))


def test_kmeans_ties_go_to_the_lower_cluster_and_empty_clusters_keep_their_centroid():
    W = np.array([[1.0, 0.0], [1.0, 0.1], [0.0, 1.0]], dtype=np.float32)
    C = np.array([[1.0, 0.0], [1.0, 0.0], [0.0, 1.0]])  # clusters 0 and 1 coincide
    assign, _ = O.kmeans_assign(W, C)
    assert assign.tolist() == [0, 0, 2]
    mu = O.kmeans_update(W, assign, 3, C)
    np.testing.assert_array_equal(mu[1], C[1])  # empty: unchanged
    assert mu[0, 1] > 0  # moved toward the second point


def test_kmeans_is_invariant_to_positive_row_scales():
    rng = np.random.default_rng(11)
    W = rng.standard_normal((300, 16)).astype(np.float32)
    scale = rng.uniform(0.1, 10.0, size=(300, 1)).astype(np.float32)
    init = rng.choice(300, size=6, replace=False)
    a1, mu1 = O.spherical_kmeans(W, 6, init, iters=4)
    a2, mu2 = O.spherical_kmeans(W * scale, 6, init, iters=4)
    np.testing.assert_array_equal(a1, a2)
    np.testing.assert_allclose(mu1, mu2, rtol=0, atol=1e-6)


def test_kmeans_steps_each_maximise_the_objective_and_end_at_a_fixed_point():
    # the assignment maximises the summed similarity to the centroids
    # given them, the update maximises it over unit centroids given the
    # assignment; brute force over all centroids confirms every final choice
    rng = np.random.default_rng(2)
    W = rng.standard_normal((60, 5)).astype(np.float32)
    M = 4
    init = rng.choice(60, size=M, replace=False)
    X = O.unit_rows(W)
    mu = X[init]
    a = np.zeros(60, dtype=np.int64)
    for it in range(30):
        a_new, _ = O.kmeans_assign(W, mu)
        if it:
            assert O.kmeans_objective(W, a_new, mu) >= O.kmeans_objective(W, a, mu) - 1e-12
        a = a_new
        mu_new = O.kmeans_update(W, a, M, mu)
        assert O.kmeans_objective(W, a, mu_new) >= O.kmeans_objective(W, a, mu) - 1e-12
        # no other unit vector does better for one cluster (random probes)
        for m in range(M):
            mem = X[a == m]
            if len(mem):
                best = float(mem.sum(0) @ mu_new[m])
                probes = rng.standard_normal((50, 5))
                probes /= np.linalg.norm(probes, axis=1, keepdims=True)
                assert np.all(mem.sum(0) @ probes.T <= best + 1e-12)
        mu = mu_new
    a, _ = O.kmeans_assign(W, mu)
    for v in range(60):
        sims = [float(np.dot(X[v], mu[m])) for m in range(M)]
        assert a[v] == min(m for m in range(M) if sims[m] == max(sims))
