"""GPU parity of libdynahead against the CPU oracle (stage-wise), small sizes.

Sizes here run in seconds on the oracle but span several 16-row tiles, ragged
cluster tails, a ragged reduction dimension (d = 200 is not a multiple of the
32-wide MFMA step nor of the 512-wide GEMV block), both logits kernels and
both router kernels.  Full-size workloads are in test_gpu_fullsize.py.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import dynaspec_oracle as O
from tests import parity as PC

pytestmark = pytest.mark.gpu

D = None


@pytest.fixture(scope="module", autouse=True)
def _lib():
    global D
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2510_13847_amd import dynahead
    D = dynahead
    D.lib()
    yield
    D.set_option(D.OPT_LOGITS_PATH, 0)
    D.set_option(D.OPT_ROUTER_PATH, 0)


DEV = "cuda"
BASE = W.WORKLOADS["llama3_8b_chain"]


def case(name, **kw):
    kw.setdefault("modes", ("topk", "sample"))
    kw.setdefault("k_t", 6)
    return W.scaled(BASE, name=name, **kw)


CASES = [
    W.WORKLOADS["tiny_fp32"],
    case("ragged_b1", V=3001, d=200, M=37, H=24, k=5, B=1),
    case("ragged_b3", V=3001, d=200, M=37, H=24, k=5, B=3),
    case("ragged_b7", V=3001, d=200, M=37, H=24, k=5, B=7),
    case("ragged_b37", V=3001, d=200, M=37, H=24, k=5, B=37),
    case("f32_b5", V=2000, d=136, M=20, H=16, k=4, B=5, dtype="f32"),
    case("linear_b20", V=2500, d=264, M=30, H=0, act="none", k=4, B=20),
    case("relu_b2", V=1500, d=128, M=16, H=32, act="relu", k=3, B=2),
    case("zipf_b9", V=6000, d=96, M=12, sizes=("zipf", 1.1, 1500), H=16, k=3, B=9),
    case("wide_k_b4", V=4096, d=512, M=64, H=64, k=64, B=4),  # k = M: shortlist = V
    # split-K router with four column groups and several k slices
    case("wide_b64", V=4000, d=520, M=40, H=48, k=4, B=64),
    # more contexts than one MFMA column pass (and than the split-K router takes)
    case("many_b130", V=3000, d=136, M=24, H=32, k=3, B=130),
]


class Problem:
    def __init__(self, w, gen_device="cpu"):
        self.w = w
        self.cluster_of = W.partition(w)
        self.W_lm = W.lm_head(w, gen_device)
        self.W1, self.W2 = W.router_weights(w, gen_device)
        self.h = W.contexts(w, gen_device)
        self.u = W.uniforms(w, gen_device)
        self.hd = self.h.to(DEV)
        self.ud = self.u.to(DEV)
        self.L = D.build_layout(torch.from_numpy(self.cluster_of).to(DEV), self.W_lm.to(DEV), w.M)
        self.R = D.Router(self.W1.to(DEV), None if self.W2 is None else self.W2.to(DEV), act=w.act)
        # host copies for the oracle
        self.h_np = W.host_array(self.h)
        self.W_np = W.host_array(self.W_lm)
        self.W1_np = W.host_array(self.W1)
        self.W2_np = None if self.W2 is None else W.host_array(self.W2)
        self.u_np = self.u.numpy().astype(np.float64)
        self.sizes, self.offsets, self.perm, self.cap = O.cluster_layout(self.cluster_of, w.M)
        self.tol = PC.TOL[w.dtype]

    def oracle_scores(self):
        return O.router_scores(self.h_np, self.W1_np, self.W2_np, act=self.w.act)


def _ids(tensor):
    return tensor.cpu().numpy().astype(np.int64)


# ---------------------------------------------------------------- layout
@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_layout_exact(w):
    p = Problem(w)
    assert _ids(p.L.perm).tolist() == p.perm.tolist()
    assert _ids(p.L.offsets).tolist() == p.offsets.tolist()
    assert p.L.cap_by_k.tolist() == p.cap.tolist()
    assert p.L.max_cluster == int(p.sizes.max())
    got = W.host_array(p.L.W_perm.cpu())
    np.testing.assert_array_equal(got, p.W_np[p.perm])


def test_layout_with_empty_clusters_and_bad_ids():
    rng = np.random.default_rng(5)
    V, M, d = 700, 40, 64
    cluster_of = rng.integers(0, M, size=V).astype(np.int32)
    cluster_of[np.isin(cluster_of, [3, 17, 39])] = 0  # three empty clusters, one big
    Wl = torch.randn(V, d).to(torch.bfloat16)
    L = D.build_layout(torch.from_numpy(cluster_of).to(DEV), Wl.to(DEV), M)
    sizes, offsets, perm, cap = O.cluster_layout(cluster_of, M)
    assert _ids(L.offsets).tolist() == offsets.tolist() and _ids(L.perm).tolist() == perm.tolist()
    assert L.cap_by_k.tolist() == cap.tolist()
    bad = cluster_of.copy()
    bad[123] = M  # out of range: flagged on the device, reported on the host
    with pytest.raises(D.DynaError) as e:
        D.build_layout(torch.from_numpy(bad).to(DEV), Wl.to(DEV), M)
    assert e.value.status == D.ERR_DEVICE_DATA


# ---------------------------------------------------------------- router
def _paths(paths, mfma_from):
    """(case, path) pairs; the MFMA paths (path >= mfma_from) take bf16 weights only."""
    return [pytest.param(w, p, id=f"{w.name}-{p}") for w in CASES for p in paths
            if p < mfma_from or w.dtype != "f32"]


@pytest.mark.parametrize("w,path", _paths([0, 1, 2, 3], 2))
def test_route_parity(w, path):
    p = Problem(w)
    D.set_option(D.OPT_ROUTER_PATH, path)
    try:
        ids, sc, scores = D.route(p.R, p.hd, w.k, want_scores=True)
        torch.cuda.synchronize()
    finally:
        D.set_option(D.OPT_ROUTER_PATH, 0)
    ref = p.oracle_scores()
    g_scores = scores.cpu().numpy().astype(np.float64)
    PC.assert_close(g_scores, ref, PC.SCORE_TOL, "router scores")
    g_ids = _ids(ids)
    # the top-k kernel is exact on its own fp32 scores (same ordering rule)
    ids_own, vals_own = O.topk_clusters(g_scores, w.k)
    np.testing.assert_array_equal(g_ids, ids_own)
    np.testing.assert_array_equal(sc.cpu().numpy().astype(np.float64), vals_own)
    strict = 0
    for b in range(w.B):
        eq, ok = PC.cluster_check(g_ids[b], ref[b], w.k)
        assert ok, f"row {b}: clusters {g_ids[b]} not a valid top-{w.k}"
        strict += int(not eq)
    assert strict <= PC.strict_limit(w.B)


@pytest.mark.parametrize("B", [5, 9, 16, 17])
@pytest.mark.parametrize("x_dtype", ["bf16", "f32"])
def test_route_hidden_from_partial_sums(B, x_dtype):
    """5..16 contexts: router layer 2 stages the hidden layer from layer 1's
    split-K partial sums (added in slice order, then bias and activation)
    instead of a reduction launch.  The scores must equal, bit for bit, those
    of the explicit split-K path with its reduction kernel (router path 2),
    and the oracle's within the score tolerance; 17 contexts take the
    reduction launch on both paths."""
    w = case(f"hid_b{B}", V=3001, d=1000, M=300, H=520, k=5, B=B)
    p = Problem(w)
    x = p.hd if x_dtype == "bf16" else p.hd.float()
    out = {}
    for path in (0, 2):
        D.set_option(D.OPT_ROUTER_PATH, path)
        try:
            _, _, scores = D.route(p.R, x, w.k, want_scores=True)
            torch.cuda.synchronize()
        finally:
            D.set_option(D.OPT_ROUTER_PATH, 0)
        out[path] = scores.cpu()
    assert torch.equal(out[0], out[2])
    # the fp32 contexts hold the bf16 values exactly: the same reference
    PC.assert_close(out[0].numpy().astype(np.float64), p.oracle_scores(), PC.SCORE_TOL, "router scores")


def test_route_nan_and_ties():
    # NaN features make every score NaN: all count as -inf, ties go to lower ids
    M, d_r = 50, 64
    W1 = torch.randn(M, d_r).to(torch.bfloat16).to(DEV)
    x = torch.full((3, d_r), float("nan")).to(torch.bfloat16).to(DEV)
    R = D.Router(W1, None, act="none")
    ids, sc, _ = D.route(R, x, 7)
    assert _ids(ids).tolist() == [list(range(7))] * 3
    # exact ties: zero weights give all-zero scores; +0 and -0 must compare equal
    W0 = torch.zeros(M, d_r).to(torch.bfloat16).to(DEV)
    xz = torch.randn(2, d_r).to(torch.bfloat16).to(DEV)
    ids, _, _ = D.route(D.Router(W0, None, act="none"), xz, 5)
    assert _ids(ids).tolist() == [list(range(5))] * 2


# ---------------------------------------------------------------- shortlist
@pytest.mark.parametrize("w", CASES[:5], ids=lambda w: w.name)
def test_shortlist_exact_union(w):
    p = Problem(w)
    rng = np.random.default_rng(11)
    B, k, M = 6, w.k, w.M
    topk = np.stack([rng.choice(M, size=k, replace=False) for _ in range(B)]).astype(np.int32)
    sel, rowoff, row_len, sl = D.shortlist(p.L, torch.from_numpy(topk).to(DEV))
    sel, rowoff, row_len, sl = _ids(sel), _ids(rowoff), _ids(row_len), _ids(sl)
    for b in range(B):
        s_o, r_o, rows_o, vids_o = O.shortlist(topk[b], p.offsets, p.perm)
        assert sel[b].tolist() == s_o.tolist()
        assert rowoff[b].tolist() == r_o.tolist()
        assert row_len[b] == len(vids_o)
        assert sl[b, :row_len[b]].tolist() == vids_o.tolist()
        assert np.all(sl[b, row_len[b]:] == -1)  # untouched past row_len


def test_shortlist_ignores_repeats_and_out_of_range():
    w = CASES[1]
    p = Problem(w)
    topk = np.array([[3, 3, 7, -1, 36], [40, 0, 0, 0, 1]], dtype=np.int32)
    sel, rowoff, row_len, sl = D.shortlist(p.L, torch.from_numpy(topk).to(DEV))
    sel, rowoff, row_len = _ids(sel), _ids(rowoff), _ids(row_len)
    assert sel[0].tolist() == [3, 7, 36, -1, -1]
    assert sel[1].tolist() == [0, 1, -1, -1, -1]
    for b, valid in enumerate([[3, 7, 36], [0, 1]]):
        assert row_len[b] == sum(p.sizes[m] for m in valid)
        assert rowoff[b, -1] == row_len[b]


# ---------------------------------------------------------------- logits
def _random_selection(p, B, k, seed):
    """Random distinct clusters per context; half the batch shares one cluster,
    like a router biased toward a popular cluster."""
    rng = np.random.default_rng(seed)
    M = p.w.M
    common = int(rng.integers(M))
    others = np.array([m for m in range(M) if m != common])
    rows = []
    for b in range(B):
        if B > 2 and b < B // 2:
            rows.append([common] + rng.choice(others, size=k - 1, replace=False).tolist())
        else:
            rows.append(rng.choice(M, size=k, replace=False).tolist())
    return np.array(rows, dtype=np.int32)


@pytest.mark.parametrize("w,path", _paths([1, 2], 2))
def test_logits_parity(w, path):
    """Paths: 1 GEMV, 2 MFMA with LDS-staged slabs (bf16 weights only)."""
    p = Problem(w)
    topk = _random_selection(p, w.B, w.k, 3)
    sel, rowoff, row_len, sl = D.shortlist(p.L, torch.from_numpy(topk).to(DEV))
    D.set_option(D.OPT_LOGITS_PATH, path)
    try:
        logits = D.shortlist_logits(p.L, p.hd, sel, rowoff, row_len)
        torch.cuda.synchronize()
    finally:
        D.set_option(D.OPT_LOGITS_PATH, 0)
    lg = logits.cpu().numpy().astype(np.float64)
    row_len, sl = _ids(row_len), _ids(sl)
    for b in range(w.B):
        n = row_len[b]
        ref = O.shortlist_logits(p.h_np[b], p.W_np, sl[b, :n])
        PC.assert_close(lg[b, :n], ref, p.tol, f"logits row {b}")
        PC.assert_tight(lg[b, :n], p.h_np[b], p.W_np[sl[b, :n]], f"logits row {b}")
        assert np.all(np.isnan(lg[b, n:])), "slots past row_len must stay untouched"


# d = 1000: four to eight k blocks for the split shapes, the last one a tail
GATHER_EXTRA = {"kdeep_b6": case("kdeep_b6", V=3001, d=1000, M=37, H=24, k=5, B=6)}


@pytest.mark.parametrize("cfg", list(range(0, 10)))
@pytest.mark.parametrize("name", ["ragged_b37", "zipf_b9", "many_b130", "kdeep_b6"])
def test_logits_gather_shapes(name, cfg):
    """Every workgroup shape of the LDS-staged MFMA gathered head, with and
    without the waves splitting the k dimension of a chunk."""
    w = GATHER_EXTRA[name] if name in GATHER_EXTRA else next(c for c in CASES if c.name == name)
    p = Problem(w)
    topk = _random_selection(p, w.B, w.k, 5)
    sel, rowoff, row_len, sl = D.shortlist(p.L, torch.from_numpy(topk).to(DEV))
    D.set_option(D.OPT_LOGITS_PATH, 2)
    D.set_option(D.OPT_GATHER_CFG, cfg)
    try:
        logits = D.shortlist_logits(p.L, p.hd, sel, rowoff, row_len)
        torch.cuda.synchronize()
    finally:
        D.set_option(D.OPT_LOGITS_PATH, 0)
        D.set_option(D.OPT_GATHER_CFG, 0)
    lg = logits.cpu().numpy().astype(np.float64)
    row_len, sl = _ids(row_len), _ids(sl)
    for b in range(w.B):
        n = row_len[b]
        ref = O.shortlist_logits(p.h_np[b], p.W_np, sl[b, :n])
        PC.assert_close(lg[b, :n], ref, p.tol, f"cfg {cfg} logits row {b}")
        PC.assert_tight(lg[b, :n], p.h_np[b], p.W_np[sl[b, :n]], f"cfg {cfg} logits row {b}")


# ---------------------------------------------------------------- select
def _select_problem(seed, B=5, with_ties=True):
    w = CASES[2]
    p = Problem(w)
    topk = _random_selection(p, B, w.k, seed)
    sel, rowoff, row_len, sl = D.shortlist(p.L, torch.from_numpy(topk).to(DEV))
    cap = p.L.cap(w.k)
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((B, cap)) * 3).astype(np.float32)
    if with_ties:
        z[:, 5:40] = np.round(z[:, 5:40])  # many exactly equal logits
        z[0, :] = 1.25                      # a row of all-equal logits
    return p, sel, rowoff, row_len, sl, torch.from_numpy(z).to(DEV), z


@pytest.mark.parametrize("k_t", [1, 4, 13, 64])
@pytest.mark.parametrize("temperature", [1.0, 0.7])
def test_select_exact_on_same_logits(k_t, temperature):
    p, sel, rowoff, row_len, sl, zd, z = _select_problem(7 + k_t)
    B = z.shape[0]
    u = torch.rand(B, generator=torch.Generator().manual_seed(k_t)).to(DEV)
    out = D.draft_select(p.L, zd, sel, rowoff, row_len, mode=D.SEL_TOPK | D.SEL_SAMPLE, k_t=k_t,
                         temperature=temperature, uniforms=u)
    torch.cuda.synchronize()
    row_len, sl = _ids(row_len), _ids(sl)
    ids, lps = _ids(out["ids"]), out["logprobs"].cpu().numpy()
    smp, slp = _ids(out["sample"]), out["sample_logprob"].cpu().numpy()
    un = u.cpu().numpy().astype(np.float64)
    strict = 0
    for b in range(B):
        n = row_len[b]
        zb = z[b, :n].astype(np.float64)
        r = O.draft_select(zb, sl[b, :n], min(k_t, n), temperature, un[b])
        m = min(k_t, n)
        assert ids[b, :m].tolist() == r["ids"].tolist(), f"row {b}"
        assert np.all(ids[b, m:] == -1)
        PC.assert_close(lps[b, :m], r["logprobs"], PC.LOGPROB_TOL, "logprobs")
        eq, ok = PC.sample_check(smp[b], zb, sl[b, :n], un[b], temperature)
        assert ok, f"row {b}: sample {smp[b]}"
        strict += int(not eq)
        j = int(np.nonzero(sl[b, :n] == smp[b])[0][0])
        PC.assert_close([slp[b]], [O.log_softmax(zb, temperature)[j]], PC.LOGPROB_TOL, "sample lp")
    assert strict <= PC.strict_limit(B), f"{strict} sampled tokens differ from the oracle's"


def test_sampling_grid_matches_probabilities():
    # a sweep of u over [0, 1) must hit every shortlist slot in proportion to q_S
    p, sel, rowoff, row_len, sl, zd, z = _select_problem(3, B=1, with_ties=False)
    N = 4096
    n = int(_ids(row_len)[0])
    zsmall = zd.clone()
    zsmall[0, :n] = torch.linspace(-2.0, 2.0, n, device=DEV)
    sel_r = sel.repeat(N, 1)
    rowoff_r = rowoff.repeat(N, 1)
    rl_r = row_len.repeat(N)
    zr = zsmall.repeat(N, 1)
    u = (torch.arange(N, dtype=torch.float32, device=DEV) + 0.5) / N
    out = D.draft_select(p.L, zr, sel_r, rowoff_r, rl_r, mode=D.SEL_SAMPLE, uniforms=u)
    smp = _ids(out["sample"])
    sl0 = _ids(sl)[0, :n]
    zb = zsmall[0, :n].cpu().numpy().astype(np.float64)
    q = np.exp(O.log_softmax(zb))
    counts = np.array([(smp == v).sum() for v in sl0])
    assert counts.sum() == N
    assert np.all(np.abs(counts - q * N) <= 1.0 + 1e-6 * N)


# ---------------------------------------------------------------- whole head
def _check_head(p, head, modes_ids=True, k=None, ref_scores=None):
    w = p.w
    k = w.k if k is None else k
    ref_scores = p.oracle_scores() if ref_scores is None else ref_scores
    clusters = _ids(head.clusters)
    logits = head.logits.cpu().numpy().astype(np.float64)
    strict_c = strict_s = 0
    for b in range(w.B):
        eq, ok = PC.cluster_check(clusters[b], ref_scores[b], k)
        assert ok, f"row {b}: clusters"
        strict_c += int(not eq)
        sel, rowoff, rows, vids = O.shortlist(clusters[b], p.offsets, p.perm)
        n = len(vids)
        z_ref = O.shortlist_logits(p.h_np[b], p.W_np, vids)
        PC.assert_close(logits[b, :n], z_ref, p.tol, f"head logits row {b}")
        PC.assert_tight(logits[b, :n], p.h_np[b], p.W_np[vids], f"head logits row {b}")
        z_gpu = logits[b, :n]
        if head.ids is not None:
            kt = head.ids.shape[1]
            got = _ids(head.ids)[b]
            r = O.draft_select(z_gpu, vids, min(kt, n))
            assert got[:min(kt, n)].tolist() == r["ids"].tolist()     # exact on own logits
            eq, ok = PC.tokens_check(got, z_ref, vids, kt)             # vs oracle logits
            assert ok
        if head.sample is not None:
            eq, ok = PC.sample_check(_ids(head.sample)[b], z_gpu, vids, p.u_np[b], head.temperature)
            assert ok, f"row {b}: sample"
            strict_s += int(not eq)
    assert strict_c <= PC.strict_limit(w.B), f"{strict_c} rows' clusters differ from the oracle's"
    assert strict_s <= PC.strict_limit(w.B), f"{strict_s} sampled tokens differ from the oracle's"
    return strict_c, strict_s


@pytest.mark.parametrize("form", [0, 1])
def test_position_aware_chain(form):
    """Draft positions t = 0..5, each routed with its cluster budget k_c(t)
    (Sec. 4.2, eq. pos_schedule; form 1: the appendix algorithm's variant)."""
    w = next(c for c in CASES if c.name == "ragged_b7")
    p = Problem(w)
    k0, k1 = min(w.M, 12), min(w.M, 6)
    mode = D.SEL_TOPK | D.SEL_SAMPLE
    for t in range(6):
        k = D.cluster_budget(t, k0, k1, 1, form)
        assert k == O.k_schedule(t, k0, k1, form=("equation", "algorithm1")[form])
        head = D.draft_head(p.R, p.L, p.hd, p.hd, k, mode=mode, k_t=w.k_t, uniforms=p.ud)
        torch.cuda.synchronize()
        _check_head(p, head, k=k)


@pytest.mark.parametrize("beta", [0.25, 0.6])
@pytest.mark.parametrize("name", ["ragged_b37", "ragged_b1"])
def test_tail_mixture(name, beta):
    """Tail mixture proposal of Sec. 5: q~ = (1 - beta) q_S + beta * uniform(V minus S).
    Shortlist ids are unchanged, log-probabilities shift by log(1 - beta), and a
    uniform past 1 - beta picks complement entry floor((u - (1 - beta)) / beta * |V minus S|)
    in layout order."""
    w = next(c for c in CASES if c.name == name)
    p = Problem(w)
    u = torch.linspace(0.0, 0.999, w.B, dtype=torch.float32) if w.B > 1 else torch.tensor([0.9])
    ud = u.to(DEV)
    # one context without sampling: the fused head (argmax and top-k)
    modes = [D.SEL_TOPK | D.SEL_SAMPLE] + ([D.SEL_ARGMAX, D.SEL_TOPK] if w.B == 1 else [])
    for mode in modes:
        kt = w.k_t if mode & D.SEL_TOPK else 1
        base = D.draft_head(p.R, p.L, p.hd, p.hd, w.k, mode=mode, k_t=kt, uniforms=ud)
        tail = D.draft_head(p.R, p.L, p.hd, p.hd, w.k, mode=mode, k_t=kt, uniforms=ud, tail_beta=beta)
        torch.cuda.synchronize()
        assert torch.equal(base.clusters, tail.clusters) and torch.equal(base.ids, tail.ids)
        lb, lt = base.logprobs.cpu().numpy(), tail.logprobs.cpu().numpy()
        fin = np.isfinite(lb)
        np.testing.assert_allclose(lt[fin], lb[fin] + np.log1p(-beta), rtol=0, atol=2e-5)
        if not mode & D.SEL_SAMPLE:
            continue
        clusters = _ids(tail.clusters)
        logits = tail.logits.cpu().numpy().astype(np.float64)
        strict = 0
        for b in range(w.B):
            sel, rowoff, rows, vids = O.shortlist(clusters[b], p.offsets, p.perm)
            comp = O.complement(p.offsets, p.perm, sel)
            ub = float(u[b])
            got = int(_ids(tail.sample)[b])
            if abs(ub - (1.0 - beta)) < 1e-6:
                continue  # branch decided at the fp32 boundary
            if ub < 1.0 - beta:
                eq, ok = PC.sample_check(got, logits[b, :len(vids)], vids, ub / (1.0 - beta), 1.0)
                assert ok, f"row {b}: shortlist branch"
                strict += int(not eq)
            else:
                x = (ub - (1.0 - beta)) / beta * len(comp)
                jj = min(len(comp) - 1, int(np.floor(x)))
                ok = got == comp[jj] or (abs(x - round(x)) < 1e-4 and got in comp[max(0, jj - 1):jj + 2])
                assert ok, f"row {b}: tail branch"
                lp = float(tail.sample_logprob.cpu().numpy()[b])
                assert abs(lp - (np.log(beta) - np.log(len(comp)))) < 1e-5
        assert strict <= PC.strict_limit(w.B)


UNION_VARIANTS = {**{f"dense{c}": (0, c) for c in range(16)}, "gemv": (1, 0), "lds": (2, 0)}
# a union longer than 16384 slots: the segmented selection
UNION_EXTRA = {"long_b8": case("long_b8", V=40000, d=64, M=48, H=16, k=12, B=8)}


# fp32 heads take the GEMV path only
@pytest.mark.parametrize("name,variant", [
    pytest.param(n, v, id=f"{n}-{v}")
    for n in ["ragged_b3", "ragged_b37", "zipf_b9", "wide_b64", "many_b130", "f32_b5", "long_b8"]
    for v in UNION_VARIANTS if n != "f32_b5" or v == "gemv"])
def test_union_shortlist_head(name, variant):
    """Union routing (Sec. 4.2): the rows of a step share one shortlist, the
    union of their selected clusters; every row's logits, tokens and sample
    are over that union (the oracle's draft_head(union=True) on the same
    clusters).  Variants: the dense union kernel (four or eight waves per
    workgroup) and the per-chunk-list kernels on the same plan."""
    w = UNION_EXTRA[name] if name in UNION_EXTRA else next(c for c in CASES if c.name == name)
    path, cfg = UNION_VARIANTS[variant]
    p = Problem(w)
    mode = D.SEL_TOPK | D.SEL_SAMPLE
    D.set_option(D.OPT_LOGITS_PATH, path)
    D.set_option(D.OPT_UNION_CFG, cfg)
    try:
        try:
            head = D.draft_head(p.R, p.L, p.hd, p.hd, w.k, mode=mode | D.SEL_UNION, k_t=w.k_t, uniforms=p.ud)
        except D.DynaError as e:
            # a fixed shape may not fit; the automatic one must always run
            if e.status == D.ERR_UNSUPPORTED and "does not fit" in str(e) and cfg != 0:
                pytest.skip("fixed union shape does not fit in LDS at this context count")
            raise
        torch.cuda.synchronize()
    finally:
        D.set_option(D.OPT_LOGITS_PATH, 0)
        D.set_option(D.OPT_UNION_CFG, 0)
    assert head.cap == min(w.V, w.B * int(p.cap[w.k]))
    ref_scores = p.oracle_scores()
    clusters = _ids(head.clusters)
    strict_c = strict_s = 0
    for b in range(w.B):
        eq, ok = PC.cluster_check(clusters[b], ref_scores[b], w.k)
        assert ok, f"row {b}: clusters"
        strict_c += int(not eq)
    union = O.union_clusters(clusters)
    sel, rowoff, rows, vids = O.shortlist(union, p.offsets, p.perm)
    n = len(vids)
    logits = head.logits.cpu().numpy().astype(np.float64)
    ids, smp = _ids(head.ids), _ids(head.sample)
    kt = min(w.k_t, n)
    for b in range(w.B):
        z_ref = O.shortlist_logits(p.h_np[b], p.W_np, vids)
        PC.assert_close(logits[b, :n], z_ref, p.tol, f"union logits row {b}")
        PC.assert_tight(logits[b, :n], p.h_np[b], p.W_np[vids], f"union logits row {b}")
        r = O.draft_select(logits[b, :n], vids, kt)
        assert ids[b, :kt].tolist() == r["ids"].tolist()  # exact on own logits
        eq, ok = PC.tokens_check(ids[b], z_ref, vids, w.k_t)
        assert ok, f"row {b}: tokens"
        eq, ok = PC.sample_check(smp[b], logits[b, :n], vids, p.u_np[b], head.temperature)
        assert ok, f"row {b}: sample"
        strict_s += int(not eq)
    assert strict_c <= PC.strict_limit(w.B) and strict_s <= PC.strict_limit(w.B), (strict_c, strict_s)
    # the oracle's union head agrees wherever its routing equals the kernels'
    ref = O.draft_head(p.h_np, p.h_np, p.W1_np, p.W2_np, w.act, p.cluster_of, w.M, p.W_np, w.k,
                       k_t=w.k_t, union=True)
    if O.union_clusters(np.stack([r["clusters"] for r in ref])).tolist() == union.tolist():
        for b in range(w.B):
            assert ref[b]["vocab_ids"].tolist() == vids.tolist()
            eq, ok = PC.tokens_check(ids[b], ref[b]["logits"], vids, w.k_t)
            assert ok
    # the per-row head on the same step is a different (smaller) shortlist
    own = D.draft_head(p.R, p.L, p.hd, p.hd, w.k, mode=mode, k_t=w.k_t, uniforms=p.ud)
    torch.cuda.synchronize()
    assert torch.equal(own.clusters, head.clusters)


def test_union_one_row_is_the_per_row_head():
    w = next(c for c in CASES if c.name == "ragged_b1")
    p = Problem(w)
    mode = D.SEL_TOPK | D.SEL_SAMPLE
    a = D.draft_head(p.R, p.L, p.hd, p.hd, w.k, mode=mode | D.SEL_UNION, k_t=w.k_t, uniforms=p.ud)
    b = D.draft_head(p.R, p.L, p.hd, p.hd, w.k, mode=mode, k_t=w.k_t, uniforms=p.ud)
    torch.cuda.synchronize()
    assert torch.equal(a.ids, b.ids) and torch.equal(a.sample, b.sample)
    assert torch.equal(a.logprobs, b.logprobs)


def test_union_rejects_small_cap_and_tail():
    w = next(c for c in CASES if c.name == "ragged_b7")
    p = Problem(w)
    head = D.DraftHead(p.R, p.L, w.B, w.k, D.SEL_TOPK | D.SEL_UNION, w.k_t, device=DEV)
    head.cap = p.L.cap(w.k)  # the per-row bound is too small for a union
    if head.cap < head.layout.V:
        with pytest.raises(D.DynaError) as e:
            head(p.hd, p.hd)
        assert e.value.status == D.ERR_CAPACITY
    t = D.DraftHead(p.R, p.L, w.B, w.k, D.SEL_TOPK | D.SEL_UNION, w.k_t, device=DEV, tail_beta=0.3)
    with pytest.raises(D.DynaError) as e:
        t(p.hd, p.hd)
    assert e.value.status == D.ERR_UNSUPPORTED


@pytest.mark.parametrize("B,k_t,n_out", [(1, 1, 1), (1, 8, 8), (6, 8, 8), (20, 12, 64), (16, 16, 16),
                                         (257, 1, 5), (37, 13, 20), (130, 63, 64), (128, 64, 64)])
def test_beam_expand(B, k_t, n_out):
    """EAGLE-2 expansion (Algorithm 1): the n_out best cumulative scores over the
    B x k_t candidates, ordered (score desc, row asc, rank asc); missing tokens
    (id -1) are never chosen.  Up to 256 candidates are ranked by counting,
    more by the radix selection (both sides of the boundary are here)."""
    rng = np.random.default_rng(B * 1000 + k_t)
    lp = -rng.exponential(3.0, size=(B, k_t)).astype(np.float32)
    lp[:, ::3] = np.round(lp[:, ::3] * 4) / 4  # exact ties across rows
    ids = rng.integers(0, 50000, size=(B, k_t)).astype(np.int32)
    ids[rng.random((B, k_t)) < 0.1] = -1
    last = (-rng.exponential(2.0, size=B)).astype(np.float32)
    last[::2] = np.round(last[::2] * 2) / 2
    for lst in (None, last):
        sc, par, tok = D.beam_expand(torch.from_numpy(lp).to(DEV), torch.from_numpy(ids).to(DEV),
                                     None if lst is None else torch.from_numpy(lst).to(DEV), n_out)
        torch.cuda.synchronize()
        cu32 = lp if lst is None else (lp + lst[:, None]).astype(np.float32)  # the kernel's fp32 sums
        r_sc, r_par, r_tok = O.beam_expand(cu32, ids, None, n_out)
        m = len(r_sc)
        assert sc.cpu().numpy()[:m].tolist() == r_sc.astype(np.float32).tolist()
        assert _ids(par)[:m].tolist() == r_par.tolist()
        assert _ids(tok)[:m].tolist() == r_tok.tolist()
        assert np.all(_ids(par)[m:] == -1) and np.all(_ids(tok)[m:] == -1)
        assert np.all(np.isneginf(sc.cpu().numpy()[m:]))


def test_beam_expand_rejects_bad_sizes():
    lp = torch.zeros((2, 4), device=DEV)
    ids = torch.zeros((2, 4), dtype=torch.int32, device=DEV)
    with pytest.raises(D.DynaError):
        D.beam_expand(lp, ids, None, 0)
    with pytest.raises(D.DynaError):
        D.beam_expand(lp, ids, None, 65)
    big = torch.zeros((200, 64), device=DEV)
    with pytest.raises(D.DynaError):
        D.beam_expand(big, torch.zeros((200, 64), dtype=torch.int32, device=DEV), None, 8)


@pytest.mark.parametrize("t", [0, 2, 5])
def test_pa_fr_static_head(t):
    """The position-aware frequency-ranked static head (appendix, PA-FR):
    the first K_fr(t) ids of the vocabulary."""
    w = CASES[4]
    p = Problem(w)
    n = D.static_budget(t, 2048)
    assert n == O.pa_fr_budget(t, 2048)
    B = w.B
    st = D.DenseHead(p.W_lm.to(DEV), n, B, D.SEL_TOPK, 5, keep_logits=True)
    st(p.hd)
    torch.cuda.synchronize()
    for b in range(B):
        r = O.dense_head(p.h_np[b:b + 1], p.W_np, k_t=5, n_rows=n)[0]
        PC.assert_close(st.logits[b].cpu().numpy(), r["logits"], p.tol, "PA-FR logits")
        eq, ok = PC.tokens_check(_ids(st.ids)[b], r["logits"], np.arange(n), 5)
        assert ok


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_draft_head_chain(w):
    p = Problem(w)
    mode = D.SEL_TOPK | D.SEL_SAMPLE
    head = D.draft_head(p.R, p.L, p.hd, p.hd, w.k, mode=mode, k_t=w.k_t, uniforms=p.ud)
    torch.cuda.synchronize()
    _check_head(p, head)
    # the fused call equals the step-by-step calls exactly
    ids, _, _ = D.route(p.R, p.hd, w.k)
    assert torch.equal(ids, head.clusters)
    sel, rowoff, row_len, _ = D.shortlist(p.L, ids, with_ids=False)
    logits = D.shortlist_logits(p.L, p.hd, sel, rowoff, row_len)
    mask = ~torch.isnan(logits)
    assert torch.equal(logits[mask], head.logits[mask])
    out = D.draft_select(p.L, logits, sel, rowoff, row_len, mode=mode, k_t=w.k_t, uniforms=p.ud)
    assert torch.equal(out["ids"], head.ids) and torch.equal(out["sample"], head.sample)


def test_k_equals_M_is_the_dense_head():
    w = CASES[-1]  # k = M = 64: the shortlist is the whole vocabulary
    p = Problem(w)
    mode = D.SEL_TOPK
    head = D.draft_head(p.R, p.L, p.hd, p.hd, w.M, mode=mode, k_t=8)
    dense = D.DenseHead(p.W_lm.to(DEV), w.V, w.B, mode, 8, keep_logits=True)(p.hd)
    torch.cuda.synchronize()
    assert torch.equal(head.ids, dense.ids)
    PC.assert_close(head.logprobs.cpu().numpy(), dense.logprobs.cpu().numpy(), PC.LOGPROB_TOL, "lp")
    # and the dense head itself against the oracle
    for b in range(w.B):
        r = O.dense_head(p.h_np[b:b + 1], p.W_np, k_t=8)[0]
        PC.assert_close(dense.logits[b].cpu().numpy(), r["logits"], p.tol, "dense logits")
        PC.assert_tight(dense.logits[b].cpu().numpy(), p.h_np[b], p.W_np, "dense logits")
        eq, ok = PC.tokens_check(_ids(dense.ids)[b], r["logits"], np.arange(w.V), 8)
        assert ok


@pytest.mark.parametrize("B", [1, 6, 37])
def test_static_head_prefix(B):
    w = CASES[4]
    p = Problem(w)
    n = 777
    hd = p.hd[:B].contiguous()
    st = D.DenseHead(p.W_lm.to(DEV), n, B, D.SEL_TOPK | D.SEL_SAMPLE, 5, keep_logits=True)
    u = p.ud[:B].contiguous()
    st(hd, u)
    torch.cuda.synchronize()
    for b in range(B):
        r = O.dense_head(p.h_np[b:b + 1], p.W_np, k_t=5, n_rows=n)[0]
        PC.assert_close(st.logits[b].cpu().numpy(), r["logits"], p.tol, "static logits")
        PC.assert_tight(st.logits[b].cpu().numpy(), p.h_np[b], p.W_np[:n], "static logits")
        eq, ok = PC.tokens_check(_ids(st.ids)[b], r["logits"], np.arange(n), 5)
        assert ok
        zg = st.logits[b].cpu().numpy().astype(np.float64)
        eq, ok = PC.sample_check(_ids(st.sample)[b], zg, np.arange(n), p.u_np[b])
        assert ok


@pytest.mark.parametrize("V,B", [(40000, 5), (300000, 5), (65536, 64)])
@pytest.mark.parametrize("k_t", [1, 10, 16, 17, 64])
def test_dense_head_long_rows(k_t, V, B):
    """Rows longer than one selection workgroup takes (segmented selection:
    per-segment partials, then one merge and the segment-level CDF walk), with
    ties across segments (duplicate LM-head rows give equal logits); 1024-slot
    segments, and 2048-slot ones for rows beyond 262144 slots; k_t up to the
    longest top-k list."""
    rng = np.random.default_rng(3)
    d = 64
    Wl = torch.from_numpy(rng.standard_normal((V, d)).astype(np.float32) / 8).to(torch.bfloat16)
    Wl[30000:30005] = Wl[17:22]  # equal logits in different segments
    h = torch.from_numpy(rng.standard_normal((B, d)).astype(np.float32)).to(torch.bfloat16)
    u = torch.tensor([0.0, 0.25, 0.5, 0.999, 0.731] + rng.random(B - 5).tolist(), dtype=torch.float32)
    W_np, h_np = W.host_array(Wl), W.host_array(h)
    dh = D.DenseHead(Wl.to(DEV), V, B, D.SEL_TOPK | D.SEL_SAMPLE, k_t, keep_logits=True)
    dh(h.to(DEV), u.to(DEV))
    torch.cuda.synchronize()
    for b in range(B):
        zg = dh.logits[b].cpu().numpy().astype(np.float64)
        r = O.dense_head(h_np[b:b + 1], W_np, k_t=k_t)[0]
        PC.assert_close(zg, r["logits"], PC.TOL["bf16"], "dense logits")
        PC.assert_tight(zg, h_np[b], W_np, "dense logits")
        own = O.draft_select(zg, np.arange(V), k_t)
        assert _ids(dh.ids)[b].tolist() == own["ids"].tolist()  # exact on its own logits
        eq, ok = PC.sample_check(_ids(dh.sample)[b], zg, np.arange(V), float(u[b]))
        assert ok, f"row {b}: sample"


def test_determinism_and_stream_overlap():
    w = CASES[4]
    p = Problem(w)
    mode = D.SEL_TOPK | D.SEL_SAMPLE
    a = D.draft_head(p.R, p.L, p.hd, p.hd, w.k, mode=mode, k_t=w.k_t, uniforms=p.ud)
    outs = [(a.ids.clone(), a.logits.clone(), a.sample.clone())]
    side = torch.cuda.Stream()
    for route_stream in [None, side, None, side]:
        a(p.hd, p.hd, p.ud, route_stream=route_stream)
        torch.cuda.synchronize()
        outs.append((a.ids.clone(), a.logits.clone(), a.sample.clone()))
    for o in outs[1:]:
        assert torch.equal(o[0], outs[0][0]) and torch.equal(o[2], outs[0][2])
        assert torch.equal(torch.nan_to_num(o[1], nan=7.0), torch.nan_to_num(outs[0][1], nan=7.0))


def test_empty_batch_is_a_no_op():
    w = CASES[1]
    p = Problem(w)
    x = p.hd[:0]
    ids, _, _ = D.route(p.R, x, w.k)
    assert ids.shape == (0, w.k)


def test_tiny_vocab_every_k():
    # brute-force scale: V = 64, M = 8, every k, B = 3
    for k in range(1, 9):
        w = case(f"tiny_k{k}", V=64, d=32, M=8, H=16, k=k, B=3, k_t=4)
        p = Problem(w)
        head = D.draft_head(p.R, p.L, p.hd, p.hd, k, mode=D.SEL_TOPK | D.SEL_SAMPLE, k_t=4,
                            uniforms=p.ud)
        torch.cuda.synchronize()
        _check_head(p, head)


FUSED_CASES = [c for c in CASES if c.B == 1] + [
    case("fused_big", V=20000, d=1024, M=100, H=64, k=12, B=1),
    case("fused_f32", V=3000, d=128, M=24, H=16, k=5, B=1, dtype="f32"),
    # one-launch step shapes: a single linear router; d above 4096 (h loaded
    # for the gathered head, two rows per wave) with more hidden units than
    # waves (two W1 rows per wave); k = M (the shortlist is the vocabulary);
    # M at its one-launch maximum of 1024
    case("chain_linear", V=6000, d=256, M=50, H=0, act="none", k=6, B=1),
    case("chain_wide", V=9000, d=5120, M=256, H=1536, k=64, B=1),
    case("chain_k_eq_m", V=2000, d=128, M=16, H=16, k=16, B=1),
    case("chain_m1024", V=50000, d=256, M=1024, H=64, k=100, B=1),
    # the other register-block instances of the one-launch step: widest of
    # d_r, H, d in 1025..2048 (four 512-element blocks) and above 6144 (16)
    case("chain_h1536", V=7000, d=1280, M=96, H=1536, k=9, B=1),
    case("chain_d8192", V=3000, d=8192, M=48, H=128, k=5, B=1),
]


def _one_launch_opt(w, route_stream=None):
    """DYNA_OPT_FUSED_B1 value that makes a step of w run as the one launch
    (3: the one launch or an error), where w's shape allows it; else 0."""
    return 3 if w.dtype == "bf16" and route_stream is None else 0


@pytest.mark.parametrize("temperature", [1.0, 0.6])
@pytest.mark.parametrize("fused_opt", [3, 2], ids=["one_launch", "four_launches"])
@pytest.mark.parametrize("w", FUSED_CASES, ids=lambda w: w.name)
def test_fused_greedy_matches_separate_kernels(w, temperature, fused_opt):
    """A greedy one-context step folds the selection into the gathered head
    (four launches), or runs the whole step as one launch; its clusters,
    logits and token must equal the separate kernels' exactly and its
    log-probability within rounding, call after call (the arrival counters
    reset themselves).  The call with a second routing stream takes the
    four-launch form."""
    p = Problem(w)
    mode = D.SEL_ARGMAX
    fused = D.DraftHead(p.R, p.L, 1, w.k, mode, 1, temperature, keep_logits=True)
    sep = D.DraftHead(p.R, p.L, 1, w.k, mode, 1, temperature, keep_logits=True)
    side = torch.cuda.Stream()
    for it, rs in enumerate([None, None, side, None, None]):
        x = W.contexts(w, "cpu", salt=it).to(DEV)
        D.set_option(D.OPT_FUSED_B1, _one_launch_opt(w, rs) if fused_opt == 3 else fused_opt)
        try:
            fused(x, x, route_stream=rs)
            D.set_option(D.OPT_FUSED_B1, 1)
            sep(x, x, route_stream=rs)
        finally:
            D.set_option(D.OPT_FUSED_B1, 0)
        torch.cuda.synchronize()
        assert torch.equal(fused.clusters, sep.clusters)
        assert torch.equal(fused.ids, sep.ids)
        PC.assert_close(fused.logprobs.cpu().numpy(), sep.logprobs.cpu().numpy(), (2e-6, 2e-6), "lp")
        vids = O.shortlist(fused.clusters[0].cpu().numpy(), p.offsets, p.perm)[3]
        n = len(vids)
        assert torch.equal(fused.logits[:, :n], sep.logits[:, :n])
        # against the oracle on the GPU's own logits
        z = fused.logits[0, :n].cpu().numpy().astype(np.float64)
        r = O.draft_select(z, vids, 1, temperature)
        assert int(fused.ids[0, 0]) == int(r["ids"][0])
        PC.assert_close(fused.logprobs[0].cpu().numpy(), r["logprobs"], PC.LOGPROB_TOL, "lp oracle")


TOPK_FUSED_CASES = [c for c in FUSED_CASES if c.name in
                    ("ragged_b1", "fused_big", "fused_f32", "chain_wide", "chain_d8192", "chain_m1024")] + [
    # a shortlist shorter than k_t = 16: the missing places are -1 / -inf
    case("short_list", V=60, d=64, M=20, H=16, k=1, B=1),
]


@pytest.mark.parametrize("temperature", [1.0, 0.6])
@pytest.mark.parametrize("k_t", [2, 7, 16])
@pytest.mark.parametrize("fused_opt", [3, 2], ids=["one_launch", "four_launches"])
@pytest.mark.parametrize("w", TOPK_FUSED_CASES, ids=lambda w: w.name)
def test_fused_topk_matches_separate_kernels(w, fused_opt, k_t, temperature):
    """TopK_{k_t} of one context (k_t up to 16) runs as the one-launch step
    (bf16 shapes), or folds the selection into the gathered head: the ids
    must equal the separate kernels' exactly, in rank order, and the
    log-probabilities within rounding, call after call (the hand-off epoch
    and the arrival counter run on); and both against the oracle's selection
    on the GPU's own logits."""
    p = Problem(w)
    mode = D.SEL_TOPK
    fused = D.DraftHead(p.R, p.L, 1, w.k, mode, k_t, temperature, keep_logits=True)
    sep = D.DraftHead(p.R, p.L, 1, w.k, mode, k_t, temperature, keep_logits=True)
    for it in range(4):
        x = W.contexts(w, "cpu", salt=it).to(DEV)
        D.set_option(D.OPT_FUSED_B1, _one_launch_opt(w) if fused_opt == 3 else fused_opt)
        try:
            fused(x, x)
            D.set_option(D.OPT_FUSED_B1, 1)
            sep(x, x)
        finally:
            D.set_option(D.OPT_FUSED_B1, 0)
        torch.cuda.synchronize()
        assert torch.equal(fused.clusters, sep.clusters)
        vids = O.shortlist(fused.clusters[0].cpu().numpy(), p.offsets, p.perm)[3]
        n = len(vids)
        assert torch.equal(fused.logits[:, :n], sep.logits[:, :n])
        assert torch.equal(fused.ids, sep.ids)
        lf, ls = fused.logprobs.cpu().numpy(), sep.logprobs.cpu().numpy()
        assert np.array_equal(np.isfinite(lf), np.isfinite(ls))
        fin = np.isfinite(ls)
        PC.assert_close(lf[fin], ls[fin], (2e-6, 2e-6), "lp")
        z = fused.logits[0, :n].cpu().numpy().astype(np.float64)
        r = O.draft_select(z, vids, k_t, temperature)
        got = fused.ids[0].cpu().numpy()
        m = min(k_t, n)
        assert got[:m].tolist() == [int(v) for v in r["ids"][:m]]
        assert (got[m:] == -1).all() and np.isneginf(lf[0, m:]).all()
        PC.assert_close(lf[0, :m], np.asarray(r["logprobs"][:m]), PC.LOGPROB_TOL, "lp oracle")


@pytest.mark.parametrize("grid", [37, 1024, 4096])
def test_fused_topk_workgroup_counts(grid):
    """The fused top-k head with a fixed number of workgroups (few, and more
    than the last workgroup has threads, so that a thread merges several
    partial lists): ids equal to the separate kernels', log-probabilities
    within rounding."""
    w = next(c for c in FUSED_CASES if c.name == "fused_big")
    p = Problem(w)
    k_t = 16
    fused = D.DraftHead(p.R, p.L, 1, w.k, D.SEL_TOPK, k_t, keep_logits=True)
    sep = D.DraftHead(p.R, p.L, 1, w.k, D.SEL_TOPK, k_t, keep_logits=True)
    for it in range(3):
        x = W.contexts(w, "cpu", salt=it).to(DEV)
        D.set_option(D.OPT_GREEDY_GRID, grid)
        D.set_option(D.OPT_FUSED_B1, 2)
        try:
            fused(x, x)
            D.set_option(D.OPT_FUSED_B1, 1)
            sep(x, x)
        finally:
            D.set_option(D.OPT_FUSED_B1, 0)
            D.set_option(D.OPT_GREEDY_GRID, 0)
        torch.cuda.synchronize()
        assert torch.equal(fused.ids, sep.ids)
        PC.assert_close(fused.logprobs.cpu().numpy(), sep.logprobs.cpu().numpy(), (2e-6, 2e-6), "lp")


@pytest.mark.parametrize("fused_opt", [3, 2], ids=["one_launch", "four_launches"])
def test_fused_topk_ties_take_lower_ids(fused_opt):
    """A zero drafter state makes every shortlist logit 0: the one-launch and
    the fused top-k must then take the k_t lowest vocabulary ids of the
    shortlist, each with log-probability -log |V_S|, as the separate kernels
    do."""
    w = next(c for c in FUSED_CASES if c.name == "fused_big")
    p = Problem(w)
    k_t = 16
    fused = D.DraftHead(p.R, p.L, 1, w.k, D.SEL_TOPK, k_t, keep_logits=True)
    sep = D.DraftHead(p.R, p.L, 1, w.k, D.SEL_TOPK, k_t, keep_logits=True)
    x = W.contexts(w, "cpu", salt=3).to(DEV)
    h = torch.zeros_like(x)
    D.set_option(D.OPT_FUSED_B1, fused_opt)
    try:
        fused(x, h)
        D.set_option(D.OPT_FUSED_B1, 1)
        sep(x, h)
    finally:
        D.set_option(D.OPT_FUSED_B1, 0)
    torch.cuda.synchronize()
    vids = O.shortlist(fused.clusters[0].cpu().numpy(), p.offsets, p.perm)[3]
    assert fused.ids[0].cpu().tolist() == sorted(int(v) for v in vids)[:k_t]
    assert torch.equal(fused.ids, sep.ids)
    np.testing.assert_allclose(fused.logprobs[0].cpu().numpy(), -np.log(len(vids)), rtol=0, atol=2e-6)


@pytest.mark.parametrize("variant", ["tied_rows", "zero_router"])
def test_one_launch_step_ties(variant):
    """Router scores with exact ties across the k-th place (layer-2 rows 3..M-1
    all equal, so 61 clusters tie and k = 7 always cuts into them), or all
    equal (a zero router): the one-launch step's selection must break them
    toward the lower cluster id exactly as the separate kernels do."""
    w = case("ties_b1", V=4000, d=256, M=64, H=32, k=7, B=1)
    p = Problem(w)
    W2 = p.W2.clone()
    if variant == "tied_rows":
        W2[3:] = W2[3]
    else:
        W2.zero_()
    R = D.Router(p.W1.to(DEV), W2.to(DEV), act=w.act)
    mode = D.SEL_ARGMAX
    one = D.DraftHead(R, p.L, 1, w.k, mode, 1, keep_logits=True)
    sep = D.DraftHead(R, p.L, 1, w.k, mode, 1, keep_logits=True)
    for it in range(4):
        x = W.contexts(w, "cpu", salt=it).to(DEV)
        D.set_option(D.OPT_FUSED_B1, 3)
        try:
            one(x, x)
            D.set_option(D.OPT_FUSED_B1, 1)
            sep(x, x)
        finally:
            D.set_option(D.OPT_FUSED_B1, 0)
        torch.cuda.synchronize()
        assert torch.equal(one.clusters, sep.clusters)
        assert torch.equal(one.ids, sep.ids)
        vids = O.shortlist(one.clusters[0].cpu().numpy(), p.offsets, p.perm)[3]
        assert torch.equal(one.logits[:, :len(vids)], sep.logits[:, :len(vids)])
        got = one.clusters[0].cpu().tolist()
        if variant == "zero_router":
            # every score is 0: the k lowest cluster ids, in id order
            assert got == list(range(w.k))
        else:
            # the tied clusters taken are the lowest ids of the tied run
            tied = sorted(c for c in got if c >= 3)
            assert tied == list(range(3, 3 + len(tied)))


@pytest.mark.parametrize("k_t", [1, 10])
def test_one_launch_step_wait_bound(k_t):
    """Every wait of the one-launch step (argmax and top-k_t) is bounded.
    With the bound forced from the host to nothing (a wait gives up at its
    first read that finds a word missing), a step must report the failure
    (ids -1, log-probabilities -inf) and never a token from half-written
    data; once the bound is back, the very next step is exact again (the
    error word carries the epoch of the launch that set it, so a late give-up
    cannot fail a later step)."""
    w = next(c for c in FUSED_CASES if c.name == "chain_wide")
    p = Problem(w)
    mode = D.SEL_ARGMAX if k_t == 1 else D.SEL_TOPK
    one = D.DraftHead(p.R, p.L, 1, w.k, mode, k_t, keep_logits=True)
    sep = D.DraftHead(p.R, p.L, 1, w.k, mode, k_t, keep_logits=True)

    def step(it, bound):
        x = W.contexts(w, "cpu", salt=it).to(DEV)
        D.set_option(D.OPT_WAIT_BOUND_US, bound)
        D.set_option(D.OPT_FUSED_B1, 3)
        try:
            one(x, x)
            D.set_option(D.OPT_FUSED_B1, 1)
            sep(x, x)
        finally:
            D.set_option(D.OPT_FUSED_B1, 0)
            D.set_option(D.OPT_WAIT_BOUND_US, 0)
        torch.cuda.synchronize()
        got, want = one.ids[0].cpu(), sep.ids[0].cpu()
        if int(got[0]) == -1:
            assert (got == -1).all() and torch.isneginf(one.logprobs[0].cpu()).all()
            return False
        assert torch.equal(got, want) and torch.equal(one.clusters, sep.clusters)
        return True

    with pytest.raises(D.DynaError):
        D.set_option(D.OPT_WAIT_BOUND_US, -2)
    assert step(0, 0)
    forced = [step(1 + i, -1) for i in range(3)]
    assert not all(forced)  # at least one forced step found a word missing
    # the error word carries the failed launch's epoch: the very next step,
    # with its wait bound restored, is exact
    assert step(4, 0) and step(5, 0) and step(6, 0)


@pytest.mark.parametrize("grid_per_cu", [2, 3])
@pytest.mark.parametrize("k_t", [1, 10])
def test_one_launch_step_grid_beyond_residency(grid_per_cu, k_t):
    """A grid request above what can be resident at once is capped by the
    occupancy check (or the step takes the four-launch form): the results stay
    exact against the separate kernels.  With more workgroups than threads in
    workgroup 0, the top-k_t merge takes several partials per thread."""
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    mode = D.SEL_ARGMAX if k_t == 1 else D.SEL_TOPK
    for name in ["chain_wide", "chain_d8192", "ragged_b1"]:
        w = next(c for c in FUSED_CASES if c.name == name)
        p = Problem(w)
        one = D.DraftHead(p.R, p.L, 1, w.k, mode, k_t, keep_logits=True)
        sep = D.DraftHead(p.R, p.L, 1, w.k, mode, k_t, keep_logits=True)
        for it in range(3):
            x = W.contexts(w, "cpu", salt=it).to(DEV)
            D.set_option(D.OPT_GREEDY_GRID, min(4096, grid_per_cu * n_cu))
            D.set_option(D.OPT_FUSED_B1, 3)
            try:
                one(x, x)
                D.set_option(D.OPT_FUSED_B1, 1)
                sep(x, x)
            finally:
                D.set_option(D.OPT_FUSED_B1, 0)
                D.set_option(D.OPT_GREEDY_GRID, 0)
            torch.cuda.synchronize()
            assert torch.equal(one.clusters, sep.clusters) and torch.equal(one.ids, sep.ids), name
            n = len(O.shortlist(one.clusters[0].cpu().numpy(), p.offsets, p.perm)[3])
            assert torch.equal(one.logits[:, :n], sep.logits[:, :n])
            PC.assert_close(one.logprobs.cpu().numpy(), sep.logprobs.cpu().numpy(), (2e-6, 2e-6), "lp")


@pytest.mark.parametrize("variant", ["nan", "pos_inf", "neg_inf", "mixed_inf", "all_equal"])
def test_one_launch_step_special_inputs(variant):
    """NaN, +-inf and all-equal router features on the one-launch step.  The
    router's scores then hold NaN (ranked as -inf) or infinities, or many
    exact ties: the step's clusters must be the canonical top-k of the
    separate router's own fp32 scores (and the oracle's, where the oracle's
    fp64 scores are finite), and its token and logits must equal the
    separate kernels' exactly; h stays finite."""
    w = case("special_b1", V=4000, d=256, M=64, H=32, k=7, B=1)
    p = Problem(w)
    x = p.hd.clone()
    if variant == "nan":
        x[0, ::3] = float("nan")
    elif variant == "pos_inf":
        x[0, 5] = float("inf")
    elif variant == "neg_inf":
        x[0, 9] = float("-inf")
    elif variant == "mixed_inf":
        x[0, 5] = float("inf")
        x[0, 77] = float("-inf")
    else:
        x[0, :] = 0.5
    h = p.hd
    one = D.DraftHead(p.R, p.L, 1, w.k, D.SEL_ARGMAX, 1, keep_logits=True)
    sep = D.DraftHead(p.R, p.L, 1, w.k, D.SEL_ARGMAX, 1, keep_logits=True)
    for _ in range(3):
        D.set_option(D.OPT_FUSED_B1, 3)
        try:
            one(x, h)
            D.set_option(D.OPT_FUSED_B1, 1)
            sep(x, h)
        finally:
            D.set_option(D.OPT_FUSED_B1, 0)
        torch.cuda.synchronize()
        assert torch.equal(one.clusters, sep.clusters)
        assert torch.equal(one.ids, sep.ids)
        n = len(O.shortlist(one.clusters[0].cpu().numpy(), p.offsets, p.perm)[3])
        assert torch.equal(one.logits[:, :n], sep.logits[:, :n])
    ids, _, scores = D.route(p.R, x, w.k, want_scores=True)
    torch.cuda.synchronize()
    g_scores = scores.cpu().numpy().astype(np.float64)
    own, _ = O.topk_clusters(g_scores, w.k)
    assert _ids(one.clusters).tolist() == own.tolist()
    if variant == "all_equal":
        ref = O.router_scores(W.host_array(x.cpu()), p.W1_np, p.W2_np, act=w.act)
        eq, ok = PC.cluster_check(_ids(one.clusters)[0], ref[0], w.k)
        assert ok
    # the token is the oracle's argmax over the GPU's shortlist and h
    vids = O.shortlist(_ids(one.clusters)[0], p.offsets, p.perm)[3]
    z_ref = O.shortlist_logits(p.h_np[0], p.W_np, vids)
    PC.assert_tight(one.logits[0, :len(vids)].cpu().numpy(), p.h_np[0], p.W_np[vids], "special logits")
    eq, ok = PC.tokens_check(_ids(one.ids)[0], z_ref, vids, 1)
    assert ok


def _special_partition(V, M, empty, single, seed):
    """cluster_of with the clusters in `empty` holding no token and those in
    `single` exactly one; the rest share the vocabulary at random."""
    rng = np.random.default_rng(seed)
    rest = np.array([m for m in range(M) if m not in empty and m not in single])
    cl = rest[rng.integers(0, len(rest), size=V)].astype(np.int32)
    for i, m in enumerate(single):
        cl[7 + 13 * i] = m
    return cl


EMPTY_CASES = [
    # (name, B, k, select mode, logits path option, union)
    ("one_launch_b1", 1, "argmax", 0, False),
    ("four_launch_b1", 1, "argmax", 0, False),
    ("gemv_b3", 3, "topk_sample", 0, False),
    ("gather_b9", 9, "topk_sample", 0, False),
    ("gemv_b9", 9, "topk_sample", 1, False),
    ("union_b9", 9, "topk_sample", 0, True),
]


@pytest.mark.parametrize("k", [3, 6, 8])
@pytest.mark.parametrize("name,B,sel,path,union", EMPTY_CASES, ids=[c[0] for c in EMPTY_CASES])
def test_empty_and_single_row_clusters(name, B, sel, path, union, k):
    """Clusters of no rows and of one row (the partition enforces no balance,
    Sec. 4.2).  A second-layer bias puts the three empty clusters first and the
    three one-row clusters next, so k = 3 selects only empty clusters (an
    empty shortlist: no token, no sample), k = 6 adds the one-row clusters (a
    shortlist of 3 tokens) and k = 8 two ordinary clusters as well."""
    V, d, M, H = 3000, 200, 40, 24
    empty, single = [3, 17, 29], [5, 11, 38]
    w = case(f"special_{name}", V=V, d=d, M=M, H=H, k=k, B=B)
    p = Problem(w)
    p.cluster_of = _special_partition(V, M, empty, single, 9)
    p.L = D.build_layout(torch.from_numpy(p.cluster_of).to(DEV), p.W_lm.to(DEV), M)
    p.sizes, p.offsets, p.perm, p.cap = O.cluster_layout(p.cluster_of, M)
    b2 = np.zeros(M, dtype=np.float32)
    b2[empty] = 60.0
    b2[single] = 50.0
    p.R = D.Router(p.W1.to(DEV), p.W2.to(DEV), b2=torch.from_numpy(b2).to(DEV), act=w.act)
    ref_scores = O.router_scores(p.h_np, p.W1_np, p.W2_np, b2=b2.astype(np.float64), act=w.act)
    mode = (D.SEL_ARGMAX if sel == "argmax" else D.SEL_TOPK | D.SEL_SAMPLE) | (D.SEL_UNION if union else 0)
    kt = 1 if sel == "argmax" else 4
    D.set_option(D.OPT_LOGITS_PATH, path)
    D.set_option(D.OPT_FUSED_B1, 2 if name.startswith("four_launch") else 3 if name.startswith("one_launch") else 0)
    try:
        head = D.draft_head(p.R, p.L, p.hd, p.hd, k, mode=mode, k_t=kt, uniforms=p.ud)
        torch.cuda.synchronize()
    finally:
        D.set_option(D.OPT_LOGITS_PATH, 0)
        D.set_option(D.OPT_FUSED_B1, 0)
    clusters = _ids(head.clusters)
    for b in range(B):
        assert sorted(clusters[b, :min(k, 6)].tolist()) == sorted((empty + single)[:min(k, 6)])
    if union:
        sel_ids = O.union_clusters(clusters)
    logits = head.logits.cpu().numpy().astype(np.float64)
    ids = _ids(head.ids)
    for b in range(B):
        eq, ok = PC.cluster_check(clusters[b], ref_scores[b], k)
        assert ok, f"row {b}: clusters"
        vids = O.shortlist(sel_ids if union else clusters[b], p.offsets, p.perm)[3]
        n = len(vids)
        assert n == {3: 0, 6: 3}.get(k, n), f"row {b}: shortlist of {n} rows"
        z_ref = O.shortlist_logits(p.h_np[b], p.W_np, vids)
        PC.assert_close(logits[b, :n], z_ref, p.tol, f"row {b} logits")
        PC.assert_tight(logits[b, :n], p.h_np[b], p.W_np[vids], f"row {b} logits")
        r = O.draft_select(logits[b, :n], vids, min(kt, n), 1.0, p.u_np[b])
        assert ids[b, :min(kt, n)].tolist() == r["ids"].tolist(), f"row {b}: ids"
        assert np.all(ids[b, min(kt, n):] == -1), f"row {b}: ids past the shortlist"
        if n == 0:
            assert np.all(np.isneginf(head.logprobs[b].cpu().numpy()))
        if head.sample is not None:
            smp = int(_ids(head.sample)[b])
            eq, ok = PC.sample_check(smp, logits[b, :n], vids, p.u_np[b])
            assert ok, f"row {b}: sample {smp}"


def test_determinism_over_many_steps():
    """The same inputs give bit-identical outputs call after call (no
    floating-point atomics, fixed-order sums): 100 one-launch steps, 100
    four-launch steps and 100 batched steps."""
    chain = next(c for c in FUSED_CASES if c.name == "chain_wide")
    pc = Problem(chain)
    for fused_opt in (3, 2):
        head = D.DraftHead(pc.R, pc.L, 1, chain.k, D.SEL_ARGMAX, 1, keep_logits=True)
        D.set_option(D.OPT_FUSED_B1, fused_opt)
        try:
            head(pc.hd, pc.hd)
            torch.cuda.synchronize()
            ref = (head.ids.clone(), head.logprobs.clone(), head.logits.clone(), head.clusters.clone())
            for _ in range(100):
                head(pc.hd, pc.hd)
            torch.cuda.synchronize()
        finally:
            D.set_option(D.OPT_FUSED_B1, 0)
        got = (head.ids, head.logprobs, head.logits, head.clusters)
        for a, b in zip(ref, got):
            assert torch.equal(torch.nan_to_num(a, nan=7.0), torch.nan_to_num(b, nan=7.0))
    w = CASES[4]
    p = Problem(w)
    mode = D.SEL_TOPK | D.SEL_SAMPLE
    head = D.DraftHead(p.R, p.L, w.B, w.k, mode, w.k_t, keep_logits=True)
    head(p.hd, p.hd, p.ud)
    torch.cuda.synchronize()
    ref = (head.ids.clone(), head.logprobs.clone(), head.sample.clone(), head.logits.clone())
    outs = []
    for i in range(100):
        head(p.hd, p.hd, p.ud)
        if i % 10 == 9:
            torch.cuda.synchronize()
            outs.append((head.ids.clone(), head.logprobs.clone(), head.sample.clone(), head.logits.clone()))
    for o in outs:
        for a, b in zip(ref, o):
            assert torch.equal(torch.nan_to_num(a, nan=7.0), torch.nan_to_num(b, nan=7.0))
