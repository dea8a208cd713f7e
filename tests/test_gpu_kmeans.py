"""GPU parity of the partition builder (spherical k-means on the unit LM-head
rows, Sec. 4.2 "Vocabulary partition") against the CPU oracle.

The oracle computes the cosine similarities exactly (float64, unrounded
centroids).  The kernel multiplies on the matrix cores with the centroids
rounded to bf16 (relative error at most 2^-8 per coordinate) and sums in
fp32.  Its similarity to centroid m therefore errs by at most
e_m = (2^-8 + (d / 4 + 64) 2^-24) * sum_i |x_i mu_m,i|, so the GPU may pick
centroid g over the oracle's r only when S[r] - S[g] <= e_r + e_g.  The rows
where the two differ are counted and bounded.  Centroids are fp32 sums of
unit rows; they match the oracle's float64 sums within 2e-5.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import dynaspec_oracle as O

pytestmark = pytest.mark.gpu
DEV = "cuda"
D = None


@pytest.fixture(scope="module", autouse=True)
def _lib():
    global D
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2510_13847_amd import dynahead
    D = dynahead
    D.lib()
    yield
    D.set_option(D.OPT_KMEANS_CFG, 0)


def _rand_head(V, d, seed):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(V, d, generator=g) / d ** 0.5).to(torch.bfloat16)


def _unit(rng, M, d):
    c = rng.standard_normal((M, d))
    return (c / np.linalg.norm(c, axis=1, keepdims=True)).astype(np.float32)


def _check_assign(got, Wh, C, S, what, limit=None):
    """got[v] equals the oracle's argmax, or the oracle's two similarities lie
    within the bf16-rounding window e_r + e_g of each other.  Returns the
    number of rows that differ (asserted below `limit`, default 1% of V + 1)."""
    ref = np.argmax(S, axis=1)
    bad = np.nonzero(got != ref)[0]
    if len(bad):
        X = O.unit_rows(Wh[bad])
        d = X.shape[1]
        eps = 2.0 ** -8 + (d / 4.0 + 64.0) * 2.0 ** -24
        Ca = np.abs(np.asarray(C, dtype=np.float64))
        for i, v in enumerate(bad):
            g, r = int(got[v]), int(ref[v])
            assert 0 <= g < S.shape[1], f"{what}: row {v} -> {g} out of range"
            win = eps * (np.abs(X[i]) @ Ca[r] + np.abs(X[i]) @ Ca[g])
            assert S[v, r] - S[v, g] <= win, (f"{what}: row {v} -> {g}, oracle {r}, gap {S[v, r] - S[v, g]:.3e} "
                                              f"above the bf16 window {win:.3e}")
    limit = max(1, S.shape[0] // 100) if limit is None else limit
    assert len(bad) <= limit, f"{what}: {len(bad)} rows differ from the oracle's assignment (limit {limit})"
    return len(bad)


SHAPES = [  # V (ragged vs 16-row tiles), d (ragged vs k blocks), M (one group, several groups)
    (1000, 64, 7), (3001, 200, 37), (2500, 520, 130), (4099, 128, 300), (2048, 1024, 513),
]


@pytest.mark.parametrize("cfg", list(range(8)))
@pytest.mark.parametrize("V,d,M", SHAPES)
def test_assign_step(V, d, M, cfg):
    rng = np.random.default_rng(V + M)
    Wl = _rand_head(V, d, V)
    C = _unit(rng, M, d)
    D.set_option(D.OPT_KMEANS_CFG, cfg)
    try:
        a, sc = D.kmeans_assign(Wl.to(DEV), torch.from_numpy(C).to(DEV), want_score=True)
        torch.cuda.synchronize()
    finally:
        D.set_option(D.OPT_KMEANS_CFG, 0)
    got = a.cpu().numpy().astype(np.int64)
    Wh = W.host_array(Wl)
    ref, S = O.kmeans_assign(Wh, C)
    n_diff = _check_assign(got, Wh, C, S, "assign")
    print(f"[kmeans] V={V} d={d} M={M} cfg={cfg}: {n_diff} assignments differ from the exact oracle", flush=True)
    # the reported product is the raw row's with the bf16-rounded centroid:
    # within the same window of the exact W[v] . mu_m
    Wf = O.as_f64(Wh)
    want = (Wf * C.astype(np.float64)[got]).sum(axis=1)
    mag = (np.abs(Wf) * np.abs(C.astype(np.float64)[got])).sum(axis=1)
    win = (2.0 ** -8 + (d / 4.0 + 64.0) * 2.0 ** -24) * mag
    err = np.abs(sc.cpu().numpy().astype(np.float64) - want)
    assert np.all(err <= win), f"scores: {int((err > win).sum())} outside the bf16 window"


def test_assign_ties_and_zero_rows():
    # duplicate centroids tie exactly: the lower id wins; a zero row scores 0
    # against every centroid and goes to cluster 0
    rng = np.random.default_rng(1)
    V, d, M = 300, 64, 6
    Wl = _rand_head(V, d, 9)
    Wl[17] = 0
    C = _unit(rng, M, d)
    C[4] = C[1]
    a, _ = D.kmeans_assign(Wl.to(DEV), torch.from_numpy(C).to(DEV))
    got = a.cpu().numpy()
    assert got[17] == 0
    assert not np.any(got == 4)
    Wh = W.host_array(Wl)
    ref, S = O.kmeans_assign(Wh, C)
    _check_assign(got.astype(np.int64), Wh, C, S, "ties")


@pytest.mark.parametrize("V,d,M", [(1000, 64, 7), (3001, 200, 37), (2048, 1024, 513), (2000, 8192, 5)])
def test_update_step(V, d, M):
    rng = np.random.default_rng(V * 7 + d)
    Wl = _rand_head(V, d, V + 1)
    assign = rng.integers(0, max(1, M - 2), size=V).astype(np.int32)  # the last clusters stay empty
    C = _unit(rng, M, d)
    mu = torch.from_numpy(C.copy()).to(DEV)
    D.kmeans_update(Wl.to(DEV), torch.from_numpy(assign).to(DEV), mu)
    torch.cuda.synchronize()
    ref = O.kmeans_update(W.host_array(Wl), assign, M, C.astype(np.float64))
    got = mu.cpu().numpy().astype(np.float64)
    np.testing.assert_allclose(got, ref, rtol=0, atol=2e-5)
    np.testing.assert_array_equal(got[M - 2:], C[M - 2:])  # empty clusters: bit-for-bit unchanged


def test_update_skips_out_of_range_ids():
    rng = np.random.default_rng(4)
    V, d, M = 500, 64, 5
    Wl = _rand_head(V, d, 3)
    assign = rng.integers(0, M, size=V).astype(np.int32)
    assign[::7] = M + 3
    assign[1::11] = -1
    C = _unit(rng, M, d)
    mu = torch.from_numpy(C.copy()).to(DEV)
    D.kmeans_update(Wl.to(DEV), torch.from_numpy(assign).to(DEV), mu)
    torch.cuda.synchronize()
    keep = (assign >= 0) & (assign < M)
    ref = O.kmeans_update(W.host_array(Wl)[keep], assign[keep], M, C.astype(np.float64))
    np.testing.assert_allclose(mu.cpu().numpy(), ref, rtol=0, atol=2e-5)


def test_planted_partition_is_recovered():
    V, d, M = 4000, 128, 24
    Wl, groups = W.planted_head(V, d, M, seed=5, noise=0.2)
    init = np.array([np.nonzero(groups == m)[0][0] for m in range(M)], dtype=np.int32)
    cl, mu = D.kmeans(Wl.to(DEV), M, torch.from_numpy(init).to(DEV), iters=4)
    torch.cuda.synchronize()
    got = cl.cpu().numpy().astype(np.int64)
    np.testing.assert_array_equal(got, groups)
    ref_a, ref_mu = O.spherical_kmeans(W.host_array(Wl), M, init, iters=4)
    np.testing.assert_array_equal(got, ref_a)
    np.testing.assert_allclose(mu.cpu().numpy(), ref_mu, rtol=0, atol=2e-5)
    # the partition feeds the layout directly
    L = D.build_layout(cl, Wl.to(DEV), M)
    assert L.cap_by_k[M] == V


@pytest.mark.parametrize("iters", [1, 4])
def test_random_head_rounds(iters):
    """No planted structure.  Every GPU round is checked against the oracle's
    round taken from the GPU's own previous centroids (so rounding in an early
    round cannot cascade): the assignment within the bf16 window, the update
    within 2e-5.  The whole builder (dyna_kmeans) must equal the chained
    steps exactly."""
    w = W.scaled(W.WORKLOADS["llama3_8b_chain"], V=5000, d=256, M=40)
    Wl = W.lm_head(w)
    Wd = Wl.to(DEV)
    init = W.kmeans_init_ids(w)
    Wh = W.host_array(Wl)
    X = O.unit_rows(Wh)
    ws = D.kmeans_workspace(Wd, w.M)
    # round 1 starts from the unit points at init (the GPU normalises them in fp32)
    cl, mu = D.kmeans(Wd, w.M, torch.from_numpy(init).to(DEV), iters=1, ws=ws)
    torch.cuda.synchronize()
    prev = X[init]
    got = cl.cpu().numpy().astype(np.int64)
    _, S = O.kmeans_assign(Wh, prev)
    diffs = [_check_assign(got, Wh, prev, S, "round 1")]
    ref_mu = O.kmeans_update(Wh, got, w.M, prev)
    np.testing.assert_allclose(mu.cpu().numpy(), ref_mu, rtol=0, atol=2e-5)
    for it in range(1, iters):
        prev = mu.cpu().numpy().astype(np.float64)   # the GPU's own centroids
        a, _ = D.kmeans_assign(Wd, mu, ws=ws)
        torch.cuda.synchronize()
        got = a.cpu().numpy().astype(np.int64)
        _, S = O.kmeans_assign(Wh, prev)
        diffs.append(_check_assign(got, Wh, prev, S, f"round {it + 1}"))
        D.kmeans_update(Wd, a, mu, ws=ws)
        torch.cuda.synchronize()
        ref_mu = O.kmeans_update(Wh, got, w.M, prev)
        np.testing.assert_allclose(mu.cpu().numpy(), ref_mu, rtol=0, atol=2e-5)
    print(f"[kmeans] rounds {iters}: assignments differing from the exact oracle per round {diffs}", flush=True)
    # the builder in one call is the chained steps
    cl_all, mu_all = D.kmeans(Wd, w.M, torch.from_numpy(init).to(DEV), iters=iters, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(cl_all, torch.from_numpy(got.astype(np.int32)).to(DEV))
    assert torch.equal(mu_all, mu)


def test_deterministic_and_errors():
    w = W.scaled(W.WORKLOADS["llama3_8b_chain"], V=3000, d=128, M=30)
    Wl = W.lm_head(w).to(DEV)
    init = torch.from_numpy(W.kmeans_init_ids(w)).to(DEV)
    a1, m1 = D.kmeans(Wl, w.M, init, iters=2)
    a2, m2 = D.kmeans(Wl, w.M, init, iters=2)
    torch.cuda.synchronize()
    assert torch.equal(a1, a2) and torch.equal(m1, m2)
    bad = init.clone()
    bad[3] = w.V
    with pytest.raises(D.DynaError) as e:
        D.kmeans(Wl, w.M, bad, iters=1)
    assert e.value.status == D.ERR_DEVICE_DATA
    with pytest.raises(D.DynaError) as e:
        D.kmeans(Wl.float(), w.M, init, iters=1)
    assert e.value.status == D.ERR_UNSUPPORTED
