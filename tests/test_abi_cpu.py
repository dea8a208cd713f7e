"""Host-side checks of the C ABI: no GPU needed (no call reaches a HIP API)."""
import ctypes
import os
import re

import pytest

from paper_2510_13847_amd import dynahead as D

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dynahead.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dyna_[a-z_]+)\s*\(", text)))


def test_library_loads_and_exports_every_declared_symbol():
    lib = D.lib()
    declared = header_functions()
    assert len(declared) >= 14
    for name in declared:
        assert hasattr(lib, name), f"{name} declared in dynahead.h but not exported"
    assert set(declared) == set(D.EXPORTED), "binding and header disagree"
    assert lib.dyna_abi_version() == D.ABI_VERSION == 2


def test_header_constants_match_the_binding():
    """Every DYNA_OPT_*, DYNA_SEL_* and DYNA_ERR_* value the header defines is
    the value the Python binding passes."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    found = dict((n, int(v, 0)) for n, v in re.findall(r"\bDYNA_((?:OPT|SEL|ERR)_[A-Z0-9_]+)\s*=\s*(-?(?:0x[0-9a-fA-F]+|\d+))", text))
    assert any(n.startswith("OPT_") for n in found)
    for name, value in found.items():
        assert getattr(D, name, None) == value, f"DYNA_{name} = {value} in the header"


def test_status_strings():
    lib = D.lib()
    for code, name in enumerate(["DYNA_OK", "DYNA_ERR_INVALID_ARG", "DYNA_ERR_CAPACITY",
                                 "DYNA_ERR_WORKSPACE", "DYNA_ERR_UNSUPPORTED", "DYNA_ERR_HIP",
                                 "DYNA_ERR_DEVICE_DATA"]):
        assert lib.dyna_status_string(code).decode() == name


def test_set_option_validation():
    lib = D.lib()
    assert lib.dyna_set_option(99, 0) == D.ERR_INVALID_ARG
    assert b"unknown option" in lib.dyna_last_error()
    assert lib.dyna_set_option(D.OPT_LOGITS_PATH, 7) == D.ERR_INVALID_ARG
    assert lib.dyna_set_option(D.OPT_LOGITS_PATH, 0) == D.OK
    assert lib.dyna_set_option(D.OPT_GATHER_CFG, 10) == D.ERR_INVALID_ARG
    assert lib.dyna_set_option(D.OPT_LOGITS_PATH, 3) == D.ERR_INVALID_ARG
    assert lib.dyna_set_option(D.OPT_GATHER_CFG, 0) == D.OK
    assert lib.dyna_set_option(D.OPT_UNION_CFG, 16) == D.ERR_INVALID_ARG
    assert lib.dyna_set_option(D.OPT_UNION_CFG, 0) == D.OK
    assert lib.dyna_set_option(D.OPT_KMEANS_CFG, 8) == D.ERR_INVALID_ARG
    assert lib.dyna_set_option(D.OPT_KMEANS_CFG, 0) == D.OK
    for v in (-2, 1000001):
        assert lib.dyna_set_option(D.OPT_WAIT_BOUND_US, v) == D.ERR_INVALID_ARG
    for v in (-1, 1, 1000000, 0):
        assert lib.dyna_set_option(D.OPT_WAIT_BOUND_US, v) == D.OK
    assert lib.dyna_set_option(12, 0) == D.ERR_INVALID_ARG  # no such option
    assert lib.dyna_set_option(D.OPT_FUSED_B1, 4) == D.ERR_INVALID_ARG
    for v in (3, 2, 1, 0):
        assert lib.dyna_set_option(D.OPT_FUSED_B1, v) == D.OK


def _layout(V=1000, d=64, M=10, cap=None, W=0x1000):
    cap_arr = (ctypes.c_int32 * (M + 1))(*([0] + [100 * (i + 1) for i in range(M)]))
    L = D._Layout(V, d, M, D.BF16, W, 0x2000, 0x3000, ctypes.addressof(cap_arr), 100)
    return L, cap_arr


def test_workspace_sizes_are_host_only():
    lib = D.lib()
    L, keep = _layout()
    n1 = lib.dyna_workspace_bytes(ctypes.byref(L), None, 4, 3, 300)
    n2 = lib.dyna_workspace_bytes(ctypes.byref(L), None, 8, 3, 300)
    assert 0 < n1 < n2
    assert lib.dyna_workspace_bytes(None, None, 4, 3, 300) == 0
    assert lib.dyna_dense_workspace_bytes(0, 4) == 0
    assert lib.dyna_dense_workspace_bytes(128256, 1) > 128256 * 4
    assert lib.dyna_layout_workspace_bytes(128256, 1024) >= 128256 * 4


def test_noalloc_scratch_covers_the_stated_shapes():
    """The allocation-free entry point's scratch (DYNA_NOALLOC_SCRATCH_BYTES
    less the 384 KiB hand-off region) holds the workspace of one context and
    of the tree-batch and serving steps, as the header states, and not the
    large-vocabulary and union batches (host-only sizing)."""
    import workloads as W
    from oracle import dynaspec_oracle as O
    lib = D.lib()
    limit = D.NOALLOC_SCRATCH_BYTES - 384 * 1024
    expect = {"llama3_8b_chain": True, "llama3_8b_tree": True, "qwen25_serving": True,
              "gemma3_large_vocab": False, "llama3_8b_tree_union": False}
    for name, fits in expect.items():
        w = W.WORKLOADS[name]
        sizes, _, _, cap = O.cluster_layout(W.partition(w), w.M)
        cap_arr = (ctypes.c_int32 * (w.M + 1))(*[int(c) for c in cap])
        L = D._Layout(w.V, w.d, w.M, D.BF16, 0x1000, 0x2000, 0x3000, ctypes.addressof(cap_arr), int(sizes.max()))
        R = D._Router(w.d, w.H, w.M, D.BF16, 2, 0x1000, 0, 0x1000 if w.H else 0, 0)
        c = min(w.V, w.B * int(cap[w.k])) if w.union else int(cap[w.k])
        need = lib.dyna_workspace_bytes(ctypes.byref(L), ctypes.byref(R), w.B, w.k, c)
        assert (0 < need <= limit) == fits, (name, need, limit)


def test_shortlist_logits_argument_errors():
    lib = D.lib()
    L, keep = _layout()
    s = lib.dyna_shortlist_logits
    P = 0x10000
    # k out of range
    assert s(ctypes.byref(L), P, D.BF16, 2, 0, P, P, P, P, 300, P, 1 << 30, None) == D.ERR_INVALID_ARG
    assert s(ctypes.byref(L), P, D.BF16, 2, 11, P, P, P, P, 300, P, 1 << 30, None) == D.ERR_INVALID_ARG
    # cap below cap_by_k[k]
    assert s(ctypes.byref(L), P, D.BF16, 2, 3, P, P, P, P, 299, P, 1 << 30, None) == D.ERR_CAPACITY
    assert b"cap=299" in lib.dyna_last_error()
    # workspace too small
    assert s(ctypes.byref(L), P, D.BF16, 2, 3, P, P, P, P, 300, P, 16, None) == D.ERR_WORKSPACE
    # misaligned h
    assert s(ctypes.byref(L), P + 2, D.BF16, 2, 3, P, P, P, P, 300, P, 1 << 30, None) == D.ERR_INVALID_ARG
    # bad dtype
    assert s(ctypes.byref(L), P, 7, 2, 3, P, P, P, P, 300, P, 1 << 30, None) == D.ERR_INVALID_ARG
    # B = 0 is a no-op even with NULL buffers
    assert s(ctypes.byref(L), None, D.BF16, 0, 3, None, None, None, None, 300, None, 0, None) == D.OK


def test_layout_struct_checks():
    lib = D.lib()
    P = 0x10000
    for field, value in [("d", 12), ("M", 0), ("M", 2000), ("wdtype", 3), ("max_cluster", 0)]:
        L, keep = _layout()
        setattr(L, field, value)
        assert lib.dyna_shortlist(ctypes.byref(L), P, 1, 1, P, P, P, None, 0, None) != D.OK
    L, keep = _layout(M=9000, V=100000)
    assert lib.dyna_shortlist(ctypes.byref(L), P, 1, 1, P, P, P, None, 0, None) == D.ERR_UNSUPPORTED


def test_select_and_head_argument_errors():
    lib = D.lib()
    L, keep = _layout()
    P = 0x10000
    sel = lib.dyna_draft_select
    # bad mode, k_t out of range, sampling without uniforms, bad temperature
    base = dict(mode=D.SEL_TOPK, k_t=4, temp=1.0, u=P)
    def call(mode, k_t, temp, u, beta=0.0):
        return sel(ctypes.byref(L), P, P, P, P, 2, 3, 300, mode, k_t, temp, beta, u, P, P, P, P, P, 1 << 30, None)
    assert call(0, 4, 1.0, P) == D.ERR_INVALID_ARG
    assert call(8, 4, 1.0, P) == D.ERR_INVALID_ARG
    assert call(D.SEL_TOPK, 0, 1.0, P) == D.ERR_INVALID_ARG
    assert call(D.SEL_TOPK, 65, 1.0, P) == D.ERR_INVALID_ARG
    assert call(D.SEL_SAMPLE, 1, 1.0, None) == D.ERR_INVALID_ARG
    assert call(D.SEL_SAMPLE, 1, 0.0, P) == D.ERR_INVALID_ARG
    assert call(D.SEL_SAMPLE, 1, float("inf"), P) == D.ERR_INVALID_ARG
    assert call(D.SEL_SAMPLE, 1, 1.0, P, beta=1.0) == D.ERR_INVALID_ARG   # tail weight in [0, 1)
    assert call(D.SEL_SAMPLE, 1, 1.0, P, beta=-0.1) == D.ERR_INVALID_ARG
    # router/layout mismatch in the fused call
    R = D._Router(64, 0, 11, D.BF16, 0, P, None, None, None)
    head = lib.dyna_draft_head
    st = head(ctypes.byref(R), ctypes.byref(L), P, P, D.BF16, 2, 3, D.SEL_ARGMAX, 1, 1.0, 0.0, None,
              P, P, None, None, None, None, 300, P, 1 << 30, None, None, None)
    assert st == D.ERR_INVALID_ARG and b"differs" in lib.dyna_last_error()
    R = D._Router(64, 12, 10, D.BF16, 2, P, None, P, None)  # H not a multiple of 8
    st = head(ctypes.byref(R), ctypes.byref(L), P, P, D.BF16, 2, 3, D.SEL_ARGMAX, 1, 1.0, 0.0, None,
              P, P, None, None, None, None, 300, P, 1 << 30, None, None, None)
    assert st == D.ERR_INVALID_ARG
    R = D._Router(64, 0, 10, D.BF16, 9, P, None, None, None)  # bad activation
    assert lib.dyna_route(ctypes.byref(R), P, D.BF16, 2, 3, P, None, None, P, 1 << 30, None) == D.ERR_INVALID_ARG


def test_build_layout_argument_errors():
    lib = D.lib()
    P = 0x10000
    cap = (ctypes.c_int32 * 11)()
    b = lib.dyna_build_layout
    assert b(None, 100, 10, P, D.BF16, 64, P + 4096, P, P, cap, None, P, 1 << 30, None) == D.ERR_INVALID_ARG
    assert b(P, 100, 101, P, D.BF16, 64, P + 4096, P, P, cap, None, P, 1 << 30, None) == D.ERR_INVALID_ARG
    assert b(P, 100, 10, P, D.BF16, 60, P + 4096, P, P, cap, None, P, 1 << 30, None) == D.ERR_INVALID_ARG
    assert b(P, 100, 10, P, D.BF16, 64, P, P, P, cap, None, P, 1 << 30, None) == D.ERR_INVALID_ARG
    assert b(P, 100, 10, P, D.BF16, 64, P + 4096, P, P, cap, None, P, 8, None) == D.ERR_WORKSPACE


def test_dense_head_argument_errors():
    lib = D.lib()
    P = 0x10000
    d = lib.dyna_dense_head
    assert d(P, D.BF16, 0, 64, P, D.BF16, 1, D.SEL_ARGMAX, 1, 1.0, None, P, None, None, None, None,
             P, 1 << 30, None) == D.ERR_INVALID_ARG
    assert d(P, D.BF16, 600000, 64, P, D.BF16, 1, D.SEL_ARGMAX, 1, 1.0, None, P, None, None, None,
             None, P, 1 << 30, None) == D.ERR_UNSUPPORTED
    assert d(P, D.BF16, 1000, 64, P, D.BF16, 1, D.SEL_ARGMAX, 1, 1.0, None, P, None, None, None,
             None, P, 4, None) == D.ERR_WORKSPACE


def test_position_budgets_match_the_oracle():
    from oracle import dynaspec_oracle as O
    lib = D.lib()
    for form, name in ((0, "equation"), (1, "algorithm1")):
        for k0, k1, k_min in ((64, 32, 1), (40, 16, 2), (8, 8, 1), (100, 63, 3)):
            for t in range(40):
                assert lib.dyna_cluster_budget(t, k0, k1, k_min, form) == O.k_schedule(t, k0, k1, k_min, form=name)
    for k_max in (1, 32, 1000, 32768):
        for t in range(40):
            assert lib.dyna_static_budget(t, k_max) == O.pa_fr_budget(t, k_max)
    assert lib.dyna_cluster_budget(-1, 64, 32, 1, 0) == -1
    assert lib.dyna_cluster_budget(3, 64, 32, 0, 0) == -1
    assert lib.dyna_cluster_budget(3, 64, 32, 1, 2) == -1
    assert lib.dyna_static_budget(3, 0) == -1
    assert D.cluster_budget(2, 64, 32) == 8 and D.static_budget(2, 32) == 10


def test_union_beam_and_kmeans_argument_errors():
    lib = D.lib()
    L, keep = _layout()
    P = 0x10000
    R = D._Router(64, 0, 10, D.BF16, 0, P, None, None, None)
    head = lib.dyna_draft_head

    def call(cap, beta=0.0, mode=D.SEL_TOPK | D.SEL_UNION):
        return head(ctypes.byref(R), ctypes.byref(L), P, P, D.BF16, 3, 3, mode, 4, 1.0, beta, None,
                    P, P, None, None, None, None, cap, P, 1 << 30, None, None, None)
    # a union of 3 rows x 3 clusters needs min(V, 3 * cap_by_k[3]) = 900 slots per row
    assert call(300) == D.ERR_CAPACITY
    assert call(900, beta=0.3) == D.ERR_UNSUPPORTED
    assert call(900, mode=D.SEL_UNION) == D.ERR_INVALID_ARG  # no selection asked for
    assert lib.dyna_set_option(D.OPT_LOGITS_PATH, 0) == D.OK
    # beam expansion: sizes are checked before any device work
    be = lib.dyna_beam_expand
    assert be(P, P, None, 2, 4, 0, P, P, P, None) == D.ERR_INVALID_ARG
    assert be(P, P, None, 2, 4, 65, P, P, P, None) == D.ERR_INVALID_ARG
    assert be(P, P, None, 2, 0, 4, P, P, P, None) == D.ERR_INVALID_ARG
    assert be(P, P, None, 200, 64, 8, P, P, P, None) == D.ERR_UNSUPPORTED  # B * k_t > 8192
    assert be(None, P, None, 2, 4, 4, P, P, P, None) == D.ERR_INVALID_ARG
    # partition builder
    assert lib.dyna_kmeans_workspace_bytes(1000, 64, 10) > 0
    km = lib.dyna_kmeans
    big = 1 << 34
    assert km(P, D.F32, 1000, 64, 10, P, 3, P, None, P, big, None) == D.ERR_UNSUPPORTED
    assert km(P, D.BF16, 1000, 60, 10, P, 3, P, None, P, big, None) == D.ERR_INVALID_ARG
    assert km(P, D.BF16, 1000, 64, 1001, P, 3, P, None, P, big, None) == D.ERR_INVALID_ARG
    assert km(P, D.BF16, 1000, 64, 10, P, 0, P, None, P, big, None) == D.ERR_INVALID_ARG
    assert km(P, D.BF16, 1000, 64, 10, None, 3, P, None, P, big, None) == D.ERR_INVALID_ARG
    assert km(P, D.BF16, 1000, 64, 10, P, 3, P, None, P, 16, None) == D.ERR_WORKSPACE
    assert km(P, D.BF16, 1000, 16384, 10, P, 3, P, None, P, big, None) == D.ERR_UNSUPPORTED
    assert lib.dyna_kmeans_assign(P, D.BF16, 1000, 64, None, 10, P, None, P, big, None) == D.ERR_INVALID_ARG
    assert lib.dyna_kmeans_update(P, D.BF16, 1000, 64, P, 10, None, P, big, None) == D.ERR_INVALID_ARG
