"""Python binding of libdynahead (ctypes).

Argument marshalling only: every step of the draft head runs in the HIP
kernels of libdynahead.so.  PyTorch supplies device memory and streams.  The
binding fails loudly when the library is missing; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdynahead.so")

OK, ERR_INVALID_ARG, ERR_CAPACITY, ERR_WORKSPACE, ERR_UNSUPPORTED, ERR_HIP, ERR_DEVICE_DATA = range(7)
F32, BF16 = 0, 1
ACT = {"none": 0, "relu": 1, "silu": 2}
SEL_ARGMAX, SEL_TOPK, SEL_SAMPLE, SEL_UNION = 1, 2, 4, 8
OPT_LOGITS_PATH, OPT_ROUTER_PATH, OPT_KERNEL_TIMING, OPT_GEMV_ROWS, OPT_FUSED_B1, OPT_MFMA_UNROLL = 1, 2, 3, 4, 5, 6
OPT_GATHER_CFG, OPT_GREEDY_GRID, OPT_UNION_CFG, OPT_KMEANS_CFG, OPT_WAIT_BOUND_US = 7, 8, 9, 10, 11
MAX_KT = 64


class DynaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


class _Layout(ctypes.Structure):
    _fields_ = [("V", ctypes.c_int32), ("d", ctypes.c_int32), ("M", ctypes.c_int32),
                ("wdtype", ctypes.c_int32), ("W_perm", ctypes.c_void_p),
                ("perm", ctypes.c_void_p), ("offsets", ctypes.c_void_p),
                ("cap_by_k", ctypes.c_void_p), ("max_cluster", ctypes.c_int32)]


class _Router(ctypes.Structure):
    _fields_ = [("d_r", ctypes.c_int32), ("H", ctypes.c_int32), ("M", ctypes.c_int32),
                ("wdtype", ctypes.c_int32), ("act", ctypes.c_int32), ("W1", ctypes.c_void_p),
                ("b1", ctypes.c_void_p), ("W2", ctypes.c_void_p), ("b2", ctypes.c_void_p)]


_lib = None
ABI_VERSION = 2  # DYNA_ABI_VERSION of include/dynahead.h

_P = ctypes.c_void_p
_I = ctypes.c_int32
_F = ctypes.c_float
_Z = ctypes.c_size_t

_SIGNATURES = {
    "dyna_abi_version": (_I, []),
    "dyna_status_string": (ctypes.c_char_p, [_I]),
    "dyna_last_error": (ctypes.c_char_p, []),
    "dyna_set_option": (_I, [_I, _I]),
    "dyna_kernel_timing": (_I, [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64), _I]),
    "dyna_layout_workspace_bytes": (_Z, [_I, _I]),
    "dyna_build_layout": (_I, [_P, _I, _I, _P, _I, _I, _P, _P, _P, _P, _P, _P, _Z, _P]),
    "dyna_workspace_bytes": (_Z, [_P, _P, _I, _I, _I]),
    "dyna_route": (_I, [_P, _P, _I, _I, _I, _P, _P, _P, _P, _Z, _P]),
    "dyna_shortlist": (_I, [_P, _P, _I, _I, _P, _P, _P, _P, _I, _P]),
    "dyna_shortlist_logits": (_I, [_P, _P, _I, _I, _I, _P, _P, _P, _P, _I, _P, _Z, _P]),
    "dyna_draft_select": (_I, [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _F, _F, _P, _P, _P, _P, _P,
                               _P, _Z, _P]),
    "dyna_draft_head": (_I, [_P, _P, _P, _P, _I, _I, _I, _I, _I, _F, _F, _P, _P, _P, _P, _P, _P, _P,
                             _I, _P, _Z, _P, _P, _P]),
    "dyna_draft_head_noalloc": (_I, [_P, _P, _P, _P, _I, _I, _I, _I, _I, _F, _F, _P, _P, _P, _P, _P, _P, _P,
                                     _I, _P]),
    "dyna_dense_workspace_bytes": (_Z, [_I, _I]),
    "dyna_cluster_budget": (_I, [_I, _I, _I, _I, _I]),
    "dyna_beam_expand": (_I, [_P, _P, _P, _I, _I, _I, _P, _P, _P, _P]),
    "dyna_kmeans_workspace_bytes": (ctypes.c_size_t, [_I, _I, _I]),
    "dyna_kmeans_assign": (_I, [_P, _I, _I, _I, _P, _I, _P, _P, _P, ctypes.c_size_t, _P]),
    "dyna_kmeans_update": (_I, [_P, _I, _I, _I, _P, _I, _P, _P, ctypes.c_size_t, _P]),
    "dyna_kmeans": (_I, [_P, _I, _I, _I, _I, _P, _I, _P, _P, _P, ctypes.c_size_t, _P]),
    "dyna_static_budget": (_I, [_I, _I]),
    "dyna_dense_head": (_I, [_P, _I, _I, _I, _P, _I, _I, _I, _I, _F, _P, _P, _P, _P, _P, _P, _P,
                             _Z, _P]),
}
EXPORTED = tuple(_SIGNATURES)


def lib():
    """Load libdynahead.so (built in-tree).  Raises if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2510_13847_amd.build` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        if L.dyna_abi_version() != ABI_VERSION:
            raise RuntimeError("libdynahead ABI version mismatch")
        _lib = L
    return _lib


def _check(status: int):
    if status != OK:
        raise DynaError(status, lib().dyna_last_error().decode())


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream(stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _need(t, name, device=True, contiguous=True):
    if t is None:
        raise ValueError(f"{name} is required")
    if device and not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if contiguous and not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def set_option(option: int, value: int):
    _check(lib().dyna_set_option(option, value))


def kernel_timing(reset=True):
    """(total_ms, launches) of the gathered-head kernel launches timed so far."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check(lib().dyna_kernel_timing(ctypes.byref(ms), ctypes.byref(n), 1 if reset else 0))
    return ms.value, n.value


# --------------------------------------------------------------------------
@dataclass
class Layout:
    """Device layout from build_layout (tensors are kept alive here)."""
    V: int
    d: int
    M: int
    W_perm: object
    perm: object
    offsets: object
    cap_by_k: np.ndarray   # host int32 [M + 1]
    max_cluster: int

    def __post_init__(self):
        self._c = _Layout(self.V, self.d, self.M, _dtype_code(self.W_perm), _ptr(self.W_perm),
                          _ptr(self.perm), _ptr(self.offsets),
                          self.cap_by_k.ctypes.data_as(ctypes.c_void_p).value, self.max_cluster)

    def with_weights(self, W_perm) -> "Layout":
        """The same layout over another copy of the permuted head (replicas)."""
        return Layout(self.V, self.d, self.M, W_perm, self.perm, self.offsets, self.cap_by_k,
                      self.max_cluster)

    @property
    def c(self):
        return ctypes.byref(self._c)

    def cap(self, k: int) -> int:
        return int(self.cap_by_k[k])


@dataclass
class Router:
    W1: object
    W2: Optional[object] = None
    b1: Optional[object] = None
    b2: Optional[object] = None
    act: str = "silu"

    def __post_init__(self):
        H = 0 if self.W2 is None else self.W1.shape[0]
        M = self.W1.shape[0] if self.W2 is None else self.W2.shape[0]
        self.d_r, self.H, self.M = self.W1.shape[1], H, M
        self._c = _Router(self.d_r, H, M, _dtype_code(self.W1), ACT[self.act], _ptr(self.W1),
                          _ptr(self.b1), _ptr(self.W2), _ptr(self.b2))

    @property
    def c(self):
        return ctypes.byref(self._c)


# --------------------------------------------------------------------------
def layout_workspace_bytes(V: int, M: int) -> int:
    return int(lib().dyna_layout_workspace_bytes(V, M))


def build_layout(cluster_of, W_lm, M: int, stream=None) -> Layout:
    """dyna_build_layout: cluster-contiguous copy of W_lm [V, d] (synchronous)."""
    import torch
    _need(cluster_of, "cluster_of")
    _need(W_lm, "W_lm")
    V, d = W_lm.shape
    dev = W_lm.device
    W_perm = torch.empty_like(W_lm)
    perm = torch.empty(V, dtype=torch.int32, device=dev)
    offsets = torch.empty(M + 1, dtype=torch.int32, device=dev)
    cap = np.zeros(M + 1, dtype=np.int32)
    mx = ctypes.c_int32(0)
    wsb = layout_workspace_bytes(V, M)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
    _check(lib().dyna_build_layout(_ptr(cluster_of), V, M, _ptr(W_lm), _dtype_code(W_lm), d,
                                   _ptr(W_perm), _ptr(perm), _ptr(offsets),
                                   cap.ctypes.data_as(ctypes.c_void_p), ctypes.byref(mx),
                                   _ptr(ws), wsb, _stream(stream)))
    return Layout(V, d, M, W_perm, perm, offsets, cap, int(mx.value))


def workspace_bytes(layout: Optional[Layout], router: Optional[Router], B: int, k: int, cap: int) -> int:
    return int(lib().dyna_workspace_bytes(layout.c if layout else None, router.c if router else None,
                                          B, k, cap))


def workspace(layout, router, B, k, cap, device="cuda"):
    """Zero-filled workspace (the one-context kernels' counters start at zero)."""
    import torch
    n = workspace_bytes(layout, router, B, k, cap)
    return torch.zeros(max(n, 1), dtype=torch.uint8, device=device)


def route(router: Router, x, k: int, ws=None, want_scores=False, stream=None):
    """dyna_route -> (topk_ids [B, k] int32, topk_scores [B, k], scores [B, M] or None)."""
    import torch
    _need(x, "x")
    B = x.shape[0]
    dev = x.device
    ids = torch.empty((B, k), dtype=torch.int32, device=dev)
    sc = torch.empty((B, k), dtype=torch.float32, device=dev)
    scores = torch.empty((B, router.M), dtype=torch.float32, device=dev) if want_scores else None
    if ws is None:
        ws = workspace(None, router, B, k, 0, dev)
    _check(lib().dyna_route(router.c, _ptr(x), _dtype_code(x), B, k, _ptr(ids), _ptr(sc),
                            _ptr(scores), _ptr(ws), ws.numel(), _stream(stream)))
    return ids, sc, scores


def shortlist(layout: Layout, topk_ids, with_ids=True, stream=None):
    """dyna_shortlist -> (sel_sorted, sel_rowoff, row_len, shortlist_ids or None)."""
    import torch
    _need(topk_ids, "topk_ids")
    B, k = topk_ids.shape
    dev = topk_ids.device
    cap = layout.cap(k)
    sel = torch.empty((B, k), dtype=torch.int32, device=dev)
    rowoff = torch.empty((B, k + 1), dtype=torch.int32, device=dev)
    row_len = torch.empty(B, dtype=torch.int32, device=dev)
    ids = torch.full((B, max(cap, 1)), -1, dtype=torch.int32, device=dev) if with_ids else None
    _check(lib().dyna_shortlist(layout.c, _ptr(topk_ids), B, k, _ptr(sel), _ptr(rowoff),
                                _ptr(row_len), _ptr(ids), cap, _stream(stream)))
    return sel, rowoff, row_len, ids


def shortlist_logits(layout: Layout, h, sel_sorted, sel_rowoff, row_len, cap=None, ws=None,
                     out=None, stream=None):
    """dyna_shortlist_logits -> logits [B, cap] fp32 (slots past row_len untouched)."""
    import torch
    _need(h, "h")
    B, k = sel_sorted.shape
    cap = layout.cap(k) if cap is None else cap
    dev = h.device
    if out is None:
        out = torch.full((B, cap), float("nan"), dtype=torch.float32, device=dev)
    if ws is None:
        ws = workspace(layout, None, B, k, cap, dev)
    _check(lib().dyna_shortlist_logits(layout.c, _ptr(h), _dtype_code(h), B, k, _ptr(sel_sorted),
                                       _ptr(sel_rowoff), _ptr(row_len), _ptr(out), cap, _ptr(ws),
                                       ws.numel(), _stream(stream)))
    return out


def _select_outputs(B, k_t, mode, dev):
    import torch
    want_ids = bool(mode & (SEL_ARGMAX | SEL_TOPK))
    kt = k_t if mode & SEL_TOPK else 1
    ids = torch.empty((B, kt), dtype=torch.int32, device=dev) if want_ids else None
    lps = torch.empty((B, kt), dtype=torch.float32, device=dev) if want_ids else None
    smp = torch.empty(B, dtype=torch.int32, device=dev) if mode & SEL_SAMPLE else None
    slp = torch.empty(B, dtype=torch.float32, device=dev) if mode & SEL_SAMPLE else None
    return ids, lps, smp, slp


def draft_select(layout: Layout, logits, sel_sorted, sel_rowoff, row_len, mode=SEL_TOPK, k_t=1,
                 temperature=1.0, uniforms=None, cap=None, ws=None, stream=None, tail_beta=0.0):
    """dyna_draft_select -> dict(ids, logprobs, sample, sample_logprob)."""
    B, k = sel_sorted.shape
    cap = logits.shape[1] if cap is None else cap
    dev = logits.device
    ids, lps, smp, slp = _select_outputs(B, k_t, mode, dev)
    if ws is None:
        ws = workspace(layout, None, B, k, cap, dev)
    _check(lib().dyna_draft_select(layout.c, _ptr(logits), _ptr(sel_sorted), _ptr(sel_rowoff),
                                   _ptr(row_len), B, k, cap, mode, k_t, temperature, tail_beta,
                                   _ptr(uniforms), _ptr(ids), _ptr(lps), _ptr(smp), _ptr(slp),
                                   _ptr(ws), ws.numel(), _stream(stream)))
    return dict(ids=ids, logprobs=lps, sample=smp, sample_logprob=slp)


class DraftHead:
    """Preallocated outputs + workspace for repeated dyna_draft_head calls."""

    def __init__(self, router: Router, layout: Layout, B: int, k: int, mode: int, k_t: int = 1,
                 temperature: float = 1.0, keep_logits=False, keep_clusters=True, device="cuda",
                 tail_beta: float = 0.0):
        import torch
        self.router, self.layout, self.B, self.k = router, layout, B, k
        self.mode, self.k_t, self.temperature, self.tail_beta = mode, k_t, temperature, tail_beta
        # DYNA_SEL_UNION: every row's logits span the step's shared shortlist
        self.cap = union_cap(layout, B, k) if (mode & SEL_UNION) and B > 1 else layout.cap(k)
        self.ids, self.logprobs, self.sample, self.sample_logprob = _select_outputs(B, k_t, mode, device)
        self.clusters = torch.empty((B, k), dtype=torch.int32, device=device) if keep_clusters else None
        self.logits = torch.full((B, self.cap), float("nan"), dtype=torch.float32,
                                 device=device) if keep_logits else None
        self.ws = workspace(layout, router, B, k, self.cap, device)

    def __call__(self, x, h, uniforms=None, stream=None, route_stream=None, x_ready=None,
                 layout: Optional[Layout] = None, router: Optional[Router] = None):
        L = layout or self.layout
        R = router or self.router
        rs = None if route_stream is None else route_stream.cuda_stream
        ev = None if x_ready is None else x_ready.cuda_event
        _check(lib().dyna_draft_head(R.c, L.c, _ptr(x), _ptr(h), _dtype_code(h), self.B, self.k,
                                     self.mode, self.k_t, self.temperature, self.tail_beta, _ptr(uniforms),
                                     _ptr(self.ids), _ptr(self.logprobs), _ptr(self.sample),
                                     _ptr(self.sample_logprob), _ptr(self.clusters),
                                     _ptr(self.logits), self.cap, _ptr(self.ws), self.ws.numel(),
                                     _stream(stream), rs, ev))
        return self


NOALLOC_SCRATCH_BYTES = 16 << 20  # DYNA_NOALLOC_SCRATCH_BYTES


def draft_head_noalloc(head: "DraftHead", x, h, uniforms=None, stream=None,
                       layout: Optional[Layout] = None, router: Optional[Router] = None):
    """dyna_draft_head_noalloc into head's preallocated outputs (its own
    workspace is not used: the library's static scratch stands in for it)."""
    L = layout or head.layout
    R = router or head.router
    _check(lib().dyna_draft_head_noalloc(R.c, L.c, _ptr(x), _ptr(h), _dtype_code(h), head.B, head.k,
                                         head.mode, head.k_t, head.temperature, head.tail_beta,
                                         _ptr(uniforms), _ptr(head.ids), _ptr(head.logprobs),
                                         _ptr(head.sample), _ptr(head.sample_logprob), _ptr(head.clusters),
                                         _ptr(head.logits), head.cap, _stream(stream)))
    return head


def draft_head(router: Router, layout: Layout, x, h, k: int, mode=SEL_ARGMAX, k_t=1,
               temperature=1.0, uniforms=None, keep_logits=True, stream=None, route_stream=None,
               tail_beta=0.0):
    """One dyna_draft_head call with fresh outputs (see DraftHead for repeated calls)."""
    head = DraftHead(router, layout, h.shape[0], k, mode, k_t, temperature, keep_logits=keep_logits,
                     device=h.device, tail_beta=tail_beta)
    head(x, h, uniforms, stream=stream, route_stream=route_stream)
    return head


def dense_workspace_bytes(n_rows: int, B: int) -> int:
    return int(lib().dyna_dense_workspace_bytes(n_rows, B))


class DenseHead:
    """dyna_dense_head over rows [0, n_rows) of W (dense when n_rows = V)."""

    def __init__(self, W, n_rows: int, B: int, mode: int, k_t: int = 1, temperature: float = 1.0,
                 keep_logits=False, device="cuda"):
        import torch
        self.W, self.n_rows, self.B = W, n_rows, B
        self.mode, self.k_t, self.temperature = mode, k_t, temperature
        self.ids, self.logprobs, self.sample, self.sample_logprob = _select_outputs(B, k_t, mode, device)
        self.logits = torch.empty((B, n_rows), dtype=torch.float32, device=device) if keep_logits else None
        n = dense_workspace_bytes(n_rows, B)
        self.ws = torch.empty(max(n, 1), dtype=torch.uint8, device=device)

    def __call__(self, h, uniforms=None, stream=None, W=None):
        W = self.W if W is None else W
        _check(lib().dyna_dense_head(_ptr(W), _dtype_code(W), self.n_rows, W.shape[1], _ptr(h),
                                     _dtype_code(h), self.B, self.mode, self.k_t, self.temperature,
                                     _ptr(uniforms), _ptr(self.ids), _ptr(self.logprobs),
                                     _ptr(self.sample), _ptr(self.sample_logprob), _ptr(self.logits),
                                     _ptr(self.ws), self.ws.numel(), _stream(stream)))
        return self


def cluster_budget(t, k0, k1, k_min=1, form=0):
    """Cluster budget k_c(t) (form 0: the paper's equation, 1: the appendix algorithm's)."""
    v = lib().dyna_cluster_budget(t, k0, k1, k_min, form)
    if v < 0:
        raise ValueError("invalid cluster budget arguments")
    return v


def static_budget(t, k_max):
    """PA-FR static shortlist size K_fr(t)."""
    v = lib().dyna_static_budget(t, k_max)
    if v < 0:
        raise ValueError("invalid static budget arguments")
    return v


def union_cap(layout: "Layout", B: int, k: int) -> int:
    """Logits row stride a DYNA_SEL_UNION step of B rows needs: min(V, B * cap_by_k[k])."""
    return min(layout.V, B * layout.cap(k))


def beam_expand(logprobs, ids, last_scores=None, n_out=None, stream=None, out=None):
    """dyna_beam_expand -> (scores[n_out], parent[n_out], ids[n_out]); out: an
    existing (scores, parent, ids) triple to write instead of fresh tensors."""
    import torch
    B, k_t = logprobs.shape
    n_out = k_t if n_out is None else n_out
    dev = logprobs.device
    if out is not None:
        sc, par, tok = out
        for t, dt in zip(out, (torch.float32, torch.int32, torch.int32)):
            _need(t, "out")
            if t.dtype != dt or t.numel() < n_out:
                raise ValueError("beam_expand: out tensors must be (float32, int32, int32) of n_out entries")
    else:
        sc = torch.empty(n_out, dtype=torch.float32, device=dev)
        par = torch.empty(n_out, dtype=torch.int32, device=dev)
        tok = torch.empty(n_out, dtype=torch.int32, device=dev)
    _check(lib().dyna_beam_expand(_ptr(logprobs), _ptr(ids), _ptr(last_scores), B, k_t, n_out, _ptr(sc),
                                  _ptr(par), _ptr(tok), _stream(stream)))
    return sc, par, tok


# ---------------------------------------------------------------- partition builder
def kmeans_workspace(W, M: int):
    import torch
    V, d = W.shape
    n = int(lib().dyna_kmeans_workspace_bytes(V, d, M))
    return torch.empty(max(n, 1), dtype=torch.uint8, device=W.device)


def kmeans_assign(W, centroids, ws=None, stream=None, want_score=False):
    """dyna_kmeans_assign -> (assign[V] int32, score[V] float32 or None)."""
    import torch
    V, d = W.shape
    M = centroids.shape[0]
    ws = kmeans_workspace(W, M) if ws is None else ws
    a = torch.empty(V, dtype=torch.int32, device=W.device)
    sc = torch.empty(V, dtype=torch.float32, device=W.device) if want_score else None
    _check(lib().dyna_kmeans_assign(_ptr(W), _dtype_code(W), V, d, _ptr(centroids), M, _ptr(a), _ptr(sc),
                                    _ptr(ws), ws.numel(), _stream(stream)))
    return a, sc


def kmeans_update(W, assign, centroids, ws=None, stream=None):
    """dyna_kmeans_update, in place on centroids (fp32 [M, d])."""
    V, d = W.shape
    M = centroids.shape[0]
    ws = kmeans_workspace(W, M) if ws is None else ws
    _check(lib().dyna_kmeans_update(_ptr(W), _dtype_code(W), V, d, _ptr(assign), M, _ptr(centroids), _ptr(ws),
                                    ws.numel(), _stream(stream)))
    return centroids


def kmeans(W, M: int, init_ids, iters: int, ws=None, stream=None, keep_centroids=True):
    """dyna_kmeans -> (cluster_of[V] int32, centroids[M, d] float32 or None)."""
    import torch
    V, d = W.shape
    ws = kmeans_workspace(W, M) if ws is None else ws
    cl = torch.empty(V, dtype=torch.int32, device=W.device)
    mu = torch.empty((M, d), dtype=torch.float32, device=W.device) if keep_centroids else None
    _check(lib().dyna_kmeans(_ptr(W), _dtype_code(W), V, d, M, _ptr(init_ids), iters, _ptr(cl), _ptr(mu),
                             _ptr(ws), ws.numel(), _stream(stream)))
    return cl, mu
