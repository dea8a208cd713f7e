"""Seeded synthetic workloads for the DynaSpec dynamic draft head.

This module only draws inputs: cluster partitions, LM-head and router weights,
context features and sampling uniforms.  It holds none of the method's
arithmetic (no routing, no top-k, no shortlist, no logits, no selection), so
that the CPU oracle and the HIP path can both be fed from it without sharing
any computation.

Shapes follow the paper's workloads (Llama-3-8B, Qwen-2.5 and Gemma-3 sized
vocabularies, Sec. 1 and Sec. 6); the paper's datasets and trained weights are
not available, so every tensor is random with the distributions below:

* cluster sizes: equal, lognormal(0, sigma) or capped Zipf(s) weights,
  rescaled to sum to V and rounded by largest remainder (ties -> lower id),
  each cluster at least one token; tokens are assigned to clusters by a seeded
  permutation of the vocabulary cut into consecutive runs;
* W_LM ~ N(0, 1/d), W1 ~ N(0, 1/d_r), W2 ~ N(0, 1/H), h = x ~ N(0, 1),
  all rounded to bf16 (round-to-nearest-even) for bf16 workloads;
* u ~ U[0, 1) in fp32, one per context row.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

BASE_SEED = 251013847


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: int            # position in the workload list; seeds derive from it
    V: int
    d: int
    M: int
    dtype: str            # "f32" or "bf16" (weights and activations)
    sizes: tuple          # ("equal",) | ("lognormal", sigma) | ("zipf", s, cap)
    H: int                # router hidden width; 0 = single linear d_r -> M
    act: str              # "none" | "relu" | "silu"
    k: int                # clusters per context
    B: int                # contexts per step
    modes: tuple          # subset of ("argmax", "topk", "sample")
    k_t: int              # tokens per context for top-k output
    seed_index: Optional[int] = None  # reuse another workload's partition/router/LM head
    overlap_gemm: Optional[tuple] = None  # (rows, K, N) stand-in draft-layer GEMM
    static_prefix: int = 32768
    union: bool = False   # the step's rows share one shortlist (union of their clusters)

    @property
    def d_r(self) -> int:
        return self.d


WORKLOADS = {
    w.name: w
    for w in [
        Workload("tiny_fp32", 0, V=8192, d=256, M=64, dtype="f32", sizes=("equal",),
                 H=0, act="none", k=4, B=4, modes=("argmax", "topk"), k_t=8,
                 static_prefix=512),
        # the draft-layer stand-in for the chain: one [4096 x 14336] projection
        # of the drafter's MLP at B = 1 (117 MB of bf16 weights)
        Workload("llama3_8b_chain", 1, V=128256, d=4096, M=1024, dtype="bf16",
                 sizes=("lognormal", 0.5), H=1024, act="silu", k=32, B=1,
                 modes=("argmax",), k_t=1, overlap_gemm=(1, 4096, 14336)),
        Workload("llama3_8b_tree", 2, V=128256, d=4096, M=1024, dtype="bf16",
                 sizes=("lognormal", 0.5), H=1024, act="silu", k=32, B=64,
                 modes=("topk",), k_t=10, seed_index=1),
        Workload("qwen25_serving", 3, V=151936, d=3584, M=2048, dtype="bf16",
                 sizes=("zipf", 1.1, 4096), H=1024, act="silu", k=64, B=16,
                 modes=("sample",), k_t=1),
        Workload("gemma3_large_vocab", 4, V=262144, d=5376, M=4096, dtype="bf16",
                 sizes=("lognormal", 0.7), H=2048, act="silu", k=64, B=128,
                 modes=("topk", "sample"), k_t=10, overlap_gemm=(128, 5376, 14336)),
        # the tree batch (same seeds: partition, weights and contexts) with one
        # union shortlist per step, the beam form of Sec. 4.2
        Workload("llama3_8b_tree_union", 2, V=128256, d=4096, M=1024, dtype="bf16",
                 sizes=("lognormal", 0.5), H=1024, act="silu", k=32, B=64,
                 modes=("topk",), k_t=10, seed_index=1, union=True),
    ]
}
WORKLOAD_ORDER = ["tiny_fp32", "llama3_8b_chain", "llama3_8b_tree",
                  "qwen25_serving", "gemma3_large_vocab", "llama3_8b_tree_union"]


def scaled(w: Workload, **changes) -> Workload:
    """A copy of a workload with some fields replaced (used for small test cases)."""
    return dataclasses.replace(w, **changes)


# One GPU's share of a batch split by context rows over eight GPUs (the rows
# are independent: no exchange between the GPUs).  The same partition, router
# and LM head; B / 8 rows.
SHARD_WORKLOADS = {
    w.name: w
    for w in [
        scaled(WORKLOADS["llama3_8b_tree"], name="llama3_8b_tree_shard8", B=8),
        scaled(WORKLOADS["gemma3_large_vocab"], name="gemma3_large_vocab_shard8", B=16, seed_index=4,
               overlap_gemm=None),
    ]
}


# --------------------------------------------------------------------------
# seeds
# --------------------------------------------------------------------------
_STREAMS = ("partition", "W1", "W2", "W_LM", "h", "u", "replicas", "spare")


def stream_seed(w: Workload, stream: str, salt: int = 0) -> int:
    """Integer seed for one named random stream of a workload."""
    idx = w.index
    if w.seed_index is not None and stream in ("partition", "W1", "W2", "W_LM"):
        idx = w.seed_index
    ss = np.random.SeedSequence(BASE_SEED + idx).spawn(len(_STREAMS))[_STREAMS.index(stream)]
    base = int(ss.generate_state(1, dtype=np.uint64)[0] & ((1 << 62) - 1))
    return (base + salt) & ((1 << 62) - 1)


# --------------------------------------------------------------------------
# cluster partitions
# --------------------------------------------------------------------------
def _largest_remainder(target: np.ndarray, total: int, lo: int = 1,
                       hi: Optional[int] = None) -> np.ndarray:
    """Round non-negative reals to integers in [lo, hi] that sum to `total`.

    Floors first, then hands out the missing units by largest remainder
    (ties -> lower index); removes surplus units (created by the lower clamp)
    from the smallest remainders that can still give one.
    """
    n = target.size
    base = np.floor(target).astype(np.int64)
    base = np.maximum(base, lo)
    if hi is not None:
        base = np.minimum(base, hi)
    rem = target - np.floor(target)
    deficit = total - int(base.sum())
    idx = np.arange(n)
    if deficit > 0:
        order = np.lexsort((idx, -rem))
        for i in order:
            if deficit == 0:
                break
            if hi is None or base[i] < hi:
                base[i] += 1
                deficit -= 1
        if deficit != 0:
            raise ValueError("cannot distribute cluster sizes")
    elif deficit < 0:
        order = np.lexsort((idx, rem))
        for i in order:
            if deficit == 0:
                break
            if base[i] > lo:
                base[i] -= 1
                deficit += 1
        if deficit != 0:
            raise ValueError("cannot distribute cluster sizes")
    return base


def cluster_sizes(w: Workload) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(stream_seed(w, "partition")))
    kind = w.sizes[0]
    if kind == "equal":
        if w.V % w.M:
            raise ValueError("equal sizes need M | V")
        return np.full(w.M, w.V // w.M, dtype=np.int64)
    if kind == "lognormal":
        sigma = float(w.sizes[1])
        x = rng.lognormal(0.0, sigma, size=w.M)
        return _largest_remainder(x / x.sum() * w.V, w.V)
    if kind == "zipf":
        s, cap = float(w.sizes[1]), int(w.sizes[2])
        r = np.arange(1, w.M + 1, dtype=np.float64)
        wgt = r ** (-s)
        lo, hi = 0.0, float(w.V) / wgt.min() + 1.0
        for _ in range(200):  # water-fill the scale so that sum(min(cap, c*w)) == V
            c = 0.5 * (lo + hi)
            if np.minimum(cap, c * wgt).sum() > w.V:
                hi = c
            else:
                lo = c
        t = np.minimum(cap, lo * wgt)
        return _largest_remainder(t, w.V, lo=1, hi=cap)
    raise ValueError(kind)


def partition(w: Workload) -> np.ndarray:
    """cluster_of[V] (int32): cluster id of every vocabulary token."""
    sizes = cluster_sizes(w)
    rng = np.random.Generator(np.random.PCG64(stream_seed(w, "partition", salt=1)))
    order = rng.permutation(w.V)
    cluster_of = np.empty(w.V, dtype=np.int32)
    start = 0
    for m, s in enumerate(sizes):
        cluster_of[order[start:start + s]] = m
        start += int(s)
    assert start == w.V
    return cluster_of


# --------------------------------------------------------------------------
# dense tensors (torch; generated on the device that will use them)
# --------------------------------------------------------------------------
def _torch():
    import torch
    return torch


def _randn(shape, seed, device, scale, dtype_name, chunk_rows=16384):
    torch = _torch()
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    out_dtype = torch.float32 if dtype_name == "f32" else torch.bfloat16
    out = torch.empty(shape, dtype=out_dtype, device=device)
    rows = shape[0]
    # chunked so the fp32 temporary of a multi-GB LM head stays small
    for r0 in range(0, rows, chunk_rows):
        r1 = min(rows, r0 + chunk_rows)
        t = torch.randn((r1 - r0,) + tuple(shape[1:]), generator=g, device=device,
                        dtype=torch.float32)
        t.mul_(scale)
        out[r0:r1].copy_(t)  # fp32 -> bf16 rounds to nearest even
    return out


def lm_head(w: Workload, device="cpu"):
    """W_LM as a [V, d] row-major tensor (one paper column per row)."""
    return _randn((w.V, w.d), stream_seed(w, "W_LM"), device, 1.0 / math.sqrt(w.d), w.dtype)


def router_weights(w: Workload, device="cpu"):
    """(W1, W2): W1 is [H, d_r] (or [M, d_r] for a single linear), W2 is [M, H] or None."""
    if w.H == 0:
        W1 = _randn((w.M, w.d_r), stream_seed(w, "W1"), device, 1.0 / math.sqrt(w.d_r), w.dtype)
        return W1, None
    W1 = _randn((w.H, w.d_r), stream_seed(w, "W1"), device, 1.0 / math.sqrt(w.d_r), w.dtype)
    W2 = _randn((w.M, w.H), stream_seed(w, "W2"), device, 1.0 / math.sqrt(w.H), w.dtype)
    return W1, W2


def contexts(w: Workload, device="cpu", batch: Optional[int] = None, salt: int = 0):
    """h[B, d] draft hidden states; the router reads the same rows as x."""
    B = w.B if batch is None else batch
    return _randn((B, w.d), stream_seed(w, "h", salt), device, 1.0, w.dtype)


def uniforms(w: Workload, device="cpu", batch: Optional[int] = None, salt: int = 0):
    """u[B] in [0, 1), fp32, one per context row."""
    torch = _torch()
    B = w.B if batch is None else batch
    g = torch.Generator(device=device)
    g.manual_seed(int(stream_seed(w, "u", salt)))
    return torch.rand(B, generator=g, device=device, dtype=torch.float32)


def overlap_gemm_operands(w: Workload, device="cpu"):
    """Stand-in draft-layer GEMM operands (rows x K) @ (K x N), bf16."""
    rows, K, N = w.overlap_gemm
    a = _randn((rows, K), stream_seed(w, "spare", 1), device, 1.0, "bf16")
    b = _randn((K, N), stream_seed(w, "spare", 2), device, 1.0 / math.sqrt(K), "bf16")
    return a, b


def kmeans_init_ids(w: Workload, M: Optional[int] = None, salt: int = 0) -> np.ndarray:
    """M distinct vocabulary ids (seeded) where the partition builder's
    centroids start."""
    M = w.M if M is None else M
    rng = np.random.default_rng(stream_seed(w, "spare", 100 + salt))
    return np.sort(rng.choice(w.V, size=M, replace=False)).astype(np.int32)


def planted_head(V: int, d: int, M: int, seed: int, noise: float = 0.3, device="cpu"):
    """A synthetic bf16 LM head with cluster structure: M random directions,
    row v = (a positive length) * direction[g_v] + isotropic noise, groups g_v
    cut from a seeded permutation into near-equal runs.  Returns (W[V, d],
    groups[V])."""
    torch = _torch()
    rng = np.random.default_rng(seed)
    groups = np.empty(V, dtype=np.int64)
    groups[rng.permutation(V)] = np.arange(V) % M
    dirs = rng.standard_normal((M, d))
    lengths = rng.uniform(0.5, 2.0, size=(V, 1))
    W = dirs[groups] * lengths + noise * rng.standard_normal((V, d))
    return torch.from_numpy(W.astype(np.float32)).to(torch.bfloat16).to(device), groups


def bf16_bits(t) -> np.ndarray:
    """Raw bf16 bit patterns (uint16) of a torch bfloat16 tensor, on the host."""
    torch = _torch()
    assert t.dtype == torch.bfloat16
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def host_array(t) -> np.ndarray:
    """Host copy of a tensor as the oracle takes it: fp32 arrays or bf16 bit patterns."""
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return bf16_bits(t)
    return t.detach().cpu().contiguous().numpy()
