// Routing top-k, shortlist construction, the gathered-head work plan and the
// draft selection.
//
//  topk_clusters_kernel  K_b = TopK_k(s_b) (Sec. 4.2): radix select of the
//                        k-th largest score on 8-bit digits, then the ties at
//                        that score taken lowest id first; optionally also the
//                        row's shortlist (Sec. 4.2: V_S = disjoint union of the
//                        selected clusters) as a prefix sum of cluster sizes.
//  shortlist_kernel      the same shortlist from any list of cluster ids.
//  plan_kernel           the batch's distinct selected clusters, cut into
//                        16-row chunks, each with the contexts that chose it,
//                        so that every selected slab is streamed once.
//  select_partial/final  Algorithm 1's log_softmax, TopK_{k_t} and remap to
//                        vocabulary ids, plus inverse-CDF sampling from the
//                        restricted draft q_S (Sec. 5), split over 1024- or
//                        2048-slot segments so long rows (the dense
//                        baseline) spread over many workgroups.
#include <atomic>
#include <mutex>

#include "topk.h"
#include "select_row.h"

namespace dyna {
namespace {

// ------------------------------------------------------------------ top-k
__global__ __launch_bounds__(kNT) void topk_clusters_kernel(TopkArgs A) {
    extern __shared__ unsigned char smem[];
    topk_row(A, blockIdx.x, smem);
}

// ------------------------------------------------------------------ shortlist
__global__ __launch_bounds__(kNT) void shortlist_kernel(
    const int32_t* __restrict__ offsets, const int32_t* __restrict__ perm, int M,
    const int32_t* __restrict__ topk_ids, int k, int32_t* __restrict__ sel_sorted,
    int32_t* __restrict__ sel_rowoff, int32_t* __restrict__ row_len,
    int32_t* __restrict__ shortlist_ids, int64_t cap) {
    extern __shared__ int32_t sl[];
    int32_t* ids = sl;            // [k] input ids, -1 when dropped
    int32_t* sid = sl + k;        // [k] kept ids ascending, then -1
    int32_t* soff = sl + 2 * k;   // [k + 1] row offsets
    __shared__ int tmp[kNT / kWave + 1];
    __shared__ int sh_nkeep;
    const int b = blockIdx.x;
    const int32_t* in = topk_ids + (int64_t)b * k;

    for (int i = threadIdx.x; i < k; i += kNT) {
        const int m = in[i];
        ids[i] = (m >= 0 && m < M) ? m : -1;
    }
    __syncthreads();
    // drop repeats: keep the first occurrence of every id
    for (int i = threadIdx.x; i < k; i += kNT) {
        const int m = ids[i];
        bool dup = false;
        if (m >= 0)
            for (int j = 0; j < i; ++j) dup |= ids[j] == m;
        sid[i] = dup ? -1 : m;   // staging: kept id or -1
    }
    __syncthreads();
    for (int i = threadIdx.x; i < k; i += kNT) ids[i] = sid[i];
    __syncthreads();
    int nkeep_local = 0;
    for (int i = threadIdx.x; i < k; i += kNT) nkeep_local += ids[i] >= 0;
    int nkeep;
    block_exclusive_scan<kNT>(nkeep_local, tmp, &nkeep);
    for (int i = threadIdx.x; i < k; i += kNT) sid[i] = -1;
    __syncthreads();
    for (int i = threadIdx.x; i < k; i += kNT) {
        const int m = ids[i];
        if (m < 0) continue;
        int rank = 0;
        for (int j = 0; j < k; ++j) rank += (ids[j] >= 0 && ids[j] < m);
        sid[rank] = m;
    }
    if (threadIdx.x == 0) sh_nkeep = nkeep;
    __syncthreads();

    const int per = (k + kNT - 1) / kNT;
    const int i0 = min(k, (int)threadIdx.x * per);
    const int i1 = min(k, i0 + per);
    int local = 0;
    for (int i = i0; i < i1; ++i) {
        const int m = sid[i];
        local += m >= 0 ? offsets[m + 1] - offsets[m] : 0;
    }
    int len;
    int run = block_exclusive_scan<kNT>(local, tmp, &len);
    for (int i = i0; i < i1; ++i) {
        const int m = sid[i];
        sel_sorted[(int64_t)b * k + i] = m;
        sel_rowoff[(int64_t)b * (k + 1) + i] = run;
        soff[i] = run;
        run += m >= 0 ? offsets[m + 1] - offsets[m] : 0;
    }
    if (threadIdx.x == 0) {
        sel_rowoff[(int64_t)b * (k + 1) + k] = len;
        row_len[b] = len;
    }
    __syncthreads();
    if (shortlist_ids != nullptr) {
        for (int i = 0; i < sh_nkeep; ++i) {
            const int m = sid[i];
            const int o = offsets[m], n = offsets[m + 1] - o;
            for (int t = threadIdx.x; t < n; t += kNT)
                shortlist_ids[(int64_t)b * cap + soff[i] + t] = perm[o + t];
        }
    }
}

// ------------------------------------------------------------------ plan
// Up to kPlanGrid workgroups.  Each one counts the contexts per cluster and
// scans the counts itself (the same result in every workgroup), then writes
// an equal share of the chunk table and the context lists of the clusters m
// with m % gridDim.x == blockIdx.x.  Global reads are issued kPlanPer at a
// time per thread so that their latencies overlap (the loops are
// latency-bound, not bandwidth-bound); the layout offsets go to LDS once.
constexpr int kPlanThreads = 1024;
constexpr int kPlanPer = 8;
constexpr int kPlanGrid = 32;  // workgroups of a batch's plan
__global__ __launch_bounds__(kPlanThreads) void plan_kernel(
    const int32_t* __restrict__ offsets, int M, const int32_t* __restrict__ sel_sorted,
    const int32_t* __restrict__ sel_rowoff, int B, int k, Plan plan) {
    extern __shared__ int32_t pl[];
    int32_t* cnt = pl;            // contexts per cluster, later the list fill counters
    int32_t* loff = pl + M;       // first list entry per cluster
    int32_t* coff = pl + 2 * M;   // first chunk per cluster
    int32_t* offs = pl + 3 * M;   // layout offsets [M + 1]
    __shared__ int tmp[kPlanThreads / kWave + 1];
    const int t = threadIdx.x;
    const int64_t n_sel = (int64_t)B * k;
    // with at most kPlanThreads * kPlanPer selections (every workload) each
    // thread loads its selections and their shortlist offsets once, in the
    // same round trip as the layout offsets, and keeps them in registers
    const bool one_round = n_sel <= (int64_t)kPlanThreads * kPlanPer;
    int mr[kPlanPer], rr[kPlanPer];
    if (one_round) {
#pragma unroll
        for (int q = 0; q < kPlanPer; ++q) {
            const int64_t e = (int64_t)q * kPlanThreads + t;
            mr[q] = e < n_sel ? sel_sorted[e] : -1;
            const uint32_t b = (uint32_t)e / (uint32_t)k, i = (uint32_t)e - b * (uint32_t)k;
            rr[q] = e < n_sel ? sel_rowoff[(size_t)b * (k + 1) + i] : 0;
        }
    }
    for (int m0 = 0; m0 <= M; m0 += kPlanThreads * kPlanPer) {
        int v[kPlanPer];
#pragma unroll
        for (int q = 0; q < kPlanPer; ++q) {
            const int m = m0 + q * kPlanThreads + t;
            v[q] = m <= M ? offsets[m] : 0;
        }
#pragma unroll
        for (int q = 0; q < kPlanPer; ++q) {
            const int m = m0 + q * kPlanThreads + t;
            if (m <= M) offs[m] = v[q];
            if (m < M) cnt[m] = 0;
        }
    }
    __syncthreads();
    if (one_round) {
#pragma unroll
        for (int q = 0; q < kPlanPer; ++q)
            if (mr[q] >= 0 && mr[q] < M) atomicAdd(&cnt[mr[q]], 1);
    } else {
        for (int64_t e0 = 0; e0 < n_sel; e0 += kPlanThreads * kPlanPer) {
            int mv[kPlanPer];
#pragma unroll
            for (int q = 0; q < kPlanPer; ++q) {
                const int64_t e = e0 + q * kPlanThreads + t;
                mv[q] = e < n_sel ? sel_sorted[e] : -1;
            }
#pragma unroll
            for (int q = 0; q < kPlanPer; ++q)
                if (mv[q] >= 0 && mv[q] < M) atomicAdd(&cnt[mv[q]], 1);
        }
    }
    __syncthreads();
    const int per = (M + kPlanThreads - 1) / kPlanThreads;
    const int m0 = min(M, t * per);
    const int m1 = min(M, m0 + per);
    int lc = 0, lch = 0;
    for (int m = m0; m < m1; ++m) {
        lc += cnt[m];
        if (cnt[m] > 0) lch += (offs[m + 1] - offs[m] + kChunkRows - 1) / kChunkRows;
    }
    int n_entries, n_chunks;
    int rl = block_exclusive_scan<kPlanThreads>(lc, tmp, &n_entries);
    int rc = block_exclusive_scan<kPlanThreads>(lch, tmp, &n_chunks);
    for (int m = m0; m < m1; ++m) {
        loff[m] = rl;
        coff[m] = rc;
        rl += cnt[m];
        if (cnt[m] > 0) rc += (offs[m + 1] - offs[m] + kChunkRows - 1) / kChunkRows;
    }
    __syncthreads();
    // chunk descriptors, all threads of all workgroups together: thread gt
    // writes an equal range of chunk indices; one binary search finds the
    // cluster of its first chunk (the last cluster whose first chunk is <= c),
    // then it walks forward
    const int nthr = (int)gridDim.x * kPlanThreads;
    const int gt = (int)blockIdx.x * kPlanThreads + t;
    const int per_c = (n_chunks + nthr - 1) / nthr;
    const int c0 = min(n_chunks, gt * per_c), c1 = min(n_chunks, c0 + per_c);
    if (c0 < c1) {
        int lo = 0, hi = M - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (coff[mid] <= c0) lo = mid; else hi = mid - 1;
        }
        while (lo > 0 && cnt[lo] == 0) --lo;  // equal offsets: the cluster that owns the chunks
        int m = lo;  // cluster 0 may have no contexts (then it owns no chunks)
        int mend = coff[m] + (cnt[m] > 0 ? (offs[m + 1] - offs[m] + kChunkRows - 1) / kChunkRows : 0);
        for (int c = c0; c < c1; ++c) {
            while (c >= mend) {  // next cluster with contexts
                ++m;
                if (cnt[m] > 0) mend = coff[m] + (offs[m + 1] - offs[m] + kChunkRows - 1) / kChunkRows;
            }
            const int ci = c - coff[m];
            const int o = offs[m], n = offs[m + 1] - o;
            plan.chunks[c] = Chunk{o + ci * kChunkRows, min(kChunkRows, n - ci * kChunkRows), loff[m], cnt[m]};
        }
    }
    __syncthreads();
    for (int m = t; m < M; m += kPlanThreads) cnt[m] = 0;
    __syncthreads();
    for (int64_t e0 = 0; e0 < n_sel; e0 += kPlanThreads * kPlanPer) {
        int mv[kPlanPer], ro[kPlanPer];
        if (one_round) {
#pragma unroll
            for (int q = 0; q < kPlanPer; ++q) {
                mv[q] = mr[q];
                ro[q] = rr[q];
            }
        } else {
#pragma unroll
            for (int q = 0; q < kPlanPer; ++q) {
                const int64_t e = e0 + q * kPlanThreads + t;
                mv[q] = e < n_sel ? sel_sorted[e] : -1;
            }
#pragma unroll
            for (int q = 0; q < kPlanPer; ++q) {
                const uint32_t e = (uint32_t)(e0 + q * kPlanThreads + t);  // B * k < 2^31
                const uint32_t b = e / (uint32_t)k, i = e - b * (uint32_t)k;
                ro[q] = (mv[q] >= 0 && mv[q] < M) ? sel_rowoff[(size_t)b * (k + 1) + i] : 0;
            }
        }
        int bq[kPlanPer];
#pragma unroll
        for (int q = 0; q < kPlanPer; ++q) {
            const uint32_t e = (uint32_t)(e0 + q * kPlanThreads + t);  // B * k < 2^31
            bq[q] = (int)(e / (uint32_t)k);
        }
#pragma unroll
        for (int q = 0; q < kPlanPer; ++q) {
            const int m = mv[q];
            // the context list of cluster m is filled by workgroup m % gridDim.x
            if (m < 0 || m >= M || m % (int)gridDim.x != (int)blockIdx.x) continue;
            const int p = atomicAdd(&cnt[m], 1);
            plan.list[loff[m] + p] = ListEntry{bq[q], ro[q] - offs[m]};
        }
    }
    if (t == 0 && blockIdx.x == 0) {
        plan.hdr->n_chunks = n_chunks;
        plan.hdr->n_entries = n_entries;
    }
}

// ------------------------------------------------------------------ union plan
// One workgroup.  The step's rows share one shortlist, the union of their
// selected clusters (Sec. 4.2: several tokens at a step take the union of
// their predicted clusters).  Union clusters are marked in an LDS bitmap and
// compacted in ascending id; each is cut into chunks whose context list is
// every row (entries i * B .. i * B + B - 1 of the list for union cluster i).
// Writes the plan, row_len[b] = |union| for every row, and the union itself
// (ascending ids, -1 past its end) to sel_u[0 .. min(M, B * k)).
// compact: the list holds one entry per union cluster (entry i, context 0)
// and a chunk's count is still B; only the dense union kernel reads this form.
__global__ __launch_bounds__(kPlanThreads) void union_plan_kernel(
    const int32_t* __restrict__ offsets, int M, const int32_t* __restrict__ topk_ids, int B, int k,
    int32_t* __restrict__ row_len, int32_t* __restrict__ sel_u, int u_cap, Plan plan, int compact) {
    extern __shared__ int32_t ul[];
    uint32_t* bits = reinterpret_cast<uint32_t*>(ul);  // [W] cluster bitmap
    const int W = (M + 31) / 32;
    int32_t* wpos = ul + W;                               // [W] union ids before each word
    int32_t* uid = ul + 2 * W;                            // [M] union ids, ascending
    int32_t* coff = uid + M;                              // [M] first chunk of union cluster i
    int32_t* roff = coff + M;                             // [M + 1] first shortlist slot of union cluster i
    __shared__ int tmp[kPlanThreads / kWave + 1];
    const int t = threadIdx.x;
    for (int i = t; i < W; i += kPlanThreads) bits[i] = 0u;
    __syncthreads();
    const int64_t n_sel = (int64_t)B * k;
    for (int64_t e0 = 0; e0 < n_sel; e0 += kPlanThreads * kPlanPer) {
        int mv[kPlanPer];
#pragma unroll
        for (int q = 0; q < kPlanPer; ++q) {
            const int64_t e = e0 + q * kPlanThreads + t;
            mv[q] = e < n_sel ? topk_ids[e] : -1;
        }
#pragma unroll
        for (int q = 0; q < kPlanPer; ++q)
            if (mv[q] >= 0 && mv[q] < M) atomicOr(&bits[mv[q] >> 5], 1u << (mv[q] & 31));
    }
    __syncthreads();
    // compact: word w's set bits take union positions wpos[w] ..
    const int per_w = (W + kPlanThreads - 1) / kPlanThreads;
    const int w0 = min(W, t * per_w), w1 = min(W, w0 + per_w);
    int cnt = 0;
    for (int w = w0; w < w1; ++w) cnt += __popc(bits[w]);
    int U;
    int run = block_exclusive_scan<kPlanThreads>(cnt, tmp, &U);
    for (int w = w0; w < w1; ++w) {
        wpos[w] = run;
        uint32_t x = bits[w];
        while (x) {
            const int bit = __builtin_ctz(x);
            uid[run++] = w * 32 + bit;
            x &= x - 1;
        }
    }
    __syncthreads();
    // union slots and chunks, in ascending id
    const int per_u = (U + kPlanThreads - 1) / kPlanThreads;
    const int i0 = min(U, t * per_u), i1 = min(U, i0 + per_u);
    int lrows = 0, lch = 0;
    for (int i = i0; i < i1; ++i) {
        const int n = offsets[uid[i] + 1] - offsets[uid[i]];
        lrows += n;
        lch += (n + kChunkRows - 1) / kChunkRows;
    }
    int len, n_chunks;
    int rr = block_exclusive_scan<kPlanThreads>(lrows, tmp, &len);
    int rc = block_exclusive_scan<kPlanThreads>(lch, tmp, &n_chunks);
    for (int i = i0; i < i1; ++i) {
        const int n = offsets[uid[i] + 1] - offsets[uid[i]];
        roff[i] = rr;
        coff[i] = rc;
        rr += n;
        rc += (n + kChunkRows - 1) / kChunkRows;
    }
    __syncthreads();
    // chunks: equal ranges per thread, one binary search, then a forward walk
    const int per_c = (n_chunks + kPlanThreads - 1) / kPlanThreads;
    const int c0 = min(n_chunks, t * per_c), c1 = min(n_chunks, c0 + per_c);
    if (c0 < c1) {
        int lo = 0, hi = U - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (coff[mid] <= c0) lo = mid; else hi = mid - 1;
        }
        int i = lo;
        for (int c = c0; c < c1; ++c) {
            while (i + 1 < U && coff[i + 1] <= c) ++i;
            const int m = uid[i];
            const int ci = c - coff[i];
            const int o = offsets[m], n = offsets[m + 1] - o;
            plan.chunks[c] = Chunk{o + ci * kChunkRows, min(kChunkRows, n - ci * kChunkRows), compact ? i : i * B, B};
        }
    }
    // every row in every union cluster's list (compact: row 0 stands for all)
    const int per = compact ? 1 : B;
    for (int64_t e = t; e < (int64_t)U * per; e += kPlanThreads) {
        const int i = (int)(e / per), b = (int)(e - (int64_t)i * per);
        plan.list[e] = ListEntry{b, roff[i] - offsets[uid[i]]};
    }
    for (int b = t; b < B; b += kPlanThreads) row_len[b] = len;
    for (int i = t; i < u_cap; i += kPlanThreads) sel_u[i] = i < U ? uid[i] : -1;
    if (t == 0) {
        plan.hdr->n_chunks = n_chunks;
        plan.hdr->n_entries = U * per;
    }
}

// ------------------------------------------------------------------ beam expansion
// One workgroup: the n_out best cumulative scores cu[b, r] = logprobs[b, r] +
// last[b] among the B x k_t candidates with a token (Algorithm 1's
// cu_scores and TopK_{k_t}), ordered (cu desc, b asc, r asc) by the key
// (ordered cu << 32) | ~(b * k_t + r).
constexpr int kBeamPer = 8;
constexpr int kBeamSmall = 256;  // candidates up to which one counting pass ranks them
__global__ __launch_bounds__(kRowThreads) void beam_expand_kernel(const float* __restrict__ logprobs,
                                                                  const int32_t* __restrict__ ids,
                                                                  const float* __restrict__ last, int B, int k_t,
                                                                  int n_out, float* out_scores, int32_t* out_parent,
                                                                  int32_t* out_ids) {
    __shared__ int hist[256];
    __shared__ uint64_t sel[DYNA_MAX_KT], top[DYNA_MAX_KT];
    const int n = B * k_t;
    if (n <= kBeamSmall) {  // uniform: a beam of a few rows, ranked by counting
        __shared__ uint64_t ks[kBeamSmall];
        __shared__ int s_nv;
        const int t = threadIdx.x;
        uint64_t key = 0;
        if (t < n && ids[t] >= 0) {
            const float cu = canon(logprobs[t]) + (last ? last[t / k_t] : 0.0f);
            key = sel_key(canon(cu), (uint32_t)t);
        }
        if (t < kBeamSmall) ks[t] = key;
        if (t == 0) s_nv = 0;
        __syncthreads();
        if (t < kBeamSmall) {
            const int nv = __popcll(__ballot(key != 0));
            if (lane_id() == 0 && nv) atomicAdd(&s_nv, nv);
        }
        if (key != 0) {
            // keys are distinct (they carry the candidate's index): the rank
            // is the number of larger keys
            int rank = 0;
            for (int j = 0; j < n; ++j) rank += ks[j] > key;
            if (rank < n_out) {
                out_scores[rank] = key_val(key);
                out_parent[rank] = t / k_t;
                out_ids[rank] = ids[t];
            }
        }
        __syncthreads();
        for (int r = s_nv + t; r < n_out; r += kRowThreads) {
            out_scores[r] = -__builtin_inff();
            out_parent[r] = -1;
            out_ids[r] = -1;
        }
        return;
    }
    uint64_t kk[kBeamPer];
    int n_valid = 0;
#pragma unroll
    for (int q = 0; q < kBeamPer; ++q) {
        const int e = q * kRowThreads + threadIdx.x;
        kk[q] = 0;
        if (e < n && ids[e] >= 0) {
            const int b = e / k_t;
            const float cu = canon(logprobs[e]) + (last ? last[b] : 0.0f);
            kk[q] = sel_key(canon(cu), (uint32_t)e);
            ++n_valid;
        }
    }
    __shared__ int sh_valid;
    if (threadIdx.x == 0) sh_valid = 0;
    __syncthreads();
    atomicAdd(&sh_valid, n_valid);
    __syncthreads();
    block_radix_topk<kRowThreads, kBeamPer>(kk, n_out, sh_valid, hist, sel, top);
    for (int r = threadIdx.x; r < n_out; r += kRowThreads) {
        const uint64_t key = top[r];
        if (key == 0) {
            out_scores[r] = -__builtin_inff();
            out_parent[r] = -1;
            out_ids[r] = -1;
        } else {
            const int e = (int)key_id(key);
            out_scores[r] = key_val(key);
            out_parent[r] = e / k_t;
            out_ids[r] = ids[e];
        }
    }
}

// ------------------------------------------------------------------ select
template <int kPer>
__global__ __launch_bounds__(kNT) void select_partial_kernel(SelectArgs a) {
    constexpr int kSegLen = kPer * kNT;
    __shared__ uint64_t top[DYNA_MAX_KT];
    __shared__ float red[kNT / kWave];
    const int p = blockIdx.x, b = blockIdx.y;
    const int len = a.row_len ? a.row_len[b] : a.fixed_len;
    const int seg0 = p * kSegLen;
    if (seg0 >= len) {  // past the row: an empty partial
        const int64_t pb = (int64_t)b * a.P + p;
        if (threadIdx.x == 0) {
            a.pmax[pb] = -__builtin_inff();
            a.psum[pb] = 0.0f;
        }
        for (int r = threadIdx.x; r < a.k_t; r += kNT) a.pkeys[pb * a.k_t + r] = 0;
        return;
    }
    const int j0 = seg0 + threadIdx.x * kPer;
    const int n = max(0, min(kPer, len - j0));
    const float* z = a.logits + (int64_t)b * a.ld;

    uint32_t vid[kPer];
    float zv[kPer];
    uint64_t list[kPer];
    if (n > 0) slot_vids(a, b, j0, n, vid);
    float zr[kPer];  // in-bounds loads (clamped to the row), issued together
#pragma unroll
    for (int q = 0; q < kPer; ++q) zr[q] = z[min(j0 + q, len - 1)];
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        zv[q] = q < n ? canon(zr[q]) : -__builtin_inff();
        list[q] = q < n ? sel_key(zv[q], vid[q]) : 0;
    }
    // the segment's k_t best keys by radix selection (measured faster than
    // per-thread sorted lists merged in k_t wave rounds: 4 us per union step
    // of 64 rows, 3.5 us per dense head)
    {
        __shared__ int rhist[256];
        __shared__ uint64_t rsel[DYNA_MAX_KT];
        block_radix_topk<kNT, kPer>(list, a.k_t, min(kSegLen, len - seg0), rhist, rsel, top);
    }
    // segment max = value of the best key (or -inf for an empty segment)
    const float smax = top[0] != 0 ? key_val(top[0]) : -__builtin_inff();
    float tsum = 0.0f;
    if (smax != -__builtin_inff()) {
#pragma unroll
        for (int q = 0; q < kPer; ++q)
            if (q < n) tsum += expf((zv[q] - smax) * a.inv_t);
    }
    tsum = wave_sum(tsum);
    if (lane_id() == 0) red[threadIdx.x / kWave] = tsum;
    __syncthreads();
    const int64_t pb = (int64_t)b * a.P + p;
    if (threadIdx.x == 0) {
        float ssum = 0.0f;
#pragma unroll
        for (int q = 0; q < kNT / kWave; ++q) ssum += red[q];
        a.pmax[pb] = smax;
        a.psum[pb] = ssum;
    }
    for (int r = threadIdx.x; r < a.k_t; r += kNT) a.pkeys[pb * a.k_t + r] = top[r];
}

template <int kPer>
__global__ __launch_bounds__(kNT) void select_final_kernel(SelectArgs a) {
    constexpr int kSegLen = kPer * kNT;
    __shared__ uint64_t wmax[8];
    __shared__ uint64_t top[DYNA_MAX_KT];
    __shared__ float sh_target, sh_base;
    __shared__ int sh_seg;
    __shared__ float red[2 * (kNT / kWave) + 1];
    __shared__ float wred[kNT / kWave];
    __shared__ int sh_pick;
    __shared__ float incl_s[kNT];
    const int b = blockIdx.x;
    const int P = a.P;
    const int len = a.row_len ? a.row_len[b] : a.fixed_len;
    const int64_t pb0 = (int64_t)b * P;

    // thread p < P holds segment p's (max, sum); the row max is a block max and
    // the segment masses c_p = sum_p * exp((max_p - max) / T) are block-scanned
    // in segment order (P <= 256 is guaranteed by the host)
    const int lane = lane_id(), w = threadIdx.x / kWave;
    const float my_m = (int)threadIdx.x < P ? a.pmax[pb0 + threadIdx.x] : -__builtin_inff();
    const float my_s = (int)threadIdx.x < P ? a.psum[pb0 + threadIdx.x] : 0.0f;
    {
        const float m = readlane_f32(wave_max_f32(my_m), kWave - 1);
        if (lane == 0) wred[w] = m;
    }
    __syncthreads();
    float mx = wred[0];
#pragma unroll
    for (int q = 1; q < kNT / kWave; ++q) mx = fmaxf(mx, wred[q]);
    const float my_c =
        (mx != -__builtin_inff() && my_m != -__builtin_inff()) ? my_s * expf((my_m - mx) * a.inv_t) : 0.0f;
    float total;
    const float my_incl = block_inclusive_scan_f32<kNT>(my_c, red, &total);
    // merge the per-segment lists: thread t walks the list of segment t
    // (P <= 256 is guaranteed by the host)
    uint64_t list[1];
    int head = 0;
    const uint64_t* mylist = a.pkeys + (pb0 + threadIdx.x) * a.k_t;
    list[0] = (int)threadIdx.x < P ? mylist[0] : 0;
    {
        for (int r = 0; r < a.k_t; ++r) {
            const uint64_t m = wave_max_u64(list[0]);
            if (lane == 0) wmax[(r & 1) * 4 + w] = m;
            __syncthreads();
            uint64_t best = wmax[(r & 1) * 4];
#pragma unroll
            for (int q = 1; q < kNT / kWave; ++q) best = max(best, wmax[(r & 1) * 4 + q]);
            if (best != 0 && list[0] == best) {
                ++head;
                list[0] = head < a.k_t ? mylist[head] : 0;
            }
            if (threadIdx.x == 0) top[r] = best;
        }
    }
    __syncthreads();
    const TailMix tail = tail_of(a, len);
    const float log_total = logf(total) - tail.lshift;
    if (a.out_ids != nullptr) {
        for (int r = threadIdx.x; r < a.k_t; r += kNT) {
            const uint64_t key = top[r];
            a.out_ids[(int64_t)b * a.k_t + r] = key != 0 ? (int32_t)key_id(key) : -1;
            if (a.out_logprobs)
                a.out_logprobs[(int64_t)b * a.k_t + r] =
                    key != 0 ? (key_val(key) - mx) * a.inv_t - log_total : -__builtin_inff();
        }
    }
    if (a.uniforms == nullptr || a.out_sample == nullptr) return;
    float u_s;
    if (tail_sample(a, b, tail, &u_s)) return;  // uniform decision for the block

    // inverse CDF: the segment whose running mass range holds u * total (the
    // first with mass past it), else the last segment with mass
    const float u_target = u_s * total;
    const float my_excl = my_incl - my_c;
    if (threadIdx.x == 0) {
        sh_seg = -1;
        sh_pick = -1;
        sh_target = u_target;
    }
    __syncthreads();
    if (my_c > 0.0f && my_excl <= u_target && u_target < my_incl) atomicMax(&sh_seg, (int)threadIdx.x);
    __syncthreads();
    const int seg_found = sh_seg;
    __syncthreads();
    if (seg_found < 0 && my_c > 0.0f) atomicMax(&sh_seg, (int)threadIdx.x);
    __syncthreads();
    if ((int)threadIdx.x == sh_seg) sh_base = my_excl;
    __syncthreads();
    const int seg = sh_seg;
    if (seg < 0) {  // empty shortlist
        if (threadIdx.x == 0) {
            a.out_sample[b] = -1;
            if (a.out_sample_logprob) a.out_sample_logprob[b] = -__builtin_inff();
        }
        return;
    }
    const float* z = a.logits + (int64_t)b * a.ld;
    const int j0 = seg * kSegLen + threadIdx.x * kPer;
    const int n = max(0, min(kPer, len - j0));
    float e[kPer];
    float tsum = 0.0f;
#pragma unroll
    for (int q = 0; q < kPer; ++q) e[q] = z[min(j0 + q, len - 1)];  // in-bounds, issued together
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        e[q] = q < n ? expf((canon(e[q]) - mx) * a.inv_t) : 0.0f;
        tsum += e[q];
    }
    float blk_total;
    const float incl = block_inclusive_scan_f32<kNT>(tsum, red, &blk_total);
    incl_s[threadIdx.x] = incl;
    __syncthreads();
    const float excl = threadIdx.x > 0 ? incl_s[threadIdx.x - 1] : 0.0f;
    const float target = sh_target - sh_base;
    // the thread whose running range holds the target picks inside its slots
    if (tsum > 0.0f && excl <= target && target < incl) {
        float acc = excl;
        int pick = -1, last = -1;
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            if (e[q] > 0.0f) last = q;
            acc += e[q];
            if (pick < 0 && e[q] > 0.0f && acc > target) pick = q;
        }
        atomicMax(&sh_pick, j0 + (pick >= 0 ? pick : last));
    }
    __syncthreads();
    if (sh_pick < 0) {  // rounding left the target at or past the segment mass: last slot with mass
        int last = -1;
#pragma unroll
        for (int q = 0; q < kPer; ++q)
            if (e[q] > 0.0f) last = j0 + q;
        if (last >= 0) atomicMax(&sh_pick, last);
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const int j = sh_pick;
        uint32_t vid[1];
        slot_vids(a, b, j, 1, vid);
        a.out_sample[b] = (int32_t)vid[0];
        if (a.out_sample_logprob) a.out_sample_logprob[b] = (canon(z[j]) - mx) * a.inv_t - log_total;
    }
}

template <int KT>
__global__ __launch_bounds__(kRowThreads) void select_row_kernel(SelectArgs a) {
    select_row<KT, kRowThreads>(a, blockIdx.x);
}

}  // namespace

// Dynamic LDS above 64 KB must be allowed per kernel and device before a
// launch; the allowance only ever grows, so launches of every size fit.
static dyna_status allow_topk_lds(size_t lds) {
    if (lds <= 65536) return DYNA_OK;
    static std::mutex mu;
    static size_t allowed[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return set_error(DYNA_ERR_HIP, "top-k: device");
    std::lock_guard<std::mutex> g(mu);
    if (allowed[dev] >= lds) return DYNA_OK;
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(topk_clusters_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
        return set_error(DYNA_ERR_UNSUPPORTED, "top-k needs %zu bytes of LDS", lds);
    allowed[dev] = lds;
    return DYNA_OK;
}

dyna_status launch_topk_clusters(const float* scores, int32_t B, int32_t M, int32_t k,
                                 int32_t* topk_ids, float* topk_scores, const int32_t* offsets,
                                 int32_t* sel_sorted, int32_t* sel_rowoff, int32_t* row_len,
                                 const Plan* plan, hipStream_t stream, const ScoreSlices& slices) {
    const size_t lds = topk_lds_bytes(M, k);
    if (dyna_status st = allow_topk_lds(lds); st != DYNA_OK) return st;
    Plan p{};
    if (plan != nullptr && B == 1) p = *plan;
    TopkArgs A{scores, slices.part, slices.slices, slices.bias, M, k, topk_ids, topk_scores, offsets,
               sel_sorted, sel_rowoff, row_len, p};
    topk_clusters_kernel<<<B, kNT, lds, stream>>>(A);
    return check_launch("topk_clusters_kernel");
}

dyna_status launch_shortlist(const int32_t* offsets, const int32_t* perm, int32_t M,
                             const int32_t* topk_ids, int32_t B, int32_t k, int32_t* sel_sorted,
                             int32_t* sel_rowoff, int32_t* row_len, int32_t* shortlist_ids,
                             int32_t cap, hipStream_t stream) {
    const size_t lds = sizeof(int32_t) * (3 * (size_t)k + 1);
    shortlist_kernel<<<B, kNT, lds, stream>>>(offsets, perm, M, topk_ids, k, sel_sorted, sel_rowoff,
                                              row_len, shortlist_ids, cap);
    return check_launch("shortlist_kernel");
}

dyna_status launch_plan(const int32_t* offsets, int32_t M, const int32_t* sel_sorted,
                        const int32_t* sel_rowoff, int32_t B, int32_t k, Plan plan,
                        hipStream_t stream) {
    const size_t lds = sizeof(int32_t) * (4 * (size_t)M + 1);
    if (lds > 64 * 1024) {
        // above 64 KiB the dynamic LDS size must be allowed, once per device
        static std::atomic<uint64_t> allowed{0};
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return set_error(DYNA_ERR_HIP, "plan: device");
        if (!(allowed.load() & (1ull << dev))) {
            if (hipFuncSetAttribute((const void*)plan_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                    (int)(sizeof(int32_t) * (4 * (size_t)DYNA_MAX_M + 1))) != hipSuccess)
                return set_error(DYNA_ERR_HIP, "plan: LDS attribute");
            allowed.fetch_or(1ull << dev);
        }
    }
    // every workgroup builds the counts and offsets itself (cheap next to a
    // hand-off between workgroups), then writes its share of the chunk table
    // and the context lists of its clusters; with one context the plan is
    // small and one workgroup does it
    const int64_t n_sel = (int64_t)B * k;
    const int grid = n_sel <= 64 ? 1 : (int)std::min<int64_t>(kPlanGrid, std::max<int64_t>(1, n_sel / 64));
    plan_kernel<<<grid, kPlanThreads, lds, stream>>>(offsets, M, sel_sorted, sel_rowoff, B, k, plan);
    return check_launch("plan_kernel");
}

dyna_status launch_union_plan(const int32_t* offsets, int32_t M, const int32_t* topk_ids, int32_t B, int32_t k,
                              int32_t* row_len, int32_t* sel_u, int32_t u_cap, Plan plan, bool compact,
                              hipStream_t stream) {
    const size_t lds = sizeof(int32_t) * (2 * (size_t)((M + 31) / 32) + 3 * (size_t)M + 1);
    if (lds > 64 * 1024) {
        static std::atomic<uint64_t> allowed{0};
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return set_error(DYNA_ERR_HIP, "union: device");
        if (!(allowed.load() & (1ull << dev))) {
            const int most = (int)(sizeof(int32_t) * (2 * (size_t)((DYNA_MAX_M + 31) / 32) + 3 * (size_t)DYNA_MAX_M + 1));
            if (hipFuncSetAttribute((const void*)union_plan_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, most) !=
                hipSuccess)
                return set_error(DYNA_ERR_HIP, "union: LDS attribute");
            allowed.fetch_or(1ull << dev);
        }
    }
    union_plan_kernel<<<1, kPlanThreads, lds, stream>>>(offsets, M, topk_ids, B, k, row_len, sel_u, u_cap, plan,
                                                        compact ? 1 : 0);
    return check_launch("union_plan_kernel");
}

dyna_status launch_beam_expand(const float* logprobs, const int32_t* ids, const float* last, int32_t B, int32_t k_t,
                               int32_t n_out, float* out_scores, int32_t* out_parent, int32_t* out_ids,
                               hipStream_t stream) {
    if ((int64_t)B * k_t > (int64_t)kRowThreads * kBeamPer)
        return set_error(DYNA_ERR_UNSUPPORTED, "beam expansion: B * k_t = %lld > %d", (long long)B * k_t,
                         kRowThreads * kBeamPer);
    beam_expand_kernel<<<1, kRowThreads, 0, stream>>>(logprobs, ids, last, B, k_t, n_out, out_scores, out_parent,
                                                     out_ids);
    return check_launch("beam_expand_kernel");
}

// Segment length of the long-row selection for rows of up to max_len slots.
// The short segments measured faster wherever they fit: 64 union rows of
// 109k slots 248.6 -> 240.4 us per step, ten union rows of 31.6k slots about
// 1.5 us less, the drafting cycle with a fixed budget of 32 clusters 505 ->
// 497 us.
static int32_t select_seg(int32_t max_len) { return max_len <= kSegShort * kNT ? kSegShort : kSeg; }

size_t select_ws_bytes(int32_t B, int32_t max_len, int32_t k_t) {
    const int32_t seg = select_seg(max_len);
    const int64_t P = std::max<int64_t>(1, ((int64_t)max_len + seg - 1) / seg);
    return (size_t)B * P * ((size_t)k_t * sizeof(uint64_t) + 2 * sizeof(float)) + 512;
}

int32_t select_max_len() { return kSeg * kNT; }

SelectArgs make_select_args(const float* logits, int64_t ld, const int32_t* row_len,
                            int32_t fixed_len, int32_t max_len, const int32_t* sel_sorted,
                            const int32_t* sel_rowoff, const int32_t* offsets,
                            const int32_t* perm, int32_t B, int32_t k, int32_t k_t,
                            float temperature, float beta, int32_t V, const float* uniforms, int32_t* out_ids,
                            float* out_logprobs, int32_t* out_sample,
                            float* out_sample_logprob, void* ws, const int32_t* slot_vid, int64_t vid_ld) {
    SelectArgs a;
    a.logits = logits;
    a.ld = ld;
    a.row_len = row_len;
    a.fixed_len = fixed_len;
    a.sel_sorted = sel_sorted;
    a.sel_rowoff = sel_rowoff;
    a.offsets = offsets;
    a.perm = perm;
    a.slot_vid = slot_vid;
    a.vid_ld = vid_ld < 0 ? ld : vid_ld;
    a.k = k;
    a.k_t = k_t;
    a.inv_t = 1.0f / temperature;
    a.uniforms = uniforms;
    a.beta = beta;
    a.V = V;
    const int32_t seg = select_seg(max_len);
    a.seg = seg;
    a.P = (int32_t)std::max<int64_t>(1, ((int64_t)max_len + seg - 1) / seg);
    char* p = static_cast<char*>(ws);
    a.pkeys = reinterpret_cast<uint64_t*>(p);
    p += (size_t)B * a.P * k_t * sizeof(uint64_t);
    a.pmax = reinterpret_cast<float*>(p);
    p += (size_t)B * a.P * sizeof(float);
    a.psum = reinterpret_cast<float*>(p);
    a.out_ids = out_ids;
    a.out_logprobs = out_logprobs;
    a.out_sample = out_sample;
    a.out_sample_logprob = out_sample_logprob;
    return a;
}

bool select_row_fits(int32_t max_len, bool fixed, int32_t k_t, int32_t k) {
    // full-vocabulary rows (fixed length) spread over many workgroups beyond 8192
    return max_len <= (fixed ? 8192 : kRowMax) && k_t <= 16 && (fixed || k <= kRowTable);
}

dyna_status launch_select(const float* logits, int64_t ld, const int32_t* row_len,
                          int32_t fixed_len, int32_t max_len, const int32_t* sel_sorted,
                          const int32_t* sel_rowoff, const int32_t* offsets, const int32_t* perm,
                          int32_t B, int32_t k, int32_t k_t, float temperature, float beta, int32_t V,
                          const float* uniforms, int32_t* out_ids, float* out_logprobs,
                          int32_t* out_sample, float* out_sample_logprob, void* ws,
                          hipStream_t stream, const int32_t* slot_vid, int64_t vid_ld, bool split_long) {
    const SelectArgs a = make_select_args(logits, ld, row_len, fixed_len, max_len, sel_sorted,
                                          sel_rowoff, offsets, perm, B, k, k_t, temperature, beta, V,
                                          uniforms, out_ids, out_logprobs, out_sample,
                                          out_sample_logprob, ws, slot_vid, vid_ld);
    // shortlist-sized rows: one workgroup per row, one launch
    const bool split = split_long && max_len > kRowSplit;
    if (!split && select_row_fits(max_len, row_len == nullptr, k_t, perm == nullptr ? 0 : k)) {
        if (k_t == 1) select_row_kernel<1><<<B, kRowThreads, 0, stream>>>(a);
        else select_row_kernel<16><<<B, kRowThreads, 0, stream>>>(a);
        return check_launch("select_row_kernel");
    }
    if (a.seg == kSegShort) {
        select_partial_kernel<kSegShort / kNT><<<dim3(a.P, B), kNT, 0, stream>>>(a);
        if (dyna_status s = check_launch("select_partial_kernel"); s != DYNA_OK) return s;
        select_final_kernel<kSegShort / kNT><<<B, kNT, 0, stream>>>(a);
    } else {
        select_partial_kernel<kSeg / kNT><<<dim3(a.P, B), kNT, 0, stream>>>(a);
        if (dyna_status s = check_launch("select_partial_kernel"); s != DYNA_OK) return s;
        select_final_kernel<kSeg / kNT><<<B, kNT, 0, stream>>>(a);
    }
    return check_launch("select_final_kernel");
}

}  // namespace dyna
