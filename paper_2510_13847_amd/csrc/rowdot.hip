// Row-dot kernels: out[b, base_b + row] = act(W[row, :] . v[b, :] + bias[row]).
//
// The same two kernels serve the router layers (every row of W against every
// context, Sec. 4.2 "Low-cost router") and the gathered head (only the rows of
// the selected cluster slabs, each against the contexts that selected that
// cluster: Sec. 4.3, the gathered LM head / FUSED_INDEX_GEMM of Algorithm 1).
//
//  * rowdot_gemv_kernel: one wave per W row.  Each lane streams 16-byte pieces
//    of the row (a wave covers 1 KiB of one row per load), keeps the row in
//    registers and dots it with each context that needs it; a butterfly sum
//    finishes each dot product.  Chosen for few contexts (B <= 4), where the
//    kernel is a pure HBM stream.
//  * rowdot_mfma_kernel: one wave per tile of 16 W rows; contexts are the 16
//    columns of v_mfma_f32_16x16x32_bf16 (G column groups per pass).  Chosen
//    for tree and serving batches, where one slab row feeds many contexts.
//    An fp32 right operand (the router's hidden layer) is split into two bf16
//    terms hi + lo, so the product keeps ~16 significant bits of it.
//
// W rows are read with non-temporal loads (each row is touched once per call);
// v rows are small and re-read from cache.  All sums have a fixed order, so
// results are bit-identical from run to run.
#include "gemv.h"

namespace dyna {
namespace {

// ------------------------------------------------------------------ GEMV
template <typename WT, typename VT, int NB, bool PLAN, int R, bool SINGLE>
__global__ __launch_bounds__(kThreads) void rowdot_gemv_kernel(RowdotArgs a) {
    if (a.zero_words != nullptr && blockIdx.x == 0 && (int)threadIdx.x < a.n_zero_words)
        a.zero_words[threadIdx.x] = 0;
    StoreEpi<PLAN> epi;
    gemv_rows<WT, VT, NB, PLAN, R, SINGLE>(a, epi);
}

// ------------------------------------------------------------------ MFMA
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 u) { return __builtin_bit_cast(bf16x8, u); }

// One item = T tiles of 16 W rows (T * 16 consecutive rows) against the
// contexts of the item, G groups of 16 contexts at a time: every B-operand
// load feeds T MFMAs and every A-operand load feeds G.  KS > 1 splits the
// k steps over the KS waves of a block (reduced through LDS in a fixed
// order); KS = 1 lets every wave take its own items.  U k-steps are loaded
// before their MFMAs are issued.
template <int T, int G, bool VF32, bool PLAN, int KS, int U>
__global__ __launch_bounds__(KS > 1 ? KS * kWave : kThreads) void rowdot_mfma_kernel(RowdotArgs a) {
    constexpr int NW = KS > 1 ? KS : kWavesPerBlock;  // waves per block
    constexpr int kItemRows = T * kMfmaRows;
    __shared__ float red[KS > 1 ? (KS - 1) * T * G * 4 * kWave : 1];
    if (a.zero_words != nullptr && blockIdx.x == 0 && (int)threadIdx.x < a.n_zero_words)
        a.zero_words[threadIdx.x] = 0;
    const int lane = lane_id();
    const int wv = threadIdx.x / kWave;
    const int col = lane & 15;   // A row inside a tile, and B / D column
    const int kq = lane >> 4;    // 8-element slice of each 32-wide k step
    const int K = a.K;
    const int nsteps = (K + 31) / 32;
    const uint16_t* __restrict__ W = static_cast<const uint16_t*>(a.W);

    // plan mode: a chunk of up to 64 rows gives 64 / kItemRows wave items
    constexpr int kSub = kChunkRows / kItemRows;
    const int64_t n_items = PLAN ? (int64_t)a.plan.hdr->n_chunks * kSub
                                 : ((int64_t)a.n_rows + kItemRows - 1) / kItemRows;
    const int64_t item0 = KS == 1 ? (int64_t)blockIdx.x * NW + wv : blockIdx.x;
    const int64_t istride = KS == 1 ? (int64_t)gridDim.x * NW : gridDim.x;
    const int s_begin = KS == 1 ? 0 : (wv * nsteps) / KS;
    const int s_end = KS == 1 ? nsteps : ((wv + 1) * nsteps) / KS;

    for (int64_t it = item0; it < n_items; it += istride) {
        int r0, nrows, lcnt;
        const ListEntry* list = nullptr;
        if constexpr (PLAN) {
            const Chunk c = a.plan.chunks[it / kSub];
            const int sub = (int)(it % kSub) * kItemRows;
            if (sub >= c.nrows) continue;  // wave-uniform
            r0 = c.r0 + sub;
            nrows = min(kItemRows, c.nrows - sub);
            lcnt = c.list_cnt;
            list = a.plan.list + c.list_off;
        } else {
            r0 = (int)(it * kItemRows);
            nrows = min(kItemRows, a.n_rows - r0);
            lcnt = a.B;
        }
        // rows past nrows (and contexts past lcnt) read a valid row whose
        // results are never stored, so every load below is unconditional
        const uint16_t* wrow[T];
#pragma unroll
        for (int t = 0; t < T; ++t) {
            const bool rvalid = t * kMfmaRows + col < nrows;
            wrow[t] = W + (int64_t)(r0 + (rvalid ? t * kMfmaRows + col : 0)) * K;
        }
        const int tiles = (nrows + kMfmaRows - 1) / kMfmaRows;  // wave-uniform

        for (int gb = 0; gb < lcnt; gb += 16 * G) {
            int cb[G], cbase[G];
            bool cvalid[G];
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const int e = gb + g * 16 + col;
                cvalid[g] = e < lcnt;
                if constexpr (PLAN) {
                    const ListEntry le = list[cvalid[g] ? e : 0];
                    cb[g] = le.b;
                    cbase[g] = le.slot_base;
                } else {
                    cb[g] = cvalid[g] ? e : 0;
                    cbase[g] = 0;
                }
            }
            f32x4 acc[T][G];
#pragma unroll
            for (int t = 0; t < T; ++t)
#pragma unroll
                for (int g = 0; g < G; ++g) acc[t][g] = f32x4{0.f, 0.f, 0.f, 0.f};

            for (int s = s_begin; s < s_end; s += U) {
                u32x4 A[U][T];
                u32x4 Bh[U][G];
                u32x4 Bl[U][VF32 ? G : 1];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    // k steps past the range (or the k tail) load element 0 and
                    // are zeroed, so they add nothing
                    const int k = (s + u) * 32 + kq * 8;
                    const bool kv = (s + u) < s_end && k < K;
                    const int ko = kv ? k : 0;
#pragma unroll
                    for (int t = 0; t < T; ++t) {
                        const u32x4 x = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wrow[t] + ko));
                        A[u][t] = kv ? x : u32x4{0u, 0u, 0u, 0u};
                    }
#pragma unroll
                    for (int g = 0; g < G; ++g) {
                        // context columns are often sparse (a few contexts per
                        // cluster): only valid columns load
                        Bh[u][g] = u32x4{0u, 0u, 0u, 0u};
                        if constexpr (VF32) Bl[u][g] = u32x4{0u, 0u, 0u, 0u};
                        if (cvalid[g] && kv) {
                            if constexpr (VF32) {
                                split8(static_cast<const float*>(a.v) + (int64_t)cb[g] * K + k, Bh[u][g],
                                       Bl[u][g]);
                            } else {
                                Bh[u][g] = *reinterpret_cast<const u32x4*>(
                                    static_cast<const uint16_t*>(a.v) + (int64_t)cb[g] * K + k);
                            }
                        }
                    }
                }
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int t = 0; t < T; ++t) {
                        if (t >= tiles) continue;  // wave-uniform
#pragma unroll
                        for (int g = 0; g < G; ++g) {
                            if (gb + g * 16 >= lcnt) continue;  // wave-uniform
                            acc[t][g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                as_bf16x8(A[u][t]), as_bf16x8(Bh[u][g]), acc[t][g], 0, 0, 0);
                            if constexpr (VF32)
                                acc[t][g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                    as_bf16x8(A[u][t]), as_bf16x8(Bl[u][g]), acc[t][g], 0, 0, 0);
                        }
                    }
            }

            if constexpr (KS > 1) {
                if (wv > 0) {
#pragma unroll
                    for (int t = 0; t < T; ++t)
#pragma unroll
                        for (int g = 0; g < G; ++g)
#pragma unroll
                            for (int r = 0; r < 4; ++r)
                                red[((((wv - 1) * T + t) * G + g) * 4 + r) * kWave + lane] = acc[t][g][r];
                }
                __syncthreads();
                if (wv == 0) {
#pragma unroll
                    for (int w = 1; w < KS; ++w)
#pragma unroll
                        for (int t = 0; t < T; ++t)
#pragma unroll
                            for (int g = 0; g < G; ++g)
#pragma unroll
                                for (int r = 0; r < 4; ++r)
                                    acc[t][g][r] += red[((((w - 1) * T + t) * G + g) * 4 + r) * kWave + lane];
                }
                __syncthreads();
                if (wv != 0) continue;
            }

#pragma unroll
            for (int g = 0; g < G; ++g) {
                if (!cvalid[g]) continue;
                float* o = a.out + (int64_t)cb[g] * a.ld + cbase[g] + r0;
#pragma unroll
                for (int t = 0; t < T; ++t)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int i = t * kMfmaRows + kq * 4 + r;
                        if (i < nrows) {
                            const float bias = a.bias ? a.bias[r0 + i] : 0.0f;
                            o[i] = apply_act(acc[t][g][r] + bias, a.act);
                            if constexpr (PLAN) {
                                if (a.vid_out) a.vid_out[(o - a.out) + i] = a.perm[r0 + i];
                            }
                        }
                    }
            }
        }
    }
}

int resident_blocks() { return 256 * 8; }  // 256 CUs x 8 blocks of 4 waves

// Rows in flight per wave: up to 4 where the registers allow it (a
// 4096-wide bf16 row takes 32 VGPRs raw), fewer for long or fp32 rows.
template <typename WT, int NB>
constexpr int gemv_max_rows() {
    return (sizeof(WT) == 2 ? NB : 2 * NB) <= 8 ? 4 : ((sizeof(WT) == 2 ? NB : 2 * NB) <= 16 ? 2 : 1);
}

template <typename WT, typename VT, bool PLAN, int NB, int R>
dyna_status launch_gemv_r(const RowdotArgs& a, bool single, hipStream_t stream) {
    const int64_t items = PLAN ? (int64_t)a.max_chunks_bound * (kChunkRows / R)
                               : ((int64_t)a.n_rows + R - 1) / R;
    int64_t blocks = std::max<int64_t>(
        1, std::min<int64_t>((items + kWavesPerBlock - 1) / kWavesPerBlock, 4096));
    if (single)
        launch_timed_kernel(rowdot_gemv_kernel<WT, VT, NB, PLAN, R, true>, dim3((unsigned)blocks),
                            dim3(kThreads), 0, stream, a);
    else
        launch_timed_kernel(rowdot_gemv_kernel<WT, VT, NB, PLAN, R, false>, dim3((unsigned)blocks),
                            dim3(kThreads), 0, stream, a);
    return check_launch("rowdot_gemv_kernel");
}

template <typename WT, typename VT, bool PLAN, int NB>
dyna_status launch_gemv_t(const RowdotArgs& a, bool single, int rows_opt, hipStream_t stream) {
    constexpr int RMAX = gemv_max_rows<WT, NB>();
    int R = rows_opt > 0 ? std::min(rows_opt, RMAX) : RMAX;
    // a small dense matrix (a router layer) spreads one row per wave so that
    // every CU takes part
    if (rows_opt == 0 && !PLAN && (int64_t)a.n_rows < 4 * 256 * 16) R = 1;
    if (R >= 4 && RMAX >= 4) return launch_gemv_r<WT, VT, PLAN, NB, (RMAX >= 4 ? 4 : 1)>(a, single, stream);
    if (R >= 2 && RMAX >= 2) return launch_gemv_r<WT, VT, PLAN, NB, (RMAX >= 2 ? 2 : 1)>(a, single, stream);
    return launch_gemv_r<WT, VT, PLAN, NB, 1>(a, single, stream);
}

template <typename WT, typename VT, bool PLAN>
dyna_status launch_gemv_nb(const RowdotArgs& a, int nb, bool single, int rows_opt, hipStream_t stream) {
#define DYNA_GEMV_CASE(N) \
    if (nb <= N) return launch_gemv_t<WT, VT, PLAN, N>(a, single, rows_opt, stream);
    DYNA_GEMV_CASE(1)
    DYNA_GEMV_CASE(2)
    DYNA_GEMV_CASE(4)
    DYNA_GEMV_CASE(8)
    DYNA_GEMV_CASE(12)
    DYNA_GEMV_CASE(16)
#undef DYNA_GEMV_CASE
    return set_error(DYNA_ERR_UNSUPPORTED, "rowdot: K > 8192");
}

template <bool PLAN>
dyna_status launch_gemv(const RowdotArgs& a, hipStream_t stream) {
    const int nb = (a.K + 511) / 512;
    const bool single = a.B == 1;
    const int rows_opt = option_gemv_rows();
    const bool wb = a.wdtype == DYNA_BF16, vb = a.vdtype == DYNA_BF16;
    if (wb && vb) return launch_gemv_nb<uint16_t, uint16_t, PLAN>(a, nb, single, rows_opt, stream);
    if (wb && !vb) return launch_gemv_nb<uint16_t, float, PLAN>(a, nb, single, rows_opt, stream);
    if (!wb && vb) return launch_gemv_nb<float, uint16_t, PLAN>(a, nb, single, rows_opt, stream);
    return launch_gemv_nb<float, float, PLAN>(a, nb, single, rows_opt, stream);
}

template <int T, int G, bool VF32, bool PLAN, int KS, int U>
dyna_status launch_mfma_t(const RowdotArgs& a, hipStream_t stream) {
    constexpr int kItemRows = T * kMfmaRows;
    const int64_t items = PLAN ? (int64_t)a.max_chunks_bound * (kChunkRows / kItemRows)
                               : ((int64_t)a.n_rows + kItemRows - 1) / kItemRows;
    const int64_t per_block = KS == 1 ? kWavesPerBlock : 1;
    const int64_t blocks =
        std::max<int64_t>(1, std::min<int64_t>((items + per_block - 1) / per_block, resident_blocks()));
    launch_timed_kernel(rowdot_mfma_kernel<T, G, VF32, PLAN, KS, U>, dim3((unsigned)blocks),
                        dim3(KS > 1 ? KS * kWave : kThreads), 0, stream, a);
    return check_launch("rowdot_mfma_kernel");
}

template <bool VF32, bool PLAN>
dyna_status launch_mfma(const RowdotArgs& a, hipStream_t stream) {
    if (PLAN) {
        // one 16-row tile per wave, U k steps loaded ahead
        if (option_mfma_unroll() == 4) return launch_mfma_t<1, 1, VF32, PLAN, 1, 4>(a, stream);
        if (option_mfma_unroll() == 16) return launch_mfma_t<1, 1, VF32, PLAN, 1, 16>(a, stream);
        return launch_mfma_t<1, 1, VF32, PLAN, 1, 8>(a, stream);
    }
    // dense (router layers, dense head): all contexts share every row; the
    // k steps of a 16-row tile are split over the 8 waves of a block
    const int groups = (a.B + 15) / 16;
    if (groups <= 1) return launch_mfma_t<1, 1, VF32, PLAN, 8, 4>(a, stream);
    if (groups <= 2) return launch_mfma_t<1, 2, VF32, PLAN, 8, 4>(a, stream);
    if (groups <= 4) return launch_mfma_t<1, 4, VF32, PLAN, 8, 4>(a, stream);
    return launch_mfma_t<1, 8, VF32, PLAN, 8, 2>(a, stream);
}

}  // namespace

// path: 0 automatic, 1 GEMV, 2 MFMA (LDS-staged where eligible), 3 MFMA (direct loads)
dyna_status launch_rowdot(const RowdotArgs& a, int path, hipStream_t stream) {
    const bool plan = a.plan.hdr != nullptr;
    const bool mfma_ok = a.wdtype == DYNA_BF16;
    if (path >= 2 && !mfma_ok)
        return set_error(DYNA_ERR_UNSUPPORTED, "rowdot: MFMA path needs bf16 weights");
    const bool use_mfma = path >= 2 || (path == 0 && mfma_ok && a.B > 4);
    // a gathered head on the matrix cores needs bf16 slabs and contexts (the
    // LDS-staged kernel); any other gathered head takes the GEMV
    if (plan && use_mfma && gather_lds_eligible(a)) return launch_gather_lds(a, stream);
    if (plan || !use_mfma) return plan ? launch_gemv<true>(a, stream) : launch_gemv<false>(a, stream);
    const bool vf32 = a.vdtype == DYNA_F32;
    return vf32 ? launch_mfma<true, false>(a, stream) : launch_mfma<false, false>(a, stream);
}

}  // namespace dyna
