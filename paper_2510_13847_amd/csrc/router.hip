// Router layers for batches of contexts (Sec. 4.2, "Low-cost router": the
// router is a small FFN applied to every context of the step).
//
// A router layer is a skinny dense product, out[b, r] = act(W[r, :] . x[b, :]
// + bias[r]) with a few thousand rows r and B <= 128 contexts.  The weights
// are streamed from HBM once; the contexts are small but every row needs all
// of them.  Work is split over (16 * NW rows) x (one k slice) workgroups:
//
//  * the workgroup stages the k slice of every context in LDS once (an fp32
//    input, the hidden layer, is split into bf16 hi + lo terms here), so the
//    NW waves of 16 rows each share it instead of re-reading it from L2;
//  * each wave streams its 16 W rows of the slice and multiplies them with
//    v_mfma_f32_16x16x32_bf16, contexts as the 16-wide columns;
//  * the k slices give enough workgroups to cover the chip and keep the
//    staged slice small; every slice writes its partial sums, and a second
//    kernel adds the slices in a fixed order and applies bias and activation,
//    so results are bit-identical from run to run;
//  * for a few contexts the second layer can stage its fp32 contexts (the
//    hidden layer) straight from the first layer's partial sums, adding the
//    slices in the same order with the same bias and activation, which saves
//    the reduction launch and gives the same values.
//
// LDS layout: context c, 16-byte piece p of the slice at position p ^ (c & 15)
// (16 lanes reading one piece index of 16 contexts hit 16 bank groups).
#include <atomic>

#include "dyna_device.h"

namespace dyna {
namespace {

constexpr int kSliceQuantum = 128;  // k-slice lengths are multiples of this
constexpr int kMaxCols = 128;       // contexts per launch (8 MFMA column groups)
constexpr int kLdsBudget = 128 * 1024;

// 32-wide k steps per slice: up to 512 with one row tile per wave, 256 with two
constexpr int max_steps(int tt) { return tt == 1 ? 16 : 8; }
// staged pieces in flight per thread (fp32 pieces take twice the registers)
template <bool VF32>
constexpr int stage_batch() { return VF32 ? 8 : 16; }

// Eight consecutive elements (k .. k + 7) of context c given as the previous
// layer's split-K partial sums: the slices added in order (sixteen slices'
// loads in flight at once), then the bias and the activation, exactly as that
// layer's reduction kernel computes them; split into bf16 hi and lo terms.
__device__ __forceinline__ void hidden8(const RowdotArgs& a, int c, int k, u32x4& hi, u32x4& lo) {
    constexpr int kSlicesInFlight = 16;
    const int64_t stride = (int64_t)a.B * a.K;
    const float* p = a.vpart + (int64_t)c * a.K + k;
    float f[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = 0.0f;
    for (int s0 = 0; s0 < a.vslices; s0 += kSlicesInFlight) {
        u32x4 y[kSlicesInFlight][2];
#pragma unroll
        for (int u = 0; u < kSlicesInFlight; ++u)
            if (s0 + u < a.vslices) {
                const u32x4* q = reinterpret_cast<const u32x4*>(p + (s0 + u) * stride);
                y[u][0] = q[0];
                y[u][1] = q[1];
            }
#pragma unroll
        for (int u = 0; u < kSlicesInFlight; ++u)
            if (s0 + u < a.vslices)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    f[i] += __uint_as_float(y[u][0][i]);
                    f[4 + i] += __uint_as_float(y[u][1][i]);
                }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = apply_act(f[i] + (a.vbias ? a.vbias[k + i] : 0.0f), a.vact);
    split8_regs(f, hi, lo);
}

// One k slice `sl` of a workgroup's row tile: stage the slice of every
// context in LDS, multiply, write the slice's partial sums.
template <int NW, int G, bool VF32, int TT, bool FP = false>
__device__ __forceinline__ void splitk_slice(const RowdotArgs& a, int ksl, int sl, float* part, uint16_t* xs) {
    constexpr int MAXS = max_steps(TT);
    constexpr int NCOL = G * 16;
    const int K = a.K, B = a.B, n = a.n_rows;
    const int k0 = sl * ksl;
    const int kn = min(ksl, K - k0);
    const int npc = ksl / 8;  // 16-byte pieces per context row of the slice

    // the wave's 16 W rows of the slice are requested first, so that their
    // HBM latency overlaps the staging of the contexts below
    const int lane = lane_id(), wv = threadIdx.x / kWave;
    const int col = lane & 15, kq = lane >> 4;
    const int r0 = (blockIdx.x * NW + wv) * kMfmaRows * TT;
    const int nsteps = (kn + 31) / 32;
    u32x4 A[TT][MAXS];
    if (r0 < n) {
#pragma unroll
        for (int t = 0; t < TT; ++t) {
            // rows past n read row n - 1 and are never stored
            const uint16_t* __restrict__ wr =
                static_cast<const uint16_t*>(a.W) + (int64_t)min(r0 + t * kMfmaRows + col, n - 1) * K + k0;
#pragma unroll
            for (int s = 0; s < MAXS; ++s) {
                const int k = s * 32 + kq * 8;
                A[t][s] = u32x4{0u, 0u, 0u, 0u};
                if (s < nsteps && k < kn)
                    A[t][s] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wr + k));
            }
        }
    }

    // stage the slice of every context, kStageBatch pieces in flight per
    // thread; piece idx = c * npc + p, stepped without divisions
    const int npieces = NCOL * npc;
    constexpr int T = NW * kWave;
    const int dc = T / npc, dp = T - dc * npc;
    int c = threadIdx.x / npc, p = threadIdx.x - c * npc;
    constexpr int kStageBatch = stage_batch<VF32>();
    // contexts given as the previous layer's partial sums: one piece at a
    // time per thread, its slices' loads in flight together
    // (FP: instances for the contexts of a few-context step only, whose
    // registers the partial-sum loads take)
    constexpr bool from_parts = VF32 && FP;
    if constexpr (from_parts) {
        for (int idx = threadIdx.x; idx < npieces; idx += T) {
            const int cc = idx / npc, pp = idx - cc * npc;
            u32x4 hi{0u, 0u, 0u, 0u}, lo{0u, 0u, 0u, 0u};
            if (cc < B && pp * 8 < kn) hidden8(a, cc, k0 + pp * 8, hi, lo);
            const int pos = cc * ksl + (pp ^ (cc & 15)) * 8;
            *reinterpret_cast<u32x4*>(xs + pos) = hi;
            *reinterpret_cast<u32x4*>(xs + NCOL * ksl + pos) = lo;
        }
    }
    for (int idx0 = from_parts ? npieces : threadIdx.x; idx0 < npieces; idx0 += T * kStageBatch) {
        u32x4 hi[kStageBatch], lo[kStageBatch];
        int cq[kStageBatch], pq[kStageBatch];
#pragma unroll
        for (int q = 0; q < kStageBatch; ++q) {
            cq[q] = c;
            pq[q] = p;
            hi[q] = u32x4{0u, 0u, 0u, 0u};
            lo[q] = u32x4{0u, 0u, 0u, 0u};
            if (c < B && p * 8 < kn) {
                if constexpr (VF32) {
                    split8(static_cast<const float*>(a.v) + (int64_t)c * K + k0 + p * 8, hi[q], lo[q]);
                } else {
                    hi[q] = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.v) + (int64_t)c * K + k0 +
                                                            p * 8);
                }
            }
            c += dc;
            p += dp;
            if (p >= npc) {
                p -= npc;
                ++c;
            }
        }
#pragma unroll
        for (int q = 0; q < kStageBatch; ++q) {
            if (cq[q] < NCOL) {
                const int pos = cq[q] * ksl + (pq[q] ^ (cq[q] & 15)) * 8;
                *reinterpret_cast<u32x4*>(xs + pos) = hi[q];
                if constexpr (VF32) *reinterpret_cast<u32x4*>(xs + NCOL * ksl + pos) = lo[q];
            }
        }
    }
    __syncthreads();
    if (r0 >= n) return;  // wave-uniform; no barrier follows in this slice

    // every context piece read from LDS feeds the TT row tiles of the wave
    f32x4 acc[TT][G];
#pragma unroll
    for (int t = 0; t < TT; ++t)
#pragma unroll
        for (int g = 0; g < G; ++g) acc[t][g] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < MAXS; ++s) {
        if (s >= nsteps) continue;  // wave-uniform
        const int p = s * 4 + kq;
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int pos = (g * 16 + col) * ksl + (p ^ col) * 8;
            const u32x4 bh = *reinterpret_cast<const u32x4*>(xs + pos);
            u32x4 bl{0u, 0u, 0u, 0u};
            if constexpr (VF32) bl = *reinterpret_cast<const u32x4*>(xs + NCOL * ksl + pos);
#pragma unroll
            for (int t = 0; t < TT; ++t) {
                acc[t][g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, A[t][s]),
                                                                    __builtin_bit_cast(bf16x8, bh), acc[t][g], 0, 0, 0);
                if constexpr (VF32)
                    acc[t][g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8, A[t][s]), __builtin_bit_cast(bf16x8, bl), acc[t][g], 0, 0, 0);
            }
        }
    }
    // partial sums of this slice: part[slice][b][row]; D row 4 * kq + r, column col
    float* pp = part + (int64_t)sl * B * n;
#pragma unroll
    for (int t = 0; t < TT; ++t)
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int b = g * 16 + col;
            if (b >= B) continue;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = r0 + t * kMfmaRows + 4 * kq + r;
                if (row < n) pp[(int64_t)b * n + row] = acc[t][g][r];
            }
        }
}

// Workgroup (x, y) takes k slice y of row tile x; each slice's partial sums
// go to their own place.
template <int NW, int G, bool VF32, int TT, bool FP>
__global__ __launch_bounds__(NW * kWave) void dense_splitk_kernel(RowdotArgs a, int ksl, float* part) {
    extern __shared__ __attribute__((aligned(16))) uint16_t xs[];  // [G*16][ksl] hi, then lo
    if (a.zero_words != nullptr && blockIdx.x == 0 && blockIdx.y == 0 && (int)threadIdx.x < a.n_zero_words)
        a.zero_words[threadIdx.x] = 0;
    splitk_slice<NW, G, VF32, TT, FP>(a, ksl, blockIdx.y, part, xs);
}

// out[b * ld + r] = act(sum over slices, in slice order, + bias[r])
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, int slices, int B, int n,
                                                            float* __restrict__ out, int64_t ld,
                                                            const float* __restrict__ bias, int act) {
    const int r = blockIdx.x * 256 + threadIdx.x;
    if (r >= n) return;
    for (int b = blockIdx.y; b < B; b += gridDim.y) {
        float s = 0.0f;
#pragma unroll 8
        for (int q = 0; q < slices; ++q) s += part[((int64_t)q * B + b) * n + r];
        out[(int64_t)b * ld + r] = apply_act(s + (bias ? bias[r] : 0.0f), act);
    }
}

template <int NW, int G, bool VF32, int TT, bool FP = false>
dyna_status launch_splitk_t(const RowdotArgs& a, const SplitShape& sh, float* part, bool reduce, hipStream_t stream) {
    const dim3 grid((unsigned)sh.row_tiles, (unsigned)sh.slices);
    const uint32_t lds = (uint32_t)sh.lds;
    if (lds > 64 * 1024) {
        // above 64 KiB the dynamic LDS size must be allowed, once per kernel and device
        static std::atomic<uint64_t> allowed{0};
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return set_error(DYNA_ERR_HIP, "router: device");
        if (!(allowed.load() & (1ull << dev))) {
            if (hipFuncSetAttribute((const void*)dense_splitk_kernel<NW, G, VF32, TT, FP>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBudget) != hipSuccess)
                return set_error(DYNA_ERR_HIP, "router: LDS attribute");
            allowed.fetch_or(1ull << dev);
        }
    }
    dense_splitk_kernel<NW, G, VF32, TT, FP><<<grid, dim3(NW * kWave), lds, stream>>>(a, sh.ksl, part);
    const dyna_status st = check_launch("dense_splitk_kernel");
    if (st != DYNA_OK || !reduce) return st;
    const int rx = (a.n_rows + 255) / 256;
    splitk_reduce_kernel<<<dim3((unsigned)rx, (unsigned)a.B), dim3(256), 0, stream>>>(
        part, sh.slices, a.B, a.n_rows, a.out, a.ld, a.bias, a.act);
    return check_launch("splitk_reduce_kernel");
}

template <int NW, bool VF32>
dyna_status launch_splitk_g(const RowdotArgs& a, const SplitShape& sh, float* part, bool reduce, hipStream_t stream) {
    // the kernel's row tiles per wave must be the shape's (they bound the slice length)
    if (a.vpart != nullptr) {
        // contexts from partial sums: up to 16 contexts (one column group)
        if constexpr (VF32) {
            if (sh.tiles == 1 && sh.groups == 1) return launch_splitk_t<NW, 1, true, 1, true>(a, sh, part, reduce, stream);
        }
        return set_error(DYNA_ERR_UNSUPPORTED, "split-K router: partial-sum contexts need fp32 and <= 16 contexts");
    }
    if (sh.tiles == 2) {
        if (sh.groups == 4) return launch_splitk_t<NW, 4, VF32, 2>(a, sh, part, reduce, stream);
        return launch_splitk_t<NW, 8, VF32, 2>(a, sh, part, reduce, stream);
    }
    switch (sh.groups) {
        case 1: return launch_splitk_t<NW, 1, VF32, 1>(a, sh, part, reduce, stream);
        case 2: return launch_splitk_t<NW, 2, VF32, 1>(a, sh, part, reduce, stream);
        case 4: return launch_splitk_t<NW, 4, VF32, 1>(a, sh, part, reduce, stream);
        default: return launch_splitk_t<NW, 8, VF32, 1>(a, sh, part, reduce, stream);
    }
}

}  // namespace

bool splitk_shape(int32_t n_rows, int32_t K, int32_t B, bool vf32, SplitShape* out) {
    if (B < 1 || B > kMaxCols || n_rows < 1 || K < 8) return false;
    SplitShape s{};
    s.groups = (B + 15) / 16;
    if (s.groups == 3) s.groups = 4;
    if (s.groups > 4) s.groups = 8;
    s.tiles = 1;  // row tiles per wave (two measured slower: fewer waves hide less latency)
    s.nw = n_rows >= 2048 * s.tiles ? 8 : 4;
    const int rows_per_block = 16 * s.nw * s.tiles;
    s.row_tiles = (n_rows + rows_per_block - 1) / rows_per_block;
    // about 256 workgroups in all, slices of at least one quantum, and the
    // staged slice within the LDS budget
    const int bytes_per_k = s.groups * 16 * 2 * (vf32 ? 2 : 1);
    const int ksl_max = std::min(max_steps(s.tiles) * 32,
                                 std::max(kSliceQuantum, (kLdsBudget / bytes_per_k) / kSliceQuantum * kSliceQuantum));
    const int want_slices = std::max(1, (256 + s.row_tiles - 1) / s.row_tiles);
    int ksl = (K + want_slices - 1) / want_slices;
    ksl = (ksl + kSliceQuantum - 1) / kSliceQuantum * kSliceQuantum;
    s.ksl = std::min(std::max(ksl, kSliceQuantum), ksl_max);
    s.slices = (K + s.ksl - 1) / s.ksl;
    s.lds = (size_t)bytes_per_k * (size_t)s.ksl;
    *out = s;
    return true;
}

size_t splitk_part_floats(int32_t n_rows, int32_t K, int32_t B, bool vf32) {
    SplitShape s;
    if (!splitk_shape(n_rows, K, B, vf32, &s)) return 0;
    return (size_t)s.slices * (size_t)B * (size_t)n_rows;
}

dyna_status launch_dense_splitk(const RowdotArgs& a, float* part, size_t part_floats, hipStream_t stream,
                                int* deferred_slices) {
    // deferred_slices set: leave the slices' partial sums in `part` for the
    // consumer to add (in slice order, then the bias; no activation)
    const bool reduce = deferred_slices == nullptr;
    const bool vf32 = a.vdtype == DYNA_F32;
    SplitShape sh;
    if (a.wdtype != DYNA_BF16 || a.plan.hdr != nullptr || !splitk_shape(a.n_rows, a.K, a.B, vf32, &sh))
        return set_error(DYNA_ERR_UNSUPPORTED, "split-K router: needs bf16 weights, 1..128 contexts");
    if (part == nullptr || (size_t)sh.slices * (size_t)a.B * (size_t)a.n_rows > part_floats)
        return set_error(DYNA_ERR_WORKSPACE, "split-K router: partial-sum buffer too small");
    if (!reduce) {
        if (a.act != DYNA_ACT_NONE) return set_error(DYNA_ERR_UNSUPPORTED, "split-K router: deferred sum with activation");
        *deferred_slices = sh.slices;
    }
    if (sh.nw == 8)
        return vf32 ? launch_splitk_g<8, true>(a, sh, part, reduce, stream)
                    : launch_splitk_g<8, false>(a, sh, part, reduce, stream);
    return vf32 ? launch_splitk_g<4, true>(a, sh, part, reduce, stream)
                : launch_splitk_g<4, false>(a, sh, part, reduce, stream);
}

}  // namespace dyna
