// Wave-per-row GEMV body shared by the row-dot kernels and the fused
// single-context kernels: out[b, base_b + row] = act(W[row, :] . v[b, :] + bias).
// One wave streams R rows per iteration (16-byte non-temporal loads, a wave
// covers 1 KiB of a row per load), keeps them raw in registers and dots them
// with each context that needs them; with SINGLE (one context) the context
// row is loaded into registers once per wave.
#pragma once
#include "dyna_device.h"

namespace dyna {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;

// Raw 16-byte pieces of a row: bf16 rows need one u32x4 per 8 elements,
// fp32 rows two.  Rows stay raw in registers and are widened inside the FMA
// loop, which halves the registers a bf16 row needs.
template <typename T>
struct Raw8;
template <>
struct Raw8<uint16_t> {
    u32x4 q;
    template <bool NT>
    __device__ __forceinline__ void load(const uint16_t* p) {
        q = NT ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p))
               : *reinterpret_cast<const u32x4*>(p);
    }
    __device__ __forceinline__ void zero() { q = u32x4{0u, 0u, 0u, 0u}; }
    __device__ __forceinline__ float at(int j) const {
        return (j & 1) ? bf16_hi(q[j >> 1]) : bf16_lo(q[j >> 1]);
    }
};
template <>
struct Raw8<float> {
    u32x4 q0, q1;
    template <bool NT>
    __device__ __forceinline__ void load(const float* p) {
        const u32x4* r = reinterpret_cast<const u32x4*>(p);
        q0 = NT ? __builtin_nontemporal_load(r) : r[0];
        q1 = NT ? __builtin_nontemporal_load(r + 1) : r[1];
    }
    __device__ __forceinline__ void zero() { q0 = q1 = u32x4{0u, 0u, 0u, 0u}; }
    __device__ __forceinline__ float at(int j) const {
        return __uint_as_float(j < 4 ? q0[j] : q1[j - 4]);
    }
};

// acc + w . x over the 8 elements of two raw pieces, in element order.  Two
// bf16 pieces use the packed bf16 dot product (two exact products and the
// accumulator per instruction, four instructions instead of eight widenings
// and eight FMAs); any fp32 operand takes FMAs.  Every kernel that must agree
// bit for bit with another (the one-context paths) accumulates through this.
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
// A 32-bit word as two bf16 lanes.  (Through memcpy: a bit cast applied to a
// vector element directly was compiled to read element 0 every time.)
__device__ __forceinline__ bf16x2 as_bf16x2(uint32_t u) {
    bf16x2 r;
    __builtin_memcpy(&r, &u, 4);
    return r;
}
__device__ __forceinline__ float dot8(const Raw8<uint16_t>& w, const Raw8<uint16_t>& x, float acc) {
#pragma unroll
    for (int p = 0; p < 4; ++p)
        acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(w.q[p]), as_bf16x2(x.q[p]), acc, false);
    return acc;
}
template <typename WT, typename VT>
__device__ __forceinline__ float dot8(const Raw8<WT>& w, const Raw8<VT>& x, float acc) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc = fmaf(w.at(j), x.at(j), acc);
    return acc;
}

// One wave computes R consecutive rows per iteration.  With SINGLE (one
// context: B = 1) the context row is loaded into registers once per wave.
// Default epilogue: store the value (and, in plan mode, the slot's vocabulary id).
// An epilogue's idle() runs while a row group's loads are in flight.
template <bool PLAN>
struct StoreEpi {
    __device__ __forceinline__ void idle() {}
    __device__ __forceinline__ void put(const RowdotArgs& a, int64_t o, float value, int32_t vid) {
        a.out[o] = value;
        if constexpr (PLAN) {
            if (a.vid_out) a.vid_out[o] = vid;
        }
    }
};

template <typename WT, typename VT, int NB, bool PLAN, int R, bool SINGLE, typename Epi = StoreEpi<PLAN>>
__device__ __forceinline__ void gemv_rows(const RowdotArgs& a, Epi& epi) {
    static_assert(kChunkRows % R == 0, "row groups must tile a chunk");
    constexpr int kGroups = kChunkRows / R;  // row groups per plan chunk
    const int lane = lane_id();
    const int64_t nwaves = (int64_t)gridDim.x * kWavesPerBlock;
    const WT* __restrict__ W = static_cast<const WT*>(a.W);
    const VT* __restrict__ v = static_cast<const VT*>(a.v);
    const int K = a.K;
    const int64_t it0 = (int64_t)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave;

    Raw8<VT> hv[SINGLE ? NB : 1];
    if constexpr (SINGLE) {
#pragma unroll
        for (int blk = 0; blk < NB; ++blk) {
            const int e = blk * 512 + lane * 8;
            if (e < K) hv[blk].template load<false>(v + e);
            else hv[blk].zero();
        }
    }

    int64_t n_items;
    Chunk pre{0, 0, 0, 0};
    if constexpr (PLAN) {
        // the first chunk descriptor is fetched together with the count
        // (in bounds: the grid never exceeds the allocated chunk table)
        const int64_t c0 = it0 / kGroups;
        if (c0 < a.plan.max_chunks) pre = a.plan.chunks[c0];
        n_items = (int64_t)a.plan.hdr->n_chunks * kGroups;
    } else {
        n_items = ((int64_t)a.n_rows + R - 1) / R;
    }

    for (int64_t it = it0; it < n_items; it += nwaves) {
        int64_t row0;
        int nrow;  // valid rows of this group
        int lcnt;
        const ListEntry* list = nullptr;
        if constexpr (PLAN) {
            const Chunk c = it == it0 ? pre : a.plan.chunks[it / kGroups];
            const int sub = (int)(it % kGroups) * R;
            if (sub >= c.nrows) continue;
            row0 = (int64_t)c.r0 + sub;
            nrow = min(R, c.nrows - sub);
            lcnt = c.list_cnt;
            list = a.plan.list + c.list_off;
        } else {
            row0 = it * R;
            nrow = (int)min<int64_t>(R, (int64_t)a.n_rows - row0);
            lcnt = a.B;
        }
        Raw8<WT> w[R][NB];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const WT* wr = W + (row0 + r) * K;
#pragma unroll
            for (int blk = 0; blk < NB; ++blk) {
                const int e = blk * 512 + lane * 8;
                if (r < nrow && e < K) w[r][blk].template load<true>(wr + e);
                else w[r][blk].zero();
            }
        }
        // lane r < nrow owns row r of the group in the epilogue
        const bool own = lane < nrow;
        const float bias = (a.bias && own) ? a.bias[row0 + lane] : 0.0f;
        int32_t vid = 0;
        if constexpr (PLAN) {
            if (a.perm && own) vid = a.perm[row0 + lane];
        }
        epi.idle();

        for (int i = 0; i < lcnt; ++i) {
            int b, base;
            if constexpr (PLAN) {
                const ListEntry le = list[i];
                b = le.b;
                base = le.slot_base;
            } else {
                b = i;
                base = 0;
            }
            float acc[R];
#pragma unroll
            for (int r = 0; r < R; ++r) acc[r] = 0.0f;
#pragma unroll
            for (int blk = 0; blk < NB; ++blk) {
                Raw8<VT> x;
                if constexpr (SINGLE) {
                    x = hv[blk];
                } else {
                    const int e = blk * 512 + lane * 8;
                    if (e < K) x.template load<false>(v + (int64_t)b * K + e);
                    else x.zero();
                }
#pragma unroll
                for (int r = 0; r < R; ++r) acc[r] = dot8(w[r][blk], x, acc[r]);
            }
            float mine = 0.0f;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const float t = wave_sum(acc[r]);
                if (lane == r) mine = t;
            }
            if (own) {
                const int64_t o = (int64_t)b * a.ld + base + row0 + lane;
                epi.put(a, o, apply_act(mine + bias, a.act), vid);
            }
        }
    }
}

}  // namespace
}  // namespace dyna
