// Device helpers shared by the libdynahead kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "dyna_internal.h"

namespace dyna {

constexpr int kNT = 256;  // threads of the per-context (select, top-k) workgroups

// ---------------------------------------------------------------- bf16
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even (finite inputs; NaN stays NaN).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

// Eight consecutive elements of a row as fp32, from bf16 (one 16-byte load)
// or fp32 (two 16-byte loads).  `nt` streams the load past the caches.
// 8 fp32 values split into bf16 hi and lo terms.
__device__ __forceinline__ void split8_regs(const float (&f)[8], u32x4& hi, u32x4& lo) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t h0 = f32_to_bf16_bits(f[2 * i]);
        const uint32_t h1 = f32_to_bf16_bits(f[2 * i + 1]);
        const uint32_t l0 = f32_to_bf16_bits(f[2 * i] - __uint_as_float(h0 << 16));
        const uint32_t l1 = f32_to_bf16_bits(f[2 * i + 1] - __uint_as_float(h1 << 16));
        hi[i] = h0 | (h1 << 16);
        lo[i] = l0 | (l1 << 16);
    }
}
// 8 consecutive fp32 values in memory split into bf16 hi and lo terms.
__device__ __forceinline__ void split8(const float* p, u32x4& hi, u32x4& lo) {
    const u32x4* q = reinterpret_cast<const u32x4*>(p);
    const u32x4 x0 = q[0], x1 = q[1];
    float f[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[i] = __uint_as_float(x0[i]);
        f[4 + i] = __uint_as_float(x1[i]);
    }
    split8_regs(f, hi, lo);
}

template <typename T, bool NT>
struct Load8;

template <bool NT>
struct Load8<uint16_t, NT> {
    __device__ __forceinline__ static void run(const uint16_t* p, float (&x)[8]) {
        u32x4 w = NT ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p))
                     : *reinterpret_cast<const u32x4*>(p);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[2 * i] = bf16_lo(w[i]);
            x[2 * i + 1] = bf16_hi(w[i]);
        }
    }
};

template <bool NT>
struct Load8<float, NT> {
    __device__ __forceinline__ static void run(const float* p, float (&x)[8]) {
        const u32x4* q = reinterpret_cast<const u32x4*>(p);
        u32x4 a = NT ? __builtin_nontemporal_load(q) : q[0];
        u32x4 b = NT ? __builtin_nontemporal_load(q + 1) : q[1];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[i] = __uint_as_float(a[i]);
            x[4 + i] = __uint_as_float(b[i]);
        }
    }
};

// ---------------------------------------------------------------- ordering
// Monotone map of a float to uint32 (larger float -> larger code).  NaN is
// mapped like -inf and -0 like +0, the ordering rule of every top-k here.
__device__ __forceinline__ uint32_t ord_f32(float f) {
    if (f != f) f = -__builtin_inff();
    if (f == 0.0f) f = 0.0f;
    uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float ord_to_f32(uint32_t o) {
    uint32_t u = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
    return __uint_as_float(u);
}
// 64-bit selection key: higher value first, then lower id first.
__device__ __forceinline__ uint64_t sel_key(float v, uint32_t id) {
    return (static_cast<uint64_t>(ord_f32(v)) << 32) | static_cast<uint64_t>(0xffffffffu - id);
}
__device__ __forceinline__ uint32_t key_id(uint64_t key) {
    return 0xffffffffu - static_cast<uint32_t>(key & 0xffffffffu);
}
__device__ __forceinline__ float key_val(uint64_t key) {
    return ord_to_f32(static_cast<uint32_t>(key >> 32));
}

// ---------------------------------------------------------------- wave ops
// Cross-lane steps use DPP row shifts and row broadcasts (ALU latency)
// instead of LDS permutes.  Source lanes outside a row read the identity.
__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

template <int CTRL, int ROW_MASK = 0xf, int BANK_MASK = 0xf>
__device__ __forceinline__ uint32_t dpp(uint32_t identity, uint32_t x) {
    // bound_ctrl off: lanes whose source is outside the row keep `identity`
    return (uint32_t)__builtin_amdgcn_update_dpp((int)identity, (int)x, CTRL, ROW_MASK, BANK_MASK, false);
}
constexpr int kRowShr1 = 0x111, kRowShr2 = 0x112, kRowShr4 = 0x114, kRowShr8 = 0x118;
constexpr int kRowBcast15 = 0x142, kRowBcast31 = 0x143;

// Inclusive scan over the 64 lanes: Hillis-Steele inside each 16-lane row,
// then the row totals are carried across rows with two row broadcasts.
template <typename T, typename Op>
__device__ __forceinline__ T wave_scan_dpp(T x, Op op, uint32_t identity) {
    auto step = [&](auto ctrl_tag, auto rmask_tag) {
        constexpr int CTRL = decltype(ctrl_tag)::value;
        constexpr int RM = decltype(rmask_tag)::value;
        T y;
        if constexpr (sizeof(T) == 4) {
            y = __builtin_bit_cast(T, dpp<CTRL, RM>(identity, __builtin_bit_cast(uint32_t, x)));
        }
        x = op(x, y);
    };
    using I = std::integral_constant<int, 0>;
    step(std::integral_constant<int, kRowShr1>{}, std::integral_constant<int, 0xf>{});
    step(std::integral_constant<int, kRowShr2>{}, std::integral_constant<int, 0xf>{});
    step(std::integral_constant<int, kRowShr4>{}, std::integral_constant<int, 0xf>{});
    step(std::integral_constant<int, kRowShr8>{}, std::integral_constant<int, 0xf>{});
    step(std::integral_constant<int, kRowBcast15>{}, std::integral_constant<int, 0xa>{});
    step(std::integral_constant<int, kRowBcast31>{}, std::integral_constant<int, 0xc>{});
    (void)sizeof(I);
    return x;
}

__device__ __forceinline__ int wave_inclusive_scan(int x) {
    return wave_scan_dpp<int>(x, [](int a, int b) { return a + b; }, 0u);
}
__device__ __forceinline__ float wave_inclusive_scan_f32(float x) {
    return wave_scan_dpp<float>(x, [](float a, float b) { return a + b; }, 0u);
}
__device__ __forceinline__ float readlane_f32(float x, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}

__device__ __forceinline__ float wave_max_f32(float x) {
    return wave_scan_dpp<float>(x, [](float a, float b) { return fmaxf(a, b); },
                                __float_as_uint(-__builtin_inff()));
}

// Sum over the wave; every lane gets the same value (fixed order).
__device__ __forceinline__ float wave_sum(float x) {
    return readlane_f32(wave_inclusive_scan_f32(x), kWave - 1);
}

// Largest 64-bit value over the wave, on every lane.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t x) {
    auto step = [&](auto ctrl_tag, auto rmask_tag) {
        constexpr int CTRL = decltype(ctrl_tag)::value;
        constexpr int RM = decltype(rmask_tag)::value;
        const uint32_t lo = dpp<CTRL, RM>(0u, (uint32_t)x);
        const uint32_t hi = dpp<CTRL, RM>(0u, (uint32_t)(x >> 32));
        const uint64_t y = ((uint64_t)hi << 32) | lo;
        x = y > x ? y : x;
    };
    step(std::integral_constant<int, kRowShr1>{}, std::integral_constant<int, 0xf>{});
    step(std::integral_constant<int, kRowShr2>{}, std::integral_constant<int, 0xf>{});
    step(std::integral_constant<int, kRowShr4>{}, std::integral_constant<int, 0xf>{});
    step(std::integral_constant<int, kRowShr8>{}, std::integral_constant<int, 0xf>{});
    step(std::integral_constant<int, kRowBcast15>{}, std::integral_constant<int, 0xa>{});
    step(std::integral_constant<int, kRowBcast31>{}, std::integral_constant<int, 0xc>{});
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, kWave - 1);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(x >> 32), kWave - 1);
    return ((uint64_t)hi << 32) | lo;
}

// Exclusive scan over a workgroup of NT threads.  `tmp` holds NT/64 + 1 ints
// of LDS.  Returns the exclusive prefix and writes the block total.
template <int NT>
__device__ __forceinline__ int block_exclusive_scan(int x, int* tmp, int* total) {
    constexpr int NW = NT / kWave;
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    int inc = wave_inclusive_scan(x);
    if (lane == kWave - 1) tmp[w] = inc;
    __syncthreads();
    if (w == 0) {
        int t = lane < NW ? tmp[lane] : 0;
        int ti = wave_inclusive_scan(t);
        if (lane < NW) tmp[lane] = ti - t;
        if (lane == NW - 1) tmp[NW] = ti;
    }
    __syncthreads();
    int res = inc - x + tmp[w];
    *total = tmp[NW];
    __syncthreads();
    return res;
}

// Float inclusive scan over a workgroup, fixed association order.
template <int NT>
__device__ __forceinline__ float block_inclusive_scan_f32(float x, float* tmp, float* total) {
    constexpr int NW = NT / kWave;
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    x = wave_inclusive_scan_f32(x);
    if (lane == kWave - 1) tmp[w] = x;
    __syncthreads();
    if (w == 0) {
        float t = lane < NW ? tmp[lane] : 0.0f;
        t = wave_inclusive_scan_f32(t);
        if (lane < NW) tmp[NW + 1 + lane] = t;  // inclusive wave prefixes
    }
    __syncthreads();
    float base = w > 0 ? tmp[NW + 1 + w - 1] : 0.0f;
    *total = tmp[NW + 1 + NW - 1];
    __syncthreads();
    return base + x;
}

// Device-coherent (agent scope) store / load: written through to, and read
// from, the point where every XCD sees the same value, without an L2
// write-back or invalidate.  Used for the few words one workgroup hands to
// another inside a kernel.
template <typename T>
__device__ __forceinline__ void store_coherent(T* p, T v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ T load_coherent(const T* p) {
    return __hip_atomic_load(const_cast<T*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float apply_act(float y, int act) {
    if (act == DYNA_ACT_RELU) return y > 0.0f ? y : 0.0f;
    if (act == DYNA_ACT_SILU) return y / (1.0f + expf(-y));
    return y;
}

}  // namespace dyna
