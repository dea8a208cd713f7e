// Selection state of a one-context head, and its cross-workgroup merge.
//
// Algorithm 1 selects with log_softmax, TopK_{k_t} and remap2realid.  For
// the argmax each lane keeps the best (logit, vocabulary id) key of the
// logits it produced and an online softmax pair (running max m, sum of
// exp((z - m)/T)); a workgroup reduces its lanes to one partial, written with
// device-coherent stores, and arrives on a counter.  The last workgroup to
// arrive merges the partials in workgroup order (deterministic).  No
// grid-wide wait and no L2 write-back is involved.  For k_t > 1 the helpers
// at the end keep a wave's best keys spread over its lanes and take the k_t
// best of many sorted lists.
#pragma once
#include "dyna_device.h"

namespace dyna {
namespace {

struct GreedyPartial {
    uint64_t key;  // best (ordered logit, inverted vocabulary id)
    float m;       // max logit
    float s;       // sum of exp((z - m) / T)
};

// Online softmax pair merge (m, s) <- (m, s) (+) (m2, s2).
__device__ __forceinline__ void softmax_merge(float& m, float& s, float m2, float s2, float inv_t) {
    if (m2 == -__builtin_inff()) return;
    if (m == -__builtin_inff()) {
        m = m2;
        s = s2;
        return;
    }
    const float M = fmaxf(m, m2);
    s = s * expf((m - M) * inv_t) + s2 * expf((m2 - M) * inv_t);
    m = M;
}

// Per-lane greedy state.
struct GreedyState {
    uint64_t best = 0;
    float m = -__builtin_inff();
    float s = 0.0f;
    __device__ __forceinline__ void add(float value, int32_t vid, float inv_t) {
        const float z = value != value ? -__builtin_inff() : value;
        const uint64_t key = sel_key(z, (uint32_t)vid);
        best = key > best ? key : best;
        softmax_merge(m, s, z, 1.0f, inv_t);
    }
};

// Workgroup of NT threads: reduce the lanes' states in a fixed order, publish
// the workgroup's partial at part[slot] and arrive on `counter`, which
// n_part workgroups reach.  Returns true in the last workgroup to arrive
// (uniform over its threads); there, thread 0's `out` is the merge of all
// n_part partials in slot order, and the counter is back at zero.
template <int NT>
__device__ bool greedy_publish_merge(const GreedyState& st, float inv_t, GreedyPartial* part, int slot,
                                     int n_part, int32_t* counter, GreedyState* out) {
    constexpr int NW = NT / kWave;
    __shared__ uint64_t w_best[NW];
    __shared__ float w_m[NW], w_s[NW];
    __shared__ int last;
    const int lane = lane_id(), w = threadIdx.x / kWave;
    const uint64_t wb = wave_max_u64(st.best);
    const float wm = readlane_f32(wave_max_f32(st.m), kWave - 1);
    const float ws = wave_sum(st.m == -__builtin_inff() ? 0.0f : st.s * expf((st.m - wm) * inv_t));
    if (lane == 0) {
        w_best[w] = wb;
        w_m[w] = wm;
        w_s[w] = ws;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t bb = w_best[0];
        float bm = w_m[0], bs = w_s[0];
        for (int q = 1; q < NW; ++q) {
            bb = w_best[q] > bb ? w_best[q] : bb;
            softmax_merge(bm, bs, w_m[q], w_s[q], inv_t);
        }
        store_coherent(&part[slot].key, bb);
        store_coherent(&part[slot].m, bm);
        store_coherent(&part[slot].s, bs);
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_s_waitcnt(0);
        last = __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == n_part - 1;
    }
    __syncthreads();
    if (!last) return false;

    // thread t merges partials t, t + NT, ... in order, then a fixed-order
    // wave and workgroup reduction
    if (threadIdx.x == 0) store_coherent(counter, 0);
    uint64_t bb = 0;
    float bm = -__builtin_inff(), bs = 0.0f;
    for (int g = threadIdx.x; g < n_part; g += NT) {
        const uint64_t k2 = load_coherent(&part[g].key);
        const float m2 = load_coherent(&part[g].m), s2 = load_coherent(&part[g].s);
        bb = k2 > bb ? k2 : bb;
        softmax_merge(bm, bs, m2, s2, inv_t);
    }
    const uint64_t gb = wave_max_u64(bb);
    const float gm = readlane_f32(wave_max_f32(bm), kWave - 1);
    const float gs = wave_sum(bm == -__builtin_inff() ? 0.0f : bs * expf((bm - gm) * inv_t));
    __syncthreads();
    if (lane == 0) {
        w_best[w] = gb;
        w_m[w] = gm;
        w_s[w] = gs;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        GreedyState f;
        f.best = w_best[0];
        f.m = w_m[0];
        f.s = w_s[0];
        for (int q = 1; q < NW; ++q) {
            f.best = w_best[q] > f.best ? w_best[q] : f.best;
            softmax_merge(f.m, f.s, w_m[q], w_s[q], inv_t);
        }
        *out = f;
    }
    return true;
}

// ---------------------------------------------------------------- top-k_t
// The key of each row goes into a list kept across the wave: lane l of
// every 16-lane row holds the wave's l-th best key so far (descending, 0 =
// empty).  A key x enters in one step, all lanes at once: place l takes
// max(key_l, min(key_{l-1}, x)), key_{l-1} read from the lane below (row
// shift; the row's first lane reads the all-ones identity).  Eight vector
// instructions per key, and no per-lane list in registers; x = 0 (no key)
// leaves the list unchanged.
__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int l) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t row_list_insert(uint64_t mine, uint64_t x) {
    const uint32_t plo = dpp<kRowShr1>(0xffffffffu, (uint32_t)mine);
    const uint32_t phi = dpp<kRowShr1>(0xffffffffu, (uint32_t)(mine >> 32));
    const uint64_t prev = ((uint64_t)phi << 32) | plo;
    const uint64_t up = prev < x ? prev : x;
    return mine > up ? mine : up;
}

// The workgroup's (m, s) over its lanes in a fixed order (thread 0 gets it).
template <int NT>
__device__ __forceinline__ void block_softmax_pair(float m, float s, float inv_t, float* w_m, float* w_s,
                                                   float* out_m, float* out_s) {
    constexpr int NW = NT / kWave;
    const int lane = lane_id(), w = threadIdx.x / kWave;
    const float wm = readlane_f32(wave_max_f32(m), kWave - 1);
    const float ws = wave_sum(m == -__builtin_inff() ? 0.0f : s * expf((m - wm) * inv_t));
    if (lane == 0) {
        w_m[w] = wm;
        w_s[w] = ws;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        float bm = w_m[0], bs = w_s[0];
        for (int q = 1; q < NW; ++q) softmax_merge(bm, bs, w_m[q], w_s[q], inv_t);
        *out_m = bm;
        *out_s = bs;
    }
}

// The k_t (<= L) best keys held in sorted lists (descending, 0 = empty;
// valid keys distinct and nonzero), one list per thread of NT.  The k_t-th
// best list head T bounds the answer from below (k_t distinct heads are
// >= T), so only entries >= T of lists whose head is >= T can be selected:
// at most k_t lists of k_t entries, ranked by counting.  No chain of k_t
// block-wide maxima.  out[0..k_t) gets the keys in descending order, 0 where
// fewer exist; ends with a barrier.
template <int L, int NT>
__device__ void block_topk_lists(const uint64_t (&list)[L], int k_t, uint64_t* heads /* LDS [NT] */,
                                 uint64_t* cand /* LDS [L * L] */, uint64_t* out /* LDS [k_t] */) {
    __shared__ uint64_t sh_T;
    __shared__ int sh_n;
    const uint64_t head = list[0];
    heads[threadIdx.x] = head;
    if (threadIdx.x == 0) {
        sh_T = 0;
        sh_n = 0;
    }
    __syncthreads();
    if (head != 0) {
        int rank = 0;
        for (int j = 0; j < NT; ++j) rank += heads[j] > head;
        if (rank == k_t - 1) sh_T = head;
    }
    __syncthreads();
    const uint64_t T = sh_T;
    if (head != 0 && head >= T) {
#pragma unroll
        for (int r = 0; r < L; ++r)
            if (r < k_t && list[r] != 0 && list[r] >= T) cand[atomicAdd(&sh_n, 1)] = list[r];
    }
    __syncthreads();
    const int n = sh_n;
    for (int c = threadIdx.x; c < n; c += NT) {
        const uint64_t key = cand[c];
        int rank = 0;
        for (int j = 0; j < n; ++j) rank += cand[j] > key;
        if (rank < k_t) out[rank] = key;
    }
    for (int r = n + threadIdx.x; r < k_t; r += NT) out[r] = 0;
    __syncthreads();
}

}  // namespace
}  // namespace dyna
