// Fused gathered head + greedy selection for one context (B = 1).
//
// A one-context step is a chain of small dependent kernels; each boundary
// costs a launch plus a cold read of the previous kernel's output.  Here the
// selection of Algorithm 1 (log_softmax, TopK_1 = argmax, remap2realid) is
// folded into the gathered head (Sec. 4.3): every wave keeps, for the logits
// it produces, the best (logit, vocabulary id) key and an online softmax pair
// (running max m, sum of exp((z - m)/T)); each workgroup reduces them to one
// partial, written with device-coherent stores.  The workgroups that had
// work arrive on a counter; the last one merges the partials in workgroup
// order (deterministic) and writes the token and its log-probability.  No
// grid-wide wait and no L2 write-back is involved.  The arrival counter is
// cleared by the step's first kernel and by the last workgroup after use.
#include "gemv.h"
#include "select_row.h"

namespace dyna {
namespace {

constexpr int kGreedyGrid = 256;  // default workgroups of the fused head (one arrival each)

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

struct GreedyEpi {
    float inv_t;
    uint64_t best = 0;
    float m = -__builtin_inff();
    float s = 0.0f;
    __device__ __forceinline__ void put(const RowdotArgs& a, int64_t o, float value, int32_t vid) {
        a.out[o] = value;
        if (a.vid_out) a.vid_out[o] = vid;
        const float z = value != value ? -__builtin_inff() : value;
        const uint64_t key = sel_key(z, (uint32_t)vid);
        best = key > best ? key : best;
        softmax_merge(m, s, z, 1.0f, inv_t);
    }
};

template <typename WT, typename VT, int NB, int R>
__global__ __launch_bounds__(kThreads) void logits_greedy_kernel(RowdotArgs lg, SelectArgs sa,
                                                                 GreedyPartial* part, int32_t* counter) {
    __shared__ uint64_t w_best[kWavesPerBlock];
    __shared__ float w_m[kWavesPerBlock], w_s[kWavesPerBlock];
    __shared__ int last;
    const int64_t n_items = (int64_t)lg.plan.hdr->n_chunks * (kChunkRows / R);
    // workgroups whose first wave has an item take part (at least workgroup 0)
    const int64_t n_part = std::max<int64_t>(
        1, std::min<int64_t>(gridDim.x, (n_items + kWavesPerBlock - 1) / kWavesPerBlock));
    if ((int64_t)blockIdx.x >= n_part) return;

    GreedyEpi epi{sa.inv_t};
    gemv_rows<WT, VT, NB, true, R, true, GreedyEpi>(lg, epi);

    // wave, then workgroup reduction in a fixed order
    const int lane = lane_id(), w = threadIdx.x / kWave;
    const uint64_t wb = wave_max_u64(epi.best);
    float m = epi.m, s = epi.s;
    const float wm = readlane_f32(wave_max_f32(m), kWave - 1);
    const float ws = wave_sum(m == -__builtin_inff() ? 0.0f : s * expf((m - wm) * sa.inv_t));
    if (lane == 0) {
        w_best[w] = wb;
        w_m[w] = wm;
        w_s[w] = ws;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t bb = w_best[0];
        float bm = w_m[0], bs = w_s[0];
        for (int q = 1; q < kWavesPerBlock; ++q) {
            bb = w_best[q] > bb ? w_best[q] : bb;
            softmax_merge(bm, bs, w_m[q], w_s[q], sa.inv_t);
        }
        store_coherent(&part[blockIdx.x].key, bb);
        store_coherent(&part[blockIdx.x].m, bm);
        store_coherent(&part[blockIdx.x].s, bs);
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_s_waitcnt(0);
        last = __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
               (int)n_part - 1;
    }
    __syncthreads();
    if (!last) return;

    // last workgroup: thread t merges partials t, t + 256, ... in order, then
    // a fixed-order wave and workgroup reduction
    if (threadIdx.x == 0) store_coherent(counter, 0);
    uint64_t bb = 0;
    float bm = -__builtin_inff(), bs = 0.0f;
    for (int64_t g = threadIdx.x; g < n_part; g += kThreads) {
        const uint64_t k2 = load_coherent(&part[g].key);
        const float m2 = load_coherent(&part[g].m), s2 = load_coherent(&part[g].s);
        bb = k2 > bb ? k2 : bb;
        softmax_merge(bm, bs, m2, s2, sa.inv_t);
    }
    const uint64_t gb = wave_max_u64(bb);
    const float gm = readlane_f32(wave_max_f32(bm), kWave - 1);
    const float gs = wave_sum(bm == -__builtin_inff() ? 0.0f : bs * expf((bm - gm) * sa.inv_t));
    __syncthreads();
    if (lane == 0) {
        w_best[w] = gb;
        w_m[w] = gm;
        w_s[w] = gs;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t fb = w_best[0];
        float fm = w_m[0], fs = w_s[0];
        for (int q = 1; q < kWavesPerBlock; ++q) {
            fb = w_best[q] > fb ? w_best[q] : fb;
            softmax_merge(fm, fs, w_m[q], w_s[q], sa.inv_t);
        }
        if (sa.out_ids) sa.out_ids[0] = fb != 0 ? (int32_t)key_id(fb) : -1;
        if (sa.out_logprobs) {
            const TailMix tail = tail_of(sa, sa.row_len ? sa.row_len[0] : sa.fixed_len);
            sa.out_logprobs[0] =
                fb != 0 ? (key_val(fb) - fm) * sa.inv_t - logf(fs) + tail.lshift : -__builtin_inff();
        }
    }
}

template <typename WT, typename VT, int NB, int R>
dyna_status launch_lg_r(const RowdotArgs& lg, const SelectArgs& sa, void* part, int32_t* counter,
                        hipStream_t s) {
    const int64_t items = (int64_t)lg.max_chunks_bound * (kChunkRows / R);
    const int cap = option_greedy_grid() > 0 ? std::min(option_greedy_grid(), kGreedyMaxBlocks) : kGreedyGrid;
    const unsigned grid = (unsigned)std::max<int64_t>(
        1, std::min<int64_t>((items + kWavesPerBlock - 1) / kWavesPerBlock, cap));
    launch_timed_kernel(logits_greedy_kernel<WT, VT, NB, R>, dim3(grid), dim3(kThreads), 0, s, lg, sa,
                        static_cast<GreedyPartial*>(part), counter);
    return check_launch("logits_greedy_kernel");
}

template <typename WT, typename VT, int NB>
dyna_status launch_lg(const RowdotArgs& lg, const SelectArgs& sa, void* part, int32_t* counter, int rows,
                      hipStream_t s) {
    constexpr int RMAX = (sizeof(WT) == 2 ? NB : 2 * NB) <= 8 ? 4 : ((sizeof(WT) == 2 ? NB : 2 * NB) <= 16 ? 2 : 1);
    const int R = rows > 0 ? std::min(rows, RMAX) : std::min(2, RMAX);
    if (R >= 4 && RMAX >= 4) return launch_lg_r<WT, VT, NB, (RMAX >= 4 ? 4 : 1)>(lg, sa, part, counter, s);
    if (R >= 2 && RMAX >= 2) return launch_lg_r<WT, VT, NB, (RMAX >= 2 ? 2 : 1)>(lg, sa, part, counter, s);
    return launch_lg_r<WT, VT, NB, 1>(lg, sa, part, counter, s);
}

}  // namespace

size_t greedy_partials_bytes() { return sizeof(GreedyPartial) * (size_t)kGreedyMaxBlocks; }

dyna_status launch_logits_greedy(const RowdotArgs& lg, const SelectArgs& sa, void* partials,
                                 int32_t* counter, hipStream_t s) {
    const int nb = (lg.K + 511) / 512;
    const int rows = option_gemv_rows();
    if (lg.B != 1 || sa.k_t != 1) return set_error(DYNA_ERR_UNSUPPORTED, "fused head: one context, argmax");
#define DYNA_LG(N)                                                                                         \
    if (nb <= N) {                                                                                         \
        if (lg.wdtype == DYNA_BF16)                                                                        \
            return lg.vdtype == DYNA_BF16 ? launch_lg<uint16_t, uint16_t, N>(lg, sa, partials, counter, rows, s) \
                                          : launch_lg<uint16_t, float, N>(lg, sa, partials, counter, rows, s);   \
        return lg.vdtype == DYNA_BF16 ? launch_lg<float, uint16_t, N>(lg, sa, partials, counter, rows, s)        \
                                      : launch_lg<float, float, N>(lg, sa, partials, counter, rows, s);          \
    }
    DYNA_LG(1)
    DYNA_LG(2)
    DYNA_LG(4)
    DYNA_LG(8)
    DYNA_LG(12)
    DYNA_LG(16)
#undef DYNA_LG
    return set_error(DYNA_ERR_UNSUPPORTED, "fused head: d > 8192");
}

}  // namespace dyna
