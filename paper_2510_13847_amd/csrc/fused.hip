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
#include "greedy.h"
#include "select_row.h"

namespace dyna {
namespace {

constexpr int kGreedyGrid = 256;  // default workgroups of the fused one-context head (one arrival each)

struct GreedyEpi {
    float inv_t;
    GreedyState st;
    __device__ __forceinline__ void idle() {}
    __device__ __forceinline__ void put(const RowdotArgs& a, int64_t o, float value, int32_t vid) {
        a.out[o] = value;
        if (a.vid_out) a.vid_out[o] = vid;
        st.add(value, vid, inv_t);
    }
};

template <typename WT, typename VT, int NB, int R>
__global__ __launch_bounds__(kThreads) void logits_greedy_kernel(RowdotArgs lg, SelectArgs sa,
                                                                 GreedyPartial* part, int32_t* counter) {
    const int64_t n_items = (int64_t)lg.plan.hdr->n_chunks * (kChunkRows / R);
    // workgroups whose first wave has an item take part (at least workgroup 0)
    const int64_t n_part = std::max<int64_t>(
        1, std::min<int64_t>(gridDim.x, (n_items + kWavesPerBlock - 1) / kWavesPerBlock));
    if ((int64_t)blockIdx.x >= n_part) return;

    GreedyEpi epi{sa.inv_t};
    gemv_rows<WT, VT, NB, true, R, true, GreedyEpi>(lg, epi);

    GreedyState f;
    if (!greedy_publish_merge<kThreads>(epi.st, sa.inv_t, part, blockIdx.x, (int)n_part, counter, &f)) return;
    if (threadIdx.x == 0) {
        const uint64_t fb = f.best;
        if (sa.out_ids) sa.out_ids[0] = fb != 0 ? (int32_t)key_id(fb) : -1;
        if (sa.out_logprobs) {
            const TailMix tail = tail_of(sa, sa.row_len ? sa.row_len[0] : sa.fixed_len);
            sa.out_logprobs[0] =
                fb != 0 ? (key_val(fb) - f.m) * sa.inv_t - logf(f.s) + tail.lshift : -__builtin_inff();
        }
    }
}

// ---------------------------------------------------------------- top-k_t
// The same fused head for TopK_{k_t} with k_t <= kTopkMax: every wave keeps
// its kTopkMax best keys (spread over its lanes) next to the lanes' online
// softmax pairs; a workgroup publishes its k_t best keys and its pair, and
// the last workgroup to arrive takes the k_t best of all published keys.
constexpr int kTopkMax = kFusedTopkMax;

struct TopkPartial {
    uint64_t key[kTopkMax];
    float m, s;
};

// Epilogue of the one-context top-k head: lanes below R own the rows of a
// group (one context: one row per lane per group); their keys are listed at
// the next group's idle point, while its loads are in flight.
template <int R>
struct TopkEpi {
    float inv_t;
    uint64_t wk = 0;    // this lane's place of the wave's list
    uint64_t pend = 0;  // key of the row this lane produced last (0: none)
    float m = -__builtin_inff(), s = 0.0f;
    __device__ __forceinline__ void idle() {
        // branch-free: an empty key 0 leaves the list as it is
#pragma unroll
        for (int r = 0; r < R; ++r) wk = row_list_insert(wk, readlane_u64(pend, r));
        pend = 0;
    }
    __device__ __forceinline__ void put(const RowdotArgs& a, int64_t o, float value, int32_t vid) {
        a.out[o] = value;
        if (a.vid_out) a.vid_out[o] = vid;
        const float z = value != value ? -__builtin_inff() : value;
        pend = sel_key(z, (uint32_t)vid);
        softmax_merge(m, s, z, 1.0f, inv_t);
    }
};

template <typename WT, typename VT, int NB, int R>
__global__ __launch_bounds__(kThreads) void logits_topk_kernel(RowdotArgs lg, SelectArgs sa, TopkPartial* part,
                                                               int32_t* counter) {
    constexpr int NW = kThreads / kWave;
    __shared__ uint64_t heads[kThreads];
    __shared__ uint64_t cand[kTopkMax * kTopkMax];
    __shared__ uint64_t top[kTopkMax];
    __shared__ float w_m[NW], w_s[NW], f_m, f_s;
    __shared__ int last;
    const int64_t n_items = (int64_t)lg.plan.hdr->n_chunks * (kChunkRows / R);
    const int64_t n_part = std::max<int64_t>(
        1, std::min<int64_t>(gridDim.x, (n_items + kWavesPerBlock - 1) / kWavesPerBlock));
    if ((int64_t)blockIdx.x >= n_part) return;
    const int k_t = sa.k_t;

    TopkEpi<R> epi;
    epi.inv_t = sa.inv_t;
    gemv_rows<WT, VT, NB, true, R, true, TopkEpi<R>>(lg, epi);
    epi.idle();

    // the workgroup's k_t best keys (the k_t best of its waves' lists, ranked
    // by counting) and softmax pair, published device-coherent
    {
        const int lane = lane_id(), w = threadIdx.x / kWave;
        if ((int)threadIdx.x < k_t) top[threadIdx.x] = 0;
        if (lane < k_t) cand[w * k_t + lane] = epi.wk;
        __syncthreads();
        if ((int)threadIdx.x < NW * k_t) {
            const uint64_t key = cand[threadIdx.x];
            int rank = 0;
            for (int j = 0; j < NW * k_t; ++j) rank += cand[j] > key;
            if (key != 0 && rank < k_t) top[rank] = key;
        }
        __syncthreads();
    }
    block_softmax_pair<kThreads>(epi.m, epi.s, sa.inv_t, w_m, w_s, &f_m, &f_s);
    TopkPartial* mine = part + blockIdx.x;
    if ((int)threadIdx.x < k_t) store_coherent(&mine->key[threadIdx.x], top[threadIdx.x]);
    if (threadIdx.x == 0) {
        store_coherent(&mine->m, f_m);
        store_coherent(&mine->s, f_s);
    }
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);  // this thread's stores have completed
    __syncthreads();
    if (threadIdx.x == 0)
        last = __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == n_part - 1;
    __syncthreads();
    if (!last) return;

    // last workgroup: thread t merges the lists of partials t, t + NT, ... into
    // its own sorted list, then the k_t best over the threads; the softmax
    // pairs in partial order
    if (threadIdx.x == 0) store_coherent(counter, 0);
    uint64_t list[kTopkMax];
#pragma unroll
    for (int r = 0; r < kTopkMax; ++r) list[r] = 0;
    float bm = -__builtin_inff(), bs = 0.0f;
    for (int64_t g = threadIdx.x; g < n_part; g += kThreads) {
        // all of the partial's loads in flight at once, then the merge
        uint64_t pk[kTopkMax];
#pragma unroll
        for (int r = 0; r < kTopkMax; ++r) pk[r] = r < k_t ? load_coherent(&part[g].key[r]) : 0;
        const float m2 = load_coherent(&part[g].m), s2 = load_coherent(&part[g].s);
        if (g == threadIdx.x) {
#pragma unroll
            for (int r = 0; r < kTopkMax; ++r) list[r] = pk[r];
        } else {
            for (int r = 0; r < k_t; ++r) {
                if (pk[r] <= list[kTopkMax - 1]) break;  // the partial's list is sorted
                list[kTopkMax - 1] = pk[r];
#pragma unroll
                for (int q = kTopkMax - 1; q > 0; --q)
                    if (list[q] > list[q - 1]) {
                        const uint64_t t = list[q];
                        list[q] = list[q - 1];
                        list[q - 1] = t;
                    }
            }
        }
        softmax_merge(bm, bs, m2, s2, sa.inv_t);
    }
    block_topk_lists<kTopkMax, kThreads>(list, k_t, heads, cand, top);
    block_softmax_pair<kThreads>(bm, bs, sa.inv_t, w_m, w_s, &f_m, &f_s);
    __syncthreads();
    const TailMix tail = tail_of(sa, sa.row_len ? sa.row_len[0] : sa.fixed_len);
    const float log_total = logf(f_s) - tail.lshift;
    for (int r = threadIdx.x; r < k_t; r += kThreads) {
        const uint64_t key = top[r];
        if (sa.out_ids) sa.out_ids[r] = key != 0 ? (int32_t)key_id(key) : -1;
        if (sa.out_logprobs)
            sa.out_logprobs[r] = key != 0 ? (key_val(key) - f_m) * sa.inv_t - log_total : -__builtin_inff();
    }
}

template <typename WT, typename VT, int NB, int R>
dyna_status launch_lg_r(const RowdotArgs& lg, const SelectArgs& sa, void* part, int32_t* counter,
                        hipStream_t s) {
    const int64_t items = (int64_t)lg.max_chunks_bound * (kChunkRows / R);
    const int cap = option_greedy_grid() > 0 ? std::min(option_greedy_grid(), kGreedyMaxBlocks) : kGreedyGrid;
    const unsigned grid = (unsigned)std::max<int64_t>(
        1, std::min<int64_t>((items + kWavesPerBlock - 1) / kWavesPerBlock, cap));
    if (sa.k_t > 1) {
        launch_timed_kernel(logits_topk_kernel<WT, VT, NB, R>, dim3(grid), dim3(kThreads), 0, s, lg, sa,
                            static_cast<TopkPartial*>(part), counter);
        return check_launch("logits_topk_kernel");
    }
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

size_t greedy_partials_bytes() {
    return std::max(sizeof(GreedyPartial), sizeof(TopkPartial)) * (size_t)kGreedyMaxBlocks;
}

dyna_status launch_logits_greedy(const RowdotArgs& lg, const SelectArgs& sa, void* partials,
                                 int32_t* counter, hipStream_t s) {
    const int nb = (lg.K + 511) / 512;
    const int rows = option_gemv_rows();
    if (lg.B != 1 || sa.k_t < 1 || sa.k_t > kTopkMax)
        return set_error(DYNA_ERR_UNSUPPORTED, "fused head: one context, k_t <= %d", kTopkMax);
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
