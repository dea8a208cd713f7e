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
