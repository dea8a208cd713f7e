// Internal declarations shared by the libdynahead translation units.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "dynahead.h"

namespace dyna {

constexpr int kWave = 64;
constexpr int kMaxDevices = 64;   // per-device tables of the library
constexpr int kMfmaRows = 16;     // rows of one MFMA A tile
// Layout rows per work chunk of the gathered head: one MFMA tile, so every
// chunk is a full work item of equal cost (partial only at a cluster's end).
constexpr int kChunkRows = kMfmaRows;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// A work chunk of the gathered head: up to kChunkRows consecutive layout rows
// of one cluster and the list of contexts that selected that cluster.
struct Chunk {
    int32_t r0;        // first layout row
    int32_t nrows;     // rows in this chunk (1..kChunkRows)
    int32_t list_off;  // first entry of the cluster's context list
    int32_t list_cnt;  // number of contexts that selected the cluster
};

// One context that selected a cluster: its row b and the shortlist slot of
// layout row r, which is slot_base + r.
struct ListEntry {
    int32_t b;
    int32_t slot_base;
};

// Device-side header of a plan; counts are written by the plan kernels.
struct PlanHeader {
    int32_t n_chunks;
    int32_t n_entries;
    int32_t pad[62];
};

// Views into a caller workspace for the gathered head.
struct Plan {
    PlanHeader* hdr;
    Chunk* chunks;       // [max_chunks]
    ListEntry* list;     // [max_entries]
    int32_t max_chunks;
    int32_t max_entries;
};

// Events for the next gathered-head launch on this host thread (kernel
// timing): stamped by the dispatch itself, so they bracket the kernel only.
struct LaunchEvents {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
};
LaunchEvents& pending_launch_events();

template <typename K, typename... Args>
void launch_timed_kernel(K kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t stream,
                         Args... args) {
    LaunchEvents& ev = pending_launch_events();
    if (ev.start != nullptr) {
        hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, ev.start, ev.stop, 0u, args...);
        ev = LaunchEvents{};
    } else {
        kernel<<<grid, block, shmem, stream>>>(args...);
    }
}

// Launch error -> status with a message.
dyna_status set_error(dyna_status s, const char* fmt, ...);
dyna_status check_launch(const char* what);

// ---------------- launchers (defined in the .hip files) ----------------

// layout.hip
dyna_status launch_build_layout(const int32_t* cluster_of, int32_t V, int32_t M,
                                const void* W_lm, int32_t wdtype, int32_t d, void* W_perm,
                                int32_t* perm, int32_t* offsets, void* ws, size_t ws_bytes,
                                int32_t* host_offsets_out, hipStream_t stream);
size_t layout_ws_bytes(int32_t V, int32_t M);

// rowdot.hip: out[b * ld + base_b + row] = act(sum_k W[row, k] * v[b, k] + bias[row])
struct RowdotArgs {
    const void* W;          // [rows, K]
    int32_t wdtype;
    int32_t K;
    const void* v;          // [B, K] (row stride K)
    int32_t vdtype;
    int32_t B;
    float* out;
    int64_t ld;             // output row stride (per context)
    const float* bias;      // [rows] or nullptr
    int32_t act;            // dyna_act
    // dense mode: rows [0, n_rows), every context, base 0
    int32_t n_rows;
    // plan mode (when plan.hdr != nullptr): chunks and context lists
    Plan plan;
    int32_t max_chunks_bound;  // host-known upper bound on plan chunks
    // plan mode, optional: vid_out[b * ld + slot] = perm[layout row of slot]
    const int32_t* perm;
    int32_t* vid_out;
    // optional: block 0 clears these words first (arrival counters that the
    // next kernels of the step use)
    int32_t* zero_words;
    int32_t n_zero_words;
    // split-K router, optional: fp32 contexts given as the previous layer's
    // split-K partial sums; context c's element k is act(sum over slices s,
    // in slice order, of vpart[(s * B + c) * K + k], + vbias[k]), the value
    // that layer's reduction would have written (v is then unused)
    const float* vpart;
    int32_t vslices;
    const float* vbias;
    int32_t vact;
};

dyna_status launch_rowdot(const RowdotArgs& a, int path, hipStream_t stream);

// router.hip: dense layers for 1..128 contexts as split-K MFMA workgroups
// (contexts staged in LDS) plus a fixed-order reduction with bias and
// activation; `part` holds the per-slice partial sums.
struct SplitShape {
    int nw;         // waves (16 rows each) per workgroup
    int groups;     // 16-context MFMA column groups
    int tiles;      // 16-row tiles per wave
    int row_tiles;  // workgroups along the rows
    int ksl;        // k-slice length
    int slices;     // workgroups along k
    size_t lds;     // staged contexts, bytes
};
bool splitk_shape(int32_t n_rows, int32_t K, int32_t B, bool vf32, SplitShape* out);
size_t splitk_part_floats(int32_t n_rows, int32_t K, int32_t B, bool vf32);
// deferred_slices != nullptr: the slices' partial sums stay in `part`
// ([slices][B][n_rows]) and *deferred_slices receives the slice count; the
// consumer adds them in slice order and then the bias (no activation).
dyna_status launch_dense_splitk(const RowdotArgs& a, float* part, size_t part_floats, hipStream_t stream,
                                int* deferred_slices = nullptr);

// gather.hip: plan mode with bf16 weights and contexts, slab rows staged
// through LDS (MFMA tiles)
bool gather_lds_eligible(const RowdotArgs& a);
dyna_status launch_gather_lds(const RowdotArgs& a, hipStream_t stream);
// union rows (every plan chunk lists contexts 0..B-1 in order): dense
// LDS-staged MFMA product; vid_out gets one shared row [slots]
dyna_status launch_union_gemm(const RowdotArgs& a, hipStream_t stream);
// Plan over rows [0, V): one chunk per 16 rows, every chunk shared by all B
// contexts (one list entry, slot base 0), so the union kernel computes the
// dense product of the rows with every context.
dyna_status launch_full_plan(int32_t V, int32_t B, const Plan& plan, hipStream_t stream);
// The same product with an argmax epilogue: every plan row against the B
// contexts (centroids); vid_out[slot] = the best context (ties to the lower
// id), out[slot] = its product (out may be null).
dyna_status launch_union_argmax(const RowdotArgs& a, int cfg, hipStream_t stream);
// kmeans.hip: spherical k-means over the LM-head rows
size_t kmeans_ws_bytes(int32_t V, int32_t d, int32_t M);
dyna_status kmeans_assign(const void* W, int32_t V, int32_t d, const float* centroids, int32_t M,
                          int32_t* out_assign, float* out_score, void* ws, hipStream_t stream);
dyna_status kmeans_update(const void* W, int32_t V, int32_t d, const int32_t* assign, int32_t M,
                          float* centroids, void* ws, hipStream_t stream);
dyna_status kmeans_run(const void* W, int32_t V, int32_t d, int32_t M, const int32_t* init_ids, int32_t iters,
                       int32_t* out_cluster_of, float* out_centroids, void* ws, hipStream_t stream);
int option_kmeans_cfg();
// layout.hip: stable counting sort of ids in [0, M) (others skipped): perm and
// CSR offsets; ws holds layout_ws_bytes(V, M)
dyna_status launch_cluster_csr(const int32_t* cluster_of, int32_t V, int32_t M, int32_t* perm,
                               int32_t* offsets, void* ws, hipStream_t stream);

// Arguments of the per-context top-k (Sec. 4.2) and of the draft selection
// (Algorithm 1), shared by the separate and the fused launches.
struct TopkArgs {
    const float* scores;   // [B, M]
    // part set: the scores are the sum of `slices` split-K partial sums
    // part[slice][B][M] in slice order, plus bias[M] (if set)
    const float* part;
    int slices;
    const float* bias;
    int M, k;
    int32_t* topk_ids;     // [B, k] rank order
    float* topk_scores;    // [B, k] or nullptr
    const int32_t* offsets;  // [M + 1] (shortlist)
    int32_t* sel_sorted;   // [B, k] or nullptr: no shortlist
    int32_t* sel_rowoff;   // [B, k + 1]
    int32_t* row_len;      // [B]
    Plan plan;             // hdr == nullptr: no plan (one context only)
};

struct SelectArgs {
    const float* logits;
    int64_t ld;
    const int32_t* row_len;   // nullptr: every row has fixed_len
    int32_t fixed_len;
    const int32_t* sel_sorted;
    const int32_t* sel_rowoff;
    const int32_t* offsets;
    const int32_t* perm;      // nullptr: vocabulary id = slot
    const int32_t* slot_vid;  // optional [B][vid_ld]: vocabulary id per slot
    int64_t vid_ld;           // row stride of slot_vid (0: one row shared by all)
    int32_t k;
    int32_t k_t;
    float inv_t;
    const float* uniforms;
    float beta;               // tail weight of the mixture proposal (0: none)
    int32_t V;                // vocabulary rows (the complement is V - row length)
    int32_t P;                // segments per row
    int32_t seg;              // slots per segment
    // partials, [B][P][...]
    uint64_t* pkeys;          // [B][P][k_t]
    float* pmax;              // [B][P]
    float* psum;              // [B][P]
    int32_t* out_ids;
    float* out_logprobs;
    int32_t* out_sample;
    float* out_sample_logprob;
};

// select.hip
struct ScoreSlices {  // split-K partial sums the top-k adds up itself
    const float* part = nullptr;
    int slices = 0;
    const float* bias = nullptr;
};
dyna_status launch_topk_clusters(const float* scores, int32_t B, int32_t M, int32_t k,
                                 int32_t* topk_ids, float* topk_scores,
                                 // optional fused shortlist outputs (all or none)
                                 const int32_t* offsets, int32_t* sel_sorted,
                                 int32_t* sel_rowoff, int32_t* row_len,
                                 // with one context, also write the gathered-head plan
                                 const Plan* plan, hipStream_t stream,
                                 const ScoreSlices& slices = ScoreSlices{});
dyna_status launch_shortlist(const int32_t* offsets, const int32_t* perm, int32_t M,
                             const int32_t* topk_ids, int32_t B, int32_t k,
                             int32_t* sel_sorted, int32_t* sel_rowoff, int32_t* row_len,
                             int32_t* shortlist_ids, int32_t cap, hipStream_t stream);
dyna_status launch_plan(const int32_t* offsets, int32_t M, const int32_t* sel_sorted,
                        const int32_t* sel_rowoff, int32_t B, int32_t k, Plan plan,
                        hipStream_t stream);
dyna_status launch_select(const float* logits, int64_t ld, const int32_t* row_len,
                          int32_t fixed_len, int32_t max_len, const int32_t* sel_sorted,
                          const int32_t* sel_rowoff, const int32_t* offsets,
                          const int32_t* perm, int32_t B, int32_t k, int32_t k_t,
                          float temperature, float beta, int32_t V, const float* uniforms, int32_t* out_ids,
                          float* out_logprobs, int32_t* out_sample,
                          float* out_sample_logprob, void* ws, hipStream_t stream,
                          // optional [B, vid_ld]: vocabulary id of every slot (written
                          // by the gathered head); saves the layout walk.  vid_ld < 0
                          // means ld; 0 means one row shared by every context row
                          const int32_t* slot_vid = nullptr, int64_t vid_ld = -1,
                          // rows longer than 16384 slots take the segmented select
                          // (many workgroups per row) instead of one workgroup per row
                          bool split_long = false);
// Workspace for launch_select with rows of at most max_len slots.
size_t select_ws_bytes(int32_t B, int32_t max_len, int32_t k_t);
// Longest row launch_select handles (256 segments).
int32_t select_max_len();
// Union plan: the rows' top-k clusters -> one shared shortlist (ascending
// cluster id), its chunk table with every row listed, row_len[b] = |union|,
// and the union's cluster ids in sel_u[0 .. u_cap) (-1 past its end).
dyna_status launch_union_plan(const int32_t* offsets, int32_t M, const int32_t* topk_ids, int32_t B, int32_t k,
                              int32_t* row_len, int32_t* sel_u, int32_t u_cap, Plan plan, bool compact,
                              hipStream_t stream);
dyna_status launch_beam_expand(const float* logprobs, const int32_t* ids, const float* last, int32_t B, int32_t k_t,
                               int32_t n_out, float* out_scores, int32_t* out_parent, int32_t* out_ids,
                               hipStream_t stream);
// Fill SelectArgs for rows of at most max_len slots; ws as for launch_select.
SelectArgs make_select_args(const float* logits, int64_t ld, const int32_t* row_len,
                            int32_t fixed_len, int32_t max_len, const int32_t* sel_sorted,
                            const int32_t* sel_rowoff, const int32_t* offsets,
                            const int32_t* perm, int32_t B, int32_t k, int32_t k_t,
                            float temperature, float beta, int32_t V, const float* uniforms, int32_t* out_ids,
                            float* out_logprobs, int32_t* out_sample,
                            float* out_sample_logprob, void* ws, const int32_t* slot_vid,
                            int64_t vid_ld = -1);
// True when the one-workgroup select handles rows of max_len slots.
bool select_row_fits(int32_t max_len, bool fixed, int32_t k_t, int32_t k);

// fused.hip (one context, argmax or top-k_t up to kFusedTopkMax): gathered
// head + selection with per-workgroup online-softmax partials; `counter` is
// zero on entry.
constexpr int kGreedyMaxBlocks = 4096;
constexpr int kFusedTopkMax = 16;
size_t greedy_partials_bytes();
dyna_status launch_logits_greedy(const RowdotArgs& lg, const SelectArgs& sa, void* partials,
                                 int32_t* counter, hipStream_t s);

// chain.hip (one context, argmax or top-k_t, bf16 throughout): the whole
// step in one launch, handing words between workgroups through an
// epoch-tagged region.
struct ChainRequest {
    bool all_bf16;  // router weights, LM head, x and h all bf16
    const void* W1;
    const float* b1;
    const void* W2;
    const float* b2;
    int32_t d_r, H, M, act;
    const void* x;
    const void* W;
    const int32_t* perm;
    const int32_t* offsets;
    int32_t d, V;
    const void* h;
    int32_t k;
    void* region;  // chain_region_bytes(H, M) of workspace, zero-filled before first use
    int32_t* out_clusters;
    float* topk_scores;
    int32_t* sel_sorted;
    int32_t* sel_rowoff;
    int32_t* row_len;
    float* out_logits;
    int32_t* out_ids;       // [k_t]
    float* out_logprobs;    // [k_t]
    int32_t k_t;            // 1 (argmax) .. 16
    float inv_t, beta;
};
size_t chain_region_bytes(int32_t H, int32_t M);
bool chain_step_eligible(const ChainRequest& q);
// Grid the one-launch step takes on the current device (capped at what can
// be resident at once), or 0 when it cannot run co-resident; fills the wall
// clock rate (kHz) for the wait bounds.
int chain_step_grid(const ChainRequest& q, int64_t* tick_khz);
dyna_status launch_chain_step(const ChainRequest& q, hipStream_t s);

// The whole head behind dyna_draft_head and its allocation-free variant:
// `chain_region` (may be null) replaces the workspace's hand-off region of
// the one-launch step; `timing` allows DYNA_OPT_KERNEL_TIMING's events.
dyna_status draft_head_core(const dyna_router* r, const dyna_layout* L, const void* x, const void* h,
                            int32_t adtype, int32_t B, int32_t k, int32_t mode, int32_t k_t, float temperature,
                            float tail_beta, const float* uniforms, int32_t* out_ids, float* out_logprobs,
                            int32_t* out_sample, float* out_sample_logprob, int32_t* out_clusters,
                            float* out_logits, int32_t cap, void* ws, size_t ws_bytes, hipStream_t stream,
                            hipStream_t route_stream, hipEvent_t x_ready, void* chain_region, bool timing);

// Global options (dyna_set_option).
int option_logits_path();
int option_router_path();
int option_gemv_rows();
int option_mfma_unroll();
int option_gather_cfg();
int option_greedy_grid();
int option_union_cfg();

}  // namespace dyna
