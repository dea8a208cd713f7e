/*
 * libdynahead -- the dynamic vocabulary draft head of DynaSpec
 * (arXiv 2510.13847), as hand-written HIP kernels for AMD CDNA4 (gfx950).
 *
 * One draft step for B contexts (Sec. 4.2 and Sec. 4.3 of the paper,
 * Algorithm 1 in its appendix):
 *
 *   route       s_b = r(x_b)                      scores over M token clusters
 *   top-k       K_b = TopK_k(s_b)                 the k best clusters per context
 *   shortlist   S_b = disjoint union of C_m, m in K_b
 *   logits      z_b = h_b . W_LM[:, S_b]          only the shortlisted LM-head rows
 *   select      log_softmax over S_b, top-k_t / argmax / inverse-CDF sample,
 *               mapped back to vocabulary ids
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers are device pointers unless the argument says "host".  The
 *    library never allocates, frees or copies caller memory on the hot calls;
 *    scratch space comes from a caller workspace sized by dyna_workspace_bytes.
 *  - Matrices are row-major.  The paper's LM head W_LM in R^{d x |V|} is held
 *    as a [V, d] array: paper column v is row v (d contiguous elements).
 *  - Every argument check runs on the host before any HIP call; a failed
 *    check returns a status and leaves device memory untouched.
 *  - Hot-path calls (everything except dyna_build_layout) are asynchronous
 *    on the given stream and never synchronise; faults inside kernels surface
 *    at the caller's next synchronisation.
 *  - Ordering rules: every top-k breaks ties toward the lower id (cluster id
 *    when routing, vocabulary id when selecting tokens); NaN counts as -inf;
 *    -0 equals +0.  A context's shortlist is ordered by ascending cluster id,
 *    then ascending vocabulary id inside each cluster (= layout order).
 *  - Results are bit-identical from run to run (no floating-point atomics).
 *  - Calls are thread-safe for distinct workspaces; dyna_last_error() is
 *    per host thread.  The options of dyna_set_option are process-wide
 *    diagnostics for tests and measurement: set them while no other thread
 *    is calling the library.
 */
#ifndef DYNAHEAD_H
#define DYNAHEAD_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DYNA_ABI_VERSION 2
#define DYNA_MAX_M 8192     /* clusters */
#define DYNA_MAX_KT 64      /* tokens per context in top-k output */

typedef enum {
    DYNA_OK = 0,
    DYNA_ERR_INVALID_ARG = 1,  /* null pointer, bad size, bad enum, misaligned */
    DYNA_ERR_CAPACITY = 2,     /* cap smaller than the largest possible shortlist */
    DYNA_ERR_WORKSPACE = 3,    /* workspace smaller than dyna_*workspace_bytes */
    DYNA_ERR_UNSUPPORTED = 4,  /* valid request outside what the kernels handle */
    DYNA_ERR_HIP = 5,          /* a HIP runtime call or launch failed */
    DYNA_ERR_DEVICE_DATA = 6   /* device-resident input failed a check (build_layout) */
} dyna_status;

typedef enum { DYNA_F32 = 0, DYNA_BF16 = 1 } dyna_dtype;

/* Router hidden activation.  The paper's router is a two-layer FFN with ReLU
 * (Sec. 4.2, "Training the router"); SiLU is offered for routers trained so. */
typedef enum { DYNA_ACT_NONE = 0, DYNA_ACT_RELU = 1, DYNA_ACT_SILU = 2 } dyna_act;

/* Selection modes, combinable bit flags (Algorithm 1: TopK_{k_t} of the
 * log-softmax over the shortlist; sampling draws from the restricted,
 * renormalised draft q_S of Sec. 5 with tail weight beta = 0). */
enum { DYNA_SEL_ARGMAX = 1, DYNA_SEL_TOPK = 2, DYNA_SEL_SAMPLE = 4, DYNA_SEL_UNION = 8 };

/* Cluster-contiguous LM head produced once by dyna_build_layout
 * (Sec. 4.2, "Vocabulary partition": V is the disjoint union of M clusters
 * of unconstrained sizes).  Layout row j holds vocabulary id perm[j];
 * cluster m occupies rows [offsets[m], offsets[m+1]). */
typedef struct dyna_layout {
    int32_t V, d, M;
    int32_t wdtype;            /* dyna_dtype of W_perm */
    const void* W_perm;        /* device [V, d], 16-byte aligned */
    const int32_t* perm;       /* device [V] */
    const int32_t* offsets;    /* device [M + 1] */
    const int32_t* cap_by_k;   /* HOST [M + 1]: sum of the k largest cluster sizes */
    int32_t max_cluster;       /* largest cluster size */
} dyna_layout;

/* Router r: R^{d_r} -> R^M (Sec. 4.2, "Low-cost router").
 * H > 0: s = W2 . act(W1 . x + b1) + b2, W1 [H, d_r], W2 [M, H].
 * H = 0: s = W1 . x + b1, W1 [M, d_r] (a single linear map).
 * The hidden activation is kept in fp32 between the layers.  The GEMV and
 * one-launch paths use it as fp32; the matrix-core path for batches feeds it
 * to the second layer as two bf16 terms, hi + lo (16 significant bits). */
typedef struct dyna_router {
    int32_t d_r, H, M;
    int32_t wdtype;            /* dyna_dtype of W1 and W2 */
    int32_t act;               /* dyna_act (ignored when H == 0) */
    const void* W1;            /* device, 16-byte aligned */
    const float* b1;           /* device [H] (or [M] when H == 0), may be NULL */
    const void* W2;            /* device [M, H]; NULL when H == 0 */
    const float* b2;           /* device [M], may be NULL */
} dyna_router;

/* ------------------------------------------------------------------ */
/* One-time layout (Sec. 4.2, "Vocabulary partition").                  */
/* ------------------------------------------------------------------ */

size_t dyna_layout_workspace_bytes(int32_t V, int32_t M);

/* Permute the LM head so that every cluster is a contiguous slab.
 *  cluster_of [V]  device int32, cluster id of each vocabulary token
 *  W_lm [V, d]     device, dtype wdtype, row v = paper column v
 *  W_perm [V, d]   device output, row j = W_lm row perm[j]
 *  perm [V]        device output: ascending cluster id, then ascending vocabulary id
 *  offsets [M+1]   device output: CSR start of each cluster (offsets[M] = V)
 *  cap_by_k_host   HOST output [M + 1] (cap_by_k[0] = 0)
 *  max_cluster_host HOST output, may be NULL
 * Synchronises `stream` before returning.  A cluster id outside [0, M)
 * gives DYNA_ERR_DEVICE_DATA (outputs are then unspecified).  Empty clusters
 * are allowed. */
dyna_status dyna_build_layout(const int32_t* cluster_of, int32_t V, int32_t M,
                              const void* W_lm, int32_t wdtype, int32_t d,
                              void* W_perm, int32_t* perm, int32_t* offsets,
                              int32_t* cap_by_k_host, int32_t* max_cluster_host,
                              void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------ */
/* Hot path, step by step.                                             */
/* ------------------------------------------------------------------ */

/* Workspace for any of the calls below with these sizes (router may be NULL
 * when only shortlist_logits / draft_select are used).  A new workspace must
 * be zero-filled once before its first dyna_draft_head call: it holds the
 * arrival counters of the one-context kernels, which every call leaves at
 * zero.  (A one-launch step that finds them nonzero does not hang: its
 * bounded waits run out and it reports out_ids = -1.) */
size_t dyna_workspace_bytes(const dyna_layout* L, const dyna_router* r,
                            int32_t B, int32_t k, int32_t cap);

/* Route (Sec. 4.2: s = r(x), K = TopK_k(s)).
 *  x [B, d_r]          device, dtype xdtype
 *  topk_ids [B, k]     device output, cluster ids in rank order (score desc, id asc)
 *  topk_scores [B, k]  device output, may be NULL
 *  scores [B, M]       device output (fp32), may be NULL
 * 1 <= k <= M.  B = 0 is a no-op. */
dyna_status dyna_route(const dyna_router* r, const void* x, int32_t xdtype,
                       int32_t B, int32_t k, int32_t* topk_ids, float* topk_scores,
                       float* scores, void* ws, size_t ws_bytes, hipStream_t stream);

/* Shortlist (Sec. 4.2: V_S = disjoint union of C_m over m in K).
 *  topk_ids [B, k]       device, distinct cluster ids per row (any order)
 *  sel_sorted [B, k]     device output, the same ids ascending
 *  sel_rowoff [B, k+1]   device output, start of each selected cluster inside
 *                        the row's shortlist (exclusive prefix of sizes)
 *  row_len [B]           device output, shortlist length
 *  shortlist_ids [B, cap] device output, may be NULL: vocabulary ids of the
 *                        shortlist in order; entries past row_len untouched
 * An id outside [0, M) or repeated in a row is ignored (counts as an empty
 * cluster) so that the shortlist never exceeds cap_by_k[k].
 * Requires cap >= cap_by_k[k] when shortlist_ids is given. */
dyna_status dyna_shortlist(const dyna_layout* L, const int32_t* topk_ids, int32_t B,
                           int32_t k, int32_t* sel_sorted, int32_t* sel_rowoff,
                           int32_t* row_len, int32_t* shortlist_ids, int32_t cap,
                           hipStream_t stream);

/* Shortlist logits (Sec. 4.3: one gathered GEMM over the shortlisted columns;
 * Algorithm 1, FUSED_INDEX_GEMM): logits[b, j] = h_b . W_perm[row of slot j].
 *  h [B, d]            device, dtype hdtype
 *  sel_* / row_len     as written by dyna_shortlist
 *  logits [B, cap]     device output fp32; slots past row_len untouched
 * Each distinct selected slab is read from HBM once per call however many
 * contexts chose it.  Requires cap >= cap_by_k[k]. */
dyna_status dyna_shortlist_logits(const dyna_layout* L, const void* h, int32_t hdtype,
                                  int32_t B, int32_t k, const int32_t* sel_sorted,
                                  const int32_t* sel_rowoff, const int32_t* row_len,
                                  float* logits, int32_t cap, void* ws, size_t ws_bytes,
                                  hipStream_t stream);

/* Draft select (Algorithm 1: p = log_softmax(z); TopK_{k_t}(p); remap2realid).
 * Log-probabilities are those of softmax(z / temperature) over the shortlist.
 *  mode                DYNA_SEL_* flags; ARGMAX alone means k_t = 1
 *  out_ids [B, k_t]    device output, vocabulary ids, (z desc, id asc); -1 past row_len
 *  out_logprobs [B, k_t] device output, may be NULL
 *  uniforms [B]        device, u in [0, 1), required with DYNA_SEL_SAMPLE
 *  out_sample [B]      device output (SAMPLE): first j in shortlist order whose
 *                      CDF exceeds u, else the last j with nonzero mass; -1
 *                      when the shortlist is empty (only empty clusters were
 *                      selected: no token is proposed)
 *  out_sample_logprob [B] device output, may be NULL
 *  tail_beta           weight beta in [0, 1) of the tail mixture proposal
 *                      q~ = (1 - beta) q_S + beta omega (Sec. 5), omega uniform
 *                      on the row's complement V \ S; 0 gives q_S.  Top-k ids
 *                      stay in the shortlist and their log-probabilities are
 *                      those of q~.  The sample takes the shortlist branch when
 *                      u < 1 - beta (at u / (1 - beta)), else complement entry
 *                      floor((u - (1 - beta)) / beta * |V \ S|), the complement
 *                      in layout order; an empty complement (k = M) has no tail.
 *  ws                  workspace of dyna_workspace_bytes(L, NULL, B, k, cap) bytes
 * 1 <= k_t <= DYNA_MAX_KT; temperature > 0. */
dyna_status dyna_draft_select(const dyna_layout* L, const float* logits,
                              const int32_t* sel_sorted, const int32_t* sel_rowoff,
                              const int32_t* row_len, int32_t B, int32_t k, int32_t cap,
                              int32_t mode, int32_t k_t, float temperature, float tail_beta,
                              const float* uniforms, int32_t* out_ids, float* out_logprobs,
                              int32_t* out_sample, float* out_sample_logprob,
                              void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------ */
/* The whole head in one call (Algorithm 1, one draft step).           */
/* ------------------------------------------------------------------ */

/* route -> top-k -> shortlist -> logits -> select.
 *  x [B, d_r], h [B, d]  device, both of dtype adtype (x may equal h)
 *  out_clusters [B, k]   device output, may be NULL (rank order)
 *  out_logits [B, cap]   device output, may be NULL
 *  route_stream          NULL: everything runs on `stream`.  Otherwise routing
 *                        (route, top-k, shortlist) runs on route_stream so it
 *                        can overlap the caller's draft layer on `stream`
 *                        (Sec. 4.2 and Sec. 4.3: the router on a parallel
 *                        stream); the logits wait for it with an event join.
 *  x_ready               with route_stream: event after which x is valid;
 *                        NULL means "x is valid when this call is made
 *                        relative to `stream`" and the library records one.
 *  mode | DYNA_SEL_UNION the B rows of the step share one shortlist, the
 *                        union of their selected clusters (Sec. 4.2: with
 *                        several tokens at a step, the union of the clusters
 *                        predicted for each), in ascending cluster id.  Every
 *                        row's logits and selection run over the union;
 *                        out_clusters stays per row.  cap must be at least
 *                        min(V, B * cap_by_k[k]); tail_beta must be 0.
 * Other arguments as in the step-by-step calls. */
dyna_status dyna_draft_head(const dyna_router* r, const dyna_layout* L,
                            const void* x, const void* h, int32_t adtype,
                            int32_t B, int32_t k, int32_t mode, int32_t k_t,
                            float temperature, float tail_beta, const float* uniforms,
                            int32_t* out_ids, float* out_logprobs, int32_t* out_sample,
                            float* out_sample_logprob, int32_t* out_clusters,
                            float* out_logits, int32_t cap, void* ws, size_t ws_bytes,
                            hipStream_t stream, hipStream_t route_stream,
                            hipEvent_t x_ready);

/* ------------------------------------------------------------------ */
/* The whole head without a workspace.                                 */
/* ------------------------------------------------------------------ */

/* Bytes of the library's static per-GPU scratch array used by
 * dyna_draft_head_noalloc (the first 384 KiB hold the one-launch step's
 * hand-off region, the rest is the step's workspace). */
#define DYNA_NOALLOC_SCRATCH_BYTES (16u << 20)

/* dyna_draft_head for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same step, arguments and results, with no workspace argument, no
 * second routing stream (everything runs on `stream`) and no kernel-timing
 * events.  It calls no allocating routine: its scratch is a static device
 * array of DYNA_NOALLOC_SCRATCH_BYTES per GPU, held until the process ends.
 * The first call on a GPU looks the array up and clears its hand-off region
 * with a small kernel on `stream` (a plain kernel, safe under capture).
 * Every call on a GPU shares that GPU's array and may leave data in it, so
 * calls that overlap on one GPU (other streams, other host threads) race;
 * order them on one stream.  A step whose workspace (dyna_workspace_bytes)
 * exceeds DYNA_NOALLOC_SCRATCH_BYTES - 384 KiB returns DYNA_ERR_WORKSPACE:
 * one context at any shape, and batches up to the tree-batch and serving
 * shapes of the paper's settings (B = 64, k = 32 at V = 128256; B = 16, k =
 * 64 at V = 151936) fit. */
dyna_status dyna_draft_head_noalloc(const dyna_router* r, const dyna_layout* L,
                                    const void* x, const void* h, int32_t adtype,
                                    int32_t B, int32_t k, int32_t mode, int32_t k_t,
                                    float temperature, float tail_beta, const float* uniforms,
                                    int32_t* out_ids, float* out_logprobs, int32_t* out_sample,
                                    float* out_sample_logprob, int32_t* out_clusters,
                                    float* out_logits, int32_t cap, hipStream_t stream);

/* ------------------------------------------------------------------ */
/* Baselines on the same kernels (Sec. 4.1).                           */
/* ------------------------------------------------------------------ */

size_t dyna_dense_workspace_bytes(int32_t n_rows, int32_t B);

/* Head over the contiguous rows [0, n_rows) of W [>= n_rows, d]: the dense
 * full-vocabulary head O = H W_LM when n_rows = V, and the static
 * fixed-shortlist head (FR-Spec's W~ = W_LM[:, V_high], here the first
 * n_rows ids) otherwise.  Token ids are row indices.  out_logits [B, n_rows]
 * may be NULL.  Selection as in dyna_draft_select. */
dyna_status dyna_dense_head(const void* W, int32_t wdtype, int32_t n_rows, int32_t d,
                            const void* h, int32_t hdtype, int32_t B, int32_t mode,
                            int32_t k_t, float temperature, const float* uniforms,
                            int32_t* out_ids, float* out_logprobs, int32_t* out_sample,
                            float* out_sample_logprob, float* out_logits,
                            void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------ */
/* Beam expansion (Algorithm 1: cu_scores, TopK_{k_t}).                */
/* ------------------------------------------------------------------ */

/* Cumulative scores cu[b, r] = logprobs[b, r] + last_scores[b] of the B x k_t
 * candidates of a step (the draft selection's outputs), and the n_out
 * largest of them, ordered (cu desc, b asc, r asc): the next beam.
 *  logprobs [B, k_t], ids [B, k_t]  device, as written by the draft head
 *                                   (a candidate with id < 0 is never chosen)
 *  last_scores [B]                  device, may be NULL (zeros: the first step)
 *  out_scores, out_parent, out_ids [n_out]  device outputs: cu, the row b the
 *                                   candidate extends, its token id; -inf, -1,
 *                                   -1 past the number of candidates
 * 1 <= k_t, n_out <= DYNA_MAX_KT; B * k_t <= 8192.  One workgroup. */
dyna_status dyna_beam_expand(const float* logprobs, const int32_t* ids, const float* last_scores,
                             int32_t B, int32_t k_t, int32_t n_out, float* out_scores,
                             int32_t* out_parent, int32_t* out_ids, hipStream_t stream);

/* ------------------------------------------------------------------ */
/* Building the partition: spherical k-means (Sec. 4.2, "Vocabulary   */
/* partition": clusters from spherical k-means on the column-          */
/* normalised LM head, one point per vocabulary entry).                */
/* ------------------------------------------------------------------ */

/* Shared argument meaning:
 *  W [V, d]    device, bf16 (DYNA_BF16 only), row-major, 16-byte aligned;
 *              row v is the paper's column v.  The points are W[v] / ||W[v]||
 *              (an all-zero row is a point with no direction).
 *  centroids   device fp32 [M, d], unit rows.
 * Similarities are taken with the centroids rounded to bf16 (the matrix
 * cores' operand type) and accumulated in fp32.  d % 8 == 0, d <= 8192,
 * 1 <= M <= min(V, DYNA_MAX_M).  ws: dyna_kmeans_workspace_bytes(V, d, M)
 * bytes of device memory, caller-owned. */
size_t dyna_kmeans_workspace_bytes(int32_t V, int32_t d, int32_t M);

/* Assignment step: out_assign[v] = argmax_m x_v . mu_m (ties to the lower
 * m); out_score[v] (optional, may be NULL) = W[v] . bf16(mu_m) for that m, the
 * raw row's product (the unit point's is this times 1 / ||W[v]||).
 * Asynchronous on `stream`.  This is the launch DYNA_OPT_KERNEL_TIMING
 * brackets for the builder. */
dyna_status dyna_kmeans_assign(const void* W, int32_t wdtype, int32_t V, int32_t d, const float* centroids,
                               int32_t M, int32_t* out_assign, float* out_score, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/* Update step, in place: centroids[m] = (sum of the unit points with
 * assign[v] == m, in ascending v) / its norm, summed in fp32; a cluster
 * with no points or a zero sum keeps its row.  Assignments outside [0, M)
 * are skipped.  Asynchronous on `stream`. */
dyna_status dyna_kmeans_update(const void* W, int32_t wdtype, int32_t V, int32_t d, const int32_t* assign,
                               int32_t M, float* centroids, void* ws, size_t ws_bytes, hipStream_t stream);

/* The whole builder: centroids start at the points init_ids[0..M) (device,
 * distinct ids in [0, V), drawn by the caller), then `iters` (>= 1) rounds
 * of assignment followed by update.  out_cluster_of [V] (device) receives
 * the last assignment, the partition that dyna_build_layout takes;
 * out_centroids (device fp32 [M, d], optional) the centroids after the last
 * update.  Synchronises `stream`; an init id outside [0, V) returns
 * DYNA_ERR_DEVICE_DATA (its centroid is zero). */
dyna_status dyna_kmeans(const void* W, int32_t wdtype, int32_t V, int32_t d, int32_t M, const int32_t* init_ids,
                        int32_t iters, int32_t* out_cluster_of, float* out_centroids, void* ws, size_t ws_bytes,
                        hipStream_t stream);

/* ------------------------------------------------------------------ */
/* Position-aware budgets (host functions, no GPU work).               */
/* ------------------------------------------------------------------ */

/* Cluster budget k_c(t) at draft position t (Sec. 4.2, eq. pos_schedule):
 * k0 at t = 0, k1 at t = 1, then floor((k1 + t) / (2t)) (form 0), or the
 * appendix algorithm's floor(k1 / (2t)) (form 1, its loop index read as the
 * draft position).  The result is clamped below at k_min: the text bounds
 * k_c(t) by k_min while both formulas reach 0 for large t.  Returns -1 for
 * t < 0, k0 < 1, k1 < 1, k_min < 1 or another form.  The value is the k a
 * caller passes to dyna_draft_head for that position. */
int32_t dyna_cluster_budget(int32_t t, int32_t k0, int32_t k1, int32_t k_min, int32_t form);

/* Shortlist size K_fr(t) of the position-aware frequency-ranked static head
 * (appendix, PA-FR): k_max for t in {0, 1}, then floor(k_max / (t + 1)).
 * Returns -1 for t < 0 or k_max < 1.  The value is the n_rows a caller
 * passes to dyna_dense_head for the static head at that position. */
int32_t dyna_static_budget(int32_t t, int32_t k_max);

/* ------------------------------------------------------------------ */
/* Diagnostics.                                                        */
/* ------------------------------------------------------------------ */

/* Kernel-path override for tests and measurement:
 * DYNA_OPT_LOGITS_PATH: 0 automatic, 1 wave-per-row GEMV, 2 MFMA tiles with
 *   the slab rows staged through LDS (bf16 weights and contexts; other types
 *   take the GEMV).
 * DYNA_OPT_ROUTER_PATH: 0 automatic, 1 GEMV, 2 split-K MFMA with the contexts
 *   staged in LDS (bf16 weights, up to 128 contexts; else 3), 3 MFMA tiles
 *   loaded straight from HBM.
 * DYNA_OPT_KERNEL_TIMING: 1 brackets every launch of the gathered-head
 *   (logits) kernel, and the k-means assignment, with two (default) events recorded on the stream it runs
 *   on; 2 hands the two events to the dispatch itself (hipExtLaunchKernelGGL);
 *   0 stops.
 * DYNA_OPT_GEMV_ROWS: rows each wave of the GEMV kernel keeps in flight:
 *   0 automatic, else 1, 2 or 4 (capped by the register budget).
 * DYNA_OPT_FUSED_B1: how dyna_draft_head runs a one-context step without
 *   sampling (argmax, or top-k_t with k_t <= 16).
 *   0 (default): one launch (router, top-k, shortlist, gathered logits and
 *   selection, the workgroups handing the hidden layer, the router scores
 *   and their partial results to each other inside the launch) when the
 *   router, LM head and activations are all bf16, d, d_r, H <= 8192,
 *   M <= 1024, V < 2^21, the step's LDS fits in 160 KB, routing stays on
 *   `stream` and the occupancy calculator finds room for the whole grid at
 *   once (its workgroups hand words to each other); otherwise as 2.
 *   2: four launches (router layer 1; router layer 2; top-k with shortlist
 *   and plan; gathered head fused with selection).  1: the separate
 *   kernels.  3: the one launch only; a step it cannot run returns
 *   DYNA_ERR_UNSUPPORTED (for tests and measurement that must know which
 *   form ran).  All forms give identical clusters, logits and ids;
 *   log-probabilities agree to rounding (the softmax sum is taken in
 *   another order).
 *   Under kernel timing the one-launch step, or the fused gathered-head +
 *   selection launch, is what is timed.
 * DYNA_OPT_MFMA_UNROLL: k steps the direct-load MFMA kernel (router path 3,
 *   and dense heads of fp32 contexts) loads ahead: 0 automatic (8), 4, 8 or 16.
 * DYNA_OPT_GATHER_CFG: shape of the LDS-staged MFMA kernel (path 2): 0
 *   automatic (slab rows staged through LDS, contexts loaded into
 *   registers, two workgroups of two waves per compute unit); 1..4 other
 *   shapes of the same kernel (waves per workgroup, ring stages, k columns
 *   per stage); 5..9 shapes whose waves split the k dimension of one chunk
 *   (for short shortlists; a shape whose split would leave a wave without
 *   k columns runs unsplit).
 * DYNA_OPT_GREEDY_GRID: workgroups of the fused one-context gathered head:
 *   0 automatic (256), else 1..4096; of the one-launch step: 0 automatic (one
 *   per compute unit), else that many, capped at 1024 and at what the
 *   occupancy calculator says can be resident at once.
 * DYNA_OPT_UNION_CFG: shape of the dense union-row kernel of
 *   DYNA_SEL_UNION steps: 0 automatic (up to 16 rows over a row stride of at
 *   most 65536 slots take the per-chunk gathered kernel instead), 1..15
 *   fixed (waves per workgroup, row tiles per wave, k columns per stage, ring
 *   depth; always the dense kernel); a shape whose ring does not fit in LDS
 *   for the batch's context count returns DYNA_ERR_UNSUPPORTED.
 * DYNA_OPT_KMEANS_CFG: shape of the k-means assignment kernel: 0
 *   automatic, 1..7 fixed.
 * DYNA_OPT_WAIT_BOUND_US: bound of every wait of the one-launch step, in
 *   microseconds of wall clock: 0 (default) 200000, 1..1000000 that many,
 *   -1 none (a wait gives up at its first read that finds a word missing;
 *   for tests of the failure path).  A step in which a wait gave up reports
 *   out_ids = -1 and out_logprobs = -inf.  The error word carries the epoch
 *   of the launch that set it, so a later step is not failed by it; only a
 *   workgroup of a failed launch that started after the failure was
 *   reported fails the next step too, which may read its stale words. */
enum { DYNA_OPT_LOGITS_PATH = 1, DYNA_OPT_ROUTER_PATH = 2, DYNA_OPT_KERNEL_TIMING = 3,
       DYNA_OPT_GEMV_ROWS = 4, DYNA_OPT_FUSED_B1 = 5, DYNA_OPT_MFMA_UNROLL = 6,
       DYNA_OPT_GATHER_CFG = 7, DYNA_OPT_GREEDY_GRID = 8, DYNA_OPT_UNION_CFG = 9,
       DYNA_OPT_KMEANS_CFG = 10, DYNA_OPT_WAIT_BOUND_US = 11 };
dyna_status dyna_set_option(int32_t option, int32_t value);

/* Waits for the events recorded under DYNA_OPT_KERNEL_TIMING and returns the
 * summed duration (ms) and number of timed launches since the last reset.
 * reset != 0 forgets them afterwards.  Host call; synchronises the events. */
dyna_status dyna_kernel_timing(double* total_ms, int64_t* launches, int32_t reset);

int32_t dyna_abi_version(void);
const char* dyna_status_string(dyna_status status);
/* Detail of the last non-OK status returned to this host thread. */
const char* dyna_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* DYNAHEAD_H */
