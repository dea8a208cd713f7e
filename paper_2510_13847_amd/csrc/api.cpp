// C ABI of libdynahead: argument checks, workspace carving, stream joins.
// Every check runs on the host before the first HIP call of an entry point.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <utility>
#include <vector>

#include "dyna_internal.h"

#define DYNA_API extern "C" __attribute__((visibility("default")))

namespace dyna {

namespace {
thread_local char g_last_error[512] = "";
std::atomic<int> g_logits_path{0};
std::atomic<int> g_router_path{0};
std::atomic<int> g_kernel_timing{0};
std::atomic<int> g_gemv_rows{0};
std::atomic<int> g_fused_off{0};
std::atomic<int> g_mfma_unroll{0};
std::atomic<int> g_gather_cfg{0};
std::atomic<int> g_greedy_grid{0};
std::atomic<int> g_union_cfg{0};
std::atomic<int> g_kmeans_cfg{0};
std::atomic<int> g_wait_bound_us{0};

// event pairs around timed gathered-head launches
std::mutex g_timing_mu;
std::vector<std::pair<hipEvent_t, hipEvent_t>> g_timing_pairs;
std::vector<hipEvent_t> g_timing_free;

thread_local hipEvent_t g_ev_x[kMaxDevices];
thread_local hipEvent_t g_ev_join[kMaxDevices];

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool valid_dtype(int32_t t) { return t == DYNA_F32 || t == DYNA_BF16; }
int elt_size(int32_t t) { return t == DYNA_BF16 ? 2 : 4; }
}  // namespace

dyna_status set_error(dyna_status s, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return s;
}

dyna_status check_launch(const char* what) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return set_error(DYNA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return DYNA_OK;
}

int option_logits_path() { return g_logits_path.load(); }

LaunchEvents& pending_launch_events() {
    static thread_local LaunchEvents ev;
    return ev;
}

static hipEvent_t timing_event() {
    std::lock_guard<std::mutex> g(g_timing_mu);
    if (!g_timing_free.empty()) {
        hipEvent_t e = g_timing_free.back();
        g_timing_free.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// Launch the gathered-head kernel, optionally between two timing events.
template <typename F>
static dyna_status timed(F launch, hipStream_t s) {
    (void)s;
    if (!g_kernel_timing.load()) return launch();
    hipEvent_t e0 = timing_event(), e1 = timing_event();
    if (!e0 || !e1) return set_error(DYNA_ERR_HIP, "kernel timing: event creation failed");
    if (g_kernel_timing.load() == 2) {
        // start/stop events handed to the gathered-head dispatch itself
        pending_launch_events() = LaunchEvents{e0, e1};
        dyna_status st = launch();
        const bool taken = pending_launch_events().start == nullptr;
        pending_launch_events() = LaunchEvents{};
        if (st != DYNA_OK) return st;
        if (!taken) return set_error(DYNA_ERR_HIP, "kernel timing: launch did not take the events");
    } else {
        if (hipEventRecord(e0, s) != hipSuccess) return set_error(DYNA_ERR_HIP, "kernel timing: event record failed");
        dyna_status st = launch();
        if (st != DYNA_OK) return st;
        if (hipEventRecord(e1, s) != hipSuccess) return set_error(DYNA_ERR_HIP, "kernel timing: event record failed");
    }
    std::lock_guard<std::mutex> g(g_timing_mu);
    g_timing_pairs.emplace_back(e0, e1);
    return DYNA_OK;
}

static dyna_status timed_rowdot(const RowdotArgs& a, int path, hipStream_t s) {
    return timed([&] { return launch_rowdot(a, path, s); }, s);
}
int option_router_path() { return g_router_path.load(); }
int option_gemv_rows() { return g_gemv_rows.load(); }
int option_mfma_unroll() { return g_mfma_unroll.load(); }
int option_gather_cfg() { return g_gather_cfg.load(); }
int option_greedy_grid() { return g_greedy_grid.load(); }
int option_union_cfg() { return g_union_cfg.load(); }
int option_kmeans_cfg() { return g_kmeans_cfg.load(); }
int option_wait_bound_us() { return g_wait_bound_us.load(); }

// ------------------------------------------------------------------ workspace
// One carving serves every hot entry point, so a single workspace can back a
// whole step; each call only touches its own regions.
struct Carve {
    float* hidden = nullptr;      // [B, H]
    float* scores = nullptr;      // [B, M]
    int32_t* topk_ids = nullptr;  // [B, k]
    float* topk_scores = nullptr; // [B, k]
    int32_t* sel_sorted = nullptr;// [B, k]
    int32_t* sel_rowoff = nullptr;// [B, k + 1]
    int32_t* row_len = nullptr;   // [B]
    float* logits = nullptr;      // [B, cap]
    int32_t* slot_vid = nullptr;  // [B, cap]
    int32_t* counters = nullptr;  // [4] arrival counters (and error word) of the fused one-context kernels
    void* partials = nullptr;     // partials of the fused one-context head
    void* chain = nullptr;        // tagged hand-off region of the one-launch step
    Plan plan{};
    float* rpart = nullptr;  // split-K partial sums of the router layers
    size_t rpart_floats = 0;
    void* select_ws = nullptr;
    size_t bytes = 0;
};

static int64_t max_chunks_for(const dyna_layout* L) {
    return ((int64_t)L->V + kChunkRows - 1) / kChunkRows + L->M;
}

// 5..16 contexts: router layer 2 stages the hidden layer straight from layer
// 1's split-K partial sums, so layer 1 needs no reduction launch (both
// layers' partial sums then share the workspace side by side; the workspace
// is sized for it whatever the router-path option says).
constexpr int32_t kHiddenFromPartsMaxB = 16;
static bool hidden_from_parts(const dyna_router* r, int32_t xdtype, int32_t B, size_t* f1, size_t* f2,
                              bool sizing = false) {
    if (r->H == 0 || B <= 4 || B > kHiddenFromPartsMaxB || r->wdtype != DYNA_BF16 ||
        (!sizing && option_router_path() != 0))
        return false;
    SplitShape s1, s2;
    if (!splitk_shape(r->H, r->d_r, B, xdtype == DYNA_F32, &s1) || !splitk_shape(r->M, r->H, B, true, &s2))
        return false;
    *f1 = (size_t)s1.slices * (size_t)B * (size_t)r->H;
    *f2 = (size_t)s2.slices * (size_t)B * (size_t)r->M;
    return true;
}

// Chunks a step can produce: the union of the selected slabs holds at most
// min(V, B * cap_by_k[k]) rows in at most min(M, B * k) clusters, and each
// cluster adds at most one partial chunk.
static int32_t chunk_bound(const dyna_layout* L, int32_t B, int32_t k) {
    const int64_t rows = std::min<int64_t>(L->V, (int64_t)B * L->cap_by_k[k]);
    const int64_t clusters = std::min<int64_t>(L->M, (int64_t)B * k);
    return (int32_t)std::min<int64_t>(max_chunks_for(L), rows / kChunkRows + clusters + 1);
}

static Carve carve(const dyna_layout* L, const dyna_router* r, int32_t B, int32_t k, int32_t cap,
                   void* base) {
    Carve c;
    char* p = static_cast<char*>(base);
    size_t off = 0;
    auto take = [&](size_t n) -> void* {
        void* q = p ? p + off : nullptr;
        off += align256(n);
        return q;
    };
    const int64_t Bl = B;
    const int32_t M = L ? L->M : (r ? r->M : 0);
    if (r && r->H > 0) c.hidden = static_cast<float*>(take(sizeof(float) * Bl * r->H));
    if (r) {
        // either input type of layer 1 (fp32 inputs use shorter slices)
        const int32_t n1 = r->H > 0 ? r->H : r->M;
        size_t f = std::max(splitk_part_floats(n1, r->d_r, B, false), splitk_part_floats(n1, r->d_r, B, true));
        if (r->H > 0) f = std::max(f, splitk_part_floats(r->M, r->H, B, true));
        // both layers' partial sums at once (either input type of layer 1)
        size_t f1 = 0, f2 = 0, g1 = 0, g2 = 0;
        if (hidden_from_parts(r, DYNA_BF16, B, &f1, &f2, true)) f = std::max(f, f1 + f2);
        if (hidden_from_parts(r, DYNA_F32, B, &g1, &g2, true)) f = std::max(f, g1 + g2);
        c.rpart_floats = f;
        if (f > 0) c.rpart = static_cast<float*>(take(sizeof(float) * f));
    }
    c.scores = static_cast<float*>(take(sizeof(float) * Bl * M));
    c.topk_ids = static_cast<int32_t*>(take(sizeof(int32_t) * Bl * k));
    c.topk_scores = static_cast<float*>(take(sizeof(float) * Bl * k));
    c.sel_sorted = static_cast<int32_t*>(take(sizeof(int32_t) * Bl * k));
    c.sel_rowoff = static_cast<int32_t*>(take(sizeof(int32_t) * Bl * (k + 1)));
    c.row_len = static_cast<int32_t*>(take(sizeof(int32_t) * Bl));
    c.logits = static_cast<float*>(take(sizeof(float) * Bl * cap));
    c.slot_vid = static_cast<int32_t*>(take(sizeof(int32_t) * Bl * cap));
    c.counters = static_cast<int32_t*>(take(4 * sizeof(int32_t)));
    if (B == 1) c.partials = take(greedy_partials_bytes());
    if (B == 1 && r) c.chain = take(chain_region_bytes(r->H, r->M));
    if (L) {
        c.plan.max_chunks = (int32_t)max_chunks_for(L);
        // per-row lists (B * k entries) or the union's (every row in each
        // of at most min(M, B * k) clusters)
        c.plan.max_entries = (int32_t)std::max<int64_t>(Bl * k, std::min<int64_t>(L->M, Bl * k) * Bl);
        c.plan.hdr = static_cast<PlanHeader*>(take(sizeof(PlanHeader)));
        c.plan.chunks = static_cast<Chunk*>(take(sizeof(Chunk) * (size_t)c.plan.max_chunks));
        c.plan.list = static_cast<ListEntry*>(take(sizeof(ListEntry) * (size_t)c.plan.max_entries));
    }
    c.select_ws = take(select_ws_bytes(B, cap, DYNA_MAX_KT));
    c.bytes = off;
    return c;
}

// ------------------------------------------------------------------ checks
#define REQUIRE(cond, ...) \
    do {                   \
        if (!(cond)) return set_error(DYNA_ERR_INVALID_ARG, __VA_ARGS__); \
    } while (0)

static dyna_status check_layout(const dyna_layout* L) {
    REQUIRE(L != nullptr, "layout is NULL");
    REQUIRE(L->V >= 1 && L->d >= 8 && L->M >= 1, "layout: bad sizes V=%d d=%d M=%d", L->V, L->d, L->M);
    REQUIRE(L->M <= L->V, "layout: M=%d > V=%d", L->M, L->V);
    if (L->M > DYNA_MAX_M)
        return set_error(DYNA_ERR_UNSUPPORTED, "layout: M=%d > DYNA_MAX_M=%d", L->M, DYNA_MAX_M);
    REQUIRE(valid_dtype(L->wdtype), "layout: bad wdtype %d", L->wdtype);
    REQUIRE(L->d % 8 == 0, "layout: d=%d is not a multiple of 8", L->d);
    if (L->d > 8192) return set_error(DYNA_ERR_UNSUPPORTED, "layout: d=%d > 8192", L->d);
    REQUIRE(L->W_perm && L->perm && L->offsets && L->cap_by_k, "layout: NULL array");
    REQUIRE(aligned16(L->W_perm), "layout: W_perm not 16-byte aligned");
    REQUIRE(L->max_cluster >= 1 && L->max_cluster <= L->V, "layout: bad max_cluster %d", L->max_cluster);
    return DYNA_OK;
}

static dyna_status check_router(const dyna_router* r) {
    REQUIRE(r != nullptr, "router is NULL");
    REQUIRE(r->d_r >= 8 && r->M >= 1 && r->H >= 0, "router: bad sizes d_r=%d H=%d M=%d", r->d_r, r->H, r->M);
    REQUIRE(r->d_r % 8 == 0, "router: d_r=%d is not a multiple of 8", r->d_r);
    REQUIRE(r->H % 8 == 0, "router: H=%d is not a multiple of 8", r->H);
    if (r->d_r > 8192 || r->H > 8192)
        return set_error(DYNA_ERR_UNSUPPORTED, "router: d_r or H > 8192");
    if (r->M > DYNA_MAX_M) return set_error(DYNA_ERR_UNSUPPORTED, "router: M > DYNA_MAX_M");
    REQUIRE(valid_dtype(r->wdtype), "router: bad wdtype %d", r->wdtype);
    REQUIRE(r->act == DYNA_ACT_NONE || r->act == DYNA_ACT_RELU || r->act == DYNA_ACT_SILU,
            "router: bad act %d", r->act);
    REQUIRE(r->W1 != nullptr && aligned16(r->W1), "router: W1 NULL or not 16-byte aligned");
    if (r->H > 0) REQUIRE(r->W2 != nullptr && aligned16(r->W2), "router: W2 NULL or not 16-byte aligned");
    return DYNA_OK;
}

static dyna_status check_k(const dyna_layout* L, int32_t k) {
    REQUIRE(k >= 1 && k <= L->M, "k=%d outside [1, M=%d]", k, L->M);
    return DYNA_OK;
}

static dyna_status check_cap(const dyna_layout* L, int32_t k, int32_t cap) {
    if (cap < L->cap_by_k[k])
        return set_error(DYNA_ERR_CAPACITY, "cap=%d < cap_by_k[%d]=%d", cap, k, L->cap_by_k[k]);
    if (cap > select_max_len())
        return set_error(DYNA_ERR_UNSUPPORTED, "cap=%d > %d", cap, select_max_len());
    return DYNA_OK;
}

static dyna_status check_select(int32_t mode, int32_t* k_t, float temperature, const float* uniforms,
                                const int32_t* out_ids, const int32_t* out_sample) {
    REQUIRE(mode > 0 && (mode & ~(DYNA_SEL_ARGMAX | DYNA_SEL_TOPK | DYNA_SEL_SAMPLE)) == 0,
            "bad select mode %d", mode);
    if (mode & DYNA_SEL_TOPK) {
        REQUIRE(*k_t >= 1 && *k_t <= DYNA_MAX_KT, "k_t=%d outside [1, %d]", *k_t, DYNA_MAX_KT);
    } else {
        *k_t = 1;  // argmax, or the max needed by sampling
    }
    if (mode & (DYNA_SEL_TOPK | DYNA_SEL_ARGMAX)) REQUIRE(out_ids != nullptr, "out_ids is NULL");
    if (mode & DYNA_SEL_SAMPLE) {
        REQUIRE(uniforms != nullptr && out_sample != nullptr, "sampling needs uniforms and out_sample");
        REQUIRE(temperature > 0.0f && temperature < 3.0e38f, "temperature must be positive and finite");
    }
    return DYNA_OK;
}

#define TRY(expr)                                   \
    do {                                            \
        dyna_status _s = (expr);                    \
        if (_s != DYNA_OK) return _s;               \
    } while (0)

// ------------------------------------------------------------------ pieces
// One router layer.  Path: 0 automatic (GEMV for up to 4 contexts, else
// split-K MFMA), 1 GEMV, 2 split-K MFMA, 3 MFMA tiles with direct loads.
// With `defer` set, a split-K layer leaves its partial sums for the top-k
// to add (defer->part stays null when the layer runs another way).
static dyna_status run_layer(const RowdotArgs& a, int path, float* part, size_t part_floats, hipStream_t s,
                             ScoreSlices* defer = nullptr) {
    const bool splitk = (path == 2 || (path == 0 && a.B > 4)) && a.wdtype == DYNA_BF16 && part != nullptr &&
                        splitk_part_floats(a.n_rows, a.K, a.B, a.vdtype == DYNA_F32) > 0;
    if (splitk && defer != nullptr && a.act == DYNA_ACT_NONE) {
        int slices = 0;
        TRY(launch_dense_splitk(a, part, part_floats, s, &slices));
        defer->part = part;
        defer->slices = slices;
        defer->bias = a.bias;
        return DYNA_OK;
    }
    if (splitk) return launch_dense_splitk(a, part, part_floats, s);
    return launch_rowdot(a, path >= 2 ? 3 : path, s);
}

static dyna_status run_router(const dyna_router* r, const void* x, int32_t xdtype, int32_t B,
                              float* scores, float* hidden, float* part, size_t part_floats, hipStream_t s,
                              int32_t* zero_words = nullptr, ScoreSlices* defer = nullptr) {
    const int path = option_router_path();
    RowdotArgs a{};
    a.zero_words = zero_words;  // cleared by block 0 of the first router kernel
    a.n_zero_words = zero_words ? 4 : 0;
    a.W = r->W1;
    a.wdtype = r->wdtype;
    a.K = r->d_r;
    a.v = x;
    a.vdtype = xdtype;
    a.B = B;
    if (r->H == 0) {
        a.out = scores;
        a.ld = r->M;
        a.bias = r->b1;
        a.act = DYNA_ACT_NONE;
        a.n_rows = r->M;
        return run_layer(a, path, part, part_floats, s, defer);
    }
    a.out = hidden;
    a.ld = r->H;
    a.bias = r->b1;
    a.act = r->act;
    a.n_rows = r->H;
    size_t f1 = 0, f2 = 0;
    if (part != nullptr && hidden_from_parts(r, xdtype, B, &f1, &f2) && f1 + f2 <= part_floats) {
        // layer 1's slices stay in part[0, f1); layer 2 adds them up (in slice
        // order, then bias and activation) while staging its contexts
        RowdotArgs a1 = a;
        a1.act = DYNA_ACT_NONE;
        a1.bias = nullptr;
        int slices1 = 0;
        TRY(launch_dense_splitk(a1, part, f1, s, &slices1));
        RowdotArgs b{};
        b.W = r->W2;
        b.wdtype = r->wdtype;
        b.K = r->H;
        b.v = hidden;  // unused: the contexts come from the partial sums
        b.vdtype = DYNA_F32;
        b.vpart = part;
        b.vslices = slices1;
        b.vbias = r->b1;
        b.vact = r->act;
        b.B = B;
        b.out = scores;
        b.ld = r->M;
        b.bias = r->b2;
        b.act = DYNA_ACT_NONE;
        b.n_rows = r->M;
        float* part2 = part + f1;
        if (defer != nullptr) {
            int slices2 = 0;
            TRY(launch_dense_splitk(b, part2, part_floats - f1, s, &slices2));
            defer->part = part2;
            defer->slices = slices2;
            defer->bias = b.bias;
            return DYNA_OK;
        }
        return launch_dense_splitk(b, part2, part_floats - f1, s);
    }
    TRY(run_layer(a, path, part, part_floats, s));
    RowdotArgs b{};
    b.W = r->W2;
    b.wdtype = r->wdtype;
    b.K = r->H;
    b.v = hidden;
    b.vdtype = DYNA_F32;
    b.B = B;
    b.out = scores;
    b.ld = r->M;
    b.bias = r->b2;
    b.act = DYNA_ACT_NONE;
    b.n_rows = r->M;
    return run_layer(b, path, part, part_floats, s, defer);
}

// Path of a gathered head with per-row shortlists: the option when set, else
// the wave-per-row GEMV for up to 32 contexts and the LDS-staged MFMA tiles
// beyond.  The GEMV's 1 KiB row loads stream better when a slab row serves
// few contexts: measured 4-12 us less per step at 8-48 contexts on the
// Llama-3-8B head and 6-7 us at 16 contexts on the Qwen- and Gemma-shaped
// heads; equal at 32 and 32 us more at 64 contexts on the Gemma-shaped head.
constexpr int32_t kGemvMaxContexts = 32;
static int gathered_path(int32_t B) {
    const int opt = option_logits_path();
    if (opt != 0) return opt;
    return B <= kGemvMaxContexts ? 1 : 0;
}

static dyna_status run_logits(const dyna_layout* L, const void* h, int32_t hdtype, int32_t B, int32_t k,
                              const int32_t* sel_sorted, const int32_t* sel_rowoff, float* logits,
                              int32_t cap, const Plan& plan, hipStream_t s) {
    TRY(launch_plan(L->offsets, L->M, sel_sorted, sel_rowoff, B, k, plan, s));
    RowdotArgs a{};
    a.W = L->W_perm;
    a.wdtype = L->wdtype;
    a.K = L->d;
    a.v = h;
    a.vdtype = hdtype;
    a.B = B;
    a.out = logits;
    a.ld = cap;
    a.bias = nullptr;
    a.act = DYNA_ACT_NONE;
    a.n_rows = 0;
    a.plan = plan;
    a.max_chunks_bound = chunk_bound(L, B, k);
    return timed_rowdot(a, gathered_path(B), s);
}

static hipEvent_t lazy_event(hipEvent_t* table) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    if (table[dev] == nullptr) {
        hipEvent_t e = nullptr;
        if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return nullptr;
        table[dev] = e;
    }
    return table[dev];
}

}  // namespace dyna

using namespace dyna;

// ====================================================================== ABI
DYNA_API int32_t dyna_abi_version(void) { return DYNA_ABI_VERSION; }

DYNA_API const char* dyna_status_string(dyna_status s) {
    switch (s) {
        case DYNA_OK: return "DYNA_OK";
        case DYNA_ERR_INVALID_ARG: return "DYNA_ERR_INVALID_ARG";
        case DYNA_ERR_CAPACITY: return "DYNA_ERR_CAPACITY";
        case DYNA_ERR_WORKSPACE: return "DYNA_ERR_WORKSPACE";
        case DYNA_ERR_UNSUPPORTED: return "DYNA_ERR_UNSUPPORTED";
        case DYNA_ERR_HIP: return "DYNA_ERR_HIP";
        case DYNA_ERR_DEVICE_DATA: return "DYNA_ERR_DEVICE_DATA";
    }
    return "unknown dyna_status";
}

DYNA_API const char* dyna_last_error(void) { return g_last_error; }

DYNA_API dyna_status dyna_set_option(int32_t option, int32_t value) {
    if (option == DYNA_OPT_MFMA_UNROLL) {
        REQUIRE(value == 0 || value == 4 || value == 8 || value == 16, "MFMA unroll %d not in {0, 4, 8, 16}", value);
        g_mfma_unroll.store(value);
        return DYNA_OK;
    }
    if (option == DYNA_OPT_GREEDY_GRID) {
        REQUIRE(value >= 0 && value <= kGreedyMaxBlocks, "greedy grid %d outside [0, %d]", value, kGreedyMaxBlocks);
        g_greedy_grid.store(value);
        return DYNA_OK;
    }
    if (option == DYNA_OPT_WAIT_BOUND_US) {
        REQUIRE(value >= -1 && value <= 1000000, "wait bound %d us outside [-1, 1000000]", value);
        g_wait_bound_us.store(value);
        return DYNA_OK;
    }
    if (option == DYNA_OPT_KMEANS_CFG) {
        REQUIRE(value >= 0 && value <= 7, "k-means shape %d outside [0, 7]", value);
        g_kmeans_cfg.store(value);
        return DYNA_OK;
    }
    if (option == DYNA_OPT_UNION_CFG) {
        REQUIRE(value >= 0 && value <= 15, "union shape %d outside [0, 15]", value);
        g_union_cfg.store(value);
        return DYNA_OK;
    }
    if (option == DYNA_OPT_GATHER_CFG) {
        REQUIRE(value >= 0 && value <= 9, "gather shape %d outside [0, 9]", value);
        g_gather_cfg.store(value);
        return DYNA_OK;
    }
    if (option == DYNA_OPT_LOGITS_PATH) {
        REQUIRE(value >= 0 && value <= 2, "logits path %d outside [0, 2]", value);
        g_logits_path.store(value);
        return DYNA_OK;
    }
    if (option == DYNA_OPT_FUSED_B1) {
        REQUIRE(value >= 0 && value <= 3, "fused option %d not in {0, 1, 2, 3}", value);
        g_fused_off.store(value);
        return DYNA_OK;
    }
    if (option == DYNA_OPT_GEMV_ROWS) {
        REQUIRE(value == 0 || value == 1 || value == 2 || value == 4, "GEMV rows %d not in {0,1,2,4}", value);
        g_gemv_rows.store(value);
        return DYNA_OK;
    }
    if (option == DYNA_OPT_ROUTER_PATH) {
        REQUIRE(value >= 0 && value <= 3, "router path %d outside [0, 3]", value);
        g_router_path.store(value);
        return DYNA_OK;
    }
    REQUIRE(value >= 0 && value <= 2, "option value %d outside [0, 2]", value);
    if (option == DYNA_OPT_KERNEL_TIMING) g_kernel_timing.store(value);
    else return set_error(DYNA_ERR_INVALID_ARG, "unknown option %d", option);
    return DYNA_OK;
}

DYNA_API dyna_status dyna_kernel_timing(double* total_ms, int64_t* launches, int32_t reset) {
    REQUIRE(total_ms != nullptr && launches != nullptr, "NULL argument");
    std::lock_guard<std::mutex> g(g_timing_mu);
    double sum = 0.0;
    dyna_status st = DYNA_OK;
    for (auto& pr : g_timing_pairs) {
        float ms = 0.0f;
        if (hipEventSynchronize(pr.second) != hipSuccess ||
            hipEventElapsedTime(&ms, pr.first, pr.second) != hipSuccess) {
            (void)hipGetLastError();
            st = set_error(DYNA_ERR_HIP, "kernel timing: elapsed time query failed");
            break;
        }
        sum += ms;
    }
    *total_ms = st == DYNA_OK ? sum : 0.0;
    *launches = st == DYNA_OK ? (int64_t)g_timing_pairs.size() : 0;
    if (reset) {
        for (auto& pr : g_timing_pairs) {
            g_timing_free.push_back(pr.first);
            g_timing_free.push_back(pr.second);
        }
        g_timing_pairs.clear();
    }
    return st;
}

DYNA_API size_t dyna_layout_workspace_bytes(int32_t V, int32_t M) {
    if (V < 1 || M < 1) return 0;
    return layout_ws_bytes(V, M);
}

DYNA_API dyna_status dyna_build_layout(const int32_t* cluster_of, int32_t V, int32_t M,
                                       const void* W_lm, int32_t wdtype, int32_t d, void* W_perm,
                                       int32_t* perm, int32_t* offsets, int32_t* cap_by_k_host,
                                       int32_t* max_cluster_host, void* ws, size_t ws_bytes,
                                       hipStream_t stream) {
    REQUIRE(cluster_of && W_lm && W_perm && perm && offsets && cap_by_k_host && ws, "NULL argument");
    REQUIRE(V >= 1 && M >= 1 && M <= V, "bad sizes V=%d M=%d", V, M);
    if (M > DYNA_MAX_M) return set_error(DYNA_ERR_UNSUPPORTED, "M=%d > DYNA_MAX_M", M);
    REQUIRE(valid_dtype(wdtype), "bad wdtype %d", wdtype);
    REQUIRE(d >= 8 && d % 8 == 0, "d=%d must be a positive multiple of 8", d);
    REQUIRE(aligned16(W_lm) && aligned16(W_perm), "W_lm / W_perm not 16-byte aligned");
    REQUIRE(W_lm != W_perm, "W_perm must not alias W_lm");
    if (ws_bytes < layout_ws_bytes(V, M))
        return set_error(DYNA_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, layout_ws_bytes(V, M));
    std::vector<int32_t> off(M + 1);
    TRY(launch_build_layout(cluster_of, V, M, W_lm, wdtype, d, W_perm, perm, offsets, ws, ws_bytes,
                            off.data(), stream));
    std::vector<int32_t> sizes(M);
    for (int m = 0; m < M; ++m) sizes[m] = off[m + 1] - off[m];
    std::sort(sizes.begin(), sizes.end(), [](int a, int b) { return a > b; });
    cap_by_k_host[0] = 0;
    for (int m = 0; m < M; ++m) cap_by_k_host[m + 1] = cap_by_k_host[m] + sizes[m];
    if (max_cluster_host) *max_cluster_host = sizes[0];
    return DYNA_OK;
}

DYNA_API size_t dyna_workspace_bytes(const dyna_layout* L, const dyna_router* r, int32_t B, int32_t k,
                                     int32_t cap) {
    if (B < 0 || k < 1 || cap < 0 || (!L && !r)) return 0;
    return carve(L, r, B, k, cap, nullptr).bytes;
}

DYNA_API dyna_status dyna_route(const dyna_router* r, const void* x, int32_t xdtype, int32_t B, int32_t k,
                                int32_t* topk_ids, float* topk_scores, float* scores, void* ws,
                                size_t ws_bytes, hipStream_t stream) {
    TRY(check_router(r));
    REQUIRE(B >= 0, "B=%d < 0", B);
    REQUIRE(k >= 1 && k <= r->M, "k=%d outside [1, M=%d]", k, r->M);
    REQUIRE(valid_dtype(xdtype), "bad xdtype %d", xdtype);
    if (B == 0) return DYNA_OK;
    REQUIRE(x != nullptr && aligned16(x) && topk_ids != nullptr, "x / topk_ids NULL or x misaligned");
    REQUIRE(ws != nullptr, "workspace is NULL");
    const Carve c0 = carve(nullptr, r, B, k, 0, nullptr);
    if (ws_bytes < c0.bytes) return set_error(DYNA_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, c0.bytes);
    const Carve c = carve(nullptr, r, B, k, 0, ws);
    float* sc = scores ? scores : c.scores;
    TRY(run_router(r, x, xdtype, B, sc, c.hidden, c.rpart, c.rpart_floats, stream));
    return launch_topk_clusters(sc, B, r->M, k, topk_ids, topk_scores, nullptr, nullptr, nullptr,
                                nullptr, nullptr, stream);
}

DYNA_API dyna_status dyna_shortlist(const dyna_layout* L, const int32_t* topk_ids, int32_t B, int32_t k,
                                    int32_t* sel_sorted, int32_t* sel_rowoff, int32_t* row_len,
                                    int32_t* shortlist_ids, int32_t cap, hipStream_t stream) {
    TRY(check_layout(L));
    TRY(check_k(L, k));
    REQUIRE(B >= 0, "B=%d < 0", B);
    if (B == 0) return DYNA_OK;
    REQUIRE(topk_ids && sel_sorted && sel_rowoff && row_len, "NULL argument");
    if (shortlist_ids) TRY(check_cap(L, k, cap));
    return launch_shortlist(L->offsets, L->perm, L->M, topk_ids, B, k, sel_sorted, sel_rowoff, row_len,
                            shortlist_ids, cap, stream);
}

DYNA_API dyna_status dyna_shortlist_logits(const dyna_layout* L, const void* h, int32_t hdtype, int32_t B,
                                           int32_t k, const int32_t* sel_sorted, const int32_t* sel_rowoff,
                                           const int32_t* row_len, float* logits, int32_t cap, void* ws,
                                           size_t ws_bytes, hipStream_t stream) {
    TRY(check_layout(L));
    TRY(check_k(L, k));
    REQUIRE(B >= 0, "B=%d < 0", B);
    REQUIRE(valid_dtype(hdtype), "bad hdtype %d", hdtype);
    TRY(check_cap(L, k, cap));
    if (B == 0) return DYNA_OK;
    REQUIRE(h && aligned16(h) && sel_sorted && sel_rowoff && row_len && logits && ws,
            "NULL argument or h misaligned");
    const Carve c0 = carve(L, nullptr, B, k, cap, nullptr);
    if (ws_bytes < c0.bytes) return set_error(DYNA_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, c0.bytes);
    const Carve c = carve(L, nullptr, B, k, cap, ws);
    return run_logits(L, h, hdtype, B, k, sel_sorted, sel_rowoff, logits, cap, c.plan, stream);
}

DYNA_API dyna_status dyna_draft_select(const dyna_layout* L, const float* logits, const int32_t* sel_sorted,
                                       const int32_t* sel_rowoff, const int32_t* row_len, int32_t B, int32_t k,
                                       int32_t cap, int32_t mode, int32_t k_t, float temperature,
                                       float tail_beta, const float* uniforms, int32_t* out_ids,
                                       float* out_logprobs,
                                       int32_t* out_sample, float* out_sample_logprob, void* ws,
                                       size_t ws_bytes, hipStream_t stream) {
    TRY(check_layout(L));
    TRY(check_k(L, k));
    TRY(check_cap(L, k, cap));
    TRY(check_select(mode, &k_t, temperature, uniforms, out_ids, out_sample));
    REQUIRE(tail_beta >= 0.0f && tail_beta < 1.0f, "tail_beta must lie in [0, 1)");
    REQUIRE(B >= 0, "B=%d < 0", B);
    if (B == 0) return DYNA_OK;
    REQUIRE(logits && sel_sorted && sel_rowoff && row_len && ws, "NULL argument");
    const Carve c0 = carve(L, nullptr, B, k, cap, nullptr);
    if (ws_bytes < c0.bytes) return set_error(DYNA_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, c0.bytes);
    const Carve c = carve(L, nullptr, B, k, cap, ws);
    const bool want_ids = (mode & (DYNA_SEL_ARGMAX | DYNA_SEL_TOPK)) != 0;
    const bool want_sample = (mode & DYNA_SEL_SAMPLE) != 0;
    return launch_select(logits, cap, row_len, 0, cap, sel_sorted, sel_rowoff, L->offsets, L->perm, B, k,
                         k_t, temperature, tail_beta, L->V, want_sample ? uniforms : nullptr,
                         want_ids ? out_ids : nullptr,
                         want_ids ? out_logprobs : nullptr, want_sample ? out_sample : nullptr,
                         want_sample ? out_sample_logprob : nullptr, c.select_ws, stream);
}

namespace dyna {

// The whole head (dyna_draft_head).  `chain_region`, when set, is the
// one-launch step's tagged hand-off region (at a fixed address, so its
// epoch survives calls of different shapes) in place of the workspace's own;
// `timing` lets DYNA_OPT_KERNEL_TIMING bracket the gathered head with events.
dyna_status draft_head_core(const dyna_router* r, const dyna_layout* L, const void* x, const void* h,
                            int32_t adtype, int32_t B, int32_t k, int32_t mode, int32_t k_t, float temperature,
                            float tail_beta, const float* uniforms, int32_t* out_ids, float* out_logprobs,
                            int32_t* out_sample, float* out_sample_logprob, int32_t* out_clusters,
                            float* out_logits, int32_t cap, void* ws, size_t ws_bytes, hipStream_t stream,
                            hipStream_t route_stream, hipEvent_t x_ready, void* chain_region, bool timing) {
    auto timed = [&](auto launch, hipStream_t s) -> dyna_status {
        return timing ? dyna::timed(launch, s) : launch();
    };
    auto timed_rowdot = [&](const RowdotArgs& a, int path, hipStream_t s) -> dyna_status {
        return timed([&] { return launch_rowdot(a, path, s); }, s);
    };
    TRY(check_router(r));
    TRY(check_layout(L));
    REQUIRE(r->M == L->M, "router M=%d differs from layout M=%d", r->M, L->M);
    REQUIRE(r->d_r > 0, "router d_r");
    TRY(check_k(L, k));
    const bool union_mode = (mode & DYNA_SEL_UNION) != 0 && B > 1;  // one row: its own shortlist
    mode &= ~DYNA_SEL_UNION;
    if (union_mode) {
        const int64_t bound = std::min<int64_t>(L->V, (int64_t)B * L->cap_by_k[k]);
        if (cap < bound)
            return set_error(DYNA_ERR_CAPACITY, "union: cap=%d < min(V, B * cap_by_k[k])=%lld", cap,
                             (long long)bound);
        if (cap > select_max_len()) return set_error(DYNA_ERR_UNSUPPORTED, "union: cap=%d > %d", cap, select_max_len());
        if (tail_beta > 0.0f) return set_error(DYNA_ERR_UNSUPPORTED, "union: no tail mixture");
    } else {
        TRY(check_cap(L, k, cap));
    }
    TRY(check_select(mode, &k_t, temperature, uniforms, out_ids, out_sample));
    REQUIRE(tail_beta >= 0.0f && tail_beta < 1.0f, "tail_beta must lie in [0, 1)");
    REQUIRE(valid_dtype(adtype), "bad adtype %d", adtype);
    REQUIRE(B >= 0, "B=%d < 0", B);
    if (B == 0) return DYNA_OK;
    REQUIRE(x && h && aligned16(x) && aligned16(h) && ws, "NULL argument or x/h misaligned");
    const Carve c0 = carve(L, r, B, k, cap, nullptr);
    if (ws_bytes < c0.bytes) return set_error(DYNA_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, c0.bytes);
    const Carve c = carve(L, r, B, k, cap, ws);

    hipStream_t rs = route_stream ? route_stream : stream;
    const bool split = rs != stream;
    if (split) {
        hipEvent_t ready = x_ready;
        if (ready == nullptr) {
            ready = lazy_event(g_ev_x);
            if (!ready || hipEventRecord(ready, stream) != hipSuccess)
                return set_error(DYNA_ERR_HIP, "draft_head: recording the x-ready event failed");
        }
        if (hipStreamWaitEvent(rs, ready, 0) != hipSuccess)
            return set_error(DYNA_ERR_HIP, "draft_head: route stream wait failed");
    }
    const bool want_ids = (mode & (DYNA_SEL_ARGMAX | DYNA_SEL_TOPK)) != 0;
    const bool want_sample = (mode & DYNA_SEL_SAMPLE) != 0;
    int32_t* clusters = out_clusters ? out_clusters : c.topk_ids;
    float* logits = out_logits ? out_logits : c.logits;
    // one context, argmax or top-k_t: the whole step in one launch, or the
    // gathered head carrying the selection (4 launches)
    const int fused_opt = g_fused_off.load();
    const bool fused = B == 1 && fused_opt != 1 && option_logits_path() <= 1 && k_t >= 1 &&
                       k_t <= kFusedTopkMax && !want_sample;
    if (fused && (fused_opt == 0 || fused_opt == 3) && !split && option_router_path() <= 1) {
        ChainRequest q{};
        q.all_bf16 = r->wdtype == DYNA_BF16 && L->wdtype == DYNA_BF16 && adtype == DYNA_BF16;
        q.W1 = r->W1;
        q.b1 = r->b1;
        q.W2 = r->W2;
        q.b2 = r->b2;
        q.d_r = r->d_r;
        q.H = r->H;
        q.M = r->M;
        q.act = r->act;
        q.x = x;
        q.W = L->W_perm;
        q.perm = L->perm;
        q.offsets = L->offsets;
        q.d = L->d;
        q.V = L->V;
        q.h = h;
        q.k = k;
        q.region = chain_region ? chain_region : c.chain;
        q.out_clusters = clusters;
        q.topk_scores = c.topk_scores;
        q.sel_sorted = c.sel_sorted;
        q.sel_rowoff = c.sel_rowoff;
        q.row_len = c.row_len;
        q.out_logits = out_logits;
        q.out_ids = want_ids ? out_ids : nullptr;
        q.out_logprobs = want_ids ? out_logprobs : nullptr;
        q.k_t = k_t;
        q.inv_t = 1.0f / temperature;
        q.beta = tail_beta;
        // the one launch needs its whole grid resident at once; a shape the
        // occupancy check rejects takes the four-launch form below
        int64_t khz = 0;
        if (q.out_ids != nullptr && chain_step_grid(q, &khz) > 0)
            return timed([&] { return launch_chain_step(q, stream); }, stream);
    }
    if (fused_opt == 3)
        return set_error(DYNA_ERR_UNSUPPORTED, "one-launch step requested (DYNA_OPT_FUSED_B1 = 3) but not possible");

    // routing (the router's stream); with several contexts a split-K last
    // layer leaves its partial sums to the top-k
    ScoreSlices slices;
    TRY(run_router(r, x, adtype, B, c.scores, c.hidden, c.rpart, c.rpart_floats, rs, fused ? c.counters : nullptr,
                   B > 1 ? &slices : nullptr));
    // union rows: one dense product of the union's slabs with every context
    // (it needs only one list entry per union cluster, and writes one shared
    // copy of the slots' vocabulary ids)
    // A few rows over a short union take the per-chunk gathered kernel (one
    // unit of every row per chunk, private rings per wave): measured at ten
    // rows, 7 us faster per step than the dense union kernel at unions of
    // 3.7-9.2k slots (row strides up to 39k) and 4 us slower at 32k.  A
    // fixed union shape (DYNA_OPT_UNION_CFG) always takes the dense kernel.
    constexpr int32_t kSmallUnionCap = 65536;
    const bool small_union = option_union_cfg() == 0 && B <= 16 && cap <= kSmallUnionCap;
    const bool dense_union = union_mode && option_logits_path() == 0 && L->wdtype == DYNA_BF16 &&
                             adtype == DYNA_BF16 && L->d % 8 == 0 && !small_union;
    if (union_mode) {
        // per-row clusters, then one shared shortlist (its ids go to sel_sorted)
        TRY(launch_topk_clusters(c.scores, B, L->M, k, clusters, c.topk_scores, nullptr, nullptr, nullptr, nullptr,
                                 nullptr, rs, slices));
        TRY(launch_union_plan(L->offsets, L->M, clusters, B, k, c.row_len, c.sel_sorted,
                              (int32_t)std::min<int64_t>(L->M, (int64_t)B * k), c.plan, dense_union, rs));
    } else {
        TRY(launch_topk_clusters(c.scores, B, L->M, k, clusters, c.topk_scores, L->offsets, c.sel_sorted,
                                 c.sel_rowoff, c.row_len, &c.plan, rs, slices));
        if (B > 1) TRY(launch_plan(L->offsets, L->M, c.sel_sorted, c.sel_rowoff, B, k, c.plan, rs));
    }
    if (split) {
        hipEvent_t join = lazy_event(g_ev_join);
        if (!join || hipEventRecord(join, rs) != hipSuccess || hipStreamWaitEvent(stream, join, 0) != hipSuccess)
            return set_error(DYNA_ERR_HIP, "draft_head: stream join failed");
    }
    // gathered head and selection (the caller's stream)
    RowdotArgs a{};
    a.W = L->W_perm;
    a.wdtype = L->wdtype;
    a.K = L->d;
    a.v = h;
    a.vdtype = adtype;
    a.B = B;
    a.out = logits;
    a.ld = cap;
    a.act = DYNA_ACT_NONE;
    a.plan = c.plan;
    a.max_chunks_bound = chunk_bound(L, B, k);
    a.perm = L->perm;
    a.vid_out = c.slot_vid;
    const SelectArgs sa = make_select_args(
        logits, cap, c.row_len, 0, cap, c.sel_sorted, c.sel_rowoff, L->offsets, L->perm, B, k, k_t,
        temperature, tail_beta, L->V, want_sample ? uniforms : nullptr, want_ids ? out_ids : nullptr,
        want_ids ? out_logprobs : nullptr, want_sample ? out_sample : nullptr,
        want_sample ? out_sample_logprob : nullptr, c.select_ws, c.slot_vid);
    if (fused) return timed([&] { return launch_logits_greedy(a, sa, c.partials, c.counters, stream); }, stream);
    if (dense_union && !gather_lds_eligible(a)) return set_error(DYNA_ERR_UNSUPPORTED, "union: kernel arguments");
    if (dense_union) TRY(timed([&] { return launch_union_gemm(a, stream); }, stream));
    else TRY(timed_rowdot(a, union_mode ? option_logits_path() : gathered_path(B), stream));
    // union rows over a few thousand slots select faster in one launch (one
    // workgroup per row); long union rows split into segments.  Measured at
    // ten rows: 6-7 us saved per step at unions of 3.7-5.9k slots (row
    // strides up to 26k), 3 us lost at 9.2k (stride 39k), 28 us at 32k; 77 us
    // lost at 64 rows of 32k.
    constexpr int32_t kUnionSplitCap = 32768;
    return launch_select(logits, cap, c.row_len, 0, cap, c.sel_sorted, c.sel_rowoff, L->offsets, L->perm, B,
                         k, k_t, temperature, tail_beta, L->V, want_sample ? uniforms : nullptr,
                         want_ids ? out_ids : nullptr,
                         want_ids ? out_logprobs : nullptr, want_sample ? out_sample : nullptr,
                         want_sample ? out_sample_logprob : nullptr, c.select_ws, stream, c.slot_vid,
                         dense_union ? 0 : cap, union_mode && cap > kUnionSplitCap);
}

}  // namespace dyna

DYNA_API dyna_status dyna_draft_head(const dyna_router* r, const dyna_layout* L, const void* x, const void* h,
                                     int32_t adtype, int32_t B, int32_t k, int32_t mode, int32_t k_t,
                                     float temperature, float tail_beta, const float* uniforms, int32_t* out_ids,
                                     float* out_logprobs, int32_t* out_sample, float* out_sample_logprob,
                                     int32_t* out_clusters, float* out_logits, int32_t cap, void* ws,
                                     size_t ws_bytes, hipStream_t stream, hipStream_t route_stream,
                                     hipEvent_t x_ready) {
    return draft_head_core(r, L, x, h, adtype, B, k, mode, k_t, temperature, tail_beta, uniforms, out_ids,
                           out_logprobs, out_sample, out_sample_logprob, out_clusters, out_logits, cap, ws,
                           ws_bytes, stream, route_stream, x_ready, nullptr, true);
}

// ------------------------------------------------------------------ beam expansion
DYNA_API dyna_status dyna_beam_expand(const float* logprobs, const int32_t* ids, const float* last_scores,
                                      int32_t B, int32_t k_t, int32_t n_out, float* out_scores,
                                      int32_t* out_parent, int32_t* out_ids, hipStream_t stream) {
    REQUIRE(B >= 1 && k_t >= 1 && k_t <= DYNA_MAX_KT, "B=%d, k_t=%d", B, k_t);
    REQUIRE(n_out >= 1 && n_out <= DYNA_MAX_KT, "n_out=%d outside [1, %d]", n_out, DYNA_MAX_KT);
    REQUIRE(logprobs && ids && out_scores && out_parent && out_ids, "NULL argument");
    return launch_beam_expand(logprobs, ids, last_scores, B, k_t, n_out, out_scores, out_parent, out_ids, stream);
}

// ------------------------------------------------------------------ budgets
DYNA_API int32_t dyna_cluster_budget(int32_t t, int32_t k0, int32_t k1, int32_t k_min, int32_t form) {
    if (t < 0 || k0 < 1 || k1 < 1 || k_min < 1 || (form != 0 && form != 1)) return -1;
    if (t == 0) return k0;
    if (t == 1) return k1;
    const int64_t num = form == 0 ? (int64_t)k1 + t : (int64_t)k1;
    return (int32_t)std::max<int64_t>(k_min, num / (2 * (int64_t)t));
}

DYNA_API int32_t dyna_static_budget(int32_t t, int32_t k_max) {
    if (t < 0 || k_max < 1) return -1;
    return t < 2 ? k_max : (int32_t)((int64_t)k_max / ((int64_t)t + 1));
}

// ------------------------------------------------------------------ partition builder
static dyna_status check_kmeans(int32_t wdtype, int32_t V, int32_t d, int32_t M) {
    if (wdtype != DYNA_BF16) return set_error(DYNA_ERR_UNSUPPORTED, "k-means: bf16 rows only");
    REQUIRE(V >= 1 && d >= 8 && d % 8 == 0, "bad sizes V=%d d=%d", V, d);
    if (d > 8192) return set_error(DYNA_ERR_UNSUPPORTED, "k-means: d=%d > 8192", d);
    REQUIRE(M >= 1 && M <= DYNA_MAX_M && M <= V, "M=%d outside [1, min(V, %d)]", M, DYNA_MAX_M);
    return DYNA_OK;
}

DYNA_API size_t dyna_kmeans_workspace_bytes(int32_t V, int32_t d, int32_t M) {
    if (V < 1 || d < 8 || M < 1) return 0;
    return kmeans_ws_bytes(V, d, M);
}

DYNA_API dyna_status dyna_kmeans_assign(const void* W, int32_t wdtype, int32_t V, int32_t d, const float* centroids,
                                        int32_t M, int32_t* out_assign, float* out_score, void* ws,
                                        size_t ws_bytes, hipStream_t stream) {
    TRY(check_kmeans(wdtype, V, d, M));
    REQUIRE(W && aligned16(W) && centroids && out_assign && ws, "NULL argument or W misaligned");
    if (ws_bytes < kmeans_ws_bytes(V, d, M))
        return set_error(DYNA_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, kmeans_ws_bytes(V, d, M));
    return timed([&] { return kmeans_assign(W, V, d, centroids, M, out_assign, out_score, ws, stream); }, stream);
}

DYNA_API dyna_status dyna_kmeans_update(const void* W, int32_t wdtype, int32_t V, int32_t d, const int32_t* assign,
                                        int32_t M, float* centroids, void* ws, size_t ws_bytes, hipStream_t stream) {
    TRY(check_kmeans(wdtype, V, d, M));
    REQUIRE(W && aligned16(W) && assign && centroids && ws, "NULL argument or W misaligned");
    if (ws_bytes < kmeans_ws_bytes(V, d, M))
        return set_error(DYNA_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, kmeans_ws_bytes(V, d, M));
    return kmeans_update(W, V, d, assign, M, centroids, ws, stream);
}

DYNA_API dyna_status dyna_kmeans(const void* W, int32_t wdtype, int32_t V, int32_t d, int32_t M,
                                 const int32_t* init_ids, int32_t iters, int32_t* out_cluster_of,
                                 float* out_centroids, void* ws, size_t ws_bytes, hipStream_t stream) {
    TRY(check_kmeans(wdtype, V, d, M));
    REQUIRE(iters >= 1, "iters=%d < 1", iters);
    REQUIRE(W && aligned16(W) && init_ids && out_cluster_of && ws, "NULL argument or W misaligned");
    if (ws_bytes < kmeans_ws_bytes(V, d, M))
        return set_error(DYNA_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, kmeans_ws_bytes(V, d, M));
    return kmeans_run(W, V, d, M, init_ids, iters, out_cluster_of, out_centroids, ws, stream);
}

// ------------------------------------------------------------------ baselines
static size_t dense_bytes(int32_t n_rows, int32_t B, float** logits, void** sel, void* base, Plan* plan = nullptr) {
    char* p = static_cast<char*>(base);
    size_t off = 0;
    const size_t lb = align256(sizeof(float) * (size_t)B * (size_t)n_rows);
    if (logits) *logits = p ? reinterpret_cast<float*>(p) : nullptr;
    off += lb;
    if (sel) *sel = p ? p + off : nullptr;
    off += align256(select_ws_bytes(B, n_rows, DYNA_MAX_KT));
    // the full-row plan of the matrix-core path (one chunk per 16 rows)
    const int64_t n_chunks = ((int64_t)n_rows + kChunkRows - 1) / kChunkRows;
    if (plan && p) {
        plan->hdr = reinterpret_cast<PlanHeader*>(p + off);
        plan->list = reinterpret_cast<ListEntry*>(p + off + sizeof(PlanHeader));
        plan->chunks = reinterpret_cast<Chunk*>(p + off + sizeof(PlanHeader) + align256(sizeof(ListEntry)));
        plan->max_chunks = (int32_t)n_chunks;
        plan->max_entries = 1;
    }
    off += sizeof(PlanHeader) + align256(sizeof(ListEntry)) + align256(sizeof(Chunk) * (size_t)n_chunks);
    return off;
}

DYNA_API size_t dyna_dense_workspace_bytes(int32_t n_rows, int32_t B) {
    if (n_rows < 1 || B < 0) return 0;
    return dense_bytes(n_rows, B, nullptr, nullptr, nullptr);
}

DYNA_API dyna_status dyna_dense_head(const void* W, int32_t wdtype, int32_t n_rows, int32_t d, const void* h,
                                     int32_t hdtype, int32_t B, int32_t mode, int32_t k_t, float temperature,
                                     const float* uniforms, int32_t* out_ids, float* out_logprobs,
                                     int32_t* out_sample, float* out_sample_logprob, float* out_logits,
                                     void* ws, size_t ws_bytes, hipStream_t stream) {
    REQUIRE(valid_dtype(wdtype) && valid_dtype(hdtype), "bad dtype");
    REQUIRE(n_rows >= 1 && d >= 8 && d % 8 == 0, "bad sizes n_rows=%d d=%d", n_rows, d);
    if (d > 8192) return set_error(DYNA_ERR_UNSUPPORTED, "d=%d > 8192", d);
    if (n_rows > select_max_len())
        return set_error(DYNA_ERR_UNSUPPORTED, "n_rows=%d > %d", n_rows, select_max_len());
    TRY(check_select(mode, &k_t, temperature, uniforms, out_ids, out_sample));
    REQUIRE(B >= 0, "B=%d < 0", B);
    if (B == 0) return DYNA_OK;
    REQUIRE(W && h && aligned16(W) && aligned16(h) && ws, "NULL argument or W/h misaligned");
    const size_t need = dense_bytes(n_rows, B, nullptr, nullptr, nullptr);
    if (ws_bytes < need) return set_error(DYNA_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, need);
    float* wl = nullptr;
    void* sel = nullptr;
    Plan plan{};
    dense_bytes(n_rows, B, &wl, &sel, ws, &plan);
    float* logits = out_logits ? out_logits : wl;
    RowdotArgs a{};
    a.W = W;
    a.wdtype = wdtype;
    a.K = d;
    a.v = h;
    a.vdtype = hdtype;
    a.B = B;
    a.out = logits;
    a.ld = n_rows;
    a.act = DYNA_ACT_NONE;
    a.n_rows = n_rows;
    if (option_logits_path() == 0 && B > 4 && wdtype == DYNA_BF16 && hdtype == DYNA_BF16) {
        // several contexts: the rows streamed once through LDS by the union
        // kernel, every context multiplied on the matrix cores
        a.plan = plan;
        a.max_chunks_bound = plan.max_chunks;
        TRY(launch_full_plan(n_rows, B, plan, stream));
        TRY(timed([&] { return launch_union_gemm(a, stream); }, stream));
    } else {
        TRY(timed_rowdot(a, option_logits_path(), stream));
    }
    const bool want_ids = (mode & (DYNA_SEL_ARGMAX | DYNA_SEL_TOPK)) != 0;
    const bool want_sample = (mode & DYNA_SEL_SAMPLE) != 0;
    return launch_select(logits, n_rows, nullptr, n_rows, n_rows, nullptr, nullptr, nullptr, nullptr, B, 0, k_t,
                         temperature, 0.0f, n_rows, want_sample ? uniforms : nullptr, want_ids ? out_ids : nullptr,
                         want_ids ? out_logprobs : nullptr, want_sample ? out_sample : nullptr,
                         want_sample ? out_sample_logprob : nullptr, sel, stream);
}
