// Building the partition: spherical k-means over the LM-head rows (Sec. 4.2,
// "Vocabulary partition": the clusters come from spherical k-means on the
// column-normalised head, one point per vocabulary entry).
//
// One round is an assignment and an update.
//  * Assignment: every row goes to the centroid of largest cosine
//    similarity.  Dividing a row by its norm does not change which centroid
//    wins, so the raw bf16 rows are scored against the bf16 unit centroids:
//    a dense V x M x d product on the matrix cores with an argmax epilogue
//    (the union-row kernel, every row against every centroid), so no V x M
//    score matrix is ever written.  Ties go to the lower centroid id.
//  * Update: a stable counting sort of the assignment (the layout's CSR
//    kernels) lists each cluster's rows in ascending id; one workgroup per
//    cluster sums its unit rows in that order in fp32 and divides by the
//    norm of the sum.  An empty cluster (or a zero sum) keeps its centroid.
// Every sum runs in a fixed order, so a run is bit-identical to the next.
#include "dyna_device.h"

namespace dyna {
namespace {

constexpr int kKmThreads = 256;
constexpr int kKmCols = 8 * kKmThreads;  // columns one pass of an update workgroup covers
constexpr int kKmUnroll = 4;             // member rows whose loads are issued together

// bf16 bits of x, rounded to nearest with ties to even (NaN stays a quiet NaN).
__device__ __forceinline__ uint16_t to_bf16_rne(float x) {
    uint32_t u = __float_as_uint(x);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// inv[v] = 1 / ||W[v]|| (0 for an all-zero row): one wave per row, 16-byte loads.
__global__ __launch_bounds__(kKmThreads) void row_inv_norm_kernel(const uint16_t* __restrict__ W, int32_t V,
                                                                  int32_t d, float* __restrict__ inv) {
    const int lane = lane_id();
    const int64_t v = (int64_t)blockIdx.x * (kKmThreads / kWave) + threadIdx.x / kWave;
    if (v >= V) return;  // whole wave
    const u32x4* row = reinterpret_cast<const u32x4*>(W + v * d);
    float s = 0.0f;
    for (int i = lane; i < d / 8; i += kWave) {
        const u32x4 q = __builtin_nontemporal_load(row + i);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float lo = bf16_lo(q[e]), hi = bf16_hi(q[e]);
            s = fmaf(lo, lo, s);
            s = fmaf(hi, hi, s);
        }
    }
    s = wave_sum(s);
    if (lane == 0) inv[v] = s > 0.0f ? 1.0f / sqrtf(s) : 0.0f;
}

// Centroid m starts at the unit row init_ids[m]; an id outside [0, V) gives a
// zero centroid and sets *bad.
__global__ __launch_bounds__(kKmThreads) void centroid_init_kernel(const uint16_t* __restrict__ W,
                                                                   const float* __restrict__ inv,
                                                                   const int32_t* __restrict__ init_ids,
                                                                   int32_t V, int32_t d, float* __restrict__ mu32,
                                                                   uint16_t* __restrict__ mu16,
                                                                   int32_t* __restrict__ bad) {
    const int64_t m = blockIdx.x;
    const int32_t v = init_ids[m];
    const bool ok = v >= 0 && v < V;
    if (!ok && threadIdx.x == 0) atomicOr(bad, 1);
    const float sc = ok ? inv[v] : 0.0f;
    for (int c = threadIdx.x; c < d; c += kKmThreads) {
        const float x = ok ? __uint_as_float((uint32_t)W[(int64_t)v * d + c] << 16) * sc : 0.0f;
        mu32[m * d + c] = x;
        mu16[m * d + c] = to_bf16_rne(x);
    }
}

__global__ void clear_word_kernel(int32_t* p) { *p = 0; }

__global__ void f32_to_bf16_kernel(const float* __restrict__ src, uint16_t* __restrict__ dst, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        dst[i] = to_bf16_rne(src[i]);
}

// Plan over every row: chunk c is rows [16c, 16c + 16), and its one list
// entry (slot base 0) stands for all B centroids.
__global__ void full_plan_kernel(int32_t V, int32_t B, Plan plan) {
    const int64_t n = ((int64_t)V + kChunkRows - 1) / kChunkRows;
    for (int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; c < n; c += (int64_t)gridDim.x * blockDim.x)
        plan.chunks[c] = Chunk{(int32_t)(c * kChunkRows), (int32_t)min<int64_t>(kChunkRows, V - c * kChunkRows), 0, B};
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        plan.list[0] = ListEntry{0, 0};
        plan.hdr->n_chunks = (int32_t)n;
        plan.hdr->n_entries = 1;
    }
}

// mu[m] = (sum of the unit rows of cluster m, in ascending row id) / its norm;
// an empty cluster or a zero sum keeps mu[m].  One workgroup per cluster;
// thread t owns columns 8t + 2048 j, j < J.
template <int J>
__global__ __launch_bounds__(kKmThreads) void centroid_update_kernel(const uint16_t* __restrict__ W,
                                                                     const float* __restrict__ inv,
                                                                     const int32_t* __restrict__ perm,
                                                                     const int32_t* __restrict__ offsets, int32_t d,
                                                                     float* __restrict__ mu32,
                                                                     uint16_t* __restrict__ mu16) {
    __shared__ float red[kKmThreads / kWave];
    const int64_t m = blockIdx.x;
    const int32_t i0 = offsets[m], i1 = offsets[m + 1];
    if (i0 >= i1) return;  // empty: unchanged (whole workgroup)
    float s[J][8];
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e) s[j][e] = 0.0f;
    for (int32_t i = i0; i < i1; i += kKmUnroll) {
        int64_t v[kKmUnroll];
        float sc[kKmUnroll];
#pragma unroll
        for (int q = 0; q < kKmUnroll; ++q) {
            const bool in = i + q < i1;
            v[q] = perm[in ? i + q : i0];
            sc[q] = in ? inv[v[q]] : 0.0f;  // a row past the cluster adds zeros
        }
        u32x4 x[kKmUnroll][J];
#pragma unroll
        for (int q = 0; q < kKmUnroll; ++q)
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const int c0 = 8 * (int)threadIdx.x + kKmCols * j;
                x[q][j] = c0 < d ? *reinterpret_cast<const u32x4*>(W + v[q] * d + c0) : u32x4{0u, 0u, 0u, 0u};
            }
#pragma unroll
        for (int q = 0; q < kKmUnroll; ++q)
#pragma unroll
            for (int j = 0; j < J; ++j)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    s[j][2 * e] = fmaf(bf16_lo(x[q][j][e]), sc[q], s[j][2 * e]);
                    s[j][2 * e + 1] = fmaf(bf16_hi(x[q][j][e]), sc[q], s[j][2 * e + 1]);
                }
    }
    float ss = 0.0f;
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e) ss = fmaf(s[j][e], s[j][e], ss);
    ss = wave_sum(ss);
    if (lane_id() == 0) red[threadIdx.x / kWave] = ss;
    __syncthreads();
    float tot = 0.0f;
#pragma unroll
    for (int w = 0; w < kKmThreads / kWave; ++w) tot += red[w];
    if (!(tot > 0.0f)) return;  // zero sum: unchanged
    const float rn = 1.0f / sqrtf(tot);
#pragma unroll
    for (int j = 0; j < J; ++j) {
        const int c0 = 8 * (int)threadIdx.x + kKmCols * j;
        if (c0 < d) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float y = s[j][e] * rn;
                mu32[m * d + c0 + e] = y;
                mu16[m * d + c0 + e] = to_bf16_rne(y);
            }
        }
    }
}

size_t al256(size_t x) { return (x + 255) & ~size_t(255); }

// Workspace views.
struct KmWs {
    float* inv;        // [V]
    uint16_t* mu16;    // [M, d]
    float* mu32;       // [M, d] (used when the caller keeps no centroids)
    int32_t* assign;   // [V] (used when the caller keeps no assignment)
    int32_t* perm;     // [V]
    int32_t* offsets;  // [M + 1]
    int32_t* bad;      // [1]
    Plan plan;
    void* csr;         // layout_ws_bytes(V, M)
    size_t bytes;
};

KmWs km_carve(int32_t V, int32_t d, int32_t M, void* base) {
    KmWs w{};
    char* p = static_cast<char*>(base);
    size_t off = 0;
    auto take = [&](size_t n) -> void* {
        void* q = p ? p + off : nullptr;
        off += al256(n);
        return q;
    };
    const int64_t n_chunks = ((int64_t)V + kChunkRows - 1) / kChunkRows;
    w.inv = static_cast<float*>(take(sizeof(float) * (size_t)V));
    w.mu16 = static_cast<uint16_t*>(take(sizeof(uint16_t) * (size_t)M * d));
    w.mu32 = static_cast<float*>(take(sizeof(float) * (size_t)M * d));
    w.assign = static_cast<int32_t*>(take(sizeof(int32_t) * (size_t)V));
    w.perm = static_cast<int32_t*>(take(sizeof(int32_t) * (size_t)V));
    w.offsets = static_cast<int32_t*>(take(sizeof(int32_t) * ((size_t)M + 1)));
    w.bad = static_cast<int32_t*>(take(sizeof(int32_t)));
    w.plan.hdr = static_cast<PlanHeader*>(take(sizeof(PlanHeader)));
    w.plan.chunks = static_cast<Chunk*>(take(sizeof(Chunk) * (size_t)n_chunks));
    w.plan.list = static_cast<ListEntry*>(take(sizeof(ListEntry)));
    w.plan.max_chunks = (int32_t)n_chunks;
    w.plan.max_entries = 1;
    w.csr = take(layout_ws_bytes(V, M));
    w.bytes = off;
    return w;
}

dyna_status launch_inv_norms(const uint16_t* W, int32_t V, int32_t d, float* inv, hipStream_t stream) {
    const int64_t blocks = ((int64_t)V + kKmThreads / kWave - 1) / (kKmThreads / kWave);
    row_inv_norm_kernel<<<(unsigned)blocks, kKmThreads, 0, stream>>>(W, V, d, inv);
    return check_launch("row_inv_norm_kernel");
}

dyna_status launch_assign(const uint16_t* W, int32_t V, int32_t d, const uint16_t* mu16, int32_t M, int32_t* assign,
                          float* score, const Plan& plan, hipStream_t stream) {
    RowdotArgs a{};
    a.W = W;
    a.wdtype = DYNA_BF16;
    a.K = d;
    a.v = mu16;
    a.vdtype = DYNA_BF16;
    a.B = M;
    a.out = score;
    a.ld = 0;
    a.act = DYNA_ACT_NONE;
    a.plan = plan;
    a.max_chunks_bound = plan.max_chunks;
    a.vid_out = assign;
    return launch_union_argmax(a, option_kmeans_cfg(), stream);
}

dyna_status launch_update(const uint16_t* W, int32_t V, int32_t d, const int32_t* assign, int32_t M,
                          const KmWs& w, float* mu32, hipStream_t stream) {
    if (dyna_status s = launch_cluster_csr(assign, V, M, w.perm, w.offsets, w.csr, stream); s != DYNA_OK) return s;
    const int J = (d + kKmCols - 1) / kKmCols;
#define DYNA_KM_UPD(NJ)                                                                                       \
    if (J <= NJ) {                                                                                            \
        centroid_update_kernel<NJ><<<M, kKmThreads, 0, stream>>>(W, w.inv, w.perm, w.offsets, d, mu32, w.mu16); \
        return check_launch("centroid_update_kernel");                                                        \
    }
    DYNA_KM_UPD(1)
    DYNA_KM_UPD(2)
    DYNA_KM_UPD(4)
#undef DYNA_KM_UPD
    return set_error(DYNA_ERR_UNSUPPORTED, "k-means: d=%d > 8192", d);
}

}  // namespace

dyna_status launch_full_plan(int32_t V, int32_t M, const Plan& plan, hipStream_t stream) {
    const int64_t n = ((int64_t)V + kChunkRows - 1) / kChunkRows;
    const unsigned blocks = (unsigned)std::min<int64_t>(1024, (n + 255) / 256);
    full_plan_kernel<<<std::max(1u, blocks), 256, 0, stream>>>(V, M, plan);
    return check_launch("full_plan_kernel");
}

size_t kmeans_ws_bytes(int32_t V, int32_t d, int32_t M) { return km_carve(V, d, M, nullptr).bytes; }

dyna_status kmeans_assign(const void* W, int32_t V, int32_t d, const float* centroids, int32_t M,
                          int32_t* out_assign, float* out_score, void* ws, hipStream_t stream) {
    const KmWs w = km_carve(V, d, M, ws);
    const int64_t n = (int64_t)M * d;
    f32_to_bf16_kernel<<<(unsigned)std::min<int64_t>(4096, (n + 255) / 256), 256, 0, stream>>>(centroids, w.mu16, n);
    if (dyna_status s = check_launch("f32_to_bf16_kernel"); s != DYNA_OK) return s;
    if (dyna_status s = launch_full_plan(V, M, w.plan, stream); s != DYNA_OK) return s;
    return launch_assign(static_cast<const uint16_t*>(W), V, d, w.mu16, M, out_assign, out_score, w.plan, stream);
}

dyna_status kmeans_update(const void* W, int32_t V, int32_t d, const int32_t* assign, int32_t M, float* centroids,
                          void* ws, hipStream_t stream) {
    const KmWs w = km_carve(V, d, M, ws);
    const uint16_t* Wb = static_cast<const uint16_t*>(W);
    if (dyna_status s = launch_inv_norms(Wb, V, d, w.inv, stream); s != DYNA_OK) return s;
    const int64_t n = (int64_t)M * d;
    // the bf16 copy of kept (empty-cluster) centroids stays consistent
    f32_to_bf16_kernel<<<(unsigned)std::min<int64_t>(4096, (n + 255) / 256), 256, 0, stream>>>(centroids, w.mu16, n);
    if (dyna_status s = check_launch("f32_to_bf16_kernel"); s != DYNA_OK) return s;
    return launch_update(Wb, V, d, assign, M, w, centroids, stream);
}

dyna_status kmeans_run(const void* W, int32_t V, int32_t d, int32_t M, const int32_t* init_ids, int32_t iters,
                       int32_t* out_cluster_of, float* out_centroids, void* ws, hipStream_t stream) {
    const KmWs w = km_carve(V, d, M, ws);
    const uint16_t* Wb = static_cast<const uint16_t*>(W);
    float* mu32 = out_centroids ? out_centroids : w.mu32;
    int32_t* assign = out_cluster_of ? out_cluster_of : w.assign;
    if (dyna_status s = launch_inv_norms(Wb, V, d, w.inv, stream); s != DYNA_OK) return s;
    clear_word_kernel<<<1, 1, 0, stream>>>(w.bad);
    centroid_init_kernel<<<M, kKmThreads, 0, stream>>>(Wb, w.inv, init_ids, V, d, mu32, w.mu16, w.bad);
    if (dyna_status s = check_launch("centroid_init_kernel"); s != DYNA_OK) return s;
    if (dyna_status s = launch_full_plan(V, M, w.plan, stream); s != DYNA_OK) return s;
    for (int32_t it = 0; it < iters; ++it) {
        if (dyna_status s = launch_assign(Wb, V, d, w.mu16, M, assign, nullptr, w.plan, stream); s != DYNA_OK)
            return s;
        if (dyna_status s = launch_update(Wb, V, d, assign, M, w, mu32, stream); s != DYNA_OK) return s;
    }
    int32_t bad = 0;
    if (hipMemcpyAsync(&bad, w.bad, sizeof(int32_t), hipMemcpyDeviceToHost, stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess)
        return set_error(DYNA_ERR_HIP, "k-means: device copy/synchronise failed");
    if (bad) return set_error(DYNA_ERR_DEVICE_DATA, "k-means: an initial id lies outside [0, V)");
    return DYNA_OK;
}

}  // namespace dyna
