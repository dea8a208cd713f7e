// One-time cluster-contiguous layout of the LM head.
//
// The paper partitions the vocabulary into M disjoint clusters of free sizes
// (Sec. 4.2, "Vocabulary partition").  Storing every cluster as one run of
// consecutive rows turns the shortlist gather of the head into whole-slab
// streams.  The layout is a stable counting sort of the tokens by cluster id
// (ties keep ascending vocabulary id), followed by a row-permuting copy.
#include "dyna_device.h"

namespace dyna {
namespace {

constexpr int kChunk = 4096;    // tokens per counting workgroup
constexpr int kThreads = 256;

__global__ void fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// Per chunk of kChunk tokens: the rank of every token among the earlier
// tokens of its cluster inside the chunk, and per-cluster counts.
__global__ __launch_bounds__(kThreads) void layout_count_kernel(
    const int32_t* __restrict__ cluster_of, int32_t V, int32_t M, int32_t* __restrict__ rank,
    int32_t* __restrict__ cnt, int32_t* __restrict__ bad) {
    extern __shared__ int32_t lds[];
    int32_t* counter = lds;        // [M]
    int32_t* ids = lds + M;        // [kThreads]
    const int64_t base = (int64_t)blockIdx.x * kChunk;
    for (int m = threadIdx.x; m < M; m += kThreads) counter[m] = 0;
    __syncthreads();
    for (int sub = 0; sub < kChunk; sub += kThreads) {
        const int64_t v = base + sub + threadIdx.x;
        int c = -1;
        if (v < V) {
            c = cluster_of[v];
            if (c < 0 || c >= M) {
                atomicOr(bad, 1);
                c = -1;
            }
        }
        ids[threadIdx.x] = c;
        __syncthreads();
        if (c >= 0) {
            int before = 0;
            for (int t = 0; t < (int)threadIdx.x; ++t) before += (ids[t] == c);
            rank[v] = counter[c] + before;
        }
        __syncthreads();
        if (c >= 0) atomicAdd(&counter[c], 1);
        __syncthreads();
    }
    for (int m = threadIdx.x; m < M; m += kThreads) cnt[(int64_t)blockIdx.x * M + m] = counter[m];
}

// Single workgroup: cluster totals, their exclusive scan (the CSR offsets),
// and per (chunk, cluster) the first layout row of that chunk's tokens.
constexpr int kScanThreads = 1024;
__global__ __launch_bounds__(kScanThreads) void layout_scan_kernel(int32_t M, int32_t nchunks,
                                                                   int32_t* __restrict__ cnt,
                                                                   int32_t* __restrict__ offsets) {
    __shared__ int tmp[kScanThreads / kWave + 1];
    const int per = (M + kScanThreads - 1) / kScanThreads;
    const int m0 = threadIdx.x * per;
    const int m1 = min(M, m0 + per);
    int local = 0;
    for (int m = m0; m < m1; ++m)
        for (int c = 0; c < nchunks; ++c) local += cnt[(int64_t)c * M + m];
    int total;
    int run = block_exclusive_scan<kScanThreads>(local, tmp, &total);
    for (int m = m0; m < m1; ++m) {
        offsets[m] = run;
        for (int c = 0; c < nchunks; ++c) {
            const int t = cnt[(int64_t)c * M + m];
            cnt[(int64_t)c * M + m] = run;
            run += t;
        }
    }
    if (threadIdx.x == 0) offsets[M] = total;
}

__global__ void layout_scatter_kernel(const int32_t* __restrict__ cluster_of, int32_t V, int32_t M,
                                      const int32_t* __restrict__ rank,
                                      const int32_t* __restrict__ base,
                                      int32_t* __restrict__ perm) {
    for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < V;
         v += (int64_t)gridDim.x * blockDim.x) {
        const int c = cluster_of[v];
        if (c < 0 || c >= M) continue;
        const int64_t chunk = v / kChunk;
        perm[base[chunk * M + c] + rank[v]] = (int32_t)v;
    }
}

// W_perm[j] = W[perm[j]]: one wave per row, 16-byte vectors.
__global__ __launch_bounds__(256) void layout_copy_rows_kernel(const u32x4* __restrict__ W,
                                                               u32x4* __restrict__ Wp,
                                                               const int32_t* __restrict__ perm,
                                                               int32_t V, int32_t vec_per_row) {
    const int lane = lane_id();
    const int64_t nw = (int64_t)gridDim.x * (blockDim.x / kWave);
    for (int64_t j = blockIdx.x * (int64_t)(blockDim.x / kWave) + threadIdx.x / kWave; j < V;
         j += nw) {
        const int64_t src = perm[j];
        const u32x4* s = W + src * vec_per_row;
        u32x4* d = Wp + j * vec_per_row;
        for (int i = lane; i < vec_per_row; i += kWave) d[i] = __builtin_nontemporal_load(s + i);
    }
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace

size_t layout_ws_bytes(int32_t V, int32_t M) {
    const int64_t nchunks = (V + kChunk - 1) / kChunk;
    return align256(sizeof(int32_t) * (size_t)V) + align256(sizeof(int32_t) * (size_t)nchunks * M) +
           256;
}

dyna_status launch_cluster_csr(const int32_t* cluster_of, int32_t V, int32_t M, int32_t* perm,
                               int32_t* offsets, void* ws, hipStream_t stream) {
    const int32_t nchunks = (V + kChunk - 1) / kChunk;
    char* p = static_cast<char*>(ws);
    int32_t* rank = reinterpret_cast<int32_t*>(p);
    p += align256(sizeof(int32_t) * (size_t)V);
    int32_t* cnt = reinterpret_cast<int32_t*>(p);
    p += align256(sizeof(int32_t) * (size_t)nchunks * M);
    int32_t* bad = reinterpret_cast<int32_t*>(p);
    fill_i32_kernel<<<1, 64, 0, stream>>>(bad, 1, 0);
    const size_t lds = sizeof(int32_t) * ((size_t)M + kThreads);
    layout_count_kernel<<<nchunks, kThreads, lds, stream>>>(cluster_of, V, M, rank, cnt, bad);
    if (dyna_status s = check_launch("layout_count_kernel"); s != DYNA_OK) return s;
    layout_scan_kernel<<<1, kScanThreads, 0, stream>>>(M, nchunks, cnt, offsets);
    if (dyna_status s = check_launch("layout_scan_kernel"); s != DYNA_OK) return s;
    layout_scatter_kernel<<<(V + 255) / 256, 256, 0, stream>>>(cluster_of, V, M, rank, cnt, perm);
    return check_launch("layout_scatter_kernel");
}

dyna_status launch_build_layout(const int32_t* cluster_of, int32_t V, int32_t M, const void* W_lm,
                                int32_t wdtype, int32_t d, void* W_perm, int32_t* perm,
                                int32_t* offsets, void* ws, size_t ws_bytes,
                                int32_t* host_offsets_out, hipStream_t stream) {
    const int32_t nchunks = (V + kChunk - 1) / kChunk;
    char* p = static_cast<char*>(ws);
    int32_t* rank = reinterpret_cast<int32_t*>(p);
    p += align256(sizeof(int32_t) * (size_t)V);
    int32_t* cnt = reinterpret_cast<int32_t*>(p);
    p += align256(sizeof(int32_t) * (size_t)nchunks * M);
    int32_t* bad = reinterpret_cast<int32_t*>(p);
    (void)ws_bytes;

    fill_i32_kernel<<<1, 64, 0, stream>>>(bad, 1, 0);
    fill_i32_kernel<<<1024, 256, 0, stream>>>(perm, V, -1);
    if (dyna_status s = check_launch("layout fill"); s != DYNA_OK) return s;
    const size_t lds = sizeof(int32_t) * ((size_t)M + kThreads);
    layout_count_kernel<<<nchunks, kThreads, lds, stream>>>(cluster_of, V, M, rank, cnt, bad);
    if (dyna_status s = check_launch("layout_count_kernel"); s != DYNA_OK) return s;
    layout_scan_kernel<<<1, kScanThreads, 0, stream>>>(M, nchunks, cnt, offsets);
    if (dyna_status s = check_launch("layout_scan_kernel"); s != DYNA_OK) return s;
    layout_scatter_kernel<<<(V + 255) / 256, 256, 0, stream>>>(cluster_of, V, M, rank, cnt, perm);
    if (dyna_status s = check_launch("layout_scatter_kernel"); s != DYNA_OK) return s;

    // A bad id leaves holes in perm; check before the copy dereferences it.
    int32_t bad_host = 0;
    if (hipMemcpyAsync(&bad_host, bad, sizeof(int32_t), hipMemcpyDeviceToHost, stream) != hipSuccess ||
        hipMemcpyAsync(host_offsets_out, offsets, sizeof(int32_t) * (size_t)(M + 1),
                       hipMemcpyDeviceToHost, stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess)
        return set_error(DYNA_ERR_HIP, "build_layout: device copy/synchronise failed");
    if (bad_host) return set_error(DYNA_ERR_DEVICE_DATA, "build_layout: cluster id outside [0, M)");
    if (host_offsets_out[M] != V)
        return set_error(DYNA_ERR_DEVICE_DATA, "build_layout: partition does not cover V");

    const int elt = wdtype == DYNA_BF16 ? 2 : 4;
    const int32_t vec_per_row = (int32_t)((int64_t)d * elt / 16);
    const int64_t blocks = std::min<int64_t>((V + 3) / 4, 8192);
    layout_copy_rows_kernel<<<(unsigned)blocks, 256, 0, stream>>>(
        static_cast<const u32x4*>(W_lm), static_cast<u32x4*>(W_perm), perm, V, vec_per_row);
    if (dyna_status s = check_launch("layout_copy_rows_kernel"); s != DYNA_OK) return s;
    if (hipStreamSynchronize(stream) != hipSuccess)
        return set_error(DYNA_ERR_HIP, "build_layout: synchronise failed");
    return DYNA_OK;
}

}  // namespace dyna
