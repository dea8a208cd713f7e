// dyna_draft_head_noalloc: the whole head with no caller workspace and no
// allocation, for callers that cannot allocate (code under HIP graph
// capture, tight serving loops).  Its scratch is one static device array per
// GPU, of DYNA_NOALLOC_SCRATCH_BYTES:
//
//   [0, kChainReserve)       the one-launch step's epoch-tagged hand-off
//                            region, at a fixed place so that its epoch runs
//                            on across calls of any shape;
//   [kChainReserve, end)     the workspace every other kernel carves, as
//                            dyna_workspace_bytes would size it.
//
// The array is shared by every call on a GPU and keeps the last call's
// contents; calls that overlap on one GPU race.
#include <atomic>
#include <mutex>

#include "dyna_internal.h"

namespace dyna {
namespace {

constexpr size_t kScratchBytes = DYNA_NOALLOC_SCRATCH_BYTES;
// 256 + 8 (H + M) + 8 * 33 * 1024 bytes for H <= 8192, M <= 1024 (the
// one-launch step's limits) is below 340 KB
constexpr size_t kChainReserve = 384 * 1024;
static_assert(kScratchBytes > kChainReserve, "scratch too small");

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` on each GPU (its host-side name is not one).
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

__global__ void clear_words_kernel(uint32_t* p, int n) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0u;
}

// First call on a device: look the array up, and clear the hand-off region
// with a fill kernel on `stream` (a memset node would not be safe to record
// under graph capture).
dyna_status scratch_of_current_device(hipStream_t stream, void** out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return set_error(DYNA_ERR_HIP, "draft_head_noalloc: no current device");
    std::lock_guard<std::mutex> g(g_mu);
    if (g_ptr[dev] == nullptr) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr)
            return set_error(DYNA_ERR_HIP, "draft_head_noalloc: hipGetSymbolAddress: %s", hipGetErrorString(e));
        hipLaunchKernelGGL(clear_words_kernel, dim3(32), dim3(256), 0, stream, static_cast<uint32_t*>(p),
                           (int)(kChainReserve / 4));
        const hipError_t le = hipGetLastError();
        if (le != hipSuccess)
            return set_error(DYNA_ERR_HIP, "draft_head_noalloc: clearing the scratch: %s", hipGetErrorString(le));
        g_ptr[dev] = p;
    }
    *out = g_ptr[dev];
    return DYNA_OK;
}

}  // namespace
}  // namespace dyna

using namespace dyna;

extern "C" __attribute__((visibility("default"))) dyna_status dyna_draft_head_noalloc(
    const dyna_router* r, const dyna_layout* L, const void* x, const void* h, int32_t adtype, int32_t B, int32_t k,
    int32_t mode, int32_t k_t, float temperature, float tail_beta, const float* uniforms, int32_t* out_ids,
    float* out_logprobs, int32_t* out_sample, float* out_sample_logprob, int32_t* out_clusters, float* out_logits,
    int32_t cap, hipStream_t stream) {
    if (B > 0 && L != nullptr && r != nullptr && k >= 1 && L->cap_by_k != nullptr && k <= L->M && cap >= 0) {
        const size_t need = dyna_workspace_bytes(L, r, B, k, cap);
        if (need > kScratchBytes - kChainReserve)
            return set_error(DYNA_ERR_WORKSPACE,
                             "draft_head_noalloc: the step needs %zu bytes of scratch; the static array "
                             "leaves %zu (DYNA_NOALLOC_SCRATCH_BYTES)",
                             need, kScratchBytes - kChainReserve);
    }
    void* base = nullptr;
    if (B > 0) {
        const dyna_status st = scratch_of_current_device(stream, &base);
        if (st != DYNA_OK) return st;
    }
    char* p = static_cast<char*>(base);
    return draft_head_core(r, L, x, h, adtype, B, k, mode, k_t, temperature, tail_beta, uniforms, out_ids,
                           out_logprobs, out_sample, out_sample_logprob, out_clusters, out_logits, cap,
                           p ? p + kChainReserve : nullptr, kScratchBytes - kChainReserve, stream, nullptr,
                           nullptr, p, false);
}
