// Top-k of the router scores for one context (Sec. 4.2, K = TopK_k(s)),
// with the context's shortlist (V_S = disjoint union of the selected
// clusters) and, for a single context, the gathered-head work plan.
#pragma once
#include "dyna_device.h"

namespace dyna {
namespace {

// One workgroup per context.  Scores (and, for the shortlist, the CSR
// offsets) are staged in LDS in one round trip.  Two 8-bit radix passes over
// the ordered score codes find the 16-bit prefix P of the k-th largest score:
// every code above P is selected, and the few codes sharing P are ranked
// exactly by (score desc, id asc) to fill the remaining places.  The k keys
// are then put in rank order and in ascending id order; with `plan` set (one
// context) the workgroup also writes the gathered-head work plan, so no
// separate plan launch is needed for a single context.
constexpr int kStagePer = 8;  // staged loads in flight per thread

__device__ __forceinline__ void radix_digit(const int* hist, int krem, uint32_t prefix, int shift,
                                            uint32_t* sh_prefix, int* sh_krem) {
    // wave 0: lane l holds digits 255-4l .. 252-4l (descending)
    const int l = lane_id();
    int c[4], sum = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        c[q] = hist[255 - 4 * l - q];
        sum += c[q];
    }
    const int inc = wave_inclusive_scan(sum);
    const int exc = inc - sum;
    if (exc < krem && krem <= inc) {
        int acc = exc;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (acc + c[q] >= krem) {
                *sh_prefix = prefix | ((uint32_t)(255 - 4 * l - q) << shift);
                *sh_krem = krem - acc;
                break;
            }
            acc += c[q];
        }
    }
}


// LDS bytes topk_row needs for M scores and k clusters.
__host__ __device__ inline size_t topk_lds_bytes(int M, int k) {
    return ((size_t)(2 * M + 1) * 4 + 7) / 8 * 8 + (size_t)(k + M) * sizeof(uint64_t) +
           (size_t)2 * k * sizeof(int32_t);
}

// The k best of the M scores sv[] (LDS) by (score desc, id asc), by one
// workgroup of kNT threads.  On return (after a barrier) sel[0..k) holds the
// k selection keys in no particular order, and the int32 arrays rk = (int32_t*)cand
// and ik = rk + k hold, for each key, its rank and its position in ascending
// id order.  `cand` is LDS scratch of M keys.
__device__ void topk_core(const float* sv, int M, int k, uint64_t* sel, uint64_t* cand) {
    __shared__ int hist[256], hist2[256];
    __shared__ uint32_t sh_prefix;
    __shared__ int sh_krem, sh_nsel, sh_ncand;
    hist[threadIdx.x] = 0;
    hist2[threadIdx.x] = 0;
    if (threadIdx.x == 0) {
        sh_nsel = 0;
        sh_ncand = 0;
    }
    __syncthreads();

    // pass 1: top byte
    for (int j = threadIdx.x; j < M; j += kNT) atomicAdd(&hist[ord_f32(sv[j]) >> 24], 1);
    __syncthreads();
    if (threadIdx.x < kWave) radix_digit(hist, k, 0u, 24, &sh_prefix, &sh_krem);
    __syncthreads();
    const uint32_t p1 = sh_prefix;
    const int krem1 = sh_krem;
    // pass 2: second byte inside the chosen top byte
    for (int j = threadIdx.x; j < M; j += kNT) {
        const uint32_t o = ord_f32(sv[j]);
        if ((o & 0xff000000u) == p1) atomicAdd(&hist2[(o >> 16) & 255u], 1);
    }
    __syncthreads();
    if (threadIdx.x < kWave) radix_digit(hist2, krem1, p1, 16, &sh_prefix, &sh_krem);
    __syncthreads();
    const uint32_t P = sh_prefix >> 16;  // 16-bit prefix of the k-th largest code
    const int need = sh_krem;             // places left for codes with prefix P

    // codes above P are in; codes with prefix P are ranked below
    for (int j = threadIdx.x; j < M; j += kNT) {
        const uint32_t o = ord_f32(sv[j]);
        const uint64_t key = (static_cast<uint64_t>(o) << 32) | (0xffffffffu - (uint32_t)j);
        if ((o >> 16) > P) sel[atomicAdd(&sh_nsel, 1)] = key;
        else if ((o >> 16) == P) cand[atomicAdd(&sh_ncand, 1)] = key;
    }
    __syncthreads();
    const int nsel0 = sh_nsel, ncand = sh_ncand;
    for (int c = threadIdx.x; c < ncand; c += kNT) {
        const uint64_t key = cand[c];
        int rank = 0;
        for (int j = 0; j < ncand; ++j) rank += cand[j] > key;
        if (rank < need) sel[nsel0 + rank] = key;
    }
    __syncthreads();

    // rank order (score desc, id asc) and ascending-id order by counting:
    // key i is compared with S slices of the k keys by S threads at once
    // (the tie-candidate array is free again and holds the two counts)
    int32_t* rk = reinterpret_cast<int32_t*>(cand);  // [k]
    int32_t* ik = rk + k;                             // [k]
    for (int i = threadIdx.x; i < k; i += kNT) {
        rk[i] = 0;
        ik[i] = 0;
    }
    __syncthreads();
    {
        const int S = max(1, kNT / k);
        const int span = (k + S - 1) / S;
        for (int wi = threadIdx.x; wi < k * S; wi += kNT) {
            const int i = wi % k, sl = wi / k;
            const uint64_t key = sel[i];
            const uint32_t id = key_id(key);
            const int j0 = sl * span, j1 = min(k, j0 + span);
            int r = 0, q = 0;
            for (int j = j0; j < j1; ++j) {
                const uint64_t o = sel[j];
                r += o > key;
                q += key_id(o) < id;
            }
            if (r) atomicAdd(&rk[i], r);
            if (q) atomicAdd(&ik[i], q);
        }
    }
    __syncthreads();
}

// Row b of the selection, by one workgroup of kTopkThreads threads; `smem`
// holds topk_lds_bytes(M, k) bytes of LDS.
__device__ void topk_row(const TopkArgs& A, int b, unsigned char* smem) {
    const int M = A.M, k = A.k;
    const float* __restrict__ scores = A.scores;
    int32_t* __restrict__ topk_ids = A.topk_ids;
    float* __restrict__ topk_scores = A.topk_scores;
    const int32_t* __restrict__ offsets = A.offsets;
    int32_t* __restrict__ sel_sorted = A.sel_sorted;
    int32_t* __restrict__ sel_rowoff = A.sel_rowoff;
    int32_t* __restrict__ row_len = A.row_len;
    const Plan& plan = A.plan;
    float* sv = reinterpret_cast<float*>(smem);                       // [M] raw scores
    int32_t* offs = reinterpret_cast<int32_t*>(sv + M);                // [M + 1]
    uint64_t* sel = reinterpret_cast<uint64_t*>(smem + ((size_t)(2 * M + 1) * 4 + 7) / 8 * 8);  // [k]
    uint64_t* cand = sel + k;                                          // [M] tie candidates
    int32_t* sid = reinterpret_cast<int32_t*>(cand + M);               // [k] ids ascending
    int32_t* ssize = sid + k;                                          // [k]
    __shared__ int tmp[kNT / kWave + 1];

    // stage scores (and offsets) with kStagePer loads in flight per thread;
    // split-K partial sums are added here in slice order, then the bias
    const float* s = scores + (int64_t)b * M;
    for (int j0 = 0; j0 < M; j0 += kNT * kStagePer) {
        float x[kStagePer];
        if (A.part != nullptr) {
            // eight slices' loads are issued together, then added in order
#pragma unroll
            for (int q = 0; q < kStagePer; ++q) x[q] = 0.0f;
            for (int sl0 = 0; sl0 < A.slices; sl0 += 8) {
                float y[8][kStagePer];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const float* ps = A.part + ((int64_t)(sl0 + u) * gridDim.x + b) * M;
#pragma unroll
                    for (int q = 0; q < kStagePer; ++q) {
                        const int j = j0 + q * kNT + threadIdx.x;
                        y[u][q] = (sl0 + u < A.slices && j < M) ? ps[j] : 0.0f;
                    }
                }
#pragma unroll
                for (int u = 0; u < 8; ++u)
#pragma unroll
                    for (int q = 0; q < kStagePer; ++q)
                        if (sl0 + u < A.slices) x[q] += y[u][q];
            }
#pragma unroll
            for (int q = 0; q < kStagePer; ++q) {
                const int j = j0 + q * kNT + threadIdx.x;
                if (j < M) x[q] = x[q] + (A.bias ? A.bias[j] : 0.0f);
            }
        } else {
#pragma unroll
            for (int q = 0; q < kStagePer; ++q) {
                const int j = j0 + q * kNT + threadIdx.x;
                x[q] = j < M ? s[j] : 0.0f;
            }
        }
#pragma unroll
        for (int q = 0; q < kStagePer; ++q) {
            const int j = j0 + q * kNT + threadIdx.x;
            if (j < M) sv[j] = x[q];
        }
    }
    if (sel_sorted != nullptr) {
        for (int j0 = 0; j0 <= M; j0 += kNT * kStagePer) {
            int x[kStagePer];
#pragma unroll
            for (int q = 0; q < kStagePer; ++q) {
                const int j = j0 + q * kNT + threadIdx.x;
                x[q] = j <= M ? offsets[j] : 0;
            }
#pragma unroll
            for (int q = 0; q < kStagePer; ++q) {
                const int j = j0 + q * kNT + threadIdx.x;
                if (j <= M) offs[j] = x[q];
            }
        }
    }
    topk_core(sv, M, k, sel, cand);
    const int32_t* rk = reinterpret_cast<const int32_t*>(cand);
    const int32_t* ik = rk + k;
    for (int i = threadIdx.x; i < k; i += kNT) {
        const uint32_t id = key_id(sel[i]);
        const int rank = rk[i], idrank = ik[i];
        topk_ids[(int64_t)b * k + rank] = (int32_t)id;
        if (topk_scores) topk_scores[(int64_t)b * k + rank] = sv[id];
        if (sel_sorted != nullptr) {
            sid[idrank] = (int32_t)id;
            ssize[idrank] = offs[id + 1] - offs[id];
        }
    }
    if (sel_sorted == nullptr) return;
    __syncthreads();

    // shortlist: exclusive prefix of the sizes in ascending id order
    const int per = (k + kNT - 1) / kNT;
    const int i0 = min(k, (int)threadIdx.x * per);
    const int i1 = min(k, i0 + per);
    int local = 0, lchunks = 0;
    for (int i = i0; i < i1; ++i) {
        local += ssize[i];
        lchunks += (ssize[i] + kChunkRows - 1) / kChunkRows;
    }
    int len, n_chunks = 0;
    int run = block_exclusive_scan<kNT>(local, tmp, &len);
    int crun = plan.hdr ? block_exclusive_scan<kNT>(lchunks, tmp, &n_chunks) : 0;
    for (int i = i0; i < i1; ++i) {
        const int m = sid[i];
        sel_sorted[(int64_t)b * k + i] = m;
        sel_rowoff[(int64_t)b * (k + 1) + i] = run;
        if (plan.hdr) {
            const int o = offs[m];
            plan.list[i] = ListEntry{b, run - o};
            for (int c = 0; c * kChunkRows < ssize[i]; ++c)
                plan.chunks[crun + c] =
                    Chunk{o + c * kChunkRows, min(kChunkRows, ssize[i] - c * kChunkRows), i, 1};
            crun += (ssize[i] + kChunkRows - 1) / kChunkRows;
        }
        run += ssize[i];
    }
    if (threadIdx.x == 0) {
        sel_rowoff[(int64_t)b * (k + 1) + k] = len;
        row_len[b] = len;
        if (plan.hdr) {
            plan.hdr->n_chunks = n_chunks;
            plan.hdr->n_entries = k;
        }
    }
}

}  // namespace
}  // namespace dyna
