// Draft selection over one context's shortlist logits (Algorithm 1:
// log_softmax, TopK_{k_t}, remap2realid; Sec. 5: inverse-CDF sampling from
// the restricted, renormalised draft q_S).
#pragma once
#include "dyna_device.h"

namespace dyna {
namespace {

// Segments of the long-row selection: 1024 slots (4 per thread) for rows of
// at most 1024 * kNT slots, else 2048 (8 per thread; rows up to kSeg * kNT).
constexpr int kSeg = 2048;
constexpr int kSegShort = 1024;
constexpr int kRowMax = 1 << 17;    // longest shortlist row the one-launch select takes
constexpr int kRowSplit = 1 << 14;  // longer rows may go to the segmented select instead


__device__ __forceinline__ float canon(float z) { return z != z ? -__builtin_inff() : z; }

// Tail mixture proposal (Sec. 5): q~ = (1 - beta) q_S + beta * omega, omega
// uniform on the complement V \ S of the row's shortlist.  An empty
// complement (the shortlist is the whole vocabulary) leaves q~ = q_S.
struct TailMix {
    float beta;    // weight in effect (0: none)
    int64_t comp;  // complement size
    float lshift;  // log(1 - beta), added to shortlist log-probabilities
};
__device__ __forceinline__ TailMix tail_of(const SelectArgs& a, int len) {
    TailMix t{0.0f, 0, 0.0f};
    if (a.beta > 0.0f && a.perm != nullptr && (int64_t)a.V > len) {
        t.beta = a.beta;
        t.comp = (int64_t)a.V - len;
        t.lshift = log1pf(-a.beta);
    }
    return t;
}

// Vocabulary id of complement entry j of row b: layout rows in ascending
// order, skipping the row's selected slabs (sel_sorted is ascending; dropped
// entries are -1 at its end).
__device__ __forceinline__ int32_t complement_vid(const SelectArgs& a, int b, int64_t j) {
    const int32_t* ss = a.sel_sorted + (int64_t)b * a.k;
    int64_t end_prev = 0;
    for (int i = 0; i < a.k; ++i) {
        const int m = ss[i];
        if (m < 0) break;
        const int64_t gap = (int64_t)a.offsets[m] - end_prev;
        if (j < gap) break;
        j -= gap;
        end_prev = a.offsets[m + 1];
    }
    return a.perm[end_prev + j];
}

// Sample draw of row b under the tail mixture: true (and the outputs
// written, by the calling thread) when u falls in the tail branch; else *u_s
// is the uniform for the shortlist branch.
__device__ __forceinline__ bool tail_sample(const SelectArgs& a, int b, const TailMix& t, float* u_s) {
    const float u = a.uniforms[b];
    if (t.beta <= 0.0f) {
        *u_s = u;
        return false;
    }
    if (u < 1.0f - t.beta) {
        *u_s = u / (1.0f - t.beta);
        return false;
    }
    int64_t j = (int64_t)floorf((u - (1.0f - t.beta)) / t.beta * (float)t.comp);
    j = j < 0 ? 0 : (j >= t.comp ? t.comp - 1 : j);
    if (threadIdx.x == 0) {
        a.out_sample[b] = complement_vid(a, b, j);
        if (a.out_sample_logprob) a.out_sample_logprob[b] = logf(t.beta) - logf((float)t.comp);
    }
    return true;
}

// Vocabulary ids of the slots [j0, j0 + n) of row b (1 <= n <= N), written
// into vid[]; with the gathered head's id table the N loads are issued
// together (entries past n repeat the last one).
template <int N>
__device__ __forceinline__ void slot_vids(const SelectArgs& a, int b, int j0, int n, uint32_t (&vid)[N]) {
    if (a.slot_vid != nullptr) {
        const int32_t* sv = a.slot_vid + (int64_t)b * a.vid_ld + j0;
#pragma unroll
        for (int q = 0; q < N; ++q) vid[q] = (uint32_t)sv[q < n ? q : n - 1];
        return;
    }
    if (a.perm == nullptr) {
        for (int q = 0; q < n; ++q) vid[q] = (uint32_t)(j0 + q);
        return;
    }
    const int32_t* ro = a.sel_rowoff + (int64_t)b * (a.k + 1);
    const int32_t* ss = a.sel_sorted + (int64_t)b * a.k;
    // largest ci with ro[ci] <= j0
    int lo = 0, hi = a.k - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (ro[mid] <= j0) lo = mid; else hi = mid - 1;
    }
    int ci = lo;
    int end = ro[ci + 1];
    for (int q = 0; q < n; ++q) {
        const int j = j0 + q;
        while (j >= end) {
            ++ci;
            end = ro[ci + 1];
        }
        const int m = ss[ci];
        vid[q] = (uint32_t)a.perm[a.offsets[m] + (j - ro[ci])];
    }
}

// Block-wide selection of the k_t largest keys (k_t <= KTMAX) from per-thread
// lists sorted descending (list[0] largest, 0 = empty).  Each wave first takes
// its own k_t best keys in k_t rounds of a wave max (no barrier), then wave 0
// takes the k_t best of the waves' candidates.  Thread 0 writes them to out[].
// Keys are unique (they carry the vocabulary id), so a round's winner is one lane.
template <int L, int NT, int KTMAX>
__device__ void block_topk_rounds(uint64_t (&list)[L], int k_t, uint64_t* cand /* LDS [NT / kWave * KTMAX] */,
                                  uint64_t* out /* LDS [k_t] */) {
    constexpr int NW = NT / kWave;
    constexpr int C = (NW * KTMAX + kWave - 1) / kWave;  // candidates per lane of wave 0
    const int lane = lane_id(), w = threadIdx.x / kWave;
    for (int r = 0; r < k_t; ++r) {
        const uint64_t m = wave_max_u64(list[0]);
        if (m != 0 && list[0] == m) {
#pragma unroll
            for (int q = 0; q < L - 1; ++q) list[q] = list[q + 1];
            list[L - 1] = 0;
        }
        if (lane == 0) cand[w * k_t + r] = m;
    }
    __syncthreads();
    if (w == 0) {
        const int nc = NW * k_t;
        uint64_t c[C];
#pragma unroll
        for (int q = 0; q < C; ++q) {
            const int i = lane + q * kWave;
            c[q] = i < nc ? cand[i] : 0;
        }
        // sort the lane's few candidates descending
#pragma unroll
        for (int r = 0; r < C; ++r)
#pragma unroll
            for (int q = r & 1; q + 1 < C; q += 2)
                if (c[q] < c[q + 1]) {
                    const uint64_t t = c[q];
                    c[q] = c[q + 1];
                    c[q + 1] = t;
                }
        for (int r = 0; r < k_t; ++r) {
            const uint64_t m = wave_max_u64(c[0]);
            if (m != 0 && c[0] == m) {
#pragma unroll
                for (int q = 0; q < C - 1; ++q) c[q] = c[q + 1];
                c[C - 1] = 0;
            }
            if (lane == 0) out[r] = m;
        }
    }
    __syncthreads();
}

// Exact top-k_t of per-thread keys held in registers (P per thread, 0 =
// empty; valid keys are distinct and nonzero), by radix selection from the
// most significant byte: each pass counts, among the keys that share the
// prefix fixed so far, the values of the next byte, and fixes the byte that
// holds the k_t-th largest key.  The search stops as soon as the keys sharing
// the prefix are exactly the ones still needed.  The selected keys, sorted
// descending, go to out[0..k_t); missing ones (short rows) are 0.
template <int NT, int P>
__device__ void block_radix_topk(const uint64_t (&kk)[P], int k_t, int n_valid, int* hist /* LDS [256] */,
                                 uint64_t* sel /* LDS [k_t] */, uint64_t* out /* LDS [k_t] */) {
    __shared__ uint64_t sh_prefix;
    __shared__ int sh_need, sh_done, sh_n;
    uint64_t prefix = 0;
    int shift = 64;
    if (n_valid > k_t) {
        uint64_t mask = 0;
        int need = k_t;
        for (int byte = 7; byte >= 0; --byte) {
            for (int i = threadIdx.x; i < 256; i += NT) hist[i] = 0;
            __syncthreads();
            const int sh = 8 * byte;
#pragma unroll
            for (int q = 0; q < P; ++q)
                if (kk[q] != 0 && (kk[q] & mask) == prefix) atomicAdd(&hist[(int)((kk[q] >> sh) & 255u)], 1);
            __syncthreads();
            if (threadIdx.x < kWave) {
                // lane l holds digits 255-4l .. 252-4l (descending)
                const int l = lane_id();
                int c[4], sum = 0;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    c[q] = hist[255 - 4 * l - q];
                    sum += c[q];
                }
                const int inc = wave_inclusive_scan(sum);
                const int exc = inc - sum;
                if (exc < need && need <= inc) {
                    int acc = exc;
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        if (acc + c[q] >= need) {
                            sh_prefix = prefix | ((uint64_t)(255 - 4 * l - q) << sh);
                            sh_need = need - acc;
                            sh_done = c[q] == need - acc;
                            break;
                        }
                        acc += c[q];
                    }
                }
            }
            __syncthreads();
            prefix = sh_prefix;
            need = sh_need;
            mask |= (uint64_t)255u << sh;
            shift = sh;
            const int done = sh_done;
            __syncthreads();  // every thread has read the shared values
            if (done) break;
        }
    }
    if (threadIdx.x == 0) sh_n = 0;
    __syncthreads();
    // selected: the keys whose bits from `shift` up are at least the prefix's
#pragma unroll
    for (int q = 0; q < P; ++q)
        if (kk[q] != 0 && (shift == 64 || (kk[q] >> shift) >= (prefix >> shift))) sel[atomicAdd(&sh_n, 1)] = kk[q];
    __syncthreads();
    const int n = sh_n;  // k_t, or fewer for a short row
    for (int i = threadIdx.x; i < k_t; i += NT) {
        if (i >= n) {
            out[i] = 0;
            continue;
        }
        const uint64_t key = sel[i];
        int rank = 0;
        for (int j = 0; j < n; ++j) rank += sel[j] > key;
        out[rank] = key;
    }
    __syncthreads();
}

// Whole-row selection in one workgroup (shortlist-sized rows, k_t <= KT).
// Max, top-k_t and the softmax sum read the row with coalesced strided loads;
// only the sampling walk uses contiguous per-thread ranges, so that the CDF
// runs in shortlist order.  Vocabulary ids come from the gathered head's
// per-slot ids when present, else from the shortlist's cluster table staged
// in LDS.
constexpr int kRowTable = 1024;  // clusters per row the LDS table holds
constexpr int kRowThreads = 1024;  // threads per row: a few slots each

template <int KT, int NT>
__device__ void select_row(const SelectArgs& a, int b) {
    __shared__ uint64_t cand[NT / kWave * KT];
    __shared__ uint64_t top[KT];
    __shared__ float red[2 * (NT / kWave) + 1];
    __shared__ float incl_s[NT];
    __shared__ int sh_pick;
    __shared__ int32_t t_ro[kRowTable + 1];
    __shared__ int32_t t_base[kRowTable];
    const int len = a.row_len ? a.row_len[b] : a.fixed_len;
    const float* z = a.logits + (int64_t)b * a.ld;
    const int32_t* sv = a.slot_vid ? a.slot_vid + (int64_t)b * a.vid_ld : nullptr;
    const bool table = sv == nullptr && a.perm != nullptr;
    if (table) {  // slot -> layout row: rows of cluster ci start at t_base[ci] + slot
        const int32_t* ro = a.sel_rowoff + (int64_t)b * (a.k + 1);
        const int32_t* ss = a.sel_sorted + (int64_t)b * a.k;
        for (int c = threadIdx.x; c <= a.k; c += NT) {
            t_ro[c] = ro[c];
            if (c < a.k) t_base[c] = ss[c] >= 0 ? a.offsets[ss[c]] - ro[c] : 0;
        }
        __syncthreads();
    }
    auto vid_of = [&](int j) -> uint32_t {
        if (sv != nullptr) return (uint32_t)sv[j];
        if (a.perm == nullptr) return (uint32_t)j;
        int lo = 0, hi = a.k - 1;  // largest ci with ro[ci] <= j
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (t_ro[mid] <= j) lo = mid; else hi = mid - 1;
        }
        return (uint32_t)a.perm[t_base[lo] + j];
    };

    constexpr int kRegPer = 8;  // rows up to NT * kRegPer slots keep their keys in registers
    if (KT > 1 && len <= NT * kRegPer) {
        __shared__ int rhist[256];
        __shared__ uint64_t rsel[KT];
        uint64_t kk[kRegPer];
#pragma unroll
        for (int q = 0; q < kRegPer; ++q) {
            const int j = q * NT + threadIdx.x;
            kk[q] = j < len ? sel_key(canon(z[j]), vid_of(j)) : 0;
        }
        block_radix_topk<NT, kRegPer>(kk, a.k_t, len, rhist, rsel, top);
    } else {
        uint64_t list[KT];
#pragma unroll
        for (int q = 0; q < KT; ++q) list[q] = 0;
        // kLoadPer slots per thread per batch, their loads issued together
        constexpr int kLoadPer = 4;
        for (int j0 = 0; j0 < len; j0 += NT * kLoadPer) {
            float zq[kLoadPer];
            uint32_t vq[kLoadPer];
#pragma unroll
            for (int q = 0; q < kLoadPer; ++q) {
                const int j = j0 + q * NT + threadIdx.x;
                zq[q] = j < len ? z[j] : 0.0f;
                vq[q] = j < len ? vid_of(j) : 0u;
            }
#pragma unroll
            for (int q = 0; q < kLoadPer; ++q) {
                if (j0 + q * NT + (int)threadIdx.x >= len) continue;
                const uint64_t key = sel_key(canon(zq[q]), vq[q]);
                if (key > list[KT - 1]) {
                    list[KT - 1] = key;
#pragma unroll
                    for (int r = KT - 1; r > 0; --r)
                        if (list[r] > list[r - 1]) {
                            const uint64_t t = list[r];
                            list[r] = list[r - 1];
                            list[r - 1] = t;
                        }
                }
            }
        }
        block_topk_rounds<KT, NT, KT>(list, a.k_t, cand, top);
    }
    const float mx = top[0] != 0 ? key_val(top[0]) : -__builtin_inff();
    const bool sampling = a.uniforms != nullptr && a.out_sample != nullptr;

    // softmax mass: strided when only top-k is asked, contiguous ranges
    // (shortlist order) when a sample must be drawn from the same sums
    const int E = (len + NT - 1) / NT;
    const int j0 = min(len, (int)threadIdx.x * E);
    const int j1 = min(len, j0 + E);
    float tsum = 0.0f;
    if (mx != -__builtin_inff()) {
        if (sampling) {
            for (int j = j0; j < j1; ++j) tsum += expf((canon(z[j]) - mx) * a.inv_t);
        } else {
#pragma unroll 4
            for (int j = threadIdx.x; j < len; j += NT) tsum += expf((canon(z[j]) - mx) * a.inv_t);
        }
    }
    float total;
    const float incl = block_inclusive_scan_f32<NT>(tsum, red, &total);
    const TailMix tail = tail_of(a, len);
    const float log_total = logf(total) - tail.lshift;
    if (a.out_ids != nullptr) {
        for (int r = threadIdx.x; r < a.k_t; r += NT) {
            const uint64_t key = top[r];
            a.out_ids[(int64_t)b * a.k_t + r] = key != 0 ? (int32_t)key_id(key) : -1;
            if (a.out_logprobs)
                a.out_logprobs[(int64_t)b * a.k_t + r] =
                    key != 0 ? (key_val(key) - mx) * a.inv_t - log_total : -__builtin_inff();
        }
    }
    if (!sampling) return;
    float u_s;
    if (tail_sample(a, b, tail, &u_s)) return;  // uniform decision for the block

    incl_s[threadIdx.x] = incl;
    if (threadIdx.x == 0) sh_pick = -1;
    __syncthreads();
    const float excl = threadIdx.x > 0 ? incl_s[threadIdx.x - 1] : 0.0f;
    const float target = u_s * total;
    if (tsum > 0.0f && excl <= target && target < incl) {
        float acc = excl;
        int pick = -1, last = -1;
        for (int j = j0; j < j1; ++j) {
            const float e = expf((canon(z[j]) - mx) * a.inv_t);
            if (e > 0.0f) last = j;
            acc += e;
            if (e > 0.0f && acc > target) {
                pick = j;
                break;
            }
        }
        atomicMax(&sh_pick, pick >= 0 ? pick : last);
    }
    __syncthreads();
    if (sh_pick < 0 && tsum > 0.0f) {  // rounding: the last slot with mass
        int last = -1;
        for (int j = j0; j < j1; ++j)
            if (expf((canon(z[j]) - mx) * a.inv_t) > 0.0f) last = j;
        atomicMax(&sh_pick, last);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        const int j = sh_pick;
        if (j < 0) {
            a.out_sample[b] = -1;
            if (a.out_sample_logprob) a.out_sample_logprob[b] = -__builtin_inff();
        } else {
            a.out_sample[b] = (int32_t)vid_of(j);
            if (a.out_sample_logprob) a.out_sample_logprob[b] = (canon(z[j]) - mx) * a.inv_t - log_total;
        }
    }
}

}  // namespace
}  // namespace dyna
