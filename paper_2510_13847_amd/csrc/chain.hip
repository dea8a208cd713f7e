// One-context draft step in a single launch (B = 1): router layer 1, router
// layer 2, top-k clusters and shortlist, gathered logits and the argmax or
// top-k_t selection (Sec. 4.2 and Sec. 4.3; Algorithm 1, one draft step).
//
// With one context every stage is small (the chain workload moves 8 MB,
// 2 MB, 4 KB and 33 MB), so as separate kernels the step is dominated by
// launch gaps and by each kernel's cold start.  Here one grid of G
// workgroups runs all of them, with two grid-wide hand-offs and a final
// gather of per-workgroup partials:
//
//   1. every wave dots its rows of W1 with x (x in registers), writes the
//      hidden units with device-coherent stores and starts loading its W2
//      row for stage 2;
//   2. after all workgroups arrived, each stages the hidden layer in LDS and
//      dots its prefetched W2 rows with it, writing the scores;
//   3. after all arrived again, every workgroup reads the M scores into LDS
//      and takes the top-k itself (the same deterministic selection in every
//      workgroup, so no further hand-off), sorts the k ids ascending and
//      forms the shortlist offsets;
//   4. the shortlist rows are split evenly over all waves as contiguous
//      ranges (a range may cross slab boundaries), streamed with
//      non-temporal 16-byte loads and dotted with h (in registers);
//   5. each workgroup publishes its greedy partial; workgroup 0 polls them,
//      merges them in workgroup order and writes the token, and the last
//      workgroup writes the selection outputs.  For top-k_t (k_t <= 16) a
//      partial also carries the workgroup's k_t best keys, and workgroup 0
//      takes the k_t best of all of them.
//
// Hand-off protocol: every handed-off word is 64 bits, a 32-bit epoch tag
// above the 32-bit value, written with one device-coherent store; readers
// poll the words themselves with coherent loads until every tag equals the
// launch's epoch, so the data carries its own ready signal (one store and
// one load round trip, no counter).  The epoch is one more than the value a
// workspace word holds at launch; workgroup 0 stores it back after the
// merge, when every workgroup has read it.  A zero-filled workspace starts
// at epoch 1, above the tags of its zero words.  Every poll is bounded in
// time: a word that never turns current (the grid is not co-resident, or a
// workspace that was not zero-filled) sets an error word and marks the
// workgroup's partial, the poll gives up, and the launch reports no token
// (out_ids = -1) but still terminates.
#include <atomic>
#include <mutex>

#include "dyna_internal.h"
#include "gemv.h"
#include "greedy.h"
#include "topk.h"

namespace dyna {
namespace {

constexpr int kChainThreads = kThreads;  // 4 waves per workgroup
constexpr int kChainWaves = kChainThreads / kWave;

// words of the chain region of the workspace: epoch, error, then tagged
// hidden [H], scores [M] and partials [G][3] (best key high, low; sum of
// exponentials: the partial's maximum logit is its best key's value).  A
// top-k_t partial adds the keys of places 1 .. k_t - 1 (high, low), at a
// stride of kPartWordsTopk words.
constexpr int kPartWords = 3;
constexpr int kChainTopkMax = 16;
constexpr int kPartWordsTopk = kPartWords + 2 * (kChainTopkMax - 1);
constexpr int kChainMaxGrid = 1024;  // workgroups at most (twice the compute units, capped)

struct ChainArgs {
    // router: H == 0 is a single linear layer W1 [M, d_r]
    const uint16_t* W1;
    const float* b1;
    const uint16_t* W2;
    const float* b2;
    int32_t d_r, H, M, act;
    const uint16_t* x;  // [d_r]
    // layout
    const uint16_t* W;  // [V, d] permuted LM head
    const int32_t* perm;
    const int32_t* offsets;
    int32_t d, V;
    const uint16_t* h;  // [d]
    int32_t k;
    // workspace (chain region)
    uint32_t* epoch;     // [1]
    uint32_t* err;       // [1]
    uint64_t* thidden;   // [H] tagged
    uint64_t* tscores;   // [M] tagged
    uint64_t* tpart;     // [G][kPartWords] tagged
    // outputs (each may be null except out_ids)
    int32_t* out_clusters;  // [k] rank order
    float* topk_scores;     // [k]
    int32_t* sel_sorted;    // [k]
    int32_t* sel_rowoff;    // [k + 1]
    int32_t* row_len;       // [1]
    float* out_logits;      // [cap], shortlist order
    int32_t* out_ids;       // [k_t]
    float* out_logprobs;    // [k_t]
    int32_t k_t;
    float inv_t, beta;
    uint64_t spin_ticks;  // bound of every wait, in wall-clock ticks
};

// Bytes of dynamic LDS: scores [M], offsets [M + 1], candidate keys [M],
// shortlist ids [k], offsets [k + 1] and slab starts [k], hidden [H].
__host__ __device__ inline size_t chain_lds_bytes(int M, int k, int H) {
    size_t b = (size_t)M * 4 + (size_t)(M + 1) * 4;
    b = (b + 15) / 16 * 16;
    b += (size_t)M * 8;
    b += (size_t)k * 4 + (size_t)(k + 1) * 4 + (size_t)k * 4;
    b = (b + 15) / 16 * 16;
    b += (size_t)H * 4;
    return b;
}

__device__ __forceinline__ uint64_t tagged(uint32_t e, uint32_t v) { return ((uint64_t)e << 32) | v; }

// Thread t reads the tagged words src[t + NT q], q < Q (those below n), into
// raw[q], re-polling its stale ones together until they carry epoch e or
// the time bound runs out.  Returns true if it gave up.
template <int NT, int Q>
__device__ __forceinline__ bool poll_own(const ChainArgs& A, const uint64_t* src, int n, uint32_t e,
                                         uint32_t (&raw)[Q]) {
    bool gave_up = false;
    const uint64_t t0 = wall_clock64();
    uint64_t v[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int j = (int)threadIdx.x + NT * q;
        v[q] = j < n ? load_coherent(src + j) : tagged(e, 0u);
    }
    for (;;) {
        bool stale = false;
#pragma unroll
        for (int q = 0; q < Q; ++q) stale |= (uint32_t)(v[q] >> 32) != e;
        if (!stale) break;
        if (wall_clock64() - t0 > A.spin_ticks) {
            store_coherent(A.err, e);
            gave_up = true;
            break;
        }
        __builtin_amdgcn_s_sleep(1);
#pragma unroll
        for (int q = 0; q < Q; ++q)
            if ((uint32_t)(v[q] >> 32) != e) v[q] = load_coherent(src + (int)threadIdx.x + NT * q);
    }
#pragma unroll
    for (int q = 0; q < Q; ++q) raw[q] = (uint32_t)v[q];
    return gave_up;
}

// Reads n tagged words src[0..n) into dst (as raw 32-bit values), workgroup
// wide, NT * 4 words per pass (poll_own per pass; passes of 8 words per
// thread measured slower).  Returns true in a thread that gave up.
template <int NT>
__device__ __forceinline__ bool poll_words(const ChainArgs& A, const uint64_t* src, int n, uint32_t e,
                                           uint32_t* dst) {
    constexpr int Q = 4;
    bool gave_up = false;
    for (int base = 0; base < n; base += NT * Q) {
        uint32_t raw[Q];
        gave_up |= poll_own<NT, Q>(A, src + base, n - base, e, raw);
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int j = base + q * NT + (int)threadIdx.x;
            if (j < n) dst[j] = raw[q];
        }
    }
    return gave_up;
}

template <int NB>
__device__ __forceinline__ void load_bf16_row(Raw8<uint16_t> (&w)[NB], const uint16_t* row, int K, int lane) {
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) {
        const int e = blk * 512 + lane * 8;
        if (e < K) w[blk].template load<true>(row + e);
        else w[blk].zero();
    }
}

template <int NB>
__device__ __forceinline__ float dot_bf16(const Raw8<uint16_t> (&w)[NB], const Raw8<uint16_t> (&v)[NB]) {
    float acc = 0.0f;
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) acc = dot8(w[blk], v[blk], acc);
    return wave_sum(acc);
}

// Row . hidden, the hidden layer (fp32) in LDS.
template <int NB>
__device__ __forceinline__ float dot_lds(const Raw8<uint16_t> (&w)[NB], const float* hid, int K, int lane) {
    float acc = 0.0f;
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) {
        const int e = blk * 512 + lane * 8;
        if (e < K) {
            const f32x4 a = *reinterpret_cast<const f32x4*>(hid + e);
            const f32x4 b = *reinterpret_cast<const f32x4*>(hid + e + 4);
#pragma unroll
            for (int j = 0; j < 4; ++j) acc = fmaf(w[blk].at(j), a[j], acc);
#pragma unroll
            for (int j = 0; j < 4; ++j) acc = fmaf(w[blk].at(4 + j), b[j], acc);
        }
    }
    return wave_sum(acc);
}

// Scores per thread in the selection: thread t holds ids kSelQ t + q.
constexpr int kSelQ = 4;
constexpr int kChainMaxM = kChainThreads * kSelQ;
// Shortlist lengths stay below 2^kLenBits (the layout scan packs the member
// count above the length in one 32-bit word).
constexpr int kLenBits = 21;

// Thread t reads the tagged words src[Q t + q], q < Q (those below n), into
// raw[q], re-polling its stale ones together until they carry epoch e or the
// time bound runs out.  Returns true if it gave up.
template <int Q>
__device__ __forceinline__ bool poll_run(const ChainArgs& A, const uint64_t* src, int n, uint32_t e,
                                         uint32_t (&raw)[Q]) {
    bool gave_up = false;
    const uint64_t t0 = wall_clock64();
    const int j0 = (int)threadIdx.x * Q;
    uint64_t v[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) v[q] = j0 + q < n ? load_coherent(src + j0 + q) : tagged(e, 0u);
    for (;;) {
        bool stale = false;
#pragma unroll
        for (int q = 0; q < Q; ++q) stale |= (uint32_t)(v[q] >> 32) != e;
        if (!stale) break;
        if (wall_clock64() - t0 > A.spin_ticks) {
            store_coherent(A.err, e);
            gave_up = true;
            break;
        }
        __builtin_amdgcn_s_sleep(1);
#pragma unroll
        for (int q = 0; q < Q; ++q)
            if ((uint32_t)(v[q] >> 32) != e) v[q] = load_coherent(src + j0 + q);
    }
#pragma unroll
    for (int q = 0; q < Q; ++q) raw[q] = (uint32_t)v[q];
    return gave_up;
}

// Minimum and maximum over the wave (on lane 63), the two reductions
// interleaved step by step.
__device__ __forceinline__ void wave_min_max(float& lo, float& hi) {
    auto step = [&](auto ctrl_tag, auto rmask_tag) {
        constexpr int CTRL = decltype(ctrl_tag)::value;
        constexpr int RM = decltype(rmask_tag)::value;
        const float l2 = __uint_as_float(dpp<CTRL, RM>(__float_as_uint(__builtin_inff()), __float_as_uint(lo)));
        const float h2 = __uint_as_float(dpp<CTRL, RM>(__float_as_uint(-__builtin_inff()), __float_as_uint(hi)));
        lo = fminf(lo, l2);
        hi = fmaxf(hi, h2);
    };
    step(std::integral_constant<int, kRowShr1>{}, std::integral_constant<int, 0xf>{});
    step(std::integral_constant<int, kRowShr2>{}, std::integral_constant<int, 0xf>{});
    step(std::integral_constant<int, kRowShr4>{}, std::integral_constant<int, 0xf>{});
    step(std::integral_constant<int, kRowShr8>{}, std::integral_constant<int, 0xf>{});
    step(std::integral_constant<int, kRowBcast15>{}, std::integral_constant<int, 0xa>{});
    step(std::integral_constant<int, kRowBcast31>{}, std::integral_constant<int, 0xc>{});
}

// Lane l of one wave reads the partials g = l + 64 (u0 + u), u < U (those
// below G; kPartWords tagged words each) into raw, re-reading them all
// together until every word carries epoch e or the time bound runs out.
// Every read is issued without a branch (lanes past G re-read partial
// G - 1), so that one round is one round trip.  Returns true if it gave up.
template <int U>
__device__ __forceinline__ bool poll_parts(const ChainArgs& A, const uint64_t* src, int G, int u0, uint32_t e,
                                           uint32_t (&raw)[U * kPartWords]) {
    constexpr int P = kPartWords;
    bool gave_up = false;
    const uint64_t t0 = wall_clock64();
    const int l = lane_id();
    const uint64_t* ps[U];
    bool in[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int g = l + kWave * (u0 + u);
        in[u] = g < G;
        ps[u] = src + (int64_t)min(g, G - 1) * P;
    }
    uint64_t v[U * P];
    for (;;) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int w = 0; w < P; ++w) v[u * P + w] = load_coherent(ps[u] + w);
        bool stale = false;
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int w = 0; w < P; ++w) stale |= in[u] && (uint32_t)(v[u * P + w] >> 32) != e;
        if (!stale) break;
        if (wall_clock64() - t0 > A.spin_ticks) {
            store_coherent(A.err, e);
            gave_up = true;
            break;
        }
        __builtin_amdgcn_s_sleep(1);
    }
#pragma unroll
    for (int q = 0; q < U * P; ++q) raw[q] = (uint32_t)v[q];
    return gave_up;
}

// One thread reads the n <= P tagged words src[0..n) into raw, re-reading its
// stale ones together until every word carries epoch e or the time bound
// runs out.  Returns true if it gave up.
template <int P>
__device__ __forceinline__ bool poll_span(const ChainArgs& A, const uint64_t* src, int n, uint32_t e,
                                          uint32_t (&raw)[P]) {
    bool gave_up = false;
    const uint64_t t0 = wall_clock64();
    uint64_t v[P];
#pragma unroll
    for (int w = 0; w < P; ++w) v[w] = w < n ? load_coherent(src + w) : tagged(e, 0u);
    for (;;) {
        bool stale = false;
#pragma unroll
        for (int w = 0; w < P; ++w) stale |= (uint32_t)(v[w] >> 32) != e;
        if (!stale) break;
        if (wall_clock64() - t0 > A.spin_ticks) {
            store_coherent(A.err, e);
            gave_up = true;
            break;
        }
        __builtin_amdgcn_s_sleep(1);
#pragma unroll
        for (int w = 0; w < P; ++w)
            if ((uint32_t)(v[w] >> 32) != e) v[w] = load_coherent(src + w);
    }
#pragma unroll
    for (int w = 0; w < P; ++w) raw[w] = (uint32_t)v[w];
    return gave_up;
}

// The k best of the M <= NT * kSelQ scores v[] (registers; thread t holds
// ids kSelQ t + q) by (score desc, id asc), as the shortlist in ascending
// cluster id: sid[0..k) the ids, mkey[0..k) their (score, id) keys,
// rowoff[0..k] the exclusive prefix of their slab sizes, sbase[0..k) their
// slabs' first layout rows.  Returns the
// shortlist length; sets `bad` in thread 0 when the members are not k.
//
// Each score gets a class that is monotone in the score: 0 for -inf and
// NaN, 255 for +inf, and for finite scores 1 + one of 254 equal-width bins
// between the finite minimum and maximum (so the bins follow the values,
// whatever their scale).  One histogram, scanned from the top by every wave,
// gives the class c* of the k-th best and the number `need` of places left
// in it; classes above c* are members, and the few scores in class c* are
// ranked exactly by their (score, id) keys.  With consecutive ids in each
// thread, thread order is id order, so one scan of (member count, slab
// length) per thread lays out the shortlist.  The member keys reuse the
// candidate area (cand[0..k)), which the ranking has finished reading by then.
template <int NT>
__device__ __forceinline__ int chain_select(const float (&v)[kSelQ], const int32_t* offs, int M, int k,
                                            uint64_t* cand, int32_t* sid, int32_t* rowoff, int32_t* sbase,
                                            uint32_t* err, uint32_t e, bool& bad) {
    static_assert(NT == 256, "one histogram bin per thread");
    constexpr int NW = NT / kWave;
    constexpr int Q = kSelQ;
    __shared__ __attribute__((aligned(16))) int hist[256];
    __shared__ float s_lo[NW], s_hi[NW];
    __shared__ int s_nc[NW];
    __shared__ uint32_t s_tot[NW];
    const float inf = __builtin_inff();
    const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
    const int id0 = t * Q;
    bool valid[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) valid[q] = id0 + q < M;

    // range of the finite scores
    float lo = inf, hi = -inf;
#pragma unroll
    for (int q = 0; q < Q; ++q)
        if (valid[q] && v[q] - v[q] == 0.0f) {
            lo = fminf(lo, v[q]);
            hi = fmaxf(hi, v[q]);
        }
    hist[t] = 0;
    wave_min_max(lo, hi);
    if (lane == kWave - 1) {
        s_lo[w] = lo;
        s_hi[w] = hi;
    }
    __syncthreads();
    lo = s_lo[0];
    hi = s_hi[0];
#pragma unroll
    for (int q = 1; q < NW; ++q) {
        lo = fminf(lo, s_lo[q]);
        hi = fmaxf(hi, s_hi[q]);
    }
    const float span = hi - lo;
    const float scale = (hi > lo && span < inf) ? 254.0f / span : 0.0f;
    int c[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const float x = v[q];
        int cl;
        if (x != x || x == -inf) cl = 0;
        else if (x == inf) cl = 255;
        else cl = 1 + min((int)((x - lo) * scale), 253);
        c[q] = valid[q] ? cl : -1;
        if (valid[q]) atomicAdd(&hist[cl], 1);
    }
    __syncthreads();

    // every wave scans the histogram from the top (lane l: classes 255 - 4l
    // down to 252 - 4l) and finds the class of the k-th best and the places
    // left in it, on every lane
    int cstar, need;
    {
        const int4 h4 = *reinterpret_cast<const int4*>(hist + 252 - 4 * lane);
        const int cc[4] = {h4.w, h4.z, h4.y, h4.x};
        const int sum = cc[0] + cc[1] + cc[2] + cc[3];
        const int inc = wave_inclusive_scan(sum);
        const int exc = inc - sum;
        const bool mine = exc < k && k <= inc;
        int cs = 0, nd = 0, acc = exc;
        bool found = false;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (!found && acc + cc[q] >= k) {
                cs = 255 - 4 * lane - q;
                nd = k - acc;
                found = true;
            }
            acc += cc[q];
        }
        const uint64_t bal = __ballot(mine);
        const int src = bal ? (int)__builtin_ctzll(bal) : 0;
        cstar = __builtin_amdgcn_readlane(cs, src);
        need = __builtin_amdgcn_readlane(nd, src);
    }

    // members above c*; the scores in c* are collected per wave and ranked
    // by their owners
    bool mem[Q], isc[Q];
    uint64_t key[Q];
    uint64_t* seg = cand + (int64_t)w * kWave * Q;
    int nc = 0;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        mem[q] = c[q] > cstar;
        isc[q] = c[q] == cstar;
        key[q] = sel_key(v[q], (uint32_t)(id0 + q));
        const uint64_t bal = __ballot(isc[q]);
        if (isc[q])
            seg[nc + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                    __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u))] = key[q];
        nc += __popcll(bal);
    }
    if (lane == 0) s_nc[w] = nc;
    __syncthreads();
    int ntot = 0;
#pragma unroll
    for (int g = 0; g < NW; ++g) ntot += s_nc[g];
#pragma unroll
    for (int q = 0; q < Q; ++q)
        if (isc[q]) {
            int rank = 0;
            if (ntot != need)
                for (int g = 0; g < NW; ++g) {
                    const uint64_t* sg = cand + (int64_t)g * kWave * Q;
                    for (int j = 0; j < s_nc[g]; ++j) rank += sg[j] > key[q];
                }
            mem[q] = rank < need;
        }

    // the shortlist in ascending id, which is thread order: one scan of the
    // packed (member count, slab length) of each thread
    int sz[Q], base[Q];
    uint32_t mine = 0;
    {
        int o[Q + 1];
        if ((M & 3) == 0 && id0 + Q <= M) {  // offs + id0 is 16-byte aligned
            const int4 o4 = *reinterpret_cast<const int4*>(offs + id0);
            o[0] = o4.x;
            o[1] = o4.y;
            o[2] = o4.z;
            o[3] = o4.w;
            o[4] = offs[id0 + Q];
        } else {
#pragma unroll
            for (int q = 0; q <= Q; ++q) o[q] = offs[min(id0 + q, M)];
        }
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            base[q] = o[q];
            sz[q] = mem[q] ? o[q + 1] - o[q] : 0;
            mine += (mem[q] ? 1u << kLenBits : 0u) + (uint32_t)sz[q];
        }
    }
    const uint32_t inc = (uint32_t)wave_inclusive_scan((int)mine);
    if (lane == kWave - 1) s_tot[w] = inc;
    __syncthreads();
    uint32_t pre = inc - mine, total = 0;
#pragma unroll
    for (int g = 0; g < NW; ++g) {
        const uint32_t tg = s_tot[g];
        if (g < w) pre += tg;
        total += tg;
    }
    constexpr uint32_t kLenMask = (1u << kLenBits) - 1u;
    int pos = (int)(pre >> kLenBits), off = (int)(pre & kLenMask);
#pragma unroll
    for (int q = 0; q < Q; ++q)
        if (mem[q]) {
            if (pos < k) {
                sid[pos] = id0 + q;
                cand[pos] = key[q];
                rowoff[pos] = off;
                sbase[pos] = base[q];
            }
            ++pos;
            off += sz[q];
        }
    const int total_cnt = (int)(total >> kLenBits), total_len = (int)(total & kLenMask);
    if (t == 0) {
        rowoff[k] = total_len;
        if (total_cnt != k) {
            store_coherent(err, e);
            bad = true;
        }
    }
    __syncthreads();
    return total_len;
}

// The selection outputs of one workgroup: the ids and slab offsets in
// ascending id, the shortlist length, and the k clusters in rank order
// (score desc, id asc) with their scores.  A member's rank is the number of
// members with a larger key; P lanes share each member's count.
template <int NT>
__device__ __forceinline__ void chain_outputs(const ChainArgs& A, const float* sv, const int32_t* sid,
                                              const uint64_t* mkey, const int32_t* rowoff, int k, int L) {
    for (int i = threadIdx.x; i <= k; i += NT) {
        if (i < k && A.sel_sorted) A.sel_sorted[i] = sid[i];
        if (A.sel_rowoff) A.sel_rowoff[i] = rowoff[i];
    }
    if (threadIdx.x == 0 && A.row_len) A.row_len[0] = L;
    if (!A.out_clusters && !A.topk_scores) return;
    constexpr int P = 8;
    const int part = threadIdx.x % P;
    for (int i0 = 0; i0 < k; i0 += NT / P) {
        const int i = i0 + (int)threadIdx.x / P;
        const uint64_t key = i < k ? mkey[i] : 0;
        int rank = 0;
        if (i < k)
            for (int j = part; j < k; j += P) rank += mkey[j] > key;
        rank += __shfl_xor(rank, 1);
        rank += __shfl_xor(rank, 2);
        rank += __shfl_xor(rank, 4);
        if (i < k && part == 0) {
            if (A.out_clusters) A.out_clusters[rank] = sid[i];
            if (A.topk_scores) A.topk_scores[rank] = sv[sid[i]];
        }
    }
}

// Stage 5 of the top-k_t step.  Every workgroup ranks its waves' k_t best
// keys by counting and publishes them with its softmax pair (tagged words);
// workgroup 0 polls the partials, one per thread, takes the k_t best of all
// of them (the k_t-th best partial head bounds the answer from below) and
// merges the softmax pairs in a fixed order; the last workgroup writes the
// selection outputs.
template <int NT>
__device__ void chain_topk_finish(const ChainArgs& A, const GreedyState& st, uint64_t wk, bool bad, uint32_t e,
                                  int G, const float* sv, const int32_t* sid, const uint64_t* mkey,
                                  const int32_t* rowoff, int k, int L) {
    constexpr int NW = NT / kWave;
    constexpr int KT = kChainTopkMax;
    __shared__ uint64_t t_cand[KT * KT];
    __shared__ uint64_t t_top[KT];
    __shared__ uint64_t t_heads[NT];
    __shared__ float w_m[NW], w_s[NW], f_m, f_s;
    __shared__ int w_bad[NW], f_bad;
    const int kt = A.k_t;
    const int lane = lane_id(), wv = threadIdx.x / kWave;
    // the wave's softmax pair (its maximum logit is its best key's value)
    const uint64_t wb = wave_max_u64(st.best);
    const float wm = wb != 0 ? key_val(wb) : -__builtin_inff();
    const float wsum = wave_sum(st.m == -__builtin_inff() ? 0.0f : st.s * expf((st.m - wm) * A.inv_t));
    const bool wbad = __ballot(bad) != 0;
    if ((int)threadIdx.x < kt) t_top[threadIdx.x] = 0;
    if (lane < kt) t_cand[wv * kt + lane] = wk;
    if (lane == 0) {
        w_m[wv] = wm;
        w_s[wv] = wsum;
        w_bad[wv] = wbad;
    }
    __syncthreads();
    if ((int)threadIdx.x < NW * kt) {
        const uint64_t key = t_cand[threadIdx.x];
        int rank = 0;
        for (int j = 0; j < NW * kt; ++j) rank += t_cand[j] > key;
        if (key != 0 && rank < kt) t_top[rank] = key;
    }
    if (threadIdx.x == 0) {
        float bm = w_m[0], bs = w_s[0];
        int any_bad = w_bad[0];
        for (int q = 1; q < NW; ++q) {
            softmax_merge(bm, bs, w_m[q], w_s[q], A.inv_t);
            any_bad |= w_bad[q];
        }
        f_s = any_bad ? -1.0f : bs;
    }
    __syncthreads();
    // publish: words 0, 1 the best key, 2 the sum, then places 1 .. kt - 1
    uint64_t* pw = A.tpart + (int64_t)blockIdx.x * kPartWordsTopk;
    if ((int)threadIdx.x < kt) {
        const uint64_t key = t_top[threadIdx.x];
        const int w0 = threadIdx.x == 0 ? 0 : kPartWords + 2 * ((int)threadIdx.x - 1);
        store_coherent(pw + w0, tagged(e, (uint32_t)(key >> 32)));
        store_coherent(pw + w0 + 1, tagged(e, (uint32_t)key));
    }
    if (threadIdx.x == 0) store_coherent(pw + 2, tagged(e, __float_as_uint(f_s)));
    if (blockIdx.x == G - 1) chain_outputs<NT>(A, sv, sid, mkey, rowoff, k, L);
    if (blockIdx.x != 0) return;

    // workgroup 0: thread t polls partials t, t + NT, ... and keeps their
    // keys as one sorted list
    const uint32_t err_word = load_coherent(A.err);
    const int nwords = kPartWords + 2 * (kt - 1);
    uint64_t list[KT];
#pragma unroll
    for (int r = 0; r < KT; ++r) list[r] = 0;
    float bm = -__builtin_inff(), bs = 0.0f;
    bool fail = false;
    for (int g = threadIdx.x; g < G; g += NT) {
        uint32_t raw[kPartWordsTopk];
        fail |= poll_span<kPartWordsTopk>(A, A.tpart + (int64_t)g * kPartWordsTopk, nwords, e, raw);
        uint64_t pk[KT];
#pragma unroll
        for (int r = 0; r < KT; ++r) {
            const int w0 = r == 0 ? 0 : kPartWords + 2 * (r - 1);
            pk[r] = r < kt ? ((uint64_t)raw[w0] << 32) | raw[w0 + 1] : 0;
        }
        const float s2 = __uint_as_float(raw[2]);
        fail |= s2 < 0.0f;
        softmax_merge(bm, bs, pk[0] != 0 ? key_val(pk[0]) : -__builtin_inff(), s2 > 0.0f ? s2 : 0.0f, A.inv_t);
        if (g == (int)threadIdx.x) {
#pragma unroll
            for (int r = 0; r < KT; ++r) list[r] = pk[r];
        } else {
            for (int r = 0; r < kt; ++r) {
                if (pk[r] <= list[KT - 1]) break;  // the partial's keys are sorted
                list[KT - 1] = pk[r];
#pragma unroll
                for (int q = KT - 1; q > 0; --q)
                    if (list[q] > list[q - 1]) {
                        const uint64_t t = list[q];
                        list[q] = list[q - 1];
                        list[q - 1] = t;
                    }
            }
        }
    }
    if (threadIdx.x == 0) f_bad = 0;
    block_topk_lists<KT, NT>(list, kt, t_heads, t_cand, t_top);
    if (fail) f_bad = 1;
    block_softmax_pair<NT>(bm, bs, A.inv_t, w_m, w_s, &f_m, &f_s);
    __syncthreads();
    const bool err = f_bad != 0 || err_word == e;
    // every workgroup has read the epoch (its partial carries it)
    if (threadIdx.x == 0) store_coherent(A.epoch, e);
    const float lshift = (A.beta > 0.0f && (int64_t)A.V > L) ? log1pf(-A.beta) : 0.0f;
    for (int r = threadIdx.x; r < kt; r += NT) {
        const uint64_t key = err ? 0 : t_top[r];
        A.out_ids[r] = key != 0 ? (int32_t)key_id(key) : -1;
        if (A.out_logprobs)
            A.out_logprobs[r] = key != 0 ? (key_val(key) - f_m) * A.inv_t - logf(f_s) + lshift : -__builtin_inff();
    }
}

template <int NB, int R, bool TOPK>
__global__ __launch_bounds__(kChainThreads) void chain_step_kernel(ChainArgs A) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const int M = A.M, k = A.k, H = A.H;
    float* sv = reinterpret_cast<float*>(smem);              // [M]
    int32_t* offs = reinterpret_cast<int32_t*>(sv + M);       // [M + 1]
    size_t o = ((size_t)M * 4 + (size_t)(M + 1) * 4 + 15) / 16 * 16;
    uint64_t* cand = reinterpret_cast<uint64_t*>(smem + o);   // [M]
    o += (size_t)M * 8;
    int32_t* sid = reinterpret_cast<int32_t*>(smem + o);      // [k] ids ascending
    int32_t* rowoff = sid + k;                                // [k + 1]
    int32_t* sbase = rowoff + k + 1;                          // [k] slab starts (layout rows)
    o = (o + (size_t)k * 4 + (size_t)(k + 1) * 4 + (size_t)k * 4 + 15) / 16 * 16;
    float* hid = reinterpret_cast<float*>(smem + o);          // [H]

    const int G = gridDim.x;
    const uint32_t e = __builtin_amdgcn_readfirstlane(load_coherent(A.epoch)) + 1u;
    const int lane = lane_id();
    const int wv = threadIdx.x / kWave;
    const int nw = G * kChainWaves;
    const int gw = blockIdx.x * kChainWaves + wv;

    // ---- loads that depend on nothing: x and the first W1 row
    constexpr bool kEarly = NB <= 8;
    Raw8<uint16_t> xv[NB], hv[NB], w2[NB];
    auto load_h = [&]() {
#pragma unroll
        for (int blk = 0; blk < NB; ++blk) {
            const int e = blk * 512 + lane * 8;
            if (e < A.d) hv[blk].template load<false>(A.h + e);
            else hv[blk].zero();
        }
    };
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) {
        const int e = blk * 512 + lane * 8;
        if (e < A.d_r) xv[blk].template load<false>(A.x + e);
        else xv[blk].zero();
    }
    const int n1 = H > 0 ? H : M;
    Raw8<uint16_t> w1[NB];
    if (gw < n1) load_bf16_row<NB>(w1, A.W1 + (int64_t)gw * A.d_r, A.d_r, lane);
    // The per-lane conditions above make the compiler wait for these loads
    // one after another.  Issuing them all at once (unconditional loads)
    // made the step 2 us slower: stage 1 then ends at more spread-out times
    // over the workgroups, and both hand-offs after it took longer, the early
    // workgroups polling words the late ones had yet to write.  The CSR
    // offsets are read in stage 3 (read here they cost 1.3 us per step).

    // ---- stage 1: layer 1 (hidden units, or the scores of a linear router)
    {
        uint64_t* out = H > 0 ? A.thidden : A.tscores;
        const int act = H > 0 ? A.act : DYNA_ACT_NONE;
        for (int j = gw; j < n1; j += nw) {
            if (j != gw) load_bf16_row<NB>(w1, A.W1 + (int64_t)j * A.d_r, A.d_r, lane);
            const float s = dot_bf16<NB>(w1, xv);
            if (lane == 0)
                store_coherent(out + j, tagged(e, __float_as_uint(apply_act(s + (A.b1 ? A.b1[j] : 0.0f), act))));
        }
    }
    // the first W2 row loads during the hand-off of the hidden layer (issued
    // with the W1 rows it only lengthens stage 1, and the hand-offs measured
    // slower that way)
    if (kEarly && H > 0 && gw < M) load_bf16_row<NB>(w2, A.W2 + (int64_t)gw * H, H, lane);

    // ---- stage 2: layer 2 over the hidden layer, polled into LDS
    bool bad = false;  // this thread gave up a wait, or the selection failed
    if (H > 0) {
        bad = poll_words<kChainThreads>(A, A.thidden, H, e, reinterpret_cast<uint32_t*>(hid));
        __syncthreads();
        for (int j = gw; j < M; j += nw) {
            if (!kEarly || j != gw) load_bf16_row<NB>(w2, A.W2 + (int64_t)j * H, H, lane);
            const float s = dot_lds<NB>(w2, hid, H, lane);
            if (lane == 0) store_coherent(A.tscores + j, tagged(e, __float_as_uint(s + (A.b2 ? A.b2[j] : 0.0f))));
        }
    }

    // ---- stage 3: top-k clusters and the shortlist, in every workgroup.
    // The CSR offsets are staged first: their round trip delays the first
    // poll of the scores, which measured faster (0.9 us per step) than
    // polling at once with the offsets in flight.  The context h for stage 4
    // loads with them (here only while the registers allow: d <= 4096).
    {
        constexpr int kOffQ = (kChainMaxM + 1 + kChainThreads - 1) / kChainThreads;
        int32_t ov[kOffQ];
#pragma unroll
        for (int u = 0; u < kOffQ; ++u) ov[u] = A.offsets[min((int)threadIdx.x + kChainThreads * u, M)];
        if constexpr (kEarly) load_h();
#pragma unroll
        for (int u = 0; u < kOffQ; ++u)
            if ((int)threadIdx.x + kChainThreads * u <= M) offs[threadIdx.x + kChainThreads * u] = ov[u];
    }
    float v[kSelQ];
    {
        uint32_t raw[kSelQ];
        bad |= poll_run<kSelQ>(A, A.tscores, M, e, raw);
#pragma unroll
        for (int q = 0; q < kSelQ; ++q) {
            v[q] = __uint_as_float(raw[q]);
            if ((int)threadIdx.x * kSelQ + q < M) sv[threadIdx.x * kSelQ + q] = v[q];
        }
    }
    const int L = chain_select<kChainThreads>(v, offs, M, k, cand, sid, rowoff, sbase, A.err, e, bad);

    // ---- stage 4: logits over the wave's contiguous range of shortlist slots
    if constexpr (!kEarly) load_h();
    GreedyState st;
    uint64_t wk = 0;  // top-k_t: this lane's place of the wave's key list
    {
        const int64_t p0 = (int64_t)gw * L / nw, p1 = (int64_t)(gw + 1) * L / nw;
        // slot q's cluster position: the number of clusters whose slabs end at
        // or before q.  With k <= 64, lane i holds cluster i's end, start
        // offset and slab start, and a ballot counts (one LDS round trip);
        // else a binary search for the first slot's cluster and a walk.
        const bool lanes = k <= kWave;
        const int my_end = lanes && lane < k ? rowoff[lane + 1] : 0x7fffffff;
        const int my_off = lanes && lane < k ? rowoff[lane] : 0;
        const int my_base = lanes && lane < k ? sbase[lane] : 0;
        int ci = 0;
        if (!lanes && p0 < p1) {
            int lo = 0, hi = k - 1;
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (rowoff[mid + 1] > p0) hi = mid;
                else lo = mid + 1;
            }
            ci = lo;
        }
        for (int64_t p = p0; p < p1; p += R) {
            const int nrow = (int)min<int64_t>(R, p1 - p);
            int64_t lrow[R];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int q = (int)p + min(r, nrow - 1);
                if (lanes) {
                    const int c = __builtin_amdgcn_readfirstlane(__popcll(__ballot(my_end <= q)));
                    lrow[r] = (int64_t)__builtin_amdgcn_readlane(my_base, c) + (q - __builtin_amdgcn_readlane(my_off, c));
                } else {
                    while (q >= rowoff[ci + 1]) ++ci;
                    lrow[r] = (int64_t)sbase[ci] + (q - rowoff[ci]);
                }
            }
            Raw8<uint16_t> w[R][NB];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                if (r < nrow) load_bf16_row<NB>(w[r], A.W + lrow[r] * A.d, A.d, lane);
                else
#pragma unroll
                    for (int blk = 0; blk < NB; ++blk) w[r][blk].zero();
            }
            int64_t my_row = lrow[0];
#pragma unroll
            for (int r = 1; r < R; ++r)
                if (lane == r) my_row = lrow[r];
            const bool own = lane < nrow;
            const int32_t vid = own ? A.perm[my_row] : 0;
            // row by row, so each row's dot starts as soon as its loads land
            float acc[R];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                acc[r] = 0.0f;
#pragma unroll
                for (int blk = 0; blk < NB; ++blk) acc[r] = dot8(w[r][blk], hv[blk], acc[r]);
            }
            float mine = 0.0f;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const float t = wave_sum(acc[r]);
                if (lane == r) mine = t;
            }
            if (own) {
                if (A.out_logits) A.out_logits[p + lane] = mine;
                st.add(mine, vid, A.inv_t);
            }
            if constexpr (TOPK) {
                // the group's keys into the wave's list, one row at a time
                // (branch-free: an empty key 0 leaves the list as it is)
                const uint64_t mykey = own ? sel_key(mine != mine ? -__builtin_inff() : mine, (uint32_t)vid) : 0;
#pragma unroll
                for (int r = 0; r < R; ++r) wk = row_list_insert(wk, readlane_u64(mykey, r));
            }
        }
    }
    if constexpr (TOPK) {
        chain_topk_finish<kChainThreads>(A, st, wk, bad, e, G, sv, sid, cand, rowoff, k, L);
        return;
    }

    // ---- stage 5: greedy partials; workgroup 0 polls and merges them.  A
    // partial whose workgroup gave up a wait (or failed the selection)
    // carries a negative sum, which fails the step.
    {
        constexpr int NW = kChainWaves;
        __shared__ uint64_t w_best[NW];
        __shared__ float w_m[NW], w_s[NW];
        __shared__ int w_bad[NW];
        // the wave's maximum logit is the value of its best key
        const uint64_t wb = wave_max_u64(st.best);
        const float wm = wb != 0 ? key_val(wb) : -__builtin_inff();
        const float wsum = wave_sum(st.m == -__builtin_inff() ? 0.0f : st.s * expf((st.m - wm) * A.inv_t));
        const bool wbad = __ballot(bad) != 0;
        if (lane == 0) {
            w_best[wv] = wb;
            w_m[wv] = wm;
            w_s[wv] = wsum;
            w_bad[wv] = wbad;
        }
        __syncthreads();
        if (wv == 0) {
            // the waves' partials side by side in lanes 0..NW-1, reduced
            // across the lanes at once (a chain of merges one after another
            // costs an exponential per wave on the critical path)
            const bool has = lane < NW;
            const uint64_t bl = has ? w_best[lane] : 0;
            const float ml = has ? w_m[lane] : -__builtin_inff();
            const float sl = has ? w_s[lane] : 0.0f;
            const bool any_bad = __ballot(has && w_bad[lane] != 0) != 0;
            const uint64_t bb = wave_max_u64(bl);
            const float bm = bb != 0 ? key_val(bb) : -__builtin_inff();
            const float bs = wave_sum(ml == -__builtin_inff() ? 0.0f : sl * expf((ml - bm) * A.inv_t));
            if (lane == 0) {
                uint64_t* pw = A.tpart + (int64_t)blockIdx.x * kPartWords;
                store_coherent(pw + 0, tagged(e, (uint32_t)(bb >> 32)));
                store_coherent(pw + 1, tagged(e, (uint32_t)bb));
                store_coherent(pw + 2, tagged(e, __float_as_uint(any_bad ? -1.0f : bs)));
            }
        }
        // the selection outputs come from the last workgroup, after its
        // partial is out (off the merging workgroup's path when G > 1)
        if (blockIdx.x == G - 1) chain_outputs<kChainThreads>(A, sv, sid, cand, rowoff, k, L);
        if (blockIdx.x != 0) return;

        // workgroup 0, wave 0: lane l polls and merges partials l, l + 64, ...
        // in order, then a fixed-order wave reduction (no barrier on this
        // path).  The error word holds the epoch of the last launch in which
        // a wait gave up; only this launch's epoch fails this launch.  (A
        // workgroup of a failed launch that starts after workgroup 0 has
        // advanced the epoch computes with the next epoch, leaves words
        // tagged with it and gives up its waits, so it marks the next launch
        // as failed, which is right: that launch may read its stale words.)
        if (wv != 0) return;
        constexpr int kLaneParts = kChainMaxGrid / kWave;
        const uint32_t err_word = lane == 0 ? load_coherent(A.err) : 0u;
        uint64_t bb = 0;
        float bm = -__builtin_inff(), bs = 0.0f;
        bool fail = false;
        for (int u0 = 0; u0 < kLaneParts; u0 += 4) {
            if (u0 * kWave >= G) break;
            uint32_t raw[4 * kPartWords];
            fail |= poll_parts<4>(A, A.tpart, G, u0, e, raw);
            // the lane's four partials: their maximum first, then the four
            // rescaled sums independently (no chain of exponentials)
            float mu[4], su[4], lm = -__builtin_inff();
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int g = lane + kWave * (u0 + u);
                const uint64_t k2 = ((uint64_t)raw[u * kPartWords] << 32) | raw[u * kPartWords + 1];
                const float s2 = __uint_as_float(raw[u * kPartWords + 2]);
                const bool in = g < G;
                fail |= in && s2 < 0.0f;
                bb = in && k2 > bb ? k2 : bb;
                mu[u] = in && k2 != 0 ? key_val(k2) : -__builtin_inff();
                su[u] = in && s2 > 0.0f ? s2 : 0.0f;
                lm = fmaxf(lm, mu[u]);
            }
            float ls = 0.0f;
#pragma unroll
            for (int u = 0; u < 4; ++u) ls += mu[u] == -__builtin_inff() ? 0.0f : su[u] * expf((mu[u] - lm) * A.inv_t);
            softmax_merge(bm, bs, lm, ls, A.inv_t);
        }
        const uint64_t gb = wave_max_u64(bb);
        const float gm = gb != 0 ? key_val(gb) : -__builtin_inff();
        const float gs = wave_sum(bm == -__builtin_inff() ? 0.0f : bs * expf((bm - gm) * A.inv_t));
        const bool gfail = __ballot(fail) != 0;
        if (lane == 0) {
            uint64_t fb = gb;
            const float fm = gm, fs = gs;
            const bool err = gfail || err_word == e;
            // every workgroup has read the epoch (its partial carries it)
            if (err) fb = 0;
            store_coherent(A.epoch, e);
            A.out_ids[0] = fb != 0 ? (int32_t)key_id(fb) : -1;
            if (A.out_logprobs) {
                const float lshift = (A.beta > 0.0f && (int64_t)A.V > L) ? log1pf(-A.beta) : 0.0f;
                A.out_logprobs[0] = fb != 0 ? (key_val(fb) - fm) * A.inv_t - logf(fs) + lshift : -__builtin_inff();
            }
        }
    }
}

template <int NB, int R, bool TOPK>
const void* chain_fn() {
    return reinterpret_cast<const void*>(chain_step_kernel<NB, R, TOPK>);
}

// The kernel instance for the widest of d_r, H and d: NB blocks of 512
// elements per row in registers, R head rows per wave in flight.
template <typename F>
auto with_chain_instance(int kmax, F f) {
    const int nb = (kmax + 511) / 512;
    if (nb <= 1) return f(std::integral_constant<int, 1>{}, std::integral_constant<int, 4>{});
    if (nb <= 2) return f(std::integral_constant<int, 2>{}, std::integral_constant<int, 4>{});
    if (nb <= 4) return f(std::integral_constant<int, 4>{}, std::integral_constant<int, 4>{});
    if (nb <= 8) return f(std::integral_constant<int, 8>{}, std::integral_constant<int, 4>{});
    if (nb <= 12) return f(std::integral_constant<int, 12>{}, std::integral_constant<int, 2>{});
    return f(std::integral_constant<int, 16>{}, std::integral_constant<int, 2>{});
}

constexpr int kChainInstances = 6;
int chain_instance_index(int kmax) {
    const int nb = (kmax + 511) / 512;
    return nb <= 1 ? 0 : nb <= 2 ? 1 : nb <= 4 ? 2 : nb <= 8 ? 3 : nb <= 12 ? 4 : 5;
}

struct ChainDevice {
    int cus = 0;
    int64_t tick_khz = 0;
    size_t lds_raised[2 * kChainInstances] = {};  // dynamic LDS limit set per instance (0: the default 64 KB)
};

std::mutex g_chain_mu;
ChainDevice g_chain_dev[kMaxDevices];

}  // namespace

size_t chain_region_bytes(int32_t H, int32_t M) {
    return 256 + (size_t)8 * (H + M) + (size_t)8 * kPartWordsTopk * kChainMaxGrid;
}

bool chain_step_eligible(const ChainRequest& q) {
    const int kmax = std::max(q.d_r, std::max(q.H, q.d));
    return q.all_bf16 && q.region != nullptr && kmax <= 8192 && q.M <= kChainMaxM && q.V < (1 << kLenBits) &&
           q.k_t >= 1 && q.k_t <= kChainTopkMax && chain_lds_bytes(q.M, q.k, q.H) <= 160 * 1024;
}

int option_wait_bound_us();  // DYNA_OPT_WAIT_BOUND_US: 0 default, -1 none, else microseconds

// The hand-offs need every workgroup resident at once.  The grid is one
// workgroup per compute unit (or the DYNA_OPT_GREEDY_GRID request), capped at
// what the occupancy calculator says can be resident together for this
// kernel instance and LDS size; 0 when no grid fits (or a query failed),
// and the caller then takes the four-launch form.  Kernels of other streams
// that hold compute units can still delay workgroups; the bounded waits
// cover that case.
int chain_step_grid(const ChainRequest& q, int64_t* tick_khz) {
    if (!chain_step_eligible(q)) return 0;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
    const int kmax = std::max(q.d_r, std::max(q.H, q.d));
    const int inst = chain_instance_index(kmax) + (q.k_t > 1 ? kChainInstances : 0);
    const size_t lds = chain_lds_bytes(q.M, q.k, q.H);
    std::lock_guard<std::mutex> g(g_chain_mu);
    ChainDevice& cd = g_chain_dev[dev];
    if (cd.cus == 0) {
        int n = 0, khz = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0 ||
            hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess || khz <= 0) {
            (void)hipGetLastError();
            return 0;
        }
        cd.cus = n;
        cd.tick_khz = khz;
    }
    const void* fn = q.k_t > 1 ? with_chain_instance(kmax, [](auto nb, auto r) {
        return chain_fn<decltype(nb)::value, decltype(r)::value, true>();
    })
                               : with_chain_instance(kmax, [](auto nb, auto r) {
                                     return chain_fn<decltype(nb)::value, decltype(r)::value, false>();
                                 });
    // dynamic LDS above the default 64 KB must be allowed per kernel first
    // (up to what the kernel's static LDS leaves of the 160 KB)
    if (lds > 64 * 1024 && lds > cd.lds_raised[inst]) {
        if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess) {
            (void)hipGetLastError();
            return 0;
        }
        cd.lds_raised[inst] = lds;
    }
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kChainThreads, lds) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    const int fit = std::min(per_cu * cd.cus, kChainMaxGrid);
    const int opt = option_greedy_grid();
    *tick_khz = cd.tick_khz;
    return std::max(0, std::min(opt > 0 ? opt : cd.cus, fit));
}

dyna_status launch_chain_step(const ChainRequest& q, hipStream_t s) {
    int64_t khz = 0;
    const int grid = chain_step_grid(q, &khz);
    if (grid <= 0) return set_error(DYNA_ERR_UNSUPPORTED, "one-launch step: no co-resident grid");
    ChainArgs a{};
    a.W1 = static_cast<const uint16_t*>(q.W1);
    a.b1 = q.b1;
    a.W2 = static_cast<const uint16_t*>(q.W2);
    a.b2 = q.b2;
    a.d_r = q.d_r;
    a.H = q.H;
    a.M = q.M;
    a.act = q.act;
    a.x = static_cast<const uint16_t*>(q.x);
    a.W = static_cast<const uint16_t*>(q.W);
    a.perm = q.perm;
    a.offsets = q.offsets;
    a.d = q.d;
    a.V = q.V;
    a.h = static_cast<const uint16_t*>(q.h);
    a.k = q.k;
    {
        char* r = static_cast<char*>(q.region);
        a.epoch = reinterpret_cast<uint32_t*>(r);
        a.err = reinterpret_cast<uint32_t*>(r + 4);
        a.thidden = reinterpret_cast<uint64_t*>(r + 256);
        a.tscores = a.thidden + q.H;
        a.tpart = a.tscores + q.M;
    }
    a.out_clusters = q.out_clusters;
    a.topk_scores = q.topk_scores;
    a.sel_sorted = q.sel_sorted;
    a.sel_rowoff = q.sel_rowoff;
    a.row_len = q.row_len;
    a.out_logits = q.out_logits;
    a.out_ids = q.out_ids;
    a.out_logprobs = q.out_logprobs;
    a.k_t = q.k_t;
    a.inv_t = q.inv_t;
    a.beta = q.beta;
    // every wait is bounded by 0.2 s of wall clock (or the bound set by
    // DYNA_OPT_WAIT_BOUND_US; -1: a wait gives up at its first read that
    // finds a word missing)
    const int bound_us = option_wait_bound_us();
    a.spin_ticks = bound_us < 0 ? 0 : (uint64_t)khz * (uint64_t)(bound_us > 0 ? bound_us : 200000) / 1000;
    const size_t lds = chain_lds_bytes(q.M, q.k, q.H);
    const int kmax = std::max(q.d_r, std::max(q.H, q.d));
    with_chain_instance(kmax, [&](auto nb, auto r) {
        if (q.k_t > 1)
            launch_timed_kernel(chain_step_kernel<decltype(nb)::value, decltype(r)::value, true>, dim3(grid),
                                dim3(kChainThreads), (uint32_t)lds, s, a);
        else
            launch_timed_kernel(chain_step_kernel<decltype(nb)::value, decltype(r)::value, false>, dim3(grid),
                                dim3(kChainThreads), (uint32_t)lds, s, a);
        return 0;
    });
    return check_launch("chain_step_kernel");
}

}  // namespace dyna
