// Gathered head for several contexts on the matrix cores, with the slab rows
// staged through LDS (Sec. 4.3: the shortlist logits of a batch are one
// gathered GEMM over the selected cluster slabs; Algorithm 1, FUSED_INDEX_GEMM).
//
// Work unit: one plan chunk (up to 16 rows of one selected cluster: one MFMA
// tile) against up to NC of the contexts that selected that cluster.  All
// chunks cost the same, and waves take them in a fixed stride, so every wave
// gets the same number of units (to one).  The tile rows
// are the A operand of v_mfma_f32_16x16x32_bf16, the contexts its B columns.
//
// Why LDS: the MFMA operand layout puts 16 different rows in one register, so
// loading A straight from HBM reads 64 bytes of each of 16 rows per wave
// instruction, a pattern HBM serves far below its streaming rate.  Here each
// wave instruction is a direct-to-LDS load (global_load_lds_dwordx4) of whole
// 256- or 512-byte row pieces, and the MFMA operands are read back from LDS.
// Each wave keeps a private ring of S stages (a stage = KB columns of the 16
// tile rows), so S - 1 stages of slab loads are always in flight; the context
// columns come straight from L2 into registers.  The wave waits on its own
// load counter only, never on a barrier (except that, for short shortlists,
// the waves of a workgroup can split one chunk's k dimension and add their
// partial tiles through LDS behind a barrier).
//
// Every other memory read inside the loop (chunk descriptors, context lists,
// the vocabulary ids of the tile rows) goes through the scalar unit, so the
// vector-memory counter only ever holds the staged loads and the output
// stores, and waiting on it never drains the ring.
//
// LDS layout of a stage: [16 rows][KB/8 pieces of 16 B].  Piece p of row r
// is stored at position p ^ r (the writer picks which global piece each lane
// fetches), so the 16 lanes that read one piece index from 16 rows hit 16
// different bank groups.
#include <atomic>

#include "dyna_device.h"

namespace dyna {
namespace {

template <typename T>
using sptr = const __attribute__((address_space(4))) T*;  // read through the scalar unit
typedef __attribute__((address_space(3))) void* lds_ptr;
typedef __attribute__((address_space(1))) void* glb_ptr;

// Cache policy of the direct-to-LDS loads of slab rows: non-temporal.  Each
// slab row is read once per step, so streaming it past the caches' normal
// allocation leaves L2 and the last-level cache to what is reused (the
// contexts, the plan); it raised the gathered head from 0.64 to 0.70 of the
// HBM peak on the tree-batch workload.  Context loads keep the default.
constexpr int kSlabPolicy = 2;

// Wait until at most N vector-memory instructions of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmem() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xF00);
}

// A work unit of one wave: plan chunk `it` and context group g (list entries
// g * NC ..).
struct Unit {
    int64_t it;
    int g;
    int kb;        // k block of the next stage of this unit
    int r0;        // first layout row of the tile
    int nrows;     // valid tile rows (1..16)
    int list_off;  // first context-list entry of the chunk
    int lcnt;      // contexts that selected the chunk's cluster
    bool valid;
};

static_assert(kChunkRows == kMfmaRows, "a plan chunk is one MFMA tile");

// Move u to the first chunk at or after u.it (stride `stride`) with rows and
// contexts; its first stage is k block kb0.
__device__ __forceinline__ void find_tile(Unit& u, const Plan& plan, int64_t n_items, int64_t stride, int kb0) {
    sptr<int32_t> ch = (sptr<int32_t>)plan.chunks;
    while (u.it < n_items) {
        const int64_t c = u.it;
        const int r0 = ch[4 * c + 0], nr = ch[4 * c + 1], lo = ch[4 * c + 2], lc = ch[4 * c + 3];
        if (nr > 0 && lc > 0) {
            u.r0 = r0;
            u.nrows = min(kMfmaRows, nr);
            u.list_off = lo;
            u.lcnt = lc;
            u.g = 0;
            u.kb = kb0;
            u.valid = true;
            return;
        }
        u.it += stride;
    }
    u.valid = false;
}

// Next stage of a unit: next k block of [kb0, kb1), else next context group,
// else next tile.
template <int NC>
__device__ __forceinline__ bool advance(Unit& u, int kb0, int kb1, const Plan& plan, int64_t n_items,
                                        int64_t stride) {
    if (++u.kb < kb1) return false;
    u.kb = kb0;
    if (++u.g * NC < u.lcnt) return true;  // same tile, next group
    u.it += stride;
    find_tile(u, plan, n_items, stride, kb0);
    return true;
}

// Lane j of v becomes x (x and j uniform).  x passes through readfirstlane
// so that the chain of selects cannot be folded back into a per-lane load.
__device__ __forceinline__ int set_lane(int v, int x, int j) {
    const int xs = __builtin_amdgcn_readfirstlane(x);
    return lane_id() == j ? xs : v;
}

__device__ __forceinline__ int from_lane(int v, int src_lane) {
    return __builtin_amdgcn_ds_bpermute(src_lane << 2, v);
}

// Context ids and slot bases of the unit's group, read through the scalar
// unit and spread over lanes: lane j of (vb, vs) holds entry j of the group
// (entries past the group repeat its first entry).  Lanes fetch the entry
// they need with ds_bpermute, which leaves the vector-memory counter alone.
template <int NC>
__device__ __forceinline__ int group_entries(const Unit& u, const Plan& plan, int& vb, int& vs) {
    sptr<int32_t> L = (sptr<int32_t>)plan.list + 2 * ((int64_t)u.list_off + (int64_t)u.g * NC);
    const int n = min(NC, u.lcnt - u.g * NC);
    const int b0 = L[0], s0 = L[1];
    vb = b0;
    vs = s0;
#pragma unroll
    for (int j = 1; j < NC; ++j) {
        if (j < n) {
            vb = set_lane(vb, L[2 * j], j);
            vs = set_lane(vs, L[2 * j + 1], j);
        }
    }
    return n;
}

// Gathered-head kernel: only the slab rows (A) go through the LDS ring; the
// context columns (B) are loaded straight into registers.  The contexts of a
// step stay in L2, and keeping them out of LDS leaves the whole ring to the
// slab rows, so each wave keeps more HBM bytes in flight.  Every stage
// issues exactly NA direct-to-LDS loads and STEPS register loads (lanes
// whose column has no context read context 0 and are zeroed when used), so
// the wave can wait for a stage with one counter value; the loop is unrolled
// by the ring depth so that a stage's B registers have fixed names.
//
// KS = NW splits the k dimension instead: all waves of a workgroup take the
// same chunk, wave w its w-th share of the k blocks, and the partial tiles
// are added through LDS in wave order at the end of each context group.  For
// a short shortlist (a few hundred chunks) that puts NW times more waves on
// the slab bytes.
template <int NW, int S, int KB, int KS = 1>
__global__ __launch_bounds__(NW * kWave) void gather_ring_kernel(RowdotArgs a) {
    constexpr int NC = 16;
    constexpr int ROWB = KB * 2;
    constexpr int PIECES = ROWB / 16;
    constexpr int RPI = kWave / PIECES;
    constexpr int NA = kMfmaRows / RPI;
    constexpr int STAGE = kMfmaRows * ROWB;
    constexpr int STEPS = KB / 32;
    constexpr int PER_STAGE = NA + STEPS;  // vector-memory instructions per stage
    static_assert(PIECES <= kWave && kWave % PIECES == 0 && kMfmaRows % RPI == 0, "stage shape");
    static_assert((S - 1) * PER_STAGE <= 63, "ring depth beyond the load counter");
    static_assert(KS == 1 || KS == NW, "k split: every wave of the workgroup on one chunk");

    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int lane = lane_id();
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    char* ring = smem + wv * (S * STAGE);
    const int K = a.K;
    const int nkb = (K + KB - 1) / KB;
    const uint16_t* __restrict__ W = static_cast<const uint16_t*>(a.W);
    const uint16_t* __restrict__ v = static_cast<const uint16_t*>(a.v);
    const int64_t n_items = (int64_t)((sptr<int32_t>)a.plan.hdr)[0];
    const int64_t stride = (int64_t)gridDim.x * (NW / KS);
    // this wave's k blocks (all of them without a split; the host makes sure
    // that every wave of a split gets at least one)
    const int kb0 = KS == 1 ? 0 : wv * nkb / KS;
    const int kb1 = KS == 1 ? nkb : (wv + 1) * nkb / KS;

    const int lsub = lane / PIECES, lpc = lane % PIECES;
    const int col = lane & 15, kq = lane >> 4;

    Unit iu;
    iu.it = (int64_t)blockIdx.x * (NW / KS) + (KS == 1 ? wv : 0);
    find_tile(iu, a.plan, n_items, stride, kb0);
    if (!iu.valid) return;
    Unit cu = iu;

    // issue side: this lane's context row; lanes whose column has no context
    // load nothing (their output column is never stored, so whatever their
    // registers hold is harmless), which keeps L2 traffic to the used columns
    const uint16_t* bsrc = v;
    bool bcol = false;
    auto issue_group = [&]() {
        int vb, vs;
        const int n = group_entries<NC>(iu, a.plan, vb, vs);
        const int b = from_lane(vb, col);
        bcol = col < n;
        bsrc = v + (int64_t)(bcol ? b : 0) * K + kq * 8;
    };
    // issue side: this lane's source of each A instruction of a stage, at k 0
    const uint16_t* arow[NA];
    auto set_rows = [&]() {
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            const int row = RPI * i + lsub;
            const int piece = lpc ^ (row % PIECES);
            arow[i] = W + (int64_t)(iu.r0 + min(row, iu.nrows - 1)) * K + piece * 8;
        }
    };
    // consume side
    int ncols = 0;
    int64_t obase = 0;
    int32_t vid[4] = {0, 0, 0, 0};
    auto consume_group = [&]() {
        int vb, vs;
        ncols = group_entries<NC>(cu, a.plan, vb, vs);
        obase = (int64_t)from_lane(vb, col) * a.ld + from_lane(vs, col) + cu.r0;
        if (a.vid_out != nullptr && cu.g == 0) {
            sptr<int32_t> P = (sptr<int32_t>)a.perm + cu.r0;
            int vp = P[0];
            if (cu.nrows == kMfmaRows) {
#pragma unroll
                for (int j = 1; j < kMfmaRows; ++j) vp = set_lane(vp, P[j], j);
            } else {
#pragma unroll
                for (int j = 1; j < kMfmaRows; ++j)
                    if (j < cu.nrows) vp = set_lane(vp, P[j], j);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) vid[r] = from_lane(vp, 4 * kq + r);
        }
    };

    u32x4 bq[S][STEPS];
    auto issue = [&](int slot, u32x4 (&bs)[STEPS]) {
        char* dst = ring + slot * STAGE;
        const int k0 = iu.kb * KB;
        if (k0 + KB <= K) {
#pragma unroll
            for (int i = 0; i < NA; ++i)
                __builtin_amdgcn_global_load_lds((glb_ptr)(arow[i] + k0), (lds_ptr)(dst + i * (RPI * ROWB)), 16, 0,
                                                 kSlabPolicy);
            if (bcol) {
#pragma unroll
                for (int st = 0; st < STEPS; ++st)
                    bs[st] = *reinterpret_cast<const u32x4*>(bsrc + k0 + st * 32);
            }
        } else {
            // k tail: pieces past K read an in-bounds piece; both operands of
            // those pieces are zeroed when the stage is consumed
#pragma unroll
            for (int i = 0; i < NA; ++i) {
                const int row = RPI * i + lsub;
                const int piece = lpc ^ (row % PIECES);
                const int off = k0 + piece * 8 < K ? k0 : -piece * 8;
                __builtin_amdgcn_global_load_lds((glb_ptr)(arow[i] + off), (lds_ptr)(dst + i * (RPI * ROWB)), 16, 0,
                                                 kSlabPolicy);
            }
            if (bcol) {
#pragma unroll
                for (int st = 0; st < STEPS; ++st) {
                    const bool in = k0 + st * 32 + kq * 8 < K;
                    bs[st] = *reinterpret_cast<const u32x4*>(bsrc + (in ? k0 + st * 32 : -kq * 8));
                }
            }
        }
    };

    // next stage of the issue side: the context group (and, on a new chunk,
    // the rows) follow the cursor
    auto advance_issue = [&]() {
        if (advance<NC>(iu, kb0, kb1, a.plan, n_items, stride) && iu.valid) {
            issue_group();
            if (iu.g == 0) set_rows();
        }
    };

    issue_group();
    set_rows();
    consume_group();
#pragma unroll
    for (int st = 0; st < S - 1; ++st) {
        if (iu.valid) {
            issue(st, bq[st]);
            advance_issue();
        }
    }

    // two accumulators take alternate k steps, so consecutive MFMAs do not
    // wait on each other
    f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    bool done = false;
    while (!done) {
#pragma unroll
        for (int u = 0; u < S; ++u) {
            if (iu.valid) {
                issue((u + S - 1) % S, bq[(u + S - 1) % S]);
                advance_issue();
                // the stage's loads are done once at most the S - 1 later
                // stages are outstanding
                wait_vmem<(S - 1) * PER_STAGE>();
            } else {
                wait_vmem<0>();
            }
            const char* st = ring + u * STAGE;
            const int k0 = cu.kb * KB;
            const bool tail = k0 + KB > K;
#pragma unroll
            for (int s2 = 0; s2 < STEPS; ++s2) {
                const int p = s2 * 4 + kq;
                u32x4 av = *reinterpret_cast<const u32x4*>(st + col * ROWB + (p ^ (col % PIECES)) * 16);
                u32x4 bv = bq[u][s2];
                if (tail && k0 + p * 8 >= K) {
                    av = u32x4{0u, 0u, 0u, 0u};
                    bv = u32x4{0u, 0u, 0u, 0u};
                }
                if (s2 & 1)
                    acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, av),
                                                                   __builtin_bit_cast(bf16x8, bv), acc1, 0, 0, 0);
                else
                    acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, av),
                                                                   __builtin_bit_cast(bf16x8, bv), acc0, 0, 0, 0);
            }
            if (cu.kb == kb1 - 1) {
                f32x4 tile;
#pragma unroll
                for (int r = 0; r < 4; ++r) tile[r] = acc0[r] + acc1[r];
                bool store = true;
                if constexpr (KS > 1) {
                    // the waves' shares of the tile, added in wave order by wave 0
                    __shared__ f32x4 part[KS][kWave];
                    part[wv][lane] = tile;
                    __syncthreads();
                    store = wv == 0;
                    if (store) {
#pragma unroll
                        for (int q = 1; q < KS; ++q) {
                            const f32x4 o = part[q][lane];
#pragma unroll
                            for (int r = 0; r < 4; ++r) tile[r] += o[r];
                        }
                    }
                    __syncthreads();
                }
                if (store && col < ncols) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int row = 4 * kq + r;
                        if (row < cu.nrows) {
                            a.out[obase + row] = tile[r];
                            if (a.vid_out != nullptr) a.vid_out[obase + row] = vid[r];
                        }
                    }
                }
                acc0 = f32x4{0.f, 0.f, 0.f, 0.f};
                acc1 = f32x4{0.f, 0.f, 0.f, 0.f};
            }
            if (advance<NC>(cu, kb0, kb1, a.plan, n_items, stride)) {
                if (!cu.valid) {
                    done = true;
                    break;
                }
                consume_group();
            }
        }
    }
}

template <int NW, int S, int KB, int KS = 1>
dyna_status launch_ring_cfg(const RowdotArgs& a, hipStream_t stream) {
    constexpr int LDS = NW * S * kMfmaRows * KB * 2;
    // a split needs at least one k block per wave
    if (KS > 1 && (a.K + KB - 1) / KB < KS) return launch_ring_cfg<NW, S, KB, 1>(a, stream);
    static_assert(LDS <= 160 * 1024, "LDS per block");
    static std::atomic<uint64_t> allowed{0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return set_error(DYNA_ERR_HIP, "gather: device");
    if (!(allowed.load() & (1ull << dev))) {
        if (hipFuncSetAttribute((const void*)gather_ring_kernel<NW, S, KB, KS>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, LDS) != hipSuccess)
            return set_error(DYNA_ERR_HIP, "gather: LDS attribute");
        allowed.fetch_or(1ull << dev);
    }
    const int per_cu = (160 * 1024) / LDS;
    const int64_t items = (int64_t)a.max_chunks_bound;
    constexpr int kItemsPerBlock = NW / KS;
    const int64_t blocks =
        std::max<int64_t>(1, std::min<int64_t>((items + kItemsPerBlock - 1) / kItemsPerBlock, 256 * per_cu));
    launch_timed_kernel(gather_ring_kernel<NW, S, KB, KS>, dim3((unsigned)blocks), dim3(NW * kWave), LDS, stream, a);
    return check_launch("gather_ring_kernel");
}

// ------------------------------------------------------------------ union head
// When the rows of a step share one shortlist (the union of their clusters,
// Sec. 4.2), the gathered head is a dense product: every union row against
// every context.  A workgroup takes NW * T consecutive plan chunks (each wave
// T chunks of 16 rows, one MFMA row tile each) against NCOL = 16 * NT
// contexts.  A stage holds KB columns of every wave's rows and of the NCOL
// contexts; the contexts are loaded once per workgroup and shared by its
// waves.  All loads are direct-to-LDS.  A stage is consumed after the wave's
// own counter wait and one workgroup barrier; that barrier also frees the
// stage read in the previous iteration, which the next load then fills.
// Workgroups are persistent (tile blockIdx.x, + gridDim.x, ...), so the ring
// runs on across tiles without refilling.  The plan lists one entry per union
// cluster (its slot base); every chunk stands for all B contexts.
template <int T>
struct UnionCursor {
    int64_t tile;
    int g;          // context group (contexts g * NCOL ..)
    int kb;         // k block
    int r0[T];      // first layout row of each of this wave's chunks
    int nrows[T];   // their valid rows (0: no chunk)
    int sb[T];      // slot base of each chunk's cluster
};

template <int NW, int T>
__device__ __forceinline__ void union_set_tile(UnionCursor<T>& u, int64_t tile, int wv, const Plan& plan,
                                               int64_t n_chunks) {
    u.tile = tile;
    u.g = 0;
    u.kb = 0;
    sptr<int32_t> ch = (sptr<int32_t>)plan.chunks;
#pragma unroll
    for (int t = 0; t < T; ++t) {
        const int64_t c = (tile * NW + wv) * T + t;
        u.r0[t] = 0;
        u.nrows[t] = 0;
        u.sb[t] = 0;
        if (c < n_chunks) {
            const int r0 = ch[4 * c + 0], nr = ch[4 * c + 1], lo = ch[4 * c + 2], lc = ch[4 * c + 3];
            if (nr > 0 && lc > 0) {
                u.r0[t] = r0;
                u.nrows[t] = min(kMfmaRows, nr);
                u.sb[t] = ((sptr<int32_t>)plan.list)[2 * (int64_t)lo + 1];
            }
        }
    }
}

template <int NW, int T>
__device__ __forceinline__ void union_advance(UnionCursor<T>& u, int nkb, int ng, int wv, const Plan& plan,
                                              int64_t n_chunks) {
    if (++u.kb < nkb) return;
    u.kb = 0;
    if (++u.g < ng) return;
    union_set_tile<NW, T>(u, u.tile + gridDim.x, wv, plan, n_chunks);
}

// LDS reads of the previous stage are complete and every wave has arrived.
__device__ __forceinline__ void stage_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0) only
    __asm__ __volatile__("s_barrier" ::: "memory");
}

constexpr int kUnionLds = 160 * 1024;

// SREQ: ring depth, or 0 for the deepest ring (at most 8) that fits in LDS
template <int NW, int T, int KB, int NT, int SREQ>
struct UnionShape {
    static constexpr int ROWB = KB * 2;
    static constexpr int STAGE = NW * T * kMfmaRows * ROWB + 16 * NT * ROWB;
    static constexpr int S = SREQ > 0 ? SREQ : (kUnionLds / STAGE < 8 ? kUnionLds / STAGE : 8);
    static constexpr int RPI = kWave / (ROWB / 16);  // rows per direct-to-LDS instruction
    static constexpr int NBI = 16 * NT / RPI;         // context instructions per stage
    // two stages only when asked for (double buffering: the barrier that
    // starts a stage frees the other one)
    static constexpr bool ok = (S >= 3 || (SREQ == 2 && S == 2)) && S * STAGE <= kUnionLds && NBI >= NW &&
                               NBI % NW == 0;
};

// Max of a 64-bit key over the 16 lanes of each DPP row (lanes 16r .. 16r + 15):
// a prefix max by row shifts, so lane 15 of the row ends with it.
__device__ __forceinline__ uint64_t row16_max_u64(uint64_t x) {
    auto step = [&](auto ctrl_tag) {
        constexpr int CTRL = decltype(ctrl_tag)::value;
        const uint32_t lo = dpp<CTRL, 0xf>(0u, (uint32_t)x);
        const uint32_t hi = dpp<CTRL, 0xf>(0u, (uint32_t)(x >> 32));
        const uint64_t y = ((uint64_t)hi << 32) | lo;
        x = y > x ? y : x;
    };
    step(std::integral_constant<int, kRowShr1>{});
    step(std::integral_constant<int, kRowShr2>{});
    step(std::integral_constant<int, kRowShr4>{});
    step(std::integral_constant<int, kRowShr8>{});
    return x;
}

// EPI 0: store every (context, slot) product to out (and the slots' ids to
// vid_out).  EPI 1: the contexts are centroids; keep, per row, the best
// (product, lower context id) over all contexts and write its context id to
// vid_out[slot] and its product to out[slot] (if out is set).
template <int NW, int T, int KB, int NT, int SREQ, int EPI>
__global__ __launch_bounds__(NW * kWave) void union_gemm_kernel(RowdotArgs a) {
    using Sh = UnionShape<NW, T, KB, NT, SREQ>;
    constexpr int S = Sh::S;
    constexpr int ROWB = KB * 2;
    constexpr int PIECES = ROWB / 16;
    constexpr int RPI = kWave / PIECES;
    constexpr int NA = T * kMfmaRows / RPI;  // A instructions per wave and stage
    constexpr int NCOL = 16 * NT;
    constexpr int NBW = NCOL / RPI / NW;     // B instructions per wave and stage
    constexpr int NI = NA + NBW;
    constexpr int A_TILE = kMfmaRows * ROWB;
    constexpr int A_WAVE = T * A_TILE;
    constexpr int A_BYTES = NW * A_WAVE;
    constexpr int STAGE = Sh::STAGE;
    constexpr int STEPS = KB / 32;
    static_assert(PIECES == 16 || PIECES == 8, "stage shape");
    static_assert(NBW >= 1 && NBW * NW * RPI == NCOL, "context loads split evenly over the waves");
    static_assert(Sh::ok && (S - 2) * NI < 64, "ring depth");

    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int lane = lane_id();
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int K = a.K, B = a.B;
    const int nkb = (K + KB - 1) / KB;
    const int ng = (B + NCOL - 1) / NCOL;
    const int64_t n_chunks = (int64_t)((sptr<int32_t>)a.plan.hdr)[0];
    const int64_t n_tiles = (n_chunks + NW * T - 1) / (NW * T);
    if ((int64_t)blockIdx.x >= n_tiles) return;  // whole workgroup
    const int64_t Q = ((n_tiles - blockIdx.x + gridDim.x - 1) / gridDim.x) * ng * nkb;
    const uint16_t* __restrict__ W = static_cast<const uint16_t*>(a.W);
    const uint16_t* __restrict__ v = static_cast<const uint16_t*>(a.v);

    const int lsub = lane / PIECES, lpc = lane % PIECES;
    const int col = lane & 15, kq = lane >> 4;

    UnionCursor<T> iu, cu;
    union_set_tile<NW, T>(iu, blockIdx.x, wv, a.plan, n_chunks);
    cu = iu;

    auto issue = [&](int slot) {
        char* dst = smem + slot * STAGE;
        const int kb = iu.kb;
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            const int t = (RPI * i) / kMfmaRows;
            const int row = RPI * i + lsub - t * kMfmaRows;
            const int piece = lpc ^ (row % PIECES);
            int e = kb * KB + piece * 8;
            e = e < K ? e : 0;  // k tail: any in-bounds piece; zeroed when read
            const int64_t grow = iu.nrows[t] > 0 ? iu.r0[t] + min(row, iu.nrows[t] - 1) : 0;
            __builtin_amdgcn_global_load_lds((glb_ptr)(W + grow * K + e),
                                             (lds_ptr)(dst + wv * A_WAVE + i * (RPI * ROWB)), 16, 0, kSlabPolicy);
        }
#pragma unroll
        for (int i = 0; i < NBW; ++i) {
            const int ii = wv * NBW + i;
            const int c = RPI * ii + lsub;
            const int piece = lpc ^ (c % PIECES);
            int e = kb * KB + piece * 8;
            e = e < K ? e : 0;
            const int b = min(iu.g * NCOL + c, B - 1);  // past B: any context; never stored
            __builtin_amdgcn_global_load_lds((glb_ptr)(v + (int64_t)b * K + e),
                                             (lds_ptr)(dst + A_BYTES + ii * (RPI * ROWB)), 16, 0, 0);
        }
    };

    // vocabulary ids of the consumed chunks' rows (lane j < 16 of vp holds row j's)
    int32_t vid[T][4];
    uint64_t run[T][4];  // EPI 1: best key per row so far (lane 15 of each DPP row)
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) run[t][r] = 0;
    auto load_vids = [&]() {
        if (EPI != 0 || a.vid_out == nullptr) return;
#pragma unroll
        for (int t = 0; t < T; ++t) {
            if (cu.nrows[t] == 0) continue;
            sptr<int32_t> P = (sptr<int32_t>)a.perm + cu.r0[t];
            int vp = P[0];
#pragma unroll
            for (int j = 1; j < kMfmaRows; ++j)
                if (j < cu.nrows[t]) vp = set_lane(vp, P[j], j);
#pragma unroll
            for (int r = 0; r < 4; ++r) vid[t][r] = from_lane(vp, 4 * kq + r);
        }
    };

    int64_t issued = 0;
#pragma unroll
    for (int s = 0; s < S - 1; ++s) {
        if (issued < Q) {
            issue((int)(issued % S));
            ++issued;
            union_advance<NW, T>(iu, nkb, ng, wv, a.plan, n_chunks);
        }
    }
    load_vids();

    f32x4 acc[T][NT];
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[t][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int64_t q = 0; q < Q; ++q) {
        // this wave's loads of stage q are done once at most the later stages remain
        if (issued - q - 1 == S - 2) wait_vmem<(S - 2) * NI>();
        else wait_vmem<0>();
        stage_barrier();
        if (issued < Q) {
            issue((int)(issued % S));
            ++issued;
            union_advance<NW, T>(iu, nkb, ng, wv, a.plan, n_chunks);
        }
        const char* st = smem + (int)(q % S) * STAGE;
        const char* sa = st + wv * A_WAVE;
        const char* sbm = st + A_BYTES;
        const int k0 = cu.kb * KB;
#pragma unroll
        for (int s = 0; s < STEPS; ++s) {
            const int p = s * 4 + kq;
            const bool tail = k0 + p * 8 >= K;
            u32x4 av[T];
#pragma unroll
            for (int t = 0; t < T; ++t) {
                av[t] = *reinterpret_cast<const u32x4*>(sa + t * A_TILE + col * ROWB + (p ^ (col % PIECES)) * 16);
                if (tail) av[t] = u32x4{0u, 0u, 0u, 0u};
            }
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                const int c = 16 * j + col;
                u32x4 bv = *reinterpret_cast<const u32x4*>(sbm + c * ROWB + (p ^ (c % PIECES)) * 16);
                if (tail) bv = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
                for (int t = 0; t < T; ++t)
                    acc[t][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8, av[t]), __builtin_bit_cast(bf16x8, bv), acc[t][j], 0, 0, 0);
            }
        }
        if (EPI == 1 && cu.kb == nkb - 1) {
            // best (product, lower centroid id) of each row over this group,
            // folded into the row's running best; written after the last group
#pragma unroll
            for (int t = 0; t < T; ++t) {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    uint64_t kb_best = 0;
#pragma unroll
                    for (int j = 0; j < NT; ++j) {
                        const int b = cu.g * NCOL + 16 * j + col;
                        const float x = acc[t][j][r];
                        const uint64_t key = sel_key(x != x ? -__builtin_inff() : x, (uint32_t)b);
                        if (b < B && key > kb_best) kb_best = key;
                    }
                    kb_best = row16_max_u64(kb_best);
                    run[t][r] = kb_best > run[t][r] ? kb_best : run[t][r];
                }
                if (cu.g == ng - 1) {
                    if (col == 15 && cu.nrows[t] > 0) {
                        const int64_t base = (int64_t)cu.sb[t] + cu.r0[t];
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const int row = 4 * kq + r;
                            if (row < cu.nrows[t]) {
                                a.vid_out[base + row] = run[t][r] != 0 ? (int32_t)key_id(run[t][r]) : 0;
                                if (a.out != nullptr) a.out[base + row] = key_val(run[t][r]);
                            }
                        }
                    }
#pragma unroll
                    for (int r = 0; r < 4; ++r) run[t][r] = 0;
                }
            }
        }
        if (EPI == 0 && cu.kb == nkb - 1) {
            // D rows 4 * kq + r, context column 16 * j + col
#pragma unroll
            for (int t = 0; t < T; ++t) {
                if (cu.nrows[t] == 0) continue;
                const int64_t base = (int64_t)cu.sb[t] + cu.r0[t];
#pragma unroll
                for (int j = 0; j < NT; ++j) {
                    const int b = cu.g * NCOL + 16 * j + col;
                    if (b < B) {
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const int row = 4 * kq + r;
                            if (row < cu.nrows[t]) a.out[(int64_t)b * a.ld + base + row] = acc[t][j][r];
                        }
                    }
                }
                // one shared copy of the slots' vocabulary ids
                if (a.vid_out != nullptr && cu.g == 0 && col == 0) {
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (4 * kq + r < cu.nrows[t]) a.vid_out[base + 4 * kq + r] = vid[t][r];
                }
            }
        }
        if (cu.kb == nkb - 1) {
#pragma unroll
            for (int t = 0; t < T; ++t)
#pragma unroll
                for (int j = 0; j < NT; ++j) acc[t][j] = f32x4{0.f, 0.f, 0.f, 0.f};
            union_advance<NW, T>(cu, nkb, ng, wv, a.plan, n_chunks);
            if (cu.g == 0) load_vids();
        } else {
            ++cu.kb;
        }
    }
}

template <int NW, int T, int KB, int NT, int SREQ = 0, int EPI = 0>
dyna_status launch_union_cfg(const RowdotArgs& a, hipStream_t stream) {
    using Sh = UnionShape<NW, T, KB, NT, SREQ>;
    if constexpr (!Sh::ok) {
        return set_error(DYNA_ERR_UNSUPPORTED, "union: shape does not fit in LDS");
    } else {
        constexpr int LDS = Sh::S * Sh::STAGE;
        static_assert(LDS <= kUnionLds, "LDS per block");
        static std::atomic<uint64_t> allowed{0};
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return set_error(DYNA_ERR_HIP, "union: device");
        if (!(allowed.load() & (1ull << dev))) {
            if (hipFuncSetAttribute((const void*)union_gemm_kernel<NW, T, KB, NT, SREQ, EPI>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, LDS) != hipSuccess)
                return set_error(DYNA_ERR_HIP, "union: LDS attribute");
            allowed.fetch_or(1ull << dev);
        }
        const int per_cu = std::max(1, kUnionLds / LDS);
        const int64_t tiles = ((int64_t)a.max_chunks_bound + NW * T - 1) / (NW * T);
        const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>(tiles, 256 * per_cu));
        launch_timed_kernel(union_gemm_kernel<NW, T, KB, NT, SREQ, EPI>, dim3((unsigned)blocks), dim3(NW * kWave), LDS,
                            stream, a);
        return check_launch("union_gemm_kernel");
    }
}

// Fixed shapes (waves, chunks per wave, k columns per stage, ring depth) of
// the union kernel; 0 picks by context count.
template <int NT>
dyna_status launch_union_nt(const RowdotArgs& a, int cfg, hipStream_t stream) {
    switch (cfg) {
        case 1: return launch_union_cfg<4, 1, 128, NT>(a, stream);
        case 2: return launch_union_cfg<8, 1, 128, NT>(a, stream);
        case 3: return launch_union_cfg<4, 2, 128, NT>(a, stream);
        case 4: return launch_union_cfg<4, 1, 64, NT>(a, stream);
        case 5: return launch_union_cfg<8, 1, 64, NT>(a, stream);
        case 6: return launch_union_cfg<4, 1, 64, NT, 4>(a, stream);
        case 7: return launch_union_cfg<8, 1, 64, NT, 3>(a, stream);
        case 8: return launch_union_cfg<4, 1, 128, NT, 3>(a, stream);
        case 9: return launch_union_cfg<8, 2, 64, NT>(a, stream);
        case 10: return launch_union_cfg<2, 1, 128, NT, 3>(a, stream);
        case 11: return launch_union_cfg<8, 1, 128, NT, 4>(a, stream);
        case 12: return launch_union_cfg<4, 1, 64, NT, 3>(a, stream);
        case 13: return launch_union_cfg<4, 2, 64, NT, 3>(a, stream);
        case 14: return launch_union_cfg<2, 2, 64, NT, 3>(a, stream);
        case 15: return launch_union_cfg<2, 1, 64, NT, 3>(a, stream);
        default:  // measured best per context count (eight waves where the context loads split)
            if constexpr (NT >= 8) return launch_union_cfg<8, 2, 64, NT>(a, stream);
            else if constexpr (NT == 4) return launch_union_cfg<8, 1, 64, NT, 3>(a, stream);
            else if constexpr (NT == 2) return launch_union_cfg<4, 1, 64, NT, 3>(a, stream);
            // up to 16 contexts: two-wave workgroups of 64-column stages
            // (many small workgroups per CU).  Measured at ten rows over a
            // union of 31.6k slots: 52.2 us against 60.3 with 128-column
            // stages and 54-81 us for deeper rings or more rows per wave;
            // the 16-context dense head 186 us (128 columns: 188; four-wave
            // workgroups: 233)
            else return launch_union_cfg<2, 1, 64, NT, 3>(a, stream);
    }
}

}  // namespace

bool gather_lds_eligible(const RowdotArgs& a) {
    return a.plan.hdr != nullptr && a.wdtype == DYNA_BF16 && a.vdtype == DYNA_BF16 && a.K % 8 == 0 &&
           a.bias == nullptr && a.act == DYNA_ACT_NONE && (a.vid_out == nullptr || a.perm != nullptr);
}

constexpr int32_t kSplitChunks = 4096;

dyna_status launch_gather_lds(const RowdotArgs& a, hipStream_t stream) {
    if (!gather_lds_eligible(a)) return set_error(DYNA_ERR_UNSUPPORTED, "gather: needs bf16 plan mode");
    switch (option_gather_cfg()) {
        case 1: return launch_ring_cfg<4, 2, 512>(a, stream);
        case 2: return launch_ring_cfg<4, 4, 256>(a, stream);
        case 3: return launch_ring_cfg<4, 8, 128>(a, stream);
        case 4: return launch_ring_cfg<8, 8, 64>(a, stream);
        case 5: return launch_ring_cfg<2, 4, 256, 2>(a, stream);
        case 6: return launch_ring_cfg<4, 4, 256, 4>(a, stream);
        case 7: return launch_ring_cfg<4, 4, 128, 4>(a, stream);
        case 8: return launch_ring_cfg<4, 3, 256, 4>(a, stream);
        case 9: return launch_ring_cfg<8, 4, 128, 8>(a, stream);
        default:
            // a short shortlist (at most a few thousand chunks, as in the
            // union steps of a few rows): four waves split each chunk's k
            // dimension.  Measured at ten rows: 19.0 -> 17.2 us over a union
            // of 5.9k rows, 26.0 -> 23.4 us over 9.2k rows; the other split
            // shapes gained less or lost.
            if (a.max_chunks_bound <= kSplitChunks) return launch_ring_cfg<4, 4, 128, 4>(a, stream);
            return launch_ring_cfg<2, 4, 256>(a, stream);  // two workgroups of two waves per CU
    }
}

dyna_status launch_union_gemm(const RowdotArgs& a, hipStream_t stream) {
    if (!gather_lds_eligible(a) || a.B < 1) return set_error(DYNA_ERR_UNSUPPORTED, "union: needs bf16 plan mode");
    const int cfg = option_union_cfg();
    if (a.B <= 16) return launch_union_nt<1>(a, cfg, stream);
    if (a.B <= 32) return launch_union_nt<2>(a, cfg, stream);
    if (a.B <= 64) return launch_union_nt<4>(a, cfg, stream);
    return launch_union_nt<8>(a, cfg, stream);
}

dyna_status launch_union_argmax(const RowdotArgs& a, int cfg, hipStream_t stream) {
    if (a.plan.hdr == nullptr || a.wdtype != DYNA_BF16 || a.vdtype != DYNA_BF16 || a.K % 8 != 0 ||
        a.vid_out == nullptr || a.B < 1)
        return set_error(DYNA_ERR_UNSUPPORTED, "nearest centroid: needs bf16 rows and centroids");
    switch (cfg) {
        case 1: return launch_union_cfg<8, 1, 64, 8, 3, 1>(a, stream);
        case 2: return launch_union_cfg<4, 1, 128, 8, 3, 1>(a, stream);
        case 3: return launch_union_cfg<8, 1, 64, 16, 3, 1>(a, stream);
        case 4: return launch_union_cfg<4, 2, 64, 16, 3, 1>(a, stream);
        case 5: return launch_union_cfg<4, 4, 64, 8, 3, 1>(a, stream);
        case 6: return launch_union_cfg<8, 2, 64, 8, 0, 1>(a, stream);
        case 7: return launch_union_cfg<8, 4, 64, 8, 2, 1>(a, stream);
        // measured best: eight waves of two row tiles (256 rows) against 256
        // centroids, double-buffered (two 64 KB stages).  The rows are
        // re-read from HBM once per group of centroids, so wider groups cut
        // the HBM bytes: 128-centroid groups measured 1.15-1.34x slower.
        default: return launch_union_cfg<8, 2, 64, 16, 2, 1>(a, stream);
    }
}

}  // namespace dyna
