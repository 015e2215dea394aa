// f2gpu.hip -- MI355X (gfx950) kernels and C ABI of the GF(2) affine-map learner.
//
// Fit (Sec. 2.2): every context is an independent streaming Gaussian
// elimination over GF(2) on augmented rows [phi | y] (Eq. 5).  Rows are taken
// in stream order in blocks of 64, one row per lane of a 64-wide wavefront:
//   1. block reduce: every row of the block is reduced against the retained
//      basis.  The basis is kept fully reduced (each pivot column is set only
//      in its own row), so the row's own bits at the pivot columns select the
//      basis rows to add, in one pass;
//   2. in-block elimination in stream order: a wavefront ballot finds the
//      earliest row with a nonzero feature residual; the rows before it are
//      redundant or contradictory (zero features, nonzero output: Eq. 8) and
//      are classified together; the earliest nonzero row gives the new pivot
//      (its highest-priority feature bit), is broadcast to the later rows that
//      hold that bit and to the retained rows that hold it (back-substitution
//      keeps the basis fully reduced), and is inserted.
// A plan kernel validates the contexts and sorts them into classes by feature
// words and length, each class list in decreasing order of estimated work:
// contexts of up to 3 feature words keep the basis in registers (one lane per
// retained row), contexts of 4-8 words keep a pivot-indexed basis in LDS (one
// wavefront, or eight for long contexts, which reduce eight blocks at once),
// wider contexts run a workgroup-per-context kernel with the basis in HBM and
// the rows it needs staged in LDS.
//
// Encode (Sec. 2.3): T(phi) is the XOR of the canonical map columns over the
// set bits of phi = [x | 1]; the support test checks phi against the
// parity-check rows of the free (non-pivot) columns, which a prepare kernel
// derives from the fitted basis.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <stdlib.h>

#include <atomic>

#include "../../include/f2gpu.h"

namespace {

constexpr int kLargeRows = 64;       // rows per block, large path
constexpr int kLargeThreads = 512;
constexpr int kEncThreads = 256;

struct FitArgs {
    const uint64_t* rows;
    int64_t rows_words;
    const int64_t* row_off;
    int32_t num_ctx;
    const int32_t* n_bits;
    const int64_t* basis_off;
    const int64_t* piv_off;
    const int64_t* map_off;
    int64_t basis_words, piv_entries, map_words;
    uint64_t* basis;
    int32_t* pivots;
    uint64_t* maps;
    uint64_t* tables;
    int32_t* rank;
    uint32_t* ctx_flags;
    int32_t* n_contra;
    int64_t* first_contra;
    int32_t* plan;  // workspace: class list offsets, group barrier counters, context lists (k_fit_plan)
    int32_t coop;   // the wide kernel runs as a cooperative launch (all workgroups resident)
    int32_t max_n;  // host hint: largest width of the batch, -1 if unknown
    int32_t spin_limit;  // polls of a group barrier before it gives up (0: never wait)
};

struct EncArgs {
    int32_t num_ctx;
    const int32_t* n_bits;
    const int64_t* basis_off;
    const int64_t* piv_off;
    const uint64_t* basis;
    const int32_t* pivots;
    const int32_t* rank;
    const uint32_t* ctx_flags;
    const int64_t* map_off;
    const uint64_t* maps;
    const uint64_t* tables;  // parity-check rows, context c at basis_off[c]
    const int32_t* ctx_id;
    const uint64_t* x;
    int32_t stride;
    int32_t x16;  // x is 16-byte aligned (then even strides allow 16-byte loads of a query)
    int64_t nq;
    uint64_t* words;
    uint8_t* qflags;
};

constexpr uint32_t kBadCtx = F2_CTX_BAD_SEGMENT | F2_CTX_BAD_WIDTH | F2_CTX_BAD_OUTPUT | F2_CTX_SYNC_TIMEOUT;

__device__ __forceinline__ int feat_words(int n) { return (n + 64) >> 6; }

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int lane) {
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(v), lane);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(v >> 32), lane);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src_lane) {
    const int lo = __builtin_amdgcn_ds_bpermute(src_lane << 2, static_cast<int>(static_cast<uint32_t>(v)));
    const int hi = __builtin_amdgcn_ds_bpermute(src_lane << 2, static_cast<int>(static_cast<uint32_t>(v >> 32)));
    return (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo);
}

__device__ __forceinline__ int ffs64(uint64_t v) { return __ffsll(static_cast<unsigned long long>(v)) - 1; }
__device__ __forceinline__ int msb64(uint64_t v) { return 63 - __clzll(static_cast<long long>(v)); }

// valid bits of the last feature word
__device__ __forceinline__ uint64_t top_mask(int n, int fw) {
    const int vb = n + 1 - 64 * (fw - 1);
    return vb >= 64 ? ~0ull : ((1ull << vb) - 1);
}

// ---------------------------------------------------------------------------
// context descriptor: width, row segment and the checks of its offsets against
// the buffer sizes (an invalid context is flagged and left at rank 0)
// ---------------------------------------------------------------------------
struct CtxDesc {
    int c, n;
    uint32_t bad;
    int64_t row0, m;
    int64_t bo, po, mo;  // output offsets: basis (and parity rows), pivots, map
};

__device__ __forceinline__ CtxDesc load_desc(const FitArgs& a, int64_t c) {
    CtxDesc ds{-1, -1, 0u, 0, 0, 0, 0, 0};  // c = -1: no context
    if (c >= a.num_ctx) return ds;
    ds.c = static_cast<int>(c);
    // every load first (one memory latency), then the checks in order
    const int n = a.n_bits[c];
    const int64_t bo = a.basis_off[c], po = a.piv_off[c], mo = a.map_off[c];
    const int64_t s0 = a.row_off[c], s1 = a.row_off[c + 1];
    ds.n = n;
    ds.bo = bo;
    ds.po = po;
    ds.mo = mo;
    if (n < 0 || n > F2_MAX_N_BITS || (a.max_n >= 0 && n > a.max_n)) {  // outside the supported or declared range
        ds.bad = F2_CTX_BAD_WIDTH;
        return ds;
    }
    const int d = n + 1;
    const int W = feat_words(n) + F2_Y_WORDS;
    if (bo < 0 || bo + static_cast<int64_t>(d) * W > a.basis_words || po < 0 || po + d > a.piv_entries || mo < 0 ||
        mo + 2 * static_cast<int64_t>(d) > a.map_words) {
        ds.bad = F2_CTX_BAD_OUTPUT;
        return ds;
    }
    if (s0 < 0 || s1 < s0 || s1 > a.rows_words || (s1 - s0) % W != 0) {
        ds.bad = F2_CTX_BAD_SEGMENT;
        return ds;
    }
    ds.row0 = s0;
    ds.m = (s1 - s0) / W;
    return ds;
}

__device__ __forceinline__ CtxDesc readlane_desc(const CtxDesc& v, int t) {
    CtxDesc ds;
    ds.c = __builtin_amdgcn_readlane(v.c, t);
    ds.n = __builtin_amdgcn_readlane(v.n, t);
    ds.bad = __builtin_amdgcn_readlane(v.bad, t);
    ds.row0 = static_cast<int64_t>(readlane64(static_cast<uint64_t>(v.row0), t));
    ds.m = static_cast<int64_t>(readlane64(static_cast<uint64_t>(v.m), t));
    ds.bo = static_cast<int64_t>(readlane64(static_cast<uint64_t>(v.bo), t));
    ds.po = static_cast<int64_t>(readlane64(static_cast<uint64_t>(v.po), t));
    ds.mo = static_cast<int64_t>(readlane64(static_cast<uint64_t>(v.mo), t));
    return ds;
}

// outputs of an invalid context (one thread)
__device__ __forceinline__ void write_bad_context(const FitArgs& a, const CtxDesc& ds) {
    a.rank[ds.c] = 0;
    a.n_contra[ds.c] = 0;
    a.first_contra[ds.c] = -1;
    a.ctx_flags[ds.c] = ds.bad;
    if (ds.bad == F2_CTX_BAD_SEGMENT) {
        const int64_t mo = a.map_off[ds.c];
        for (int j = 0; j < 2 * (ds.n + 1); ++j) a.maps[mo + j] = 0;
    }
}

// ---------------------------------------------------------------------------
// fit plan.  Contexts are validated (an invalid one gets rank 0 and its flag
// here), assigned to the kernel of their class, and each class list is sorted
// by an estimate of the elimination work, largest first:
//   class 0: fw <= 3, at most kLongRows rows  -> register basis, one wavefront
//   class 1: fw 4-8, at most kLongRows rows   -> LDS basis, kPivWaves wavefronts
//   class 2: fw <= 8, more than kLongRows rows -> LDS basis, kPivWaves wavefronts
//   class 3: fw > 8                           -> large-context kernel
// A class kernel with G workgroups deals its list out in stripes of G entries,
// alternating direction from stripe to stripe, so that every workgroup gets a
// similar share of the work and the longest contexts start first.  The sort is
// a counting sort over (class, cost bucket) bins in two kernels (per-block
// histograms; a scatter that scans them) with no device-wide atomics: on a chip
// of eight dies those serialise far from the compute units.
// Workspace (int32): [0, 5) list offsets per class, [kPivNext] the work counter
// of the LDS-basis kernel, [kBarHead, kPlanHead) barrier counters of workgroup
// groups, [kPlanHead, kPlanHead + C) the lists, then C sort keys and a
// kPlanBins histogram per plan block.
// ---------------------------------------------------------------------------
constexpr int kRegMaxFW = 3;
constexpr int kPivMaxFW = 8;
constexpr int kLongRows = 256;  // contexts with more rows take the multi-wavefront kernel
enum { kClsReg = 0, kClsPiv = 1, kClsPivLong = 2, kClsLarge = 3, kNumCls = 4 };
constexpr int kPivNext = 8;                 // plan word: next list position for the LDS-basis kernel
constexpr int kBarHead = 16;                // plan words kBarHead ..: barrier counters of workgroup groups
constexpr int kMaxGroups = 128;
constexpr int kPlanHead = kBarHead + kMaxGroups;
constexpr int kBuckets = 256;
constexpr int kPlanBins = kNumCls * kBuckets;
constexpr int kPlanThreads = 1024;  // one context per thread; one bin per thread in the scan
static_assert(kPlanBins == kPlanThreads, "the scan gives one bin to each thread");

__device__ __forceinline__ int fit_class(const CtxDesc& ds) {
    const int fw = feat_words(ds.n);
    if (fw > kPivMaxFW) return kClsLarge;
    if (ds.m > kLongRows) return kClsPivLong;
    return fw <= kRegMaxFW ? kClsReg : kClsPiv;
}

// log-scale bucket (4 per octave) of rows x min(rows, d) x row words
__device__ __forceinline__ int cost_bucket(const CtxDesc& ds) {
    const uint64_t d = static_cast<uint64_t>(ds.n) + 1, W = static_cast<uint64_t>(feat_words(ds.n)) + F2_Y_WORDS;
    const uint64_t m = ds.m < (1ll << 32) ? static_cast<uint64_t>(ds.m) : (1ull << 32);
    const uint64_t cost = m * (m < d ? m : d) * W + 1;
    const int e = 63 - __clzll(static_cast<long long>(cost));
    const int frac = e >= 2 ? static_cast<int>((cost >> (e - 2)) & 3) : 0;
    const int b = 4 * e + frac;
    return b < kBuckets ? b : kBuckets - 1;
}

struct PlanView {
    int32_t* cls_off;  // [kNumCls + 1]
    int32_t* order;    // [C]
    int32_t* key;      // [C]
    int32_t* hist;     // [blocks][kPlanBins]
};

__device__ __forceinline__ PlanView plan_view(const FitArgs& a) {
    PlanView v;
    v.cls_off = a.plan;
    v.order = a.plan + kPlanHead;
    v.key = v.order + a.num_ctx;
    v.hist = v.key + a.num_ctx;
    return v;
}

// (1) per context: validate, class and bin; per block: histogram of the bins
__global__ __launch_bounds__(kPlanThreads) void k_plan_count(FitArgs a) {
    __shared__ int sBin[kPlanBins];
    const PlanView P = plan_view(a);
    const int tid = threadIdx.x;
    sBin[tid] = 0;
    __syncthreads();
    if (blockIdx.x == 0 && tid < kMaxGroups) a.plan[kBarHead + tid] = 0;
    if (blockIdx.x == 0 && tid == 0) a.plan[kPivNext] = 0;
    const int64_t c = static_cast<int64_t>(blockIdx.x) * kPlanThreads + tid;
    if (c < a.num_ctx) {
        const CtxDesc ds = load_desc(a, c);
        int k = -1;
        if (ds.bad) {
            write_bad_context(a, ds);
        } else {
            const int cls = fit_class(ds);
            k = cls * kBuckets + (kBuckets - 1 - cost_bucket(ds));
            atomicAdd(&sBin[k], 1);
            // the workgroups of a wide context OR their flags in (contradiction, wait timeout)
            if (cls == kClsLarge) a.ctx_flags[c] = 0u;
        }
        P.key[c] = k;
    }
    __syncthreads();
    P.hist[static_cast<int64_t>(blockIdx.x) * kPlanBins + tid] = sBin[tid];
}

// (2) scatter.  Thread b of every block sums bin b over all blocks (its total) and
// over the blocks before this one; a block scan of the totals gives the bin bases.
// List position = bin base + earlier blocks' count + rank within the block.
__global__ __launch_bounds__(kPlanThreads) void k_plan_scatter(FitArgs a, int blocks) {
    __shared__ int sBin[kPlanBins];
    __shared__ int sWave[kPlanThreads / 64];
    const PlanView P = plan_view(a);
    const int tid = threadIdx.x, lane = tid & 63;
    const int g0 = static_cast<int>(blockIdx.x);
    int total = 0, before = 0;
    int g = 0;
    for (; g + 8 <= blocks; g += 8) {  // eight loads in flight
        int v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = P.hist[static_cast<int64_t>(g + k) * kPlanBins + tid];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            before += g + k < g0 ? v[k] : 0;
            total += v[k];
        }
    }
    for (; g < blocks; ++g) {
        const int v = P.hist[static_cast<int64_t>(g) * kPlanBins + tid];
        before += g < g0 ? v : 0;
        total += v;
    }
    int x = total;
    for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(x, o);
        if (lane >= o) x += t;
    }
    if (lane == 63) sWave[tid >> 6] = x;
    __syncthreads();
    int base = 0;
    for (int w = 0; w < (tid >> 6); ++w) base += sWave[w];
    const int excl = base + x - total;
    if (g0 == 0) {
        if (tid % kBuckets == 0) P.cls_off[tid / kBuckets] = excl;
        if (tid == kPlanThreads - 1) P.cls_off[kNumCls] = excl + total;
    }
    sBin[tid] = excl + before;
    __syncthreads();
    const int64_t c = static_cast<int64_t>(g0) * kPlanThreads + tid;
    if (c < a.num_ctx) {
        const int k = P.key[c];
        if (k >= 0) P.order[atomicAdd(&sBin[k], 1)] = static_cast<int32_t>(c);
    }
}

// the i-th context of classes cls .. cls_last (adjacent lists) dealt to taker g
// of G (snake order), or -1; by default the takers are the workgroups
__device__ __forceinline__ int class_ctx(const FitArgs& a, int cls, int i, int cls_last = -1, int G = -1, int g = -1) {
    const int lo = a.plan[cls], cnt = a.plan[(cls_last < 0 ? cls : cls_last) + 1] - lo;
    if (G < 0) {
        G = static_cast<int>(gridDim.x);
        g = static_cast<int>(blockIdx.x);
    }
    const int64_t e = static_cast<int64_t>(i) * G + ((i & 1) ? G - 1 - g : g);
    return e < cnt ? a.plan[kPlanHead + lo + static_cast<int>(e)] : -1;
}

// ---------------------------------------------------------------------------
// parity-check rows, written by every fit kernel next to the canonical map:
// for the i-th free (non-pivot) column f in ascending order, row i (fw words,
// at the context's basis offset in the tables buffer) is h_f = e_f plus e_p for
// every pivot p whose basis row holds bit f.  Since the basis is fully reduced,
// the residual of reducing phi at column f is the parity of phi & h_f, so phi
// lies in the span exactly when every row has even overlap with it.  Word w of
// h_f is one ballot: lane b tests bit f of the basis row of pivot 64 w + b.
// The rows exist only when t = d - rank <= rank; a context with more free
// columns than basis rows is encoded by reducing phi with the basis itself.
// ---------------------------------------------------------------------------
__device__ __forceinline__ bool has_parity_rows(int d, int rank) { return d - rank <= rank; }
// orders a wavefront's own LDS accesses: used where a wavefront works alone on
// its LDS region, so that no workgroup barrier couples it to the others
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---------------------------------------------------------------------------
// register-basis fit (fw <= 3): one wavefront per context.  Lane s of register
// set k holds retained row 64k + s (fw + 2 words and its pivot); the rows of
// the current block are one per lane.  An LDS mirror of the retained rows
// feeds the block reduce with broadcast reads.
// ---------------------------------------------------------------------------
template <int FW>
__device__ __forceinline__ uint64_t word_at(const uint64_t (&f)[FW], int wi) {
    // branch-free select of word wi (wi is usually wavefront-uniform)
    if constexpr (FW == 1) {
        return f[0];
    } else if constexpr (FW == 2) {
        const uint64_t s1 = 0ull - static_cast<uint64_t>(wi == 1);
        return f[0] ^ ((f[0] ^ f[1]) & s1);
    } else {
        static_assert(FW == 3, "register basis holds at most 3 feature words");
        const uint64_t s1 = 0ull - static_cast<uint64_t>(wi == 1);
        const uint64_t s2 = 0ull - static_cast<uint64_t>(wi == 2);
        return f[0] ^ ((f[0] ^ f[1]) & s1) ^ ((f[0] ^ f[2]) & s2);
    }
}

// all-ones when bit b of w is set, else zero (32-bit: one mask serves both halves)
__device__ __forceinline__ uint32_t bit_mask(uint64_t w, int b) {
    const uint32_t dw = (b & 32) ? static_cast<uint32_t>(w >> 32) : static_cast<uint32_t>(w);
    return static_cast<uint32_t>(__builtin_amdgcn_sbfe(static_cast<int>(dw), b & 31, 1));  // sign of a 1-bit field
}

// 64 x 64 bit-matrix transpose across a wavefront: lane b holds row b; returned,
// lane f holds bit f of every row (bit b of the result = bit f of row b).  Six
// rounds that swap the off-diagonal blocks of size 32, 16, .., 1 with the partner
// lane (lane xor j).
template <int J, uint64_t M>
__device__ __forceinline__ uint64_t transpose_round(uint64_t v, int lane) {
    const uint32_t plo = static_cast<uint32_t>(__shfl_xor(static_cast<int>(static_cast<uint32_t>(v)), J));
    const uint32_t phi = static_cast<uint32_t>(__shfl_xor(static_cast<int>(static_cast<uint32_t>(v >> 32)), J));
    const uint64_t p = (static_cast<uint64_t>(phi) << 32) | plo;
    return (lane & J) ? ((v & ~M) | ((p & ~M) >> J)) : ((v & M) | ((p & M) << J));
}
__device__ __forceinline__ uint64_t transpose64(uint64_t v, int lane) {
    v = transpose_round<32, 0x00000000ffffffffull>(v, lane);
    v = transpose_round<16, 0x0000ffff0000ffffull>(v, lane);
    v = transpose_round<8, 0x00ff00ff00ff00ffull>(v, lane);
    v = transpose_round<4, 0x0f0f0f0f0f0f0f0full>(v, lane);
    v = transpose_round<2, 0x3333333333333333ull>(v, lane);
    return transpose_round<1, 0x5555555555555555ull>(v, lane);
}

// f ^ (m & d) with m a 32-bit all-ones/zero mask: one v_bitop3 per half
__device__ __forceinline__ uint64_t xor_and(uint64_t f, uint32_t m, uint64_t d) {
    const uint32_t lo = __builtin_amdgcn_bitop3_b32(static_cast<uint32_t>(f), m, static_cast<uint32_t>(d), 0x78);
    const uint32_t hi =
        __builtin_amdgcn_bitop3_b32(static_cast<uint32_t>(f >> 32), m, static_cast<uint32_t>(d >> 32), 0x78);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

// a ^ b ^ c: one v_bitop3 per half
__device__ __forceinline__ uint64_t xor3(uint64_t a, uint64_t b, uint64_t c) {
    const uint32_t lo = __builtin_amdgcn_bitop3_b32(static_cast<uint32_t>(a), static_cast<uint32_t>(b),
                                                    static_cast<uint32_t>(c), 0x96);
    const uint32_t hi = __builtin_amdgcn_bitop3_b32(static_cast<uint32_t>(a >> 32), static_cast<uint32_t>(b >> 32),
                                                    static_cast<uint32_t>(c >> 32), 0x96);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

constexpr int kRecWords = 6;  // LDS record: fw feature words, 2 output words, pivot (<= 6 words)

template <int FW>
__device__ __forceinline__ void fit_ctx_reg(const FitArgs& a, const CtxDesc& ds, uint64_t* sRec, int16_t* sPos) {
    constexpr int W = FW + F2_Y_WORDS;
    constexpr int NB = kLongRows / 64;  // blocks of a context in this class
    const int lane = threadIdx.x & 63;
    const int c = ds.c, n = ds.n, d = n + 1;
    const int64_t m = ds.m;  // at most kLongRows
    const uint64_t* R = a.rows + ds.row0;
    const uint64_t tmask = top_mask(n, FW);
    const int cw = n >> 6;
    const uint64_t cbit = 1ull << (n & 63);
    const uint64_t lane_lt = (1ull << lane) - 1;

    // block b's rows in register set b, one per lane; every row is loaded up front
    uint64_t f[NB][FW], y0[NB], y1[NB];
    int bp[NB];         // pivot of this lane's row, where the row is a basis row
    uint64_t piv[NB];   // lanes of set b that hold basis rows (uniform)
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int64_t i = 64 * b + lane;
        const bool valid = i < m;
#pragma unroll
        for (int w = 0; w < FW; ++w) f[b][w] = valid ? R[i * W + w] : 0ull;
        f[b][FW - 1] &= tmask;
        y0[b] = valid ? R[i * W + FW] : 0ull;
        y1[b] = valid ? R[i * W + FW + 1] : 0ull;
        bp[b] = 0;
        piv[b] = 0;
    }
    uint64_t xm[FW];  // the x columns of each feature word (the constant column cleared)
#pragma unroll
    for (int w = 0; w < FW; ++w) xm[w] = (w == cw) ? ~cbit : ~0ull;
    int rank = 0, ncontra = 0;
    int64_t first = -1;

    // dense copy of the basis rows (record = fw words, 2 output words, pivot) for
    // the broadcast reads of the block reduce; sPos[p] = record of pivot p
    auto store_mirror = [&](int nsets, bool positions) {
        int base = 0;
#pragma unroll
        for (int k = 0; k < NB; ++k) {
            if (k < nsets) {
                if ((piv[k] >> lane) & 1ull) {
                    const int s = base + __popcll(piv[k] & lane_lt);
                    uint64_t* rec = sRec + s * kRecWords;
#pragma unroll
                    for (int w = 0; w < FW; ++w) rec[w] = f[k][w];
                    rec[FW] = y0[k];
                    rec[FW + 1] = y1[k];
                    rec[W] = static_cast<uint64_t>(bp[k]);
                    if (positions) sPos[bp[k]] = static_cast<int16_t>(s);
                }
                base += __popcll(piv[k]);
            }
        }
    };

#pragma unroll
    for (int b = 0; b < NB; ++b) {
        if (64 * b >= m) break;
        const bool valid = 64 * b + lane < m;
        // (1) reduce against the basis of the earlier blocks: it is fully reduced,
        //     so the row's own (unreduced) bits at the pivot columns select the
        //     records to add; the selection masks do not depend on one another
        if (rank > 0) {
            uint64_t f0[FW];
#pragma unroll
            for (int w = 0; w < FW; ++w) f0[w] = f[b][w];
            constexpr int U = FW >= 3 ? 1 : FW == 2 ? 2 : 4;  // records read ahead (register budget)
            int s = 0;
            for (; s + U <= rank; s += U) {
                uint64_t rv[U][W];
                int pv[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const uint64_t* rec = sRec + (s + u) * kRecWords;
#pragma unroll
                    for (int w = 0; w < W; ++w) rv[u][w] = rec[w];
                    pv[u] = static_cast<int>(rec[W]);
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const uint32_t mm = bit_mask(word_at<FW>(f0, pv[u] >> 6), pv[u] & 63);
#pragma unroll
                    for (int w = 0; w < FW; ++w) f[b][w] = xor_and(f[b][w], mm, rv[u][w]);
                    y0[b] = xor_and(y0[b], mm, rv[u][FW]);
                    y1[b] = xor_and(y1[b], mm, rv[u][FW + 1]);
                }
            }
            for (; s < rank; ++s) {
                const uint64_t* rec = sRec + s * kRecWords;
                const int p = static_cast<int>(rec[W]);
                const uint32_t mm = bit_mask(word_at<FW>(f0, p >> 6), p & 63);
#pragma unroll
                for (int w = 0; w < FW; ++w) f[b][w] = xor_and(f[b][w], mm, rec[w]);
                y0[b] = xor_and(y0[b], mm, rec[FW]);
                y1[b] = xor_and(y1[b], mm, rec[FW + 1]);
            }
        }

        // (2) elimination in stream order: the earliest row with a nonzero
        //     feature residual becomes a basis row where it stands; its pivot is
        //     cleared from the later rows of the block and from the basis rows
        //     of this and the earlier blocks (the basis stays fully reduced)
        uint64_t pending = __ballot(valid);
        for (;;) {
            uint64_t any = f[b][0];
#pragma unroll
            for (int w = 1; w < FW; ++w) any |= f[b][w];
            const uint64_t nz = __ballot(any != 0) & pending;
            if (!nz) break;
            const int j = ffs64(nz);
            uint64_t F[FW];
#pragma unroll
            for (int w = 0; w < FW; ++w) F[w] = readlane64(f[b][w], j);
            const uint64_t Y0 = readlane64(y0[b], j), Y1 = readlane64(y1[b], j);
            // pivot: highest-priority set feature bit (x_{n-1} .. x_0, else the
            // constant: the row is nonzero)
            int p = n;
#pragma unroll
            for (int w = 0; w < FW; ++w) {
                const uint64_t v = F[w] & xm[w];
                p = v ? 64 * w + msb64(v) : p;
            }
            const int pw = p >> 6, pb = p & 63;
            {  // this block: every row holding bit p except the new basis row itself
                const uint32_t mm = bit_mask(word_at<FW>(f[b], pw), pb) & (lane == j ? 0u : ~0u);
#pragma unroll
                for (int w = 0; w < FW; ++w) f[b][w] = xor_and(f[b][w], mm, F[w]);
                y0[b] = xor_and(y0[b], mm, Y0);
                y1[b] = xor_and(y1[b], mm, Y1);
            }
#pragma unroll
            for (int k = 0; k < NB; ++k) {  // earlier blocks: only their basis rows are nonzero
                if (k < b && piv[k]) {
                    const uint32_t mm = bit_mask(word_at<FW>(f[k], pw), pb);
#pragma unroll
                    for (int w = 0; w < FW; ++w) f[k][w] = xor_and(f[k][w], mm, F[w]);
                    y0[k] = xor_and(y0[k], mm, Y0);
                    y1[k] = xor_and(y1[k], mm, Y1);
                }
            }
            if (lane == j) bp[b] = p;
            piv[b] |= 1ull << j;
            pending &= ~(1ull << j);
            ++rank;
        }
        // (3) every other row of the block now has zero features: redundant, or
        //     contradictory when its output is nonzero (Eq. 8)
        const uint64_t cm = __ballot(valid && !((piv[b] >> lane) & 1ull) && (y0[b] | y1[b]) != 0);
        if (cm) {
            if (ncontra == 0) first = 64 * b + ffs64(cm);
            ncontra += __popcll(cm);
        }
        if (piv[b] && 64 * (b + 1) < m) {
            store_mirror(b + 1, false);
            wave_sync();
        }
    }

    // outputs: basis rows and pivots in descending priority, canonical map, scalars
    for (int j = lane; j < d; j += 64) sPos[j] = -1;
    wave_sync();
    store_mirror(NB, true);
    wave_sync();
    uint64_t pm[FW];  // pivot columns (uniform): the positions that received a record
#pragma unroll
    for (int w = 0; w < FW; ++w) pm[w] = __ballot(64 * w + lane < d && sPos[64 * w + lane] >= 0);
    const int64_t bo = ds.bo, po = ds.po, mo = ds.mo;
#pragma unroll
    for (int k = 0; k < NB; ++k) {
        if ((piv[k] >> lane) & 1ull) {
            const int p = bp[k];
            int kout = rank - 1;
            if (p != n) {  // pivots of higher priority: x bits above p
                kout = 0;
#pragma unroll
                for (int w = 0; w < FW; ++w) {
                    uint64_t v = pm[w];
                    if (w == cw) v &= ~cbit;
                    if (w < (p >> 6)) v = 0;
                    if (w == (p >> 6)) v &= ((p & 63) == 63) ? 0ull : (~0ull << ((p & 63) + 1));
                    kout += __popcll(v);
                }
            }
            uint64_t* out = a.basis + bo + static_cast<int64_t>(kout) * W;
#pragma unroll
            for (int w = 0; w < FW; ++w) out[w] = f[k][w];
            out[FW] = y0[k];
            out[FW + 1] = y1[k];
            a.pivots[po + kout] = p;
        }
    }
    for (int j = lane; j < d; j += 64) {
        const int sl = sPos[j];
        a.maps[mo + 2 * j] = sl >= 0 ? sRec[sl * kRecWords + FW] : 0ull;
        a.maps[mo + 2 * j + 1] = sl >= 0 ? sRec[sl * kRecWords + FW + 1] : 0ull;
    }
    // parity-check rows of the free columns (sRec holds the final rows, sPos their
    // records).  Word v of the row of free column fc = 64 w + f holds, at bit b, bit fc
    // of the basis row of pivot 64 v + b: with lane b holding word w of that basis row
    // (zero for a free column), a bit-matrix transpose across the wavefront gives lane
    // f exactly that word; the free lanes then store their rows in ascending order.
    uint64_t* H = a.tables + bo;
    if (has_parity_rows(d, rank)) {
        // (no arrays indexed by the loop counters: where these loops stay rolled,
        // such an array would live in scratch memory)
        int base = 0;  // free columns in the words before w
#pragma unroll
        for (int w = 0; w < FW; ++w) {
            const int sw = (64 * w + lane < d) ? sPos[64 * w + lane] : -1;
            const uint64_t fr = ~__ballot(sw >= 0) & (w == FW - 1 ? tmask : ~0ull);
            if (!fr) continue;  // no free column in this word (full rank: none at all)
            const bool mine = (fr >> lane) & 1ull;
            const int64_t i = base + __popcll(fr & lane_lt);
#pragma unroll
            for (int v = 0; v < FW; ++v) {
                const int sv = (64 * v + lane < d) ? sPos[64 * v + lane] : -1;
                const uint64_t col = transpose64(sv >= 0 ? sRec[sv * kRecWords + w] : 0ull, lane);
                if (mine) H[i * FW + v] = col | (v == w ? (1ull << lane) : 0ull);
            }
            base += __popcll(fr);
        }
    }
    if (lane == 0) {
        a.rank[c] = rank;
        a.n_contra[c] = ncontra;
        a.first_contra[c] = first;
        a.ctx_flags[c] = ncontra ? F2_CTX_CONTRADICTION : 0u;
    }
    wave_sync();
}

// One workgroup of kRegWaves wavefronts per compute unit, each wavefront fitting
// its own contexts in its own LDS region.  The workgroup's share of the class
// list (dealt in snake order, so shares carry similar work) starts with one
// context per wavefront in snake order over the four SIMDs (wavefront w runs on
// SIMD w mod 4), largest first; then wavefronts take the next context of the
// share as they finish, through a counter in LDS.
constexpr int kRegWaves = 16;

__global__ __launch_bounds__(64 * kRegWaves) void k_fit_reg(FitArgs a) {
    __shared__ __align__(16) uint64_t sRec[kRegWaves][64 * kRegMaxFW * kRecWords];
    __shared__ int16_t sPos[kRegWaves][64 * kRegMaxFW];
    __shared__ int sNext;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    if (tid == 0) sNext = kRegWaves;
    __syncthreads();
    const int r = wave >> 2, simd = wave & 3;
    // the share's list positions (the class bounds read once)
    const int lo = a.plan[kClsReg], cnt = a.plan[kClsReg + 1] - lo;
    const int G = static_cast<int>(gridDim.x), g = static_cast<int>(blockIdx.x);
    auto ctx_at = [&](int i) {  // context at position i of the share, or num_ctx past its end
        const int64_t e = static_cast<int64_t>(i) * G + ((i & 1) ? G - 1 - g : g);
        return __builtin_amdgcn_readfirstlane(e < cnt ? a.plan[kPlanHead + lo + static_cast<int>(e)] : a.num_ctx);
    };
    auto next_pos = [&]() {
        int nk = 0;
        if (lane == 0) nk = atomicAdd(&sNext, 1);
        return __builtin_amdgcn_readfirstlane(nk);
    };
    // a two-deep pipeline: while a context is fitted, the next one's descriptor
    // and the one after's id are already loading
    CtxDesc ds = readlane_desc(load_desc(a, ctx_at(4 * r + ((r & 1) ? 3 - simd : simd))), 0);
    int c1 = ctx_at(next_pos());
    while (ds.c >= 0) {
        const CtxDesc dn = readlane_desc(load_desc(a, c1), 0);
        const int c2 = ctx_at(next_pos());
        switch (feat_words(ds.n)) {
            case 1: fit_ctx_reg<1>(a, ds, sRec[wave], sPos[wave]); break;
            case 2: fit_ctx_reg<2>(a, ds, sRec[wave], sPos[wave]); break;
            default: fit_ctx_reg<3>(a, ds, sRec[wave], sPos[wave]); break;
        }
        ds = dn;
        c1 = c2;
    }
}

// ---------------------------------------------------------------------------
// pivot-indexed LDS-basis fit: retained row of pivot p in record p (fw + 2
// words), a pivot-column bitmask beside it, for contexts of 4-8 feature words
// and for long contexts of up to 8 feature words.  With NW > 1 wavefronts (the
// kernel runs kPivWaves) the next NW blocks of 64 rows are reduced
// in parallel, one per wavefront; the first block (in stream order) that still
// holds a nonzero feature residual runs the insertion loop in its own
// wavefront (in registers), the blocks before it are only classified, the
// blocks after it are redone against the grown basis; then every wavefront
// clears the new pivots from the retained records.  Once the basis stops
// growing every round completes NW blocks, and a large basis reduces through
// Four-Russians tables.
// ---------------------------------------------------------------------------
constexpr int kPivRec = kPivMaxFW + F2_Y_WORDS;  // record words
constexpr int kPivCap = 64 * kPivMaxFW;          // d <= 512
constexpr int kPivWaves = 4;
constexpr int kPivThreads = 64 * kPivWaves;

template <int FW>
__device__ __forceinline__ uint64_t sel_word(const uint64_t (&f)[FW], int wi) {
    uint64_t v = f[0];
#pragma unroll
    for (int k = 1; k < FW; ++k) v ^= (f[k] ^ f[0]) & (0ull - static_cast<uint64_t>(wi == k));
    return v;
}

// Four-Russians tables for contexts of up to 4 feature words (d <= 256): their
// records use rec[0, 256), and the tables take the rest of rec plus tabx (the
// two are adjacent): table g holds the 16 XOR combinations of the retained rows
// of positions 4g .. 4g+3 (fw + 2 words each; absent pivots contribute zero)
constexpr int kPivTabExtra = 1480;  // keeps three workgroups per compute unit within the LDS
constexpr int kPivTabWords = (kPivCap / 2) * kPivRec + kPivTabExtra;
constexpr int kPivTabMinRank = 32;   // smaller bases reduce as fast record by record
constexpr int kPivTabMinRows = 512;  // tables are built only with two rounds of rows or more to go

struct alignas(16) PivShared {  // 16-byte aligned: the tables are read 16 bytes at a time
    uint64_t rec[kPivCap][kPivRec];
    uint64_t tabx[kPivTabExtra];  // continues rec (tables)
    int ntab;                     // valid tables (positions [0, 4 ntab)), 0: none
    uint64_t pm[kPivMaxFW];   // pivot columns of the retained rows
    uint64_t npm[kPivMaxFW];  // pivot columns of the rows the current round added
    int flag[8];  // per wavefront (up to 8)
    int contra, nnew;
    long long first, round_first;
};

// all threads: the tables of the first positions (as many as fit) from the records
template <int FW, int NW>
__device__ __forceinline__ void piv_build_tables(PivShared& S, int d) {
    constexpr int W = FW + F2_Y_WORDS;
    constexpr int cap = kPivTabWords / (16 * W);
    const int nt = (d + 3) / 4 < cap ? (d + 3) / 4 : cap;
    uint64_t* tab = &S.rec[kPivCap / 2][0];
    for (int t = threadIdx.x; t < nt * W; t += 64 * NW) {  // one (table, word) per step
        const int g = t / W, w = t - g * W;
        uint64_t* e = tab + g * 16 * W + w;  // entry k of table g at e[k W]
        e[0] = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int p = 4 * g + b;
            const bool piv = p < d && ((S.pm[p >> 6] >> (p & 63)) & 1ull);
            const uint64_t r = piv ? S.rec[p][w] : 0ull;
            for (int k = 0; k < (1 << b); ++k) e[((1 << b) + k) * W] = e[k * W] ^ r;
        }
    }
    if (threadIdx.x == 0) S.ntab = nt;
}

// one table entry of W words from LDS, 16 bytes per read where W is even (the
// entries then start 16-byte aligned)
typedef unsigned long long u64x2_t __attribute__((ext_vector_type(2)));
template <int W>
__device__ __forceinline__ void load_entry(const uint64_t* e, uint64_t (&v)[W]) {
    if constexpr (W % 2 == 0) {
#pragma unroll
        for (int u = 0; u < W / 2; ++u) {
            const u64x2_t p = reinterpret_cast<const u64x2_t*>(e)[u];
            v[2 * u] = p.x;
            v[2 * u + 1] = p.y;
        }
    } else {
#pragma unroll
        for (int u = 0; u < W; ++u) v[u] = e[u];
    }
}

// reduce this wavefront's block rows against the retained basis (one pass: the
// basis is fully reduced).  Positions [0, 4 ntab) by table lookups: the row's own
// 4 bits at positions 4g .. 4g+3, masked to the pivots, select entry of table g.
template <int FW>
__device__ __forceinline__ void piv_reduce(PivShared& S, int fw, int ntab, uint64_t (&f)[FW], uint64_t& y0,
                                           uint64_t& y1) {
    constexpr int W = FW + F2_Y_WORDS;
    uint64_t f0[FW];
#pragma unroll
    for (int w = 0; w < FW; ++w) f0[w] = f[w];
    if constexpr (FW <= 4) {
        const uint64_t* tab = &S.rec[kPivCap / 2][0];
#pragma unroll
        for (int w = 0; w < FW; ++w) {
            if (16 * w >= ntab) break;
            const uint64_t pmw = S.pm[w];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const uint32_t half = h ? static_cast<uint32_t>(f0[w] >> 32) : static_cast<uint32_t>(f0[w]);
                const uint32_t pmh = h ? static_cast<uint32_t>(pmw >> 32) : static_cast<uint32_t>(pmw);
#pragma unroll
                for (int k = 0; k < 8; k += 4) {  // four tables per step: every entry read issued first
                    const int g = 16 * w + 8 * h + k;
                    if (g >= ntab) break;
                    uint64_t ev[4][W];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        // past the last table: entry 0 of table g (zero)
                        const bool in = g + q < ntab;
                        const uint32_t iq = in ? __builtin_amdgcn_ubfe(half, 4 * (k + q), 4) &
                                                     ((pmh >> (4 * (k + q))) & 0xFu)
                                               : 0u;
                        load_entry<W>(tab + (16 * (in ? g + q : g) + static_cast<int>(iq)) * W, ev[q]);
                    }
#pragma unroll
                    for (int u = 0; u < FW; ++u) f[u] = xor3(xor3(f[u], ev[0][u], ev[1][u]), ev[2][u], ev[3][u]);
                    y0 = xor3(xor3(y0, ev[0][FW], ev[1][FW]), ev[2][FW], ev[3][FW]);
                    y1 = xor3(xor3(y1, ev[0][FW + 1], ev[1][FW + 1]), ev[2][FW + 1], ev[3][FW + 1]);
                }
            }
        }
    }
    const int done = FW <= 4 ? 4 * ntab : 0;  // positions below are reduced
    for (int pw = done >> 6; pw < fw; ++pw) {
        uint64_t pm = S.pm[pw];
        if (pw == (done >> 6) && (done & 63)) pm &= ~0ull << (done & 63);
        if (!pm) continue;
        const uint64_t ow = sel_word<FW>(f0, pw);  // unreduced word pw of this lane's row
        while (pm) {
            int bb[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                bb[u] = pm ? ffs64(pm) : -1;
                pm &= pm - 1;
            }
            uint64_t rv[4][FW + 2];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const uint64_t* rec = S.rec[64 * pw + (bb[u] < 0 ? 0 : bb[u])];
#pragma unroll
                for (int w = 0; w < FW + 2; ++w) rv[u][w] = rec[w];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const uint32_t mk = bb[u] < 0 ? 0u : bit_mask(ow, bb[u]);
#pragma unroll
                for (int w = 0; w < FW; ++w) f[w] = xor_and(f[w], mk, rv[u][w]);
                y0 = xor_and(y0, mk, rv[u][FW]);
                y1 = xor_and(y1, mk, rv[u][FW + 1]);
            }
        }
    }
}

// in-block elimination of one wavefront's block, in registers: the earliest row
// with a nonzero feature residual becomes a new basis row and stays in its lane;
// its pivot is cleared from every other row of the block, earlier new rows
// included, so the new rows end fully reduced among themselves (and hold no
// retained pivot: the block was reduced first).  Rows before it with a zero
// residual are classified on the way.  The new rows then go to their records,
// their pivots to npm and their count to nnew; the retained rows are cleared of
// the new pivots afterwards by all wavefronts (piv_backsub).
template <int FW>
__device__ void piv_insert(PivShared& S, int n, int64_t b0, bool valid, uint64_t (&f)[FW], uint64_t& y0, uint64_t& y1,
                           int& ncon, long long& firstc) {
    const int lane = threadIdx.x & 63;
    const int cw = n >> 6;
    const uint64_t cbit = 1ull << (n & 63);
    uint64_t xm[FW];  // the x columns of each feature word (the constant column cleared)
#pragma unroll
    for (int w = 0; w < FW; ++w) xm[w] = (w == cw) ? ~cbit : ~0ull;
    if (lane < FW) S.npm[lane] = 0;
    uint64_t pending = __ballot(valid);
    uint64_t ins = 0;  // lanes holding new basis rows
    int mypiv = 0;     // this lane's pivot, where it holds a new basis row
    while (pending) {
        uint64_t any = f[0];
#pragma unroll
        for (int w = 1; w < FW; ++w) any |= f[w];
        const uint64_t nz = __ballot(any != 0) & pending;
        // pending rows before the earliest nonzero one have zero residuals
        const uint64_t zr = nz ? pending & ((nz & (0ull - nz)) - 1) : pending;
        if (zr) {
            const uint64_t cm = __ballot((y0 | y1) != 0) & zr;
            if (cm) {
                if (ncon == 0) firstc = b0 + ffs64(cm);
                ncon += __popcll(cm);
            }
            pending &= ~zr;
        }
        if (!nz) break;
        const int j = ffs64(nz);
        uint64_t F[FW];
#pragma unroll
        for (int w = 0; w < FW; ++w) F[w] = readlane64(f[w], j);
        const uint64_t Y0 = readlane64(y0, j), Y1 = readlane64(y1, j);
        // pivot: the highest-priority set feature bit, x_{n-1} .. x_0, else the
        // constant (the row is nonzero)
        int p = n;
#pragma unroll
        for (int w = 0; w < FW; ++w) {
            const uint64_t v = F[w] & xm[w];
            p = v ? 64 * w + msb64(v) : p;
        }
        const int pw = p >> 6, pb = p & 63;
        const uint32_t mm = bit_mask(sel_word<FW>(f, pw), pb) & (lane == j ? 0u : ~0u);
#pragma unroll
        for (int w = 0; w < FW; ++w) f[w] = xor_and(f[w], mm, F[w]);
        y0 = xor_and(y0, mm, Y0);
        y1 = xor_and(y1, mm, Y1);
        if (lane == j) mypiv = p;
        ins |= 1ull << j;
        pending &= ~(1ull << j);
    }
    wave_sync();  // npm cleared before the new pivots are added
    if ((ins >> lane) & 1ull) {
        uint64_t* rec = S.rec[mypiv];
#pragma unroll
        for (int w = 0; w < FW; ++w) rec[w] = f[w];
        rec[FW] = y0;
        rec[FW + 1] = y1;
        atomicOr(reinterpret_cast<unsigned long long*>(&S.npm[mypiv >> 6]), 1ull << (mypiv & 63));
    }
    if (lane == 0) S.nnew = __popcll(ins);
}

// clear the round's new pivots from the retained rows (records of S.pm), one
// record per thread.  The new rows hold no other new pivot, so a record's bits
// at the new pivots, read once before any addition, select the rows to add.
template <int FW, int NW>
__device__ __forceinline__ void piv_backsub(PivShared& S, int d, int fw) {
    for (int s = threadIdx.x; s < d; s += 64 * NW) {
        if (!((S.pm[s >> 6] >> (s & 63)) & 1ull)) continue;
        uint64_t* rec = S.rec[s];
        uint64_t R[FW + 2];
#pragma unroll
        for (int w = 0; w < FW + 2; ++w) R[w] = rec[w];
        uint64_t R0[FW];
#pragma unroll
        for (int w = 0; w < FW; ++w) R0[w] = R[w];
#pragma unroll
        for (int w = 0; w < FW; ++w) {
            if (w >= fw) break;
            uint64_t m = S.npm[w];
            while (m) {
                const int b = ffs64(m);
                m &= m - 1;
                const uint32_t mk = bit_mask(R0[w], b);
                const uint64_t* nr = S.rec[64 * w + b];
#pragma unroll
                for (int u = 0; u < FW + 2; ++u) R[u] = xor_and(R[u], mk, nr[u]);
            }
        }
#pragma unroll
        for (int w = 0; w < FW + 2; ++w) rec[w] = R[w];
    }
}

template <int FW, int NW>
__device__ __forceinline__ void fit_ctx_piv(const FitArgs& a, const CtxDesc& ds, PivShared& S) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int c = ds.c, n = ds.n, d = n + 1;
    const int fw = feat_words(n);  // <= FW; records keep FW feature words, then the two output words
    const int Wr = fw + F2_Y_WORDS;
    const int64_t m = ds.m;
    const uint64_t* R = a.rows + ds.row0;
    const uint64_t tmask = top_mask(n, fw);

    static_assert(NW > 1, "rounds of several wavefronts");
    if (tid < kPivMaxFW) {
        S.pm[tid] = 0;
        S.npm[tid] = 0;
    }
    if (tid == 0) {
        S.contra = 0;
        S.nnew = 0;
        S.ntab = 0;
        S.first = -1;
    }
    __syncthreads();
    // the next round's block is loaded while this round runs, on the guess that
    // the round completes all NW blocks (it does once the basis stops growing);
    // not for the widest records, whose registers it would cost occupancy
    constexpr bool kPrefetch = FW <= 4;
    // raw words of this wavefront's row in the block at base, row index clamped
    // into the segment (lanes past its end are masked at use).  Up to 4 feature
    // words every load is issued (fw >= FW - 1 there, so word FW - 1 is still in
    // the row): a fixed count of loads in flight, which the wait for them can count.
    auto load_raw = [&](int64_t base, uint64_t (&raw)[FW + 2]) {
        const int64_t ii = base + 64 * wave + lane;
        const uint64_t* row = R + (ii < m ? ii : m - 1) * Wr;
#pragma unroll
        for (int w = 0; w < FW; ++w) raw[w] = (kPrefetch || w < fw) ? row[w] : 0ull;
        raw[FW] = row[fw];
        raw[FW + 1] = row[fw + 1];
    };
    uint64_t pre[FW + 2];
    int64_t pre_b0 = -1;
    int rank = 0;
    int64_t b0 = 0;
    while (b0 < m) {
        const int64_t bw = b0 + 64 * wave;  // this wavefront's block
        const int64_t i = bw + lane;
        const bool valid = i < m;
        uint64_t raw[FW + 2];
        if (kPrefetch && pre_b0 == b0) {
#pragma unroll
            for (int w = 0; w < FW + 2; ++w) raw[w] = pre[w];
        } else {
            load_raw(b0, raw);
        }
        if constexpr (kPrefetch) {  // issued unconditionally (a block past the end reads the last row)
            pre_b0 = b0 + 64 * NW;
            load_raw(pre_b0, pre);
        }
        uint64_t f[FW], y0, y1;
#pragma unroll
        for (int w = 0; w < FW; ++w) f[w] = (valid && w < fw) ? raw[w] : 0ull;
#pragma unroll
        for (int w = 0; w < FW; ++w)
            if (w == fw - 1) f[w] &= tmask;
        y0 = valid ? raw[FW] : 0ull;
        y1 = valid ? raw[FW + 1] : 0ull;
        if constexpr (FW <= 4) {  // a large basis that will serve two rounds or more: tables
            if (S.ntab == 0 && rank >= kPivTabMinRank && m - b0 >= kPivTabMinRows) {
                piv_build_tables<FW, NW>(S, d);
                __syncthreads();
            }
        }
        if (rank > 0) piv_reduce<FW>(S, fw, S.ntab, f, y0, y1);
        uint64_t any = f[0];
#pragma unroll
        for (int w = 1; w < FW; ++w) any |= f[w];
        const bool has_nz = __ballot(valid && any != 0) != 0;
        if (lane == 0) S.flag[wave] = has_nz ? 1 : 0;
        if (tid == 0) S.round_first = 0x7fffffffffffffffll;
        __syncthreads();
        int wstar = NW;
        for (int w = NW - 1; w >= 0; --w)
            if (S.flag[w]) wstar = w;
        int ncon = 0;
        long long firstc = -1;
        if (wave < wstar) {  // every residual is zero: redundant or contradictory rows
            const uint64_t cm = __ballot(valid && (y0 | y1) != 0);
            if (cm) {
                ncon = __popcll(cm);
                firstc = bw + ffs64(cm);
            }
        } else if (wave == wstar) {
            piv_insert<FW>(S, n, bw, valid, f, y0, y1, ncon, firstc);
        }
        if (lane == 0 && ncon) {
            atomicAdd(&S.contra, ncon);
            atomicMin(&S.round_first, firstc);
        }
        __syncthreads();
        if (S.nnew) {  // retained rows lose the new pivots, then the new rows join them
            piv_backsub<FW, NW>(S, d, fw);
            __syncthreads();
            if (tid < fw) S.pm[tid] |= S.npm[tid];
            if (tid == 0) S.ntab = 0;  // the tables no longer match the basis
            __syncthreads();
        }
        if (tid == 0 && S.first < 0 && S.round_first != 0x7fffffffffffffffll) S.first = S.round_first;
        rank = 0;
        for (int w = 0; w < fw; ++w) rank += __popcll(S.pm[w]);
        __syncthreads();
        if (tid == 0) S.nnew = 0;
        b0 += 64 * static_cast<int64_t>(wstar < NW ? wstar + 1 : NW);
    }
    __syncthreads();

    // outputs: basis rows and pivots in descending priority, canonical map, encode table, scalars
    const int64_t bo = ds.bo, po = ds.po, mo = ds.mo;
    const int cw = n >> 6;
    const uint64_t cbit = 1ull << (n & 63);
    for (int j = tid; j < d; j += 64 * NW) {
        const bool present = (S.pm[j >> 6] >> (j & 63)) & 1ull;
        a.maps[mo + 2 * j] = present ? S.rec[j][FW] : 0ull;
        a.maps[mo + 2 * j + 1] = present ? S.rec[j][FW + 1] : 0ull;
        if (!present) continue;
        int k = rank - 1;
        if (j != n) {  // pivots of higher priority: x bits above j
            k = 0;
            for (int w = j >> 6; w < fw; ++w) {
                uint64_t v = S.pm[w];
                if (w == (j >> 6)) v &= (j & 63) == 63 ? 0ull : (~0ull << ((j & 63) + 1));
                if (w == cw) v &= ~cbit;
                k += __popcll(v);
            }
        }
        uint64_t* out = a.basis + bo + static_cast<int64_t>(k) * Wr;
#pragma unroll
        for (int w = 0; w < FW; ++w)
            if (w < fw) out[w] = S.rec[j][w];
        out[fw] = S.rec[j][FW];
        out[fw + 1] = S.rec[j][FW + 1];
        a.pivots[po + k] = j;
    }
    // parity-check rows of the free columns (word v of the row of free column 64 w + f
    // holds, at bit b, bit f of word w of the retained row of pivot 64 v + b): per word
    // pair (w, v), taken by wavefront v mod NW, a bit-matrix transpose of word w of the
    // retained rows 64 v .. 64 v + 63 (zero for free columns) gives lane f its word
    uint64_t* H = a.tables + bo;
    if (has_parity_rows(d, rank)) {
        const uint64_t lane_lt = (1ull << lane) - 1;
        int base = 0;  // free columns in the words before w
        for (int w = 0; w < fw; ++w) {
            const uint64_t fr = ~S.pm[w] & (w == fw - 1 ? tmask : ~0ull);
            if (!fr) continue;  // no free column in this word
            const bool mine = (fr >> lane) & 1ull;
            const int64_t i = base + __popcll(fr & lane_lt);
            for (int v = wave; v < fw; v += NW) {
                const bool piv = (S.pm[v] >> lane) & 1ull;
                const uint64_t col = transpose64(piv ? S.rec[64 * v + lane][w] : 0ull, lane);
                if (mine) H[i * fw + v] = col | (v == w ? (1ull << lane) : 0ull);
            }
            base += __popcll(fr);
        }
    }
    if (tid == 0) {
        a.rank[c] = rank;
        a.n_contra[c] = S.contra;
        a.first_contra[c] = S.first;
        a.ctx_flags[c] = S.contra ? F2_CTX_CONTRADICTION : 0u;
    }
    __syncthreads();
}

// ---------------------------------------------------------------------------
// large-context fit (fw > 8): one workgroup of 8 wavefronts per context.  Lanes
// span the feature words of a row (lane w holds word w); the two output words of
// the 8 rows a wavefront holds sit in lanes 2k, 2k+1 of one more register.  The
// working basis lives in the caller's basis buffer, one slot per priority
// position (slot t holds the row whose pivot is the t-th highest-priority
// feature), and is kept fully reduced, so the final descending-priority order is
// an in-place compaction.  Rows go in blocks of 64, rows 8w .. 8w+7 of a block
// held by wavefront w:
//   (1) block reduce with Four-Russians tables (the method of Arlazarov, Dinic,
//       Kronrod and Faradzev): the retained rows of four consecutive pivot
//       positions give a 16-entry LDS table of all their XOR combinations, and a
//       row's own four bits at those positions (unchanged by the other retained
//       rows, the basis being fully reduced) select the entry to add.  Eight
//       tables (32 pivot positions) are built per round while the previous
//       round's tables are read;
//   (2) in-block elimination in stream order, one wavefront at a time over its
//       own eight rows, each new pivot cleared from that wavefront's other rows at
//       once and from the other wavefronts' rows after a barrier (earlier new rows
//       included, so the block's new rows end fully reduced);
//   (3) back-substitution: the new rows, in descending priority, form tables of
//       four rows each, and every retained row adds the entry its bits at those
//       pivots select; (4) the new rows are stored at their priority slots.
// A feature word whose columns are all retained pivots is zero in every reduced
// row and in every new row, so steps (1) and (3) read and write only the other
// words (the "active" lanes); the words left alone keep the unreduced bits the
// selections are read from.  Once the rank reaches d every later row lies in the
// span and the basis is the identity on the features, so a row's residual is
// y + M phi (the canonical map, staged in LDS): those rows are only checked for
// contradictions.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int prio_slot(int p, int n) { return p < n ? n - 1 - p : n; }
__device__ __forceinline__ int slot_pivot(int t, int n) { return t < n ? n - 1 - t : n; }

constexpr int kLargeWaves = kLargeThreads / 64;      // 8
constexpr int kLgSlots = kLargeRows / kLargeWaves;   // block rows per wavefront: 8
constexpr int kLgEnt = 16;                           // entries of a 4-bit table
constexpr int kLgRoundTables = kLargeWaves;          // reduce: one table per wavefront per round
constexpr int kLgBuf = kLgRoundTables * kLgEnt;      // entries of one round's tables
static_assert(kLgSlots == 8, "a wavefront's output words occupy lanes 0-15");
static_assert(kLgRoundTables * 4 == 32, "a round covers half a pivot word");

struct LargeShared {
    uint64_t tf[2 * kLgBuf][64];  // table entries, feature words (lane = word); the map in the full-rank phase
    uint64_t tz[2 * kLgBuf][2];   // table entries, output words
    int pubP[2][kLgSlots];        // in-block elimination: pivots published by one wavefront (tables in tf)
    int pubN[2];
    int rowPiv[kLargeRows];       // pivot of each block row that became a basis row, else -1
    int nsorted[kLargeRows];      // the block's new pivots in descending priority
    int above[64];                // new pivots (constant excluded) in feature words above w
    uint64_t pm[64];              // pivot columns of the retained basis
    uint64_t npm[64];             // pivot columns found in the current block
    int contra, nnew;
    int timeout;                  // a group barrier of this context gave up
    long long firstMin;
};

// per-lane value of slot lane/2 for lanes 0-15 (the output-word lanes), 0 elsewhere
template <typename T>
__device__ __forceinline__ T spread_slots(const T (&v)[kLgSlots], int lane) {
    T r = 0;
#pragma unroll
    for (int k = 0; k < kLgSlots; ++k) r = ((lane >> 1) == k) ? v[k] : r;
    return r;
}

// all-ones in the lanes whose bit is set in the 64-bit mask e
__device__ __forceinline__ uint32_t lanes_of(uint64_t e, int lane) {
    return 0u - static_cast<uint32_t>((e >> lane) & 1ull);
}

// the next half pivot word (2 pw + h) after r that holds retained pivots and
// belongs to member g of a group of G (a power of 2; pivot words pw = g mod G), or -1
__device__ __forceinline__ int next_round(const LargeShared& L, int fw, int r, int G, int g) {
    for (int t = r + 1; t < 2 * fw; ++t) {
        if (((t >> 1) & (G - 1)) != g) continue;
        const uint64_t v = L.pm[t >> 1];
        if ((t & 1) ? (v >> 32) != 0 : (v & 0xffffffffull) != 0) return t;
    }
    return -1;
}

// barrier of the G workgroups that fit one context together (all resident: the
// launch is cooperative); counter `bar` only grows, epoch counts this member's
// arrivals.  The wait is bounded (spin_limit polls) so that a kernel can never
// hang on it; a wait that gives up sets *timed_out (LDS, read after the
// workgroup barrier that ends this call), and the context is reported
// F2_CTX_SYNC_TIMEOUT.  spin_limit 0 never waits: every call gives up.
// full: release and acquire fences around it (every earlier global write of the
// group visible after it); otherwise only the arrival order: the data exchanged
// across it must be written and read with device-scope atomic stores and loads.
__device__ __forceinline__ void group_barrier(int* bar, int& epoch, int G, int spin_limit, int* timed_out,
                                              bool full = true) {
    if (full) __threadfence();
    __builtin_amdgcn_s_waitcnt(0);  // this thread's stores performed before the arrival is counted
    __syncthreads();
    ++epoch;
    if (threadIdx.x == 0) {
        __hip_atomic_fetch_add(bar, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const int target = G * epoch;
        bool arrived = false;
        for (int spin = 0; spin < spin_limit; ++spin) {
            if (__hip_atomic_load(bar, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target) {
                arrived = true;
                break;
            }
            __builtin_amdgcn_s_sleep(2);
        }
        if (!arrived) *timed_out = 1;
        if (full) __threadfence();
    }
    __syncthreads();
}

__device__ __forceinline__ void put_dev(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// device-scope (sc1) loads through a buffer resource: the same coherence as a
// device-scope atomic load, but the compiler keeps many of them in flight
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ __amdgpu_buffer_rsrc_t dev_rsrc(const uint64_t* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint64_t*>(base), 0, static_cast<int>(bytes), 0x00020000);
}
__device__ __forceinline__ uint64_t get_dev(__amdgpu_buffer_rsrc_t r, uint32_t word) {
    const u32x2_t v = __builtin_amdgcn_raw_buffer_load_b64(r, static_cast<int>(8 * word), 0, 16 /* sc1 */);
    return (static_cast<uint64_t>(v.y) << 32) | v.x;
}

struct GroupRows {
    uint64_t f[4];     // feature word `lane` of four retained rows, as loaded
    uint64_t z[4];     // output word (lane & 1) of the same rows, as loaded
    uint32_t present;  // rows that exist (bit i), wavefront-uniform
};

// retained rows of pivot positions q0 .. q0+3 of round r (pivot word r/2).  The
// loads are unconditional (in-bounds addresses) and their values are masked only
// where they are used, so that they stay in flight across the preceding round.
__device__ __forceinline__ void load_group(const LargeShared& L, const uint64_t* B, int W, int fw, int n, int r,
                                           int wave, int lane, GroupRows& gr) {
    const int pw = r >> 1, q0 = 32 * (r & 1) + 4 * wave;
    gr.present = static_cast<uint32_t>((L.pm[pw] >> q0) & 15ull);
    const int fl = lane < fw ? lane : 0, zl = fw + (lane & 1);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint64_t* row = B + static_cast<int64_t>(prio_slot(64 * pw + q0 + i, n)) * W;
        gr.f[i] = row[fl];
        gr.z[i] = row[zl];
    }
}

// the 16 XOR combinations of four rows, entry e = rows of the set bits of e
__device__ __forceinline__ void write_table(LargeShared& L, int base, const GroupRows& gr, int lane, bool act) {
    const uint64_t f1 = (act && (gr.present & 1u)) ? gr.f[0] : 0ull, f2 = (act && (gr.present & 2u)) ? gr.f[1] : 0ull;
    const uint64_t f4 = (act && (gr.present & 4u)) ? gr.f[2] : 0ull, f8 = (act && (gr.present & 8u)) ? gr.f[3] : 0ull;
    const uint64_t f3 = f1 ^ f2, f5 = f4 ^ f1, f6 = f4 ^ f2, f7 = f6 ^ f1;
    {  // inactive lanes get zero entries, so that adding an entry leaves them unchanged
        uint64_t (*T)[64] = L.tf + base;
        T[0][lane] = 0ull;
        T[1][lane] = f1;
        T[2][lane] = f2;
        T[3][lane] = f3;
        T[4][lane] = f4;
        T[5][lane] = f5;
        T[6][lane] = f6;
        T[7][lane] = f7;
        T[8][lane] = f8;
        T[9][lane] = f8 ^ f1;
        T[10][lane] = f8 ^ f2;
        T[11][lane] = f8 ^ f3;
        T[12][lane] = f8 ^ f4;
        T[13][lane] = f8 ^ f5;
        T[14][lane] = f8 ^ f6;
        T[15][lane] = f8 ^ f7;
    }
    // output words: lane l < 32 writes word l & 1 of entry l >> 1
    const int e = lane >> 1, q = lane & 1;
    uint64_t z = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint64_t zi = ((gr.present >> i) & 1u) ? (q ? readlane64(gr.z[i], 1) : readlane64(gr.z[i], 0)) : 0ull;
        z ^= ((e >> i) & 1) ? zi : 0ull;
    }
    if (lane < 32) L.tz[base + e][q] = z;
}

// reduce the wavefront's block rows by the tables of round r in buffer buf
__device__ __forceinline__ void apply_round(const LargeShared& L, int r, int buf, uint64_t (&acc)[kLgSlots],
                                            uint64_t& yv, int lane, bool act) {
    const int pw = r >> 1, h = r & 1;
    const uint64_t pmw = L.pm[pw];
    uint32_t s[kLgSlots];
#pragma unroll
    for (int k = 0; k < kLgSlots; ++k) s[k] = static_cast<uint32_t>((readlane64(acc[k], pw) & pmw) >> (32 * h));
    const uint32_t sy = spread_slots(s, lane);
    const uint32_t present = static_cast<uint32_t>(pmw >> (32 * h));
#pragma unroll
    for (int g = 0; g < kLgRoundTables; g += 2) {  // two tables at a time, one three-input XOR
        if (((present >> (4 * g)) & 0xffu) == 0) continue;
        const int b0 = buf * kLgBuf + kLgEnt * g, b1 = b0 + kLgEnt;
        // all reads issued before the first use (entries are zero in the inactive lanes,
        // and every table of the round is written, absent rows as zero)
        uint64_t t0[kLgSlots], t1[kLgSlots];
#pragma unroll
        for (int k = 0; k < kLgSlots; ++k) {
            t0[k] = L.tf[b0 + ((s[k] >> (4 * g)) & 15u)][lane];
            t1[k] = L.tf[b1 + ((s[k] >> (4 * g + 4)) & 15u)][lane];
        }
        const uint64_t ty0 = L.tz[b0 + ((sy >> (4 * g)) & 15u)][lane & 1];
        const uint64_t ty1 = L.tz[b1 + ((sy >> (4 * g + 4)) & 15u)][lane & 1];
#pragma unroll
        for (int k = 0; k < kLgSlots; ++k) acc[k] = xor3(acc[k], t0[k], t1[k]);
        yv = xor3(yv, ty0, ty1);
    }
}

// new pivot of a row (lane = word): highest-priority set feature, the constant last; -1 if none
__device__ __forceinline__ int row_pivot(uint64_t F, int n, int cw, uint64_t cbit, int lane) {
    const uint64_t Fx = (lane == cw) ? (F & ~cbit) : F;
    const uint64_t nzx = __ballot(Fx != 0);
    if (nzx) {
        const int top = msb64(nzx);
        return 64 * top + msb64(readlane64(Fx, top));
    }
    return (readlane64(F, cw) & cbit) ? n : -1;
}

// G workgroups may fit one context together (member g): each reduces the block
// by the tables of its own pivot words and the partial sums are exchanged
// through the context's tables buffer (free until the outputs are written); the
// in-block elimination runs in every member on identical data; each member
// back-substitutes and stores the rows of its own pivot words; member 0 writes
// the outputs.
__device__ __forceinline__ void fit_ctx_large(const FitArgs& a, const CtxDesc& ds, LargeShared& L, int G, int g,
                                              int* bar, int& epoch) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = ds.c;
    const int n = ds.n;
    const int fw = feat_words(n), W = fw + F2_Y_WORDS, d = n + 1;
    const int64_t m = ds.m;
    const uint64_t* R = a.rows + ds.row0;
    const uint64_t tmask = top_mask(n, fw);
    const uint64_t lmask = lane < fw ? (lane == fw - 1 ? tmask : ~0ull) : 0ull;  // valid bits of word `lane`
    const int cw = n >> 6;
    const uint64_t cbit = 1ull << (n & 63);
    uint64_t* B = a.basis + a.basis_off[c];
    constexpr long long kNone = 0x7fffffffffffffffll;

    if (tid < 64) L.pm[tid] = 0;
    if (tid == 0) {
        L.contra = 0;
        L.timeout = 0;
        L.firstMin = kNone;
    }
    int rank = 0;
    int64_t b0 = 0;
    for (int blk = 0; b0 < m && rank < d; b0 += kLargeRows, ++blk) {
        const int nb = static_cast<int>((m - b0) < kLargeRows ? (m - b0) : kLargeRows);
        if (tid < 64) {
            L.npm[tid] = 0;
            L.rowPiv[tid] = -1;
        }
        // block rows: slot k of wavefront w is block row 8w + k
        uint64_t acc[kLgSlots], yv;
#pragma unroll
        for (int k = 0; k < kLgSlots; ++k) {
            const int i = kLgSlots * wave + k;
            acc[k] = (i < nb && lane < fw) ? (R[(b0 + i) * W + lane] & lmask) : 0ull;
        }
        {
            const int i = kLgSlots * wave + (lane >> 1);
            yv = (lane < 2 * kLgSlots && i < nb) ? R[(b0 + i) * W + fw + (lane & 1)] : 0ull;
        }
        // drain the row loads here: left outstanding, they would make every later wait
        // inside the reduce loop a wait for all memory operations
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        // active lanes: feature words with at least one column that is not a retained pivot
        const bool act = lane < fw && (L.pm[lane] | ~lmask) != ~0ull;

        // (1) block reduce against the retained basis, half a pivot word per round
        if (rank > 0) {
            GroupRows gA, gB;
            int r = next_round(L, fw, -1, G, g);
            if (r >= 0) {
                load_group(L, B, W, fw, n, r, wave, lane, gA);
                write_table(L, kLgEnt * wave, gA, lane, act);
            }
            int rn = r >= 0 ? next_round(L, fw, r, G, g) : -1;
            if (rn >= 0) load_group(L, B, W, fw, n, rn, wave, lane, gA);
            __syncthreads();
            int buf = 0;
            while (r >= 0) {
                const int rnn = rn >= 0 ? next_round(L, fw, rn, G, g) : -1;
                if (rnn >= 0) load_group(L, B, W, fw, n, rnn, wave, lane, gB);
                apply_round(L, r, buf, acc, yv, lane, act);
                if (rn >= 0) write_table(L, (buf ^ 1) * kLgBuf + kLgEnt * wave, gA, lane, act);
                __syncthreads();
                r = rn;
                rn = rnn;
                gA = gB;
                buf ^= 1;
            }
            if (G > 1) {
                // member o holds X + P_o (X the unreduced rows, P_o its tables' sum); the
                // reduced rows are X + sum P_o = X + sum (X + P_o) for an even G
                uint64_t* X = a.tables + a.basis_off[c];
                const int64_t xs = static_cast<int64_t>(kLargeRows) * W;  // one member's block
                uint64_t* mine = X + ((blk & 1) * G + g) * xs;
                const int yi = kLgSlots * wave + (lane >> 1);
#pragma unroll
                for (int k = 0; k < kLgSlots; ++k)
                    if (act) put_dev(mine + (kLgSlots * wave + k) * W + lane, acc[k]);
                if (lane < 2 * kLgSlots) put_dev(mine + yi * W + fw + (lane & 1), yv);
                group_barrier(bar, epoch, G, a.spin_limit, &L.timeout, false);
                // reads past a partial's rows land in another partial or past the
                // resource (zero); their values are masked off
                const __amdgpu_buffer_rsrc_t xr = dev_rsrc(X + (blk & 1) * G * xs, static_cast<uint32_t>(8 * G * xs));
                for (int o = 0; o < G; ++o) {
                    if (o == g) continue;
                    const uint32_t ob = static_cast<uint32_t>(o * xs);
                    uint64_t v[kLgSlots];
#pragma unroll
                    for (int k = 0; k < kLgSlots; ++k) v[k] = get_dev(xr, ob + (kLgSlots * wave + k) * W + lane);
                    const uint64_t vy = get_dev(xr, ob + yi * W + fw + (lane & 1));
#pragma unroll
                    for (int k = 0; k < kLgSlots; ++k) acc[k] ^= act ? v[k] : 0ull;
                    yv ^= lane < 2 * kLgSlots ? vy : 0ull;
                }
#pragma unroll
                for (int k = 0; k < kLgSlots; ++k) {  // + X, reloaded
                    const int i = kLgSlots * wave + k;
                    if (act && i < nb) acc[k] ^= R[(b0 + i) * W + lane] & lmask;
                }
                if (lane < 2 * kLgSlots && yi < nb) yv ^= R[(b0 + yi) * W + fw + (lane & 1)];
            }
#pragma unroll
            for (int k = 0; k < kLgSlots; ++k) acc[k] = act ? acc[k] : 0ull;
        }

        // (2) in-block elimination.  Rows whose features reduced to zero are
        //     redundant or contradictory whatever the other block rows hold.
        int ncon = 0;
        long long firstc = kNone;
        unsigned long long mine = 0;
#pragma unroll
        for (int k = 0; k < kLgSlots; ++k) {
            const int i = kLgSlots * wave + k;
            if (__ballot(acc[k] != 0)) {
                mine |= 1ull << k;
            } else if (i < nb) {
                if ((readlane64(yv, 2 * k) | readlane64(yv, 2 * k + 1)) != 0) {
                    ++ncon;
                    if (firstc == kNone) firstc = b0 + i;
                }
            }
        }
        for (int ph = 0; ph < kLargeWaves; ++ph) {
            const int bq = ph & 1;
            const int tb = kLgSlots * bq;  // this phase's published rows in tf (the reduce is done with it)
            if (wave == ph) {  // this wavefront's rows in order; earlier wavefronts' pivots already applied
                unsigned newSlots = 0;
#pragma unroll
                for (int s = 0; s < kLgSlots; ++s) {
                    if (!((mine >> s) & 1ull)) continue;
                    const int i = kLgSlots * ph + s;
                    const uint64_t F = acc[s];
                    const int p = row_pivot(F, n, cw, cbit, lane);
                    const uint64_t Y0 = readlane64(yv, 2 * s), Y1 = readlane64(yv, 2 * s + 1);
                    if (p < 0) {  // dependent on the earlier rows: redundant, or contradictory
                        if ((Y0 | Y1) != 0) {
                            ++ncon;
                            if (firstc > b0 + i) firstc = b0 + i;
                        }
                        continue;
                    }
                    const int pw = p >> 6, pb = p & 63;
                    // bit p of the wavefront's rows: gathered in every lane, read from lane pw
                    uint32_t bits = 0;
#pragma unroll
                    for (int t = 0; t < kLgSlots; ++t) bits |= static_cast<uint32_t>((acc[t] >> pb) & 1ull) << t;
                    const uint32_t hits = __builtin_amdgcn_readlane(bits, pw) & ~(1u << s);
#pragma unroll
                    for (int t = 0; t < kLgSlots; ++t) acc[t] = xor_and(acc[t], ((hits >> t) & 1u) ? ~0u : 0u, F);
                    uint32_t em = hits;  // slot t -> output-word lanes 2t, 2t+1
                    em = (em | (em << 4)) & 0x0f0fu;
                    em = (em | (em << 2)) & 0x3333u;
                    em = (em | (em << 1)) & 0x5555u;
                    em |= em << 1;
                    yv = xor_and(yv, lanes_of(em, lane), (lane & 1) ? Y1 : Y0);
                    newSlots |= 1u << s;
                    if (lane == 0) {
                        L.rowPiv[i] = p;
                        atomicOr(reinterpret_cast<unsigned long long*>(&L.npm[pw]), 1ull << pb);
                    }
                }
                // publish the new rows, now fully reduced among themselves, in slot order
                const int np = __popc(newSlots);
#pragma unroll
                for (int s = 0; s < kLgSlots; ++s) {
                    if (!((newSlots >> s) & 1u)) continue;
                    const int q = __popc(newSlots & ((1u << s) - 1u));
                    L.tf[tb + q][lane] = acc[s];
                    if ((lane >> 1) == s) L.tz[tb + q][lane & 1] = yv;
                    if (lane == 0) L.pubP[bq][q] = L.rowPiv[kLgSlots * ph + s];
                }
                if (lane == 0) L.pubN[bq] = np;
            }
            __syncthreads();
            const int np = L.pubN[bq];
            if (wave != ph && np > 0) {  // the published rows: selection bits at their pivots, then the rows
                const int pk = lane < np ? L.pubP[bq][lane] : 0;
                const int pkw = pk >> 6, pkb = pk & 63;
                uint32_t sel[kLgSlots];
                uint64_t wv[kLgSlots];
#pragma unroll
                for (int k = 0; k < kLgSlots; ++k) wv[k] = shfl64(acc[k], pkw);
#pragma unroll
                for (int k = 0; k < kLgSlots; ++k)
                    sel[k] = static_cast<uint32_t>(__ballot(lane < np && ((wv[k] >> pkb) & 1ull)));
                const uint32_t sy = spread_slots(sel, lane);
                for (int q = 0; q < np; ++q) {
                    const uint64_t Fv = L.tf[tb + q][lane];
                    const uint64_t Zv = L.tz[tb + q][lane & 1];
#pragma unroll
                    for (int k = 0; k < kLgSlots; ++k) acc[k] = xor_and(acc[k], ((sel[k] >> q) & 1u) ? ~0u : 0u, Fv);
                    yv = xor_and(yv, 0u - ((sy >> q) & 1u), Zv);
                }
            }
        }
        if (lane == 0 && ncon) {
            atomicAdd(&L.contra, ncon);
            atomicMin(&L.firstMin, firstc);
        }
        __syncthreads();

        // (3) new rows in descending priority: position = new pivots above it
        if (wave == 0) {
            const uint64_t v = L.npm[lane] & ((lane == cw) ? ~cbit : ~0ull);
            const int cnt = lane < fw ? __popcll(v) : 0;
            int x = cnt;  // inclusive scan from the top word down
            for (int o = 1; o < 64; o <<= 1) {
                const int t = __shfl_down(x, o);
                if (lane + o < 64) x += t;
            }
            L.above[lane] = x - cnt;
            const int total = __shfl(x, 0) + ((L.npm[cw] & cbit) ? 1 : 0);
            if (lane == 0) L.nnew = total;
        }
        __syncthreads();
        const int K = L.nnew;
        if (K > 0) {
#pragma unroll
            for (int k = 0; k < kLgSlots; ++k) {
                const int i = kLgSlots * wave + k;
                const int p = L.rowPiv[i];
                if (p < 0) continue;
                int pos = K - 1;
                if (p != n) {
                    uint64_t v = L.npm[p >> 6];
                    if ((p >> 6) == cw) v &= ~cbit;
                    v &= (p & 63) == 63 ? 0ull : (~0ull << ((p & 63) + 1));
                    pos = L.above[p >> 6] + __popcll(v);
                }
                const int e = kLgEnt * (pos >> 2) + (1 << (pos & 3));
                L.tf[e][lane] = acc[k];
                if ((lane >> 1) == k) L.tz[e][lane & 1] = yv;
                if (lane == 0) L.nsorted[pos] = p;
            }
            __syncthreads();
            // complete the tables: groups w and w + 8, missing rows of the last group are zero
            const int NG = (K + 3) >> 2;
            for (int g = wave; g < NG; g += kLargeWaves) {
                GroupRows gr;
                gr.present = 0;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const bool has = 4 * g + q < K;
                    gr.present |= has ? (1u << q) : 0u;
                    gr.f[q] = has ? L.tf[kLgEnt * g + (1 << q)][lane] : 0ull;
                    gr.z[q] = has ? L.tz[kLgEnt * g + (1 << q)][lane & 1] : 0ull;
                }
                __builtin_amdgcn_wave_barrier();
                write_table(L, kLgEnt * g, gr, lane, true);
            }
            __syncthreads();

            // (3') clear the new pivots from the retained rows: positions wave, wave + 8, ...
            //      of every retained pivot word, one register per row, the next word's rows
            //      loaded while this word's are updated
            const int pk = lane < K ? L.nsorted[lane] : 0;
            const int pkw = pk >> 6, pkb = pk & 63;
            const uint64_t mineBits = 0x0101010101010101ull << wave;
            auto next_word = [&](int pw) {  // this member's pivot words only
                for (++pw; pw < fw; ++pw)
                    if ((pw & (G - 1)) == g && (L.pm[pw] & mineBits)) return pw;
                return -1;
            };
            auto load_rows = [&](int pw, uint64_t (&Bv)[kLgSlots], uint64_t& yb) {  // raw: masked where used
#pragma unroll
                for (int q = 0; q < kLgSlots; ++q) {
                    const int b = wave + kLargeWaves * q;
                    Bv[q] = B[static_cast<int64_t>(prio_slot(64 * pw + b, n)) * W + (lane < fw ? lane : 0)];
                }
                const int b = wave + kLargeWaves * ((lane >> 1) & 7);
                yb = B[static_cast<int64_t>(prio_slot(64 * pw + b, n)) * W + fw + (lane & 1)];
            };
            uint64_t Bv[kLgSlots], yb, Bn[kLgSlots], ybn;
            int pw = next_word(-1);
            if (pw >= 0) load_rows(pw, Bv, yb);
            while (pw >= 0) {
                const int pwn = next_word(pw);
                if (pwn >= 0) load_rows(pwn, Bn, ybn);
                const uint64_t pmw = L.pm[pw];
#pragma unroll
                for (int q = 0; q < kLgSlots; ++q) Bv[q] = (act && ((pmw >> (wave + kLargeWaves * q)) & 1ull)) ? Bv[q] : 0ull;
                yb = (lane < 2 * kLgSlots && ((pmw >> (wave + kLargeWaves * (lane >> 1))) & 1ull)) ? yb : 0ull;
                uint64_t sv[kLgSlots], wv[kLgSlots];
#pragma unroll
                for (int q = 0; q < kLgSlots; ++q) wv[q] = shfl64(Bv[q], pkw);  // all exchanges in flight together
#pragma unroll
                for (int q = 0; q < kLgSlots; ++q) sv[q] = __ballot(lane < K && ((wv[q] >> pkb) & 1ull));
                const uint64_t svy = spread_slots(sv, lane);
                for (int g = 0; g < NG; g += 2) {  // two tables at a time (the second may not exist)
                    const bool two = g + 1 < NG;
                    uint64_t t0[kLgSlots], t1[kLgSlots];
#pragma unroll
                    for (int q = 0; q < kLgSlots; ++q) {
                        t0[q] = L.tf[kLgEnt * g + ((sv[q] >> (4 * g)) & 15u)][lane];
                        t1[q] = two ? L.tf[kLgEnt * (g + 1) + ((sv[q] >> (4 * g + 4)) & 15u)][lane] : 0ull;
                    }
                    const uint64_t ty0 = L.tz[kLgEnt * g + ((svy >> (4 * g)) & 15u)][lane & 1];
                    const uint64_t ty1 = two ? L.tz[kLgEnt * (g + 1) + ((svy >> (4 * g + 4)) & 15u)][lane & 1] : 0ull;
#pragma unroll
                    for (int q = 0; q < kLgSlots; ++q) Bv[q] = xor3(Bv[q], t0[q], t1[q]);
                    yb = xor3(yb, ty0, ty1);
                }
#pragma unroll
                for (int q = 0; q < kLgSlots; ++q) {
                    const int b = wave + kLargeWaves * q;
                    if (!((pmw >> b) & 1ull)) continue;
                    uint64_t* row = B + static_cast<int64_t>(prio_slot(64 * pw + b, n)) * W;
                    if (act) row[lane] = Bv[q];
                    if ((lane >> 1) == q) row[fw + (lane & 1)] = yb;
                }
                pw = pwn;
#pragma unroll
                for (int q = 0; q < kLgSlots; ++q) Bv[q] = Bn[q];
                yb = ybn;
            }
            // (4) insert the new rows at their priority slots (every word: fresh slots)
            for (int pos = wave; pos < K; pos += kLargeWaves) {
                if (((L.nsorted[pos] >> 6) & (G - 1)) != g) continue;  // another member's pivot word
                const int e = kLgEnt * (pos >> 2) + (1 << (pos & 3));
                uint64_t* row = B + static_cast<int64_t>(prio_slot(L.nsorted[pos], n)) * W;
                if (lane < fw) row[lane] = L.tf[e][lane];
                if (lane < 2) row[fw + lane] = L.tz[e][lane];
            }
            __syncthreads();
            if (tid < 64) L.pm[tid] |= L.npm[tid];
        }
        __syncthreads();
        rank += K;
    }

    if (G > 1) group_barrier(bar, epoch, G, a.spin_limit, &L.timeout);  // every member's basis rows written
    if (b0 < m) {
        // full rank: every remaining row lies in the span; its residual is y + M phi
        // (members of a group take every G-th 512-row chunk)
        uint64_t (*sZ)[2] = reinterpret_cast<uint64_t (*)[2]>(&L.tf[0][0]);
        long long firstCons = kNone;
        int ncons = 0;
        for (int jj = tid; jj < d; jj += kLargeThreads) {
            const uint64_t* row = B + static_cast<int64_t>(prio_slot(jj, n)) * W;
            sZ[jj][0] = row[fw];
            sZ[jj][1] = row[fw + 1];
        }
        __syncthreads();
        for (int64_t r0 = b0 + static_cast<int64_t>(g) * kLargeThreads; r0 < m; r0 += static_cast<int64_t>(G) * kLargeThreads) {
            const int64_t i = r0 + tid;
            if (i < m) {
                const uint64_t* row = R + i * W;
                uint64_t z0 = row[fw], z1 = row[fw + 1];
                for (int w = 0; w < fw; ++w) {
                    uint64_t v = row[w];
                    if (w == fw - 1) v &= tmask;
                    while (v) {
                        const int jj = 64 * w + ffs64(v);
                        v &= v - 1;
                        z0 ^= sZ[jj][0];
                        z1 ^= sZ[jj][1];
                    }
                }
                if (z0 | z1) {
                    ++ncons;
                    if (firstCons == kNone) firstCons = i;
                }
            }
        }
        if (G == 1) {
            if (ncons) {
                atomicAdd(&L.contra, ncons);
                atomicMin(&L.firstMin, firstCons);
            }
            __syncthreads();
        } else {  // members' counts through the exchange area, combined by member 0
            __shared__ int sCnt;
            __shared__ long long sFirst;
            if (tid == 0) {
                sCnt = 0;
                sFirst = kNone;
            }
            __syncthreads();
            if (ncons) {
                atomicAdd(&sCnt, ncons);
                atomicMin(&sFirst, firstCons);
            }
            __syncthreads();
            int64_t* X = reinterpret_cast<int64_t*>(a.tables + a.basis_off[c]);
            if (tid == 0) {
                X[2 * g] = sCnt;
                X[2 * g + 1] = sFirst;
            }
            group_barrier(bar, epoch, G, a.spin_limit, &L.timeout);
            if (g == 0 && tid == 0) {
                for (int o = 1; o < G; ++o) {
                    L.contra += static_cast<int>(X[2 * o]);
                    if (X[2 * o + 1] < L.firstMin) L.firstMin = X[2 * o + 1];
                }
                L.contra += sCnt;
                if (sFirst < L.firstMin) L.firstMin = sFirst;
            }
            __syncthreads();
        }
    }
    // the rank as the pivot set holds it: equal to the running count unless a
    // timed-out exchange left members with different data, and then it keeps
    // every output position below d
    if (tid == 0) L.nnew = 0;
    __syncthreads();
    if (wave == 0 && lane < fw) atomicAdd(&L.nnew, __popcll(L.pm[lane] & lmask));
    __syncthreads();
    rank = L.nnew;
    if (g != 0) {  // member 0 writes the outputs; the others only report a wait that gave up
        if (tid == 0 && L.timeout) atomicOr(&a.ctx_flags[c], F2_CTX_SYNC_TIMEOUT);
        return;
    }

    // outputs: canonical map and encode table from the slots, then compaction into descending priority
    const int64_t po = a.piv_off[c], mo = a.map_off[c];
    for (int jj = tid; jj < d; jj += kLargeThreads) {
        const bool present = (L.pm[jj >> 6] >> (jj & 63)) & 1ull;
        const uint64_t* row = B + static_cast<int64_t>(prio_slot(jj, n)) * W;
        a.maps[mo + 2 * jj] = present ? row[fw] : 0ull;
        a.maps[mo + 2 * jj + 1] = present ? row[fw + 1] : 0ull;
    }
    {  // parity-check rows of the free columns: per word pair (w, v), taken by wavefront
       // v mod 8, a bit-matrix transpose of word w of the retained rows of pivots
       // 64 v .. 64 v + 63 (zero for free columns) gives lane f word v of the row of
       // free column 64 w + f
        uint64_t* H = a.tables + a.basis_off[c];
        if (has_parity_rows(d, rank)) {
            const uint64_t lane_lt = (1ull << lane) - 1;
            int base = 0;  // free columns in the words before w
            for (int w = 0; w < fw; ++w) {
                const uint64_t fr = ~L.pm[w] & (w == fw - 1 ? tmask : ~0ull);
                if (!fr) continue;  // no free column in this word
                const bool mine = (fr >> lane) & 1ull;
                const int64_t i = base + __popcll(fr & lane_lt);
                for (int v = wave; v < fw; v += kLargeWaves) {
                    const int p = 64 * v + lane;
                    const bool piv = (L.pm[v] >> lane) & 1ull;
                    const uint64_t col = transpose64(piv ? B[static_cast<int64_t>(prio_slot(p, n)) * W + w] : 0ull, lane);
                    if (mine) H[i * fw + v] = col | (v == w ? (1ull << lane) : 0ull);
                }
                base += __popcll(fr);
            }
        }
    }
    // pivots, and the basis rows moved from their slots to positions 0 .. rank-1: the
    // row of slot t goes to position (present slots before t) <= t, so slots are moved
    // in increasing order, 64 at a time (read all, barrier, write all)
    if (wave == 0) {  // present slots in words above w (slot order = descending feature index, constant last)
        const uint64_t v = L.pm[lane] & ((lane == cw) ? ~cbit : ~0ull);
        const int cnt = lane < fw ? __popcll(v) : 0;
        int x = cnt;
        for (int o = 1; o < 64; o <<= 1) {
            const int t = __shfl_down(x, o);
            if (lane + o < 64) x += t;
        }
        L.above[lane] = x - cnt;
    }
    __syncthreads();
    if (rank < d) {
        for (int t0 = 0; t0 < d; t0 += kLargeRows) {
            uint64_t w0[kLgSlots], w1[kLgSlots];
            int kk[kLgSlots];
#pragma unroll
            for (int q = 0; q < kLgSlots; ++q) {
                const int t = t0 + kLgSlots * wave + q;
                const int pt = t < d ? slot_pivot(t, n) : 0;
                const bool present = t < d && ((L.pm[pt >> 6] >> (pt & 63)) & 1ull);
                kk[q] = -1;
                w0[q] = w1[q] = 0;
                if (present) {
                    const uint64_t* row = B + static_cast<int64_t>(t) * W;
                    if (lane < W) w0[q] = row[lane];
                    if (64 + lane < W) w1[q] = row[64 + lane];
                    if (pt == n) {
                        kk[q] = rank - 1;
                    } else {
                        uint64_t v = L.pm[pt >> 6];
                        if ((pt >> 6) == cw) v &= ~cbit;
                        v &= (pt & 63) == 63 ? 0ull : (~0ull << ((pt & 63) + 1));
                        kk[q] = L.above[pt >> 6] + __popcll(v);
                    }
                }
            }
            __syncthreads();
#pragma unroll
            for (int q = 0; q < kLgSlots; ++q) {
                if (kk[q] < 0) continue;
                uint64_t* out = B + static_cast<int64_t>(kk[q]) * W;
                if (lane < W) out[lane] = w0[q];
                if (64 + lane < W) out[64 + lane] = w1[q];
            }
            __syncthreads();
        }
    }
    for (int t = tid; t < d; t += kLargeThreads) {  // full rank: every slot present, position = slot
        const int pt = slot_pivot(t, n);
        if (!((L.pm[pt >> 6] >> (pt & 63)) & 1ull)) continue;
        int k = rank - 1;
        if (pt != n) {
            uint64_t v = L.pm[pt >> 6];
            if ((pt >> 6) == cw) v &= ~cbit;
            v &= (pt & 63) == 63 ? 0ull : (~0ull << ((pt & 63) + 1));
            k = L.above[pt >> 6] + __popcll(v);
        }
        a.pivots[po + k] = pt;
    }
    if (tid == 0) {
        a.rank[c] = rank;
        a.n_contra[c] = L.contra;
        a.first_contra[c] = L.firstMin == kNone ? -1 : L.firstMin;
        // OR: the other members may report a timeout (the plan cleared the word)
        atomicOr(&a.ctx_flags[c], (L.contra ? F2_CTX_CONTRADICTION : 0u) | (L.timeout ? F2_CTX_SYNC_TIMEOUT : 0u));
    }
    __syncthreads();
}

// contexts of classes 1-2 (fw <= 8 beyond the register kernel): pivot-indexed LDS
// basis, kPivWaves wavefronts per workgroup, several workgroups per compute unit.
// The list (largest first) is taken greedily: workgroup g starts at position g,
// then each takes the next free position from a counter as it finishes one (the
// fetch is issued when a context starts, so its latency hides behind the work).
__global__ __launch_bounds__(kPivThreads, 3) void k_fit_piv(FitArgs a) {
    __shared__ PivShared S;
    __shared__ int sNext;
    const int lo = a.plan[kClsPiv], cnt = a.plan[kClsPivLong + 1] - lo;
    for (int i = static_cast<int>(blockIdx.x); i < cnt;) {
        const int c = __builtin_amdgcn_readfirstlane(a.plan[kPlanHead + lo + i]);
        int next = 0;
        if (threadIdx.x == 0) next = atomicAdd(&a.plan[kPivNext], 1) + static_cast<int>(gridDim.x);
        const CtxDesc ds = readlane_desc(load_desc(a, c), 0);
        switch (feat_words(ds.n)) {
            case 1: fit_ctx_piv<1, kPivWaves>(a, ds, S); break;
            case 2: fit_ctx_piv<2, kPivWaves>(a, ds, S); break;
            case 3: case 4: fit_ctx_piv<4, kPivWaves>(a, ds, S); break;
            default: fit_ctx_piv<8, kPivWaves>(a, ds, S); break;
        }
        if (threadIdx.x == 0) sNext = next;
        __syncthreads();
        i = sNext;
        __syncthreads();
    }
}

// Small batches (up to kSmallBatch contexts, declared widths below 512): one
// launch, one workgroup of 8 wavefronts per context, the context's class choosing
// the path (one wavefront for the register basis, all eight for the LDS basis).
// No plan: its two launches would cost more than the fit of a batch this size,
// and one workgroup per context needs no load balance.  Invalid contexts, and any
// wider than the declared bound, are flagged here.
constexpr int kSmallBatch = 64;
union SmallShared {
    struct {
        uint64_t rec[64 * kRegMaxFW * kRecWords];
        int16_t pos[64 * kRegMaxFW];
    } reg;
    PivShared piv;
};

__global__ __launch_bounds__(kLargeThreads) void k_fit_small(FitArgs a) {
    __shared__ SmallShared U;
    const CtxDesc ds = readlane_desc(load_desc(a, blockIdx.x), 0);
    if (ds.c < 0) return;
    if (ds.bad) {
        if (threadIdx.x == 0) write_bad_context(a, ds);
        return;
    }
    const int fw = feat_words(ds.n);
    switch (fit_class(ds)) {
        case kClsReg:
            if (threadIdx.x < 64) {
                if (fw == 1) fit_ctx_reg<1>(a, ds, U.reg.rec, U.reg.pos);
                else if (fw == 2) fit_ctx_reg<2>(a, ds, U.reg.rec, U.reg.pos);
                else fit_ctx_reg<3>(a, ds, U.reg.rec, U.reg.pos);
            }
            break;
        case kClsLarge:  // not launched for a batch that may hold one (the bound is below 512)
            break;
        default:
            switch (fw) {
                case 1: fit_ctx_piv<1, kLargeWaves>(a, ds, U.piv); break;
                case 2: fit_ctx_piv<2, kLargeWaves>(a, ds, U.piv); break;
                case 3: case 4: fit_ctx_piv<4, kLargeWaves>(a, ds, U.piv); break;
                default: fit_ctx_piv<8, kLargeWaves>(a, ds, U.piv); break;
            }
            break;
    }
}

// Wide contexts (class 3): with few of them (as many as a quarter of the
// workgroups or fewer) each is fitted by a group of 4 workgroups, by 2 with up to
// half, else by one.  Under a cooperative launch every workgroup is resident,
// which the group barriers need; otherwise groups are single workgroups.  A
// group's workgroups are blockIdx values congruent mod 8, which the dispatcher
// places on one die (shared L2 for the exchange).
__global__ __launch_bounds__(kLargeThreads) void k_fit_wide(FitArgs a) {
    __shared__ LargeShared U;
    const int nl = a.plan[kClsLarge + 1] - a.plan[kClsLarge];
    const int nwg = static_cast<int>(gridDim.x);
    int G = 1;
    if (a.coop && nwg % 32 == 0 && nwg / 4 <= kMaxGroups && 4 * nl <= nwg) G = 4;
    else if (a.coop && nwg % 16 == 0 && nwg / 2 <= kMaxGroups && 2 * nl <= nwg) G = 2;
    const int x = static_cast<int>(blockIdx.x), idx = x / 8;
    const int g = idx % G, grp = (x % 8) + 8 * (idx / G), ngrp = nwg / G;
    int epoch = 0;
    for (int i = 0;; ++i) {
        const int c = __builtin_amdgcn_readfirstlane(class_ctx(a, kClsLarge, i, -1, ngrp, grp));
        if (c < 0) break;
        fit_ctx_large(a, readlane_desc(load_desc(a, c), 0), U, G, g, a.plan + kBarHead + grp, epoch);
    }
}

// ---------------------------------------------------------------------------
// encode (Sec. 2.3), one lane per query, queries in any order: the table
// entries of the set bits of phi = [x | 1] are XORed (the constant column is
// always set).  The z part is T(phi) = M phi; the h part is the reduction
// residual on the free columns and must vanish for phi to lie in the span.
// ---------------------------------------------------------------------------

// x words of a query, with bits past the stride read as zero
template <int SMAX>
struct QueryX {
    uint64_t xr[SMAX > 0 ? SMAX : 1];
    const uint64_t* xq;
    int S;
    __device__ __forceinline__ void load(const uint64_t* p, int stride) {
        xq = p;
        S = stride;
        if constexpr (SMAX > 0) {
#pragma unroll
            for (int k = 0; k < SMAX; ++k) xr[k] = k < S ? p[k] : 0ull;
        }
    }
    __device__ __forceinline__ uint64_t word(int w) const {
        if constexpr (SMAX > 0) {
            uint64_t v = 0;
#pragma unroll
            for (int k = 0; k < SMAX; ++k) v = (w == k) ? xr[k] : v;
            return v;
        } else {
            return w < S ? xq[w] : 0ull;
        }
    }
};

// any x bit at or above the width n: outside the context's ambient space
template <int SMAX>
__device__ __forceinline__ bool outside_width(const QueryX<SMAX>& x, int n) {
    bool outside = false;
    for (int w = (n >> 6); w < x.S; ++w) {
        const uint64_t v = x.word(w);
        const int lo = 64 * w;
        outside |= (lo >= n) ? (v != 0) : ((v >> (n - lo)) != 0);
    }
    return outside;
}

struct alignas(16) Word2 {
    uint64_t x, y;
};

// T(phi): XOR of the map columns of the set bits, four gathers in flight
template <int SMAX>
__device__ __forceinline__ void map_gather(const uint64_t* M, int n, const QueryX<SMAX>& x, uint64_t& z0,
                                           uint64_t& z1) {
    const Word2 zc = *reinterpret_cast<const Word2*>(M + 2 * n);  // constant column: always set
    z0 = zc.x;
    z1 = zc.y;
    const int fw = feat_words(n);
    const int xw = x.S < fw ? x.S : fw;
    for (int w = 0; w < xw; ++w) {
        const uint64_t v = x.word(w);
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            uint32_t u = half ? static_cast<uint32_t>(v >> 32) : static_cast<uint32_t>(v);
            const uint64_t* Mh = M + 2 * (64 * w + 32 * half);
            while (u) {  // a missing gather re-reads the first column and is masked off
                int jj[4];
                uint64_t mk[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    mk[k] = u ? ~0ull : 0ull;
                    jj[k] = u ? __builtin_ctz(u) : jj[0];
                    u &= u - 1;
                }
                Word2 a[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) a[k] = *reinterpret_cast<const Word2*>(Mh + 2 * jj[k]);
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    z0 ^= a[k].x & mk[k];
                    z1 ^= a[k].y & mk[k];
                }
            }
        }
    }
}

// support test: even overlap of phi = [x | 1] with every parity-check row
// (all rows are read, several at a time: no early exit to serialise the loads)
template <int SMAX>
__device__ __forceinline__ bool parity_ok(const uint64_t* H, int t, int n, const QueryX<SMAX>& x) {
    const int fw = feat_words(n), cw = n >> 6;
    const uint64_t cbit = 1ull << (n & 63);
    int odd = 0;  // bit 0 of an OR of popcounts is the OR of their parities
    if (fw == 1) {
        const uint64_t q = x.word(0) | cbit;
        int f = 0;
        for (; f + 4 <= t; f += 4) {
            const uint64_t h0 = H[f], h1 = H[f + 1], h2 = H[f + 2], h3 = H[f + 3];
            odd |= __popcll(h0 & q) | __popcll(h1 & q) | __popcll(h2 & q) | __popcll(h3 & q);
        }
        for (; f < t; ++f) odd |= __popcll(H[f] & q);
    } else {
        for (int f = 0; f < t; ++f) {
            const uint64_t* h = H + static_cast<int64_t>(f) * fw;
            uint64_t acc = 0;
            for (int w = 0; w < fw; ++w) {
                uint64_t qw = x.word(w);
                if (w == cw) qw |= cbit;
                acc ^= h[w] & qw;
            }
            odd |= __popcll(acc);
        }
    }
    return (odd & 1) == 0;
}

// low-rank contexts: reduce phi by the basis rows (descending priority); the
// rows whose pivot bit phi holds sum to [phi | T(phi)] exactly when phi is in the span
template <int SMAX>
__device__ __forceinline__ bool basis_scan(const uint64_t* B, const int32_t* piv, int rank, int n,
                                           const QueryX<SMAX>& x, uint64_t& z0, uint64_t& z1) {
    const int fw = feat_words(n), W = fw + F2_Y_WORDS, cw = n >> 6;
    const uint64_t cbit = 1ull << (n & 63);
    uint64_t diff = 0;  // features: phi XOR the selected rows, word by word
    z0 = z1 = 0;
    if (fw <= 4) {
        uint64_t acc[4] = {0, 0, 0, 0};
        auto add_row = [&](int p, const uint64_t (&rv)[6]) {
            uint64_t qw = x.word(p >> 6);
            if ((p >> 6) == cw) qw |= cbit;
            const uint64_t mk = 0ull - ((qw >> (p & 63)) & 1ull);
#pragma unroll
            for (int w = 0; w < 4; ++w) acc[w] ^= rv[w] & mk;
            z0 ^= rv[4] & mk;
            z1 ^= rv[5] & mk;
        };
        int k = 0;
        for (; k + 2 <= rank; k += 2) {  // two rows in flight (four cost a third of the occupancy of the per-lane passes)
            int p[2];
            uint64_t rv[2][6];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                p[u] = piv[k + u];
                const uint64_t* row = B + static_cast<int64_t>(k + u) * W;
#pragma unroll
                for (int w = 0; w < 4; ++w) rv[u][w] = w < fw ? row[w] : 0ull;
                rv[u][4] = row[fw];
                rv[u][5] = row[fw + 1];
            }
#pragma unroll
            for (int u = 0; u < 2; ++u) add_row(p[u], rv[u]);
        }
        for (; k < rank; ++k) {
            const uint64_t* row = B + static_cast<int64_t>(k) * W;
            uint64_t rv[6];
#pragma unroll
            for (int w = 0; w < 4; ++w) rv[w] = w < fw ? row[w] : 0ull;
            rv[4] = row[fw];
            rv[5] = row[fw + 1];
            add_row(piv[k], rv);
        }
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            if (w >= fw) break;
            uint64_t qw = x.word(w);
            if (w == cw) qw |= cbit;
            diff |= acc[w] ^ qw;
        }
    } else {
        for (int w = 0; w < fw; ++w) {  // one feature word at a time
            uint64_t acc = 0;
            for (int k = 0; k < rank; ++k) {
                const int p = piv[k];
                uint64_t qw = x.word(p >> 6);
                if ((p >> 6) == cw) qw |= cbit;
                if ((qw >> (p & 63)) & 1ull) {
                    const uint64_t* row = B + static_cast<int64_t>(k) * W;
                    acc ^= row[w];
                    if (w == 0) {
                        z0 ^= row[fw];
                        z1 ^= row[fw + 1];
                    }
                }
            }
            uint64_t qw = x.word(w);
            if (w == cw) qw |= cbit;
            diff |= acc ^ qw;
        }
    }
    return diff == 0;
}

template <int SMAX>
__device__ __forceinline__ bool encode_query(const EncArgs& e, int c, const uint64_t* xq, uint64_t& z0,
                                             uint64_t& z1) {
    QueryX<SMAX> x;
    x.load(xq, e.stride);
    const int n = e.n_bits[c];
    if (outside_width(x, n)) return false;
    const int d = n + 1;
    const int r0 = e.rank[c];
    const int r = r0 < 0 ? 0 : (r0 > d ? d : r0);  // 0 <= rank <= d for a fitted context
    if (!has_parity_rows(d, r))
        return basis_scan(e.basis + e.basis_off[c], e.pivots + e.piv_off[c], r, n, x, z0, z1);
    map_gather(e.maps + e.map_off[c], n, x, z0, z1);
    return parity_ok(e.tables + e.basis_off[c], d - r, n, x);
}

// flags and word of one query of context id c
__device__ __forceinline__ uint8_t encode_one(const EncArgs& e, int c, int64_t q, uint64_t& z0, uint64_t& z1) {
    z0 = z1 = 0;
    if (c < 0 || c >= e.num_ctx || (e.ctx_flags[c] & kBadCtx)) return F2_Q_BAD_CTX;
    uint8_t fl = (e.ctx_flags[c] & F2_CTX_CONTRADICTION) ? F2_Q_CTX_CONTRADICTORY : 0;
    const uint64_t* xq = e.x + q * e.stride;
    const bool in = e.stride <= 4 ? encode_query<4>(e, c, xq, z0, z1) : encode_query<0>(e, c, xq, z0, z1);
    if (!in) {
        fl |= F2_Q_OUT_OF_SPAN;
        z0 = z1 = 0;
    }
    return fl;
}

__global__ __launch_bounds__(kEncThreads) void k_encode(EncArgs e) {
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kEncThreads + threadIdx.x;
    if (q >= e.nq) return;
    Word2 out;
    const uint8_t fl = encode_one(e, e.ctx_id[q], q, out.x, out.y);
    *reinterpret_cast<Word2*>(e.words + 2 * q) = out;
    e.qflags[q] = fl;
}

// ---------------------------------------------------------------------------
// context-grouped encode for large batches.  In arbitrary order the lanes of a
// wavefront gather from as many maps as they hold contexts, one cache line per
// lane.  A counting sort by bin (2^k consecutive contexts per bin, at most
// kSortMaxBins bins, or kSortMaxBinsLarge for batches above kFineBinQueries
// (finer bins, an LDS histogram of up to 160 KB), one more bin for out-of-range
// ids) first groups the queries; the encode then runs over the sorted order,
// where the lanes of a wavefront share a few contexts and their gathers hit the
// same lines, and writes each result straight to its query.
//
// The batch is sorted window by window (bpw consecutive count blocks, about
// kWindowQueries queries): a query's sorted position stays inside its window.
// The sorted passes walk the positions in order, so the results they scatter
// at any time land in the queries of about one window (128 MB of words), which
// the last-level cache merges before they reach HBM; scattered 16-byte writes
// over a whole 100M-query batch run at a third of that rate.  The flag bytes
// are cleared in query order by the scatter; the sorted passes write only the
// nonzero ones.  The sort uses per-block LDS histograms and scans (no
// device-wide counters):
//   count (per block)  ->  column scan (per window and bin, over the window's
//   blocks)  ->  scatter (bin scan per block, query -> sorted position)  ->
//   sorted encode  ->  second pass over the positions it leaves
// ---------------------------------------------------------------------------
constexpr int kSortThreads = 1024;
constexpr int kSortMaxBins = 8192;
constexpr int kSortMaxBinsLarge = 40000;  // 160,004 bytes of LDS histogram: up to two of 80,000 contexts per bin
constexpr int64_t kWindowQueries = int64_t{1} << 23;

struct SortArgs {
    int32_t nb;       // bins, the last one for out-of-range context ids
    int32_t bin_shift;  // 2^bin_shift contexts per bin
    int32_t blocks;   // count / scatter blocks
    int32_t bpw;      // count / scatter blocks per window
    int64_t qc;       // queries per count / scatter block
    int32_t* hist;    // [blocks][nb], then exclusive offsets within each bin (of the block's window)
    int32_t* total;   // [windows][nb]
    int2* perm;       // [nq] sorted position -> (query, context id)
    int32_t regroup;  // 1: each chunk of kRegroupChunk positions regrouped by context (k_enc_regroup)
    int32_t staged;   // 1: k_encode_sorted stages the wavefronts' contexts; 0: every position per lane
    uint64_t* rest;   // [ceil(nq / 64)] positions the staged pass left to the second pass (bit per lane; set for the listed groups only)
    int32_t* rest_list;   // [ceil(nq / 64)] the 64-position groups with such positions, in no order
    int32_t* rest_count;  // [1] entries of rest_list (cleared by the count)
};

__device__ __forceinline__ int query_bin(const EncArgs& e, const SortArgs& s, int c) {
    return (c < 0 || c >= e.num_ctx) ? s.nb - 1 : (c >> s.bin_shift);
}

__global__ __launch_bounds__(kSortThreads) void k_enc_count(EncArgs e, SortArgs s) {
    extern __shared__ int sBin[];  // [s.nb] (dynamic)
    const int tid = threadIdx.x;
    for (int b = tid; b < s.nb; b += kSortThreads) sBin[b] = 0;
    __syncthreads();
    const int64_t q0 = static_cast<int64_t>(blockIdx.x) * s.qc;
    const int64_t q1 = q0 + s.qc < e.nq ? q0 + s.qc : e.nq;
    // eight ids per thread and step, the next step's loaded before this step's
    // counts (sixteen loads in flight per thread)
    constexpr int U = 8;
    int64_t q = q0 + tid;
    if (q + (U - 1) * kSortThreads < q1) {
        int c[U];
#pragma unroll
        for (int u = 0; u < U; ++u) c[u] = e.ctx_id[q + u * kSortThreads];
        for (;;) {
            const int64_t qn = q + U * kSortThreads;
            const bool more = qn + (U - 1) * kSortThreads < q1;
            int cn[U];
#pragma unroll
            for (int u = 0; u < U; ++u) cn[u] = e.ctx_id[more ? qn + u * kSortThreads : q];  // (a valid address)
#pragma unroll
            for (int u = 0; u < U; ++u) atomicAdd(&sBin[query_bin(e, s, c[u])], 1);
            q = qn;
            if (!more) break;
#pragma unroll
            for (int u = 0; u < U; ++u) c[u] = cn[u];
        }
    }
    for (; q < q1; q += kSortThreads) atomicAdd(&sBin[query_bin(e, s, e.ctx_id[q])], 1);
    if (blockIdx.x == 0 && tid == 0) *s.rest_count = 0;
    __syncthreads();
    int32_t* h = s.hist + static_cast<int64_t>(blockIdx.x) * s.nb;
    for (int b = tid; b < s.nb; b += kSortThreads) h[b] = sBin[b];
}

// exclusive prefix of each bin over the blocks of its window, in place, and the
// bin's total in the window.  A workgroup takes 64 bins of one window (a lane
// each) and splits the window's blocks among its kColWaves wavefronts, so every lane
// has all of its loads in flight at once.
constexpr int kColWaves = 8;  // 16: 39 us on 100M queries in 12 windows of ~21 blocks; 8: 32 us
constexpr int kMaxSortBlocks = 256;
constexpr int kColPerWave = kMaxSortBlocks / kColWaves;  // blocks per wavefront (at most)
__global__ __launch_bounds__(64 * kColWaves) void k_enc_colscan(SortArgs s) {
    __shared__ int sPart[kColWaves][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int groups = (s.nb + 63) / 64;  // bin groups per window
    const int win = blockIdx.x / groups;
    const int b = (blockIdx.x - win * groups) * 64 + lane;
    const int bpw = s.bpw > 0 ? s.bpw : s.blocks;  // (no window size: one window of every block)
    const int wb0 = win * bpw;
    const int wblocks = s.blocks - wb0 < bpw ? s.blocks - wb0 : bpw;  // <= kMaxSortBlocks
    const int per = (wblocks + kColWaves - 1) / kColWaves;  // <= kColPerWave
    const int gb = wb0 + wave * per, ge = wb0 + wblocks;
    int v[kColPerWave];
#pragma unroll
    for (int k = 0; k < kColPerWave; ++k)
        v[k] = (b < s.nb && k < per && gb + k < ge) ? s.hist[static_cast<int64_t>(gb + k) * s.nb + b] : 0;
    int sum = 0;
#pragma unroll
    for (int k = 0; k < kColPerWave; ++k) sum += v[k];
    sPart[wave][lane] = sum;
    __syncthreads();
    int run = 0, total = 0;
    for (int w = 0; w < kColWaves; ++w) {
        const int t = sPart[w][lane];
        run += w < wave ? t : 0;
        total += t;
    }
    if (b >= s.nb) return;
#pragma unroll
    for (int k = 0; k < kColPerWave; ++k)
        if (k < per && gb + k < ge) {
            s.hist[static_cast<int64_t>(gb + k) * s.nb + b] = run;
            run += v[k];
        }
    if (wave == 0) s.total[static_cast<int64_t>(win) * s.nb + b] = total;
}

// exclusive scan of the bin totals by one workgroup of kSortThreads threads,
// added into sBin, which holds the block's own offsets within each bin (h, copied
// here while the totals are loading).  Up to kBinsPerThread bins per thread the
// totals stay in registers; more bins (large batches) read them twice.
constexpr int kBinsPerThread = (kSortMaxBins + 1 + kSortThreads - 1) / kSortThreads;
__device__ __forceinline__ void bin_offsets(const SortArgs& s, const int32_t* h, const int32_t* total, int* sBin,
                                            int* sWave) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int per = (s.nb + kSortThreads - 1) / kSortThreads;
    const int b0 = tid * per;
    const bool in_regs = per <= kBinsPerThread;
    int tv[kBinsPerThread];
    int sum = 0;
    if (in_regs) {
#pragma unroll
        for (int k = 0; k < kBinsPerThread; ++k) tv[k] = (k < per && b0 + k < s.nb) ? total[b0 + k] : 0;
#pragma unroll
        for (int k = 0; k < kBinsPerThread; ++k) sum += tv[k];
    } else {
        for (int k = 0; k < per; ++k)
            if (b0 + k < s.nb) sum += total[b0 + k];
    }
    for (int b = tid; b < s.nb; b += kSortThreads) sBin[b] = h[b];
    int x = sum;
    for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(x, o);
        if (lane >= o) x += t;
    }
    if (lane == 63) sWave[tid >> 6] = x;
    __syncthreads();
    int run = x - sum;
    for (int w = 0; w < (tid >> 6); ++w) run += sWave[w];
    if (in_regs) {
#pragma unroll
        for (int k = 0; k < kBinsPerThread; ++k)
            if (k < per && b0 + k < s.nb) {
                sBin[b0 + k] += run;
                run += tv[k];
            }
    } else {
        for (int k = 0; k < per; ++k)
            if (b0 + k < s.nb) {
                sBin[b0 + k] += run;
                run += total[b0 + k];
            }
    }
}

__global__ __launch_bounds__(kSortThreads) void k_enc_scatter(EncArgs e, SortArgs s) {
    extern __shared__ int sBin[];  // [s.nb] (dynamic)
    __shared__ int sWave[kSortThreads / 64];
    const int tid = threadIdx.x;
    const int win = blockIdx.x / s.bpw;
    // every block scans its window's bin totals itself (a few thousand words)
    // instead of a one-workgroup scan kernel between the column scan and the scatter
    bin_offsets(s, s.hist + static_cast<int64_t>(blockIdx.x) * s.nb, s.total + static_cast<int64_t>(win) * s.nb, sBin,
                sWave);
    __syncthreads();
    const int64_t q0 = static_cast<int64_t>(blockIdx.x) * s.qc;
    const int64_t q1 = q0 + s.qc < e.nq ? q0 + s.qc : e.nq;
    const int64_t base = static_cast<int64_t>(win) * s.bpw * s.qc;  // the window's first query and position
    // the flag bytes of the block's queries, cleared in order (the sorted passes
    // write the nonzero ones), 8 at a time from the first 8-byte aligned one
    {
        const int mis = static_cast<int>((0 - reinterpret_cast<uintptr_t>(e.qflags)) & 7u);  // qflags + mis is aligned
        const int64_t a0 = q0 + ((mis - q0) & 7);
        const int64_t a1 = a0 + (q1 > a0 ? ((q1 - a0) & ~int64_t{7}) : 0);
        if (a0 < q1) {
            for (int64_t w = tid; w < ((a1 - a0) >> 3); w += kSortThreads)
                reinterpret_cast<uint64_t*>(e.qflags + a0)[w] = 0;
            if (tid < a0 - q0) e.qflags[q0 + tid] = 0;
            if (tid < q1 - a1) e.qflags[a1 + tid] = 0;
        } else {
            for (int64_t q = q0 + tid; q < q1; q += kSortThreads) e.qflags[q] = 0;
        }
    }
    auto place = [&](int64_t q, int c, int p) { s.perm[base + p] = make_int2(static_cast<int>(q), c); };
    // four queries per thread and step, the next step's ids loaded before this
    // step's entries are stored and taken (bins computed) after them: the wait
    // for those loads then leaves the scattered stores in flight (the memory
    // counter retires in issue order), and the ids of the first step are taken
    // before the loop, so that no wait at its top covers the stores either
    int64_t q = q0 + tid;
    if (q + 3 * kSortThreads < q1) {
        int c[4], b[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) c[u] = e.ctx_id[q + u * kSortThreads];
#pragma unroll
        for (int u = 0; u < 4; ++u) b[u] = query_bin(e, s, c[u]);
        for (;;) {
            const int64_t qn = q + 4 * kSortThreads;
            const bool more = qn + 3 * kSortThreads < q1;
            int cn[4], p[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) cn[u] = e.ctx_id[more ? qn + u * kSortThreads : q];  // (a valid address)
#pragma unroll
            for (int u = 0; u < 4; ++u) p[u] = atomicAdd(&sBin[b[u]], 1);
#pragma unroll
            for (int u = 0; u < 4; ++u) place(q + u * kSortThreads, c[u], p[u]);
            q = qn;
            if (!more) break;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                c[u] = cn[u];
                b[u] = query_bin(e, s, cn[u]);
            }
        }
    }
    for (; q < q1; q += kSortThreads) {
        const int c = e.ctx_id[q];
        place(q, c, atomicAdd(&sBin[query_bin(e, s, c)], 1));
    }
}

// A bin of 2^bin_shift contexts keeps its queries in batch order, so its contexts
// interleave.  With many queries per context the sorted positions are regrouped
// chunk by chunk (kRegroupChunk positions, in LDS): key = the bin's offset from
// the chunk's first bin (clamped) and the context's low bits, so within a chunk
// spanning few bins every context's entries end contiguous.  Entries only move
// inside their chunk (chunks never straddle a window).
constexpr int kRegroupThreads = 1024;
constexpr int kRegroupPer = 4;
constexpr int kRegroupChunk = kRegroupThreads * kRegroupPer;  // 4096 positions, 12-bit keys

__global__ __launch_bounds__(kRegroupThreads) void k_enc_regroup(EncArgs e, SortArgs s) {
    __shared__ int sCount[kRegroupChunk];
    __shared__ int sWave[kRegroupThreads / 64];
    __shared__ int2 sEnt[kRegroupChunk];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t c0 = static_cast<int64_t>(blockIdx.x) * kRegroupChunk;
    const int n = e.nq - c0 < kRegroupChunk ? static_cast<int>(e.nq - c0) : kRegroupChunk;
    const int b0 = query_bin(e, s, s.perm[c0].y);
    const int lb = s.bin_shift < 12 ? s.bin_shift : 12;  // keys stay below kRegroupChunk
    const int span = (kRegroupChunk >> lb) - 1;
    int2 ent[kRegroupPer];
    int key[kRegroupPer], rank[kRegroupPer];
#pragma unroll
    for (int u = 0; u < kRegroupPer; ++u) {
        const int k = tid + u * kRegroupThreads;
        ent[u] = k < n ? s.perm[c0 + k] : make_int2(0, 0);
        sCount[k] = 0;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kRegroupPer; ++u) {
        const int k = tid + u * kRegroupThreads;
        key[u] = 0;
        rank[u] = 0;
        if (k < n) {  // positions past the batch take no slot
            const int db = query_bin(e, s, ent[u].y) - b0;  // >= 0: the chunk is in bin order
            key[u] = ((db < span ? db : span) << lb) | (ent[u].y & ((1 << lb) - 1));
            rank[u] = atomicAdd(&sCount[key[u]], 1);
        }
    }
    __syncthreads();
    // exclusive scan of the 4096 key counts: four consecutive keys per thread
    int cnt[kRegroupPer], sum = 0;
#pragma unroll
    for (int u = 0; u < kRegroupPer; ++u) {
        cnt[u] = sCount[kRegroupPer * tid + u];
        sum += cnt[u];
    }
    int x = sum;
    for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(x, o);
        if (lane >= o) x += t;
    }
    if (lane == 63) sWave[wave] = x;
    __syncthreads();
    int base = x - sum;
    for (int w = 0; w < wave; ++w) base += sWave[w];
#pragma unroll
    for (int u = 0; u < kRegroupPer; ++u) {
        sCount[kRegroupPer * tid + u] = base;
        base += cnt[u];
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kRegroupPer; ++u) {
        const int k = tid + u * kRegroupThreads;
        if (k < n) sEnt[sCount[key[u]] + rank[u]] = ent[u];
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kRegroupPer; ++u) {
        const int k = tid + u * kRegroupThreads;
        if (k < n) s.perm[c0 + k] = sEnt[k];
    }
}

// In grouped order the lanes of a wavefront mostly share one context.  Such a
// context's map columns and parity-check rows (or, with few basis rows, its
// basis rows and pivots) are staged in LDS by the whole wavefront with coalesced
// loads, and each lane masks the broadcast columns with its own phi bits: one
// sign-extended bit per column, where the per-lane path gathers a column per
// set bit with divergent addresses.  Staging capacity: contexts of up to 2
// feature words (d <= 128); the positions of wider ones, and of wavefronts with
// more than kSharedCtxPerWave contexts, are left to a second pass (k_encode_rest),
// which keeps this kernel's registers and LDS small (more wavefronts in flight
// to cover its three dependent memory round trips: entry, context scalars, stage).
// The second pass stages, in a stage of up to 4 feature words, each context that
// holds at least kRestStageLanes of a wavefront's remaining lanes, and gathers per
// lane for the others.
//
// A stage of SFW feature words: 64 SFW map columns of 16 bytes at words
// [0, 128 SFW), the parity-check rows (fewer than d / 2 + 1 of up to SFW words)
// from word 128 SFW; or, with few basis rows (r < d / 2), the basis rows and then
// the pivots as words.
template <int SFW>
struct StageGeom {
    static constexpr int cols = 64 * SFW;
    static constexpr int rows = 2 * cols;                  // first word of the parity-check rows
    static constexpr int words = rows + cols / 2 * SFW;    // SFW = 2: 3 KB, SFW = 4: 8 KB
    static_assert((cols / 2 - 1) * (SFW + F2_Y_WORDS + 1) <= words, "few-basis-row contexts fit the stage too");
};
constexpr int kEncStageFW = 2;  // the staged pass
constexpr int kEncWideFW = 4;   // the second pass
struct EncStage {
    uint64_t w[kEncThreads / 64][StageGeom<kEncStageFW>::words];
};
struct EncStageWide {
    uint64_t w[kEncThreads / 64][StageGeom<kEncWideFW>::words];
};

// the staged context's geometry (uniform)
struct StageCtx {
    int n, d, fw, r;
    bool rows;  // parity-check rows (else: basis rows)
};

// a context's scalars, all loads issued together (c valid)
struct CtxScalars {
    uint32_t flags;
    int n, r0;
    int64_t mo, bo, po;
};
__device__ __forceinline__ CtxScalars ctx_scalars(const EncArgs& e, int c) {
    CtxScalars v;
    v.flags = e.ctx_flags[c];
    v.n = e.n_bits[c];
    v.r0 = e.rank[c];
    v.mo = e.map_off[c];
    v.bo = e.basis_off[c];
    v.po = e.piv_off[c];
    // all six values taken here: the six loads go out together (else each is
    // sunk to its first use, behind the branches on the ones before)
    __asm__ volatile("" : : "s"(v.flags), "s"(v.n), "s"(v.r0), "s"(v.mo), "s"(v.bo), "s"(v.po));
    return v;
}

// whole wavefront: stage the context of v (valid, fw <= SFW) in the wavefront's LDS area
template <int SFW>
__device__ __forceinline__ StageCtx stage_context(const EncArgs& e, const CtxScalars& v, uint64_t* st) {
    const int lane = threadIdx.x & 63;
    StageCtx g;
    g.n = v.n;
    g.d = g.n + 1;
    g.fw = feat_words(g.n);
    g.r = v.r0 < 0 ? 0 : (v.r0 > g.d ? g.d : v.r0);
    g.rows = has_parity_rows(g.d, g.r);
    // every load of the stage is issued before the first LDS store (one round trip)
    using G = StageGeom<SFW>;
    if (g.rows) {  // columns at words [0, 2d), the t fw words of parity-check rows from G::rows
        constexpr int NM = 2 * G::cols / 64, NH = (G::words - G::rows) / 64;  // words per lane (d <= cols, t <= d / 2)
        const uint64_t* M = e.maps + v.mo;
        const uint64_t* H = e.tables + v.bo;
        const int nm = 2 * g.d, nh = (g.d - g.r) * g.fw;
        uint64_t a[NM], b[NH];
#pragma unroll
        for (int u = 0; u < NM; ++u) a[u] = lane + 64 * u < nm ? M[lane + 64 * u] : 0ull;
#pragma unroll
        for (int u = 0; u < NH; ++u) b[u] = lane + 64 * u < nh ? H[lane + 64 * u] : 0ull;
#pragma unroll
        for (int u = 0; u < NM; ++u)
            if (lane + 64 * u < nm) st[lane + 64 * u] = a[u];
#pragma unroll
        for (int u = 0; u < NH; ++u)
            if (lane + 64 * u < nh) st[G::rows + lane + 64 * u] = b[u];
    } else {  // basis rows (r (fw + 2) words, r < d / 2), then the pivots as words
        constexpr int NB = (G::cols / 2 * (SFW + F2_Y_WORDS) + 63) / 64, NP = (G::cols / 2 + 63) / 64;
        const uint64_t* B = e.basis + v.bo;
        const int32_t* P = e.pivots + v.po;
        const int nw = g.r * (g.fw + F2_Y_WORDS);
        uint64_t a[NB];
        int32_t b[NP];
#pragma unroll
        for (int u = 0; u < NB; ++u) a[u] = lane + 64 * u < nw ? B[lane + 64 * u] : 0ull;
#pragma unroll
        for (int u = 0; u < NP; ++u) b[u] = lane + 64 * u < g.r ? P[lane + 64 * u] : 0;
#pragma unroll
        for (int u = 0; u < NB; ++u)
            if (lane + 64 * u < nw) st[lane + 64 * u] = a[u];
#pragma unroll
        for (int u = 0; u < NP; ++u)
            if (lane + 64 * u < g.r) st[nw + lane + 64 * u] = static_cast<uint64_t>(b[u]);
    }
    wave_sync();
    return g;
}

template <int FW, int SFW>
__device__ __forceinline__ bool encode_staged(const EncArgs& e, const StageCtx& g, const uint64_t* st,
                                              const uint64_t* xq, const uint64_t (&xv)[4], uint64_t& z0,
                                              uint64_t& z1) {
    const int S = e.stride, n = g.n, d = g.d, fw = g.fw, cw = n >> 6;
    const uint64_t cbit = 1ull << (n & 63);
    bool outside = false;  // x bits at or above n
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        if (w >= S) break;
        if (w > cw) outside |= xv[w] != 0;
        else if (w == cw) outside |= (xv[w] >> (n & 63)) != 0;
    }
    for (int w = 4; w < S; ++w) outside |= xq[w] != 0;  // staged contexts have fw <= 4: all of these are outside
    uint64_t ph[FW];
#pragma unroll
    for (int w = 0; w < FW; ++w) ph[w] = (w < fw ? xv[w] : 0ull) | (w == cw ? cbit : 0ull);
    if (g.rows) {
        // T(phi): every staged column, masked by its bit of phi (the columns past
        // n hold stale words, and their mask is zero).  A loop over 32-column
        // steps, unrolled within a step: fully unrolled, the code of every width
        // runs to several KB per wavefront and instruction fetch bounds the pass.
        const uint4* col = reinterpret_cast<const uint4*>(st);
        uint32_t a0 = 0, a1 = 0, a2 = 0, a3 = 0;
#pragma unroll 1
        for (int j0 = 0; j0 < d; j0 += 32) {
            uint64_t pw = ph[0];
#pragma unroll
            for (int k = 1; k < FW; ++k) pw = (j0 >> 6) == k ? ph[k] : pw;
            const uint32_t half = static_cast<uint32_t>(pw >> (j0 & 32));
#pragma unroll
            for (int u0 = 0; u0 < 32; u0 += 8) {
                if (j0 + u0 >= d) break;
#pragma unroll
                for (int u = u0; u < u0 + 8; ++u) {
                    const uint4 v = col[j0 + u];
                    const uint32_t mk = static_cast<uint32_t>(__builtin_amdgcn_sbfe(static_cast<int>(half), u, 1));
                    a0 = __builtin_amdgcn_bitop3_b32(a0, mk, v.x, 0x78);
                    a1 = __builtin_amdgcn_bitop3_b32(a1, mk, v.y, 0x78);
                    a2 = __builtin_amdgcn_bitop3_b32(a2, mk, v.z, 0x78);
                    a3 = __builtin_amdgcn_bitop3_b32(a3, mk, v.w, 0x78);
                }
            }
        }
        z0 = (static_cast<uint64_t>(a1) << 32) | a0;
        z1 = (static_cast<uint64_t>(a3) << 32) | a2;
        // support: even overlap with every parity-check row
        const uint64_t* H = st + StageGeom<SFW>::rows;
        const int t = d - g.r;
        uint32_t odd = 0;
        for (int f = 0; f < t; ++f) {
            uint64_t acc = 0;
#pragma unroll
            for (int w = 0; w < FW; ++w)
                if (w < fw) acc ^= H[f * fw + w] & ph[w];
            odd |= static_cast<uint32_t>(__popcll(acc));
        }
        return (odd & 1u) == 0 && !outside;
    }
    // few basis rows: the rows whose pivot bit phi holds sum to [phi | T(phi)]
    // exactly when phi is in the span
    const int W = fw + F2_Y_WORDS;
    const uint64_t* piv = st + g.r * W;
    uint64_t acc[FW];
#pragma unroll
    for (int w = 0; w < FW; ++w) acc[w] = 0;
    uint64_t y0 = 0, y1 = 0;
    for (int k = 0; k < g.r; ++k) {
        const int p = static_cast<int>(piv[k]);
        uint64_t pwd = ph[0];
#pragma unroll
        for (int w = 1; w < FW; ++w) pwd = (p >> 6) == w ? ph[w] : pwd;
        const uint32_t mk = bit_mask(pwd, p & 63);
        const uint64_t* row = st + k * W;
#pragma unroll
        for (int w = 0; w < FW; ++w)
            if (w < fw) acc[w] = xor_and(acc[w], mk, row[w]);
        y0 = xor_and(y0, mk, row[fw]);
        y1 = xor_and(y1, mk, row[fw + 1]);
    }
    uint64_t diff = 0;
#pragma unroll
    for (int w = 0; w < FW; ++w) diff |= acc[w] ^ ph[w];
    z0 = y0;
    z1 = y1;
    return diff == 0 && !outside;
}

constexpr int kSharedCtxPerWave = 8;  // contexts of a wavefront taken through the stage

// a query's first x words (up to 4), 16 bytes at a time where the stride and
// the alignment allow
__device__ __forceinline__ void load_x4(const EncArgs& e, const uint64_t* xq, uint64_t (&xv)[4]) {
    const int S = e.stride;
    if (e.x16 && (S == 2 || S == 4)) {  // a query's words start 16-byte aligned
        const uint4* x4 = reinterpret_cast<const uint4*>(xq);
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            if (k >= S / 2) break;
            const uint4 v = x4[k];
            xv[2 * k] = (static_cast<uint64_t>(v.y) << 32) | v.x;
            xv[2 * k + 1] = (static_cast<uint64_t>(v.w) << 32) | v.z;
        }
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (k < S) xv[k] = xq[k];
    }
}

__global__ __launch_bounds__(kEncThreads) void k_encode_sorted(EncArgs e, SortArgs s) {
    __shared__ EncStage sStage;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kEncThreads + threadIdx.x;
    const bool live = i < e.nq;
    const int2 qc = live ? s.perm[i] : make_int2(0, 0);
    uint64_t* st = sStage.w[threadIdx.x >> 6];
    Word2 out, fl;
    out.x = out.y = 0;
    fl.x = fl.y = 0;
    bool done = !live;
    // the query's x words (up to 4) are loaded first: their latency overlaps the
    // context's scalars and the staging
    const uint64_t* xq = e.x + static_cast<int64_t>(live ? qc.x : 0) * e.stride;
    uint64_t xv[4] = {0, 0, 0, 0};
    if (live) load_x4(e, xq, xv);
    for (int k = 0; k < kSharedCtxPerWave; ++k) {  // the wavefront's contexts, first lane's first
        const uint64_t todo = __ballot(!done);
        if (!todo) break;
        const int c0 = __builtin_amdgcn_readlane(qc.y, ffs64(todo));
        const bool valid = c0 >= 0 && c0 < e.num_ctx;
        const CtxScalars v = ctx_scalars(e, valid ? c0 : 0);
        if (!valid || (v.flags & kBadCtx)) {
            if (!done && qc.y == c0) {
                fl.x = F2_Q_BAD_CTX;
                done = true;
            }
            continue;
        }
        if (feat_words(v.n) > kEncStageFW) break;  // wider: per-lane pass
        const StageCtx g = stage_context<kEncStageFW>(e, v, st);
        if (!done && qc.y == c0) {
            fl.x = (v.flags & F2_CTX_CONTRADICTION) ? F2_Q_CTX_CONTRADICTORY : 0;
            const bool in = encode_staged<kEncStageFW, kEncStageFW>(e, g, st, xq, xv, out.x, out.y);
            if (!in) {
                fl.x |= F2_Q_OUT_OF_SPAN;
                out.x = out.y = 0;
            }
            done = true;
        }
        wave_sync();  // the stage is rewritten for the next context
    }
    const uint64_t left = __ballot(!done);  // lanes of further or wider contexts: second pass
    if (left && (threadIdx.x & 63) == 0) {  // a few percent of the groups (the second pass reads only these)
        s.rest[i >> 6] = left;
        s.rest_list[atomicAdd(s.rest_count, 1)] = static_cast<int32_t>(i >> 6);
    }
    if (!done || !live) return;
    *reinterpret_cast<Word2*>(e.words + 2 * static_cast<int64_t>(qc.x)) = out;
    if (fl.x) e.qflags[qc.x] = static_cast<uint8_t>(fl.x);  // the scatter cleared the others
}

// the second pass over the grouped order: the positions the staged pass left
// (their groups in s.rest_list, their lanes in s.rest).  Each context of the
// group (up to kEncWideFW feature words) is staged in turn, however few of the
// group's lanes it holds: on 100M Zipf queries that is 0.55 ms against 0.64 with
// per-lane gathers for contexts of fewer than 16 lanes; wider and bad contexts go
// per lane.  A fixed grid whose wavefronts take the listed groups in turn: a grid
// over every position would launch (and allocate the stage for) a workgroup per
// 256 positions, almost all of them idle (1.2 against 0.42 ms on 100M queries).
constexpr int kRestStageLanes = 1;
constexpr int kRestCtxPerWave = 64;  // contexts of a wavefront considered for the stage (all of them)
constexpr int kRestGrid = 2048;     // workgroups of the listed-group pass (100M queries: 0.50 ms; 1,024: 0.54)

// one wavefront: the lanes of bits among positions i0 .. i0 + 63
__device__ __forceinline__ void rest_group(const EncArgs& e, const SortArgs& s, uint64_t* st, int64_t i0,
                                           uint64_t bits) {
    const int lane = threadIdx.x & 63;
    const int64_t i = i0 + lane;
    const bool live = i < e.nq && ((bits >> lane) & 1ull);
    if (!__ballot(live)) return;
    const int2 qc = live ? s.perm[i] : make_int2(0, 0);
    const uint64_t* xq = e.x + static_cast<int64_t>(live ? qc.x : 0) * e.stride;
    uint64_t xv[4] = {0, 0, 0, 0};
    if (live) load_x4(e, xq, xv);
    Word2 out;
    out.x = out.y = 0;
    uint8_t fl = 0;
    bool done = !live, lane_path = false;
    for (int k = 0; k < kRestCtxPerWave; ++k) {
        const uint64_t todo = __ballot(!done && !lane_path);
        if (!todo) break;
        const int c0 = __builtin_amdgcn_readlane(qc.y, ffs64(todo));
        const bool mine = !done && !lane_path && qc.y == c0;
        bool stage = c0 >= 0 && c0 < e.num_ctx && __popcll(__ballot(mine)) >= kRestStageLanes;
        CtxScalars v;
        if (stage) {
            v = ctx_scalars(e, c0);
            stage = !(v.flags & kBadCtx) && feat_words(v.n) <= kEncWideFW;
        }
        if (!stage) {  // few lanes, or a bad or wide context: per lane
            if (mine) lane_path = true;
            continue;
        }
        const StageCtx g = stage_context<kEncWideFW>(e, v, st);
        if (mine) {
            fl = (v.flags & F2_CTX_CONTRADICTION) ? F2_Q_CTX_CONTRADICTORY : 0;
            const bool in = encode_staged<kEncWideFW, kEncWideFW>(e, g, st, xq, xv, out.x, out.y);
            if (!in) {
                fl |= F2_Q_OUT_OF_SPAN;
                out.x = out.y = 0;
            }
            done = true;
        }
        wave_sync();  // the stage is rewritten for the next context
    }
    if (!done) fl = encode_one(e, qc.y, qc.x, out.x, out.y);
    if (!live) return;
    *reinterpret_cast<Word2*>(e.words + 2 * static_cast<int64_t>(qc.x)) = out;
    if (fl) e.qflags[qc.x] = fl;
}

__global__ __launch_bounds__(kEncThreads) void k_encode_rest(EncArgs e, SortArgs s) {
    __shared__ EncStageWide sStage;
    const int wave = threadIdx.x >> 6;
    uint64_t* st = sStage.w[wave];
    const int cnt = *s.rest_count;
    const int waves = static_cast<int>(gridDim.x) * (kEncThreads / 64);
    for (int k = static_cast<int>(blockIdx.x) * (kEncThreads / 64) + wave; k < cnt; k += waves) {
        const int g = __builtin_amdgcn_readfirstlane(s.rest_list[k]);
        rest_group(e, s, st, static_cast<int64_t>(g) * 64, s.rest[g]);
    }
}

// grouped order without the staged pass (bins of several contexts, not
// regrouped): every position per lane, the lanes of a wavefront gathering from
// the few maps of its bins
__global__ __launch_bounds__(kEncThreads) void k_encode_lanes(EncArgs e, SortArgs s) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kEncThreads + threadIdx.x;
    if (i >= e.nq) return;
    const int2 qc = s.perm[i];
    Word2 out;
    const uint8_t fl = encode_one(e, qc.y, qc.x, out.x, out.y);
    *reinterpret_cast<Word2*>(e.words + 2 * static_cast<int64_t>(qc.x)) = out;
    if (fl) e.qflags[qc.x] = fl;
}

// ---------------------------------------------------------------------------
// feature vectors of Eq. 1 as fit rows, and the post-encode word merges: plain
// streaming kernels, one output word (vectorize) or one 128-bit word (merge)
// per thread, reads and writes coalesced
// ---------------------------------------------------------------------------
constexpr int kStreamThreads = 256;

// each workgroup writes the kVecRows rows from blockIdx * kVecRows on; the row of
// an output word is its index in the workgroup's span times magic = ceil(2^32 / rw)
// (exact: the span is under 2^15 words and rw <= 66)
constexpr int kVecRows = 256;

__global__ __launch_bounds__(kStreamThreads) void k_vectorize(const uint64_t* values, const uint64_t* y,
                                                              int64_t num_rows, int k, uint64_t keep0,
                                                              uint64_t keep1, uint64_t* rows, uint32_t magic) {
    const int rw = k + 3;
    const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kVecRows;
    const int nr = num_rows - r0 < kVecRows ? static_cast<int>(num_rows - r0) : kVecRows;
    const uint64_t* vals = values + r0 * k;
    const uint64_t* yr = y ? y + 2 * r0 : nullptr;
    uint64_t* out = rows + r0 * rw;
    for (int w = threadIdx.x; w < nr * rw; w += kStreamThreads) {
        const int r = static_cast<int>(__umulhi(static_cast<uint32_t>(w), magic));
        const int j = w - r * rw;
        uint64_t v;
        if (j < k) v = vals[r * k + j];
        else if (j == k) v = 1;  // the constant feature
        else v = yr ? (yr[2 * r + (j - k - 1)] & (j == k + 1 ? keep0 : keep1)) : 0ull;
        out[w] = v;
    }
}

__global__ __launch_bounds__(kStreamThreads) void k_merge(const uint64_t* words, const uint64_t* field, int shift,
                                                          int width, uint64_t mask0, uint64_t mask1,
                                                          const uint64_t* state, int64_t n, uint64_t* out) {
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kStreamThreads + threadIdx.x;
    if (q >= n) return;
    const Word2 w = *reinterpret_cast<const Word2*>(words + 2 * q);
    uint64_t lo = w.x, hi = w.y;
    if (field) {
        const uint64_t f = width >= 64 ? field[q] : (field[q] & ((1ull << width) - 1));
        if (shift == 0) {
            lo ^= f;
        } else if (shift < 64) {
            lo ^= f << shift;
            hi ^= f >> (64 - shift);
        } else {
            hi ^= f << (shift - 64);
        }
    }
    uint64_t s0 = 0, s1 = 0;
    if (state) {
        const Word2 st = *reinterpret_cast<const Word2*>(state + 2 * q);
        s0 = st.x;
        s1 = st.y;
    }
    Word2 r;
    r.x = (lo & ~mask0) | (s0 & mask0);
    r.y = (hi & ~mask1) | (s1 & mask1);
    *reinterpret_cast<Word2*>(out + 2 * q) = r;
}

// ---------------------------------------------------------------------------
// basis pooling: contexts trained separately (one per exact group) are tested
// for one shared map by eliminating their bases together.  The members' basis
// rows are concatenated per pool (count -> scan -> copy) and fitted by the fit
// kernels as ordinary row streams; a pool is shared when that fit finds no
// contradiction and its members are valid, consistent and of equal width and
// output mask.
// ---------------------------------------------------------------------------
struct PoolArgs {
    int32_t num_ctx;  // members' model
    const int32_t* n_bits;
    const int64_t* basis_off;
    const uint64_t* basis;
    const int32_t* rank;
    const uint32_t* ctx_flags;
    const uint64_t* out_mask;  // [2 num_ctx] or null
    int32_t num_pools;
    const int64_t* pool_off;   // [num_pools + 1] into members
    const int32_t* members;
    int64_t num_members;
    const int32_t* pooled_n;   // widths of the pooled contexts
    const uint32_t* pooled_flags;
    uint32_t* pool_flags;
    int64_t* row_off;          // [num_pools + 1]: row words per pool, then their offsets
    uint64_t* rows;
    int64_t rows_cap;
    int64_t* blk;              // [ceil(num_pools / 256) + 1]: words per block of 256 pools, then their
                               // offsets; last: the total, or -1 when it exceeds rows_cap
};

constexpr uint32_t kPoolNoRows = F2_POOL_BAD_MEMBER | F2_POOL_WIDTH_MISMATCH;

__global__ __launch_bounds__(256) void k_pool_count(PoolArgs P) {
    const int p0 = blockIdx.x * 256 + threadIdx.x;
    const bool live = p0 < P.num_pools;
    const int p = live ? p0 : P.num_pools - 1;  // lanes past the end redo the last pool and store nothing
    const int64_t lo = P.pool_off[p], hi = P.pool_off[p + 1];
    const int n = P.pooled_n[p];
    const int64_t W = feat_words(n < 0 ? 0 : n) + F2_Y_WORDS;
    uint32_t fl = (lo < 0 || hi < lo || hi > P.num_members || n < 0 || n > F2_MAX_N_BITS) ? F2_POOL_BAD_MEMBER : 0u;
    int64_t words = 0;
    uint64_t m0 = 0, m1 = 0;
    for (int64_t e = lo; e < hi && !(fl & F2_POOL_BAD_MEMBER); ++e) {
        const int c = P.members[e];
        if (c < 0 || c >= P.num_ctx || P.ctx_flags[c] != 0) {  // out of range, malformed or contradictory
            fl |= F2_POOL_BAD_MEMBER;
            break;
        }
        if (P.n_bits[c] != n) fl |= F2_POOL_WIDTH_MISMATCH;
        if (P.out_mask) {
            const uint64_t a0 = P.out_mask[2 * c], a1 = P.out_mask[2 * c + 1];
            if (e == lo) {
                m0 = a0;
                m1 = a1;
            } else if (a0 != m0 || a1 != m1) {
                fl |= F2_POOL_MASK_MISMATCH;
            }
        }
        words += static_cast<int64_t>(P.rank[c]) * W;
    }
    if (live) {
        P.pool_flags[p] = fl;
        P.row_off[p] = (fl & kPoolNoRows) ? 0 : words;
    }
    // the block's words
    __shared__ int64_t sSum[4];
    int64_t v = (!live || (fl & kPoolNoRows)) ? 0 : words;
    for (int o = 32; o > 0; o >>= 1) v += __shfl_down(v, o);
    if ((threadIdx.x & 63) == 0) sSum[threadIdx.x >> 6] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t t = 0;
        for (int w = 0; w < 4; ++w) t += sSum[w];
        P.blk[blockIdx.x] = t;
    }
}

// one workgroup: exclusive scan of the blocks' words (1024 blocks at a time,
// coalesced); the last entry gets the total, or -1 beyond the buffer (a context
// in several pools), which empties every pool and flags it
__global__ __launch_bounds__(1024) void k_pool_scan(PoolArgs P) {
    __shared__ int64_t sWave[16];
    const int tid = threadIdx.x, lane = tid & 63;
    const int nblk = (P.num_pools + 255) / 256;
    int64_t carry = 0;
    for (int b0 = 0; b0 < nblk; b0 += 1024) {
        const int b = b0 + tid;
        const int64_t v = b < nblk ? P.blk[b] : 0;
        int64_t x = v;
        for (int o = 1; o < 64; o <<= 1) {
            const int64_t t = __shfl_up(x, o);
            if (lane >= o) x += t;
        }
        if (lane == 63) sWave[tid >> 6] = x;
        __syncthreads();
        int64_t run = x - v, total = 0;
        for (int w = 0; w < 16; ++w) {
            total += sWave[w];
            if (w < (tid >> 6)) run += sWave[w];
        }
        if (b < nblk) P.blk[b] = carry + run;
        carry += total;
        __syncthreads();  // sWave is rewritten by the next chunk
    }
    if (tid == 0) P.blk[nblk] = carry > P.rows_cap ? -1 : carry;
}

// the pools' row offsets: their block's offset plus the scan within the block
__global__ __launch_bounds__(256) void k_pool_offsets(PoolArgs P) {
    __shared__ int64_t sWave[4];
    const int tid = threadIdx.x, lane = tid & 63;
    const int p = blockIdx.x * 256 + tid;
    const int nblk = (P.num_pools + 255) / 256;
    const bool live = p < P.num_pools;
    const int64_t v = live ? P.row_off[p] : 0;
    const int64_t total = P.blk[nblk], base = P.blk[blockIdx.x];
    int64_t x = v;
    for (int o = 1; o < 64; o <<= 1) {
        const int64_t t = __shfl_up(x, o);
        if (lane >= o) x += t;
    }
    if (lane == 63) sWave[tid >> 6] = x;
    __syncthreads();
    int64_t run = base + x - v;
    for (int w = 0; w < (tid >> 6); ++w) run += sWave[w];
    const bool over = total < 0;
    if (live) {
        P.row_off[p] = over ? 0 : run;
        if (over) P.pool_flags[p] |= F2_POOL_BAD_MEMBER;
    }
    if (p == P.num_pools - 1) P.row_off[P.num_pools] = over ? 0 : total;
}

// one wavefront per pool: the members' basis rows, in member order, each in its
// stored order.  Up to 64 members at a time, one per lane (their ranks and
// offsets loaded together); every lane then copies words of the group's output,
// the member of each word found among the lanes' prefixes.
__global__ __launch_bounds__(256) void k_pool_copy(PoolArgs P) {
    const int lane = threadIdx.x & 63;
    const int p = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (p >= P.num_pools) return;
    if (P.pool_flags[p] & kPoolNoRows) return;
    const int64_t lo = P.pool_off[p], hi = P.pool_off[p + 1];
    const int64_t W = feat_words(P.pooled_n[p]) + F2_Y_WORDS;
    int64_t dst = P.row_off[p];
    for (int64_t e0 = lo; e0 < hi; e0 += 64) {
        const int64_t e = e0 + lane;
        int64_t words = 0, src = 0;
        if (e < hi) {
            const int c = P.members[e];
            words = static_cast<int64_t>(P.rank[c]) * W;
            src = P.basis_off[c];
        }
        int64_t x = words;  // inclusive prefix over the group's members
        for (int o = 1; o < 64; o <<= 1) {
            const int64_t t = __shfl_up(x, o);
            if (lane >= o) x += t;
        }
        const int64_t pre = x - words;
        const int64_t total = __shfl(x, 63);
        const int nm = hi - e0 < 64 ? static_cast<int>(hi - e0) : 64;
        for (int64_t k = lane; k < total; k += 64) {
            // the member holding output word k: the last with prefix <= k (its prefix
            // and source offset read from its lane by readlane, which, unlike a
            // permute, also reads lanes this loop has left inactive)
            int64_t ps = 0;
            int64_t ss = (static_cast<int64_t>(__builtin_amdgcn_readlane(static_cast<int32_t>(src >> 32), 0)) << 32) |
                         (static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int32_t>(src), 0)));
            for (int i = 1; i < nm; ++i) {
                const int64_t pi = (static_cast<int64_t>(__builtin_amdgcn_readlane(static_cast<int32_t>(pre >> 32), i)) << 32) |
                                   (static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int32_t>(pre), i)));
                if (k >= pi) {
                    ps = pi;
                    ss = (static_cast<int64_t>(__builtin_amdgcn_readlane(static_cast<int32_t>(src >> 32), i)) << 32) |
                         (static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int32_t>(src), i)));
                }
            }
            P.rows[dst + k] = P.basis[ss + (k - ps)];
        }
        dst += total;
    }
}

__global__ __launch_bounds__(256) void k_pool_finish(PoolArgs P) {
    const int p = blockIdx.x * 256 + threadIdx.x;
    if (p >= P.num_pools) return;
    uint32_t fl = P.pool_flags[p];
    if (P.pooled_flags[p] & F2_CTX_CONTRADICTION) fl |= F2_POOL_CONTRADICTION;
    P.pool_flags[p] = fl ? fl : F2_POOL_SHARED;
}


// ---------------------------------------------------------------------------
// interleaved-stream ingestion: the rows of many contexts arrive mixed, in
// stream order (Sec. 3: observations are gathered across a corpus); the fit takes
// each context's rows contiguous and in stream order.  A stable LSD radix sort of
// (context, row) pairs by context, 9 bits per pass (per-block LDS histograms, the
// column scan of the encode sort, a stable scatter), then each context's rows are
// copied, trimmed to its row width, to their offsets.  Rows of an out-of-range
// context, of a width outside [0, F2_MAX_N_BITS], or wider than the stride sort
// last and are dropped.
// ---------------------------------------------------------------------------
constexpr int kGrpDigitBits = 9;  // two passes up to 2^18 - 1 contexts
constexpr int kGrpBins = 1 << kGrpDigitBits;
constexpr int kGrpThreads = 1024;
constexpr int kGrpWaves = kGrpThreads / 64;

struct GroupArgs {
    int32_t num_ctx;
    const int32_t* n_bits;
    const int32_t* ctx_id;
    const uint64_t* rows;
    int32_t stride;
    int64_t nr;             // rows
    int32_t blocks;
    int64_t qc;             // rows per count / scatter block
    int32_t shift;          // digit of this pass: (key >> shift) & (kGrpBins - 1)
    const int2* in;         // pairs (key, row) of the previous pass, or null (first pass: from ctx_id)
    int2* out;
    int32_t* hist;          // [blocks][kGrpBins]
    int32_t* total;         // [kGrpBins]
    int32_t* first;         // [num_ctx] first sorted position of each context
    int32_t* count;         // [num_ctx] rows of each context
    int64_t* blk;           // [ceil(num_ctx / 1024) + 1] words per block of contexts, then their offsets
    uint64_t* rows_out;
    int64_t* row_off;       // [num_ctx + 1]
    int64_t* dropped;       // [1]
};

// the sort key of a row: its context, or num_ctx for a row that is dropped
__device__ __forceinline__ int group_key(const GroupArgs& g, int64_t r) {
    const int c = g.ctx_id[r];
    if (c < 0 || c >= g.num_ctx) return g.num_ctx;
    const int n = g.n_bits[c];
    if (n < 0 || n > F2_MAX_N_BITS || feat_words(n) + F2_Y_WORDS > g.stride) return g.num_ctx;
    return c;
}

__device__ __forceinline__ int2 group_pair(const GroupArgs& g, int64_t r) {
    return g.in ? g.in[r] : make_int2(group_key(g, r), static_cast<int>(r));
}

__global__ __launch_bounds__(kGrpThreads) void k_grp_count(GroupArgs g) {
    __shared__ int sBin[kGrpBins];
    const int tid = threadIdx.x;
    if (tid < kGrpBins) sBin[tid] = 0;
    __syncthreads();
    const int64_t r0 = static_cast<int64_t>(blockIdx.x) * g.qc;
    const int64_t r1 = r0 + g.qc < g.nr ? r0 + g.qc : g.nr;
    for (int64_t r = r0 + tid; r < r1; r += kGrpThreads)
        atomicAdd(&sBin[(group_pair(g, r).x >> g.shift) & (kGrpBins - 1)], 1);
    __syncthreads();
    if (tid < kGrpBins) g.hist[static_cast<int64_t>(blockIdx.x) * kGrpBins + tid] = sBin[tid];
}

// stable scatter: the block's rows in rounds of kGrpThreads, wavefront w taking
// the round's w-th 64 rows; within a wavefront a row's rank among equal digits
// comes from the ballots of the digit bits, across wavefronts from per-wavefront
// digit counts, across rounds from the running cursor of each digit
__global__ __launch_bounds__(kGrpThreads) void k_grp_scatter(GroupArgs g) {
    __shared__ int sCur[kGrpBins];
    __shared__ int sCnt[kGrpWaves][kGrpBins];
    __shared__ int sBase[kGrpBins];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid < kGrpBins) {  // the bin's start: bins before it over every block, then the blocks before this one
        int base = 0;
        for (int b = 0; b < tid; ++b) base += g.total[b];
        sCur[tid] = base + g.hist[static_cast<int64_t>(blockIdx.x) * kGrpBins + tid];
    }
    const int64_t r0 = static_cast<int64_t>(blockIdx.x) * g.qc;
    const int64_t r1 = r0 + g.qc < g.nr ? r0 + g.qc : g.nr;
    const uint64_t lt = (1ull << lane) - 1;
    for (int64_t rb = r0; rb < r1; rb += kGrpThreads) {
        for (int k = tid; k < kGrpWaves * kGrpBins; k += kGrpThreads) (&sCnt[0][0])[k] = 0;
        const int64_t r = rb + 64 * wave + lane;
        const bool live = r < r1;
        const int2 pr = live ? group_pair(g, r) : make_int2(0, 0);
        const int dg = (pr.x >> g.shift) & (kGrpBins - 1);
        uint64_t peers = __ballot(live);
#pragma unroll
        for (int b = 0; b < kGrpDigitBits; ++b) {
            const uint64_t m = __ballot(live && ((dg >> b) & 1));
            peers &= ((dg >> b) & 1) ? m : ~m;
        }
        const int rank = __popcll(peers & lt);
        __syncthreads();  // counts cleared
        if (live && rank == __popcll(peers) - 1) sCnt[wave][dg] = __popcll(peers);  // the group's last lane
        __syncthreads();
        if (tid < kGrpBins) {  // per digit: exclusive prefix over the wavefronts, the round's count to the cursor
            int run = sCur[tid];
            for (int w = 0; w < kGrpWaves; ++w) {
                const int c = sCnt[w][tid];
                sCnt[w][tid] = run;
                run += c;
            }
            sBase[tid] = run;
        }
        __syncthreads();
        if (live) g.out[sCnt[wave][dg] + rank] = pr;
        __syncthreads();
        if (tid < kGrpBins) sCur[tid] = sBase[tid];
    }
}

// first position and row count of each context, rows dropped (contexts zeroed first)
__global__ __launch_bounds__(256) void k_grp_clear(GroupArgs g) {
    const int c = blockIdx.x * 256 + threadIdx.x;
    if (c < g.num_ctx) {
        g.first[c] = 0;
        g.count[c] = 0;
    }
    if (c == 0) *g.dropped = 0;
}

__global__ __launch_bounds__(256) void k_grp_bounds(GroupArgs g) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= g.nr) return;
    const int k = g.in[i].x;
    const bool start = i == 0 || g.in[i - 1].x != k;
    if (k == g.num_ctx) {
        if (start) *g.dropped = g.nr - i;
        return;
    }
    if (start) g.first[k] = static_cast<int32_t>(i);
    if (i == g.nr - 1 || g.in[i + 1].x != k) g.count[k] = static_cast<int32_t>(i + 1);  // end, made a count below
}

// words per block of 1024 contexts (end positions made counts)
__global__ __launch_bounds__(1024) void k_grp_words(GroupArgs g) {
    __shared__ int64_t sW[16];
    const int c = blockIdx.x * 1024 + threadIdx.x;
    int64_t v = 0;
    if (c < g.num_ctx) {
        const int cnt = g.count[c] ? g.count[c] - g.first[c] : 0;
        g.count[c] = cnt;
        v = static_cast<int64_t>(cnt) * (feat_words(g.n_bits[c]) + F2_Y_WORDS);
        g.row_off[c] = v;
    }
    for (int o = 32; o > 0; o >>= 1) v += __shfl_down(v, o);
    if ((threadIdx.x & 63) == 0) sW[threadIdx.x >> 6] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t t = 0;
        for (int w = 0; w < 16; ++w) t += sW[w];
        g.blk[blockIdx.x] = t;
    }
}

// one workgroup: exclusive scan of the blocks' words, the total last
__global__ __launch_bounds__(1024) void k_grp_scan(GroupArgs g) {
    __shared__ int64_t sWave[16];
    const int tid = threadIdx.x, lane = tid & 63;
    const int nblk = (g.num_ctx + 1023) / 1024;
    int64_t carry = 0;
    for (int b0 = 0; b0 < nblk; b0 += 1024) {
        const int b = b0 + tid;
        const int64_t v = b < nblk ? g.blk[b] : 0;
        int64_t x = v;
        for (int o = 1; o < 64; o <<= 1) {
            const int64_t t = __shfl_up(x, o);
            if (lane >= o) x += t;
        }
        if (lane == 63) sWave[tid >> 6] = x;
        __syncthreads();
        int64_t run = x - v, total = 0;
        for (int w = 0; w < 16; ++w) {
            total += sWave[w];
            if (w < (tid >> 6)) run += sWave[w];
        }
        if (b < nblk) g.blk[b] = carry + run;
        carry += total;
        __syncthreads();
    }
    if (tid == 0) g.blk[nblk] = carry;
}

// each context's word offset: its block's offset plus the scan within the block
__global__ __launch_bounds__(1024) void k_grp_offsets(GroupArgs g) {
    __shared__ int64_t sWave[16];
    const int tid = threadIdx.x, lane = tid & 63;
    const int c = blockIdx.x * 1024 + tid;
    const int64_t v = c < g.num_ctx ? g.row_off[c] : 0;
    int64_t x = v;
    for (int o = 1; o < 64; o <<= 1) {
        const int64_t t = __shfl_up(x, o);
        if (lane >= o) x += t;
    }
    if (lane == 63) sWave[tid >> 6] = x;
    __syncthreads();
    int64_t run = g.blk[blockIdx.x] + x - v;
    for (int w = 0; w < (tid >> 6); ++w) run += sWave[w];
    if (c < g.num_ctx) g.row_off[c] = run;
    if (c == g.num_ctx - 1) g.row_off[g.num_ctx] = g.blk[(g.num_ctx + 1023) / 1024];
}

// the dropped-row count out, and row_off[0] = 0 when there are no contexts
__global__ __launch_bounds__(64) void k_grp_finish(GroupArgs g, int64_t* dropped_out, int no_ctx) {
    if (threadIdx.x == 0) {
        *dropped_out = g.nr > 0 ? *g.dropped : 0;
        if (no_ctx) g.row_off[0] = 0;
    }
}

// output rows: sorted position i copies its row, trimmed to the context's width
// eight lanes per row: lane j copies words j, j + 8, ... of its row, so one
// instruction moves up to 64 contiguous bytes of each of 8 rows and no lane waits on
// a chain of single-word copies
constexpr int kGrpCopyLanes = 8;
constexpr int kGrpCopyRowsPerBlock = 256 / kGrpCopyLanes;
__global__ __launch_bounds__(256) void k_grp_copy(GroupArgs g) {
    const int j = threadIdx.x % kGrpCopyLanes;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kGrpCopyRowsPerBlock + threadIdx.x / kGrpCopyLanes;
         i < g.nr; i += static_cast<int64_t>(gridDim.x) * kGrpCopyRowsPerBlock) {
        const int2 pr = g.in[i];
        if (pr.x >= g.num_ctx) continue;
        const int W = feat_words(g.n_bits[pr.x]) + F2_Y_WORDS;
        const uint64_t* __restrict__ src = g.rows + static_cast<int64_t>(pr.y) * g.stride;
        uint64_t* __restrict__ dst = g.rows_out + g.row_off[pr.x] + static_cast<int64_t>(i - g.first[pr.x]) * W;
        for (int w = j; w < W; w += kGrpCopyLanes) dst[w] = src[w];
    }
}

inline size_t align256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }


// workspace of the grouping: two pair buffers, histograms, per-context bounds
struct GroupPlan {
    int blocks;
    int64_t qc;
    size_t off_a, off_b, off_hist, off_total, off_first, off_count, off_blk, off_drop, bytes;
};
GroupPlan group_workspace(int32_t num_ctx, int64_t nr) {
    GroupPlan p{};
    int64_t blocks = (nr + 8191) / 8192;
    if (blocks > kMaxSortBlocks) blocks = kMaxSortBlocks;
    if (blocks < 1) blocks = 1;
    p.qc = (nr + blocks - 1) / blocks;
    if (p.qc < 1) p.qc = 1;
    p.blocks = static_cast<int>((nr + p.qc - 1) / p.qc);
    if (p.blocks < 1) p.blocks = 1;
    size_t o = 0;
    p.off_a = o;
    o = align256(o + sizeof(int2) * static_cast<size_t>(nr));
    p.off_b = o;
    o = align256(o + sizeof(int2) * static_cast<size_t>(nr));
    p.off_hist = o;
    o = align256(o + sizeof(int32_t) * static_cast<size_t>(p.blocks) * kGrpBins);
    p.off_total = o;
    o = align256(o + sizeof(int32_t) * kGrpBins);
    p.off_first = o;
    o = align256(o + sizeof(int32_t) * static_cast<size_t>(num_ctx));
    p.off_count = o;
    o = align256(o + sizeof(int32_t) * static_cast<size_t>(num_ctx));
    p.off_blk = o;
    o = align256(o + sizeof(int64_t) * (static_cast<size_t>((num_ctx + 1023) / 1024) + 1));
    p.off_drop = o;
    o = align256(o + sizeof(int64_t));
    p.bytes = o;
    return p;
}

// workgroups of a fit class kernel: at most one per context, at most `cap`
unsigned fit_grid(int num_ctx, int cap) { return static_cast<unsigned>(num_ctx < cap ? num_ctx : cap); }

// encode workspace: empty for the gather path; the sort buffers when the batch is
// large enough for grouping by context to pay off
struct EncPlan {
    bool sorted;
    int windows;
    SortArgs s;
    size_t off_hist, off_total, off_perm, off_rest, off_rest_list, off_rest_count, bytes;
};

int64_t encode_window();

// batches above this take the fine bins (an LDS histogram of up to 160 KB)
constexpr int64_t kFineBinQueries = int64_t{1} << 22;

EncPlan encode_workspace(int32_t num_ctx, int64_t nq) {
    EncPlan p{};
    p.bytes = 256;
    // grouping pays from about 160k queries on (4,096 contexts of 17-97 bits: the
    // gather path takes 31 us for 131k queries, the grouped one 36 us; at 197k 45 and 42 us)
    p.sorted = nq >= 3 * (1 << 16) && nq >= 4 * static_cast<int64_t>(num_ctx) && nq <= 0x7fffffff;
    if (!p.sorted) return p;
    const int64_t C = num_ctx > 0 ? num_ctx : 1;
    int shift = 0;
    // finer bins for large batches (100M Zipf queries over 80,000 contexts in
    // windows of 8M: 6.44 ms with 4 contexts per bin, 6.19 with 2); smaller ones
    // keep the small histogram (a 160 KB one costs its occupancy there)
    const int maxb = nq > kFineBinQueries ? kSortMaxBinsLarge : kSortMaxBins;
    while ((C + (int64_t{1} << shift) - 1) >> shift > maxb) ++shift;
    p.s.bin_shift = shift;
    p.s.nb = static_cast<int>((C + (int64_t{1} << shift) - 1) >> shift) + 1;
    // about 256 count / scatter blocks in all (one per compute unit, each with its
    // histogram), of at least 8k queries: enough blocks for the scatter, few
    // histogram rows to scan (1M queries: 83 us with 8k, 86 with 16k, 88 with 4k).
    // Above the window size the blocks form windows of bpw blocks; their size is a
    // multiple of kRegroupChunk, so no regrouped chunk straddles two windows.
    const int64_t wq = encode_window();
    const int64_t windows = (nq + wq - 1) / wq;
    int64_t qc, bpw;
    if (windows <= 1) {
        int64_t blocks = (nq + 8191) / 8192;
        if (blocks > kMaxSortBlocks) blocks = kMaxSortBlocks;
        qc = (nq + blocks - 1) / blocks;
        bpw = blocks;
    } else {
        bpw = kMaxSortBlocks / windows > 1 ? kMaxSortBlocks / windows : 1;
        const int64_t per_window = (nq + windows - 1) / windows;
        qc = (per_window + bpw - 1) / bpw;
        qc = (qc + kRegroupChunk - 1) / kRegroupChunk * kRegroupChunk;
    }
    p.s.qc = qc;
    p.s.blocks = static_cast<int>((nq + qc - 1) / qc);
    p.s.bpw = static_cast<int>(bpw < p.s.blocks ? bpw : p.s.blocks);
    p.windows = (p.s.blocks + p.s.bpw - 1) / p.s.bpw;
    size_t o = 0;
    p.off_hist = o;
    o = align256(o + sizeof(int32_t) * static_cast<size_t>(p.s.blocks) * p.s.nb);
    p.off_total = o;
    o = align256(o + sizeof(int32_t) * static_cast<size_t>(p.windows) * p.s.nb);
    p.off_perm = o;
    o = align256(o + sizeof(int2) * static_cast<size_t>(nq));
    // above kFineBinQueries bins of up to 4 contexts go to the staged pass as they
    // come (no regroup: 6.95 against 7.09 ms on 100M Zipf queries over 80,000
    // contexts); smaller batches regroup when bins hold several contexts and
    // contexts average 16 queries or more
    const bool fine = nq > kFineBinQueries && shift <= 2;
    p.s.regroup = !fine && shift > 0 && nq >= 16 * C;
    // with one context per bin, fine bins, or after the regroup, a wavefront holds
    // a few contexts and the staged pass applies; otherwise every position goes per lane
    p.s.staged = shift == 0 || fine || p.s.regroup;
    p.off_rest = o;
    o = align256(o + sizeof(uint64_t) * static_cast<size_t>((nq + 63) / 64));
    p.off_rest_list = o;
    o = align256(o + sizeof(int32_t) * static_cast<size_t>((nq + 63) / 64));
    p.off_rest_count = o;
    o = align256(o + sizeof(int32_t));
    p.bytes = o > 256 ? o : 256;
    return p;
}

// every output buffer of a model present and its sizes non-negative
bool model_complete(const f2_model* m) {
    return m->n_bits && m->basis_off && m->piv_off && m->map_off && m->basis && m->pivots && m->maps && m->tables &&
           m->rank && m->ctx_flags && m->n_contra && m->first_contra_row && m->basis_words >= 0 &&
           m->piv_entries >= 0 && m->map_words >= 0;
}

// polls of a group barrier before it gives up: 2^24 (seconds), or the value of
// F2GPU_GROUP_SPIN_LIMIT (a test hook for the timeout report)
int group_spin_limit() {
    const char* v = getenv("F2GPU_GROUP_SPIN_LIMIT");
    if (!v || !*v) return 1 << 24;
    char* end = nullptr;
    const long x = strtol(v, &end, 10);
    if (*end != '\0' || x < 0) return 1 << 24;
    return x > (1 << 24) ? (1 << 24) : static_cast<int>(x);
}

// queries per encode chunk: the grouped path indexes a batch's positions in 32
// bits, so larger batches are encoded in chunks of 2^30 (each grouped on its own,
// one after the other through one chunk-sized workspace); F2GPU_ENCODE_CHUNK may
// set a smaller chunk (a test hook for the chunking)
constexpr int64_t kEncChunk = int64_t{1} << 30;
int64_t encode_chunk() {
    const char* v = getenv("F2GPU_ENCODE_CHUNK");
    if (!v || !*v) return kEncChunk;
    char* end = nullptr;
    const long long x = strtoll(v, &end, 10);
    if (*end != '\0' || x < 1 || x > kEncChunk) return kEncChunk;
    return x;
}

// queries per sort window: kWindowQueries, or the value of F2GPU_ENCODE_WINDOW
// (a test hook: several windows at sizes the oracle checks quickly), at least
// 2^16 so that the per-window bin totals stay a small part of the workspace
int64_t encode_window() {
    const char* v = getenv("F2GPU_ENCODE_WINDOW");
    if (!v || !*v) return kWindowQueries;
    char* end = nullptr;
    const long long x = strtoll(v, &end, 10);
    if (*end != '\0' || x < 1 || x > kEncChunk) return kWindowQueries;
    return x < (int64_t{1} << 16) ? (int64_t{1} << 16) : x;
}

FitArgs fit_args(const uint64_t* rows, int64_t rows_words, const int64_t* row_off, const f2_model* m, int32_t* plan) {
    FitArgs a;
    a.rows = rows;
    a.rows_words = rows_words;
    a.row_off = row_off;
    a.num_ctx = m->num_ctx;
    a.n_bits = m->n_bits;
    a.basis_off = m->basis_off;
    a.piv_off = m->piv_off;
    a.map_off = m->map_off;
    a.basis_words = m->basis_words;
    a.piv_entries = m->piv_entries;
    a.map_words = m->map_words;
    a.basis = m->basis;
    a.pivots = m->pivots;
    a.maps = m->maps;
    a.tables = m->tables;
    a.rank = m->rank;
    a.ctx_flags = m->ctx_flags;
    a.n_contra = m->n_contra;
    a.first_contra = m->first_contra_row;
    a.plan = plan;
    a.coop = 0;
    a.max_n = m->max_n_bits;
    a.spin_limit = group_spin_limit();
    return a;
}

// the fit: plan (two kernels), then the class kernels, each keeping about as
// many workgroups as fit on the chip at once
// workgroups of the wide kernel that can be resident at once on the current
// device, or 0 where cooperative launches are unavailable (queried once per device)
int wide_resident_workgroups() {
    static std::atomic<int> cache[64];  // value + 1; 0 = not queried yet
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 0;
    if (dev < 64) {
        const int v = cache[dev].load(std::memory_order_relaxed);
        if (v > 0) return v - 1;
    }
    int coop = 0, cus = 0, per_cu = 0;
    int r = 0;
    if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) == hipSuccess && coop &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(k_fit_wide), kLargeThreads,
                                                     0) == hipSuccess)
        r = cus * per_cu;
    (void)hipGetLastError();
    if (dev < 64) cache[dev].store(r + 1, std::memory_order_relaxed);
    return r;
}

// the fit: plan (two kernels), then the class kernels.  The wide kernel runs one
// workgroup per compute unit as a cooperative launch (so that a group of
// workgroups can fit one context together), else a plain launch of up to 256.
constexpr int kPivGrid = 768;  // LDS-basis workgroups: three per compute unit (LDS-bound)
void launch_fit(FitArgs a, hipStream_t s) {
    const int32_t C = a.num_ctx;
    if (C <= kSmallBatch && a.max_n >= 0 && a.max_n < 512) {
        a.coop = 0;
        hipLaunchKernelGGL(k_fit_small, dim3(static_cast<unsigned>(C)), dim3(kLargeThreads), 0, s, a);
        return;
    }
    const int plan_blocks = static_cast<int>((static_cast<int64_t>(C) + kPlanThreads - 1) / kPlanThreads);
    hipLaunchKernelGGL(k_plan_count, dim3(plan_blocks), dim3(kPlanThreads), 0, s, a);
    hipLaunchKernelGGL(k_plan_scatter, dim3(plan_blocks), dim3(kPlanThreads), 0, s, a, plan_blocks);
    hipLaunchKernelGGL(k_fit_reg, dim3(fit_grid((C + kRegWaves - 1) / kRegWaves, 256)), dim3(64 * kRegWaves), 0, s, a);
    hipLaunchKernelGGL(k_fit_piv, dim3(fit_grid(C, kPivGrid)), dim3(kPivThreads), 0, s, a);
    // a batch whose declared widths stay below 512 holds no wide context (wider
    // ones are rejected by the plan), so the wide kernel is not launched at all
    if (a.max_n >= 0 && a.max_n < 512) return;
    const int res = wide_resident_workgroups();
    if (res >= 32) {
        a.coop = 1;
        void* args[] = {&a};
        if (hipLaunchCooperativeKernel(reinterpret_cast<const void*>(k_fit_wide), dim3(res < 1024 ? res : 1024),
                                       dim3(kLargeThreads), args, 0, s) == hipSuccess)
            return;
        (void)hipGetLastError();
    }
    a.coop = 0;
    hipLaunchKernelGGL(k_fit_wide, dim3(fit_grid(C, 256)), dim3(kLargeThreads), 0, s, a);
}

}  // namespace

extern "C" {

const char* f2_status_string(int status) {
    switch (status) {
        case F2_OK: return "ok";
        case F2_EINVAL: return "invalid argument";
        case F2_EWORKSPACE: return "workspace missing or too small";
        case F2_EDEVICE: return "HIP error while enqueuing device work";
        case F2_ETOOWIDE: return "context width above F2_MAX_N_BITS";
        case F2_ESCRATCH: return "batch above the allocation-free fit's fixed plan size (F2_NOALLOC_MAX_CTX contexts)";
        default: return "unknown status";
    }
}

int f2_fit_layout(const int32_t* n_bits_host, int32_t num_ctx, int64_t* basis_off_host, int64_t* piv_off_host,
                  int64_t* map_off_host) {
    if (num_ctx < 0 || !basis_off_host || !piv_off_host || !map_off_host || (num_ctx > 0 && !n_bits_host))
        return F2_EINVAL;
    int64_t bo = 0, po = 0, mo = 0;
    for (int32_t c = 0; c < num_ctx; ++c) {
        const int n = n_bits_host[c];
        if (n < 0) return F2_EINVAL;
        if (n > F2_MAX_N_BITS) return F2_ETOOWIDE;
        const int64_t d = n + 1, W = (n + 64) / 64 + F2_Y_WORDS;
        basis_off_host[c] = bo;
        piv_off_host[c] = po;
        map_off_host[c] = mo;
        bo += d * W;
        po += d;
        mo += 2 * d;
    }
    basis_off_host[num_ctx] = bo;
    piv_off_host[num_ctx] = po;
    map_off_host[num_ctx] = mo;
    return F2_OK;
}

size_t f2_fit_workspace_bytes(int32_t num_ctx) {
    if (num_ctx < 0) return 0;
    const size_t blocks = (static_cast<size_t>(num_ctx) + kPlanThreads - 1) / kPlanThreads;
    return align256(sizeof(int32_t) * (kPlanHead + 2 * static_cast<size_t>(num_ctx) + kPlanBins * blocks));
}

}  // extern "C"

namespace {

// ---------------------------------------------------------------------------
// allocation-free fit: the plan lives in a fixed device array instead of a
// caller workspace.  The array's name is a host-side stand-in; its device address
// is looked up once per device (hipGetSymbolAddress with that device current)
// and kept, and only that address is handed to kernels.  Every call on a device
// shares its array: calls that overlap on one device race.  The plan kernels
// initialise every plan word they read, so nothing stale carries over.
// ---------------------------------------------------------------------------
constexpr int32_t kScratchMaxCtx = F2_NOALLOC_MAX_CTX;
constexpr size_t kScratchBytes =
    (sizeof(int32_t) * (kPlanHead + 2 * static_cast<size_t>(kScratchMaxCtx) +
                        kPlanBins * ((static_cast<size_t>(kScratchMaxCtx) + kPlanThreads - 1) / kPlanThreads)) +
     255) / 256 * 256;
constexpr int kScratchDevices = 64;

__device__ __align__(256) uint8_t scratch[kScratchBytes];

// device address of this device's scratch array, or nullptr if it cannot be found
void* scratch_address() {
    static std::atomic<void*> addr[kScratchDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices) return nullptr;
    void* p = addr[dev].load(std::memory_order_acquire);
    if (p) return p;
    void* q = nullptr;
    if (hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)) != hipSuccess || !q) {
        (void)hipGetLastError();
        return nullptr;
    }
    addr[dev].store(q, std::memory_order_release);  // the same address whichever thread looks it up
    return q;
}

}  // namespace

extern "C" {

int f2_fit_batch_noalloc(const uint64_t* rows, int64_t rows_words, const int64_t* row_off, const f2_model* m,
                         void* stream) {
    if (!m || m->num_ctx < 0 || rows_words < 0) return F2_EINVAL;
    const int32_t C = m->num_ctx;
    if (C == 0) return F2_OK;
    if (!row_off || !model_complete(m) || (rows_words > 0 && !rows)) return F2_EINVAL;
    if (C > kScratchMaxCtx || f2_fit_workspace_bytes(C) > kScratchBytes) return F2_ESCRATCH;
    void* plan = scratch_address();
    if (!plan) return F2_EDEVICE;
    launch_fit(fit_args(rows, rows_words, row_off, m, static_cast<int32_t*>(plan)), static_cast<hipStream_t>(stream));
    return hipGetLastError() == hipSuccess ? F2_OK : F2_EDEVICE;
}

int f2_fit_batch(const uint64_t* rows, int64_t rows_words, const int64_t* row_off, const f2_model* m,
                 void* workspace, size_t workspace_bytes, void* stream) {
    if (!m || m->num_ctx < 0 || rows_words < 0) return F2_EINVAL;
    const int32_t C = m->num_ctx;
    if (C == 0) return F2_OK;
    if (!row_off || !model_complete(m) || (rows_words > 0 && !rows)) return F2_EINVAL;
    if (!workspace || workspace_bytes < f2_fit_workspace_bytes(C) ||
        (reinterpret_cast<uintptr_t>(workspace) & 255u))
        return F2_EWORKSPACE;
    launch_fit(fit_args(rows, rows_words, row_off, m, static_cast<int32_t*>(workspace)), static_cast<hipStream_t>(stream));
    return hipGetLastError() == hipSuccess ? F2_OK : F2_EDEVICE;
}

size_t f2_encode_workspace_bytes(const f2_model* m, int64_t num_queries) {
    if (!m || m->num_ctx < 0 || num_queries < 0) return 0;
    const int64_t chunk = encode_chunk();
    return encode_workspace(m->num_ctx, num_queries < chunk ? num_queries : chunk).bytes;
}

}  // extern "C"

namespace {

// one chunk of at most encode_chunk() queries (arguments checked by the caller)
int encode_range(const f2_model* m, const int32_t* ctx_id, const uint64_t* x, int32_t x_stride_words,
                 int64_t num_queries, uint64_t* words_out, uint8_t* qflags_out, void* workspace, hipStream_t s) {
    EncArgs e;
    e.num_ctx = m->num_ctx;
    e.n_bits = m->n_bits;
    e.basis_off = m->basis_off;
    e.piv_off = m->piv_off;
    e.basis = m->basis;
    e.pivots = m->pivots;
    e.rank = m->rank;
    e.ctx_flags = m->ctx_flags;
    e.map_off = m->map_off;
    e.maps = m->maps;
    e.tables = m->tables;
    e.ctx_id = ctx_id;
    e.x = x;
    e.stride = x_stride_words;
    e.x16 = (reinterpret_cast<uintptr_t>(x) & 15u) == 0;
    e.nq = num_queries;
    e.words = words_out;
    e.qflags = qflags_out;
    const int64_t blocks = (num_queries + kEncThreads - 1) / kEncThreads;
    if (blocks > 0x7fffffff) return F2_EINVAL;
    EncPlan p = encode_workspace(m->num_ctx, num_queries);
    if (!p.sorted) {
        hipLaunchKernelGGL(k_encode, dim3(static_cast<unsigned>(blocks)), dim3(kEncThreads), 0, s, e);
        return hipGetLastError() == hipSuccess ? F2_OK : F2_EDEVICE;
    }
    char* ws = static_cast<char*>(workspace);
    p.s.hist = reinterpret_cast<int32_t*>(ws + p.off_hist);
    p.s.total = reinterpret_cast<int32_t*>(ws + p.off_total);
    p.s.perm = reinterpret_cast<int2*>(ws + p.off_perm);
    p.s.rest = reinterpret_cast<uint64_t*>(ws + p.off_rest);
    p.s.rest_list = reinterpret_cast<int32_t*>(ws + p.off_rest_list);
    p.s.rest_count = reinterpret_cast<int32_t*>(ws + p.off_rest_count);
    const size_t bin_lds = sizeof(int) * static_cast<size_t>(p.s.nb);
    hipLaunchKernelGGL(k_enc_count, dim3(p.s.blocks), dim3(kSortThreads), bin_lds, s, e, p.s);
    hipLaunchKernelGGL(k_enc_colscan, dim3(static_cast<unsigned>(p.windows) * ((p.s.nb + 63) / 64)),
                       dim3(64 * kColWaves), 0, s, p.s);
    hipLaunchKernelGGL(k_enc_scatter, dim3(p.s.blocks), dim3(kSortThreads), bin_lds, s, e, p.s);
    if (p.s.regroup)
        hipLaunchKernelGGL(k_enc_regroup, dim3(static_cast<unsigned>((num_queries + kRegroupChunk - 1) / kRegroupChunk)),
                           dim3(kRegroupThreads), 0, s, e, p.s);
    if (p.s.staged) {
        hipLaunchKernelGGL(k_encode_sorted, dim3(static_cast<unsigned>(blocks)), dim3(kEncThreads), 0, s, e, p.s);
        hipLaunchKernelGGL(k_encode_rest, dim3(static_cast<unsigned>(blocks < kRestGrid ? blocks : kRestGrid)),
                           dim3(kEncThreads), 0, s, e, p.s);
    } else {
        hipLaunchKernelGGL(k_encode_lanes, dim3(static_cast<unsigned>(blocks)), dim3(kEncThreads), 0, s, e, p.s);
    }
    return hipGetLastError() == hipSuccess ? F2_OK : F2_EDEVICE;
}

}  // namespace

extern "C" {

int f2_encode_batch(const f2_model* m, const int32_t* ctx_id, const uint64_t* x, int32_t x_stride_words,
                    int64_t num_queries, uint64_t* words_out, uint8_t* qflags_out, void* workspace,
                    size_t workspace_bytes, void* stream) {
    if (!m || m->num_ctx < 0 || num_queries < 0 || x_stride_words < 1) return F2_EINVAL;
    if (num_queries == 0) return F2_OK;
    if (!ctx_id || !x || !words_out || !qflags_out) return F2_EINVAL;
    if (m->num_ctx > 0 && (!m->n_bits || !m->basis_off || !m->piv_off || !m->map_off || !m->basis || !m->pivots ||
                           !m->maps || !m->tables || !m->rank || !m->ctx_flags))
        return F2_EINVAL;
    if (!workspace || workspace_bytes < f2_encode_workspace_bytes(m, num_queries) ||
        (reinterpret_cast<uintptr_t>(workspace) & 255u))
        return F2_EWORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    // chunks in stream order through the one workspace
    const int64_t chunk = encode_chunk();
    for (int64_t q0 = 0; q0 < num_queries; q0 += chunk) {
        const int64_t n = num_queries - q0 < chunk ? num_queries - q0 : chunk;
        const int st = encode_range(m, ctx_id + q0, x + q0 * x_stride_words, x_stride_words, n, words_out + 2 * q0,
                                    qflags_out + q0, workspace, s);
        if (st != F2_OK) return st;
    }
    return F2_OK;
}

int f2_vectorize_rows(const uint64_t* values, const uint64_t* y, int64_t num_rows, int32_t k,
                      const uint64_t* keep_host, uint64_t* rows_out, void* stream) {
    if (num_rows < 0 || k < 0 || k > 63 || !keep_host) return F2_EINVAL;
    if (num_rows == 0) return F2_OK;
    if ((k > 0 && !values) || !rows_out) return F2_EINVAL;
    const int64_t blocks = (num_rows + kVecRows - 1) / kVecRows;
    if (num_rows > (int64_t{1} << 56) || blocks > 0x7fffffff) return F2_EINVAL;
    const uint32_t rw = static_cast<uint32_t>(k + 3);
    const uint32_t magic = static_cast<uint32_t>(((uint64_t{1} << 32) + rw - 1) / rw);  // ceil(2^32 / rw)
    hipLaunchKernelGGL(k_vectorize, dim3(static_cast<unsigned>(blocks)), dim3(kStreamThreads), 0,
                       static_cast<hipStream_t>(stream), values, y, num_rows, k, keep_host[0], keep_host[1], rows_out,
                       magic);
    return hipGetLastError() == hipSuccess ? F2_OK : F2_EDEVICE;
}

int f2_merge_words(const uint64_t* words, const uint64_t* field, int32_t shift, int32_t width,
                   const uint64_t* mask_host, const uint64_t* state, int64_t num_words, uint64_t* out,
                   void* stream) {
    if (num_words < 0 || !mask_host) return F2_EINVAL;
    if (field && (width < 1 || width > 64 || shift < 0 || shift + width > 128)) return F2_EINVAL;
    if (num_words == 0) return F2_OK;
    if (!words || !out) return F2_EINVAL;
    const int64_t blocks = (num_words + kStreamThreads - 1) / kStreamThreads;
    if (blocks > 0x7fffffff) return F2_EINVAL;
    hipLaunchKernelGGL(k_merge, dim3(static_cast<unsigned>(blocks)), dim3(kStreamThreads), 0,
                       static_cast<hipStream_t>(stream), words, field, field ? shift : 0, field ? width : 64,
                       mask_host[0], mask_host[1], state, num_words, out);
    return hipGetLastError() == hipSuccess ? F2_OK : F2_EDEVICE;
}

size_t f2_pool_workspace_bytes(const f2_model* members_model, int32_t num_pools) {
    if (!members_model || members_model->basis_words < 0 || num_pools < 0) return 0;
    return align256(sizeof(int64_t) * (static_cast<size_t>(num_pools) + 1)) +
           align256(sizeof(uint64_t) * static_cast<size_t>(members_model->basis_words)) +
           align256(sizeof(int64_t) * (static_cast<size_t>((num_pools + 255) / 256) + 1)) +
           f2_fit_workspace_bytes(num_pools);
}

size_t f2_group_workspace_bytes(int32_t num_ctx, int64_t num_rows) {
    if (num_ctx < 0 || num_rows < 0 || num_rows > 0x7fffffff) return 0;
    return group_workspace(num_ctx, num_rows).bytes;
}

int f2_group_rows(const int32_t* ctx_id, const uint64_t* rows, int32_t row_stride_words, int64_t num_rows,
                  const int32_t* n_bits, int32_t num_ctx, uint64_t* rows_out, int64_t rows_out_words,
                  int64_t* row_off_out, int64_t* dropped_out, void* workspace, size_t workspace_bytes, void* stream) {
    if (num_ctx < 0 || num_rows < 0 || num_rows > 0x7fffffff || row_stride_words < F2_Y_WORDS + 1) return F2_EINVAL;
    if (!row_off_out || !dropped_out || (num_ctx > 0 && !n_bits)) return F2_EINVAL;
    if (num_rows > 0 && (!ctx_id || !rows || !rows_out || rows_out_words < num_rows * row_stride_words))
        return F2_EINVAL;
    if (!workspace || workspace_bytes < f2_group_workspace_bytes(num_ctx, num_rows) ||
        (reinterpret_cast<uintptr_t>(workspace) & 255u))
        return F2_EWORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const GroupPlan p = group_workspace(num_ctx, num_rows);
    char* ws = static_cast<char*>(workspace);
    GroupArgs g;
    g.num_ctx = num_ctx;
    g.n_bits = n_bits;
    g.ctx_id = ctx_id;
    g.rows = rows;
    g.stride = row_stride_words;
    g.nr = num_rows;
    g.blocks = p.blocks;
    g.qc = p.qc;
    g.hist = reinterpret_cast<int32_t*>(ws + p.off_hist);
    g.total = reinterpret_cast<int32_t*>(ws + p.off_total);
    g.first = reinterpret_cast<int32_t*>(ws + p.off_first);
    g.count = reinterpret_cast<int32_t*>(ws + p.off_count);
    g.blk = reinterpret_cast<int64_t*>(ws + p.off_blk);
    g.rows_out = rows_out;
    g.row_off = row_off_out;
    g.dropped = reinterpret_cast<int64_t*>(ws + p.off_drop);
    int2* bufs[2] = {reinterpret_cast<int2*>(ws + p.off_a), reinterpret_cast<int2*>(ws + p.off_b)};
    // passes: kGrpDigitBits bits of the key (0 .. num_ctx) each
    int bits = 1;
    while ((int64_t{1} << bits) <= num_ctx) ++bits;
    const int passes = (bits + kGrpDigitBits - 1) / kGrpDigitBits;
    SortArgs cs{};
    cs.nb = kGrpBins;
    cs.blocks = p.blocks;
    cs.bpw = p.blocks;  // one window: every block
    cs.hist = g.hist;
    cs.total = g.total;
    g.in = nullptr;
    if (num_rows > 0) {
        for (int k = 0; k < passes; ++k) {
            g.shift = kGrpDigitBits * k;
            g.out = bufs[k & 1];
            hipLaunchKernelGGL(k_grp_count, dim3(p.blocks), dim3(kGrpThreads), 0, s, g);
            hipLaunchKernelGGL(k_enc_colscan, dim3((kGrpBins + 63) / 64), dim3(64 * kColWaves), 0, s, cs);
            hipLaunchKernelGGL(k_grp_scatter, dim3(p.blocks), dim3(kGrpThreads), 0, s, g);
            g.in = g.out;
        }
    }
    const unsigned cb = static_cast<unsigned>((num_ctx + 255) / 256);
    if (num_ctx > 0) hipLaunchKernelGGL(k_grp_clear, dim3(cb), dim3(256), 0, s, g);
    else hipLaunchKernelGGL(k_grp_clear, dim3(1), dim3(256), 0, s, g);
    if (num_rows > 0)
        hipLaunchKernelGGL(k_grp_bounds, dim3(static_cast<unsigned>((num_rows + 255) / 256)), dim3(256), 0, s, g);
    const unsigned kb = static_cast<unsigned>((num_ctx + 1023) / 1024);
    if (num_ctx > 0) {
        hipLaunchKernelGGL(k_grp_words, dim3(kb), dim3(1024), 0, s, g);
        hipLaunchKernelGGL(k_grp_scan, dim3(1), dim3(1024), 0, s, g);
        hipLaunchKernelGGL(k_grp_offsets, dim3(kb), dim3(1024), 0, s, g);
    } else {
        hipLaunchKernelGGL(k_grp_scan, dim3(1), dim3(1024), 0, s, g);  // row_off[0] = 0 below
    }
    if (num_rows > 0 && num_ctx > 0)
        hipLaunchKernelGGL(k_grp_copy,
                           dim3(static_cast<unsigned>(std::min<int64_t>((num_rows + kGrpCopyRowsPerBlock - 1) / kGrpCopyRowsPerBlock, 1 << 20))),
                           dim3(256), 0, s, g);
    hipLaunchKernelGGL(k_grp_finish, dim3(1), dim3(64), 0, s, g, dropped_out, num_ctx == 0 ? 1 : 0);
    return hipGetLastError() == hipSuccess ? F2_OK : F2_EDEVICE;
}

int f2_pool_bases(const f2_model* members_model, const uint64_t* out_mask, const int64_t* pool_off,
                  const int32_t* members, int64_t num_members, const f2_model* pooled, uint32_t* pool_flags,
                  void* workspace, size_t workspace_bytes, void* stream) {
    if (!members_model || !pooled || members_model->num_ctx < 0 || pooled->num_ctx < 0 || num_members < 0)
        return F2_EINVAL;
    const int32_t P = pooled->num_ctx;
    if (P == 0) return F2_OK;
    if (!pool_off || !pool_flags || (num_members > 0 && !members) || !model_complete(pooled)) return F2_EINVAL;
    if (members_model->num_ctx > 0 && (!members_model->n_bits || !members_model->basis_off || !members_model->basis ||
                                       !members_model->rank || !members_model->ctx_flags || members_model->basis_words < 0))
        return F2_EINVAL;
    if (!workspace || workspace_bytes < f2_pool_workspace_bytes(members_model, P) ||
        (reinterpret_cast<uintptr_t>(workspace) & 255u))
        return F2_EWORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    char* ws = static_cast<char*>(workspace);
    PoolArgs A;
    A.num_ctx = members_model->num_ctx;
    A.n_bits = members_model->n_bits;
    A.basis_off = members_model->basis_off;
    A.basis = members_model->basis;
    A.rank = members_model->rank;
    A.ctx_flags = members_model->ctx_flags;
    A.out_mask = out_mask;
    A.num_pools = P;
    A.pool_off = pool_off;
    A.members = members;
    A.num_members = num_members;
    A.pooled_n = pooled->n_bits;
    A.pooled_flags = pooled->ctx_flags;
    A.pool_flags = pool_flags;
    A.row_off = reinterpret_cast<int64_t*>(ws);
    const size_t off_rows = align256(sizeof(int64_t) * (static_cast<size_t>(P) + 1));
    A.rows = reinterpret_cast<uint64_t*>(ws + off_rows);
    A.rows_cap = members_model->basis_words;
    const size_t off_blk = off_rows + align256(sizeof(uint64_t) * A.rows_cap);
    const unsigned pb = static_cast<unsigned>((P + 255) / 256);
    A.blk = reinterpret_cast<int64_t*>(ws + off_blk);
    int32_t* plan = reinterpret_cast<int32_t*>(ws + off_blk + align256(sizeof(int64_t) * (static_cast<size_t>(pb) + 1)));
    hipLaunchKernelGGL(k_pool_count, dim3(pb), dim3(256), 0, s, A);
    hipLaunchKernelGGL(k_pool_scan, dim3(1), dim3(1024), 0, s, A);
    hipLaunchKernelGGL(k_pool_offsets, dim3(pb), dim3(256), 0, s, A);
    hipLaunchKernelGGL(k_pool_copy, dim3(static_cast<unsigned>((P + 3) / 4)), dim3(256), 0, s, A);
    launch_fit(fit_args(A.rows, A.rows_cap, A.row_off, pooled, plan), s);
    hipLaunchKernelGGL(k_pool_finish, dim3(pb), dim3(256), 0, s, A);
    return hipGetLastError() == hipSuccess ? F2_OK : F2_EDEVICE;
}

}  // extern "C"
