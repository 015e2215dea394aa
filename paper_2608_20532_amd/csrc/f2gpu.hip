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
// Contexts are sorted into width classes by a plan kernel; each class runs a
// kernel specialised for its feature-word count, one wavefront per context
// with the basis in LDS.  Contexts wider than 8 feature words run a
// workgroup-per-context kernel with the basis in HBM and rows staged in LDS.
//
// Encode (Sec. 2.3): a prepare kernel turns each fitted basis into a
// per-column table [z_j | h_j]: z_j is the canonical map column and h_j the
// column of the parity check on the non-pivot (free) columns.  A query then
// XORs the table entries of its set feature bits: the z part is T(phi) and
// the h part is the reduction residual on the free columns, zero exactly when
// phi lies in the span.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/f2gpu.h"

namespace {

constexpr int kClasses = 5;          // feature words 1, 2, 3-4, 5-8, >8
constexpr int kLargeRows = 64;       // rows per block, large path
constexpr int kLargeThreads = 256;
constexpr int kMaxW = 66;            // widest row: 64 feature words + 2 output words
constexpr int kEncThreads = 256;
constexpr int kEncHW = 8;            // parity-check words kept in registers

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
    int32_t* rank;
    uint32_t* ctx_flags;
    int32_t* n_contra;
    int64_t* first_contra;
    int32_t* counters;  // [0, kClasses): contexts per class
    int32_t* lists;     // kClasses x num_ctx context ids
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
    uint64_t* tables;  // same offsets as the basis: context c at basis_off[c]
    const int32_t* ctx_id;
    const uint64_t* x;
    int32_t stride;
    int64_t nq;
    uint64_t* words;
    uint8_t* qflags;
};

constexpr uint32_t kBadCtx = F2_CTX_BAD_SEGMENT | F2_CTX_BAD_WIDTH | F2_CTX_BAD_OUTPUT;

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
// plan: validate every context, write the outputs of invalid ones, and sort
// the valid ones into width classes.
// ---------------------------------------------------------------------------
__global__ void k_fit_init(int32_t* counters) {
    if (threadIdx.x < 16) counters[threadIdx.x] = 0;
}

__global__ __launch_bounds__(256) void k_fit_plan(FitArgs a) {
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    int cls = -1;
    if (c < a.num_ctx) {
        const int n = a.n_bits[c];
        uint32_t flags = 0;
        int64_t mo = 0;
        int d = 0;
        if (n < 0 || n > F2_MAX_N_BITS) {
            flags = F2_CTX_BAD_WIDTH;
        } else {
            d = n + 1;
            const int W = feat_words(n) + F2_Y_WORDS;
            const int64_t bo = a.basis_off[c], po = a.piv_off[c];
            mo = a.map_off[c];
            if (bo < 0 || bo + static_cast<int64_t>(d) * W > a.basis_words || po < 0 || po + d > a.piv_entries ||
                mo < 0 || mo + 2 * static_cast<int64_t>(d) > a.map_words) {
                flags = F2_CTX_BAD_OUTPUT;
            } else {
                const int64_t s0 = a.row_off[c], s1 = a.row_off[c + 1];
                if (s0 < 0 || s1 < s0 || s1 > a.rows_words || (s1 - s0) % W != 0) flags = F2_CTX_BAD_SEGMENT;
            }
        }
        if (flags) {
            a.rank[c] = 0;
            a.n_contra[c] = 0;
            a.first_contra[c] = -1;
            a.ctx_flags[c] = flags;
            if (flags == F2_CTX_BAD_SEGMENT)
                for (int j = 0; j < 2 * d; ++j) a.maps[mo + j] = 0;
        } else {
            const int fw = feat_words(n);
            cls = fw == 1 ? 0 : fw == 2 ? 1 : fw <= 4 ? 2 : fw <= 8 ? 3 : 4;
        }
    }
    // wave-aggregated append: one atomic per class per wavefront
    const int lane = threadIdx.x & 63;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int k = 0; k < kClasses; ++k) {
        const uint64_t mask = __ballot(cls == k);
        if (!mask) continue;
        int base = 0;
        const int leader = ffs64(mask);
        if (lane == leader) base = atomicAdd(&a.counters[k], __popcll(mask));
        base = __shfl(base, leader);
        if (cls == k) a.lists[static_cast<int64_t>(k) * a.num_ctx + base + __popcll(mask & below)] = c;
    }
}

// ---------------------------------------------------------------------------
// small-context fit: one wavefront per context, basis in LDS, FW = feature
// words of the class (contexts of the class have fw <= FW)
// ---------------------------------------------------------------------------
template <int FW>
__device__ __forceinline__ uint64_t pick_word(const uint64_t (&f)[FW], int w) {
    uint64_t v = f[0];
#pragma unroll
    for (int k = 1; k < FW; ++k) v = (w == k) ? f[k] : v;
    return v;
}

template <int FW>
__global__ __launch_bounds__(64) void k_fit_small(FitArgs a, int cls) {
    constexpr int CAP = 64 * FW;  // d <= 64 FW retained rows at most
    __shared__ uint64_t sBf[FW][CAP];
    __shared__ uint64_t sBy[2][CAP];
    __shared__ int16_t sPiv[CAP];
    __shared__ int16_t sPos[CAP];
    const int lane = threadIdx.x;
    const int count = a.counters[cls];
    const int32_t* list = a.lists + static_cast<int64_t>(cls) * a.num_ctx;

    for (int idx = blockIdx.x; idx < count; idx += gridDim.x) {
        const int c = list[idx];
        const int n = a.n_bits[c];
        const int fw = feat_words(n), W = fw + F2_Y_WORDS, d = n + 1;
        const int64_t s0 = a.row_off[c];
        const int64_t m = (a.row_off[c + 1] - s0) / W;
        const uint64_t* R = a.rows + s0;
        const uint64_t tmask = top_mask(n, fw);
        const int cw = n >> 6;
        const uint64_t cbit = 1ull << (n & 63);

        for (int j = lane; j < d; j += 64) sPos[j] = -1;
        int rank = 0, ncontra = 0;
        int64_t first = -1;
        __syncthreads();

        for (int64_t b0 = 0; b0 < m; b0 += 64) {
            const int64_t i = b0 + lane;
            const bool valid = i < m;
            uint64_t f[FW];
            uint64_t y0 = 0, y1 = 0;
#pragma unroll
            for (int w = 0; w < FW; ++w) f[w] = 0;
            if (valid) {
                const uint64_t* row = R + i * W;
#pragma unroll
                for (int w = 0; w < FW; ++w)
                    if (w < fw) f[w] = row[w];
                y0 = row[fw];
                y1 = row[fw + 1];
#pragma unroll
                for (int w = 0; w < FW; ++w)
                    if (w == fw - 1) f[w] &= tmask;
            }
            // (1) reduce against the retained basis (one pass: it is fully reduced)
            for (int s = 0; s < rank; ++s) {
                const int p = sPiv[s];
                if ((pick_word<FW>(f, p >> 6) >> (p & 63)) & 1ull) {
#pragma unroll
                    for (int w = 0; w < FW; ++w) f[w] ^= sBf[w][s];
                    y0 ^= sBy[0][s];
                    y1 ^= sBy[1][s];
                }
            }
            // (2) in-block elimination in stream order
            uint64_t pending = __ballot(valid);
            while (pending) {
                bool nzf = false;
#pragma unroll
                for (int w = 0; w < FW; ++w) nzf |= (f[w] != 0);
                const uint64_t nz = __ballot(nzf) & pending;
                const int j = nz ? ffs64(nz) : 64;
                const uint64_t before = (j >= 64) ? pending : (pending & ((1ull << j) - 1));
                const uint64_t cm = __ballot((y0 | y1) != 0) & before;
                if (cm) {
                    if (ncontra == 0) first = b0 + ffs64(cm);
                    ncontra += __popcll(cm);
                }
                pending &= ~before;
                if (j >= 64) break;
                uint64_t F[FW];
#pragma unroll
                for (int w = 0; w < FW; ++w) F[w] = readlane64(f[w], j);
                const uint64_t Y0 = readlane64(y0, j), Y1 = readlane64(y1, j);
                // pivot: highest-priority set feature bit (x_{n-1} .. x_0, then the constant)
                int p = -1;
#pragma unroll
                for (int w = FW - 1; w >= 0; --w) {
                    uint64_t v = F[w];
                    if (w == cw) v &= ~cbit;
                    if (p < 0 && v) p = 64 * w + msb64(v);
                }
                if (p < 0) p = n;
                // later rows of the block holding bit p
                if (lane > j && ((pick_word<FW>(f, p >> 6) >> (p & 63)) & 1ull)) {
#pragma unroll
                    for (int w = 0; w < FW; ++w) f[w] ^= F[w];
                    y0 ^= Y0;
                    y1 ^= Y1;
                }
                // clear p from every retained row, then insert
                for (int s = lane; s < rank; s += 64) {
                    if ((sBf[p >> 6][s] >> (p & 63)) & 1ull) {
#pragma unroll
                        for (int w = 0; w < FW; ++w) sBf[w][s] ^= F[w];
                        sBy[0][s] ^= Y0;
                        sBy[1][s] ^= Y1;
                    }
                }
                if (lane == 0) {
#pragma unroll
                    for (int w = 0; w < FW; ++w) sBf[w][rank] = F[w];
                    sBy[0][rank] = Y0;
                    sBy[1][rank] = Y1;
                    sPiv[rank] = static_cast<int16_t>(p);
                    sPos[p] = static_cast<int16_t>(rank);
                }
                ++rank;
                pending &= ~(1ull << j);
                __syncthreads();
            }
        }
        __syncthreads();

        // outputs: basis rows and pivots in descending priority, canonical map, scalars
        const int64_t bo = a.basis_off[c], po = a.piv_off[c], mo = a.map_off[c];
        for (int s = lane; s < rank; s += 64) {
            const int p = sPiv[s];
            int k = 0;
            if (p == n) {
                k = rank - 1;
            } else {
                for (int t = 0; t < rank; ++t) {
                    const int q = sPiv[t];
                    k += (q > p && q < n);
                }
            }
            uint64_t* out = a.basis + bo + static_cast<int64_t>(k) * W;
            for (int w = 0; w < fw; ++w) out[w] = sBf[w][s];
            out[fw] = sBy[0][s];
            out[fw + 1] = sBy[1][s];
            a.pivots[po + k] = p;
        }
        for (int j = lane; j < d; j += 64) {
            const int s = sPos[j];
            a.maps[mo + 2 * j] = s >= 0 ? sBy[0][s] : 0ull;
            a.maps[mo + 2 * j + 1] = s >= 0 ? sBy[1][s] : 0ull;
        }
        if (lane == 0) {
            a.rank[c] = rank;
            a.n_contra[c] = ncontra;
            a.first_contra[c] = first;
            a.ctx_flags[c] = ncontra ? F2_CTX_CONTRADICTION : 0u;
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// large-context fit: one workgroup of 4 wavefronts per context.  The working
// basis lives in the caller's basis buffer, one slot per priority position
// (slot t holds the row whose pivot is the t-th highest-priority feature), so
// that the final descending-priority order is an in-place compaction.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int prio_slot(int p, int n) { return p < n ? n - 1 - p : n; }
__device__ __forceinline__ int slot_pivot(int t, int n) { return t < n ? n - 1 - t : n; }

__global__ __launch_bounds__(kLargeThreads) void k_fit_large(FitArgs a, int cls) {
    __shared__ uint64_t sRow[kLargeRows][kMaxW];
    __shared__ uint64_t sPmask[64];
    __shared__ int sNewRow[kLargeRows];  // block row of the k-th new pivot
    __shared__ int sNewPiv[kLargeRows];  // its pivot
    __shared__ int sP, sNumNew, sContra;
    __shared__ long long sFirst;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int count = a.counters[cls];
    const int32_t* list = a.lists + static_cast<int64_t>(cls) * a.num_ctx;

    for (int idx = blockIdx.x; idx < count; idx += gridDim.x) {
        const int c = list[idx];
        const int n = a.n_bits[c];
        const int fw = feat_words(n), W = fw + F2_Y_WORDS, d = n + 1;
        const int64_t s0 = a.row_off[c];
        const int64_t m = (a.row_off[c + 1] - s0) / W;
        const uint64_t* R = a.rows + s0;
        const uint64_t tmask = top_mask(n, fw);
        const int cw = n >> 6;
        const uint64_t cbit = 1ull << (n & 63);
        uint64_t* B = a.basis + a.basis_off[c];

        if (tid < 64) sPmask[tid] = 0;
        if (tid == 0) {
            sContra = 0;
            sFirst = -1;
        }
        __syncthreads();

        for (int64_t b0 = 0; b0 < m; b0 += kLargeRows) {
            const int nb = static_cast<int>((m - b0) < kLargeRows ? (m - b0) : kLargeRows);
            for (int k = tid; k < nb * W; k += kLargeThreads) {
                const int r = k / W, w = k - r * W;
                uint64_t v = R[(b0 + r) * W + w];
                if (w == fw - 1) v &= tmask;
                sRow[r][w] = v;
            }
            if (tid == 0) sNumNew = 0;
            __syncthreads();

            // (1) block reduce against the retained basis, lanes over words
            for (int r = wave; r < nb; r += 4) {
                uint64_t acc0 = 0, acc1 = 0;
                for (int w = 0; w < fw; ++w) {
                    uint64_t v = sRow[r][w] & sPmask[w];
                    while (v) {
                        const int p = 64 * w + ffs64(v);
                        v &= v - 1;
                        const uint64_t* src = B + static_cast<int64_t>(prio_slot(p, n)) * W;
                        if (lane < W) acc0 ^= src[lane];
                        if (64 + lane < W) acc1 ^= src[64 + lane];
                    }
                }
                if (lane < W) sRow[r][lane] ^= acc0;
                if (64 + lane < W) sRow[r][64 + lane] ^= acc1;
            }
            __syncthreads();

            // (2) in-block elimination in stream order
            for (int j = 0; j < nb; ++j) {
                if (wave == 0) {
                    const uint64_t v = (lane < fw) ? sRow[j][lane] : 0ull;
                    const uint64_t vx = (lane == cw) ? (v & ~cbit) : v;
                    const uint64_t nzm = __ballot(v != 0);
                    const uint64_t nxm = __ballot(vx != 0);
                    int p = -1;
                    if (nxm) {
                        const int top = msb64(nxm);
                        p = 64 * top + msb64(readlane64(vx, top));
                    } else if (nzm) {
                        p = n;
                    }
                    if (lane == 0) {
                        sP = p;
                        if (p < 0 && (sRow[j][fw] | sRow[j][fw + 1])) {
                            if (sContra == 0) sFirst = b0 + j;
                            ++sContra;
                        }
                        if (p >= 0) {
                            sNewRow[sNumNew] = j;
                            sNewPiv[sNumNew] = p;
                            ++sNumNew;
                        }
                    }
                }
                __syncthreads();
                const int p = sP;
                if (p >= 0) {
                    for (int r = j + 1 + wave; r < nb; r += 4) {
                        if ((sRow[r][p >> 6] >> (p & 63)) & 1ull) {
                            if (lane < W) sRow[r][lane] ^= sRow[j][lane];
                            if (64 + lane < W) sRow[r][64 + lane] ^= sRow[j][64 + lane];
                        }
                    }
                }
                __syncthreads();
            }

            // (3) fully reduce the new rows among themselves (latest pivot first)
            const int K = sNumNew;
            for (int k = K - 1; k > 0; --k) {
                const int jk = sNewRow[k], pk = sNewPiv[k];
                for (int e = wave; e < k; e += 4) {
                    const int je = sNewRow[e];
                    if ((sRow[je][pk >> 6] >> (pk & 63)) & 1ull) {
                        if (lane < W) sRow[je][lane] ^= sRow[jk][lane];
                        if (64 + lane < W) sRow[je][64 + lane] ^= sRow[jk][64 + lane];
                    }
                }
                __syncthreads();
            }

            if (K > 0) {
                // (4) clear the new pivots from every retained row
                for (int t = wave; t < d; t += 4) {
                    const int pt = slot_pivot(t, n);
                    if (!((sPmask[pt >> 6] >> (pt & 63)) & 1ull)) continue;
                    uint64_t* row = B + static_cast<int64_t>(t) * W;
                    uint64_t w0 = (lane < W) ? row[lane] : 0ull;
                    uint64_t w1 = (64 + lane < W) ? row[64 + lane] : 0ull;
                    const int pk = (lane < K) ? sNewPiv[lane] : 0;
                    const uint64_t wk = shfl64(w0, pk >> 6);
                    uint64_t sel = __ballot(lane < K && ((wk >> (pk & 63)) & 1ull));
                    if (!sel) continue;
                    while (sel) {
                        const int k = ffs64(sel);
                        sel &= sel - 1;
                        const int jk = sNewRow[k];
                        if (lane < W) w0 ^= sRow[jk][lane];
                        if (64 + lane < W) w1 ^= sRow[jk][64 + lane];
                    }
                    if (lane < W) row[lane] = w0;
                    if (64 + lane < W) row[64 + lane] = w1;
                }
                // (5) insert the new rows at their priority slots
                for (int k = wave; k < K; k += 4) {
                    const int jk = sNewRow[k];
                    uint64_t* row = B + static_cast<int64_t>(prio_slot(sNewPiv[k], n)) * W;
                    if (lane < W) row[lane] = sRow[jk][lane];
                    if (64 + lane < W) row[64 + lane] = sRow[jk][64 + lane];
                }
                __syncthreads();
                if (tid == 0)
                    for (int k = 0; k < K; ++k) sPmask[sNewPiv[k] >> 6] |= 1ull << (sNewPiv[k] & 63);
            }
            __syncthreads();
        }

        // outputs: canonical map from the slots, then compaction into descending priority
        const int64_t po = a.piv_off[c], mo = a.map_off[c];
        for (int j = tid; j < d; j += kLargeThreads) {
            const bool present = (sPmask[j >> 6] >> (j & 63)) & 1ull;
            const uint64_t* row = B + static_cast<int64_t>(prio_slot(j, n)) * W;
            a.maps[mo + 2 * j] = present ? row[fw] : 0ull;
            a.maps[mo + 2 * j + 1] = present ? row[fw + 1] : 0ull;
        }
        int rank = 0;
        for (int w = 0; w < fw; ++w) rank += __popcll(sPmask[w]);
        __syncthreads();
        for (int t0 = 0; t0 < d; t0 += 4) {
            const int t = t0 + wave;
            const int pt = t < d ? slot_pivot(t, n) : 0;
            const bool present = t < d && ((sPmask[pt >> 6] >> (pt & 63)) & 1ull);
            uint64_t w0 = 0, w1 = 0;
            int k = 0;
            if (present) {
                const uint64_t* row = B + static_cast<int64_t>(t) * W;
                if (lane < W) w0 = row[lane];
                if (64 + lane < W) w1 = row[64 + lane];
                if (pt == n) {
                    k = rank - 1;
                } else {
                    // pivots of higher priority: x bits above pt
                    for (int w = pt >> 6; w < fw; ++w) {
                        uint64_t v = sPmask[w];
                        if (w == (pt >> 6)) v &= (pt & 63) == 63 ? 0ull : (~0ull << ((pt & 63) + 1));
                        if (w == cw) v &= ~cbit;
                        k += __popcll(v);
                    }
                }
            }
            __syncthreads();
            if (present) {
                uint64_t* out = B + static_cast<int64_t>(k) * W;
                if (lane < W) out[lane] = w0;
                if (64 + lane < W) out[64 + lane] = w1;
                if (lane == 0) a.pivots[po + k] = pt;
            }
            __syncthreads();
        }
        if (tid == 0) {
            a.rank[c] = rank;
            a.n_contra[c] = sContra;
            a.first_contra[c] = sFirst;
            a.ctx_flags[c] = sContra ? F2_CTX_CONTRADICTION : 0u;
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// encode tables: entry j of context c (stride 2 + hw words, hw = ceil((d-rank)/64)):
//   pivot column j  : [z_j | the bits of r_j at the free columns, compacted]
//   free column j   : [0   | the unit vector of j among the free columns]
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_enc_prepare(EncArgs e) {
    __shared__ uint64_t sFree[64];
    __shared__ int sFreeBefore[65];
    __shared__ int16_t sSlot[F2_MAX_N_BITS + 1];
    const int c = blockIdx.x, lane = threadIdx.x;
    if (e.ctx_flags[c] & kBadCtx) return;
    const int n = e.n_bits[c];
    const int fw = feat_words(n), W = fw + F2_Y_WORDS, d = n + 1;
    const int r = min(max(e.rank[c], 0), d);  // a model from f2_fit_batch always satisfies 0 <= rank <= d
    const int hw = (d - r + 63) >> 6, ES = 2 + hw;
    const uint64_t* B = e.basis + e.basis_off[c];
    const int32_t* piv = e.pivots + e.piv_off[c];
    uint64_t* T = e.tables + e.basis_off[c];
    const uint64_t tmask = top_mask(n, fw);
    for (int w = lane; w < fw; w += 64) sFree[w] = (w == fw - 1) ? tmask : ~0ull;
    for (int j = lane; j < d; j += 64) sSlot[j] = -1;
    __syncthreads();
    for (int k = lane; k < r; k += 64) {
        const int p = min(max(piv[k], 0), n);
        sSlot[p] = static_cast<int16_t>(k);
        atomicAnd(reinterpret_cast<unsigned long long*>(&sFree[p >> 6]), ~(1ull << (p & 63)));
    }
    __syncthreads();
    if (lane == 0) {
        int acc = 0;
        for (int w = 0; w < fw; ++w) {
            sFreeBefore[w] = acc;
            acc += __popcll(sFree[w]);
        }
    }
    __syncthreads();
    for (int j = lane; j < d; j += 64) {
        uint64_t* ent = T + static_cast<int64_t>(j) * ES;
        for (int k = 0; k < hw; ++k) ent[2 + k] = 0;
        const int k = sSlot[j];
        if (k < 0) {
            ent[0] = 0;
            ent[1] = 0;
            const int w = j >> 6;
            const int idx = sFreeBefore[w] + __popcll(sFree[w] & ((1ull << (j & 63)) - 1));
            ent[2 + (idx >> 6)] |= 1ull << (idx & 63);
        } else {
            const uint64_t* row = B + static_cast<int64_t>(k) * W;
            ent[0] = row[fw];
            ent[1] = row[fw + 1];
            for (int w = 0; w < fw; ++w) {
                uint64_t v = row[w] & sFree[w];
                while (v) {
                    const int b = ffs64(v);
                    v &= v - 1;
                    const int idx = sFreeBefore[w] + __popcll(sFree[w] & ((1ull << b) - 1));
                    ent[2 + (idx >> 6)] |= 1ull << (idx & 63);
                }
            }
        }
    }
}

// encode: one lane per query
__global__ __launch_bounds__(kEncThreads) void k_encode(EncArgs e) {
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kEncThreads + threadIdx.x;
    if (q >= e.nq) return;
    const int c = e.ctx_id[q];
    uint64_t z0 = 0, z1 = 0;
    uint8_t fl = 0;
    if (c < 0 || c >= e.num_ctx || (e.ctx_flags[c] & kBadCtx)) {
        fl = F2_Q_BAD_CTX;
    } else {
        if (e.ctx_flags[c] & F2_CTX_CONTRADICTION) fl = F2_Q_CTX_CONTRADICTORY;
        const int n = e.n_bits[c];
        const int fw = feat_words(n), d = n + 1;
        const int hw = (d - min(max(e.rank[c], 0), d) + 63) >> 6, ES = 2 + hw;
        const uint64_t* T = e.tables + e.basis_off[c];
        const uint64_t* xq = e.x + q * e.stride;
        bool outside = false;
        for (int w = 0; w < e.stride; ++w) {
            const int lo = 64 * w;
            const uint64_t v = xq[w];
            if (lo >= n) outside |= (v != 0);
            else if (n - lo < 64) outside |= (v >> (n - lo)) != 0;
        }
        if (outside) {
            fl |= F2_Q_OUT_OF_SPAN;
        } else {
            bool inspan = true;
            const int xw = e.stride < fw ? e.stride : fw;
            for (int h0 = 0; h0 < (hw > 0 ? hw : 1); h0 += kEncHW) {
                uint64_t h[kEncHW];
#pragma unroll
                for (int k = 0; k < kEncHW; ++k) h[k] = 0;
                const bool first = (h0 == 0);
                const int hn = (hw - h0) < kEncHW ? (hw - h0) : kEncHW;
                // constant feature (storage bit n) is always set
                {
                    const uint64_t* ent = T + static_cast<int64_t>(n) * ES;
                    if (first) {
                        z0 ^= ent[0];
                        z1 ^= ent[1];
                    }
#pragma unroll
                    for (int k = 0; k < kEncHW; ++k)
                        if (k < hn) h[k] ^= ent[2 + h0 + k];
                }
                for (int w = 0; w < xw; ++w) {
                    uint64_t v = xq[w];
                    while (v) {
                        const int j = 64 * w + ffs64(v);
                        v &= v - 1;
                        const uint64_t* ent = T + static_cast<int64_t>(j) * ES;
                        if (first) {
                            z0 ^= ent[0];
                            z1 ^= ent[1];
                        }
#pragma unroll
                        for (int k = 0; k < kEncHW; ++k)
                            if (k < hn) h[k] ^= ent[2 + h0 + k];
                    }
                }
#pragma unroll
                for (int k = 0; k < kEncHW; ++k) inspan &= (h[k] == 0);
            }
            if (!inspan) {
                fl |= F2_Q_OUT_OF_SPAN;
                z0 = z1 = 0;
            }
        }
    }
    if (fl & (F2_Q_BAD_CTX | F2_Q_OUT_OF_SPAN)) z0 = z1 = 0;
    e.words[2 * q] = z0;
    e.words[2 * q + 1] = z1;
    e.qflags[q] = fl;
}

inline size_t align256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

int grid_for_class(int cls, int num_ctx) {
    static const int caps[kClasses] = {4096, 4096, 2048, 1024, 512};
    int g = caps[cls];
    return num_ctx < g ? (num_ctx > 0 ? num_ctx : 1) : g;
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
    return 256 + align256(sizeof(int32_t) * static_cast<size_t>(kClasses) * static_cast<size_t>(num_ctx));
}

int f2_fit_batch(const uint64_t* rows, int64_t rows_words, const int64_t* row_off, const f2_model* m,
                 void* workspace, size_t workspace_bytes, void* stream) {
    if (!m || m->num_ctx < 0 || rows_words < 0) return F2_EINVAL;
    const int32_t C = m->num_ctx;
    if (C == 0) return F2_OK;
    if (!row_off || !m->n_bits || !m->basis_off || !m->piv_off || !m->map_off || !m->basis || !m->pivots ||
        !m->maps || !m->rank || !m->ctx_flags || !m->n_contra || !m->first_contra_row || (rows_words > 0 && !rows) ||
        m->basis_words < 0 || m->piv_entries < 0 || m->map_words < 0)
        return F2_EINVAL;
    if (!workspace || workspace_bytes < f2_fit_workspace_bytes(C) ||
        (reinterpret_cast<uintptr_t>(workspace) & 255u))
        return F2_EWORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    FitArgs a;
    a.rows = rows;
    a.rows_words = rows_words;
    a.row_off = row_off;
    a.num_ctx = C;
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
    a.rank = m->rank;
    a.ctx_flags = m->ctx_flags;
    a.n_contra = m->n_contra;
    a.first_contra = m->first_contra_row;
    a.counters = static_cast<int32_t*>(workspace);
    a.lists = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + 256);

    hipLaunchKernelGGL(k_fit_init, dim3(1), dim3(64), 0, s, a.counters);
    hipLaunchKernelGGL(k_fit_plan, dim3((C + 255) / 256), dim3(256), 0, s, a);
    hipLaunchKernelGGL(k_fit_small<1>, dim3(grid_for_class(0, C)), dim3(64), 0, s, a, 0);
    hipLaunchKernelGGL(k_fit_small<2>, dim3(grid_for_class(1, C)), dim3(64), 0, s, a, 1);
    hipLaunchKernelGGL(k_fit_small<4>, dim3(grid_for_class(2, C)), dim3(64), 0, s, a, 2);
    hipLaunchKernelGGL(k_fit_small<8>, dim3(grid_for_class(3, C)), dim3(64), 0, s, a, 3);
    hipLaunchKernelGGL(k_fit_large, dim3(grid_for_class(4, C)), dim3(kLargeThreads), 0, s, a, 4);
    return hipGetLastError() == hipSuccess ? F2_OK : F2_EDEVICE;
}

size_t f2_encode_workspace_bytes(const f2_model* m) {
    if (!m || m->basis_words < 0) return 0;
    return align256(sizeof(uint64_t) * static_cast<size_t>(m->basis_words)) + 256;
}

int f2_encode_batch(const f2_model* m, const int32_t* ctx_id, const uint64_t* x, int32_t x_stride_words,
                    int64_t num_queries, uint64_t* words_out, uint8_t* qflags_out, void* workspace,
                    size_t workspace_bytes, void* stream) {
    if (!m || m->num_ctx < 0 || num_queries < 0 || x_stride_words < 1) return F2_EINVAL;
    if (num_queries == 0) return F2_OK;
    if (!ctx_id || !x || !words_out || !qflags_out) return F2_EINVAL;
    if (m->num_ctx > 0 && (!m->n_bits || !m->basis_off || !m->piv_off || !m->basis || !m->pivots || !m->rank ||
                           !m->ctx_flags))
        return F2_EINVAL;
    if (!workspace || workspace_bytes < f2_encode_workspace_bytes(m) ||
        (reinterpret_cast<uintptr_t>(workspace) & 255u))
        return F2_EWORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    EncArgs e;
    e.num_ctx = m->num_ctx;
    e.n_bits = m->n_bits;
    e.basis_off = m->basis_off;
    e.piv_off = m->piv_off;
    e.basis = m->basis;
    e.pivots = m->pivots;
    e.rank = m->rank;
    e.ctx_flags = m->ctx_flags;
    e.tables = static_cast<uint64_t*>(workspace);
    e.ctx_id = ctx_id;
    e.x = x;
    e.stride = x_stride_words;
    e.nq = num_queries;
    e.words = words_out;
    e.qflags = qflags_out;
    if (m->num_ctx > 0) hipLaunchKernelGGL(k_enc_prepare, dim3(m->num_ctx), dim3(64), 0, s, e);
    const int64_t blocks = (num_queries + kEncThreads - 1) / kEncThreads;
    if (blocks > 0x7fffffff) return F2_EINVAL;
    hipLaunchKernelGGL(k_encode, dim3(static_cast<unsigned>(blocks)), dim3(kEncThreads), 0, s, e);
    return hipGetLastError() == hipSuccess ? F2_OK : F2_EDEVICE;
}

}  // extern "C"
