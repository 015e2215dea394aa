/*
 * f2_oracle.c -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT PATH.
 *
 * A plain, single-threaded, deliberately slow CPU reference of the GF(2)
 * affine-map learner of F2Asm ("Learning Exact NVIDIA SASS Encoders with F2
 * Linear Algebra").  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load it.  It shares no code, header or table with the
 * GPU library: it is written from the paper alone.
 *
 *   fit    -- streaming Gaussian elimination over GF(2), Sec. 2.2 (Eq. 5 and
 *             the five per-row steps that follow it), worked through in App. B.
 *   encode -- reduction of a query against the retained basis with an output
 *             accumulator, Sec. 2.3 (Eqs. 6-9 and the encoding paragraph after
 *             them), App. B query traces.
 *
 * Storage convention of one context of input width n (d = n + 1 features):
 *   fw = ceil(d / 64) feature words, storage bit i < n holds x_i, storage bit
 *   n holds the constant feature, higher bits of the last feature word are
 *   padding; then 2 words of the 128-bit output (bits 0-63, then 64-127).
 * Pivot priority is the paper's feature index of Eq. 1, phi = [1 | bits(x)]:
 * the constant has index 0 and x_i has index i + 1, so the highest-priority
 * bit is x_{n-1} and the constant comes last.
 *
 * Readings where the paper is silent (listed with reasons in the design notes):
 *   - after a contradiction the row is discarded and fitting continues; the
 *     context is flagged, the count and the first such row are reported;
 *   - the canonical dense map has column p = z_p for every pivot p and zero
 *     columns elsewhere (the paper allows any linear extension, Sec. 2.3);
 *   - an unsupported query yields a zero word plus a flag;
 *   - query bits at or above the context width lie outside its ambient space
 *     and make the query unsupported;
 *   - padding bits of training rows are ignored.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_Y_WORDS 2
#define OR_MAX_N 4095

/* per-context flags (same values as documented in the library header, defined here independently) */
#define OR_CTX_CONTRADICTION 1u
#define OR_CTX_BAD_SEGMENT 2u
#define OR_CTX_BAD_WIDTH 4u
#define OR_CTX_BAD_OUTPUT 8u
/* per-query flags */
#define OR_Q_OUT_OF_SPAN 1u
#define OR_Q_CTX_CONTRADICTORY 2u
#define OR_Q_BAD_CTX 4u

static int feature_words(int n) { return (n + 1 + 63) / 64; }
static int bit_of(const uint64_t* v, int i) { return (int)((v[i / 64] >> (i % 64)) & 1u); }
static void xor_into(uint64_t* dst, const uint64_t* src, int words) {
    for (int w = 0; w < words; ++w) dst[w] ^= src[w];
}
static int all_zero(const uint64_t* v, int words) {
    for (int w = 0; w < words; ++w)
        if (v[w]) return 0;
    return 1;
}

/* Storage bit visited t-th in descending priority: x_{n-1}, ..., x_0, then the constant. */
static int storage_at_priority(int n, int t) { return t < n ? n - 1 - t : n; }

/* Highest-priority set feature bit of r (storage index), or -1 when the feature part is zero. */
static int highest_feature(const uint64_t* r, int n) {
    for (int t = 0; t <= n; ++t) {
        int s = storage_at_priority(n, t);
        if (bit_of(r, s)) return s;
    }
    return -1;
}

/*
 * Fit one context from m rows in stream order.
 * Outputs: basis rows [0, rank) in descending pivot priority (fw + 2 words
 * each), their pivots (storage bit index), the canonical map (d columns of 2
 * words, column j = storage bit j), contradiction count and first
 * contradictory row (-1 if none).  Returns the rank.
 */
int oracle_fit_context(const uint64_t* rows, int64_t m, int n, uint64_t* basis_out, int32_t* pivots_out,
                       uint64_t* map_out, int32_t* n_contra, int64_t* first_contra) {
    const int fw = feature_words(n), W = fw + OR_Y_WORDS, d = n + 1;
    /* retained basis indexed by pivot: B[k] = (r_k, z_k) */
    uint64_t* B = (uint64_t*)calloc((size_t)d * W, sizeof(uint64_t));
    char* present = (char*)calloc((size_t)d, 1);
    uint64_t* cur = (uint64_t*)malloc(sizeof(uint64_t) * W);
    const int valid_top = d - 64 * (fw - 1); /* meaningful bits in the last feature word */
    const uint64_t top_mask = valid_top == 64 ? ~0ULL : ((1ULL << valid_top) - 1);
    int rank = 0;
    *n_contra = 0;
    *first_contra = -1;

    for (int64_t i = 0; i < m; ++i) {
        memcpy(cur, rows + i * W, sizeof(uint64_t) * W);
        cur[fw - 1] &= top_mask;
        /* (1) XOR-reduce against the stored pivots, highest priority first */
        for (int t = 0; t <= n; ++t) {
            int k = storage_at_priority(n, t);
            if (present[k] && bit_of(cur, k)) xor_into(cur, B + (size_t)k * W, W);
        }
        int p = highest_feature(cur, n);
        if (p < 0) {
            /* (2) zero/zero residual: redundant.  (3) zero/nonzero: contradiction. */
            if (!all_zero(cur + fw, OR_Y_WORDS)) {
                if (*n_contra == 0) *first_contra = i;
                ++*n_contra;
            }
            continue;
        }
        /* (4) pivot = highest set input bit; (5) clear it from stored rows, then insert */
        for (int k = 0; k < d; ++k)
            if (present[k] && bit_of(B + (size_t)k * W, p)) xor_into(B + (size_t)k * W, cur, W);
        memcpy(B + (size_t)p * W, cur, sizeof(uint64_t) * W);
        present[p] = 1;
        ++rank;
    }

    int out = 0;
    for (int t = 0; t <= n; ++t) {
        int k = storage_at_priority(n, t);
        if (!present[k]) continue;
        memcpy(basis_out + (size_t)out * W, B + (size_t)k * W, sizeof(uint64_t) * W);
        pivots_out[out] = k;
        ++out;
    }
    for (int j = 0; j < d; ++j) {
        map_out[2 * j] = present[j] ? B[(size_t)j * W + fw] : 0;
        map_out[2 * j + 1] = present[j] ? B[(size_t)j * W + fw + 1] : 0;
    }
    free(cur);
    free(present);
    free(B);
    return rank;
}

/*
 * Reduce an explicit feature vector q (fw words, storage layout, constant bit
 * included as given) by a fitted basis whose rows are in descending pivot
 * priority.  Every XOR of r_k into the residual XORs z_k into the accumulator.
 * Returns 1 when the residual is zero (q in the training span), else 0.
 */
int oracle_reduce_query(const uint64_t* basis, const int32_t* pivots, int rank, int n, const uint64_t* q,
                        uint64_t* acc_out, uint64_t* residual_out) {
    const int fw = feature_words(n), W = fw + OR_Y_WORDS;
    memcpy(residual_out, q, sizeof(uint64_t) * fw);
    acc_out[0] = acc_out[1] = 0;
    for (int k = 0; k < rank; ++k) {
        if (!bit_of(residual_out, pivots[k])) continue;
        xor_into(residual_out, basis + (size_t)k * W, fw);
        xor_into(acc_out, basis + (size_t)k * W + fw, OR_Y_WORDS);
    }
    return all_zero(residual_out, fw);
}

/* Segment/offset validation shared by the batch fit; returns per-context flags. */
static uint32_t check_context(int32_t c, const int64_t* row_off, int64_t rows_words, const int32_t* n_bits,
                              const int64_t* basis_off, int64_t basis_words, const int64_t* piv_off,
                              int64_t piv_entries, const int64_t* map_off, int64_t map_words, int64_t* m_out) {
    const int n = n_bits[c];
    *m_out = 0;
    if (n < 0 || n > OR_MAX_N) return OR_CTX_BAD_WIDTH;
    const int d = n + 1, W = feature_words(n) + OR_Y_WORDS;
    if (basis_off[c] < 0 || basis_off[c] + (int64_t)d * W > basis_words || piv_off[c] < 0 ||
        piv_off[c] + d > piv_entries || map_off[c] < 0 || map_off[c] + 2 * (int64_t)d > map_words)
        return OR_CTX_BAD_OUTPUT;
    int64_t a = row_off[c], b = row_off[c + 1];
    if (a < 0 || b < a || b > rows_words || (b - a) % W != 0) return OR_CTX_BAD_SEGMENT;
    *m_out = (b - a) / W;
    return 0;
}

/*
 * Fit every context of a batch.  Offsets are in uint64 words (rows, basis,
 * maps) or int32 entries (pivots), as produced by the layout rule
 * basis capacity (n+1)(fw+2) words, pivot capacity n+1, map 2(n+1) words.
 */
void oracle_fit_batch(const uint64_t* rows, int64_t rows_words, const int64_t* row_off, const int32_t* n_bits,
                      int32_t num_ctx, const int64_t* basis_off, int64_t basis_words, const int64_t* piv_off,
                      int64_t piv_entries, const int64_t* map_off, int64_t map_words, uint64_t* basis,
                      int32_t* pivots, uint64_t* maps, int32_t* rank, uint32_t* ctx_flags, int32_t* n_contra,
                      int64_t* first_contra) {
    for (int32_t c = 0; c < num_ctx; ++c) {
        int64_t m = 0;
        uint32_t f = check_context(c, row_off, rows_words, n_bits, basis_off, basis_words, piv_off, piv_entries,
                                   map_off, map_words, &m);
        rank[c] = 0;
        n_contra[c] = 0;
        first_contra[c] = -1;
        ctx_flags[c] = f;
        if (f & (OR_CTX_BAD_WIDTH | OR_CTX_BAD_OUTPUT)) continue;
        const int n = n_bits[c];
        if (f & OR_CTX_BAD_SEGMENT) {
            memset(maps + map_off[c], 0, sizeof(uint64_t) * 2 * (size_t)(n + 1));
            continue;
        }
        int32_t nc;
        int64_t fc;
        rank[c] = oracle_fit_context(rows + row_off[c], m, n, basis + basis_off[c], pivots + piv_off[c],
                                     maps + map_off[c], &nc, &fc);
        n_contra[c] = nc;
        first_contra[c] = fc;
        if (nc > 0) ctx_flags[c] |= OR_CTX_CONTRADICTION;
    }
}

/*
 * Encode a batch of queries (Sec. 2.3).  Query i names context ctx_id[i] and
 * carries x in x[i*stride .. i*stride+stride); the feature vector is
 * q = [x | 1].  A query whose context id is out of range or whose context
 * could not be fitted gets a zero word and OR_Q_BAD_CTX.
 */
void oracle_encode_batch(int32_t num_ctx, const int32_t* n_bits, const int64_t* basis_off, const int64_t* piv_off,
                         const uint64_t* basis, const int32_t* pivots, const int32_t* rank,
                         const uint32_t* ctx_flags, const int32_t* ctx_id, const uint64_t* x, int32_t stride,
                         int64_t num_queries, uint64_t* words_out, uint8_t* qflags_out) {
    uint64_t q[OR_MAX_N / 64 + 1], res[OR_MAX_N / 64 + 1], acc[2];
    for (int64_t i = 0; i < num_queries; ++i) {
        const int32_t c = ctx_id[i];
        const uint64_t* xq = x + i * stride;
        words_out[2 * i] = words_out[2 * i + 1] = 0;
        if (c < 0 || c >= num_ctx || (ctx_flags[c] & (OR_CTX_BAD_SEGMENT | OR_CTX_BAD_WIDTH | OR_CTX_BAD_OUTPUT))) {
            qflags_out[i] = OR_Q_BAD_CTX;
            continue;
        }
        uint8_t fl = (ctx_flags[c] & OR_CTX_CONTRADICTION) ? OR_Q_CTX_CONTRADICTORY : 0;
        const int n = n_bits[c], fw = feature_words(n);
        int outside = 0;
        for (int b = n; b < 64 * stride; ++b)
            if (bit_of(xq, b)) outside = 1;
        if (outside) {
            qflags_out[i] = fl | OR_Q_OUT_OF_SPAN;
            continue;
        }
        memset(q, 0, sizeof(uint64_t) * fw);
        for (int b = 0; b < n && b < 64 * stride; ++b) /* bits past the stride are zero */
            if (bit_of(xq, b)) q[b / 64] |= 1ULL << (b % 64);
        q[n / 64] |= 1ULL << (n % 64); /* constant feature of Eq. 1 */
        if (oracle_reduce_query(basis + basis_off[c], pivots + piv_off[c], rank[c], n, q, acc, res)) {
            words_out[2 * i] = acc[0];
            words_out[2 * i + 1] = acc[1];
            qflags_out[i] = fl;
        } else {
            qflags_out[i] = fl | OR_Q_OUT_OF_SPAN;
        }
    }
}
