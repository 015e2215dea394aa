/*
 * Seeded synthetic workloads for the GF(2) affine-map learner.
 *
 * This module only draws data: context widths, row counts, planted affine
 * maps, feature vectors from full or rank-deficient subspaces, injected
 * contradictions and query streams.  The training output of a row is the
 * planted map evaluated on its feature vector (the data model of the
 * encoding equation, Sec. 2.1, Eq. 2); nothing here eliminates, reduces or
 * encodes.  Both the CPU oracle and the GPU library are fed from these
 * buffers, so the generator shares no code with either of them.
 *
 * Randomness: splitmix64 (Steele, Lea and Flood, 2014) used counter-style.
 * Every context and every query owns a key derived from the run seed, so any
 * prefix of contexts or queries is reproducible on its own and OpenMP
 * threads produce identical bytes regardless of scheduling.
 *
 * Row storage (little-endian uint64 words), for a context of input width n:
 *   fw = ceil((n + 1) / 64) feature words holding x_0..x_{n-1} at storage
 *   bits 0..n-1 and the constant feature at storage bit n, then two words of
 *   the 128-bit output y (bits 0-63, then 64-127).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define GAMMA 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}
/* i-th draw of the stream identified by key */
static inline uint64_t draw_at(uint64_t key, uint64_t i) { return mix64(key + (i + 1) * GAMMA); }
/* independent child key */
static inline uint64_t child(uint64_t key, uint64_t tag) { return mix64(key ^ mix64(tag * GAMMA + 0x5851F42D4C957F2DULL)); }

typedef struct { uint64_t key, ctr; } stream_t;
static inline uint64_t next(stream_t* s) { return draw_at(s->key, s->ctr++); }
static inline uint64_t below(stream_t* s, uint64_t range) {
    return (uint64_t)(((unsigned __int128)next(s) * range) >> 64);
}
static inline double unit_open(stream_t* s) { /* in (0,1) */
    return ((double)(next(s) >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}

enum { TAG_SHAPE = 1, TAG_MAP = 2, TAG_SUB = 3, TAG_ROWS = 4, TAG_CONTRA = 5 };
enum { KIND_FULL = 0, KIND_RESERVED = 1, KIND_SUBSPACE = 2 };

static int cfg_kind(int cfg) {
    switch (cfg) {
        case 1: case 2: return KIND_RESERVED;
        case 3: return KIND_SUBSPACE;
        default: return KIND_FULL;
    }
}

static inline int feat_words(int n) { return (n + 1 + 63) / 64; }

/*
 * Per-context shapes.
 *   cfg 1: n = 33 (x_0..x_31 drawn, x_32 reserved), 200 rows.
 *   cfg 2: 16..96 drawn input bits plus one reserved top bit, rows = 2 (active + 1),
 *          one injected contradiction with probability 5%.
 *   cfg 3: n = 8 + Geometric(1/33) redrawn while > 256, rows = clip(round(exp(N(ln 30, 1.5^2))), 1, 4000),
 *          injected contradiction with probability 1% when rows >= 2.
 *   cfg 4: n = 4095, 8192 rows.
 */
int syn_shapes(int cfg, uint64_t seed, int32_t num_ctx, int32_t* n_bits, int64_t* m_rows, uint8_t* contra) {
    if (cfg < 1 || cfg > 4 || num_ctx < 0) return -1;
    for (int32_t c = 0; c < num_ctx; ++c) {
        stream_t s = {child(child(seed, (uint64_t)c), TAG_SHAPE), 0};
        int n = 0; int64_t m = 0; int inj = 0;
        if (cfg == 1) { n = 33; m = 200; }
        else if (cfg == 2) {
            int active = 16 + (int)below(&s, 81);
            n = active + 1; m = 2 * (int64_t)(active + 1);
            inj = unit_open(&s) < 0.05;
        } else if (cfg == 3) {
            const double lq = log1p(-1.0 / 33.0);
            do {
                double g = floor(log(unit_open(&s)) / lq);
                n = 8 + (g > 1e6 ? 1000000 : (int)g);
            } while (n > 256);
            double u1 = unit_open(&s), u2 = unit_open(&s);
            double z = sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2);
            double r = floor(exp(log(30.0) + 1.5 * z) + 0.5);
            if (r < 1) r = 1;
            if (r > 4000) r = 4000;
            m = (int64_t)r;
            double u3 = unit_open(&s);
            inj = (m >= 2) && (u3 < 0.01);
        } else { n = 4095; m = 8192; }
        n_bits[c] = n; m_rows[c] = m; contra[c] = (uint8_t)inj;
    }
    return 0;
}

/* subspace structure of a cfg-3 context: x = P [s ; B s], s in F2^k, k = ceil(0.7 n) */
typedef struct { int n, k; int perm[256]; uint64_t B[256][3]; } subspace_t;

static void make_subspace(uint64_t ckey, int n, subspace_t* S) {
    stream_t s = {child(ckey, TAG_SUB), 0};
    S->n = n; S->k = (7 * n + 9) / 10;
    for (int i = 0; i < n; ++i) S->perm[i] = i;
    for (int i = n - 1; i > 0; --i) { int j = (int)below(&s, (uint64_t)i + 1); int t = S->perm[i]; S->perm[i] = S->perm[j]; S->perm[j] = t; }
    int kw = (S->k + 63) / 64;
    for (int t = 0; t < n - S->k; ++t)
        for (int w = 0; w < 3; ++w) {
            uint64_t v = w < kw ? next(&s) : 0;
            int hi = S->k - 64 * w;
            if (hi < 64) v = hi <= 0 ? 0 : (v & ((1ULL << hi) - 1));
            S->B[t][w] = v;
        }
}

static inline void setbit(uint64_t* v, int i) { v[i >> 6] |= 1ULL << (i & 63); }
static inline int getbit(const uint64_t* v, int i) { return (int)((v[i >> 6] >> (i & 63)) & 1ULL); }

/* draw the x bits (storage bits 0..n-1) of one training row */
static void draw_x(int kind, int n, const subspace_t* S, stream_t* s, uint64_t* x, int fw) {
    memset(x, 0, sizeof(uint64_t) * (size_t)fw);
    if (kind == KIND_SUBSPACE) {
        uint64_t sv[3] = {0, 0, 0};
        for (int w = 0; w < (S->k + 63) / 64; ++w) sv[w] = next(s);
        int hi = S->k & 63;
        if (hi) sv[(S->k - 1) / 64] &= (1ULL << hi) - 1;
        for (int i = 0; i < S->k; ++i) if (getbit(sv, i)) setbit(x, S->perm[i]);
        for (int t = 0; t < n - S->k; ++t) {
            int par = __builtin_popcountll(S->B[t][0] & sv[0]) + __builtin_popcountll(S->B[t][1] & sv[1]) +
                      __builtin_popcountll(S->B[t][2] & sv[2]);
            if (par & 1) setbit(x, S->perm[S->k + t]);
        }
    } else {
        int act = kind == KIND_RESERVED ? n - 1 : n;
        for (int w = 0; w < fw && 64 * w < act; ++w) {
            uint64_t v = next(s);
            int hi = act - 64 * w;
            if (hi < 64) v &= (1ULL << hi) - 1;
            x[w] = v;
        }
    }
}

/*
 * Fill training rows.  row_off[c] is the first uint64 word of context c.
 * contra_row[c] receives the in-context index of the injected contradictory
 * row (a copy of an earlier row's x with one output bit flipped), or -1.
 */
int syn_rows(int cfg, uint64_t seed, int32_t num_ctx, const int32_t* n_bits, const int64_t* m_rows,
             const uint8_t* contra, const int64_t* row_off, uint64_t* rows, int64_t* contra_row) {
    if (cfg < 1 || cfg > 4) return -1;
    const int kind = cfg_kind(cfg);
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(| : bad)
    for (int32_t c = 0; c < num_ctx; ++c) {
        const int n = n_bits[c], fw = feat_words(n), W = fw + 2;
        const int64_t m = m_rows[c];
        const uint64_t ckey = child(seed, (uint64_t)c);
        if (kind == KIND_SUBSPACE && n > 256) { bad = 1; continue; }
        /* planted affine map: w_i for x_i (i < n) and the bias w_n, 128 bits each */
        uint64_t* Wp = (uint64_t*)malloc(sizeof(uint64_t) * 2 * (size_t)(n + 1));
        stream_t sm = {child(ckey, TAG_MAP), 0};
        for (int i = 0; i <= n; ++i) { Wp[2 * i] = next(&sm); Wp[2 * i + 1] = next(&sm); }
        subspace_t* S = NULL;
        if (kind == KIND_SUBSPACE) { S = (subspace_t*)malloc(sizeof(subspace_t)); make_subspace(ckey, n, S); }
        stream_t sr = {child(ckey, TAG_ROWS), 0};
        uint64_t* base = rows + row_off[c];
        for (int64_t r = 0; r < m; ++r) {
            uint64_t* row = base + r * W;
            draw_x(kind, n, S, &sr, row, fw);
            uint64_t y0 = Wp[2 * n], y1 = Wp[2 * n + 1];
            for (int i = 0; i < n; ++i)
                if (getbit(row, i)) { y0 ^= Wp[2 * i]; y1 ^= Wp[2 * i + 1]; }
            setbit(row, n); /* constant feature */
            row[fw] = y0; row[fw + 1] = y1;
        }
        contra_row[c] = -1;
        if (contra[c] && m >= 2) {
            stream_t sc = {child(ckey, TAG_CONTRA), 0};
            int64_t j = 1 + (int64_t)below(&sc, (uint64_t)(m - 1));
            int64_t i = (int64_t)below(&sc, (uint64_t)j);
            int b = (int)below(&sc, 128);
            memcpy(base + j * W, base + i * W, sizeof(uint64_t) * (size_t)W);
            base[j * W + fw + (b >> 6)] ^= 1ULL << (b & 63);
            contra_row[c] = j;
        }
        free(S);
        free(Wp);
    }
    return bad ? -2 : 0;
}

/*
 * Queries.  Context choice: uniform (zipf_s <= 0) or Zipf(zipf_s) over ranks
 * mapped through a seeded permutation of context ids.  An in-span query is
 * the XOR of three training feature vectors of its context (odd count, so the
 * constant feature stays 1), which lies in the training span by construction.
 * With probability out_frac it is pushed out of the span:
 *   reserved-bit contexts: set the reserved top input bit;
 *   subspace contexts: flip one coordinate that is a dependent coordinate of
 *   the context's subspace (no vector of the subspace differs from another in
 *   that coordinate alone).
 * x is written with `stride` words per query (x bits only, no constant).
 * planted_out[i] = 1 when the query was built outside the span.
 */
int syn_queries(int cfg, uint64_t seed, int32_t num_ctx, const int32_t* n_bits, const int64_t* m_rows,
                const int64_t* row_off, const uint64_t* rows, int64_t nq, int32_t stride, double out_frac,
                double zipf_s, int32_t* ctx_id, uint64_t* x, uint8_t* planted_out) {
    if (cfg < 1 || cfg > 4 || num_ctx <= 0 || stride < 1) return -1;
    for (int32_t c = 0; c < num_ctx; ++c)
        if ((n_bits[c] + 63) / 64 > stride) return -3;
    const int kind = cfg_kind(cfg);
    const uint64_t qkey = child(seed, 0xABCDEF0123ULL);
    int32_t* perm = NULL;
    double* cdf = NULL;
    int32_t* guide = NULL;
    const int G = 1 << 16;
    if (zipf_s > 0) {
        perm = (int32_t*)malloc(sizeof(int32_t) * (size_t)num_ctx);
        for (int32_t i = 0; i < num_ctx; ++i) perm[i] = i;
        stream_t sp = {child(qkey, 1), 0};
        for (int32_t i = num_ctx - 1; i > 0; --i) { int32_t j = (int32_t)below(&sp, (uint64_t)i + 1); int32_t t = perm[i]; perm[i] = perm[j]; perm[j] = t; }
        cdf = (double*)malloc(sizeof(double) * (size_t)num_ctx);
        double acc = 0;
        for (int32_t r = 0; r < num_ctx; ++r) { acc += pow((double)(r + 1), -zipf_s); cdf[r] = acc; }
        for (int32_t r = 0; r < num_ctx; ++r) cdf[r] /= acc;
        cdf[num_ctx - 1] = 1.0;
        guide = (int32_t*)malloc(sizeof(int32_t) * (size_t)(G + 1));
        int32_t r = 0;
        for (int g = 0; g <= G; ++g) { double t = (double)g / G; while (r < num_ctx - 1 && cdf[r] < t) ++r; guide[g] = r; }
    }
    int bad = 0;
#pragma omp parallel
    {
        subspace_t* S = (subspace_t*)malloc(sizeof(subspace_t));
        int32_t cached = -1;
#pragma omp for schedule(static, 65536) reduction(| : bad)
        for (int64_t q = 0; q < nq; ++q) {
            stream_t s = {qkey, (uint64_t)q * 8};
            int32_t c;
            if (zipf_s > 0) {
                double u = unit_open(&s);
                int32_t r = guide[(int)(u * G)];
                while (r < num_ctx - 1 && cdf[r] < u) ++r;
                c = perm[r];
            } else c = (int32_t)below(&s, (uint64_t)num_ctx);
            const int n = n_bits[c], fw = feat_words(n), W = fw + 2;
            const int64_t m = m_rows[c];
            uint64_t* xq = x + q * stride;
            for (int w = 0; w < stride; ++w) xq[w] = 0;
            int out = 0;
            if (m > 0) {
                const uint64_t* base = rows + row_off[c];
                for (int t = 0; t < 3; ++t) {
                    const uint64_t* row = base + (int64_t)below(&s, (uint64_t)m) * W;
                    for (int w = 0; w < fw && w < stride; ++w) xq[w] ^= row[w];
                }
                /* strip the constant feature: only x_0..x_{n-1} are query bits */
                if ((n >> 6) < stride) xq[n >> 6] &= ~(1ULL << (n & 63));
            } else out = 1;
            if (unit_open(&s) < out_frac) {
                if (kind == KIND_RESERVED) { xq[(n - 1) >> 6] |= 1ULL << ((n - 1) & 63); out = 1; }
                else if (kind == KIND_SUBSPACE) {
                    if (cached != c) { make_subspace(child(seed, (uint64_t)c), n, S); cached = c; }
                    if (n > S->k) {
                        int j = S->perm[S->k + (int)below(&s, (uint64_t)(n - S->k))];
                        xq[j >> 6] ^= 1ULL << (j & 63);
                        out = 1;
                    }
                } else bad = 1;
            }
            ctx_id[q] = c;
            if (planted_out) planted_out[q] = (uint8_t)out;
        }
        free(S);
    }
    free(perm); free(cdf); free(guide);
    return bad ? -2 : 0;
}
