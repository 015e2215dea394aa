/*
 * f2gpu.h -- C ABI of the MI355X (gfx950) GF(2) affine-map learner.
 *
 * Method: F2Asm, "Learning Exact NVIDIA SASS Encoders with F2 Linear Algebra".
 *   Fitting solves, for every encoding context, the training system Phi W = Y
 *   over GF(2) (Sec. 2.1, Eq. 3) by streaming Gaussian elimination on
 *   augmented rows [phi | y] (Sec. 2.2, Eq. 5): each row is reduced against
 *   the retained pivot basis, a zero-feature residual with a nonzero output
 *   is a contradiction (Eq. 8), otherwise its highest-priority feature bit
 *   becomes a new pivot, that pivot is cleared from the stored rows and the
 *   row is inserted.  Encoding reduces a query phi(x) by the stored rows and
 *   XORs their outputs; a nonzero residual proves the query lies outside the
 *   observed span S = rowspan(Phi) (Sec. 2.3, Eqs. 6-9).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every pointer argument is DEVICE memory allocated and owned by the
 *    caller unless its name ends in _host.  The library allocates nothing and
 *    keeps no state between calls beyond a per-device cache of how many
 *    workgroups of the wide-context fit can be resident at once (queried on
 *    first use) and the fixed per-device plan array of f2_fit_batch_noalloc
 *    (a file-scope device array, part of the loaded library); concurrent
 *    calls need distinct workspaces.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *    device work is enqueued on it; outputs are valid once it has synchronised.
 *  - A negative return value means nothing was enqueued (argument errors that
 *    the host can check, or a HIP launch failure).  Data conditions found on
 *    the device (contradictions, unsupported queries, malformed segments, bad
 *    context ids) are never errors: they are reported per context or per query.
 *
 * Row layout of a context with input width n (d = n + 1 features)
 * -----------------------------------------------------------------
 *  fw = ceil(d / 64) little-endian uint64 feature words, then 2 output words:
 *    storage bit i < n  : input bit x_i
 *    storage bit n      : the constant feature (the leading 1 of Eq. 1); it is
 *                         taken from the row as given, so linear systems such
 *                         as the worked example of App. B can be expressed
 *    bits above n       : padding, ignored
 *    word fw, fw + 1    : output y, bits 0-63 then 64-127 (a 128-bit word)
 *  Pivot priority follows the feature index of Eq. 1: the constant has index
 *  0 and x_i has index i + 1, so x_{n-1} has the highest priority and the
 *  constant the lowest.  A pivot is reported as its storage bit index.
 */
#ifndef F2GPU_H
#define F2GPU_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    F2_OK = 0,
    F2_EINVAL = -1,      /* null pointer, negative count, bad stride, ... */
    F2_EWORKSPACE = -2,  /* workspace missing or smaller than required */
    F2_EDEVICE = -3,     /* HIP error while enqueuing */
    F2_ETOOWIDE = -4,    /* host-side layout helper: a width above F2_MAX_N_BITS */
    F2_ESCRATCH = -5     /* f2_fit_batch_noalloc: more contexts than F2_NOALLOC_MAX_CTX */
} f2_status;

#define F2_MAX_N_BITS 4095 /* widest supported context: fw <= 64 feature words */
#define F2_Y_WORDS 2       /* the 128-bit output word */

/* per-context flags (ctx_flags) */
enum {
    F2_CTX_CONTRADICTION = 1u, /* n_contra > 0: some row had a zero-feature, nonzero-output residual */
    F2_CTX_BAD_SEGMENT = 2u,   /* row segment negative, past rows_words, or not a multiple of fw+2 words */
    F2_CTX_BAD_WIDTH = 4u,     /* n_bits outside [0, F2_MAX_N_BITS], or above a declared max_n_bits */
    F2_CTX_BAD_OUTPUT = 8u,    /* output offsets of this context fall outside the output buffers */
    F2_CTX_SYNC_TIMEOUT = 16u  /* a wide context fitted by several workgroups together: a bounded wait
                                  for the other workgroups gave up, so the outputs of this context
                                  are not trustworthy; encoding treats it like a malformed context.
                                  The wait bound is 2^24 polls; the environment variable
                                  F2GPU_GROUP_SPIN_LIMIT (read at every f2_fit_batch call) overrides
                                  it, 0 meaning "never wait" (a test hook for this report) */
};

/* per-query flags (qflags_out) */
enum {
    F2_Q_OUT_OF_SPAN = 1u,       /* phi(x) is not in the observed span: word is 0 */
    F2_Q_CTX_CONTRADICTORY = 2u, /* the context's training data held a contradiction */
    F2_Q_BAD_CTX = 4u            /* context id out of range, or context malformed or flagged
                                    F2_CTX_SYNC_TIMEOUT: word is 0 */
};

/*
 * Fit outputs, and the model that encoding reads.  A host struct holding
 * device pointers.  Per context c:
 *   basis[basis_off[c] ...]   rank[c] rows of fw+2 words in descending pivot
 *                             priority (capacity (n+1)(fw+2) words; rows past
 *                             the rank are scratch, their content unspecified)
 *   pivots[piv_off[c] ...]    rank[c] storage bit indices, same order
 *                             (capacity n+1 entries)
 *   maps[map_off[c] ...]      the canonical dense map: n+1 columns of 2 words,
 *                             column j = storage bit j; column p = z_p for every
 *                             pivot p and 0 for every other column (one linear
 *                             extension of T beyond the span, Sec. 2.3)
 *   tables[basis_off[c] ...]  parity-check rows read by f2_encode_batch, present
 *                             when t = n+1-rank <= rank: one row of fw words per
 *                             free (non-pivot) column f, in ascending f: h_f = e_f
 *                             plus e_p for every pivot p whose basis row holds
 *                             bit f (t rows, within the basis capacity).  phi lies
 *                             in the span exactly when every row has even overlap
 *                             with it.  When t > rank the region is not written
 *                             and encoding reduces phi by the basis rows instead.
 *   rank[c], ctx_flags[c], n_contra[c] (rows flagged contradictory),
 *   first_contra_row[c] (index within the context's segment, -1 if none).
 * For a contradictory context the stored map is defined by the rows kept in
 * stream order (each row independent of all earlier rows), which is what the
 * streaming elimination retains.
 */
typedef struct f2_model {
    int32_t num_ctx;
    const int32_t* n_bits;    /* [num_ctx] input width n of each context */
    const int64_t* basis_off; /* [num_ctx+1] uint64-word offsets into basis */
    const int64_t* piv_off;   /* [num_ctx+1] int32-entry offsets into pivots */
    const int64_t* map_off;   /* [num_ctx+1] uint64-word offsets into maps */
    int64_t basis_words;      /* size of basis in uint64 words */
    int64_t piv_entries;      /* size of pivots in int32 entries */
    int64_t map_words;        /* size of maps in uint64 words */
    uint64_t* basis;
    int32_t* pivots;
    uint64_t* maps;
    uint64_t* tables;         /* basis_words words */
    int32_t* rank;            /* [num_ctx] */
    uint32_t* ctx_flags;      /* [num_ctx] */
    int32_t* n_contra;        /* [num_ctx] */
    int64_t* first_contra_row;/* [num_ctx] */
    int32_t max_n_bits;       /* -1, or an upper bound on the widths n of the batch, known on the
                                 host: f2_fit_batch flags a wider context F2_CTX_BAD_WIDTH, and
                                 below 512 (every context within 8 feature words) it does not
                                 launch the wide-context kernel at all. */
} f2_model;

/*
 * Host helper: output offsets for a batch (num_ctx+1 entries each, caller-
 * allocated host arrays), packed in context order with the capacities above.
 * Returns F2_OK, F2_EINVAL (null pointer, num_ctx < 0) or F2_ETOOWIDE.
 */
int f2_fit_layout(const int32_t* n_bits_host, int32_t num_ctx, int64_t* basis_off_host, int64_t* piv_off_host,
                  int64_t* map_off_host);

/* Workspace bytes f2_fit_batch needs for num_ctx contexts (any widths): the
 * per-batch plan that sorts contexts into kernel classes. */
size_t f2_fit_workspace_bytes(int32_t num_ctx);

/*
 * Fit every context of a batch (Sec. 2.2).
 *   rows      [rows_words] packed rows (layout above); context c owns the words
 *             rows[row_off[c] .. row_off[c+1]), i.e. (row_off[c+1]-row_off[c])/(fw+2)
 *             rows, processed in stream order
 *   row_off   [num_ctx+1] uint64-word offsets
 *   model     outputs; model->num_ctx contexts, model->n_bits their widths
 *   workspace at least f2_fit_workspace_bytes(num_ctx) bytes, 256-byte aligned
 * Returns F2_OK, F2_EINVAL, F2_EWORKSPACE or F2_EDEVICE.  Contexts are
 * independent; results do not depend on launch geometry.
 */
int f2_fit_batch(const uint64_t* rows, int64_t rows_words, const int64_t* row_off, const f2_model* model_host,
                 void* workspace, size_t workspace_bytes, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): f2_fit_batch without a
 * workspace.  The per-batch plan lives in a fixed device array of the library
 * (about 1.5 MB on each device the library runs on, held until the process
 * ends), so the call allocates nothing; inputs, outputs and semantics are those
 * of f2_fit_batch.  Every call on a device shares that device's array: calls
 * that overlap on one device (concurrent streams, threads) race and must be
 * serialised by the caller.  The array's address is looked up on the first call
 * on each device.
 * Returns F2_OK, F2_EINVAL, F2_ESCRATCH (more than F2_NOALLOC_MAX_CTX contexts:
 * nothing enqueued) or F2_EDEVICE.
 */
#define F2_NOALLOC_MAX_CTX 131072
int f2_fit_batch_noalloc(const uint64_t* rows, int64_t rows_words, const int64_t* row_off, const f2_model* model_host,
                         void* stream);

/*
 * Workspace bytes f2_encode_batch needs for a fitted model and a batch size
 * (scratch for the batch; the model's tables are part of the fit outputs).
 * Batches above 2^30 queries are encoded in chunks of 2^30, so the workspace
 * is that of one chunk.  The environment variable F2GPU_ENCODE_CHUNK, read at
 * each call, may set a smaller chunk (1 .. 2^30; a test hook): the size must be
 * the same when this is called and when f2_encode_batch runs.  Within a chunk,
 * a large batch is grouped by context window by window (about 2^23 queries each);
 * F2GPU_ENCODE_WINDOW (1 .. 2^30, raised to 2^16 at least; read the same way; a
 * test hook) sets a smaller window, and must likewise be the same for both calls.
 */
size_t f2_encode_workspace_bytes(const f2_model* model_host, int64_t num_queries);

/*
 * Encode a batch of queries against a fitted model (Sec. 2.3).
 *   ctx_id     [num_queries] context of each query
 *   x          [num_queries * x_stride_words] input bits x_0.. of each query,
 *              little-endian; bits past the stride count as 0.  The feature
 *              vector is phi = [x | 1] (Eq. 1): the constant is always 1.
 *   words_out  [2 * num_queries] the 128-bit word T(phi) (0 when unsupported)
 *   qflags_out [num_queries] F2_Q_* flags
 * A query with any x bit at or above its context's width n lies outside that
 * context's ambient space and is reported unsupported.
 * The model must come from f2_fit_batch (or f2_pool_bases): the parity-check
 * rows in tables are written by the fit.  A batch of more than one chunk (see
 * f2_encode_workspace_bytes) is enqueued chunk after chunk on the stream; the
 * results do not depend on the chunking.
 * Returns F2_OK, F2_EINVAL, F2_EWORKSPACE or F2_EDEVICE.
 */
int f2_encode_batch(const f2_model* model_host, const int32_t* ctx_id, const uint64_t* x, int32_t x_stride_words,
                    int64_t num_queries, uint64_t* words_out, uint8_t* qflags_out, void* workspace,
                    size_t workspace_bytes, void* stream);

/*
 * Feature vectors of Eq. 1 as fit rows.  Eq. 1 builds phi = [1 | bits64(v_0) |
 * ... | bits64(v_{k-1})] from k parsed 64-bit values, d = 1 + 64k features;
 * feature index 1 + 64j + b is bit b of v_j (the numbering of App. C).  In the
 * row layout above (n = 64k) that is storage bit 64j + b, with the constant in
 * word k, so row r becomes
 *     [v_{r,0} .. v_{r,k-1} | 1 | y_r AND keep]         (k + 3 words)
 *   values     [num_rows * k] row-major
 *   y          [2 * num_rows] output words, or NULL for zero outputs
 *   keep_host  [2] host words: output bits that are learned (all ones, or an
 *              opaque mask cleared: those bits are restored after encoding by
 *              f2_merge_words)
 *   rows_out   [num_rows * (k + 3)]
 * 0 <= k <= 63.  Queries need no conversion: x is the values, stride k words.
 * Returns F2_OK, F2_EINVAL or F2_EDEVICE.
 */
int f2_vectorize_rows(const uint64_t* values, const uint64_t* y, int64_t num_rows, int32_t k,
                      const uint64_t* keep_host, uint64_t* rows_out, void* stream);

/*
 * Final words from learned words (Sec. 4, the worked example that assembles an
 * instruction word): a separately supplied field is shifted into place and
 * XORed in, then the bits of an opaque mask (excluded from learning) are
 * restored from recorded state.  For each q < num_words:
 *     w = words[q] XOR ((field[q] AND (2^width - 1)) << shift)    (128-bit)
 *     out[q] = (w AND NOT mask) OR (state[q] AND mask)
 *   words, out [2 * num_words] (may be the same buffer)
 *   field      [num_words], or NULL for no field (then width and shift are ignored)
 *   width      1..64 bits, shift + width <= 128
 *   mask_host  [2] host words; state [2 * num_words] or NULL (masked bits cleared)
 * Returns F2_OK, F2_EINVAL or F2_EDEVICE.
 */
int f2_merge_words(const uint64_t* words, const uint64_t* field, int32_t shift, int32_t width,
                   const uint64_t* mask_host, const uint64_t* state, int64_t num_words, uint64_t* out,
                   void* stream);

/* per-pool flags (pool_flags) */
enum {
    F2_POOL_SHARED = 1u,          /* one map serves every member */
    F2_POOL_CONTRADICTION = 2u,   /* the members' equations contradict each other */
    F2_POOL_WIDTH_MISMATCH = 4u,  /* a member's width differs from the pool's (pool fitted from no rows) */
    F2_POOL_MASK_MISMATCH = 8u,   /* the members' output masks differ */
    F2_POOL_BAD_MEMBER = 16u      /* a member id out of range, a malformed or contradictory member, bad
                                     pool offsets, or members used by several pools beyond the buffer
                                     (pool fitted from no rows) */
};

/*
 * Pooling of separately fitted contexts (Sec. 2.1: groups with the same
 * instruction form are trained apart, then their bases are combined and
 * eliminated; a single map serves the whole group when the combined system has
 * no contradiction and every member learned the same output bits, else each
 * member keeps its own; Sec. 2.2 merges shard
 * bases the same way).  Pool p has the member contexts
 * members[pool_off[p] .. pool_off[p+1]) of members_model; their basis rows, in
 * member order and each member's stored order, are fitted as one row stream
 * (f2_fit_batch semantics) into context p of pooled.
 *   out_mask   [2 * members_model->num_ctx] learned-bit mask per member context,
 *              or NULL (all equal)
 *   pooled     outputs; pooled->num_ctx pools, pooled->n_bits[p] the pool's width
 *   pool_flags [pooled->num_ctx] F2_POOL_* flags: SHARED alone, or the reasons
 * Each context should appear in at most one pool (the row buffer holds every
 * member basis once).  For consistent members the pooled basis is the fully
 * reduced basis of the union of their spans.
 * Returns F2_OK, F2_EINVAL, F2_EWORKSPACE or F2_EDEVICE.
 */
size_t f2_pool_workspace_bytes(const f2_model* members_model, int32_t num_pools);
int f2_pool_bases(const f2_model* members_model, const uint64_t* out_mask, const int64_t* pool_off,
                  const int32_t* members, int64_t num_members, const f2_model* pooled, uint32_t* pool_flags,
                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * Interleaved-stream ingestion: group a stream of fit rows of many contexts,
 * mixed in stream order (observations gathered across a corpus, Sec. 3), by
 * context, keeping each context's rows in stream order (the kept-row semantics
 * of the streaming elimination, Sec. 2.2, depend on it).
 *   ctx_id      [num_rows] context of each row
 *   rows        [num_rows * row_stride_words] each row in the packed layout of
 *               its context (fw + 2 words, see the top of this file) at the
 *               start of its stride; the words past fw + 2 are ignored
 *   n_bits      [num_ctx] width of each context
 *   rows_out    [rows_out_words >= num_rows * row_stride_words] the grouped
 *               rows, trimmed to fw + 2 words: a valid f2_fit_batch input
 *   row_off_out [num_ctx + 1] word offsets of each context's rows in rows_out
 *               (f2_fit_batch's row_off)
 *   dropped_out [1] rows dropped: context id out of range, context width
 *               outside [0, F2_MAX_N_BITS], or fw + 2 above the stride
 *   workspace   f2_group_workspace_bytes(num_ctx, num_rows) bytes, 256-byte aligned
 * Returns F2_OK, F2_EINVAL (also for num_rows above 2^31 - 1 or a stride below
 * 3 words), F2_EWORKSPACE or F2_EDEVICE.
 */
size_t f2_group_workspace_bytes(int32_t num_ctx, int64_t num_rows);
int f2_group_rows(const int32_t* ctx_id, const uint64_t* rows, int32_t row_stride_words, int64_t num_rows,
                  const int32_t* n_bits, int32_t num_ctx, uint64_t* rows_out, int64_t rows_out_words,
                  int64_t* row_off_out, int64_t* dropped_out, void* workspace, size_t workspace_bytes, void* stream);

/* Static description of a status code. */
const char* f2_status_string(int status);

#ifdef __cplusplus
}
#endif
#endif /* F2GPU_H */
