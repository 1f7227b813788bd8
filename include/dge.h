/*
 * dge.h - C ABI of the Draft-Guided Eviction (DGE) eviction step on AMD Instinct
 * MI355X (gfx950).
 *
 * The paper (arxiv 2609.33334) defers KV-cache eviction until k answer tokens
 * have been drafted on the full cache, then, once per layer (Alg. 1, steps B-C):
 *   1. scores every cached key by the softmax attention the scoring queries pay
 *      to it (window and/or draft queries; fp32 softmax, score summed over the
 *      queries, meaned over each GQA group, 1-D max-pooled: App. "Diagnostic details",
 *      App. "Complexity and overheads");
 *   2. keeps the top (B - w) past keys per KV head (R_E of Alg. 1);
 *   3. rewrites the cache as [retained past, ascending] || [window + draft tail]
 *      (App. "Draft-guided eviction implementation", implementation notes).
 * Alternative retention rules the paper composes with DGE: H2O accumulated
 * attention (Table "Complexity and measured overhead", footnote a), StreamingLLM sinks + recency (Sec. 6)
 * and PyramidKV layer budgets (App. "Additional analysis").
 *
 * Conventions shared by every call
 * --------------------------------
 * - Tensor pointers are DEVICE pointers unless the name ends in _host.  The
 *   caller owns all memory; the library never allocates device memory.
 * - Calls are asynchronous on the given HIP stream.  All arguments are validated
 *   on the host BEFORE anything is launched: a call that returns an error has
 *   launched nothing and written nothing.  A failed launch returns DGE_ERR_HIP.
 * - Outputs must not alias inputs.  Device pointers must be 16-byte aligned.
 * - Results are deterministic: no floating-point atomics; reruns are bit-identical.
 * - Layouts are packed and head-major.  For a batch of sequences, sequence b owns
 *   cached rows [kv_offsets[b], kv_offsets[b+1]) of every KV head: N_b rows, of
 *   which the first L_b = N_b - k are prompt rows and the last k draft rows.
 *     K, V      : [H_kv][kv_head_stride] elements; row r of head h starts at
 *                 h*kv_head_stride + r*head_dim; head_dim elements contiguous.
 *     scores    : [H_kv][T] float32, T = kv_offsets[batch] (total cached rows).
 *   Element type of Q, K, V: bfloat16 (DGE_BF16) or float32 (DGE_F32).
 * - Thread safety: no global mutable state except the per-GPU scratch of
 *   dge_score_noalloc; concurrent calls on different streams with disjoint outputs and
 *   workspaces are safe (dge_score_noalloc calls on one GPU excepted).
 * - Row counts are bounded by INT32_MAX / 2: a longer sequence is DGE_ERR_UNSUPPORTED,
 *   a larger n_select DGE_ERR_INVALID (so that n_select + n_tail fits in int32).
 */
#ifndef DGE_H_
#define DGE_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DGE_ABI_VERSION 1

typedef enum {
  DGE_OK = 0,
  DGE_ERR_INVALID = 1,      /* argument violates the documented contract */
  DGE_ERR_UNSUPPORTED = 2,  /* valid request this build does not implement (e.g. head_dim) */
  DGE_ERR_WORKSPACE = 3,    /* workspace pointer NULL or smaller than dge_workspace_size */
  DGE_ERR_HIP = 4           /* a HIP launch or runtime call failed */
} dge_status_t;

typedef enum { DGE_BF16 = 0, DGE_F32 = 1 } dge_dtype_t;

/* Which cached rows score the keys (Alg. 1, step B).  For a sequence with
 * N = L + k cached rows:
 *   WINDOW_DRAFT : the last w prompt rows and the k draft rows, positions [N-w-k, N)
 *   DRAFT        : the k draft rows only (DGE's own scorer),     positions [N-k, N)
 *   WINDOW       : the last w prompt rows only (DGE-W / SnapKV),  positions [L-w, L)
 * A row at position p attends keys j <= p (causal). */
typedef enum {
  DGE_ROWS_WINDOW_DRAFT = 0,
  DGE_ROWS_DRAFT = 1,
  DGE_ROWS_WINDOW = 2
} dge_rows_t;

typedef enum { DGE_OP_SCORE = 0, DGE_OP_SELECT = 1, DGE_OP_H2O = 2 } dge_op_t;

/* Geometry of one layer's cache and the eviction parameters it is read with. */
typedef struct {
  int32_t batch;        /* sequences, >= 1 */
  int32_t n_q_heads;    /* H_q, a multiple of n_kv_heads (G = H_q / H_kv <= 64) */
  int32_t n_kv_heads;   /* H_kv >= 1 */
  int32_t head_dim;     /* d: 64 or 128 */
  int32_t window;       /* w >= 0 observation-window rows (last prompt rows) */
  int32_t k_draft;      /* k >= 0 draft rows cached after the prompt */
  const int64_t *kv_offsets;       /* device [batch+1], kv_offsets[0] == 0, non-decreasing */
  const int64_t *kv_offsets_host;  /* host copy with the same values (validation, launch sizing) */
  int64_t kv_head_stride;          /* elements between KV heads of K and V, >= T*head_dim */
  int32_t dtype;                   /* dge_dtype_t of Q, K and V */
} dge_geom_t;

/* DGE_ABI_VERSION of the built library. */
int dge_abi_version(void);

/* Static, human-readable name of a status code (never NULL). */
const char *dge_status_string(int status);

/* Bytes of device workspace the given operation needs for this geometry.
 * DGE_OP_SCORE: per-row softmax partials of dge_score (sized for w + k scoring rows).
 * DGE_OP_SELECT: radix keys of dge_select_topb.
 * DGE_OP_H2O: partial column sums of dge_h2o_colsum, plus the per-row log-sum-exp
 *             for calls where the caller supplies none.
 * Writes *bytes (host pointer).  Errors: DGE_ERR_INVALID for a bad geometry. */
dge_status_t dge_workspace_size(const dge_geom_t *geom, int32_t op, size_t *bytes);

/* Step 1 of the eviction (Alg. 1 step B; App. "Diagnostic details"; App. "Complexity and overheads"):
 *   raw[h][j] = (1/G) sum_{g in group h} sum_{scoring rows r} softmax_j(q_{g,r} . k_j / sqrt(d))
 * for every cached row j of every sequence (tail rows included), softmax in fp32
 * over keys j <= p_r, scores accumulated in fp32.  Each sequence's scores sum to
 * the number of scoring rows.
 *   q   : [H_q][batch * n_rows][d], the rows of `rows` for each sequence in ascending
 *         position, n_rows = w+k, k or w (see dge_rows_t); query head hq belongs to KV
 *         head hq / G.
 *   k   : keys, layout above.
 *   raw : [H_kv][T] float32 output.
 *   ws  : workspace of at least dge_workspace_size(geom, DGE_OP_SCORE) bytes.
 * Errors: DGE_ERR_INVALID if a sequence has fewer than w + k rows or n_rows == 0;
 * DGE_ERR_UNSUPPORTED for head_dim outside {64, 128}. */
dge_status_t dge_score(const dge_geom_t *geom, int32_t rows, const void *q, const void *k,
                       float *raw, void *ws, size_t ws_bytes, hipStream_t stream);

/* dge_score that also returns the softmax normaliser of every scoring row, which the
 * scoring computes anyway (the full-cache log-partition log Z(q) of the attention-matching
 * loss, App. "Attention-matching loss"; with dge_evicted_mass it gives the rows' evicted
 * mass without a second pass over the full cache):
 *   row_lse : [H_q][batch * n_rows] float32 output, natural log:
 *             row_lse[hq][b * n_rows + r] = log sum_{j <= p_r} exp(q_{hq,r} . k_j / sqrt(d)),
 *             rows in the order of q.
 * Other arguments, the raw output and errors are those of dge_score (DGE_ERR_INVALID for a
 * NULL or misaligned row_lse). */
dge_status_t dge_score_with_lse(const dge_geom_t *geom, int32_t rows, const void *q,
                                const void *k, float *raw, float *row_lse, void *ws,
                                size_t ws_bytes, hipStream_t stream);

/* dge_score for callers that cannot allocate device memory or pass a workspace (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * kernels and results as dge_score (bit-identical), with the softmax partials kept in a
 * fixed scratch array that the library holds in every GPU's memory until the process
 * ends.  No allocation of any kind is made by this call.
 *   Limit: the call needs dge_workspace_size(geom, DGE_OP_SCORE)-style scratch for its
 *   rows mode of at most DGE_NOALLOC_SCRATCH_BYTES (16 MiB: e.g. 64 layers x 8 KV heads x
 *   8 sequences of up to 32K rows, 34 scoring rows, G = 4); larger geometries return
 *   DGE_ERR_WORKSPACE before anything is launched.
 *   Every call on one GPU shares that GPU's scratch, and calls keep no state in it between
 *   them (each value read was written earlier in the same call): calls whose executions
 *   overlap on one GPU (different streams or threads) RACE and must be serialised by the
 *   caller.  The stream must belong to the current device; the scratch address is
 *   resolved on the first call on each device (hipGetSymbolAddress, no allocation).
 * Arguments and other errors are those of dge_score; DGE_ERR_HIP if the scratch address
 * cannot be resolved. */
#define DGE_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
dge_status_t dge_score_noalloc(const dge_geom_t *geom, int32_t rows, const void *q,
                               const void *k, float *raw, hipStream_t stream);

/* dge_score with the scoring rows' softmax normalisers supplied by the caller, e.g. the
 * log-sum-exp an attention forward already produced for the window and draft rows.
 * Only the column-sum pass runs, so K is read once.
 *   row_lse : [H_q][batch * n_rows] float32, natural log: log sum_{j <= p_r} exp(q_r . k_j / sqrt(d)),
 *             rows in the order of q.
 * Other arguments and the output are those of dge_score; no workspace is needed.
 * Errors: as dge_score; DGE_ERR_UNSUPPORTED when G * n_rows exceeds what one workgroup
 * keeps in registers (more than 576 query rows per KV head for bf16, d = 128). */
dge_status_t dge_score_lse(const dge_geom_t *geom, int32_t rows, const void *q, const void *k,
                           const float *row_lse, float *raw, hipStream_t stream);

/* Steps 1b-2 (SnapKV max-pool, then R_E = per-head top-B; Alg. 1; App. "Draft-guided eviction implementation").
 * For every (sequence b, KV head h), with C_b = N_b - n_tail candidate rows:
 *   pooled[j] = max{ scores[h][off_b + i] : |i - j| <= pool_kernel/2, 0 <= i < C_b }
 *   idx[b][h][0 .. n_kept[b]) = the n_kept[b] = min(n_select, C_b) candidates with the
 *   largest pooled score, ties to the lower position, in ascending order; entries
 *   [n_kept[b], n_select) are set to -1.
 *   scores      : [H_kv][T] float32, non-negative (dge_score or dge_h2o_colsum output).
 *   pool_kernel : odd >= 1 (1 = no pooling).
 *   n_tail      : protected rows at the end of each sequence (w + k for DGE; the recent
 *                 window for H2O); 0 <= n_tail <= N_b.
 *   n_select    : B - w for DGE (B - n_recent for H2O), >= 0.
 *   idx         : [batch][H_kv][n_select] int32 output (row index within the sequence);
 *                 may be NULL when n_select == 0.
 *   n_kept      : [batch] int32 output.
 *   ws          : at least dge_workspace_size(geom, DGE_OP_SELECT) bytes.
 * Selection is exact on the float32 scores (radix select on their bit patterns).
 * Errors: DGE_ERR_INVALID for an even or < 1 pool_kernel, n_select < 0, or
 * n_tail outside [0, N_b]. */
dge_status_t dge_select_topb(const dge_geom_t *geom, const float *scores, int32_t pool_kernel,
                             int32_t n_tail, int32_t n_select, int32_t *idx, int32_t *n_kept,
                             void *ws, size_t ws_bytes, hipStream_t stream);

/* Steps 1b-3 in one call: dge_select_topb followed by dge_compact with the same
 * n_tail and n_select (Alg. 1 steps B-C; App. "Draft-guided eviction implementation").  Writes idx, n_kept, k_out
 * and v_out exactly as the two separate calls would; the selection is repeated by
 * several workgroups per KV head so that the row copies spread over the chip.
 * Arguments, layouts and errors are those of the two calls; ws is the
 * DGE_OP_SELECT workspace. */
dge_status_t dge_select_compact(const dge_geom_t *geom, const float *scores, int32_t pool_kernel,
                                int32_t n_tail, int32_t n_select, int32_t *idx, int32_t *n_kept,
                                const void *k, const void *v, void *k_out, void *v_out, void *ws,
                                size_t ws_bytes, hipStream_t stream);

/* dge_select_compact for n_layers layers at once (Alg. 1 steps B-C run for every layer
 * after drafting), each layer with its own budget: one launch per group of up to 64
 * layers (one launch per layer when a sequence has more than 32768 candidates or the
 * pool radius exceeds 8, as dge_select_compact does then).  The caches are
 * layer-major: layer l's scores are heads [l*H_kv, (l+1)*H_kv) of a [n_layers*H_kv][T]
 * array (one dge_score call over the layer-major geometry writes them), and its K and V
 * heads start at element l * H_kv * kv_head_stride of k and v.  geom describes one layer.
 * Outputs are packed layer after layer, with nb = batch * H_kv:
 *   idx    : layer l's [batch][H_kv][n_select_host[l]] block starts at int32 element
 *            nb * (n_select_host[0] + ... + n_select_host[l-1]);
 *   n_kept : [n_layers][batch];
 *   k_out, v_out : layer l's [batch][H_kv][n_select_host[l] + n_tail][head_dim] block
 *            starts at row nb * sum over l' < l of (n_select_host[l'] + n_tail).
 * Every block equals what dge_select_compact writes for that layer's slices.
 *   n_select_host : host array [n_layers], each >= 0 (B_l - w for per-layer budgets).
 *   ws     : the DGE_OP_SELECT workspace of one layer.
 * Errors: those of dge_select_compact; DGE_ERR_INVALID for n_layers < 1, a NULL
 * n_select_host or a negative entry. */
dge_status_t dge_select_compact_layers(const dge_geom_t *geom, int32_t n_layers,
                                       const float *scores, int32_t pool_kernel, int32_t n_tail,
                                       const int32_t *n_select_host, int32_t *idx,
                                       int32_t *n_kept, const void *k, const void *v, void *k_out,
                                       void *v_out, void *ws, size_t ws_bytes,
                                       hipStream_t stream);

/* StreamingLLM retention (Sec. 6; App. "Additional analysis": four sinks and a recency window):
 * idx[b][h][0 .. n_kept[b]) = 0, 1, ..., n_kept[b]-1 with n_kept[b] = min(n_sink, N_b - n_recent);
 * remaining entries up to n_sink are -1.  The n_recent rows are the tail passed to
 * dge_compact.  No scores are read.
 *   idx    : [batch][H_kv][n_sink] int32 output;  n_kept : [batch] int32 output.
 * Errors: DGE_ERR_INVALID if n_sink < 0 or n_recent outside [0, N_b]. */
dge_status_t dge_select_streaming(const dge_geom_t *geom, int32_t n_sink, int32_t n_recent,
                                  int32_t *idx, int32_t *n_kept, hipStream_t stream);

/* Step 3 (Alg. 1 step C; App. "Draft-guided eviction implementation": [retained past] || [window + draft tail]).
 * For every (b, h), with C_b = N_b - n_tail and n_out = n_select + n_tail:
 *   out[b][h][r] = K[h][off_b + idx[b][h][r]]        for r < n_kept[b]
 *   out[b][h][r] = K[h][off_b + C_b + r - n_kept[b]] for n_kept[b] <= r < n_kept[b] + n_tail
 *   out[b][h][r] = 0                                for the remaining rows up to n_out
 * and the same for V.  Bit-exact copies of the stored elements.
 *   idx, n_kept : dge_select_topb / dge_select_streaming output (n_kept[b] <= min(n_select, C_b),
 *                 idx entries in [0, C_b)).
 *   k_out, v_out: [batch][H_kv][n_out][d] outputs, same element type as K/V.
 * Errors: DGE_ERR_INVALID for n_select < 0 or n_tail outside [0, N_b]. */
dge_status_t dge_compact(const dge_geom_t *geom, const int32_t *idx, const int32_t *n_kept,
                         int32_t n_select, int32_t n_tail, const void *k, const void *v,
                         void *k_out, void *v_out, hipStream_t stream);

/* Step 3 as an edit of the live cache (Alg. 1 step C rewrites the cache the continuation
 * decodes from): for every (b, h), with C_b = N_b - n_tail and nk = n_kept[b],
 *   K[h][off_b + r] <- K[h][off_b + idx[b][h][r]]   for r < nk
 *   K[h][off_b + nk + t] <- K[h][off_b + C_b + t]   for t < n_tail
 * and the same for V, with every source read before it is overwritten: afterwards the
 * first nk + n_tail rows of each segment hold exactly the rows dge_compact writes to
 * out[b][h][0 .. nk + n_tail).  Rows from nk + n_tail to N_b keep stale contents, and no
 * zero rows are written; the caller's new sequence length is nk + n_tail (the segment
 * offsets are unchanged).
 *   idx, n_kept : dge_select_topb / dge_select_streaming output: ascending, so that
 *                 idx[b][h][r] >= r (an entry below r is raised to r, one past C_b - 1
 *                 lowered to C_b - 1; rows are never moved upwards).
 *   k, v        : the cache, layout above; distinct buffers.
 * No workspace.  Two launches: the rows whose source lies below n_kept[b] + n_tail (a short
 * prefix, typically) are moved in order by one workgroup per (KV head, sequence); every
 * other row's source is never overwritten, and those rows are copied by many workgroups
 * at once.
 * Errors: DGE_ERR_INVALID for n_select < 0, n_tail outside [0, N_b], k == v or a NULL /
 * misaligned pointer. */
dge_status_t dge_compact_inplace(const dge_geom_t *geom, const int32_t *idx,
                                 const int32_t *n_kept, int32_t n_select, int32_t n_tail,
                                 void *k, void *v, hipStream_t stream);

/* Continuation check on the evicted cache (Sec. 3 Eq. 1; App. "Why deferral can recover
 * FullKV", the eviction-mass equation; App. "Attention-matching loss"): attention of
 * query rows over the compacted caches that dge_compact / dge_select_compact write.
 * For sequence b, KV head h and each of its G = H_q / H_kv query heads, query row r
 * (position N_b - q_from_end + r) attends
 *   the retained past rows  k_c[b][h][0 .. n_kept[b])      (all precede the tail), and
 *   the tail rows           k_c[b][h][n_kept[b] + t], t <= n_tail - q_from_end + r
 *                           (tail row t sits at position N_b - n_tail + t),
 * with weights softmax_j(q . k_j / sqrt(d)) (float32 logits, normalisers and sums; for
 * bf16 caches each weight enters the product with V as a high and a low bf16 part, which
 * keep about 16 of its significant bits):
 *   out[hq][b * n_q + r][:] = sum_j a_j v_j,
 *   lse[hq][b * n_q + r]    = log sum_j exp(q . k_j / sqrt(d))  (natural log; -inf and a
 *                             zero output when the row attends nothing).
 * q_from_end = n_tail gives the window + draft scoring rows (their evicted mass is
 * rho_q = 1 - exp(lse_R - lse_full), lse_full from a keep-all compaction); q_from_end <= 0
 * gives continuation (decode) queries, which attend every kept row.
 *   q        : [H_q][batch * n_q][d], the cache's element type.
 *   k_c, v_c : [batch][H_kv][n_select + n_tail][d] (dge_compact layout).
 *   n_kept   : [batch] int32 (clamped to [0, n_select]).
 *   out      : [H_q][batch * n_q][d] float32 output;  lse : [H_q][batch * n_q] float32 output.
 * No workspace.  Errors: DGE_ERR_INVALID for n_q < 1, n_select < 0, n_tail < 0,
 * q_from_end > n_tail, n_select + n_tail < 1 or a NULL / misaligned pointer;
 * DGE_ERR_UNSUPPORTED for more than 8 query heads per KV head. */
dge_status_t dge_cache_attention(const dge_geom_t *geom, const void *q, int32_t n_q,
                                 int32_t q_from_end, const void *k_c, const void *v_c,
                                 int32_t n_select, int32_t n_tail, const int32_t *n_kept,
                                 float *out, float *lse, hipStream_t stream);

/* Evicted attention mass of the observation rows and the attention-matching loss of a
 * selection (App. "Attention-matching loss", Eq. match; Sec. 3 Eq. 1, where beta is the
 * missed mass; App. "Why deferral can recover FullKV", the eviction-mass equation), from
 * the compacted cache and the full-cache normalisers dge_score_with_lse returns, with no
 * second pass over the full cache.  For sequence b, query head hq and observation row r
 * (position N_b - q_from_end + r, inside the tail, so every candidate precedes it):
 *   lse_R          = log sum over the retained rows k_c[b][h][0 .. n_kept[b]) and the tail
 *                    rows at positions <= its own of exp(q . k_j / sqrt(d))   (float32)
 *   rho[hq][b*n_q + r] = 1 - exp(lse_R - lse_full[hq][b*n_q + r]), the softmax mass the row
 *                    places on the evicted keys (computed as -expm1 of the clamped deficit)
 *   beta[b][h]     = mean of rho over the G query heads of KV head h and the n_q rows
 *   l_match[b][h]  = mean of -log(1 - rho) over the same rows (= mean |log Z - log Z_R|)
 *   q        : [H_q][batch * n_q][d] observation rows (dge_score's q for the window + draft
 *              rows: n_q = q_from_end = w + k); element type of the cache.
 *   k_c      : [batch][H_kv][n_select + n_tail][d], the dge_compact layout (V is not read).
 *   n_kept   : [batch] int32 (clamped to [0, n_select]).
 *   lse_full : [H_q][batch * n_q] float32, natural-log partition of each row over the full
 *              cache (dge_score_with_lse's row_lse for the same rows).
 *   rho      : [H_q][batch * n_q] float32 output; beta, l_match : [batch][H_kv] float32 outputs.
 * Accuracy: rho is the difference of two float32 log-partitions, so its absolute error is
 * about their rounding (~1e-6 for rows of 32K keys), not relative to rho.
 * No workspace.  Errors: DGE_ERR_INVALID for n_q < 1, n_select < 0, n_tail < 1,
 * q_from_end > n_tail or < n_q, or a NULL / misaligned pointer; DGE_ERR_UNSUPPORTED for more
 * than 8 query heads per KV head. */
dge_status_t dge_evicted_mass(const dge_geom_t *geom, const void *q, int32_t n_q,
                              int32_t q_from_end, const void *k_c, int32_t n_select,
                              int32_t n_tail, const int32_t *n_kept, const float *lse_full,
                              float *rho, float *beta, float *l_match, hipStream_t stream);

/* Rotary position embedding of query or key rows, in place (the post-RoPE Q and K the
 * scoring reads; App. "Draft-guided eviction implementation": queries recomputed post-RoPE
 * from each layer's input; rotate-half pairs (i, i + d/2) as in the compensation-token
 * appendix; theta = 500,000 for the Table "Backbones" models).  For head h, row r with
 * position p = positions[r], and pair i < head_dim/2:
 *   x_i       <- x_i cos(p w_i) - x_{i+d/2} sin(p w_i)
 *   x_{i+d/2} <- x_{i+d/2} cos(p w_i) + x_i sin(p w_i),     w_i = theta^(-2i/head_dim)
 * computed in double and rounded once to the stored type (bf16: round to nearest even).
 *   x         : [n_heads][head_stride] elements, row r of head h at h*head_stride + r*head_dim
 *               (the Q layout [H_q][rows][d] or the K layout [H_kv][T][d]); 16-byte aligned.
 *   positions : [n_rows] int32 device array (the rows' absolute positions).
 * Errors: DGE_ERR_INVALID for n_heads < 1, n_rows < 0, theta <= 1 or not finite,
 * head_stride < n_rows * head_dim or a head stride that is not a multiple of 8 bytes, a
 * bad dtype or a NULL / misaligned pointer; DGE_ERR_UNSUPPORTED for a head_dim that is not
 * a multiple of 4 or is above 128. */
dge_status_t dge_rope(int32_t n_heads, int32_t n_rows, int32_t head_dim, int32_t dtype,
                      int64_t head_stride, const int32_t *positions, double theta, void *x,
                      hipStream_t stream);

/* Query/key capture from a layer's input (App. "Draft-guided eviction implementation": the
 * post-RoPE queries are recomputed from each layer's input by forward pre-hooks): the
 * projection by a Linear weight and the rotary embedding of dge_rope in one call,
 *   out[h][r][:] = RoPE_{positions[r]}( (x W^T)[r][h*head_dim .. (h+1)*head_dim) ),
 * products on the matrix cores (bf16 in, float32 accumulate), each rotate-half pair
 * (i, i + head_dim/2) turned by positions[r] * theta^(-2i/head_dim) (the angle formed and
 * reduced modulo 2 pi in double, the rotation applied in float to the float32 sums), rounded
 * once to bf16 (round to nearest even).  For up to 64 rows (the window and draft rows) the
 * hidden dimension is split over several workgroups whose float32 partial sums go to the
 * workspace and are added in a fixed order by a second launch, so results are deterministic.
 *   x         : [n_rows][hidden] bf16, the layer input rows (e.g. the window and draft rows).
 *   w         : [n_heads * head_dim][hidden] bf16, the Linear weight (W_q, W_k, or a fused
 *               [W_q; W_k] whose heads come out in that order), rows = output features, as
 *               torch.nn.Linear stores it.
 *   positions : [n_rows] int32 absolute positions.
 *   out       : [n_heads][n_rows][head_dim] bf16 output, the Q layout dge_score reads.
 *   ws        : at least dge_project_rope_workspace(...) bytes (may be NULL when that is 0).
 * n_rows == 0 does nothing.  Errors: DGE_ERR_INVALID for n_rows < 0, n_heads < 1, hidden < 1,
 * theta <= 1 or not finite, a NULL / misaligned pointer (16 bytes; positions 4);
 * DGE_ERR_WORKSPACE for a missing or short workspace; DGE_ERR_UNSUPPORTED for head_dim
 * outside {64, 128}, hidden not a multiple of 128 or more than 4,194,240 rows. */
dge_status_t dge_project_rope(int32_t n_rows, int32_t hidden, const void *x, int32_t n_heads,
                              int32_t head_dim, const void *w, const int32_t *positions,
                              double theta, void *out, void *ws, size_t ws_bytes,
                              hipStream_t stream);

/* Bytes of workspace dge_project_rope needs for these sizes (0 when it needs none); writes
 * *bytes (host pointer).  Errors: those of dge_project_rope's size checks, DGE_ERR_INVALID
 * for a NULL bytes pointer. */
dge_status_t dge_project_rope_workspace(int32_t n_rows, int32_t hidden, int32_t n_heads,
                                        int32_t head_dim, size_t *bytes);

/* Contiguity of the retained sets (Sec. 4, "Selection trades coverage for contiguity";
 * Table "Selection decomposition", column "run len."): for sequence b and KV head h,
 *   runs[b][h]     = number of maximal runs of consecutive positions among the first
 *                    n_kept[b] entries of idx[b][h][.] (0 when none is kept),
 *   mean_len[b][h] = n_kept[b] / runs[b][h] (float32; 0 when none is kept).
 * Counted over the selected past keys; the protected window/draft tail, one run under
 * every rule, is not included.
 *   idx      : [batch][H_kv][n_select] int32, strictly ascending within each row's kept
 *              prefix (as dge_select_topb and dge_select_streaming write it); entries past
 *              n_kept[b] are ignored.  Unsorted or repeated entries give a count that is
 *              not the run count (no error is raised).
 *   n_kept   : [batch] int32 (clamped to [0, n_select]).
 *   runs     : [batch][H_kv] int32 output;  mean_len : [batch][H_kv] float32 output.
 * No workspace.  Errors: DGE_ERR_INVALID for n_select < 0 or a NULL / misaligned pointer. */
dge_status_t dge_retained_runs(const dge_geom_t *geom, const int32_t *idx, const int32_t *n_kept,
                               int32_t n_select, int32_t *runs, float *mean_len,
                               hipStream_t stream);

/* H2O accumulated attention, kept running through the draft rows
 * (Table "Complexity and measured overhead", footnote a; App. "Draft-guided eviction implementation" on H2O's prompt-query buffer):
 *   colsum[h][j] = (1/G) sum_{g in group h} sum_{p = j}^{N_b - 1} softmax_j(q_{g,p} . k_j / sqrt(d))
 * over every cached row p of the sequence (all prompt rows and the k draft rows).
 *   q_all  : [H_q][T][d] queries of every cached row (same element type as K).
 *   lse    : NULL, or [H_q][T] float32 natural-log partition log sum_{j<=p} exp(q_p . k_j / sqrt(d))
 *            supplied by the caller (e.g. from its attention forward); when NULL the
 *            library computes it first into the workspace.
 *   colsum : [H_kv][T] float32 output; each sequence's colsum sums to N_b.
 *   ws     : dge_workspace_size(geom, DGE_OP_H2O) bytes (per-segment partial column sums,
 *            and the row LSE when lse == NULL).
 * Only bfloat16 inputs with head_dim 128 are supported, and computing the LSE in the
 * library needs G <= 4 query heads per KV head (DGE_ERR_UNSUPPORTED otherwise). */
dge_status_t dge_h2o_colsum(const dge_geom_t *geom, const void *q_all, const void *k,
                            const float *lse, float *colsum, void *ws, size_t ws_bytes,
                            hipStream_t stream);

/* PyramidKV per-layer budgets (App. "Additional analysis"), host only:
 *   c = B - w;  max = 2c - floor(c/beta);  min = floor(c/beta);
 *   steps = floor((max - min) / (n_layers - 1));  out_host[l] = max - l*steps + w.
 * Errors: DGE_ERR_INVALID for B < w, n_layers < 1, beta < 1 or a NULL output. */
dge_status_t dge_pyramid_budgets(int32_t B, int32_t w, int32_t n_layers, int32_t beta,
                                 int32_t *out_host);

#ifdef __cplusplus
}
#endif

#endif /* DGE_H_ */
