/*
 * cc.h -- C ABI of the counter-causal refresh-scoring library (libcc.so, gfx950).
 *
 * The library implements the memory-refresh cycle of counter-causal KV-cache
 * eviction (Gould & van den Hengel, "Back from the Future: Key-Value Cache
 * Management by Counter-Causal Surprise"):
 *
 *   cc_score        per-entry surprise scores of the cached tokens (Sec. 3.1):
 *                   attention over the stored keys/values under the
 *                   counter-causal mask, the output projection, the LM head and
 *                   the log-softmax at the cached token id;
 *   cc_select_keep  the k highest-scoring entries of each segment (Sec. 3.2,
 *                   memory refresh: argsort and keep the top J);
 *   cc_compact_kv   gather the kept entries of the KV cache, token ids and
 *                   position ids (Sec. 3.2, memory refresh: K', V', X updates).
 *
 * Conventions shared by every entry point
 *   - Pointers are device pointers unless the name ends in _h (host memory).
 *   - Every call only enqueues work on `stream` (a hipStream_t; NULL is the
 *     default stream) and returns; results are ready when the stream is.
 *     Host arrays (_h) are read before the call returns.
 *   - The caller owns every buffer.  The library allocates no device memory;
 *     scratch space comes from the caller's workspace, whose size the matching
 *     *_workspace query returns (a NULL workspace with size 0 is valid when the
 *     query returned 0).  Small planning tables are copied from host memory
 *     into the workspace on `stream`.
 *   - Arguments are checked on the host before anything is enqueued.  A call
 *     that returns a status other than CC_OK has enqueued nothing and written
 *     nothing.  Faults inside kernels surface at the caller's next
 *     synchronisation.  Token ids outside [0, vocab) and position ids outside
 *     the cache are a caller error with undefined results for that row.
 *   - Element types: CC_BF16 tensors are bfloat16, CC_F32 tensors are float32;
 *     scores are always float32.  Matrices are row-major.
 *   - Calls that share a workspace must be ordered (same stream or synchronised).
 */
#ifndef CC_H
#define CC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum cc_status {
  CC_OK = 0,
  CC_ERR_ARG = 1,          /* a NULL required pointer, a bad enum value, a bad count */
  CC_ERR_SHAPE = 2,        /* inconsistent sizes (e.g. n_heads_q % n_heads_kv != 0) */
  CC_ERR_DTYPE = 3,        /* dtype not valid for this call */
  CC_ERR_WORKSPACE = 4,    /* workspace smaller than the query returned */
  CC_ERR_UNSUPPORTED = 5,  /* a valid problem this library has no kernel for */
  CC_ERR_HIP = 6,          /* the HIP runtime rejected a launch or copy */
  CC_ERR_SCRATCH = 7       /* the call needs more than the static scratch of the
                              allocation-free entry point holds */
} cc_status;

typedef enum cc_dtype { CC_F32 = 0, CC_BF16 = 1 } cc_dtype;

/* Counter-causal mask (Sec. 3.1): position i attends to cache positions j > i of
 * its own sequence (STRICT, the paper's mask).  INCLUSIVE (j >= i) is provided for
 * testing.  A row with no allowed key has a zero attention output. */
typedef enum cc_diag { CC_DIAG_STRICT = 0, CC_DIAG_INCLUSIVE = 1 } cc_diag;

/* LAST_LAYER: the fast single-layer approximation (Sec. 3.1): queries are given,
 * attention runs on the cache's last layer, then W_o and the LM head.
 * FULL: every layer runs with fresh queries from the token embeddings against the
 * stored keys/values of that layer (Sec. 3.1, full counter-causal pass).
 * LAST_LAYER_H: the fast approximation in its exact form (Sec. 3.1, fast single-layer
 * approximation): from the stored activations H entering the last layer, RMSNorm,
 * W_q and RoPE at the original positions, attention on the cache's last layer, the
 * layer's output processing (W_o + residual, RMSNorm, SwiGLU MLP + residual), the
 * final RMSNorm and the LM head.
 * LAST_LAYER_FUSED: LAST_LAYER with W_o folded into the LM head.  With queries given,
 * the output processing of the fast approximation (Sec. 3.1) is the bare projection
 * W_o, so z = W_lm (W_o y) = (W_lm W_o) y: inputs.w_lm holds the product
 * [V][Hq*head_dim] (from cc_fuse_wo_lmhead, once per model) and inputs.w_o is unused.
 * The scores equal LAST_LAYER's up to rounding. */
typedef enum cc_mode {
  CC_MODE_LAST_LAYER = 0,
  CC_MODE_FULL = 1,
  CC_MODE_LAST_LAYER_H = 2,
  CC_MODE_LAST_LAYER_FUSED = 3
} cc_mode;

typedef enum cc_kv_layout { CC_KV_CONTIGUOUS = 0, CC_KV_PAGED = 1 } cc_kv_layout;

/* A view of the KV cache (keys and values share the layout).  head_dim elements of
 * one (layer, KV head, token) are contiguous; strides are in elements.
 *   CONTIGUOUS: element (seq b, layer l, head h, token t, e) is at
 *       base + b*seq_stride + l*layer_stride + h*head_stride + t*tok_stride + e
 *   PAGED: token t of sequence b lives in page block_table[b*max_pages + t/page_size],
 *       slot t % page_size:
 *       base + l*layer_stride + page*page_stride + h*head_stride + slot*tok_stride + e
 * Token t is the t-th cached entry of its sequence in cache order (ascending
 * original position after any number of refreshes). */
typedef struct cc_kv {
  int32_t layout;              /* cc_kv_layout */
  int32_t n_layers;            /* layers held by the cache */
  void* k;                     /* device base of keys */
  void* v;                     /* device base of values */
  int64_t seq_stride;          /* CONTIGUOUS only */
  int64_t layer_stride;
  int64_t head_stride;
  int64_t tok_stride;
  int64_t page_stride;         /* PAGED only: one page spans less than 4 GiB, i.e.
                                  page_stride and page_size*tok_stride, in bytes, are
                                  below 2^32 (CC_ERR_UNSUPPORTED otherwise) */
  const int32_t* block_table;  /* PAGED only: device [n_seqs][max_pages] page ids */
  int32_t page_size;           /* PAGED only: tokens per page, a power of two >= 16 */
  int32_t max_pages;           /* PAGED only: row length of block_table */
} cc_kv;

/* Shape of one refresh.  Sequences are ragged: sequence b holds cache entries
 * [cu_seqlens[b], cu_seqlens[b+1]) of every token-major array (N = cu_seqlens[n_seqs]).
 * With GQA, query head h reads KV head h / (n_heads_q / n_heads_kv). */
typedef struct cc_problem {
  int32_t dtype;               /* cc_dtype of q, k, v and all weights */
  int32_t mode;                /* cc_mode */
  int32_t diag;                /* cc_diag */
  int32_t n_seqs;              /* >= 1 */
  const int32_t* cu_seqlens_h; /* host [n_seqs+1], cu[0] = 0, non-decreasing */
  const int32_t* cu_seqlens_d; /* the same values in device memory */
  int32_t n_heads_q;
  int32_t n_heads_kv;          /* divides n_heads_q */
  int32_t head_dim;            /* 64 or 128 (FULL and LAST_LAYER_H: 128) */
  int32_t hidden;              /* D: model width, rows of W_o (bf16: a multiple of 64) */
  int32_t vocab;               /* V: rows of the LM head */
  int32_t n_layers;            /* FULL only: transformer layers (<= kv.n_layers) */
  int32_t ffn;                 /* FULL, LAST_LAYER_H: SwiGLU width */
  float softmax_scale;         /* 0 selects 1/sqrt(head_dim) (Eq. (2)) */
  float rope_theta;            /* FULL, LAST_LAYER_H: rotary base */
  float rms_eps;               /* FULL, LAST_LAYER_H: RMSNorm epsilon */
  int32_t n_frozen;            /* first n_frozen entries of each sequence are sink
                                  slots that are never evicted (score +inf) */
  int32_t lmhead_packed;       /* bf16 only: 1 = the LM head reads the packed weight
                                  cc_inputs.w_lm_packed (cc_pack_lmhead) and packs its
                                  input rows in the workspace (cc_inputs.w_lm is then
                                  not read and may be NULL); 0 = row-major w_lm */
} cc_problem;

/* Weights of one transformer layer (FULL, LAST_LAYER_H), device pointers in `dtype`. */
typedef struct cc_layer_weights {
  const void* attn_norm;       /* [D] RMSNorm gain before attention */
  const void* wq;              /* [Hq*d][D] query projection */
  const void* wo;              /* [D][Hq*d] output projection */
  const void* mlp_norm;        /* [D] RMSNorm gain before the MLP */
  const void* w_gate;          /* [F][D] */
  const void* w_up;            /* [F][D] */
  const void* w_down;          /* [D][F] */
} cc_layer_weights;

typedef struct cc_inputs {
  const void* q;               /* LAST_LAYER(_FUSED): [N][Hq][d] queries (already
                                  rotated) */
  cc_kv kv;                    /* LAST_LAYER scores layer kv.n_layers-1; FULL uses
                                  layers 0..n_layers-1 (keys already rotated) */
  const int32_t* token_ids;    /* [N] cached token ids X */
  const int32_t* pos_ids;      /* FULL, LAST_LAYER_H: [N] original positions,
                                  NULL -> 0..n_b-1 */
  const void* w_o;             /* LAST_LAYER: [D][Hq*d] */
  const void* w_lm;            /* [V][D] LM head; LAST_LAYER_FUSED: [V][Hq*d], the
                                  product W_lm W_o.  Not read (may be NULL) when
                                  lmhead_packed = 1 */
  const void* embed;           /* FULL: [V][D] token embeddings */
  const cc_layer_weights* layers_h; /* FULL: host array [n_layers]; LAST_LAYER_H:
                                  host array [1], the last layer's weights */
  const void* final_norm;      /* FULL, LAST_LAYER_H: [D] final RMSNorm gain */
  const void* h_last;          /* LAST_LAYER_H: [N][D] stored activations entering
                                  the last layer (dtype), token-major like ids */
  const void* w_lm_packed;     /* lmhead_packed = 1: the LM head in the packed layout
                                  of cc_pack_lmhead */
} cc_inputs;

/* Human-readable name of a status code (static string). */
const char* cc_status_str(cc_status s);

/* Library build identifier, e.g. "libcc gfx950 <date>". */
const char* cc_version(void);

/* ------------------------------------------------------------------ scoring */

/* Workspace bytes cc_score needs for problem p (sizes only; pointers unused). */
cc_status cc_score_workspace(const cc_problem* p, size_t* bytes);

/* Surprise score of every cached entry (Eq. (5), Sec. 3.1):
 *   scores[i] = logsumexp_v(z_i) - z_i[x_i] = -log P(x_i | x_{i+1..n_b-1}),
 * a strictly decreasing function of P, where z_i are the LM-head logits of entry i
 * after the counter-causal pass.  The last entry of each sequence (no future) and
 * the first n_frozen entries score +inf.  scores: device float32 [N].
 * The [N][V] logits are never materialised. */
cc_status cc_score(const cc_problem* p, const cc_inputs* in, float* scores,
                   void* workspace, size_t workspace_bytes, void* stream);

/* Sub-steps of cc_score, exposed for testing and measurement. */

/* Workspace for cc_attention_cc. */
cc_status cc_attention_workspace(const cc_problem* p, size_t* bytes);

/* Counter-causal attention (Eq. (2) under the mask of Sec. 3.1) over cache layer
 * `layer`: o[i][h][:] = sum_{j allowed} softmax_j(scale * q[i][h].k[j][c]) v[j][c],
 * c = h / g.  q, o: [N][Hq][d] in dtype (o may not alias q). */
cc_status cc_attention_cc(const cc_problem* p, const void* q, const cc_kv* kv,
                          int32_t layer, void* o, void* workspace,
                          size_t workspace_bytes, void* stream);

/* Workspace for cc_lmhead_score. */
cc_status cc_lmhead_workspace(const cc_problem* p, size_t* bytes);

/* LM head, log-softmax and target gather (Eq. (5)): for hidden rows u [N][D]
 * (dtype), scores[i] = logsumexp(W_lm u_i) - (W_lm u_i)[ids[i]], with the
 * last-entry / frozen rule applied.  The target logit is taken from the same
 * accumulators as the log-sum-exp, and a difference that rounding takes below zero is
 * returned as 0 (-log P >= 0).  lse (nullable) receives logsumexp.  This is the
 * log-probability sub-step: log P(x_i | future) = -scores[i] for every finite score. */
cc_status cc_lmhead_score(const cc_problem* p, const void* u, const void* w_lm,
                          const int32_t* token_ids, float* scores, float* lse,
                          void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of the static device scratch behind cc_lmhead_score_noalloc (per GPU). */
#define CC_NOALLOC_SCRATCH_BYTES (32u << 20)

/* cc_lmhead_score without a workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid allocation).
 * Arguments, results and errors are those of cc_lmhead_score with p->lmhead_packed = 0
 * (a packed problem returns CC_ERR_ARG); the scratch that cc_lmhead_workspace(p) would
 * size -- the per-(vocabulary tile, entry) log-sum-exp partials and the target logits,
 * written in full by every call -- lives in a static device array of
 * CC_NOALLOC_SCRATCH_BYTES that each GPU the library runs on holds until the process
 * ends.  A problem whose cc_lmhead_workspace exceeds it returns CC_ERR_SCRATCH before
 * anything is enqueued (32 MiB covers, e.g., 4096 entries of a 128256-word vocabulary:
 * about 8 B per entry per 256 words).  The call allocates nothing.  Every call on one GPU
 * shares that GPU's array: calls whose execution overlaps on one GPU (two streams, or two
 * host threads) race and must be ordered by the caller. */
cc_status cc_lmhead_score_noalloc(const cc_problem* p, const void* u, const void* w_lm,
                                  const int32_t* token_ids, float* scores, float* lse,
                                  void* stream);

/* Workspace for cc_fuse_wo_lmhead: the transposed W_o. */
cc_status cc_fuse_wo_lmhead_workspace(int32_t dtype, int32_t hidden, int32_t qdim,
                                      size_t* bytes);

/* The weight of mode LAST_LAYER_FUSED: out[v][c] = sum_d w_lm[v][d] w_o[d][c], with
 * w_lm [V][hidden], w_o [hidden][qdim] (qdim = Hq*head_dim) and out [V][qdim], all in
 * dtype (fp32 accumulation, one rounding to dtype).  A one-time weight preparation,
 * not part of a refresh.  bf16 needs hidden % 64 == 0 and 16-byte aligned pointers. */
cc_status cc_fuse_wo_lmhead(int32_t dtype, const void* w_lm, const void* w_o, void* out,
                            int32_t vocab, int32_t hidden, int32_t qdim, void* workspace,
                            size_t workspace_bytes, void* stream);

/* Dense projection y[m][n] = sum_k x[m][k] w[n][k] (x: [M][K], w: [N][K], y: [M][N],
 * all in dtype), the layer's output projection of the fast variant. */
cc_status cc_linear(int32_t dtype, const void* x, const void* w, void* y, int32_t M,
                    int32_t N, int32_t K, void* stream);

/* ------------------------------------------------------------------ FP8 LM head */

/* Workspace for cc_quantize_fp8 on `rows` rows. */
cc_status cc_quantize_fp8_workspace(int64_t rows, size_t* bytes);

/* OCP FP8 E4M3 quantization of x [rows][cols] (dtype): per_row = 1 gives each row its own
 * scale, per_row = 0 one scale for the matrix.  amax = max |x| over the row (matrix),
 * codes = E4M3(x * (448 / amax)) rounded to nearest even, scale = amax / 448, every step
 * in fp32; an all-zero row (matrix) gets codes 0 and scale 0.  x aligned to four
 * elements; codes: device uint8 [rows][cols] (4-byte aligned); scale: device float
 * [rows] (per_row) or [1].
 * cols must be a positive multiple of 4.  A weight preparation for cc_lmhead_score_fp8
 * (the LM head, one scale); not part of the method (the paper fixes no precision). */
cc_status cc_quantize_fp8(int32_t dtype, const void* x, int64_t rows, int32_t cols,
                          int32_t per_row, uint8_t* codes, float* scale, void* workspace,
                          size_t workspace_bytes, void* stream);

/* Workspace for cc_lmhead_score_fp8. */
cc_status cc_lmhead_fp8_workspace(const cc_problem* p, size_t* bytes);

/* cc_lmhead_score on an FP8 LM head: u [N][D] (dtype) is quantized per row into the
 * workspace as in cc_quantize_fp8; w_codes [V][D] are the LM head's E4M3 codes with one
 * device scale w_scale[0]; the logits are z = (sum_d code products) * scale_u * scale_w,
 * accumulated in fp32 on the FP8 matrix cores, and the score follows Eq. (5) as in
 * cc_lmhead_score.  D = p->hidden must be a multiple of 128; w_codes 16-byte aligned. */
cc_status cc_lmhead_score_fp8(const cc_problem* p, const void* u, const uint8_t* w_codes,
                              const float* w_scale, const int32_t* token_ids, float* scores,
                              float* lse, void* workspace, size_t workspace_bytes,
                              void* stream);

/* Bytes of the packed LM-head layout of a bf16 [rows][cols] matrix: rows rounded up
 * to a multiple of 256, times cols, times 2. */
cc_status cc_pack_lmhead_bytes(int64_t rows, int32_t cols, size_t* bytes);

/* Packs a bf16 matrix x [rows][cols] (row stride cols; cols a positive multiple of 32;
 * x 16-byte aligned) into the layout the packed LM head stages: for each 256-row tile
 * and 32-column step, one 16 KB block in which row r (64 bytes at 64r) holds its
 * 16-byte chunk c (columns 8c .. 8c+7 of the step) at chunk position c ^ ((r >> 1) & 3);
 * rows past `rows` are zero.  A bit copy that changes the layout only: the weight
 * preparation for lmhead_packed = 1, made once per model (the LM-head input rows are
 * packed inside each call).  out: device, cc_pack_lmhead_bytes bytes, 16-byte aligned,
 * not overlapping x. */
cc_status cc_pack_lmhead(const void* x, int64_t rows, int32_t cols, void* out,
                         size_t out_bytes, void* stream);

/* cc_lmhead_score with p->lmhead_packed = 1: w_packed is w_lm [V][D] packed by
 * cc_pack_lmhead (the row-major weight is not needed).  The result equals
 * cc_lmhead_score up to fp32 summation order (the packed kernel accumulates in another
 * order on the 16x16x32 matrix-core shape).  Workspace: cc_lmhead_workspace(p). */
cc_status cc_lmhead_score_packed(const cc_problem* p, const void* u, const void* w_packed,
                                 const int32_t* token_ids, float* scores, float* lse,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------ selection */

/* Workspace for cc_select_keep with n_segs segments. */
cc_status cc_select_workspace(int32_t n_segs, size_t* bytes);

/* Keep selection (Sec. 3.2): segment s is scores[seg_start_h[s] .. +seg_len_h[s]).
 * Its k = k_h[s] kept entries are the first k under the order (score descending,
 * -0 == +0, NaN below -inf; ties to the lower index), written in ascending order as
 * segment-local indices to keep_idx[off_s .. off_s + k), off_s = sum_{t<s} k_h[t].
 * 0 <= k <= seg_len.  Segments may overlap (e.g. one per KV head over the same
 * per-token scores).  keep_idx: device int32 [sum k]. */
cc_status cc_select_keep(const float* scores, int32_t n_segs, const int64_t* seg_start_h,
                         const int32_t* seg_len_h, const int32_t* k_h, int32_t* keep_idx,
                         void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------ compaction */

/* Workspace for cc_compact_kv on a cache of cache_layers layers. */
cc_status cc_compact_workspace(const cc_problem* p, int32_t cache_layers, int32_t per_head,
                               size_t* bytes);

/* KV compaction (Sec. 3.2): for every cache layer, KV head and sequence b,
 *   dst[j] = src[keep[j]] for j < k_b   (a bit copy of head_dim elements),
 * with keep the list from cc_select_keep.  Lists are packed back to back:
 * per_head = 0: one list per sequence (k_h[b]); per_head = 1: one list per
 * (sequence, KV head) in order b*n_heads_kv + h (k_h[b*Hkv+h]).
 * dst is `out` (same geometry as `kv`) or, when out is NULL, `kv` itself (in
 * place; safe because lists are ascending so keep[j] >= j).  token_ids and pos_ids
 * (nullable, device int32 [N], token-major by cu_seqlens) are compacted in place
 * with the first list of each sequence: ids[cu_b + j] = ids[cu_b + keep[j]].
 * Entries at and past k_b are left untouched (paged: pages past ceil(k_b/P) are free
 * for the caller to reuse). */
cc_status cc_compact_kv(const cc_problem* p, const cc_kv* kv, const int32_t* keep_idx,
                        const int32_t* k_h, int32_t per_head, int32_t* token_ids,
                        int32_t* pos_ids, const cc_kv* out, void* workspace,
                        size_t workspace_bytes, void* stream);

/* Workspace for cc_compact_rows. */
cc_status cc_compact_rows_workspace(const cc_problem* p, int32_t row_bytes, int32_t per_head,
                                    size_t* bytes);

/* Compaction of a token-major per-entry array that travels with the cache, such as the
 * stored activations H of the exact fast variant (Sec. 3.1: H is recorded per cache
 * entry, so the memory refresh of Sec. 3.2 keeps the same rows):
 *   rows[cu[b] + j] = rows[cu[b] + keep_b[j]] for j < k_b,
 * with the same keep lists as cc_compact_kv (per_head = 1: the first list of each
 * sequence is used).  rows: device [N][row_bytes] (row_bytes a multiple of 16, rows
 * 16-byte aligned); out_rows NULL compacts in place, else writes out_rows (same shape,
 * no overlap with rows).  A bit copy. */
cc_status cc_compact_rows(const cc_problem* p, void* rows, int32_t row_bytes,
                          const int32_t* keep_idx, const int32_t* k_h, int32_t per_head,
                          void* out_rows, void* workspace, size_t workspace_bytes,
                          void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CC_H */
