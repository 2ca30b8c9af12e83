/*
 * hs2.h -- C ABI of libhs2.so: decode-time attention of one HySparse2 hybrid
 * block on MI355X (gfx950).
 *
 * A hybrid block is one full-attention (FA) layer followed by sparse-attention
 * (SA) layers (HySparse2, Sec. "HySparse2 Overview").  The FA layer attends
 * over the whole KV cache and doubles as the indexer: its exact softmax
 * probabilities are the token scores (Sec. "The Role of Full Attention").
 * Per query, the most recent `window` tokens are always selected and the `k`
 * highest-scoring tokens before that window are added (Sec. "Cross-Layer KV
 * Reuse", removal of the separate SWA branch; token-level selection in the
 * same section).  The SA layers reuse the FA layer's KV cache and those
 * indices (KV Reuse, same section).  FA and SA use no positional encoding
 * (Sec. "Experimental Setup").
 *
 * Readings where the paper is silent, fixed by this ABI:
 *   - score of token t for KV head g and query c: the sum, over the query
 *     heads h of g, of head h's softmax probability of t (each head
 *     normalised over its own causal range);
 *   - top-k is drawn only from tokens outside the window; equal scores go to
 *     the lower token index; scores below FLT_MIN rank as zero;
 *   - the cache of sequence b holds tokens [0, len[b]) including the decode
 *     tokens; query c of a C-token chunk sits at pos = len[b] - C + c and sees
 *     tokens [0, pos]; its window is [max(0, pos - window + 1), pos];
 *   - query head h reads KV head h / G with G = n_q_heads / n_kv_heads;
 *   - SA layers use a plain softmax over the selected tokens (no sink).
 *
 * Conventions for every entry point:
 *   - tensor pointers are DEVICE pointers (HIP device memory of the current
 *     device) unless stated otherwise; bf16 tensors are passed as uint16_t
 *     bit patterns; every work-issuing call is asynchronous on `stream`
 *     (a hipStream_t; NULL = the default stream) and results are valid once
 *     the caller synchronises that stream;
 *   - the caller owns every buffer, including the workspace; the library
 *     never allocates or frees device memory and never synchronises;
 *   - inputs are read-only; outputs must not alias inputs or the workspace;
 *   - every condition checkable on the host is checked before anything is
 *     launched; on error nothing is launched, outputs are untouched and a
 *     negative status is returned (hs2_status_string / hs2_last_error give a
 *     message).  Nothing throws across this ABI.
 *   - len[] lives on the device and is not read by the host.  Precondition:
 *     n_queries <= len[b] <= max_len.  The kernels clamp len[b] to
 *     [0, max_len]; a query whose position is negative gets an all -1 index
 *     row and a zero output.
 *
 * Planner overrides (environment, read on every call; for tests and tuning,
 * invalid values fall back to the planner's choice): HS2_FA_VARIANT
 * (full-attention kernel shape), HS2_FA_SPLIT / HS2_POOL_SPLIT /
 * HS2_SA_SPLIT (tokens or slots per workgroup), HS2_FA_ROUNDS (workgroup
 * rounds the full-attention splits are sized for), HS2_POOL_FROM_K=1
 * (recompute the scores from K even where the stored logits would serve),
 * HS2_FA_CACHE_POLICY (0: every full-attention load cacheable, 1: V rows
 * non-temporal, 2: K and V non-temporal, 3: V and the leading K rows of
 * each token group non-temporal; 1 and 2 exist for one query row tile, 3
 * for more) and HS2_FA_K_KEEP (percent of each token group's K rows that
 * policy 3 keeps cacheable).  None changes a result beyond floating-point
 * summation order; the cache policies change none at all.
 */
#ifndef HS2_H
#define HS2_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum hs2_status {
  HS2_OK = 0,
  HS2_ERR_NULL = -1,        /* a required pointer is NULL                         */
  HS2_ERR_SHAPE = -2,       /* inconsistent or out-of-range dimensions / budgets  */
  HS2_ERR_UNSUPPORTED = -3, /* valid request this build does not implement        */
  HS2_ERR_WORKSPACE = -4,   /* workspace smaller than hs2_workspace_bytes()       */
  HS2_ERR_ALIGN = -5,       /* pointer or stride not 16-byte aligned              */
  HS2_ERR_HIP = -6          /* a HIP runtime call or a kernel launch failed       */
} hs2_status;

/* Shapes shared by every call of one hybrid block.
 *   q, out:  [batch, n_queries, n_q_heads, head_dim] contiguous bf16
 *   K, V:    element (b, g, t, d) at b*kv_stride_b + g*kv_stride_h + t*kv_stride_t + d
 *            (bf16, or E4M3 bytes for the _fp8 entry points; K and V share
 *            this layout; each token row is contiguous)                         */
typedef struct hs2_dims {
  int32_t batch;       /* B >= 1                                                  */
  int32_t n_queries;   /* C: decode tokens per sequence, 1 .. 16                  */
  int32_t n_q_heads;   /* Hq >= 1                                                 */
  int32_t n_kv_heads;  /* Hkv >= 1, Hq % Hkv == 0, G = Hq / Hkv <= 64,            */
                       /*   C * (G rounded up to a power of two) <= 128,          */
                       /*   B * Hkv * C <= 65535 (HS2_ERR_UNSUPPORTED)            */
  int32_t head_dim;    /* D: 128, or 256 (the paper's head dim, Sec. "Experimental */
                       /*   Setup"); other values: HS2_ERR_UNSUPPORTED            */
  int32_t max_len;     /* Lmax: cache capacity per sequence, 1 .. 2^27 tokens     */
  int64_t kv_stride_b; /* elements; multiple of 8                                 */
  int64_t kv_stride_h; /* elements; multiple of 8                                 */
  int64_t kv_stride_t; /* elements; >= head_dim, multiple of 8, <= 2^24           */
  float scale;         /* softmax scale; <= 0 selects 1/sqrt(head_dim)            */
} hs2_dims;

/* Bytes of device workspace that every call below needs for these dims and
 * budgets (the same buffer may serve all calls of a block, one at a time).
 * Host-only, launches nothing.  Returns 0 if the dims or budgets are invalid. */
size_t hs2_workspace_bytes(const hs2_dims* dims, int32_t k, int32_t window);

/* Full-attention layer + token scores + selection (the block's first layer).
 * Passages: the full-attention layer attends over the whole cache and its
 * exact attention scores select the tokens (Sec. "The Role of Full
 * Attention"); the selection is the forced recent window followed by the
 * highest-scoring tokens outside it, chosen per token (Sec. "Cross-Layer KV
 * Reuse", paragraphs "Removing the Separate SWA Branch" and "Token-Level
 * Sparse Selection").
 *
 *   q       [B, C, Hq, D] bf16         FA-layer queries
 *   K, V    cache, layout of hs2_dims  (read over [0, len[b]) per sequence)
 *   len     [B] int32 (device)         tokens in each sequence's cache
 *   k       >= 0                       top-k budget outside the window
 *   window  >= 0                       forced recent window; k + window >= 1
 *   out     [B, C, Hq, D] bf16         attention output (fp32 accumulation,
 *                                      rounded to nearest even)
 *   idx     [B, Hkv, C, k + window] int32   selected token indices of each
 *           (sequence, KV head, query): ascending, then -1 padding.  Row
 *           length min(pos + 1, k + window): min(k, N) top-k tokens of the
 *           N = max(0, pos - window + 1) tokens before the window, then the
 *           window itself.
 *   stats   [B, C, Hq, 2] float or NULL: per head (M, Z) with M the largest
 *           logit scale*<q, k_t> over [0, pos] and Z = sum_t exp(logit_t - M)
 *   scores  [B, Hkv, C, max_len] float or NULL: pooled scores of the
 *           candidate tokens [0, N); entries from N on are unspecified
 *   workspace / workspace_bytes: device scratch, >= hs2_workspace_bytes()
 *   stream  hipStream_t                                                        */
hs2_status hs2_full_attn_score_select(const hs2_dims* dims, const uint16_t* q, const uint16_t* K,
                                      const uint16_t* V, const int32_t* len, int32_t k, int32_t window,
                                      uint16_t* out, int32_t* idx, float* stats, float* scores,
                                      void* workspace, size_t workspace_bytes, void* stream);

/* Sparse-attention layer reusing the FA layer's cache and selection.
 * Passage: the sparse layers of a hybrid block reuse the preceding
 * full-attention layer's KV cache and its selected indices and attend only
 * over the selected tokens (Sec. "HySparse2 Overview"; Sec. "Cross-Layer KV
 * Reuse", KV Reuse).
 *
 *   q       [B, C, Hq, D] bf16         this SA layer's own queries
 *   K, V    the same cache the FA layer read
 *   len     [B] int32 (device)         as for the FA call
 *   idx     [B, Hkv, C, n_slots] int32 (device) selection rows; entries < 0
 *           or >= len[b] are skipped.  Query head h uses row (b, h / G, c).
 *   out     [B, C, Hq, D] bf16         softmax attention over the selected
 *           tokens only (a row with no valid entry gives 0)                    */
hs2_status hs2_sparse_attn(const hs2_dims* dims, const uint16_t* q, const uint16_t* K, const uint16_t* V,
                           const int32_t* len, const int32_t* idx, int32_t n_slots, uint16_t* out,
                           void* workspace, size_t workspace_bytes, void* stream);

/* The same sparse-attention layer with the two per-layer parts the paper's
 * sparse layers carry (Sec. "Experimental Setup": learnable per-head sink
 * biases and sigmoid output gates).  Either may be NULL, and with both NULL
 * this is hs2_sparse_attn.
 *
 *   sink    [Hq] float (device) or NULL: one logit per query head, in the
 *           units of the scaled logits scale*<q, k_t>, that joins the softmax
 *           normaliser without a value row:
 *             out = sum_t e^(s_t - M) v_t / (e^(sink_h - M) + sum_t e^(s_t - M))
 *   gate    [B, C, Hq, D] bf16 (device, 8-byte aligned) or NULL: gate logits;
 *           the output is multiplied elementwise by 1 / (1 + e^(-gate))
 *           before rounding to bf16 (the logits come from the layer's own
 *           trained projection, outside this library)
 * Other arguments, ownership and errors as for hs2_sparse_attn.               */
hs2_status hs2_sparse_attn_ex(const hs2_dims* dims, const uint16_t* q, const uint16_t* K, const uint16_t* V,
                              const int32_t* len, const int32_t* idx, int32_t n_slots, const float* sink,
                              const uint16_t* gate, uint16_t* out, void* workspace, size_t workspace_bytes,
                              void* stream);

/* FP8 KV cache.  The paper sizes every KV cache it reports in FP8 storage
 * (Sec. "Evaluation", paragraph on prefill computation and KV-cache storage);
 * it does not fix the format or the scaling, so these entry points take
 * OCP E4M3 bytes (bias 7, subnormals, no infinities, 0x7F/0xFF = NaN, largest
 * finite 448) with one fp32 scale per KV head and tensor: the cache stands for
 *   K(b, g, t, d) = k_scale[g] * e4m3(K8[...]),  V likewise with v_scale[g].
 * The math is that of the bf16 entry points on these dequantised values
 * (fp32 accumulation), so a cache holding the same values gives the same
 * selection and, up to rounding order, the same outputs.
 *
 *   K8, V8   uint8 [..] with the element offsets of hs2_dims (one byte each);
 *            kv_stride_b, kv_stride_h and kv_stride_t must be multiples of 16
 *            (HS2_ERR_ALIGN), K8 and V8 16-byte aligned
 *   k_scale, v_scale  [Hkv] float (device, 4-byte aligned), both required
 *            (HS2_ERR_NULL); finite and > 0 for meaningful results
 * Other arguments, outputs, ownership and errors as for
 * hs2_full_attn_score_select and hs2_sparse_attn_ex respectively; the same
 * hs2_workspace_bytes() covers both cache formats.                            */
hs2_status hs2_full_attn_score_select_fp8(const hs2_dims* dims, const uint16_t* q, const uint8_t* K8,
                                          const uint8_t* V8, const float* k_scale, const float* v_scale,
                                          const int32_t* len, int32_t k, int32_t window, uint16_t* out,
                                          int32_t* idx, float* stats, float* scores, void* workspace,
                                          size_t workspace_bytes, void* stream);
hs2_status hs2_sparse_attn_fp8(const hs2_dims* dims, const uint16_t* q, const uint8_t* K8, const uint8_t* V8,
                               const float* k_scale, const float* v_scale, const int32_t* len, const int32_t* idx,
                               int32_t n_slots, const float* sink, const uint16_t* gate, uint16_t* out,
                               void* workspace, size_t workspace_bytes, void* stream);

/* hs2_sparse_attn without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the layer's scratch (its split
 * partials) is a static device array of 16 MiB inside the library, one per
 * GPU, held until the process ends.  The call itself allocates nothing.
 *   - arguments, outputs and results as for hs2_sparse_attn (same kernels,
 *     same splits: the output is bit-identical to hs2_sparse_attn's);
 *   - a layer needing more than 16 MiB of scratch (rows B * Hkv * C times
 *     its splits times the head rows) is rejected with HS2_ERR_WORKSPACE
 *     before anything is launched; the benchmark shapes need 6-10 MiB;
 *   - every call on one GPU uses that GPU's one array: calls that overlap on
 *     one GPU (other streams, other host threads) race and must be ordered
 *     by the caller; nothing in the array needs clearing between calls.   */
hs2_status hs2_sparse_attn_noalloc(const hs2_dims* dims, const uint16_t* q, const uint16_t* K, const uint16_t* V,
                                   const int32_t* len, const int32_t* idx, int32_t n_slots, uint16_t* out,
                                   void* stream);

/* Block-level selection: the granularity of the predecessor HySparse, which
 * the paper compares against (Sec. "Ablation 1: Token-Level versus
 * Block-Level Sparsity": blocks of 64 tokens, the same global budget and the
 * same local window).  The same full-attention layer and pooled scores as
 * hs2_full_attn_score_select; then the N candidates before the window are
 * cut into blocks [j*block, (j+1)*block), the last one cut short at N; a
 * block's score is the sum of its candidates' pooled scores (each below
 * FLT_MIN counting as zero; the paper does not restate how a block is
 * scored), summed in fp32; the k / block best blocks (score descending,
 * lower block first among equal scores) are selected.  idx rows hold the
 * tokens of the selected blocks, then the window: ascending, -1 padded to
 * k + window.  The sparse layers take these rows unchanged.
 *
 *   block   a power of two in [16, 256], k a multiple of it (HS2_ERR_SHAPE);
 *           ceil(max_len / block) <= 16384 (HS2_ERR_UNSUPPORTED)
 * Other arguments, outputs, ownership and errors as for
 * hs2_full_attn_score_select (bf16 cache).                                   */
hs2_status hs2_full_attn_score_select_blocks(const hs2_dims* dims, const uint16_t* q, const uint16_t* K,
                                             const uint16_t* V, const int32_t* len, int32_t k, int32_t window,
                                             int32_t block, uint16_t* out, int32_t* idx, float* stats,
                                             float* scores, void* workspace, size_t workspace_bytes,
                                             void* stream);

/* Block-level selection alone, from caller-given pooled scores
 * [B, Hkv, C, max_len] float (device; entries [0, N) of each row are read,
 * >= 0 and finite), exactly the selection kernels of
 * hs2_full_attn_score_select_blocks (test and diagnostics).                  */
hs2_status hs2_select_blocks_from_scores(const hs2_dims* dims, const float* scores, const int32_t* len, int32_t k,
                                         int32_t window, int32_t block, int32_t* idx, void* workspace,
                                         size_t workspace_bytes, void* stream);

/* Selection alone, from caller-given pooled scores (test and diagnostics).
 * Runs exactly the selection kernels of hs2_full_attn_score_select on
 * scores [B, Hkv, C, max_len] float (device; entries [0, N) of each row are
 * read, must be >= 0 and finite) and writes idx as described there.          */
hs2_status hs2_select_from_scores(const hs2_dims* dims, const float* scores, const int32_t* len, int32_t k,
                                  int32_t window, int32_t* idx, void* workspace, size_t workspace_bytes,
                                  void* stream);

/* Streaming-read probe (diagnostics): reads the `bytes` bytes at device
 * address `src` once and xors a fold of them into *sink.  Over a buffer much
 * larger than the 256 MB last-level cache its rate is the device's practical
 * streaming-read ceiling, which the streaming kernels of this library are
 * reported against next to the nominal HBM peak.
 *   mode    0: 16-byte register loads; 1: the same with the non-temporal
 *           hint; 2: 16-byte direct-to-LDS loads, the loads the
 *           full-attention and score kernels issue; 3: the same
 *           non-temporal; 4 and 5: gathers, the rate of the sparse
 *           layers' access pattern -- the buffer as records of 512 (mode 4:
 *           a token's K and V in a bf16 cache of head dim 128) or 256 bytes
 *           (mode 5: E4M3) read in a scattered order (a fixed permutation,
 *           each record once) by the same direct-to-LDS loads; bytes must
 *           be the record size times a power of two, else HS2_ERR_SHAPE
 *           (other modes: HS2_ERR_SHAPE)
 *   src     16-byte aligned, bytes a multiple of 16 (HS2_ERR_ALIGN), bytes > 0
 *   sink    device array of HS2_STREAM_PROBE_SINK_WORDS uint32, 4-byte
 *           aligned (HS2_ERR_NULL if NULL); overwritten
 * Asynchronous on `stream`; launches one kernel of HS2_STREAM_PROBE_SINK_WORDS
 * workgroups, each of which stores the xor of the 32-bit words of its slice
 * to its own word of sink (the xor of all sink words is the xor of the
 * buffer).                                                                    */
#define HS2_STREAM_PROBE_SINK_WORDS 4096
hs2_status hs2_stream_read_probe(const void* src, size_t bytes, int32_t mode, uint32_t* sink, void* stream);

/* Static description of a status code. */
const char* hs2_status_string(int32_t status);

/* Message of the last failed call on this host thread ("" if none). */
const char* hs2_last_error(void);

/* Per-kernel timing (diagnostics).  While enabled, every kernel launch of this
 * library is bracketed by a pair of HIP events recorded on the launch stream
 * (up to a fixed number of launches).  hs2_timing_read() waits for the
 * recorded events, then fills, for up to `max_kernels` kernel kinds that ran,
 * their names (NUL-separated into `names`), launch counts and total
 * milliseconds; it returns the number of kinds written, or a negative status.
 * hs2_timing_reset() discards the records.  Not thread-safe.                  */
hs2_status hs2_timing_enable(int32_t on);
void hs2_timing_reset(void);
int32_t hs2_timing_read(char* names, size_t names_len, int32_t* counts, double* total_ms, int32_t max_kernels);

#ifdef __cplusplus
}
#endif
#endif /* HS2_H */
