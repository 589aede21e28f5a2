/*
 * litevlm.h - C ABI of the LiteVLM select + prefill path on MI355X (gfx950).
 *
 * Paper: "LiteVLM: A Low-Latency Vision-Language Model Inference Pipeline for
 * Resource-Constrained Environments" (arXiv 2506.07416).
 *
 * Calls in pipeline order, all enqueued on one HIP stream:
 *   litevlm_psm_forward       the Patch Selection Module's view logits from the query
 *   litevlm_patch_select      view selection and per-view patch masking
 *   litevlm_token_score_topk  text-guided visual-token scoring, top-k, compaction
 *                             (litevlm_token_score_topk_rows: the last n text rows only;
 *                             litevlm_select_score_topk: with the patch selection inside)
 *   litevlm_prefill_attn      causal GQA prefill attention over the compacted sequence
 * in front of the scoring, from the hidden states:
 *   litevlm_tsm_qk            the Token Selection Module's scoring queries and keys
 *                             (litevlm_tsm_fold_gain prepares its weights;
 *                             litevlm_gather_hidden compacts the hidden states for the LLM)
 * and, for the token generated after the prefill:
 *   litevlm_decode_attn       extend-one decode attention over the compacted KV cache
 *
 * Conventions shared by every call
 *   - Pointers marked "dev" are device pointers owned by the caller; the library
 *     never allocates, frees or keeps them after the call returns. "host" pointers
 *     are read during the call only.
 *   - Device pointers to tensors of Q/K/V/O and the workspace must be 16-byte
 *     aligned; other device pointers 4-byte aligned (1-byte for uint8 arrays).
 *     Tensors are dense and row-major in the stated layout (last index fastest).
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream). Calls
 *     only enqueue work and return; results are valid after the stream is
 *     synchronised. Nothing in the three calls synchronises with the host.
 *   - Every argument is validated on the host before anything is enqueued. On
 *     any error status nothing is launched and no output is written.
 *     LITEVLM_ERR_HIP reports a failed launch; faults inside kernels surface at
 *     the caller's next synchronisation, as usual in HIP.
 *   - Results are deterministic: identical inputs give bitwise-identical outputs
 *     (fixed reduction orders, no floating-point atomics).
 *   - Calls are reentrant and keep no global mutable state, except
 *     litevlm_token_score_topk_noalloc, which works in a device array of the
 *     library (see there).
 *
 * Sequence layout: visual tokens of view v occupy positions
 * [view_offsets[v], view_offsets[v+1]), views in order, view_offsets[0] = 0,
 * view_offsets[N] = V_full; text tokens occupy [V_full, S), T = S - V_full.
 */
#ifndef LITEVLM_H
#define LITEVLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LITEVLM_OK = 0,
  LITEVLM_ERR_NULL_POINTER = 1, /* a required pointer is NULL */
  LITEVLM_ERR_BAD_SHAPE = 2,    /* a size is out of range or inconsistent */
  LITEVLM_ERR_BAD_VALUE = 3,    /* a scalar argument is out of range or not finite */
  LITEVLM_ERR_UNSUPPORTED = 4,  /* valid request this build does not implement */
  LITEVLM_ERR_MISALIGNED = 5,   /* a pointer violates the alignment rule */
  LITEVLM_ERR_WORKSPACE = 6,    /* workspace NULL or smaller than required */
  LITEVLM_ERR_HIP = 7           /* a HIP runtime call or kernel launch failed */
} litevlm_status_t;

typedef enum {
  LITEVLM_F32 = 0,      /* IEEE binary32 */
  LITEVLM_BF16 = 1,     /* bfloat16 */
  LITEVLM_FP8_E4M3 = 2  /* OCP E4M3FN (bias 7, max 448, no inf), with a per-tensor fp32 scale */
} litevlm_dtype_t;

/* Limits of this build. */
#define LITEVLM_MAX_VIEWS 64      /* N */
#define LITEVLM_MAX_VISUAL 16384  /* V_full (top-k keeps every key of a sample in LDS) */
#define LITEVLM_MAX_BATCH 256     /* B */
#define LITEVLM_MAX_HEADS 128     /* Hq (the gather copies a token's Q, K, V rows in one pass) */

/* Library version as major*10000 + minor*100 + patch. */
int32_t litevlm_version(void);

/* Static string naming a status code (never NULL). */
const char* litevlm_status_string(int32_t status);

/*
 * litevlm_patch_select - view selection and patch masking.
 *
 * Paper: Design section, Patch Selection Module paragraph (the final view score
 * is a weighted sum of a lexical mapping and the module's logits; views scoring
 * above a threshold are kept, and only their patches proceed); Experiments
 * section, Training paragraph (only the selected views' patches reach the
 * vision encoder, hence the LLM).
 *
 * Per sample b and view v:
 *   s_v = w_lexical * lex_v + (1 - w_lexical) * sigmoid(logit_v)   (fp32, no FMA contraction)
 *   keep_v = (s_v > threshold); if no view passes, the single best view is kept
 *   (the lowest v among equal best scores).
 *
 *   B, N, S            batch, views (1..LITEVLM_MAX_VIEWS), sequence length
 *   view_offsets_host  host int32 [N+1]: ascending, off[0] = 0, off[N] = V_full <= S
 *   view_logit         dev fp32 [B, N]: the selection module's per-view logits
 *   view_lexical       dev fp32 [B, N] lexical scores in [0, 1], or NULL (= 0)
 *   w_lexical          weight of the lexical term, in [0, 1]
 *   threshold          keep threshold on the fused score (finite)
 *   view_keep          dev out uint8 [B, N]: 1 = view kept
 *   token_keep         dev out uint8 [B, S]: 1 for tokens of kept views and for all text tokens
 *   n_visual_kept      dev out int32 [B]: V_b, the visual tokens that survive (may be NULL)
 */
litevlm_status_t litevlm_patch_select(int32_t B, int32_t N, int32_t S,
                                      const int32_t* view_offsets_host,
                                      const float* view_logit, const float* view_lexical,
                                      float w_lexical, float threshold,
                                      uint8_t* view_keep, uint8_t* token_keep,
                                      int32_t* n_visual_kept, void* stream);

/* Bytes of device workspace litevlm_token_score_topk needs for these sizes
 * (0 when the sizes are invalid). */
size_t litevlm_token_score_topk_workspace(int32_t B, int32_t S, int32_t V_full,
                                          int32_t Hq, int32_t Hkv, int32_t D);

/*
 * litevlm_token_score_topk - visual-token importance, top-k and compaction.
 *
 * Paper: Design section, Token Selection Module paragraph (the first decoder
 * layer, run standalone, scores visual tokens from self-attention, in the
 * manner of FastV; pruning happens before the LLM); Results section, Visual
 * Token Compression paragraph and Table 1 (compression ratio r; token counts).
 *
 * Per sample b, with the patch-selected sequence = kept visual tokens (in
 * order) followed by all T text tokens, V_b = kept visual count:
 *   score_b(j) = 1/(Hq*T) * sum_h sum_t softmax_j'(q_{t,h} . k_{j',h/G} * scale)[j]
 *     where text token t sits at position V_b + t of that sequence and its
 *     causal row spans positions 0..V_b+t; scale = softmax_scale*q_scale*k_scale.
 *     Visual tokens of dropped views score -INFINITY.
 *   k_b = min(V_b, floor(keep_ratio*V_b + 1e-6)), in IEEE double.
 *   Kept visual tokens: the first k_b in (score descending, position ascending)
 *     order; exactly equal scores keep the lower position.
 *   Compacted sequence: kept visual positions ascending, then text positions
 *     V_full..S-1. cu_seqlens[b+1] - cu_seqlens[b] = k_b + T.
 *
 *   dtype              LITEVLM_F32, LITEVLM_BF16 or LITEVLM_FP8_E4M3 (Q, K, V, qc, kc, vc)
 *   B, S, V_full       batch (1..LITEVLM_MAX_BATCH), sequence length, visual tokens (T = S - V_full >= 1)
 *   Hq, Hkv, D         query heads (1..LITEVLM_MAX_HEADS), KV heads (Hq % Hkv == 0),
 *                      head dim (64 or 128)
 *   q                  dev [B, S, Hq, D]
 *   k                  dev [B, S, Hkv, D]
 *   v                  dev [B, S, Hkv, D] (may be NULL when vc is NULL)
 *   softmax_scale      logit scale, normally 1/sqrt(D) (finite, > 0)
 *   q_scale, k_scale, v_scale   fp8 dequantisation scales (finite, > 0); must be 1 otherwise
 *   token_keep         dev uint8 [B, S] from litevlm_patch_select, or NULL = all kept;
 *                      only positions < V_full are read (text is always kept)
 *   keep_ratio         r in [0, 1]
 *   scores             dev out fp32 [B, V_full]
 *   kept_index         dev out int32, capacity B*S: packed compacted positions
 *                      (positions within the sample), segment b at cu_seqlens[b]
 *   cu_seqlens         dev out int32 [B+1]
 *   qc, kc, vc         dev out packed rows of Q, K, V at kept_index, capacity B*S
 *                      rows of Hq*D / Hkv*D / Hkv*D elements, exact copies of the
 *                      input bits; each may be NULL to skip that copy
 *   workspace          dev scratch of litevlm_token_score_topk_workspace() bytes;
 *                      its contents on entry are ignored, and calls that may run
 *                      concurrently must not share one workspace
 */
litevlm_status_t litevlm_token_score_topk(int32_t dtype, int32_t B, int32_t S, int32_t V_full,
                                          int32_t Hq, int32_t Hkv, int32_t D,
                                          const void* q, const void* k, const void* v,
                                          float softmax_scale, float q_scale, float k_scale,
                                          float v_scale, const uint8_t* token_keep,
                                          double keep_ratio, float* scores, int32_t* kept_index,
                                          int32_t* cu_seqlens, void* qc, void* kc, void* vc,
                                          void* workspace, size_t workspace_bytes, void* stream);

/* Most views litevlm_select_score_topk takes (the selection is taken inside
 * every scoring workgroup, one comparison per view offset). */
#define LITEVLM_MAX_FUSED_VIEWS 8

/*
 * litevlm_select_score_topk - litevlm_patch_select and litevlm_token_score_topk
 * in one call: the scoring kernels take the view selection themselves from the
 * view logits, so the step needs no token mask between the two.
 *
 * Paper: Design section, Patch Selection Module and Token Selection Module
 * paragraphs (the selected views' patches are what the token scoring sees);
 * the rest as for the two calls.
 *
 * The view decision (view_keep, the token mask, n_visual_kept) is that of
 * litevlm_patch_select with these N, view offsets, logits, lexical scores,
 * w_lexical and threshold, bit for bit: the same fp32 decision, evaluated by
 * the same device code. The rest is litevlm_token_score_topk on that token
 * mask:
 *   - bit for bit for B = 1;
 *   - for 2 <= B <= 16 (where the shape gives the first sweep at least two
 *     key splits per (sample, KV group, 512-row block) and at most 256 key
 *     tiles of 64 per sample; bit for bit otherwise) the first score sweep
 *     splits the live key tiles (those of kept views, and the text) in
 *     proportion over the samples. That split
 *     follows from the view masks, which this call has and the two-call path
 *     does not. Its partial sums round differently, so a score may differ
 *     from the two-call path in its last bits (well within 1e-5 relative), and
 *     the kept set only where scores tie within such a difference.
 * Both paths are deterministic.
 *
 *   N                  views, 1..LITEVLM_MAX_FUSED_VIEWS (N up to LITEVLM_MAX_VIEWS:
 *                      LITEVLM_ERR_UNSUPPORTED; use the two calls)
 *   view_offsets_host  host int32 [N+1]: view v holds visual positions
 *                      [off[v], off[v+1]), off[0] = 0, non-decreasing, off[N] = V_full
 *   view_logit, view_lexical, w_lexical, threshold   as for litevlm_patch_select
 *   view_keep          dev out uint8 [B, N], or NULL
 *   token_keep         dev out uint8 [B, S] (the token mask), or NULL
 *   n_visual_kept      dev out int32 [B], or NULL
 *   other arguments    as for litevlm_token_score_topk (the workspace size is
 *                      litevlm_token_score_topk_workspace())
 */
litevlm_status_t litevlm_select_score_topk(int32_t dtype, int32_t B, int32_t S, int32_t V_full, int32_t Hq,
                                           int32_t Hkv, int32_t D, int32_t N, const int32_t* view_offsets_host,
                                           const float* view_logit, const float* view_lexical, float w_lexical,
                                           float threshold, const void* q, const void* k, const void* v,
                                           float softmax_scale, float q_scale, float k_scale, float v_scale,
                                           double keep_ratio, uint8_t* view_keep, uint8_t* token_keep,
                                           int32_t* n_visual_kept, float* scores, int32_t* kept_index,
                                           int32_t* cu_seqlens, void* qc, void* kc, void* vc, void* workspace,
                                           size_t workspace_bytes, void* stream);

/* Size of the device scratch array of litevlm_token_score_topk_noalloc (8 MiB
 * per GPU, held from the first such call on a GPU until the process ends). */
#define LITEVLM_NOALLOC_SCRATCH_BYTES (8u << 20)

/*
 * litevlm_token_score_topk_noalloc - litevlm_token_score_topk for callers that
 * cannot allocate device memory (code under HIP graph capture, serving loops
 * that forbid allocation): the same computation, arguments, layouts and
 * results, with the workspace taken from a static device array of the library
 * instead of a caller buffer. It calls no hipMalloc, hipFree or allocating
 * routine; the array's device address is looked up once per device (on the
 * first call made with that device current).
 *
 * Limit: the workspace of the sizes, litevlm_token_score_topk_workspace(B, S,
 * V_full, Hq, Hkv, D), must fit LITEVLM_NOALLOC_SCRATCH_BYTES, else the call
 * returns LITEVLM_ERR_WORKSPACE and launches nothing. Every call on one GPU
 * shares that GPU's array, so calls that may overlap on one GPU (other
 * streams, other host threads) race and give undefined results; calls on one
 * stream are ordered and safe. The array keeps the last call's contents, which
 * no call reads before writing.
 */
litevlm_status_t litevlm_token_score_topk_noalloc(int32_t dtype, int32_t B, int32_t S, int32_t V_full,
                                                  int32_t Hq, int32_t Hkv, int32_t D,
                                                  const void* q, const void* k, const void* v,
                                                  float softmax_scale, float q_scale, float k_scale,
                                                  float v_scale, const uint8_t* token_keep,
                                                  double keep_ratio, float* scores, int32_t* kept_index,
                                                  int32_t* cu_seqlens, void* qc, void* kc, void* vc,
                                                  void* stream);

/* Bytes of device workspace litevlm_token_score_topk_rows needs for these
 * sizes (0 when the sizes or query_rows are invalid). */
size_t litevlm_token_score_topk_rows_workspace(int32_t B, int32_t S, int32_t V_full,
                                               int32_t Hq, int32_t Hkv, int32_t D,
                                               int32_t query_rows);

/*
 * litevlm_token_score_topk_rows - litevlm_token_score_topk with only the last
 * query_rows text tokens as query rows.
 *
 * Paper: Related Work, Visual Token Compression (FastV prunes visual tokens by
 * the attention that the last token pays them, inside the LLM after an early
 * layer); the scoring of litevlm_token_score_topk is otherwise unchanged.
 *
 *   score_b(j) = 1/(Hq*n) * sum_h sum_{t = T-n}^{T-1} softmax(...)[j], n = query_rows,
 * with the rows, masks, k_b rule, top-k order and compaction exactly as in
 * litevlm_token_score_topk (the compacted sequence still keeps every text
 * token). query_rows = 1 is the last-token readout; query_rows = T is
 * litevlm_token_score_topk. query_rows outside 1..T gives LITEVLM_ERR_BAD_VALUE.
 * The workspace comes from litevlm_token_score_topk_rows_workspace(); every
 * other argument, its layout, ownership and errors are those of
 * litevlm_token_score_topk.
 */
litevlm_status_t litevlm_token_score_topk_rows(int32_t dtype, int32_t B, int32_t S, int32_t V_full,
                                               int32_t Hq, int32_t Hkv, int32_t D, int32_t query_rows,
                                               const void* q, const void* k, const void* v,
                                               float softmax_scale, float q_scale, float k_scale,
                                               float v_scale, const uint8_t* token_keep,
                                               double keep_ratio, float* scores, int32_t* kept_index,
                                               int32_t* cu_seqlens, void* qc, void* kc, void* vc,
                                               void* workspace, size_t workspace_bytes, void* stream);

/*
 * litevlm_prefill_attn - causal GQA prefill attention over packed sequences.
 *
 * Paper: Introduction and Related Work, Visual Token Compression (prefill
 * processes the whole sequence, and self-attention's quadratic cost is what
 * token compression saves); Figure 3b (prefill latency against input tokens,
 * FP16 and FP8); Experiments section, Deployment paragraph (FP8 PTQ).
 *
 * For each sample b (rows cu_seqlens[b]..cu_seqlens[b+1]-1) and query head h:
 *   O[i,h] = sum_j softmax_j(l_ij) V[j, h/G],  l_ij = q_i . k_j * softmax_scale*q_scale*k_scale,
 *   keys j <= i when causal (positions within the sample), all keys otherwise;
 *   the result is multiplied by v_scale. Softmax and accumulation in fp32.
 *
 *   in_dtype           LITEVLM_F32, LITEVLM_BF16 or LITEVLM_FP8_E4M3
 *   out_dtype          LITEVLM_F32 or LITEVLM_BF16 (BF16 is the normal output for BF16/FP8 input)
 *   B, Hq, Hkv, D      batch, heads (Hq % Hkv == 0), head dim (64 or 128)
 *   qc                 dev [total, Hq, D]; kc, vc dev [total, Hkv, D]; total = cu_seqlens[B]
 *   cu_seqlens         dev int32 [B+1], non-decreasing, cu_seqlens[0] = 0
 *   max_seqlen         host upper bound on every cu_seqlens[b+1]-cu_seqlens[b]; the
 *                      grid is sized from it and surplus tiles exit at once.
 *                      Segments longer than max_seqlen are undefined behaviour.
 *   softmax_scale, q_scale, k_scale, v_scale   finite, > 0; scales must be 1 unless FP8
 *   causal             1 = causal (the prefill path), 0 = full attention
 *   o                  dev out [total, Hq, D] in out_dtype
 */
litevlm_status_t litevlm_prefill_attn(int32_t in_dtype, int32_t out_dtype, int32_t B,
                                      int32_t Hq, int32_t Hkv, int32_t D,
                                      const void* qc, const void* kc, const void* vc,
                                      const int32_t* cu_seqlens, int32_t max_seqlen,
                                      float softmax_scale, float q_scale, float k_scale,
                                      float v_scale, int32_t causal, void* o, void* stream);

/*
 * litevlm_tsm_qk - the Token Selection Module's scoring queries and keys from
 * the hidden states entering its decoder layer.
 *
 * Paper: Design section, Token Selection Module paragraph (the first decoder
 * layer of the finetuned LLM, run standalone, scores the visual tokens);
 * Experiments section (the decoder is InternLM2.5). The layer's attention takes
 * its queries and keys from RMS-normalised hidden states through bias-free
 * projections and rotary position embeddings:
 *   r_j      = 1 / sqrt(mean_c x[b,j,c]^2 + eps)
 *   k[b,j,h] = rope(r_j * (x[b,j] . W_k'[h*D:(h+1)*D]), pos_j)   for every kept token j
 *   q[b,t,h] = rope(r_t * (x[b,t] . W_q'[h*D:(h+1)*D]), pos_t)   for the text tokens t
 *   rope pairs element d < D/2 of a head with element d + D/2 and rotates the
 *   pair by the angle pos * rope_theta^(-2d/D);
 *   pos_j = the number of kept tokens before j (its position in the
 *   patch-selected sequence; token_keep NULL: pos_j = j).
 * Products in bf16 on MFMA with fp32 accumulation; the outputs are rounded to
 * bf16. The results are the q and k that litevlm_token_score_topk reads.
 *
 *   B, S, V_full       batch, sequence length, visual tokens (T = S - V_full >= 1)
 *   Dm                 model width: a multiple of 64, at most 65536
 *   Hq, Hkv, D         heads (Hq % Hkv == 0), head dim 64 or 128; Hq*D and Hkv*D must
 *                      be multiples of 128 (else LITEVLM_ERR_UNSUPPORTED)
 *   hidden             dev bf16 [B, S, Dm]
 *   token_keep         dev uint8 [B, S] from litevlm_patch_select, or NULL
 *   w_q, w_k           dev bf16 [Hq*D, Dm], [Hkv*D, Dm]: the projections with the RMS
 *                      normalisation gain folded in (litevlm_tsm_fold_gain)
 *   eps                RMS normalisation epsilon (finite, > 0)
 *   rope_theta         rotary base (finite, > 1)
 *   q                  dev out bf16 [B, S, Hq, D]: rows V_full..S-1 of every sample are
 *                      written, the visual rows are left untouched
 *   k                  dev out bf16 [B, S, Hkv, D]: the rows of kept tokens are written
 *                      (every row when token_keep is NULL); the rows of dropped tokens
 *                      are left untouched, since the scoring never reads them
 */
litevlm_status_t litevlm_tsm_qk(int32_t B, int32_t S, int32_t V_full, int32_t Dm, int32_t Hq, int32_t Hkv,
                                int32_t D, const void* hidden, const uint8_t* token_keep, const void* w_q,
                                const void* w_k, float eps, float rope_theta, void* q, void* k,
                                void* stream);

/* Number of float32 parameters of the Patch Selection Module (0 if a size is < 1). */
size_t litevlm_psm_param_count(int32_t d, int32_t d_ff, int32_t n_views, int32_t n_layers);

/* Bytes of device workspace litevlm_psm_forward needs (0 when the sizes are invalid). */
size_t litevlm_psm_workspace(int32_t B, int32_t T, int32_t d, int32_t n_heads, int32_t d_ff);

/*
 * litevlm_psm_forward - the Patch Selection Module: view logits from the text
 * query's token embeddings.
 *
 * Paper: Design section, Patch Selection Module paragraph (a small transformer
 * encoder of 4 layers over the tokenised query; a cross-attention with N
 * learnable latent queries, one per camera view; each view's result mapped to
 * an independent logit). Its logits are the view_logit of litevlm_patch_select.
 *
 * Per sample, with h = emb (T tokens of width d):
 *   each of n_layers layers:  h += MHA(LN1(h));  h += W_down GELU(W_up LN2(h) + b_up) + b_down
 *     (pre-norm; LayerNorm eps 1e-5 with gain and bias; MHA with n_heads heads and
 *     biased in/out projections; exact erf GELU)
 *   X = LNf(h);  q_v = latent_v W_cq^T + b_cq;  K = X W_ck^T + b_ck;  V = X W_cv^T + b_cv
 *   logit_v = w_head_v . (softmax(q_v K^T / sqrt(d)) V) + b_head_v
 * The GEMM and attention inputs are rounded to bf16 (MFMA, fp32 accumulation);
 * the residual stream, the norms and the cross-attention run in fp32.
 *
 *   B, T               batch (1..LITEVLM_MAX_BATCH), query tokens (1..8192)
 *   d, n_heads, d_ff   width 256 or 512; d / n_heads = 64 or 128 (else
 *                      LITEVLM_ERR_UNSUPPORTED); d_ff a multiple of 64 (<= 16384)
 *   n_views, n_layers  N (1..LITEVLM_MAX_VIEWS), encoder layers (1..64)
 *   emb                dev fp32 [B, T, d]
 *   params             dev fp32, n_params = litevlm_psm_param_count(d, d_ff, n_views,
 *                      n_layers) values in this order: per layer ln1 gain [d], ln1 bias
 *                      [d], QKV weight [3d, d] (rows: q, k, v outputs), QKV bias [3d],
 *                      output weight [d, d], output bias [d], ln2 gain [d], ln2 bias [d],
 *                      up weight [d_ff, d], up bias [d_ff], down weight [d, d_ff], down
 *                      bias [d]; then final-norm gain [d], bias [d], latents [N, d],
 *                      cross Q weight [d, d], bias [d], cross K weight [d, d], bias [d],
 *                      cross V weight [d, d], bias [d], head weights [N, d], head biases [N]
 *                      (a weight [out, in] maps x to x W^T); another count gives
 *                      LITEVLM_ERR_BAD_SHAPE
 *   view_logit         dev out fp32 [B, n_views]
 *   workspace          dev scratch of litevlm_psm_workspace() bytes (contents on entry
 *                      ignored; calls that may run concurrently must not share one)
 */
litevlm_status_t litevlm_psm_forward(int32_t B, int32_t T, int32_t d, int32_t n_heads, int32_t d_ff,
                                     int32_t n_views, int32_t n_layers, const float* emb, const float* params,
                                     size_t n_params, float* view_logit, void* workspace,
                                     size_t workspace_bytes, void* stream);

/*
 * litevlm_gather_hidden - the compacted hidden states for the LLM: packed row r
 * of sample b (rows cu_seqlens[b]..cu_seqlens[b+1]-1) is an exact copy of row
 * kept_index[r] of that sample's hidden states.
 *
 * Paper: Design section, Token Selection Module paragraph (the pruned visual
 * tokens do not enter the LLM: what the LLM prefills is the kept tokens' hidden
 * states, which its own first layer projects).
 *
 *   B, S               batch, rows per sample of hidden
 *   row_bytes          bytes per row (a multiple of 16, at most 196608)
 *   hidden             dev [B, S, row_bytes]
 *   kept_index, cu_seqlens   dev int32, as written by litevlm_token_score_topk
 *                      (values of kept_index must lie in [0, S))
 *   out                dev [total, row_bytes], total = cu_seqlens[B] (capacity B*S rows;
 *                      rows past total are untouched)
 */
litevlm_status_t litevlm_gather_hidden(int32_t B, int32_t S, int32_t row_bytes, const void* hidden,
                                       const int32_t* kept_index, const int32_t* cu_seqlens, void* out,
                                       void* stream);

/*
 * litevlm_tsm_fold_gain - w_out[n, c] = bf16(w[n, c] * gamma[c]): folds the RMS
 * normalisation gain into the projection that follows it, once per set of
 * weights (the form litevlm_tsm_qk takes). w and w_out are dev bf16
 * [rows, cols] (may be the same buffer), gamma dev fp32 [cols].
 */
litevlm_status_t litevlm_tsm_fold_gain(int32_t rows, int32_t cols, const void* w, const float* gamma,
                                       void* w_out, void* stream);

/* Bytes of device workspace litevlm_decode_attn needs for these sizes (0 when
 * the sizes are invalid or unsupported). */
size_t litevlm_decode_attn_workspace(int32_t in_dtype, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
                                     int32_t max_seqlen);

/*
 * litevlm_decode_attn - extend-one decode attention over the compacted KV cache.
 *
 * Paper: Results section (after the prefill, each output token is decoded
 * against the cached keys and values; the paper measures how little a 3x
 * token cut saves in this phase, because each decoded token makes one pass
 * over the cache).
 *
 * For each sample b, with the cache rows cu_seqlens[b]..cu_seqlens[b+1]-1 of
 * kc, vc (n_b = cu_seqlens[b+1]-cu_seqlens[b] rows, the compacted sequence of
 * the prefill) followed by the new token's own key k1[b] and value v1[b]:
 *   o[b,h] = v_scale * sum_j softmax_j(l_j) V_j,  l_j = q1[b,h] . K_j * softmax_scale*q_scale*k_scale,
 *   j over the n_b cached tokens and the new token (which comes last and sees
 *   everything before it, so no mask applies); query head h reads KV head h/G.
 *   Softmax and accumulation in fp32.
 *
 *   in_dtype           LITEVLM_F32, LITEVLM_BF16 or LITEVLM_FP8_E4M3 (q1, k1, v1, kc, vc)
 *   out_dtype          LITEVLM_F32 or LITEVLM_BF16
 *   B, Hq, Hkv, D      batch, heads (G = Hq/Hkv in {1, 2, 4, 8}, else
 *                      LITEVLM_ERR_UNSUPPORTED), head dim (64 or 128)
 *   q1                 dev [B, Hq, D]: the new token's queries
 *   k1, v1             dev [B, Hkv, D]: the new token's key and value
 *   kc, vc             dev [total, Hkv, D], total = cu_seqlens[B]: the compacted cache
 *                      (the kc, vc of litevlm_token_score_topk)
 *   cu_seqlens         dev int32 [B+1], non-decreasing, cu_seqlens[0] = 0
 *   max_seqlen         host upper bound on every n_b; the split grid is sized from it
 *                      and surplus splits exit at once. Longer segments give
 *                      undefined values (no out-of-range access).
 *   softmax_scale, q_scale, k_scale, v_scale   finite, > 0; scales must be 1 unless FP8
 *   o                  dev out [B, Hq, D] in out_dtype
 *   workspace          dev scratch of litevlm_decode_attn_workspace() bytes (partial
 *                      results of the key splits); contents on entry are ignored, and
 *                      calls that may run concurrently must not share one workspace
 */
litevlm_status_t litevlm_decode_attn(int32_t in_dtype, int32_t out_dtype, int32_t B, int32_t Hq,
                                     int32_t Hkv, int32_t D, const void* q1, const void* k1,
                                     const void* v1, const void* kc, const void* vc,
                                     const int32_t* cu_seqlens, int32_t max_seqlen,
                                     float softmax_scale, float q_scale, float k_scale,
                                     float v_scale, void* o, void* workspace,
                                     size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LITEVLM_H */
