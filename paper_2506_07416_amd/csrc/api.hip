// C ABI of the LiteVLM select + prefill path: host-side validation, workspace
// sizing and dispatch to the kernel launchers. Every check runs before any
// HIP call, so an error status means nothing was enqueued or written.
#include <math.h>

#include <mutex>

#include "launch.hpp"

using namespace litevlm;

namespace {

constexpr int32_t kVersion = 100;  // 0.1.0

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
bool finite_pos(float x) { return isfinite(x) && x > 0.f; }
bool valid_dtype(int dt) { return dt == LITEVLM_F32 || dt == LITEVLM_BF16 || dt == LITEVLM_FP8_E4M3; }

litevlm_status_t hip_status(hipError_t e) { return e == hipSuccess ? LITEVLM_OK : LITEVLM_ERR_HIP; }

litevlm_status_t check_score_shape(int32_t B, int32_t S, int32_t V_full, int32_t Hq, int32_t Hkv,
                                   int32_t D) {
  if (B < 1 || B > LITEVLM_MAX_BATCH) return LITEVLM_ERR_BAD_SHAPE;
  if (V_full < 0 || V_full > LITEVLM_MAX_VISUAL || S <= V_full) return LITEVLM_ERR_BAD_SHAPE;
  if (Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || Hq > LITEVLM_MAX_HEADS) return LITEVLM_ERR_BAD_SHAPE;
  if (D != 64 && D != 128) return LITEVLM_ERR_BAD_SHAPE;
  // keep every index computed in int32 inside range
  if ((int64_t)B * S * Hq * D > ((int64_t)1 << 40)) return LITEVLM_ERR_BAD_SHAPE;
  if ((int64_t)B * S > INT32_MAX / 2) return LITEVLM_ERR_BAD_SHAPE;
  return LITEVLM_OK;
}

// Decode: G = Hq/Hkv query heads per KV head must be 1, 2, 4 or 8 (the kernel
// holds every query head of a KV head in registers).
litevlm_status_t check_decode_shape(int32_t in_dtype, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
                                    int32_t max_seqlen) {
  if (!valid_dtype(in_dtype)) return LITEVLM_ERR_UNSUPPORTED;
  if (B < 1 || B > LITEVLM_MAX_BATCH || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 ||
      Hq > LITEVLM_MAX_HEADS || (D != 64 && D != 128) || max_seqlen < 0)
    return LITEVLM_ERR_BAD_SHAPE;
  if ((int64_t)B * (max_seqlen + 1) > INT32_MAX / 2) return LITEVLM_ERR_BAD_SHAPE;
  // the split grid (at most B*Hkv*((max_seqlen+64)/64) workgroups) must fit an int
  if ((int64_t)B * Hkv * ((max_seqlen + 64) / 64) > INT32_MAX) return LITEVLM_ERR_BAD_SHAPE;
  const int G = Hq / Hkv;
  if (G != 1 && G != 2 && G != 4 && G != 8) return LITEVLM_ERR_UNSUPPORTED;
  return LITEVLM_OK;
}

}  // namespace

extern "C" {

int32_t litevlm_version(void) { return kVersion; }

const char* litevlm_status_string(int32_t s) {
  switch (s) {
    case LITEVLM_OK: return "ok";
    case LITEVLM_ERR_NULL_POINTER: return "null pointer";
    case LITEVLM_ERR_BAD_SHAPE: return "bad shape";
    case LITEVLM_ERR_BAD_VALUE: return "bad value";
    case LITEVLM_ERR_UNSUPPORTED: return "unsupported";
    case LITEVLM_ERR_MISALIGNED: return "misaligned pointer";
    case LITEVLM_ERR_WORKSPACE: return "workspace too small";
    case LITEVLM_ERR_HIP: return "hip error";
    default: return "unknown status";
  }
}

litevlm_status_t litevlm_patch_select(int32_t B, int32_t N, int32_t S,
                                      const int32_t* view_offsets_host, const float* view_logit,
                                      const float* view_lexical, float w_lexical, float threshold,
                                      uint8_t* view_keep, uint8_t* token_keep,
                                      int32_t* n_visual_kept, void* stream) {
  if (!view_offsets_host || !view_logit || !view_keep || !token_keep) return LITEVLM_ERR_NULL_POINTER;
  if (B < 1 || B > LITEVLM_MAX_BATCH || N < 1 || N > LITEVLM_MAX_VIEWS || S < 1)
    return LITEVLM_ERR_BAD_SHAPE;
  ViewOffsets vo;
  if (view_offsets_host[0] != 0) return LITEVLM_ERR_BAD_SHAPE;
  for (int v = 0; v <= N; ++v) {
    vo.off[v] = view_offsets_host[v];
    if (v > 0 && vo.off[v] < vo.off[v - 1]) return LITEVLM_ERR_BAD_SHAPE;
  }
  if (vo.off[N] > S) return LITEVLM_ERR_BAD_SHAPE;
  if (!(w_lexical >= 0.f && w_lexical <= 1.f) || !isfinite(threshold)) return LITEVLM_ERR_BAD_VALUE;
  if (!aligned(view_logit, 4) || (view_lexical && !aligned(view_lexical, 4)) ||
      (n_visual_kept && !aligned(n_visual_kept, 4)))
    return LITEVLM_ERR_MISALIGNED;
  return hip_status(launch_patch_select(B, N, S, vo, view_logit, view_lexical, w_lexical, threshold,
                                        view_keep, token_keep, n_visual_kept,
                                        static_cast<hipStream_t>(stream)));
}

size_t litevlm_token_score_topk_rows_workspace(int32_t B, int32_t S, int32_t V_full, int32_t Hq,
                                               int32_t Hkv, int32_t D, int32_t query_rows) {
  if (check_score_shape(B, S, V_full, Hq, Hkv, D) != LITEVLM_OK) return 0;
  if (query_rows < 1 || query_rows > S - V_full) return 0;
  return score_workspace_layout(B, S, V_full, Hq, Hkv, query_rows).total;
}

size_t litevlm_token_score_topk_workspace(int32_t B, int32_t S, int32_t V_full, int32_t Hq,
                                          int32_t Hkv, int32_t D) {
  return litevlm_token_score_topk_rows_workspace(B, S, V_full, Hq, Hkv, D, S - V_full);
}

}  // extern "C"

namespace {

// Validation of every argument of the scoring call except the workspace.
litevlm_status_t check_score_args(int32_t dtype, int32_t B, int32_t S, int32_t V_full, int32_t Hq,
                                  int32_t Hkv, int32_t D, int32_t query_rows, const void* q, const void* k,
                                  const void* v, float softmax_scale, float q_scale, float k_scale,
                                  float v_scale, double keep_ratio, const float* scores,
                                  const int32_t* kept_index, const int32_t* cu_seqlens, const void* qc,
                                  const void* kc, const void* vc) {
  if (!q || !k || !scores || !kept_index || !cu_seqlens) return LITEVLM_ERR_NULL_POINTER;
  if (vc && !v) return LITEVLM_ERR_NULL_POINTER;
  if (!valid_dtype(dtype)) return LITEVLM_ERR_UNSUPPORTED;
  const litevlm_status_t sh = check_score_shape(B, S, V_full, Hq, Hkv, D);
  if (sh != LITEVLM_OK) return sh;
  if (query_rows < 1 || query_rows > S - V_full) return LITEVLM_ERR_BAD_VALUE;
  if (!finite_pos(softmax_scale) || !finite_pos(q_scale) || !finite_pos(k_scale) ||
      !finite_pos(v_scale))
    return LITEVLM_ERR_BAD_VALUE;
  if (dtype != LITEVLM_FP8_E4M3 && (q_scale != 1.f || k_scale != 1.f || v_scale != 1.f))
    return LITEVLM_ERR_BAD_VALUE;
  if (!(keep_ratio >= 0.0 && keep_ratio <= 1.0)) return LITEVLM_ERR_BAD_VALUE;
  const void* big[] = {q, k, v, qc, kc, vc};
  for (const void* p : big)
    if (p && !aligned(p, 16)) return LITEVLM_ERR_MISALIGNED;
  if (!aligned(scores, 4) || !aligned(kept_index, 4) || !aligned(cu_seqlens, 4))
    return LITEVLM_ERR_MISALIGNED;
  return LITEVLM_OK;
}

litevlm_status_t launch_score(int32_t dtype, int32_t B, int32_t S, int32_t V_full, int32_t Hq, int32_t Hkv,
                              int32_t D, int32_t query_rows, const void* q, const void* k, const void* v,
                              float softmax_scale, float q_scale, float k_scale, const uint8_t* token_keep,
                              double keep_ratio, float* scores, int32_t* kept_index, int32_t* cu_seqlens,
                              void* qc, void* kc, void* vc, void* workspace, void* stream,
                              const ViewSel* vs = nullptr, uint8_t* view_keep = nullptr,
                              uint8_t* token_keep_out = nullptr, int32_t* n_visual_kept = nullptr) {
  ScoreArgs a;
  a.dtype = dtype;
  a.B = B;
  a.S = S;
  a.V_full = V_full;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.D = D;
  a.query_rows = query_rows;
  a.q = q;
  a.k = k;
  a.v = v;
  a.logit_scale_log2 = (float)((double)softmax_scale * q_scale * k_scale * 1.4426950408889634);
  a.token_keep = token_keep;
  a.keep_ratio = keep_ratio;
  a.scores = scores;
  a.kept_index = kept_index;
  a.cu_seqlens = cu_seqlens;
  a.qc = qc;
  a.kc = kc;
  a.vc = vc;
  a.workspace = workspace;
  if (vs) {
    a.vs = *vs;
    a.view_keep = view_keep;
    a.token_keep_out = token_keep_out;
    a.n_visual_kept = n_visual_kept;
  }
  return hip_status(launch_token_score_topk(a, static_cast<hipStream_t>(stream)));
}

// Device scratch of litevlm_token_score_topk_noalloc: the workspace of the
// scoring call (per-split row statistics, fixed-point column sums) for callers
// that cannot allocate. Each GPU holds its own copy for the life of the
// process. In host code the name is only a host-side stand-in: its device
// address comes from hipGetSymbolAddress, once per device, and only that
// address is ever passed to kernels.
static __device__ __align__(256) uint8_t scratch[LITEVLM_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};  // device address of `scratch` per device ordinal

// The scratch array's device address on the current device, looked up on the
// first call made with that device current.
litevlm_status_t device_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return LITEVLM_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return LITEVLM_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return LITEVLM_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return LITEVLM_OK;
}

}  // namespace

extern "C" {

litevlm_status_t litevlm_token_score_topk_noalloc(int32_t dtype, int32_t B, int32_t S, int32_t V_full,
                                                  int32_t Hq, int32_t Hkv, int32_t D, const void* q,
                                                  const void* k, const void* v, float softmax_scale,
                                                  float q_scale, float k_scale, float v_scale,
                                                  const uint8_t* token_keep, double keep_ratio, float* scores,
                                                  int32_t* kept_index, int32_t* cu_seqlens, void* qc, void* kc,
                                                  void* vc, void* stream) {
  const int32_t T = S > V_full ? S - V_full : 1;
  const litevlm_status_t st =
      check_score_args(dtype, B, S, V_full, Hq, Hkv, D, T, q, k, v, softmax_scale, q_scale, k_scale, v_scale,
                       keep_ratio, scores, kept_index, cu_seqlens, qc, kc, vc);
  if (st != LITEVLM_OK) return st;
  if (score_workspace_layout(B, S, V_full, Hq, Hkv, T).total > LITEVLM_NOALLOC_SCRATCH_BYTES)
    return LITEVLM_ERR_WORKSPACE;
  void* ws = nullptr;
  const litevlm_status_t sc = device_scratch(&ws);
  if (sc != LITEVLM_OK) return sc;
  // the kernels need the scratch contents on entry to be nothing in particular
  // (sweep 1 clears the column sums itself), so no clearing is enqueued here
  return launch_score(dtype, B, S, V_full, Hq, Hkv, D, T, q, k, v, softmax_scale, q_scale, k_scale, token_keep,
                      keep_ratio, scores, kept_index, cu_seqlens, qc, kc, vc, ws, stream);
}

litevlm_status_t litevlm_token_score_topk_rows(int32_t dtype, int32_t B, int32_t S, int32_t V_full,
                                               int32_t Hq, int32_t Hkv, int32_t D, int32_t query_rows,
                                               const void* q, const void* k, const void* v,
                                               float softmax_scale, float q_scale, float k_scale,
                                               float v_scale, const uint8_t* token_keep, double keep_ratio,
                                               float* scores, int32_t* kept_index, int32_t* cu_seqlens,
                                               void* qc, void* kc, void* vc, void* workspace,
                                               size_t workspace_bytes, void* stream) {
  const litevlm_status_t st =
      check_score_args(dtype, B, S, V_full, Hq, Hkv, D, query_rows, q, k, v, softmax_scale, q_scale, k_scale,
                       v_scale, keep_ratio, scores, kept_index, cu_seqlens, qc, kc, vc);
  if (st != LITEVLM_OK) return st;
  if (workspace && !aligned(workspace, 16)) return LITEVLM_ERR_MISALIGNED;
  const size_t need = score_workspace_layout(B, S, V_full, Hq, Hkv, query_rows).total;
  if (!workspace || workspace_bytes < need) return LITEVLM_ERR_WORKSPACE;
  return launch_score(dtype, B, S, V_full, Hq, Hkv, D, query_rows, q, k, v, softmax_scale, q_scale, k_scale,
                      token_keep, keep_ratio, scores, kept_index, cu_seqlens, qc, kc, vc, workspace, stream);
}

litevlm_status_t litevlm_select_score_topk(int32_t dtype, int32_t B, int32_t S, int32_t V_full, int32_t Hq,
                                           int32_t Hkv, int32_t D, int32_t N, const int32_t* view_offsets_host,
                                           const float* view_logit, const float* view_lexical, float w_lexical,
                                           float threshold, const void* q, const void* k, const void* v,
                                           float softmax_scale, float q_scale, float k_scale, float v_scale,
                                           double keep_ratio, uint8_t* view_keep, uint8_t* token_keep,
                                           int32_t* n_visual_kept, float* scores, int32_t* kept_index,
                                           int32_t* cu_seqlens, void* qc, void* kc, void* vc, void* workspace,
                                           size_t workspace_bytes, void* stream) {
  const int32_t T = S > V_full ? S - V_full : 1;
  const litevlm_status_t st =
      check_score_args(dtype, B, S, V_full, Hq, Hkv, D, T, q, k, v, softmax_scale, q_scale, k_scale, v_scale,
                       keep_ratio, scores, kept_index, cu_seqlens, qc, kc, vc);
  if (st != LITEVLM_OK) return st;
  if (!view_offsets_host || !view_logit) return LITEVLM_ERR_NULL_POINTER;
  if (N < 1 || N > LITEVLM_MAX_VIEWS || view_offsets_host[0] != 0) return LITEVLM_ERR_BAD_SHAPE;
  if (N > kFusedViews) return LITEVLM_ERR_UNSUPPORTED;
  ViewSel vs{};
  for (int v = 0; v <= N; ++v) {
    vs.off[v] = view_offsets_host[v];
    if (v > 0 && vs.off[v] < vs.off[v - 1]) return LITEVLM_ERR_BAD_SHAPE;
  }
  if (vs.off[N] != V_full) return LITEVLM_ERR_BAD_SHAPE;  // the views tile the visual positions
  if (!(w_lexical >= 0.f && w_lexical <= 1.f) || !isfinite(threshold)) return LITEVLM_ERR_BAD_VALUE;
  if (!aligned(view_logit, 4) || (view_lexical && !aligned(view_lexical, 4)) ||
      (n_visual_kept && !aligned(n_visual_kept, 4)))
    return LITEVLM_ERR_MISALIGNED;
  if (workspace && !aligned(workspace, 16)) return LITEVLM_ERR_MISALIGNED;
  const size_t need = score_workspace_layout(B, S, V_full, Hq, Hkv, T).total;
  if (!workspace || workspace_bytes < need) return LITEVLM_ERR_WORKSPACE;
  vs.logit = view_logit;
  vs.lexical = view_lexical;
  vs.w = w_lexical;
  vs.tau = threshold;
  vs.N = N;
  return launch_score(dtype, B, S, V_full, Hq, Hkv, D, T, q, k, v, softmax_scale, q_scale, k_scale, nullptr,
                      keep_ratio, scores, kept_index, cu_seqlens, qc, kc, vc, workspace, stream, &vs, view_keep,
                      token_keep, n_visual_kept);
}

litevlm_status_t litevlm_token_score_topk(int32_t dtype, int32_t B, int32_t S, int32_t V_full,
                                          int32_t Hq, int32_t Hkv, int32_t D, const void* q,
                                          const void* k, const void* v, float softmax_scale,
                                          float q_scale, float k_scale, float v_scale,
                                          const uint8_t* token_keep, double keep_ratio,
                                          float* scores, int32_t* kept_index, int32_t* cu_seqlens,
                                          void* qc, void* kc, void* vc, void* workspace,
                                          size_t workspace_bytes, void* stream) {
  // every text token is a query row (S > V_full is checked by the callee)
  return litevlm_token_score_topk_rows(dtype, B, S, V_full, Hq, Hkv, D, S > V_full ? S - V_full : 1, q, k, v,
                                       softmax_scale, q_scale, k_scale, v_scale, token_keep, keep_ratio,
                                       scores, kept_index, cu_seqlens, qc, kc, vc, workspace, workspace_bytes,
                                       stream);
}

litevlm_status_t litevlm_prefill_attn(int32_t in_dtype, int32_t out_dtype, int32_t B, int32_t Hq,
                                      int32_t Hkv, int32_t D, const void* qc, const void* kc,
                                      const void* vc, const int32_t* cu_seqlens, int32_t max_seqlen,
                                      float softmax_scale, float q_scale, float k_scale,
                                      float v_scale, int32_t causal, void* o, void* stream) {
  if (!qc || !kc || !vc || !cu_seqlens || !o) return LITEVLM_ERR_NULL_POINTER;
  if (!valid_dtype(in_dtype) || (out_dtype != LITEVLM_F32 && out_dtype != LITEVLM_BF16))
    return LITEVLM_ERR_UNSUPPORTED;
  if (B < 1 || B > LITEVLM_MAX_BATCH || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 ||
      (D != 64 && D != 128) || max_seqlen < 0)
    return LITEVLM_ERR_BAD_SHAPE;
  if ((int64_t)B * max_seqlen > INT32_MAX / 2) return LITEVLM_ERR_BAD_SHAPE;
  if (causal != 0 && causal != 1) return LITEVLM_ERR_BAD_VALUE;
  if (!finite_pos(softmax_scale) || !finite_pos(q_scale) || !finite_pos(k_scale) ||
      !finite_pos(v_scale))
    return LITEVLM_ERR_BAD_VALUE;
  if (in_dtype != LITEVLM_FP8_E4M3 && (q_scale != 1.f || k_scale != 1.f || v_scale != 1.f))
    return LITEVLM_ERR_BAD_VALUE;
  if (!aligned(qc, 16) || !aligned(kc, 16) || !aligned(vc, 16) || !aligned(o, 16) ||
      !aligned(cu_seqlens, 4))
    return LITEVLM_ERR_MISALIGNED;

  AttnArgs a;
  a.in_dtype = in_dtype;
  a.out_dtype = out_dtype;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.D = D;
  a.max_seqlen = max_seqlen;
  a.causal = causal;
  a.q = qc;
  a.k = kc;
  a.v = vc;
  a.cu_seqlens = cu_seqlens;
  a.logit_scale_log2 = (float)((double)softmax_scale * q_scale * k_scale * 1.4426950408889634);
  a.out_scale = v_scale;
  a.o = o;
  return hip_status(launch_prefill_attn(a, static_cast<hipStream_t>(stream)));
}

size_t litevlm_decode_attn_workspace(int32_t in_dtype, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
                                     int32_t max_seqlen) {
  if (check_decode_shape(in_dtype, B, Hq, Hkv, D, max_seqlen) != LITEVLM_OK) return 0;
  return decode_layout(in_dtype, B, Hq, Hkv, D, max_seqlen).total;
}

litevlm_status_t litevlm_decode_attn(int32_t in_dtype, int32_t out_dtype, int32_t B, int32_t Hq,
                                     int32_t Hkv, int32_t D, const void* q1, const void* k1,
                                     const void* v1, const void* kc, const void* vc,
                                     const int32_t* cu_seqlens, int32_t max_seqlen,
                                     float softmax_scale, float q_scale, float k_scale,
                                     float v_scale, void* o, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  if (!q1 || !k1 || !v1 || !kc || !vc || !cu_seqlens || !o) return LITEVLM_ERR_NULL_POINTER;
  if (!valid_dtype(in_dtype) || (out_dtype != LITEVLM_F32 && out_dtype != LITEVLM_BF16))
    return LITEVLM_ERR_UNSUPPORTED;
  const litevlm_status_t sh = check_decode_shape(in_dtype, B, Hq, Hkv, D, max_seqlen);
  if (sh != LITEVLM_OK) return sh;
  if (!finite_pos(softmax_scale) || !finite_pos(q_scale) || !finite_pos(k_scale) ||
      !finite_pos(v_scale))
    return LITEVLM_ERR_BAD_VALUE;
  if (in_dtype != LITEVLM_FP8_E4M3 && (q_scale != 1.f || k_scale != 1.f || v_scale != 1.f))
    return LITEVLM_ERR_BAD_VALUE;
  const void* big[] = {q1, k1, v1, kc, vc, o, workspace};
  for (const void* p : big)
    if (p && !aligned(p, 16)) return LITEVLM_ERR_MISALIGNED;
  if (!aligned(cu_seqlens, 4)) return LITEVLM_ERR_MISALIGNED;
  const size_t need = decode_layout(in_dtype, B, Hq, Hkv, D, max_seqlen).total;
  if (!workspace || workspace_bytes < need) return LITEVLM_ERR_WORKSPACE;

  DecodeArgs a;
  a.in_dtype = in_dtype;
  a.out_dtype = out_dtype;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.D = D;
  a.max_seqlen = max_seqlen;
  a.q1 = q1;
  a.k1 = k1;
  a.v1 = v1;
  a.kc = kc;
  a.vc = vc;
  a.cu_seqlens = cu_seqlens;
  a.logit_scale_log2 = (float)((double)softmax_scale * q_scale * k_scale * 1.4426950408889634);
  a.out_scale = v_scale;
  a.o = o;
  a.workspace = workspace;
  return hip_status(launch_decode_attn(a, static_cast<hipStream_t>(stream)));
}

litevlm_status_t litevlm_gather_hidden(int32_t B, int32_t S, int32_t row_bytes, const void* hidden,
                                       const int32_t* kept_index, const int32_t* cu_seqlens, void* out,
                                       void* stream) {
  if (!hidden || !kept_index || !cu_seqlens || !out) return LITEVLM_ERR_NULL_POINTER;
  if (B < 1 || B > LITEVLM_MAX_BATCH || S < 1 || (int64_t)B * S > INT32_MAX / 2) return LITEVLM_ERR_BAD_SHAPE;
  if (row_bytes < 16 || row_bytes % 16 != 0 || row_bytes > 48 * 256 * 16) return LITEVLM_ERR_BAD_SHAPE;
  if (!aligned(hidden, 16) || !aligned(out, 16) || !aligned(kept_index, 4) || !aligned(cu_seqlens, 4))
    return LITEVLM_ERR_MISALIGNED;
  return hip_status(launch_gather_hidden(B, S, row_bytes, hidden, kept_index, cu_seqlens, out,
                                         static_cast<hipStream_t>(stream)));
}

// Patch Selection Module sizes: d 256 or 512 (the LayerNorm and cross kernels
// hold a row in registers / LDS), head dim d / n_heads of 64 or 128 (the
// prefill attention kernel), d_ff a multiple of 64.
static litevlm_status_t check_psm_shape(int32_t B, int32_t T, int32_t d, int32_t n_heads, int32_t d_ff,
                                 int32_t n_views, int32_t n_layers) {
  if (B < 1 || B > LITEVLM_MAX_BATCH || T < 1 || T > 8192 || n_views < 1 || n_views > LITEVLM_MAX_VIEWS ||
      n_layers < 1 || n_layers > 64)
    return LITEVLM_ERR_BAD_SHAPE;
  if ((d != 256 && d != 512) || n_heads < 1 || d % n_heads != 0) return LITEVLM_ERR_BAD_SHAPE;
  const int dh = d / n_heads;
  if (dh != 64 && dh != 128) return LITEVLM_ERR_UNSUPPORTED;
  if (d_ff < 64 || d_ff % 64 != 0 || d_ff > 16384) return LITEVLM_ERR_BAD_SHAPE;
  return LITEVLM_OK;
}

size_t litevlm_psm_param_count(int32_t d, int32_t d_ff, int32_t n_views, int32_t n_layers) {
  if (d < 1 || d_ff < 1 || n_views < 1 || n_layers < 1) return 0;
  return psm_layout(1, 1, d, d_ff, n_views, n_layers).params;
}

size_t litevlm_psm_workspace(int32_t B, int32_t T, int32_t d, int32_t n_heads, int32_t d_ff) {
  if (check_psm_shape(B, T, d, n_heads, d_ff, 1, 1) != LITEVLM_OK) return 0;
  return psm_layout(B, T, d, d_ff, 1, 1).total;
}

litevlm_status_t litevlm_psm_forward(int32_t B, int32_t T, int32_t d, int32_t n_heads, int32_t d_ff,
                                     int32_t n_views, int32_t n_layers, const float* emb, const float* params,
                                     size_t n_params, float* view_logit, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  if (!emb || !params || !view_logit) return LITEVLM_ERR_NULL_POINTER;
  const litevlm_status_t sh = check_psm_shape(B, T, d, n_heads, d_ff, n_views, n_layers);
  if (sh != LITEVLM_OK) return sh;
  const PsmLayout L = psm_layout(B, T, d, d_ff, n_views, n_layers);
  if (n_params != L.params) return LITEVLM_ERR_BAD_SHAPE;
  if (!aligned(emb, 16) || !aligned(params, 16) || !aligned(view_logit, 4) || (workspace && !aligned(workspace, 16)))
    return LITEVLM_ERR_MISALIGNED;
  if (!workspace || workspace_bytes < L.total) return LITEVLM_ERR_WORKSPACE;
  PsmArgs a;
  a.B = B;
  a.T = T;
  a.d = d;
  a.n_heads = n_heads;
  a.d_ff = d_ff;
  a.n_views = n_views;
  a.n_layers = n_layers;
  a.emb = emb;
  a.params = params;
  a.view_logit = view_logit;
  a.workspace = workspace;
  return hip_status(launch_psm_forward(a, static_cast<hipStream_t>(stream)));
}

litevlm_status_t litevlm_tsm_fold_gain(int32_t rows, int32_t cols, const void* w, const float* gamma,
                                       void* w_out, void* stream) {
  if (!w || !gamma || !w_out) return LITEVLM_ERR_NULL_POINTER;
  if (rows < 1 || cols < 1 || (int64_t)rows * cols > ((int64_t)1 << 40)) return LITEVLM_ERR_BAD_SHAPE;
  if (!aligned(w, 2) || !aligned(w_out, 2) || !aligned(gamma, 4)) return LITEVLM_ERR_MISALIGNED;
  return hip_status(launch_tsm_fold_gain(w, gamma, w_out, rows, cols, static_cast<hipStream_t>(stream)));
}

litevlm_status_t litevlm_tsm_qk(int32_t B, int32_t S, int32_t V_full, int32_t Dm, int32_t Hq, int32_t Hkv,
                                int32_t D, const void* hidden, const uint8_t* token_keep, const void* w_q,
                                const void* w_k, float eps, float rope_theta, void* q, void* k,
                                void* stream) {
  if (!hidden || !w_q || !w_k || !q || !k) return LITEVLM_ERR_NULL_POINTER;
  if (B < 1 || B > LITEVLM_MAX_BATCH || V_full < 0 || S <= V_full || Hq < 1 || Hkv < 1 ||
      Hq > LITEVLM_MAX_HEADS || Hq % Hkv != 0 || (D != 64 && D != 128))
    return LITEVLM_ERR_BAD_SHAPE;
  if (Dm < 64 || Dm % 64 != 0 || Dm > 65536) return LITEVLM_ERR_BAD_SHAPE;
  // a workgroup covers 128 output features: whole heads, rotary partners together
  if ((Hq * D) % 128 != 0 || (Hkv * D) % 128 != 0) return LITEVLM_ERR_UNSUPPORTED;
  if ((int64_t)B * S > INT32_MAX / 2 || (int64_t)B * S * Dm > ((int64_t)1 << 40)) return LITEVLM_ERR_BAD_SHAPE;
  if (!(eps > 0.f) || !isfinite(eps) || !(rope_theta > 1.f) || !isfinite(rope_theta))
    return LITEVLM_ERR_BAD_VALUE;
  if (!aligned(hidden, 16) || !aligned(w_q, 16) || !aligned(w_k, 16) || !aligned(q, 16) || !aligned(k, 16))
    return LITEVLM_ERR_MISALIGNED;
  TsmArgs a;
  a.B = B;
  a.S = S;
  a.V_full = V_full;
  a.Dm = Dm;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.D = D;
  a.hidden = hidden;
  a.token_keep = token_keep;
  a.w_q = w_q;
  a.w_k = w_k;
  a.eps = eps;
  a.rope_theta = rope_theta;
  a.q = q;
  a.k = k;
  return hip_status(launch_tsm_qk(a, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
