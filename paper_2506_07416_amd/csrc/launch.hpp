// Host-side launch entry points of the device kernels, called by api.hip after
// argument validation. Each returns the HIP error of its launches.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/litevlm.h"
#include "viewsel.hpp"

namespace litevlm {

struct ViewOffsets {
  int32_t off[LITEVLM_MAX_VIEWS + 1];
};

hipError_t launch_patch_select(int B, int N, int S, const ViewOffsets& vo, const float* logit,
                               const float* lexical, float w, float tau, uint8_t* view_keep,
                               uint8_t* token_keep, int32_t* n_visual_kept, hipStream_t stream);

// Workspace of the scoring step, carved from one caller buffer:
//   rowpart  float2 [B][Hkv][ns1][R]  per-key-split (max, sum) of each text row
//   acc      u64    [B][V_full]       fixed-point column sums of sweep 2
// with R = (Hq/Hkv)*n_query rows per KV group (the last n_query text tokens
// are the query rows); ns1 (key splits of sweep 1) is a function of the shape.
struct ScoreWorkspace {
  size_t rowpart_off, acc_off, total;
};
ScoreWorkspace score_workspace_layout(int B, int S, int V_full, int Hq, int Hkv, int n_query);

struct ScoreArgs {
  int dtype, B, S, V_full, Hq, Hkv, D;
  int query_rows;  // the last query_rows text tokens are the query rows (1..T)
  const void* q;
  const void* k;
  const void* v;
  float logit_scale_log2;  // softmax_scale*q_scale*k_scale*log2(e)
  const uint8_t* token_keep;
  double keep_ratio;
  float* scores;
  int32_t* kept_index;
  int32_t* cu_seqlens;
  void* qc;
  void* kc;
  void* vc;
  void* workspace;
  // in-call patch selection (vs.N > 0, token_keep NULL): the keep flags come
  // from the view scores, and the selection's outputs are written (each may be NULL)
  ViewSel vs{};
  uint8_t* view_keep = nullptr;
  uint8_t* token_keep_out = nullptr;
  int32_t* n_visual_kept = nullptr;
};
hipError_t launch_token_score_topk(const ScoreArgs& a, hipStream_t stream);

// Row gather behind the compaction: rows kept_index[r] of each sample of q, k,
// v (qvec / kvvec 16-byte pieces per row) into packed qc, kc, vc (each may be
// NULL, kvvec may be 0).
void launch_gather(int B, int S, const int32_t* kept_index, const int32_t* cu_seqlens, const void* q,
                   const void* k, const void* v, void* qc, void* kc, void* vc, int qvec, int kvvec,
                   hipStream_t stream);
hipError_t launch_gather_hidden(int B, int S, int row_bytes, const void* hidden, const int32_t* kept_index,
                                const int32_t* cu_seqlens, void* out, hipStream_t stream);

struct AttnArgs {
  int in_dtype, out_dtype, B, Hq, Hkv, D, max_seqlen, causal;
  const void* q;
  const void* k;
  const void* v;
  const int32_t* cu_seqlens;
  float logit_scale_log2;  // softmax_scale*q_scale*k_scale*log2(e)
  float out_scale;         // v_scale
  void* o;
};
hipError_t launch_prefill_attn(const AttnArgs& a, hipStream_t stream);

// Workspace of the decode step: per (sample, query head, key split) the
// unnormalised output float [D] and the split's (max, sum) float2. The split
// length and count follow from the shape and the host bound max_seqlen.
struct DecodeLayout {
  int split_len, nsplit;
  size_t part_o_off, part_ml_off, total;
};
DecodeLayout decode_layout(int in_dtype, int B, int Hq, int Hkv, int D, int max_seqlen);

struct DecodeArgs {
  int in_dtype, out_dtype, B, Hq, Hkv, D, max_seqlen;
  const void* q1;
  const void* k1;
  const void* v1;
  const void* kc;
  const void* vc;
  const int32_t* cu_seqlens;
  float logit_scale_log2;  // softmax_scale*q_scale*k_scale*log2(e)
  float out_scale;         // v_scale
  void* o;
  void* workspace;
};
hipError_t launch_decode_attn(const DecodeArgs& a, hipStream_t stream);

struct TsmArgs {
  int B, S, V_full, Dm, Hq, Hkv, D;
  const void* hidden;
  const uint8_t* token_keep;
  const void* w_q;
  const void* w_k;
  float eps, rope_theta;
  void* q;
  void* k;
};
hipError_t launch_tsm_qk(const TsmArgs& a, hipStream_t stream);

// Patch Selection Module: parameter count and workspace carving.
struct PsmLayout {
  size_t layer_params, params;
  size_t h_off, q_off, k_off, v_off, att_off, ff_off, cu_off, total;
};
PsmLayout psm_layout(int B, int T, int d, int d_ff, int n_views, int n_layers);

struct PsmArgs {
  int B, T, d, n_heads, d_ff, n_views, n_layers;
  const float* emb;
  const float* params;
  float* view_logit;
  void* workspace;
};
hipError_t launch_psm_forward(const PsmArgs& a, hipStream_t stream);
hipError_t launch_tsm_fold_gain(const void* w, const float* gamma, void* w_out, int rows, int cols,
                                hipStream_t stream);

}  // namespace litevlm
