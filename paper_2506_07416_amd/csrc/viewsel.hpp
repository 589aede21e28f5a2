// View selection of the Patch Selection Module (Design section, Patch Selection
// Module paragraph), as device functions shared by the patch-select kernel and
// the scoring kernels that take the selection themselves.
//
// View v of a sample scores s_v = w * lexical_v + (1 - w) * sigmoid(logit_v),
// evaluated in fp32 with IEEE operations and no contraction; it is kept when
// s_v > tau. When no view passes, the view with the highest score is kept (the
// lowest index among equal scores). The views tile the visual positions
// off[0] = 0 .. off[N] in order; later positions are text and always kept.
#pragma once

#include "../../include/litevlm.h"
#include "common.hpp"

namespace litevlm {

// Most views the in-call selection handles (the per-key view lookup is an
// unrolled comparison against the offsets).
constexpr int kFusedViews = LITEVLM_MAX_FUSED_VIEWS;

// The selection inputs of one call, passed by value to the kernels.
struct ViewSel {
  const float* logit;    // [B, N]
  const float* lexical;  // [B, N] or NULL (lexical scores 0)
  float w, tau;
  int N;                 // 1..kFusedViews (0: no in-call selection)
  int off[kFusedViews + 1];
};

// The raw inputs of view min(lane, N-1) of sample b, one view per lane: both
// loads are unconditional (the lexical one reads the logit when there is no
// lexical score), so issuing them waits on nothing.
struct ViewIn {
  float x, lex;
};
__device__ __forceinline__ ViewIn view_load(const float* logit, const float* lexical, int N, int b, int lane) {
  const int v = b * N + min(lane, N - 1);
  ViewIn in;
  in.x = logit[v];
  in.lex = (lexical ? lexical : logit)[v];
  return in;
}

// Score of one view from its inputs.
__device__ __forceinline__ float view_score(float x, float lex, float w) {
  const float sig = __fdiv_rn(1.0f, __fadd_rn(1.0f, expf(-x)));
  return __fadd_rn(__fmul_rn(w, lex), __fmul_rn(__fsub_rn(1.0f, w), sig));
}

// Kept views of a sample as a bit mask (bit v = view v), from the inputs one
// wave loaded with view_load; every lane of the wave returns the same mask.
// MAXN bounds N. Branch-free, so that no wait for the loads in flight is
// placed before it: the fallback (no view passes: the first view whose score
// no later view exceeds, a strict scan in view order as the definition reads)
// is evaluated always and selected at the end.
template <int MAXN>
__device__ __forceinline__ uint64_t view_keep_mask(const ViewIn& in, bool has_lexical, float w, float tau, int N,
                                                   int lane) {
  const float s = view_score(in.x, has_lexical ? in.lex : 0.0f, w);
  const uint64_t pass = __ballot(lane < N && s > tau);
  float best = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(s), 0));
  int bv = 0;
#pragma unroll
  for (int u = 1; u < MAXN; ++u) {
    const float su = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(s), u));
    const bool better = u < N && su > best;
    best = better ? su : best;
    bv = better ? u : bv;
  }
  return pass ? pass : (1ull << bv);
}

// Keep flag of position j of a sample under a mask of its (at most
// kFusedViews) views: the view holding j, or 1 past the last view.
__device__ __forceinline__ uint32_t view_token_flag(const ViewSel& vs, uint32_t mask, int j) {
  int v = 0;
#pragma unroll
  for (int u = 1; u <= kFusedViews; ++u) v += (u <= vs.N && j >= vs.off[u]) ? 1 : 0;
  return v < vs.N ? (mask >> v) & 1u : 1u;
}

}  // namespace litevlm
