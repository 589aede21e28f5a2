// View selection and per-view patch masking (Design section, Patch Selection
// Module paragraph): fused view score, strict threshold, best-view fallback,
// token mask over the view-major visual layout plus the always-kept text.
#include "common.hpp"
#include "launch.hpp"

namespace litevlm {

__global__ void __launch_bounds__(256)
patch_select_kernel(int N, int S, ViewOffsets vo, const float* __restrict__ logit,
                    const float* __restrict__ lexical, float w, float tau,
                    uint8_t* __restrict__ view_keep, uint8_t* __restrict__ token_keep,
                    int32_t* __restrict__ n_visual_kept) {
  const int b = blockIdx.x;
  __shared__ uint8_t keep_s[LITEVLM_MAX_VIEWS];
  if (threadIdx.x == 0) {
    // N <= 64 views: one thread, written as the definition reads. No FMA
    // contraction, IEEE division, so the decision matches an fp32 evaluation.
    float best = 0.f;
    int best_v = 0, any = 0;
    for (int v = 0; v < N; ++v) {
      const float x = logit[b * N + v];
      const float sig = __fdiv_rn(1.0f, __fadd_rn(1.0f, expf(-x)));
      const float lex = lexical ? lexical[b * N + v] : 0.0f;
      const float s = __fadd_rn(__fmul_rn(w, lex), __fmul_rn(__fsub_rn(1.0f, w), sig));
      const int k = s > tau;
      keep_s[v] = (uint8_t)k;
      any |= k;
      if (v == 0 || s > best) { best = s; best_v = v; }
    }
    if (!any) keep_s[best_v] = 1;
    int nvis = 0;
    for (int v = 0; v < N; ++v) {
      view_keep[b * N + v] = keep_s[v];
      if (keep_s[v]) nvis += vo.off[v + 1] - vo.off[v];
    }
    if (n_visual_kept) n_visual_kept[b] = nvis;
  }
  __syncthreads();
  const int V_full = vo.off[N];
  uint8_t* row = token_keep + (size_t)b * S;
  for (int v = 0; v < N; ++v) {
    const uint8_t k = keep_s[v];
    for (int p = vo.off[v] + threadIdx.x; p < vo.off[v + 1]; p += blockDim.x) row[p] = k;
  }
  for (int p = V_full + threadIdx.x; p < S; p += blockDim.x) row[p] = 1;
}

hipError_t launch_patch_select(int B, int N, int S, const ViewOffsets& vo, const float* logit,
                               const float* lexical, float w, float tau, uint8_t* view_keep,
                               uint8_t* token_keep, int32_t* n_visual_kept, hipStream_t stream) {
  hipLaunchKernelGGL(patch_select_kernel, dim3(B), dim3(256), 0, stream, N, S, vo, logit, lexical,
                     w, tau, view_keep, token_keep, n_visual_kept);
  return hipGetLastError();
}

}  // namespace litevlm
