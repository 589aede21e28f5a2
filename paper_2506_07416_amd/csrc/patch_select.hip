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
  __shared__ float s_s[LITEVLM_MAX_VIEWS];
  // One thread per view, written as the definition reads: no FMA
  // contraction and IEEE division, so the decision matches an fp32 evaluation.
  if (threadIdx.x < N) {
    const int v = threadIdx.x;
    const float x = logit[b * N + v];
    const float sig = __fdiv_rn(1.0f, __fadd_rn(1.0f, expf(-x)));
    const float lex = lexical ? lexical[b * N + v] : 0.0f;
    const float s = __fadd_rn(__fmul_rn(w, lex), __fmul_rn(__fsub_rn(1.0f, w), sig));
    s_s[v] = s;
    keep_s[v] = (uint8_t)(s > tau);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    // if no view passes, keep the best one (lowest index among equal scores)
    int any = 0, best_v = 0;
    for (int v = 0; v < N; ++v) {
      any |= keep_s[v];
      if (s_s[v] > s_s[best_v]) best_v = v;
    }
    if (!any) keep_s[best_v] = 1;
  }
  __syncthreads();
  if (threadIdx.x < N) view_keep[b * N + threadIdx.x] = keep_s[threadIdx.x];
  if (threadIdx.x == 0 && n_visual_kept) {
    int nvis = 0;
    for (int v = 0; v < N; ++v)
      if (keep_s[v]) nvis += vo.off[v + 1] - vo.off[v];
    n_visual_kept[b] = nvis;
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
