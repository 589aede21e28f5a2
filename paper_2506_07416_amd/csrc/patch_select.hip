// View selection and per-view patch masking (Design section, Patch Selection
// Module paragraph): fused view score, strict threshold, best-view fallback,
// token mask over the view-major visual layout plus the always-kept text.
#include "common.hpp"
#include "launch.hpp"
#include "viewsel.hpp"

namespace litevlm {

__global__ void __launch_bounds__(256)
patch_select_kernel(int N, int S, ViewOffsets vo, const float* __restrict__ logit,
                    const float* __restrict__ lexical, float w, float tau,
                    uint8_t* __restrict__ view_keep, uint8_t* __restrict__ token_keep,
                    int32_t* __restrict__ n_visual_kept) {
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  __shared__ int off_s[LITEVLM_MAX_VIEWS + 1];
  // the view offsets go to LDS once, so that no loop below waits on a
  // dependent load of them
  if (tid <= N) off_s[tid] = vo.off[tid];
  // every wave takes the decision, one view per lane (N <= 64), with the
  // function the scoring kernels use when they select the views themselves
  const ViewIn in = view_load(logit, lexical, N, b, lane);
  const uint64_t mask = view_keep_mask<LITEVLM_MAX_VIEWS>(in, lexical != nullptr, w, tau, N, lane);
  __syncthreads();
  if (tid < N) view_keep[b * N + tid] = (uint8_t)((mask >> tid) & 1u);
  if (tid == 0 && n_visual_kept) {
    int nvis = 0;
    for (int v = 0; v < N; ++v)
      if ((mask >> v) & 1u) nvis += off_s[v + 1] - off_s[v];
    n_visual_kept[b] = nvis;
  }
  // token mask: visual token p takes its view's flag (views are contiguous
  // and view-major), text tokens are 1; 16 bytes per thread and store
  uint8_t* row = token_keep + (size_t)b * S;
  const bool vec = (reinterpret_cast<uintptr_t>(row) & 15) == 0;
  for (int p0 = 16 * tid; p0 < S; p0 += 16 * 256) {
    // view of p0: the number of views ending at or before it (N independent
    // LDS reads rather than a dependent walk); v == N for text tokens
    int v = 0;
    for (int u = 0; u < N; ++u) v += p0 >= off_s[u + 1] ? 1 : 0;
    const int n = min(16, S - p0);
    uint32_t wd[4];
    if (p0 + n <= (v < N ? off_s[v + 1] : S)) {
      // the whole chunk lies in one view (or in the text)
      const uint32_t k = v < N ? (uint32_t)((mask >> v) & 1u) : 1u;
      wd[0] = wd[1] = wd[2] = wd[3] = k * 0x01010101u;
    } else {
      wd[0] = wd[1] = wd[2] = wd[3] = 0u;
      for (int j = 0; j < n; ++j) {
        const int p = p0 + j;
        while (v < N && p >= off_s[v + 1]) ++v;
        const uint32_t k = v < N ? (uint32_t)((mask >> v) & 1u) : 1u;
        wd[j >> 2] |= k << (8 * (j & 3));
      }
    }
    if (vec && n == 16) {
      *reinterpret_cast<uint4*>(row + p0) = make_uint4(wd[0], wd[1], wd[2], wd[3]);
    } else {
      for (int j = 0; j < n; ++j) row[p0 + j] = (uint8_t)(wd[j >> 2] >> (8 * (j & 3)));
    }
  }
}

hipError_t launch_patch_select(int B, int N, int S, const ViewOffsets& vo, const float* logit,
                               const float* lexical, float w, float tau, uint8_t* view_keep,
                               uint8_t* token_keep, int32_t* n_visual_kept, hipStream_t stream) {
  hipLaunchKernelGGL(patch_select_kernel, dim3(B), dim3(256), 0, stream, N, S, vo, logit, lexical,
                     w, tau, view_keep, token_keep, n_visual_kept);
  return hipGetLastError();
}

}  // namespace litevlm
