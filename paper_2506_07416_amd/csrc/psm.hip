// Patch Selection Module forward pass: a small pre-norm transformer encoder
// over the text query's token embeddings, then a single-headed cross-attention
// of N learnable latent queries (one per camera view) over the encoded tokens
// and one linear head per view, giving the view logits that the patch
// selection fuses with its lexical scores.
//
// The module is tiny (d = 256, 4 layers, 128 tokens at the benchmark shape),
// so every step is latency-bound: the kernels favour few dependent global
// round trips over peak rates.
//   - psm_ln_kernel: LayerNorm, one wave per row (fp32 math, bf16 out); the
//     first call also copies the embeddings into the fp32 residual stream and
//     writes the per-sample row offsets the attention call reads.
//   - psm_gemm_kernel: bf16 MFMA (v_mfma_f32_32x32x16_bf16) on x [M, K] times
//     W^T, W [N, K] fp32 from the parameter vector (rounded to bf16 as it is
//     loaded), with the bias and either a bf16 output (split into equal column
//     ranges, for Q/K/V), GELU, or an add into the fp32 residual stream. A wave
//     owns a 32 x 32 output block and reads its operands straight from global
//     memory (the weights are re-read from L2 by the few row blocks).
//   - self-attention: the library's prefill attention kernel, non-causal.
//   - psm_cross_kernel: per (view, sample): the latent's query, its softmax over
//     the encoded tokens, the attended value and the view's head.
#include "common.hpp"
#include "launch.hpp"

namespace litevlm {
namespace {

typedef uint32_t psm_u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int psm_acc_row(int r, int hl) { return 8 * (r >> 2) + 4 * hl + (r & 3); }

__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.f + erff(x * 0.7071067811865476f)); }

// LayerNorm of one row per wave: y = (x - mean) / sqrt(var + 1e-5) * g + b.
template <int EPL>
__global__ __launch_bounds__(256) void psm_ln_kernel(const float* __restrict__ init, float* __restrict__ h,
                                                     const float* __restrict__ g, const float* __restrict__ bta,
                                                     uint16_t* __restrict__ y, int M, int B, int T,
                                                     int32_t* __restrict__ cu) {
  constexpr int d = EPL * kWave;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (cu && blockIdx.x == 0)
    for (int t = threadIdx.x; t <= B; t += 256) cu[t] = t * T;
  if (row >= M) return;
  float x[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    const size_t i = (size_t)row * d + lane + kWave * e;
    x[e] = init ? init[i] : h[i];
    if (init) h[i] = x[e];
  }
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < EPL; ++e) s += x[e];
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) s += __shfl_xor(s, m, kWave);
  const float mu = s / d;
  float v = 0.f;
#pragma unroll
  for (int e = 0; e < EPL; ++e) v = fmaf(x[e] - mu, x[e] - mu, v);
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) v += __shfl_xor(v, m, kWave);
  const float r = 1.f / sqrtf(v / d + 1e-5f);
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    const int c = lane + kWave * e;
    y[(size_t)row * d + c] = f32_to_bf16_bits((x[e] - mu) * r * g[c] + bta[c]);
  }
}

enum { kOutBf16 = 0, kOutGelu = 1, kOutResid = 2 };

// out = x W^T + bias over a 64 x 64 tile per workgroup (2 x 2 waves of 32 x 32).
// kOutBf16: columns split into nsplit equal ranges, range j to out[j] [M, N/nsplit];
// kOutGelu: bf16 gelu(.) to out[0] [M, N]; kOutResid: h [M, N] += (.).
template <int MODE>
__global__ __launch_bounds__(256) void psm_gemm_kernel(const uint16_t* __restrict__ x, const float* __restrict__ W,
                                                       const float* __restrict__ bias, int M, int N, int K,
                                                       uint16_t* out0, uint16_t* out1, uint16_t* out2, int nsplit,
                                                       float* __restrict__ h) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int l32 = lane & 31, hl = lane >> 5;
  const int m0 = blockIdx.x * 64 + 32 * (w & 1), n0 = blockIdx.y * 64 + 32 * (w >> 1);
  const int arow = min(m0 + l32, M - 1);
  const uint16_t* ap = x + (size_t)arow * K + 8 * hl;
  const float* bp = W + (size_t)(n0 + l32) * K + 8 * hl;
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
  // Chunks of CH k16 steps: every load of a chunk is issued before its MFMAs,
  // so a chunk costs one memory round trip instead of CH.
  constexpr int CH = 8;
  int k = 0;
  for (; k + 16 * CH <= K; k += 16 * CH) {
    psm_u32x4 av[CH];
    float4 bv0[CH], bv1[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      av[c] = *reinterpret_cast<const psm_u32x4*>(ap + k + 16 * c);
      bv0[c] = *reinterpret_cast<const float4*>(bp + k + 16 * c);
      bv1[c] = *reinterpret_cast<const float4*>(bp + k + 16 * c + 4);
    }
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const float bv[8] = {bv0[c].x, bv0[c].y, bv0[c].z, bv0[c].w, bv1[c].x, bv1[c].y, bv1[c].z, bv1[c].w};
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, av[c]), pack_bf16x8(bv), acc, 0, 0, 0);
    }
  }
  for (; k < K; k += 16) {
    const bf16x8 a = __builtin_bit_cast(bf16x8, *reinterpret_cast<const psm_u32x4*>(ap + k));
    const float4 b0 = *reinterpret_cast<const float4*>(bp + k);
    const float4 b1 = *reinterpret_cast<const float4*>(bp + k + 4);
    const float bv[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pack_bf16x8(bv), acc, 0, 0, 0);
  }
  const int col = n0 + l32;
  const float bc = bias[col];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int row = m0 + psm_acc_row(r, hl);
    if (row >= M) continue;
    const float val = acc[r] + bc;
    if constexpr (MODE == kOutResid) {
      h[(size_t)row * N + col] += val;
    } else if constexpr (MODE == kOutGelu) {
      out0[(size_t)row * N + col] = f32_to_bf16_bits(gelu_erf(val));
    } else {
      const int wsplit = N / nsplit, j = col / wsplit;
      uint16_t* o = j == 0 ? out0 : (j == 1 ? out1 : out2);
      o[(size_t)row * wsplit + (col - j * wsplit)] = f32_to_bf16_bits(val);
    }
  }
}

// View logit of (view blockIdx.x, sample blockIdx.y): q = latent W_cq^T + b_cq,
// p = softmax_t(q . k_t / sqrt(d)), z = sum_t p_t v_t, logit = w_head . z + b_head.
template <int EPT>
__global__ __launch_bounds__(256) void psm_cross_kernel(const uint16_t* __restrict__ kc,
                                                        const uint16_t* __restrict__ vc,
                                                        const float* __restrict__ latents,
                                                        const float* __restrict__ w_cq, const float* __restrict__ b_cq,
                                                        const float* __restrict__ w_head,
                                                        const float* __restrict__ b_head, float* __restrict__ logit,
                                                        int T, int n_views) {
  constexpr int d = EPT * 256;
  const int v = blockIdx.x, b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  __shared__ float q[d];
  __shared__ float red[8];
  extern __shared__ float p[];  // [T]
  // query of the latent: thread j computes elements j, j + 256, ...
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int j = tid + 256 * e;
    float s = b_cq[j];
    const float* wr = w_cq + (size_t)j * d;
    const float* lr = latents + (size_t)v * d;
#pragma unroll 16
    for (int i = 0; i < d; ++i) s = fmaf(lr[i], wr[i], s);
    q[j] = s;
  }
  __syncthreads();
  const float scale = 1.f / sqrtf((float)d);
  float mx = -INFINITY;
  for (int t = tid; t < T; t += 256) {
    const uint16_t* kr = kc + ((size_t)b * T + t) * d;
    float s = 0.f;
#pragma unroll 16
    for (int i = 0; i < d; ++i) s = fmaf(q[i], bf16_bits_to_f32(kr[i]), s);
    s *= scale;
    p[t] = s;
    mx = fmaxf(mx, s);
  }
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) mx = fmaxf(mx, __shfl_xor(mx, m, kWave));
  if (lane == 0) red[w] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  float sum = 0.f;
  for (int t = tid; t < T; t += 256) {
    const float e = __expf(p[t] - mx);
    p[t] = e;
    sum += e;
  }
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) sum += __shfl_xor(sum, m, kWave);
  __syncthreads();
  if (lane == 0) red[4 + w] = sum;
  __syncthreads();
  const float inv = 1.f / (((red[4] + red[5]) + red[6]) + red[7]);
  // z and its dot with the head weights
  float dotp = 0.f;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int j = tid + 256 * e;
    float z = 0.f;
    for (int t = 0; t < T; ++t) z = fmaf(p[t], bf16_bits_to_f32(vc[((size_t)b * T + t) * d + j]), z);
    dotp = fmaf(z * inv, w_head[(size_t)v * d + j], dotp);
  }
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) dotp += __shfl_xor(dotp, m, kWave);
  __syncthreads();
  if (lane == 0) red[w] = dotp;
  __syncthreads();
  if (tid == 0) logit[(size_t)b * n_views + v] = ((red[0] + red[1]) + red[2]) + red[3] + b_head[v];
}

template <int EPL>
void ln(const float* init, float* h, const float* g, const float* bt, uint16_t* y, int M, int B, int T, int32_t* cu,
        hipStream_t s) {
  hipLaunchKernelGGL((psm_ln_kernel<EPL>), dim3((M + 3) / 4), dim3(256), 0, s, init, h, g, bt, y, M, B, T, cu);
}

template <int MODE>
void gemm(const uint16_t* x, const float* W, const float* bias, int M, int N, int K, uint16_t* o0, uint16_t* o1,
          uint16_t* o2, int nsplit, float* h, hipStream_t s) {
  hipLaunchKernelGGL((psm_gemm_kernel<MODE>), dim3((M + 63) / 64, N / 64), dim3(256), 0, s, x, W, bias, M, N, K, o0,
                     o1, o2, nsplit, h);
}

template <int EPL>
hipError_t run(const PsmArgs& a, hipStream_t s) {
  const PsmLayout L = psm_layout(a.B, a.T, a.d, a.d_ff, a.n_views, a.n_layers);
  const int M = a.B * a.T, d = a.d, dff = a.d_ff;
  uint8_t* ws = static_cast<uint8_t*>(a.workspace);
  float* h = reinterpret_cast<float*>(ws + L.h_off);
  uint16_t* xl = reinterpret_cast<uint16_t*>(ws + L.x_off);
  uint16_t* q = reinterpret_cast<uint16_t*>(ws + L.q_off);
  uint16_t* k = reinterpret_cast<uint16_t*>(ws + L.k_off);
  uint16_t* v = reinterpret_cast<uint16_t*>(ws + L.v_off);
  uint16_t* att = reinterpret_cast<uint16_t*>(ws + L.att_off);
  uint16_t* ff = reinterpret_cast<uint16_t*>(ws + L.ff_off);
  int32_t* cu = reinterpret_cast<int32_t*>(ws + L.cu_off);
  const float* P = a.params;
  for (int i = 0; i < a.n_layers; ++i) {
    const float* lp = P + (size_t)i * L.layer_params;
    const float* ln1_g = lp;
    const float* ln1_b = ln1_g + d;
    const float* w_qkv = ln1_b + d;
    const float* b_qkv = w_qkv + (size_t)3 * d * d;
    const float* w_o = b_qkv + 3 * d;
    const float* b_o = w_o + (size_t)d * d;
    const float* ln2_g = b_o + d;
    const float* ln2_b = ln2_g + d;
    const float* w_up = ln2_b + d;
    const float* b_up = w_up + (size_t)dff * d;
    const float* w_dn = b_up + dff;
    const float* b_dn = w_dn + (size_t)d * dff;
    ln<EPL>(i == 0 ? a.emb : nullptr, h, ln1_g, ln1_b, xl, M, a.B, a.T, i == 0 ? cu : nullptr, s);
    gemm<kOutBf16>(xl, w_qkv, b_qkv, M, 3 * d, d, q, k, v, 3, nullptr, s);
    AttnArgs at;
    at.in_dtype = LITEVLM_BF16;
    at.out_dtype = LITEVLM_BF16;
    at.B = a.B;
    at.Hq = a.n_heads;
    at.Hkv = a.n_heads;
    at.D = d / a.n_heads;
    at.max_seqlen = a.T;
    at.causal = 0;
    at.q = q;
    at.k = k;
    at.v = v;
    at.cu_seqlens = cu;
    at.logit_scale_log2 = (float)(1.4426950408889634 / sqrt((double)at.D));
    at.out_scale = 1.f;
    at.o = att;
    const hipError_t e = launch_prefill_attn(at, s);
    if (e != hipSuccess) return e;
    gemm<kOutResid>(att, w_o, b_o, M, d, d, nullptr, nullptr, nullptr, 1, h, s);
    ln<EPL>(nullptr, h, ln2_g, ln2_b, xl, M, a.B, a.T, nullptr, s);
    gemm<kOutGelu>(xl, w_up, b_up, M, dff, d, ff, nullptr, nullptr, 1, nullptr, s);
    gemm<kOutResid>(ff, w_dn, b_dn, M, d, dff, nullptr, nullptr, nullptr, 1, h, s);
  }
  const float* fp = P + (size_t)a.n_layers * L.layer_params;
  const float* lnf_g = fp;
  const float* lnf_b = lnf_g + d;
  const float* lat = lnf_b + d;
  const float* w_cq = lat + (size_t)a.n_views * d;
  const float* b_cq = w_cq + (size_t)d * d;
  const float* w_ck = b_cq + d;
  const float* b_ck = w_ck + (size_t)d * d;
  const float* w_cv = b_ck + d;
  const float* b_cv = w_cv + (size_t)d * d;
  const float* w_hd = b_cv + d;
  const float* b_hd = w_hd + (size_t)a.n_views * d;
  ln<EPL>(nullptr, h, lnf_g, lnf_b, xl, M, a.B, a.T, nullptr, s);
  gemm<kOutBf16>(xl, w_ck, b_ck, M, d, d, q, nullptr, nullptr, 1, nullptr, s);
  gemm<kOutBf16>(xl, w_cv, b_cv, M, d, d, k, nullptr, nullptr, 1, nullptr, s);
  const size_t pbytes = (size_t)a.T * sizeof(float);
  if (d == 512)
    hipLaunchKernelGGL((psm_cross_kernel<2>), dim3(a.n_views, a.B), dim3(256), pbytes, s, q, k, lat, w_cq, b_cq, w_hd,
                       b_hd, a.view_logit, a.T, a.n_views);
  else
    hipLaunchKernelGGL((psm_cross_kernel<1>), dim3(a.n_views, a.B), dim3(256), pbytes, s, q, k, lat, w_cq, b_cq, w_hd,
                       b_hd, a.view_logit, a.T, a.n_views);
  return hipGetLastError();
}

}  // namespace

PsmLayout psm_layout(int B, int T, int d, int d_ff, int n_views, int n_layers) {
  PsmLayout L;
  L.layer_params = (size_t)4 * d + (size_t)3 * d * d + 3 * d + (size_t)d * d + d + (size_t)d_ff * d + d_ff +
                   (size_t)d * d_ff + d;
  L.params = (size_t)n_layers * L.layer_params + 2 * (size_t)d + (size_t)n_views * d + 3 * ((size_t)d * d + d) +
             (size_t)n_views * d + n_views;
  const size_t M = (size_t)B * T;
  auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
  size_t off = 0;
  L.h_off = off;
  off = a256(off + M * d * 4);
  L.x_off = off;
  off = a256(off + M * d * 2);
  L.q_off = off;
  off = a256(off + M * d * 2);
  L.k_off = off;
  off = a256(off + M * d * 2);
  L.v_off = off;
  off = a256(off + M * d * 2);
  L.att_off = off;
  off = a256(off + M * d * 2);
  L.ff_off = off;
  off = a256(off + M * d_ff * 2);
  L.cu_off = off;
  off = a256(off + (size_t)(B + 1) * 4);
  L.total = off;
  return L;
}

hipError_t launch_psm_forward(const PsmArgs& a, hipStream_t stream) {
  if (a.d == 256) return run<4>(a, stream);
  return run<8>(a, stream);
}

}  // namespace litevlm
