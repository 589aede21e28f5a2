// Patch Selection Module forward pass: a small pre-norm transformer encoder
// over the text query's token embeddings, then a single-headed cross-attention
// of N learnable latent queries (one per camera view) over the encoded tokens
// and one linear head per view, giving the view logits that the patch
// selection fuses with its lexical scores.
//
// The module is tiny (d = 256, 4 layers, 128 tokens at the benchmark shape),
// so every step is latency-bound: the kernels favour few launches and few
// dependent global round trips over peak rates.
//   - psm_gemm_kernel: bf16 MFMA (v_mfma_f32_32x32x16_bf16) on A [M, K] times
//     W^T, W [N, K] fp32 from the parameter vector (rounded to bf16 as it is
//     loaded). A workgroup owns one 32 x 32 output block and splits the k range
//     over its 4 waves (more workgroups, fewer round trips each); A is either
//     bf16 or the LayerNorm of fp32 rows formed as the operands load (the norm
//     needs no launch of its own). Epilogues: bias plus a split bf16 output
//     (Q/K/V), GELU, or an add into the fp32 residual stream.
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

enum { kOutBf16 = 0, kOutGelu = 1, kOutResid = 2 };

// out = A W^T + bias for one 32 x 32 output block per workgroup, the k range
// split over its 4 waves (wave w: columns [w*K/4, (w+1)*K/4)) and the partial
// blocks summed through LDS in wave order. A is either bf16 x [M, K] or, with
// LNIN, the LayerNorm of the fp32 rows src [M, K] (gain g, bias bt, eps 1e-5),
// formed as the operands load; every wave first takes the mean and variance of
// the block's 32 rows (lane l32 / half hl: half hl of row l32).
// Output: kOutBf16 columns split into nsplit equal ranges, range j to out[j]
// [M, N/nsplit]; kOutGelu bf16 gelu(.) to out[0] [M, N]; kOutResid
// h [M, N] = (rsrc ? rsrc : h) + (.). The block at (0, 0) also writes the
// per-sample row offsets cu[t] = t*T (t <= B) when cu is given.
template <int MODE, bool LNIN>
__global__ __launch_bounds__(256) void psm_gemm_kernel(const uint16_t* __restrict__ x, const float* __restrict__ src,
                                                       const float* __restrict__ g, const float* __restrict__ bt,
                                                       const float* __restrict__ W, const float* __restrict__ bias,
                                                       int M, int N, int K, uint16_t* out0, uint16_t* out1,
                                                       uint16_t* out2, int nsplit, float* h,
                                                       const float* __restrict__ rsrc, int32_t* cu, int B, int T) {
  __shared__ float red[4][16][kWave];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int l32 = lane & 31, hl = lane >> 5;
  const int m0 = blockIdx.x * 32, n0 = blockIdx.y * 32;
  if (cu && blockIdx.x == 0 && blockIdx.y == 0)
    for (int t = threadIdx.x; t <= B; t += 256) cu[t] = t * T;
  const int arow = min(m0 + l32, M - 1);
  float mu = 0.f, rstd = 1.f;
  if constexpr (LNIN) {
    const float4* rp = reinterpret_cast<const float4*>(src + (size_t)arow * K) + hl * (K / 8);
    float s1 = 0.f, s2 = 0.f;
#pragma unroll 8
    for (int i = 0; i < K / 8; ++i) {
      const float4 v = rp[i];
      s1 += (v.x + v.y) + (v.z + v.w);
      s2 = fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, fmaf(v.w, v.w, s2))));
    }
    s1 = sum_xor32(s1);
    s2 = sum_xor32(s2);
    mu = s1 / K;
    rstd = 1.f / sqrtf(fmaxf(s2 / K - mu * mu, 0.f) + 1e-5f);
  }
  const int kw = K / 4, kbeg = w * kw;
  const float* bp = W + (size_t)(n0 + l32) * K + kbeg + 8 * hl;
  auto a_op = [&](int k) __attribute__((always_inline)) {
    if constexpr (LNIN) {
      const int c = kbeg + k + 8 * hl;
      const float* xr = src + (size_t)arow * K + c;
      const float4 x0 = *reinterpret_cast<const float4*>(xr), x1 = *reinterpret_cast<const float4*>(xr + 4);
      const float4 g0 = *reinterpret_cast<const float4*>(g + c), g1 = *reinterpret_cast<const float4*>(g + c + 4);
      const float4 b0 = *reinterpret_cast<const float4*>(bt + c), b1 = *reinterpret_cast<const float4*>(bt + c + 4);
      const float y[8] = {(x0.x - mu) * rstd * g0.x + b0.x, (x0.y - mu) * rstd * g0.y + b0.y,
                          (x0.z - mu) * rstd * g0.z + b0.z, (x0.w - mu) * rstd * g0.w + b0.w,
                          (x1.x - mu) * rstd * g1.x + b1.x, (x1.y - mu) * rstd * g1.y + b1.y,
                          (x1.z - mu) * rstd * g1.z + b1.z, (x1.w - mu) * rstd * g1.w + b1.w};
      return pack_bf16x8(y);
    } else {
      return __builtin_bit_cast(bf16x8, *reinterpret_cast<const psm_u32x4*>(x + (size_t)arow * K + kbeg + k + 8 * hl));
    }
  };
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
  // chunks of CH k16 steps: the chunk's loads are issued before its MFMAs
  constexpr int CH = 4;
  int k = 0;
  for (; k + 16 * CH <= kw; k += 16 * CH) {
    bf16x8 av[CH];
    float4 bv0[CH], bv1[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      av[c] = a_op(k + 16 * c);
      bv0[c] = *reinterpret_cast<const float4*>(bp + k + 16 * c);
      bv1[c] = *reinterpret_cast<const float4*>(bp + k + 16 * c + 4);
    }
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const float bv[8] = {bv0[c].x, bv0[c].y, bv0[c].z, bv0[c].w, bv1[c].x, bv1[c].y, bv1[c].z, bv1[c].w};
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[c], pack_bf16x8(bv), acc, 0, 0, 0);
    }
  }
  for (; k < kw; k += 16) {
    const bf16x8 a = a_op(k);
    const float4 b0 = *reinterpret_cast<const float4*>(bp + k);
    const float4 b1 = *reinterpret_cast<const float4*>(bp + k + 4);
    const float bv[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pack_bf16x8(bv), acc, 0, 0, 0);
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) red[w][r][lane] = acc[r];
  __syncthreads();
  // wave w finishes accumulator registers 4w .. 4w+3 of the block
  const int col = n0 + l32;
  const float bc = bias[col];
#pragma unroll
  for (int rr = 0; rr < 4; ++rr) {
    const int r = 4 * w + rr;
    const int row = m0 + psm_acc_row(r, hl);
    const float val = (((red[0][r][lane] + red[1][r][lane]) + red[2][r][lane]) + red[3][r][lane]) + bc;
    if (row >= M) continue;
    if constexpr (MODE == kOutResid) {
      const size_t i = (size_t)row * N + col;
      h[i] = (rsrc ? rsrc[i] : h[i]) + val;
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

template <int MODE, bool LNIN>
void gemm(const uint16_t* x, const float* src, const float* g, const float* bt, const float* W, const float* bias,
          int M, int N, int K, uint16_t* o0, uint16_t* o1, uint16_t* o2, int nsplit, float* h, const float* rsrc,
          int32_t* cu, int B, int T, hipStream_t s) {
  hipLaunchKernelGGL((psm_gemm_kernel<MODE, LNIN>), dim3((M + 31) / 32, N / 32), dim3(256), 0, s, x, src, g, bt, W,
                     bias, M, N, K, o0, o1, o2, nsplit, h, rsrc, cu, B, T);
}

hipError_t run(const PsmArgs& a, hipStream_t s) {
  const PsmLayout L = psm_layout(a.B, a.T, a.d, a.d_ff, a.n_views, a.n_layers);
  const int M = a.B * a.T, d = a.d, dff = a.d_ff, B = a.B, T = a.T;
  uint8_t* ws = static_cast<uint8_t*>(a.workspace);
  float* h = reinterpret_cast<float*>(ws + L.h_off);
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
    // the first layer reads the embeddings; its first residual add seeds h
    const float* hin = i == 0 ? a.emb : h;
    gemm<kOutBf16, true>(nullptr, hin, ln1_g, ln1_b, w_qkv, b_qkv, M, 3 * d, d, q, k, v, 3, nullptr, nullptr,
                         i == 0 ? cu : nullptr, B, T, s);
    AttnArgs at;
    at.in_dtype = LITEVLM_BF16;
    at.out_dtype = LITEVLM_BF16;
    at.B = B;
    at.Hq = a.n_heads;
    at.Hkv = a.n_heads;
    at.D = d / a.n_heads;
    at.max_seqlen = T;
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
    gemm<kOutResid, false>(att, nullptr, nullptr, nullptr, w_o, b_o, M, d, d, nullptr, nullptr, nullptr, 1, h,
                           i == 0 ? a.emb : nullptr, nullptr, B, T, s);
    gemm<kOutGelu, true>(nullptr, h, ln2_g, ln2_b, w_up, b_up, M, dff, d, ff, nullptr, nullptr, 1, nullptr, nullptr,
                         nullptr, B, T, s);
    gemm<kOutResid, false>(ff, nullptr, nullptr, nullptr, w_dn, b_dn, M, d, dff, nullptr, nullptr, nullptr, 1, h,
                           nullptr, nullptr, B, T, s);
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
  gemm<kOutBf16, true>(nullptr, h, lnf_g, lnf_b, w_ck, b_ck, M, d, d, q, nullptr, nullptr, 1, nullptr, nullptr,
                       nullptr, B, T, s);
  gemm<kOutBf16, true>(nullptr, h, lnf_g, lnf_b, w_cv, b_cv, M, d, d, k, nullptr, nullptr, 1, nullptr, nullptr,
                       nullptr, B, T, s);
  const size_t pbytes = (size_t)T * sizeof(float);
  if (d == 512)
    hipLaunchKernelGGL((psm_cross_kernel<2>), dim3(a.n_views, B), dim3(256), pbytes, s, q, k, lat, w_cq, b_cq, w_hd,
                       b_hd, a.view_logit, T, a.n_views);
  else
    hipLaunchKernelGGL((psm_cross_kernel<1>), dim3(a.n_views, B), dim3(256), pbytes, s, q, k, lat, w_cq, b_cq, w_hd,
                       b_hd, a.view_logit, T, a.n_views);
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

hipError_t launch_psm_forward(const PsmArgs& a, hipStream_t stream) { return run(a, stream); }

}  // namespace litevlm
