// Causal GQA prefill attention over packed variable-length sequences: the
// quadratic part of the LLM prefill that token compression shrinks
// (Introduction; Related Work, Visual Token Compression; Figure 3b).
//
// bf16 path: flash-style forward on v_mfma_f32_32x32x16_bf16 with fp32
// accumulation and an online softmax in the exp2 domain. A workgroup owns 128
// query rows of one query head (4 waves x 32 rows) and streams the keys of its
// KV head in tiles of 64 through LDS.
//
// Both products are formed transposed so that a lane owns one query row
// throughout: S^T = K Q^T puts query (lane % 32) in the accumulator columns,
// and O^T = V^T P^T keeps the same ownership for the output, so the running
// max / sum / rescale of a row never leave the two lanes (lane, lane ^ 32)
// that hold it. Q stays in registers as the B operand. K rows are read from
// LDS as the A operand in a permuted order (bits 2 and 3 of the row index
// swapped) chosen so that the exponentiated accumulator of S^T is already the
// B operand of the P.V product, 8 consecutive keys per lane. V is stored
// transposed in LDS ([d][key]) so its A-operand reads are 16-byte rows.
#include "common.hpp"
#include "launch.hpp"

namespace litevlm {

struct AttnParams {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* cu;
  void* o;
  int B, Hq, Hkv, G, n_mtiles;
  float scale_log2, out_scale;
};

// Row of the 32x32 accumulator held in register r by lane half hl.
__device__ __forceinline__ int acc_row32(int r, int hl) { return 8 * (r >> 2) + 4 * hl + (r & 3); }
// Swap bits 2 and 3: the K-row order that lines S^T up with the P.V operand.
__device__ __forceinline__ int swap23(int x) { return (x & ~12) | ((x & 4) << 1) | ((x & 8) >> 1); }

template <int OUT>
__device__ __forceinline__ void store_out(void* o, size_t idx, float x) {
  if (OUT == LITEVLM_BF16) static_cast<uint16_t*>(o)[idx] = f32_to_bf16_bits(x);
  else static_cast<float*>(o)[idx] = x;
}

template <int D, bool CAUSAL, int OUT>
__global__ void __launch_bounds__(256)
attn_fwd_bf16_kernel(AttnParams p) {
  constexpr int BM = 128, BN = 64;
  constexpr int KS = D / 16;   // k-steps of S^T (contraction over head dims)
  constexpr int DB = D / 32;   // 32-row blocks of O^T
  constexpr int KPAD = D + 8;  // LDS row stride of the K tile [BN][KPAD]
  constexpr int VPAD = BN + 8; // LDS row stride of the V^T tile [D][VPAD]
  __shared__ __attribute__((aligned(16))) uint16_t Ks[BN * KPAD];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D * VPAD];

  const uint16_t* __restrict__ q = static_cast<const uint16_t*>(p.q);
  const uint16_t* __restrict__ k = static_cast<const uint16_t*>(p.k);
  const uint16_t* __restrict__ v = static_cast<const uint16_t*>(p.v);

  // heaviest query tiles first: the tile index is the slowest grid dimension, reversed
  const int hb_count = p.Hq * p.B;
  const int hb = blockIdx.x % hb_count;
  const int mt = p.n_mtiles - 1 - (int)(blockIdx.x / hb_count);
  const int h = hb % p.Hq, b = hb / p.Hq;
  const int seq0 = p.cu[b];
  const int len = p.cu[b + 1] - seq0;
  const int m0 = mt * BM;
  if (m0 >= len) return;
  const int g = h / p.G;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lq = lane & 31, hl = lane >> 5;
  const int qi = m0 + w * 32 + lq;
  const bool q_ok = qi < len;

  bf16x8 qreg[KS];
  {
    const uint16_t* qr = q + ((size_t)(seq0 + qi) * p.Hq + h) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qreg[ks] = q_ok ? *reinterpret_cast<const bf16x8*>(qr + ks * 16 + 8 * hl) : bf16x8{};
  }

  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  const int kend = CAUSAL ? min(len, m0 + BM) : len;
  const int wave_q0 = m0 + w * 32;
  const size_t kvrow = (size_t)p.Hkv * D;
  const uint16_t* kbase = k + ((size_t)seq0 * p.Hkv + g) * D;
  const uint16_t* vbase = v + ((size_t)seq0 * p.Hkv + g) * D;

  for (int k0 = 0; k0 < kend; k0 += BN) {
    __syncthreads();
    // K tile, row-major
    for (int c = tid; c < BN * D / 8; c += 256) {
      const int key = c / (D / 8), d8 = (c % (D / 8)) * 8;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (k0 + key < len) val = *reinterpret_cast<const uint4*>(kbase + (k0 + key) * kvrow + d8);
      *reinterpret_cast<uint4*>(&Ks[key * KPAD + d8]) = val;
    }
    // V tile, transposed: each thread packs 4 keys x 8 dims into 8 row writes
    for (int c = tid; c < (BN / 4) * (D / 8); c += 256) {
      const int kq = c / (D / 8), d8 = (c % (D / 8)) * 8;
      uint4 r4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = 4 * kq + i;
        r4[i] = (k0 + key < len) ? *reinterpret_cast<const uint4*>(vbase + (k0 + key) * kvrow + d8)
                                 : make_uint4(0, 0, 0, 0);
      }
      const uint16_t* e0 = reinterpret_cast<const uint16_t*>(&r4[0]);
      const uint16_t* e1 = reinterpret_cast<const uint16_t*>(&r4[1]);
      const uint16_t* e2 = reinterpret_cast<const uint16_t*>(&r4[2]);
      const uint16_t* e3 = reinterpret_cast<const uint16_t*>(&r4[3]);
#pragma unroll
      for (int dd = 0; dd < 8; ++dd) {
        uint2 pk;
        pk.x = (uint32_t)e0[dd] | ((uint32_t)e1[dd] << 16);
        pk.y = (uint32_t)e2[dd] | ((uint32_t)e3[dd] << 16);
        *reinterpret_cast<uint2*>(&Vt[(d8 + dd) * VPAD + 4 * kq]) = pk;
      }
    }
    __syncthreads();
    if (CAUSAL && k0 > wave_q0 + 31) continue;  // every key of the tile is after this wave's rows

    f32x16 s[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[nb][r] = 0.f;
      const uint16_t* krow = &Ks[(nb * 32 + swap23(lq)) * KPAD + 8 * hl];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        s[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            *reinterpret_cast<const bf16x8*>(krow + ks * 16), qreg[ks], s[nb], 0, 0, 0);
    }

    const bool need_mask = (k0 + BN > len) || (CAUSAL && k0 + BN - 1 > wave_q0);
    float mx = -INFINITY;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float x = s[nb][r] * p.scale_log2;
        if (need_mask) {
          const int key = k0 + nb * 32 + swap23(acc_row32(r, hl));
          if (key >= len || (CAUSAL && key > qi)) x = -INFINITY;
        }
        s[nb][r] = x;
        mx = fmaxf(mx, x);
      }
    mx = wave_max_xor(mx, 32);
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = exp2f(m_run - m_use);
    m_run = m_new;
    float rowsum = 0.f;
    bf16x8 pb[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      float pv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        pv[e] = exp2f(s[kk >> 1][8 * (kk & 1) + e] - m_use);
        rowsum += pv[e];
      }
      pb[kk] = pack_bf16x8(pv);
    }
    l_run = l_run * alpha + rowsum;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const uint16_t* vrow = &Vt[(db * 32 + lq) * VPAD + 8 * hl];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            *reinterpret_cast<const bf16x8*>(vrow + kk * 16), pb[kk], o[db], 0, 0, 0);
    }
  }

  const float l = l_run + __shfl_xor(l_run, 32, kWave);
  const float inv = (l > 0.f) ? p.out_scale / l : 0.f;
  if (q_ok) {
    const size_t obase = ((size_t)(seq0 + qi) * p.Hq + h) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) store_out<OUT>(p.o, obase + db * 32 + acc_row32(r, hl), o[db][r] * inv);
  }
}

// fp32 path: one lane per query row, K/V tiles of 64 keys staged in LDS,
// plain FMAs. Meant for small fp32 problems.
template <int D, bool CAUSAL, int OUT>
__global__ void __launch_bounds__(64)
attn_fwd_f32_kernel(AttnParams p) {
  constexpr int BN = 64;
  __shared__ float Ksh[BN][D];
  __shared__ float Vsh[BN][D];
  const float* __restrict__ q = static_cast<const float*>(p.q);
  const float* __restrict__ k = static_cast<const float*>(p.k);
  const float* __restrict__ v = static_cast<const float*>(p.v);
  const int hb_count = p.Hq * p.B;
  const int hb = blockIdx.x % hb_count;
  const int mt = p.n_mtiles - 1 - (int)(blockIdx.x / hb_count);
  const int h = hb % p.Hq, b = hb / p.Hq;
  const int seq0 = p.cu[b];
  const int len = p.cu[b + 1] - seq0;
  const int m0 = mt * 64;
  if (m0 >= len) return;
  const int g = h / p.G;
  const int qi = m0 + threadIdx.x;
  const bool q_ok = qi < len;
  float qr[D], acc[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    qr[d] = q_ok ? q[((size_t)(seq0 + qi) * p.Hq + h) * D + d] : 0.f;
    acc[d] = 0.f;
  }
  float m_run = -INFINITY, l_run = 0.f;
  const int kend = CAUSAL ? min(len, m0 + 64) : len;
  for (int k0 = 0; k0 < kend; k0 += BN) {
    __syncthreads();
    for (int c = threadIdx.x; c < BN * D; c += 64) {
      const int key = c / D, d = c % D;
      const bool ok = k0 + key < len;
      const size_t idx = ((size_t)(seq0 + k0 + key) * p.Hkv + g) * D + d;
      Ksh[key][d] = ok ? k[idx] : 0.f;
      Vsh[key][d] = ok ? v[idx] : 0.f;
    }
    __syncthreads();
    const int nk = min(BN, kend - k0);
    for (int j = 0; j < nk; ++j) {
      const int key = k0 + j;
      if (CAUSAL && key > qi) break;
      float s = 0.f;
#pragma unroll
      for (int d = 0; d < D; ++d) s = fmaf(qr[d], Ksh[j][d], s);
      const float x = s * p.scale_log2;
      const float m_new = fmaxf(m_run, x);
      const float alpha = exp2f(m_run - m_new);
      const float pj = exp2f(x - m_new);
      l_run = l_run * alpha + pj;
#pragma unroll
      for (int d = 0; d < D; ++d) acc[d] = fmaf(pj, Vsh[j][d], acc[d] * alpha);
      m_run = m_new;
    }
  }
  if (q_ok) {
    const float inv = (l_run > 0.f) ? p.out_scale / l_run : 0.f;
    const size_t obase = ((size_t)(seq0 + qi) * p.Hq + h) * D;
#pragma unroll
    for (int d = 0; d < D; ++d) store_out<OUT>(p.o, obase + d, acc[d] * inv);
  }
}

template <int D, bool CAUSAL, int OUT>
static void launch_typed(const AttnArgs& a, AttnParams& p, hipStream_t stream) {
  if (a.in_dtype == LITEVLM_BF16) {
    p.n_mtiles = (a.max_seqlen + 127) / 128;
    hipLaunchKernelGGL((attn_fwd_bf16_kernel<D, CAUSAL, OUT>), dim3(p.n_mtiles * a.Hq * a.B),
                       dim3(256), 0, stream, p);
  } else {
    p.n_mtiles = (a.max_seqlen + 63) / 64;
    hipLaunchKernelGGL((attn_fwd_f32_kernel<D, CAUSAL, OUT>), dim3(p.n_mtiles * a.Hq * a.B),
                       dim3(64), 0, stream, p);
  }
}

template <int D>
static void launch_d(const AttnArgs& a, AttnParams& p, hipStream_t stream) {
  if (a.causal) {
    if (a.out_dtype == LITEVLM_BF16) launch_typed<D, true, LITEVLM_BF16>(a, p, stream);
    else launch_typed<D, true, LITEVLM_F32>(a, p, stream);
  } else {
    if (a.out_dtype == LITEVLM_BF16) launch_typed<D, false, LITEVLM_BF16>(a, p, stream);
    else launch_typed<D, false, LITEVLM_F32>(a, p, stream);
  }
}

hipError_t launch_prefill_attn(const AttnArgs& a, hipStream_t stream) {
  if (a.max_seqlen <= 0) return hipSuccess;
  AttnParams p;
  p.q = a.q;
  p.k = a.k;
  p.v = a.v;
  p.cu = a.cu_seqlens;
  p.o = a.o;
  p.B = a.B;
  p.Hq = a.Hq;
  p.Hkv = a.Hkv;
  p.G = a.Hq / a.Hkv;
  p.scale_log2 = a.logit_scale_log2;
  p.out_scale = a.out_scale;
  if (a.D == 128) launch_d<128>(a, p, stream);
  else launch_d<64>(a, p, stream);
  return hipGetLastError();
}

}  // namespace litevlm
