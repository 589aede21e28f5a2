// Extend-one decode attention over the compacted KV cache.
//
// After the prefill, each generated token attends to the S'_b cached tokens of
// its sample's compacted sequence and to itself. The work per token is one pass
// over the cached keys and values, so the step is bound by HBM reads of the
// cache, not by arithmetic: at G query heads per KV head it does 2*G flops per
// cached element read. That is far below the VALU rate needed to keep up with
// HBM, so the products run as fp32 FMAs on the vector units (exact bf16 and E4M3
// products) and every byte of the cache is read once.
//
// Split-K over the key axis (flash decoding): a workgroup owns L consecutive
// keys of one (sample, KV head) and all G query heads that read that KV head,
// so each cached row is fetched by one workgroup only. It writes the split's
// running max, sum and unnormalised output per query head; a second kernel
// merges the splits of each (sample, head) in split order, so the result does
// not depend on which workgroup finishes first.
#include "common.hpp"
#include "launch.hpp"

namespace litevlm {
namespace {

constexpr int kDecThreads = 256;  // 4 waves = 16 key groups of 16 lanes
constexpr int kKeyGroups = kDecThreads / 16;

// Keys per split when the grid is already large (64 otherwise): 128 for every
// dtype. Longer splits (256 keys) hold more K and V rows in registers per
// workgroup but leave fewer workgroups in flight; on the batch-8 caches of
// 1-2K tokens 128 was faster (bf16 20.4 -> 18.0 us, E4M3 20.0 -> 17.5 us).
constexpr int split_len_big(int, int) { return 128; }

template <int DT>
constexpr int elem_bytes() {
  return DT == LITEVLM_F32 ? 4 : DT == LITEVLM_BF16 ? 2 : 1;
}

// The raw bits of EPL consecutive elements of one row (one lane's share).
template <int DT, int EPL>
struct Raw {
  static constexpr int kBytes = EPL * elem_bytes<DT>();
  static constexpr int kWords = kBytes / 4;
  uint32_t w[kWords];
};

template <int DT, int EPL>
__device__ __forceinline__ Raw<DT, EPL> load_raw(const uint8_t* p) {
  Raw<DT, EPL> r;
  constexpr int W = Raw<DT, EPL>::kWords;
  static_assert(W == 1 || W == 2 || W % 4 == 0, "row share must be 4, 8 or 16n bytes");
  if constexpr (W % 4 == 0) {
#pragma unroll
    for (int i = 0; i < W / 4; ++i) {
      const uint4 x = reinterpret_cast<const uint4*>(p)[i];
      r.w[4 * i] = x.x;
      r.w[4 * i + 1] = x.y;
      r.w[4 * i + 2] = x.z;
      r.w[4 * i + 3] = x.w;
    }
  } else if constexpr (W == 2) {
    const uint2 x = *reinterpret_cast<const uint2*>(p);
    r.w[0] = x.x;
    r.w[1] = x.y;
  } else {
    r.w[0] = *reinterpret_cast<const uint32_t*>(p);
  }
  return r;
}

// Exact widening to fp32.
template <int DT, int EPL>
__device__ __forceinline__ void widen(const Raw<DT, EPL>& r, float* x) {
  if constexpr (DT == LITEVLM_F32) {
#pragma unroll
    for (int i = 0; i < EPL; ++i) x[i] = __uint_as_float(r.w[i]);
  } else if constexpr (DT == LITEVLM_BF16) {
#pragma unroll
    for (int i = 0; i < EPL / 2; ++i) {
      x[2 * i] = __uint_as_float(r.w[i] << 16);
      x[2 * i + 1] = __uint_as_float(r.w[i] & 0xFFFF0000u);
    }
  } else {
    // gfx950's fp8 conversions use the OCP E4M3FN encoding
#pragma unroll
    for (int i = 0; i < EPL / 4; ++i) {
      const auto lo = __builtin_amdgcn_cvt_pk_f32_fp8((int)r.w[i], false);
      const auto hi = __builtin_amdgcn_cvt_pk_f32_fp8((int)r.w[i], true);
      x[4 * i] = lo[0];
      x[4 * i + 1] = lo[1];
      x[4 * i + 2] = hi[0];
      x[4 * i + 3] = hi[1];
    }
  }
}

struct DecodeParams {
  const uint8_t* q1;  // [B, Hq, D]
  const uint8_t* k1;  // [B, Hkv, D]
  const uint8_t* v1;  // [B, Hkv, D]
  const uint8_t* kc;  // [total, Hkv, D]
  const uint8_t* vc;  // [total, Hkv, D]
  const int32_t* cu;  // [B + 1]
  float* part_o;      // [B, Hq, nsplit, D]   unnormalised split outputs
  float2* part_ml;    // [B, Hq, nsplit]      split (max, sum), log2 domain
  void* o;            // [B, Hq, D]
  int B, Hq, Hkv, nsplit;
  float scale_log2, out_scale;
};

// Work item of a split workgroup. The grid is sized from the host bound on the
// cache length, so most of it may be surplus. The live items (splits holding at
// least one key) are numbered first, sample by sample and KV head by KV head
// (a head's splits consecutive), so the surplus workgroups, which exit at once,
// are dispatched after every live one instead of between them. Called by every
// thread of the workgroup; the result is uniform across it.
struct SplitItem {
  int b, g, split;
};
template <int L>
__device__ __forceinline__ bool split_item(const DecodeParams& p, int* s_scan, SplitItem& it) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int c = 0;
  if (tid < p.B) {
    const int n = p.cu[tid + 1] - p.cu[tid];
    c = p.Hkv * min(max(n, 0) / L + 1, p.nsplit);
  }
#pragma unroll
  for (int x = 1; x < kWave; x <<= 1) {
    const int y = __shfl_up(c, x, kWave);
    if (lane >= x) c += y;
  }
  if (lane == kWave - 1) s_scan[LITEVLM_MAX_BATCH + 1 + w] = c;  // wave totals
  __syncthreads();
  for (int k = 0; k < w; ++k) c += s_scan[LITEVLM_MAX_BATCH + 1 + k];
  if (tid < p.B) s_scan[tid + 1] = c;
  if (tid == 0) s_scan[0] = 0;
  __syncthreads();
  const int i = blockIdx.x;
  if (i >= s_scan[p.B]) return false;
  int lo = 0, hi = p.B;  // s_scan[lo] <= i < s_scan[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (s_scan[mid] <= i) lo = mid;
    else hi = mid;
  }
  const int r = i - s_scan[lo];
  const int ns = (s_scan[lo + 1] - s_scan[lo]) / p.Hkv;
  it.b = lo;
  it.g = r / ns;
  it.split = r % ns;
  return true;
}

// One workgroup: one split (keys [s*L, s*L + L) of the sequence cache ++ new
// token, i.e. keys 0..n with key n the new token) of one KV head of one sample,
// from split_item. Key group c (16 lanes) takes keys c, c+16, ...
// of the split; lane i of a group holds elements [i*EPL, i*EPL + EPL) of a row.
template <int D, int DT, int G, int L>
__global__ __launch_bounds__(kDecThreads) void decode_split_kernel(DecodeParams p) {
  constexpr int EPL = D / 16;
  constexpr int KPG = L / kKeyGroups;  // keys per group
  constexpr int E = elem_bytes<DT>();
  static_assert(KPG >= 1 && EPL >= 4, "shape");

  __shared__ int s_scan[LITEVLM_MAX_BATCH + 1 + 4];
  SplitItem it;
  if (!split_item<L>(p, s_scan, it)) return;  // surplus workgroup (uniform)
  const int split = it.split, g = it.g, b = it.b;
  const int lo = p.cu[b];
  const int n = p.cu[b + 1] - lo;  // cached tokens of this sample
  const int k0 = split * L;        // <= n for a live item

  const int tid = threadIdx.x;
  const int grp = tid >> 4, li = tid & 15, w = tid >> 6, lane = tid & 63;
  const int64_t row_bytes = (int64_t)p.Hkv * D * E;
  const int share = li * EPL * E;

  // Every K and V row share of the split is requested before any arithmetic.
  Raw<DT, EPL> kr[KPG], vr[KPG];
  const uint8_t* knew = p.k1 + ((int64_t)b * p.Hkv + g) * D * E + share;
  const uint8_t* vnew = p.v1 + ((int64_t)b * p.Hkv + g) * D * E + share;
#pragma unroll
  for (int i = 0; i < KPG; ++i) {
    const int j = k0 + grp + kKeyGroups * i;
    // keys past the new token are masked below; they read the new token's row
    const bool cached = j < n;
    const int64_t off = ((int64_t)(lo + (cached ? j : 0)) * row_bytes) + (int64_t)g * D * E + share;
    kr[i] = load_raw<DT, EPL>(cached ? p.kc + off : knew);
    vr[i] = load_raw<DT, EPL>(cached ? p.vc + off : vnew);
  }
  float qf[G][EPL];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const Raw<DT, EPL> qr = load_raw<DT, EPL>(p.q1 + ((int64_t)b * p.Hq + g * G + h) * D * E + share);
    widen(qr, qf[h]);
  }

  __shared__ float lg[L * G];              // logits, then probabilities: [key][head]
  __shared__ float2 stat[G];               // split (max, sum) per head
  __shared__ float red[4 * G * D];         // per-wave output partials

  // Logits (log2 domain). The 16 lanes of a group reduce by DPP within their row.
#pragma unroll
  for (int i = 0; i < KPG; ++i) {
    float kf[EPL];
    widen(kr[i], kf);
    const int jj = grp + kKeyGroups * i;
    const bool live = k0 + jj <= n;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc = fmaf(qf[h][e], kf[e], acc);
      acc = row16_sum(acc);
      if (li == h) lg[jj * G + h] = live ? acc * p.scale_log2 : -INFINITY;
    }
  }
  __syncthreads();

  // Split softmax statistics: wave w takes heads w, w+4, ...; lane l keys l, l+64, ...
  for (int h = w; h < G; h += 4) {
    float m = -INFINITY;
    for (int j = lane; j < L; j += kWave) m = fmaxf(m, lg[j * G + h]);
#pragma unroll
    for (int x = 1; x < kWave; x <<= 1) m = wave_max_xor(m, x);
    float s = 0.f;
    for (int j = lane; j < L; j += kWave) {
      const float e = __builtin_amdgcn_exp2f(lg[j * G + h] - m);  // masked keys: exp2(-inf) = 0
      lg[j * G + h] = e;
      s += e;
    }
#pragma unroll
    for (int x = 1; x < kWave; x <<= 1) s += __shfl_xor(s, x, kWave);
    if (lane == 0) stat[h] = make_float2(m, s);
  }
  __syncthreads();

  // P V: each lane accumulates its EPL output elements for every head.
  float acc[G][EPL];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[h][e] = 0.f;
#pragma unroll
  for (int i = 0; i < KPG; ++i) {
    float vf[EPL];
    widen(vr[i], vf);
    const int jj = grp + kKeyGroups * i;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float ph = lg[jj * G + h];
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[h][e] = fmaf(ph, vf[e], acc[h][e]);
    }
  }
  // Sum the wave's four key groups (lanes 16 and 32 apart), then the four waves.
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[h][e] = sum_xor32(sum_xor16(acc[h][e]));
  if (lane < 16) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < EPL; ++e) red[(w * G + h) * D + li * EPL + e] = acc[h][e];
  }
  __syncthreads();

  const int64_t head0 = (int64_t)b * p.Hq + g * G;
  for (int t = tid; t < G * D; t += kDecThreads) {
    const int h = t / D, d = t % D;
    const float s = ((red[(0 * G + h) * D + d] + red[(1 * G + h) * D + d]) + red[(2 * G + h) * D + d]) +
                    red[(3 * G + h) * D + d];
    p.part_o[((head0 + h) * p.nsplit + split) * D + d] = s;
  }
  if (tid < G) p.part_ml[(head0 + tid) * p.nsplit + split] = stat[tid];
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c,
                                         false);
}

// bf16 split: the same work as decode_split_kernel with the products on the
// packed bf16 dot unit (two products per instruction, fp32 accumulate), which
// halves the vector instructions per cached byte.
//   Logits: 8 lanes per key, lane i holding the 16-byte pieces i, i+8, ... of
//     the key and of each query head (so each load instruction reads whole
//     128-byte lines), as stored bf16 pairs; the dots are summed over the 8 lanes.
//   P V: 16 lanes per key as in decode_split_kernel; keys c+16i and c+16(i+1)
//     of a group are paired so that one dot takes the pair's (p, v) products;
//     p is rounded to bf16 first and the split's sum is taken over the rounded
//     values, so the weights of the output still sum to the normaliser.
template <int D, int G, int L>
__global__ __launch_bounds__(kDecThreads) void decode_split_bf16_kernel(DecodeParams p) {
  constexpr int E = 2;
  constexpr int WK = D / 16;          // K dwords per lane (8 lanes per key)
  constexpr int KK = L / 32;          // keys per 8-lane group
  constexpr int WV = D / 32;          // V dwords per lane (16 lanes per key)
  constexpr int KV = L / kKeyGroups;  // keys per 16-lane group
  static_assert(KK >= 1 && KV % 2 == 0 && WV >= 2, "shape");

  __shared__ int s_scan[LITEVLM_MAX_BATCH + 1 + 4];
  SplitItem it;
  if (!split_item<L>(p, s_scan, it)) return;
  const int split = it.split, g = it.g, b = it.b;
  const int lo = p.cu[b];
  const int n = p.cu[b + 1] - lo;
  const int k0 = split * L;

  const int tid = threadIdx.x;
  const int g8 = tid >> 3, l8 = tid & 7, g16 = tid >> 4, l16 = tid & 15, w = tid >> 6, lane = tid & 63;
  const int64_t row_bytes = (int64_t)p.Hkv * D * E;
  const int64_t head_off = (int64_t)g * D * E;
  const uint8_t* knew = p.k1 + ((int64_t)b * p.Hkv + g) * D * E;
  const uint8_t* vnew = p.v1 + ((int64_t)b * p.Hkv + g) * D * E;

  uint32_t kw[KK][WK], vw[KV][WV];
#pragma unroll
  for (int i = 0; i < KK; ++i) {
    const int j = k0 + g8 + 32 * i;
    const uint8_t* src = (j < n ? p.kc + (int64_t)(lo + j) * row_bytes + head_off : knew) + 16 * l8;
#pragma unroll
    for (int t = 0; t < WK; t += 4) {
      const uint4 x = *reinterpret_cast<const uint4*>(src + 32 * t);  // piece l8 + 8*(t/4)
      kw[i][t] = x.x;
      kw[i][t + 1] = x.y;
      kw[i][t + 2] = x.z;
      kw[i][t + 3] = x.w;
    }
  }
#pragma unroll
  for (int i = 0; i < KV; ++i) {
    const int j = k0 + g16 + kKeyGroups * i;
    const uint8_t* src = (j < n ? p.vc + (int64_t)(lo + j) * row_bytes + head_off : vnew) + l16 * WV * 4;
    if constexpr (WV == 4) {
      const uint4 x = *reinterpret_cast<const uint4*>(src);
      vw[i][0] = x.x;
      vw[i][1] = x.y;
      vw[i][2] = x.z;
      vw[i][3] = x.w;
    } else {
      const uint2 x = *reinterpret_cast<const uint2*>(src);
      vw[i][0] = x.x;
      vw[i][1] = x.y;
    }
  }
  uint32_t qw[G][WK];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const uint8_t* src = p.q1 + ((int64_t)b * p.Hq + g * G + h) * D * E + 16 * l8;
#pragma unroll
    for (int t = 0; t < WK; t += 4) {
      const uint4 x = *reinterpret_cast<const uint4*>(src + 32 * t);
      qw[h][t] = x.x;
      qw[h][t + 1] = x.y;
      qw[h][t + 2] = x.z;
      qw[h][t + 3] = x.w;
    }
  }

  __shared__ float lg[L * G];
  __shared__ float2 stat[G];
  __shared__ float red[4 * G * D];

#pragma unroll
  for (int i = 0; i < KK; ++i) {
    const int jj = g8 + 32 * i;
    float mine = 0.f;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float acc = 0.f;
#pragma unroll
      for (int t = 0; t < WK; ++t) acc = dot2_bf16(qw[h][t], kw[i][t], acc);
      acc += dpp<0xB1>(acc);   // quad_perm [1,0,3,2]
      acc += dpp<0x4E>(acc);   // quad_perm [2,3,0,1]
      acc += dpp<0x141>(acc);  // row_half_mirror: the other quad of the 8 lanes
      mine = (l8 == h) ? acc : mine;
    }
    if (l8 < G) lg[jj * G + l8] = (k0 + jj <= n) ? mine * p.scale_log2 : -INFINITY;
  }
  __syncthreads();

  for (int h = w; h < G; h += 4) {
    float m = -INFINITY;
    for (int j = lane; j < L; j += kWave) m = fmaxf(m, lg[j * G + h]);
#pragma unroll
    for (int x = 1; x < kWave; x <<= 1) m = wave_max_xor(m, x);
    float s = 0.f;
    for (int j = lane; j < L; j += kWave) {
      const float e = bf16_bits_to_f32(f32_to_bf16_bits(__builtin_amdgcn_exp2f(lg[j * G + h] - m)));
      lg[j * G + h] = e;
      s += e;
    }
#pragma unroll
    for (int x = 1; x < kWave; x <<= 1) s += __shfl_xor(s, x, kWave);
    if (lane == 0) stat[h] = make_float2(m, s);
  }
  __syncthreads();

  float acc[G][2 * WV];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 2 * WV; ++e) acc[h][e] = 0.f;
#pragma unroll
  for (int i = 0; i < KV; i += 2) {
    const int ja = g16 + kKeyGroups * i, jb = ja + kKeyGroups;
    uint32_t pk[G];
#pragma unroll
    for (int h = 0; h < G; ++h)
      pk[h] = (__float_as_uint(lg[ja * G + h]) >> 16) | (__float_as_uint(lg[jb * G + h]) & 0xFFFF0000u);
#pragma unroll
    for (int t = 0; t < WV; ++t) {
      const uint32_t even = __builtin_amdgcn_perm(vw[i + 1][t], vw[i][t], 0x05040100u);  // (v_a[2t], v_b[2t])
      const uint32_t odd = __builtin_amdgcn_perm(vw[i + 1][t], vw[i][t], 0x07060302u);   // (v_a[2t+1], v_b[2t+1])
#pragma unroll
      for (int h = 0; h < G; ++h) {
        acc[h][2 * t] = dot2_bf16(even, pk[h], acc[h][2 * t]);
        acc[h][2 * t + 1] = dot2_bf16(odd, pk[h], acc[h][2 * t + 1]);
      }
    }
  }
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 2 * WV; ++e) acc[h][e] = sum_xor32(sum_xor16(acc[h][e]));
  if (lane < 16) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 2 * WV; ++e) red[(w * G + h) * D + l16 * 2 * WV + e] = acc[h][e];
  }
  __syncthreads();

  const int64_t head0 = (int64_t)b * p.Hq + g * G;
  for (int t = tid; t < G * D; t += kDecThreads) {
    const int h = t / D, d = t % D;
    const float s = ((red[(0 * G + h) * D + d] + red[(1 * G + h) * D + d]) + red[(2 * G + h) * D + d]) +
                    red[(3 * G + h) * D + d];
    p.part_o[((head0 + h) * p.nsplit + split) * D + d] = s;
  }
  if (tid < G) p.part_ml[(head0 + tid) * p.nsplit + split] = stat[tid];
}

// One workgroup per (sample, query head) merges the live splits. Thread t reads
// float4 piece t % (D/4) of splits t / (D/4), t / (D/4) + SLOTS, ... (coalesced
// rows, several splits in flight per thread); the slots are then summed in slot
// order, so the result does not depend on timing.
template <int D, bool OUT_BF16>
__global__ __launch_bounds__(kDecThreads) void decode_combine_kernel(DecodeParams p, int L) {
  constexpr int V4 = D / 4;                // float4 pieces per row
  constexpr int SLOTS = kDecThreads / V4;  // splits read side by side
  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63;
  const int n = p.cu[b + 1] - p.cu[b];
  const int ns = min(n / L + 1, p.nsplit);  // splits holding keys 0..n
  const int64_t head = (int64_t)b * p.Hq + h;
  const float2* ml = p.part_ml + head * p.nsplit;
  const float4* po = reinterpret_cast<const float4*>(p.part_o + head * p.nsplit * D);

  __shared__ float wmax[4];
  __shared__ float4 racc[SLOTS][V4];
  __shared__ float rl[SLOTS];

  // The first R splits of the thread's slot are requested together with their
  // statistics before the maximum is known (addresses clamped to the last
  // split, so every load is valid and none waits on a branch); splits beyond
  // R*SLOTS, for very long caches, are read after it.
  constexpr int R = 8;
  const int slot = tid / V4, c = tid % V4;
  float2 mr[R];
  float4 xr[R];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int s = min(slot + i * SLOTS, ns - 1);
    mr[i] = ml[s];
    xr[i] = po[(int64_t)s * V4 + c];
  }
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < R; ++i) m = fmaxf(m, mr[i].x);  // clamped repeats change no maximum
  for (int s = slot + R * SLOTS; s < ns; s += SLOTS) m = fmaxf(m, ml[s].x);
#pragma unroll
  for (int x = 1; x < kWave; x <<= 1) m = wave_max_xor(m, x);
  if (lane == 0) wmax[w] = m;
  __syncthreads();
  m = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));

  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float l = 0.f;
  auto add = [&](const float2 st, const float4 x) __attribute__((always_inline)) {
    const float wgt = __builtin_amdgcn_exp2f(st.x - m);
    l = fmaf(st.y, wgt, l);
    acc.x = fmaf(x.x, wgt, acc.x);
    acc.y = fmaf(x.y, wgt, acc.y);
    acc.z = fmaf(x.z, wgt, acc.z);
    acc.w = fmaf(x.w, wgt, acc.w);
  };
#pragma unroll
  for (int i = 0; i < R; ++i)
    if (slot + i * SLOTS < ns) add(mr[i], xr[i]);
#pragma unroll 4
  for (int s = slot + R * SLOTS; s < ns; s += SLOTS) add(ml[s], po[(int64_t)s * V4 + c]);
  racc[slot][c] = acc;
  if (c == 0) rl[slot] = l;
  __syncthreads();
  if (tid < V4) {
    float4 t = racc[0][tid];
    float lt = rl[0];
    for (int q = 1; q < SLOTS; ++q) {
      const float4 u = racc[q][tid];
      t.x += u.x;
      t.y += u.y;
      t.z += u.z;
      t.w += u.w;
      lt += rl[q];
    }
    const float f = p.out_scale / lt;
    if constexpr (OUT_BF16) {
      uint2 pk;
      pk.x = (uint32_t)f32_to_bf16_bits(t.x * f) | ((uint32_t)f32_to_bf16_bits(t.y * f) << 16);
      pk.y = (uint32_t)f32_to_bf16_bits(t.z * f) | ((uint32_t)f32_to_bf16_bits(t.w * f) << 16);
      reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.o) + head * D)[tid] = pk;
    } else {
      reinterpret_cast<float4*>(static_cast<float*>(p.o) + head * D)[tid] =
          make_float4(t.x * f, t.y * f, t.z * f, t.w * f);
    }
  }
}

template <int D, int DT, int G, int L>
void launch_split(const DecodeParams& p, int B, hipStream_t stream) {
  hipLaunchKernelGGL((decode_split_kernel<D, DT, G, L>), dim3(p.nsplit * p.Hkv * B), dim3(kDecThreads), 0,
                     stream, p);
}

template <int D, int DT, int G>
void launch_g(const DecodeParams& p, int B, int L, hipStream_t stream) {
  constexpr int LBIG = split_len_big(DT, G);
  if constexpr (DT == LITEVLM_BF16) {
    if (L == 64)
      hipLaunchKernelGGL((decode_split_bf16_kernel<D, G, 64>), dim3(p.nsplit * p.Hkv * B), dim3(kDecThreads),
                         0, stream, p);
    else
      hipLaunchKernelGGL((decode_split_bf16_kernel<D, G, LBIG>), dim3(p.nsplit * p.Hkv * B),
                         dim3(kDecThreads), 0, stream, p);
  } else {
    if (L == 64) launch_split<D, DT, G, 64>(p, B, stream);
    else launch_split<D, DT, G, LBIG>(p, B, stream);
  }
}

template <int D, int DT>
void launch_dt(const DecodeParams& p, int B, int G, int L, hipStream_t stream) {
  switch (G) {
    case 1: launch_g<D, DT, 1>(p, B, L, stream); break;
    case 2: launch_g<D, DT, 2>(p, B, L, stream); break;
    case 4: launch_g<D, DT, 4>(p, B, L, stream); break;
    default: launch_g<D, DT, 8>(p, B, L, stream); break;
  }
}

template <int D>
void launch_d(const DecodeParams& p, int dt, int B, int G, int L, bool out_bf16, hipStream_t stream) {
  if (dt == LITEVLM_F32) launch_dt<D, LITEVLM_F32>(p, B, G, L, stream);
  else if (dt == LITEVLM_BF16) launch_dt<D, LITEVLM_BF16>(p, B, G, L, stream);
  else launch_dt<D, LITEVLM_FP8_E4M3>(p, B, G, L, stream);
  if (out_bf16)
    hipLaunchKernelGGL((decode_combine_kernel<D, true>), dim3(p.Hq, B), dim3(kDecThreads), 0, stream, p, L);
  else
    hipLaunchKernelGGL((decode_combine_kernel<D, false>), dim3(p.Hq, B), dim3(kDecThreads), 0, stream, p, L);
}

}  // namespace

DecodeLayout decode_layout(int in_dtype, int B, int Hq, int Hkv, int D, int max_seqlen) {
  DecodeLayout lay;
  // Keys per split: the largest of {LBIG, 64} that still gives about two
  // workgroups per CU over the upper-bound length (keys 0..max_seqlen).
  const int lbig = split_len_big(in_dtype, Hq / Hkv);
  const int64_t want = 512;
  lay.split_len = ((int64_t)B * Hkv * ((max_seqlen + lbig) / lbig) >= want) ? lbig : 64;
  lay.nsplit = (max_seqlen + lay.split_len) / lay.split_len;
  const size_t heads = (size_t)B * Hq * lay.nsplit;
  lay.part_o_off = 0;
  lay.part_ml_off = (heads * D * sizeof(float) + 255) & ~(size_t)255;
  lay.total = lay.part_ml_off + heads * sizeof(float2);
  return lay;
}

hipError_t launch_decode_attn(const DecodeArgs& a, hipStream_t stream) {
  const DecodeLayout lay = decode_layout(a.in_dtype, a.B, a.Hq, a.Hkv, a.D, a.max_seqlen);
  DecodeParams p;
  p.q1 = static_cast<const uint8_t*>(a.q1);
  p.k1 = static_cast<const uint8_t*>(a.k1);
  p.v1 = static_cast<const uint8_t*>(a.v1);
  p.kc = static_cast<const uint8_t*>(a.kc);
  p.vc = static_cast<const uint8_t*>(a.vc);
  p.cu = a.cu_seqlens;
  p.part_o = reinterpret_cast<float*>(static_cast<uint8_t*>(a.workspace) + lay.part_o_off);
  p.part_ml = reinterpret_cast<float2*>(static_cast<uint8_t*>(a.workspace) + lay.part_ml_off);
  p.o = a.o;
  p.B = a.B;
  p.Hq = a.Hq;
  p.Hkv = a.Hkv;
  p.nsplit = lay.nsplit;
  p.scale_log2 = a.logit_scale_log2;
  p.out_scale = a.out_scale;
  const int G = a.Hq / a.Hkv;
  const bool out_bf16 = a.out_dtype == LITEVLM_BF16;
  if (a.D == 128) launch_d<128>(p, a.in_dtype, a.B, G, lay.split_len, out_bf16, stream);
  else launch_d<64>(p, a.in_dtype, a.B, G, lay.split_len, out_bf16, stream);
  return hipGetLastError();
}

}  // namespace litevlm
