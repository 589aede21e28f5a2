// Text-guided visual-token scoring (Design section, Token Selection Module
// paragraph): the attention mass that the text rows of the first decoder layer
// put on each visual token, averaged over query heads and text rows.
//
// For KV group g the R = G*T text query rows (row r = t*G + hh is query head
// g*G+hh of text token t) attend causally over the patch-selected sequence.
// In original positions that is: kept visual keys (token_keep = 1) and text
// keys V_full+t' with t' <= t. Exact column mass needs each row's softmax
// normaliser first, so the work is two sweeps over K:
//   sweep 1  per (key tile, row): max m and sum Z of exp2(logit) over the tile
//   merge    per row: m = max over tiles, Z = sum Z_tile * exp2(m_tile - m)
//   sweep 2  per visual key: sum over rows of exp2(logit - m) / Z
// Logits are formed transposed, S^T = K Q^T, on MFMA: the key tile stays in
// registers as the A operand and 16 query rows at a time stream through the B
// operand. In the 16x16 accumulator a lane owns one query row (lane % 16) and
// four keys per 16-key block (4*(lane/16) + e). Every reduction runs in a
// fixed order, so results are deterministic.
#include "common.hpp"
#include "launch.hpp"

namespace litevlm {

constexpr int KT = kScoreKeyTile;  // keys per tile: 4 blocks of 16
constexpr int kScoreWaves = 4;

// ---------------------------------------------------------------- logit tiles
// Each tile policy holds 64 keys of one KV head and produces, for 16 query
// rows, acc[kb][e] = k(kb*16 + 4*(lane/16) + e) . q(lane % 16) in fp32.

template <int D>
struct TileBf16 {
  static constexpr int KS = D / 32;  // k-steps of v_mfma_f32_16x16x32_bf16
  bf16x8 kreg[4][KS];

  __device__ __forceinline__ void load_keys(const uint16_t* kbase, size_t kstride, int nvalid,
                                            int lane) {
    const int c = lane & 15, g4 = lane >> 4;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const int key = kb * 16 + c;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if (key < nvalid)
          kreg[kb][ks] = *reinterpret_cast<const bf16x8*>(kbase + key * kstride + ks * 32 + 8 * g4);
        else
          kreg[kb][ks] = bf16x8{};
      }
    }
  }

  // qrow: this lane's query row (row lane % 16), or nullptr for a padding row.
  __device__ __forceinline__ void logits(const uint16_t* qrow, int lane, f32x4 acc[4]) const {
    const int g4 = lane >> 4;
    bf16x8 qreg[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qreg[ks] = qrow ? *reinterpret_cast<const bf16x8*>(qrow + ks * 32 + 8 * g4) : bf16x8{};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kreg[kb][ks], qreg[ks], a, 0, 0, 0);
      acc[kb] = a;
    }
  }
};

template <int D>
struct TileFp8 {
  // v_mfma_f32_16x16x128_f8f6f4: one k-step covers 128 head dims; a lane
  // supplies 32 consecutive E4M3 bytes. D = 64 zero-pads the upper half.
  i32x8 kreg[4];

  __device__ __forceinline__ void load_keys(const uint8_t* kbase, size_t kstride, int nvalid,
                                            int lane) {
    const int c = lane & 15, g4 = lane >> 4;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const int key = kb * 16 + c;
      if (key < nvalid && 32 * g4 < D)
        kreg[kb] = *reinterpret_cast<const i32x8*>(kbase + key * kstride + 32 * g4);
      else
        kreg[kb] = i32x8{};
    }
  }

  __device__ __forceinline__ void logits(const uint8_t* qrow, int lane, f32x4 acc[4]) const {
    const int g4 = lane >> 4;
    const i32x8 qreg = (qrow && 32 * g4 < D) ? *reinterpret_cast<const i32x8*>(qrow + 32 * g4) : i32x8{};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
      // format 0 = E4M3 for both operands; zero scale operands select the
      // unscaled instruction.
      acc[kb] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(kreg[kb], qreg, z, 0, 0, 0, 0, 0, 0);
    }
  }
};

template <int D>
struct TileF32 {
  // Plain fp32 FMAs (no fp32 matrix path is worth it at the sizes fp32 is
  // used for). The lane's own 16 keys are read from global memory per row
  // block; Q stays in registers per row block.
  const float* kbase;
  size_t kstride;
  int nvalid;

  __device__ __forceinline__ void load_keys(const float* kb_, size_t ks_, int nv, int) {
    kbase = kb_;
    kstride = ks_;
    nvalid = nv;
  }

  __device__ __forceinline__ void logits(const float* qrow, int lane, f32x4 acc[4]) const {
    const int g4 = lane >> 4;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = kb * 16 + 4 * g4 + e;
        float s = 0.f;
        if (qrow && key < nvalid) {
          const float* kr = kbase + key * kstride;
          for (int d = 0; d < D; ++d) s = fmaf(qrow[d], kr[d], s);
        }
        acc[kb][e] = s;
      }
    }
  }
};

template <int DT, int D>
struct TileOf;
template <int D> struct TileOf<LITEVLM_BF16, D> { using T = TileBf16<D>; using E = uint16_t; };
template <int D> struct TileOf<LITEVLM_FP8_E4M3, D> { using T = TileFp8<D>; using E = uint8_t; };
template <int D> struct TileOf<LITEVLM_F32, D> { using T = TileF32<D>; using E = float; };

struct ScoreDims {
  int S, V_full, T, Hq, Hkv, G, R, n_kt;
  float scale_log2;
};

// Bitmask over the lane's 16 accumulator keys (bit kb*4+e): key is visual and kept.
__device__ __forceinline__ uint32_t kept_visual_mask(const uint8_t* keep_row, int key0, int V_full,
                                                     int lane) {
  const int g4 = lane >> 4;
  uint32_t m = 0;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int key = key0 + kb * 16 + 4 * g4 + e;
      if (key < V_full && (keep_row == nullptr || keep_row[key])) m |= 1u << (kb * 4 + e);
    }
  return m;
}

template <class E>
__device__ __forceinline__ const E* text_row_ptr(const E* q, int b, int g, int r, const ScoreDims& d,
                                                 int Dh) {
  const int t = r / d.G, hh = r - t * d.G;
  return q + (((size_t)b * d.S + d.V_full + t) * d.Hq + (size_t)g * d.G + hh) * Dh;
}

// ---------------------------------------------------------------- sweep 1

template <int DT, int D>
__global__ void __launch_bounds__(256)
score_rowstats_kernel(ScoreDims d, const void* __restrict__ qv, const void* __restrict__ kv,
                      const uint8_t* __restrict__ token_keep, float2* __restrict__ rowpart) {
  using Tile = typename TileOf<DT, D>::T;
  using E = typename TileOf<DT, D>::E;
  const E* q = static_cast<const E*>(qv);
  const E* k = static_cast<const E*>(kv);
  const int kt = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, g4 = lane >> 4;
  const int key0 = kt * KT;
  const int nvalid = min(KT, d.S - key0);
  const uint8_t* keep_row = token_keep ? token_keep + (size_t)b * d.S : nullptr;

  Tile tile;
  tile.load_keys(k + (((size_t)b * d.S + key0) * d.Hkv + g) * D, (size_t)d.Hkv * D, nvalid, lane);
  const uint32_t vis = kept_visual_mask(keep_row, key0, d.V_full, lane);

  const int nchunks = (d.R + 15) / 16;
  for (int ch = wave; ch < nchunks; ch += kScoreWaves) {
    const int r = ch * 16 + c;
    const bool row_ok = r < d.R;
    f32x4 acc[4];
    tile.logits(row_ok ? text_row_ptr(q, b, g, r, d, D) : nullptr, lane, acc);
    const int t = row_ok ? r / d.G : -1;
    float x[16];
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = kb * 4 + e;
        const int key = key0 + kb * 16 + 4 * g4 + e;
        // visible: a kept visual key, or a text key at or before this row's token
        const bool ok = ((vis >> i) & 1u) || (key >= d.V_full && key < d.S && key - d.V_full <= t);
        x[i] = ok ? acc[kb][e] * d.scale_log2 : -INFINITY;
        mx = fmaxf(mx, x[i]);
      }
    mx = wave_max_xor(mx, 16);
    mx = wave_max_xor(mx, 32);
    float z = 0.f;
    if (mx != -INFINITY) {
#pragma unroll
      for (int i = 0; i < 16; ++i) z += exp2f(x[i] - mx);
    }
    z += __shfl_xor(z, 16, kWave);
    z += __shfl_xor(z, 32, kWave);
    if (g4 == 0 && row_ok)
      rowpart[(((size_t)b * d.Hkv + g) * d.n_kt + kt) * d.R + r] = make_float2(mx, z);
  }
}

// ---------------------------------------------------------------- merge

__global__ void __launch_bounds__(256)
score_rowmerge_kernel(int rows_total, int R, int n_kt, const float2* __restrict__ rowpart,
                      float2* __restrict__ rowstat) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows_total) return;
  const int bg = idx / R, r = idx - bg * R;
  const float2* p = rowpart + (size_t)bg * n_kt * R + r;
  float m = -INFINITY;
  for (int kt = 0; kt < n_kt; ++kt) m = fmaxf(m, p[(size_t)kt * R].x);
  float z = 0.f;
  for (int kt = 0; kt < n_kt; ++kt) {
    const float2 v = p[(size_t)kt * R];
    if (v.x != -INFINITY) z += v.y * exp2f(v.x - m);
  }
  rowstat[idx] = make_float2(m, 1.0f / z);
}

// ---------------------------------------------------------------- sweep 2

template <int DT, int D>
__global__ void __launch_bounds__(256)
score_colmass_kernel(ScoreDims d, const void* __restrict__ qv, const void* __restrict__ kv,
                     const uint8_t* __restrict__ token_keep, const float2* __restrict__ rowstat,
                     float* __restrict__ colpart) {
  using Tile = typename TileOf<DT, D>::T;
  using E = typename TileOf<DT, D>::E;
  const E* q = static_cast<const E*>(qv);
  const E* k = static_cast<const E*>(kv);
  const int vt = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, g4 = lane >> 4;
  const int key0 = vt * KT;
  const int nvalid = min(KT, d.V_full - key0);
  const uint8_t* keep_row = token_keep ? token_keep + (size_t)b * d.S : nullptr;
  float* out = colpart + ((size_t)b * d.Hkv + g) * d.V_full + key0;

  // A tile whose keys all belong to dropped views contributes nothing.
  bool any = false;
  if (threadIdx.x < nvalid) any = keep_row == nullptr || keep_row[key0 + threadIdx.x];
  if (!__syncthreads_or(any)) {
    if (threadIdx.x < nvalid) out[threadIdx.x] = 0.f;
    return;
  }

  Tile tile;
  tile.load_keys(k + (((size_t)b * d.S + key0) * d.Hkv + g) * D, (size_t)d.Hkv * D, nvalid, lane);
  const uint32_t vis = kept_visual_mask(keep_row, key0, d.V_full, lane);
  const float2* rs = rowstat + ((size_t)b * d.Hkv + g) * d.R;

  float col[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) col[i] = 0.f;
  const int nchunks = (d.R + 15) / 16;
  for (int ch = wave; ch < nchunks; ch += kScoreWaves) {
    const int r = ch * 16 + c;
    const bool row_ok = r < d.R;
    f32x4 acc[4];
    tile.logits(row_ok ? text_row_ptr(q, b, g, r, d, D) : nullptr, lane, acc);
    const float2 st = row_ok ? rs[r] : make_float2(0.f, 0.f);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = kb * 4 + e;
        // every text row sees every kept visual key
        if (row_ok && ((vis >> i) & 1u)) col[i] += exp2f(acc[kb][e] * d.scale_log2 - st.x) * st.y;
      }
  }
  // sum over the 16 rows of the lane's group (lanes sharing lane/16), fixed tree
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    float v = col[i];
    v += __shfl_xor(v, 1, kWave);
    v += __shfl_xor(v, 2, kWave);
    v += __shfl_xor(v, 4, kWave);
    v += __shfl_xor(v, 8, kWave);
    col[i] = v;
  }
  __shared__ float red[kScoreWaves][KT];
  if (c == 0) {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) red[wave][kb * 16 + 4 * g4 + e] = col[kb * 4 + e];
  }
  __syncthreads();
  if (threadIdx.x < nvalid) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kScoreWaves; ++w) s += red[w][threadIdx.x];
    out[threadIdx.x] = s;
  }
}

// ---------------------------------------------------------------- top-k + compaction

__device__ __forceinline__ uint32_t order_key(float s) {
  // monotone map fp32 -> uint32: larger float, larger key
  const uint32_t u = __float_as_uint(s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Visual tokens kept at compression ratio r: floor(r*V + 1e-6) in IEEE double
// without contraction, capped at V.
__device__ __forceinline__ int keep_count(double r, int V) {
  const double x = __dadd_rn(__dmul_rn(r, (double)V), 1e-6);
  const int k = (int)floor(x);
  return k < V ? k : V;
}

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;

// Block-wide exclusive scan of one int per thread; returns the exclusive
// prefix and writes the block total to *total.
__device__ __forceinline__ int block_exclusive_scan(int v, int* wsum, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off, kWave);
    if (lane >= off) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < kTopkWaves; ++w) {
      const int t = wsum[w];
      wsum[w] = run;
      run += t;
    }
    wsum[kTopkWaves] = run;
  }
  __syncthreads();
  const int excl = wsum[wave] + x - v;
  *total = wsum[kTopkWaves];
  __syncthreads();
  return excl;
}

__device__ __forceinline__ int block_count_kept(const uint8_t* row, int n, int* wsum) {
  int c = 0;
  for (int j = threadIdx.x; j < n; j += kTopkThreads) c += row[j] != 0;
  int total;
  block_exclusive_scan(c, wsum, &total);
  return total;
}

__global__ void __launch_bounds__(kTopkThreads)
topk_compact_kernel(int S, int V_full, int Hkv, float count, double keep_ratio,
                    const float* __restrict__ colpart, const uint8_t* __restrict__ token_keep,
                    float* __restrict__ scores, int32_t* __restrict__ kept_index,
                    int32_t* __restrict__ cu_seqlens) {
  __shared__ uint32_t keys[LITEVLM_MAX_VISUAL];
  __shared__ int hist[256];
  __shared__ int wsum[kTopkWaves + 1];
  __shared__ int sel_digit, sel_above;
  const int b = blockIdx.x;
  const int T = S - V_full;
  const int tid = threadIdx.x;

  // Compacted offsets: every sample's length is k_b + T with k_b from its own
  // kept-visual count, so the prefix is recomputed here from token_keep.
  int cu_b = 0, V_b = V_full;
  for (int bb = 0; bb <= b; ++bb) {
    const int Vbb = token_keep ? block_count_kept(token_keep + (size_t)bb * S, V_full, wsum) : V_full;
    if (bb < b) cu_b += keep_count(keep_ratio, Vbb) + T;
    else V_b = Vbb;
  }
  const int kb_ = keep_count(keep_ratio, V_b);

  // Scores: fixed-order sum over KV groups, then the mean over Hq*T rows.
  const uint8_t* keep_row = token_keep ? token_keep + (size_t)b * S : nullptr;
  for (int j = tid; j < V_full; j += kTopkThreads) {
    float s = -INFINITY;
    if (keep_row == nullptr || keep_row[j]) {
      float acc = 0.f;
      for (int g = 0; g < Hkv; ++g) acc += colpart[((size_t)b * Hkv + g) * V_full + j];
      s = acc / count;
    }
    scores[(size_t)b * V_full + j] = s;
    keys[j] = order_key(s);
  }
  __syncthreads();

  // Radix select of the kb_-th largest key, 8 bits at a time from the top.
  uint32_t prefix = 0, pmask = 0;
  int krem = kb_;
  if (kb_ > 0) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      if (tid < 256) hist[tid] = 0;
      __syncthreads();
      for (int j = tid; j < V_full; j += kTopkThreads) {
        const uint32_t kk = keys[j];
        if ((kk & pmask) == prefix) atomicAdd(&hist[(kk >> shift) & 255u], 1);
      }
      __syncthreads();
      if (tid < 64) {
        // lane l owns bins 4l..4l+3; suffix sums over lanes find the bin that
        // holds the krem-th largest candidate
        const int l = tid;
        const int c0 = hist[4 * l], c1 = hist[4 * l + 1], c2 = hist[4 * l + 2], c3 = hist[4 * l + 3];
        int suf = c0 + c1 + c2 + c3;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const int y = __shfl_down(suf, off, kWave);
          if (l + off < 64) suf += y;
        }
        int above = __shfl_down(suf, 1, kWave);  // candidates in bins of lanes > l
        if (l == 63) above = 0;
        if (above < krem && suf >= krem) {
          // walk this lane's bins from the top; a = candidates in higher bins
          int a = above, dsel;
          if (a + c3 >= krem) {
            dsel = 4 * l + 3;
          } else if ((a += c3) + c2 >= krem) {
            dsel = 4 * l + 2;
          } else if ((a += c2) + c1 >= krem) {
            dsel = 4 * l + 1;
          } else {
            a += c1;
            dsel = 4 * l;
          }
          sel_digit = dsel;
          sel_above = a;
        }
      }
      __syncthreads();
      prefix |= ((uint32_t)sel_digit) << shift;
      pmask |= 0xFFu << shift;
      krem -= sel_above;
      __syncthreads();
    }
  }
  // prefix is now the kb_-th largest key; take every larger key plus the first
  // krem equal keys in position order.
  const uint32_t thr = prefix;
  const int per = (V_full + kTopkThreads - 1) / kTopkThreads;
  const int j0 = min(V_full, tid * per), j1 = min(V_full, j0 + per);
  int neq = 0;
  if (kb_ > 0)
    for (int j = j0; j < j1; ++j) neq += keys[j] == thr;
  int tot;
  int eq_before = block_exclusive_scan(neq, wsum, &tot);
  int nsel = 0;
  if (kb_ > 0) {
    int eqr = eq_before;
    for (int j = j0; j < j1; ++j) {
      const uint32_t kk = keys[j];
      if (kk > thr) ++nsel;
      else if (kk == thr) { nsel += eqr < krem; ++eqr; }
    }
  }
  int sel_before = block_exclusive_scan(nsel, wsum, &tot);
  int32_t* out = kept_index + cu_b;
  if (kb_ > 0) {
    int eqr = eq_before, pos = sel_before;
    for (int j = j0; j < j1; ++j) {
      const uint32_t kk = keys[j];
      bool take = false;
      if (kk > thr) take = true;
      else if (kk == thr) { take = eqr < krem; ++eqr; }
      if (take) out[pos++] = j;
    }
  }
  for (int t = tid; t < T; t += kTopkThreads) out[kb_ + t] = V_full + t;
  if (tid == 0) {
    cu_seqlens[b + 1] = cu_b + kb_ + T;
    if (b == 0) cu_seqlens[0] = 0;
  }
}

// ---------------------------------------------------------------- gather

__global__ void __launch_bounds__(256)
gather_rows_kernel(int B, int S, const int32_t* __restrict__ kept_index,
                   const int32_t* __restrict__ cu_seqlens, const uint4* __restrict__ q,
                   const uint4* __restrict__ k, const uint4* __restrict__ v, uint4* __restrict__ qc,
                   uint4* __restrict__ kc, uint4* __restrict__ vc, int qvec, int kvvec) {
  __shared__ int cu[LITEVLM_MAX_BATCH + 1];
  for (int i = threadIdx.x; i <= B; i += blockDim.x) cu[i] = cu_seqlens[i];
  __syncthreads();
  const int total = cu[B];
  for (int i = blockIdx.x; i < total; i += gridDim.x) {
    int lo = 0, hi = B - 1;  // last b with cu[b] <= i
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (cu[mid] <= i) lo = mid; else hi = mid - 1;
    }
    const size_t src = (size_t)lo * S + kept_index[i];
    if (qc)
      for (int c = threadIdx.x; c < qvec; c += blockDim.x) qc[(size_t)i * qvec + c] = q[src * qvec + c];
    if (kc)
      for (int c = threadIdx.x; c < kvvec; c += blockDim.x) kc[(size_t)i * kvvec + c] = k[src * kvvec + c];
    if (vc)
      for (int c = threadIdx.x; c < kvvec; c += blockDim.x) vc[(size_t)i * kvvec + c] = v[src * kvvec + c];
  }
}

// ---------------------------------------------------------------- host launch

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

ScoreWorkspace score_workspace_layout(int B, int S, int V_full, int Hq, int Hkv) {
  const int T = S - V_full;
  const size_t R = (size_t)(Hq / Hkv) * T;
  const size_t n_kt = (size_t)(S + KT - 1) / KT;
  ScoreWorkspace w;
  w.rowpart_off = 0;
  w.rowstat_off = align256(w.rowpart_off + sizeof(float2) * B * Hkv * n_kt * R);
  w.colpart_off = align256(w.rowstat_off + sizeof(float2) * B * Hkv * R);
  w.total = align256(w.colpart_off + sizeof(float) * B * Hkv * (size_t)V_full);
  return w;
}

template <int DT, int D>
static void launch_sweeps(const ScoreArgs& a, const ScoreDims& d, float2* rowpart, float2* rowstat,
                          float* colpart, hipStream_t stream) {
  hipLaunchKernelGGL((score_rowstats_kernel<DT, D>), dim3(d.n_kt, a.Hkv, a.B), dim3(256), 0, stream,
                     d, a.q, a.k, a.token_keep, rowpart);
  const int rows_total = a.B * a.Hkv * d.R;
  hipLaunchKernelGGL(score_rowmerge_kernel, dim3((rows_total + 255) / 256), dim3(256), 0, stream,
                     rows_total, d.R, d.n_kt, rowpart, rowstat);
  const int n_vt = (a.V_full + KT - 1) / KT;
  if (n_vt > 0)
    hipLaunchKernelGGL((score_colmass_kernel<DT, D>), dim3(n_vt, a.Hkv, a.B), dim3(256), 0, stream,
                       d, a.q, a.k, a.token_keep, rowstat, colpart);
}

hipError_t launch_token_score_topk(const ScoreArgs& a, hipStream_t stream) {
  const ScoreWorkspace w = score_workspace_layout(a.B, a.S, a.V_full, a.Hq, a.Hkv);
  char* ws = static_cast<char*>(a.workspace);
  float2* rowpart = reinterpret_cast<float2*>(ws + w.rowpart_off);
  float2* rowstat = reinterpret_cast<float2*>(ws + w.rowstat_off);
  float* colpart = reinterpret_cast<float*>(ws + w.colpart_off);
  ScoreDims d;
  d.S = a.S;
  d.V_full = a.V_full;
  d.T = a.S - a.V_full;
  d.Hq = a.Hq;
  d.Hkv = a.Hkv;
  d.G = a.Hq / a.Hkv;
  d.R = d.G * d.T;
  d.n_kt = (a.S + KT - 1) / KT;
  d.scale_log2 = a.logit_scale_log2;

#define LITEVLM_SWEEPS(DT)                                                         \
  (a.D == 128 ? launch_sweeps<DT, 128>(a, d, rowpart, rowstat, colpart, stream) \
              : launch_sweeps<DT, 64>(a, d, rowpart, rowstat, colpart, stream))
  if (a.dtype == LITEVLM_BF16) LITEVLM_SWEEPS(LITEVLM_BF16);
  else if (a.dtype == LITEVLM_FP8_E4M3) LITEVLM_SWEEPS(LITEVLM_FP8_E4M3);
  else LITEVLM_SWEEPS(LITEVLM_F32);
#undef LITEVLM_SWEEPS

  hipLaunchKernelGGL(topk_compact_kernel, dim3(a.B), dim3(kTopkThreads), 0, stream, a.S, a.V_full,
                     a.Hkv, (float)a.Hq * (float)d.T, a.keep_ratio, colpart, a.token_keep, a.scores,
                     a.kept_index, a.cu_seqlens);
  if (a.qc || a.kc || a.vc) {
    const int esz = a.dtype == LITEVLM_F32 ? 4 : (a.dtype == LITEVLM_BF16 ? 2 : 1);
    const int qvec = a.Hq * a.D * esz / 16, kvvec = a.Hkv * a.D * esz / 16;
    const int grid = min(a.B * a.S, 4096);
    hipLaunchKernelGGL(gather_rows_kernel, dim3(grid), dim3(256), 0, stream, a.B, a.S, a.kept_index,
                       a.cu_seqlens, static_cast<const uint4*>(a.q), static_cast<const uint4*>(a.k),
                       static_cast<const uint4*>(a.v), static_cast<uint4*>(a.qc),
                       static_cast<uint4*>(a.kc), static_cast<uint4*>(a.vc), qvec, kvvec);
  }
  return hipGetLastError();
}

}  // namespace litevlm
