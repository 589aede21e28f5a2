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
#include <algorithm>
#include <climits>

#include "common.hpp"
#include "launch.hpp"

namespace litevlm {

constexpr int KW = 32;             // keys per wave: 2 blocks of 16
constexpr int kScoreWaves = 4;
constexpr int KT = KW * kScoreWaves;  // keys per workgroup
static_assert(KT == kScoreKeyTile, "workspace layout and kernels disagree on the key tile");

// ---------------------------------------------------------------- logit tiles
// Each tile policy holds one wave's 32 keys of one KV head and produces, for
// the 16 query rows of a chunk staged in LDS,
//   acc[kb][e] = k(kb*16 + 4*(lane/16) + e) . q(lane % 16)   in fp32.

template <int D>
struct TileBf16 {
  static constexpr int KS = D / 32;  // k-steps of v_mfma_f32_16x16x32_bf16
  static constexpr int ROW_BYTES = D * 2;
  bf16x8 kreg[2][KS];

  __device__ __forceinline__ void load_keys(const uint16_t* kbase, size_t kstride, int nvalid,
                                            int lane) {
    const int c = lane & 15, g4 = lane >> 4;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int key = kb * 16 + c;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        kreg[kb][ks] = key < nvalid
            ? *reinterpret_cast<const bf16x8*>(kbase + key * kstride + ks * 32 + 8 * g4)
            : bf16x8{};
    }
  }

  // qrow: LDS address of this lane's query row (row lane % 16 of the chunk).
  __device__ __forceinline__ void logits(const uint8_t* qrow, int lane, f32x4 acc[2]) const {
    const int g4 = lane >> 4;
    bf16x8 qreg[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qreg[ks] = *reinterpret_cast<const bf16x8*>(qrow + (ks * 32 + 8 * g4) * 2);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
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
  static constexpr int ROW_BYTES = D;
  i32x8 kreg[2];

  __device__ __forceinline__ void load_keys(const uint8_t* kbase, size_t kstride, int nvalid,
                                            int lane) {
    const int c = lane & 15, g4 = lane >> 4;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int key = kb * 16 + c;
      kreg[kb] = (key < nvalid && 32 * g4 < D)
          ? *reinterpret_cast<const i32x8*>(kbase + key * kstride + 32 * g4)
          : i32x8{};
    }
  }

  __device__ __forceinline__ void logits(const uint8_t* qrow, int lane, f32x4 acc[2]) const {
    const int g4 = lane >> 4;
    i32x8 qreg = i32x8{};
    if (32 * g4 < D) {
      const i32x4 lo = *reinterpret_cast<const i32x4*>(qrow + 32 * g4);
      const i32x4 hi = *reinterpret_cast<const i32x4*>(qrow + 32 * g4 + 16);
      qreg = i32x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
      // format 0 = E4M3 for both operands; zero scale operands select the
      // unscaled instruction.
      acc[kb] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(kreg[kb], qreg, z, 0, 0, 0, 0, 0, 0);
    }
  }
};

template <int D>
struct TileF32 {
  // Plain fp32 FMAs; fp32 inputs are only used at small sizes. The lane's own
  // 8 keys are read from global memory, its query row from LDS.
  static constexpr int ROW_BYTES = D * 4;
  const float* kbase;
  size_t kstride;
  int nvalid;

  __device__ __forceinline__ void load_keys(const float* kb_, size_t ks_, int nv, int) {
    kbase = kb_;
    kstride = ks_;
    nvalid = nv;
  }

  __device__ __forceinline__ void logits(const uint8_t* qrow, int lane, f32x4 acc[2]) const {
    const int g4 = lane >> 4;
    const float* qf = reinterpret_cast<const float*>(qrow);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = kb * 16 + 4 * g4 + e;
        float s = 0.f;
        if (key < nvalid) {
          const float* kr = kbase + key * kstride;
          for (int d = 0; d < D; ++d) s = fmaf(qf[d], kr[d], s);
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
  int S, V_full, T, Hq, Hkv, G, R, n_kt, rs1, rs2;
  float scale_log2;
};

// Keep flags of the lane's 8 accumulator keys (bit kb*4+e): all 8 byte loads
// are issued from clamped addresses before any is used.
__device__ __forceinline__ uint32_t lane_keep_bits(const uint8_t* keep_row, int key0, int S, int lane) {
  if (keep_row == nullptr) return 0xFFu;
  const int g4 = lane >> 4;
  uint8_t f[8];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int e = 0; e < 4; ++e) f[kb * 4 + e] = keep_row[min(key0 + kb * 16 + 4 * g4 + e, S - 1)];
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) m |= (f[i] ? 1u : 0u) << i;
  return m;
}

// Bitmask over the lane's 8 accumulator keys (bit kb*4+e): key is visual and kept.
__device__ __forceinline__ uint32_t kept_visual_mask(const uint8_t* keep_row, int key0, int V_full,
                                                     int S, int lane) {
  const int g4 = lane >> 4;
  const uint32_t kf = lane_keep_bits(keep_row, key0, S, lane);
  uint32_t m = 0;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int i = kb * 4 + e;
      const int key = key0 + kb * 16 + 4 * g4 + e;
      if (key < V_full && ((kf >> i) & 1u)) m |= 1u << i;
    }
  return m;
}

// Byte address of text query row r of KV group g: query head g*G + r%G of text token r/G.
__device__ __forceinline__ const uint8_t* text_row(const uint8_t* q, int b, int g, int r,
                                                   const ScoreDims& d, int row_bytes) {
  const int t = r / d.G, hh = r - t * d.G;
  return q + (((size_t)b * d.S + d.V_full + t) * d.Hq + (size_t)g * d.G + hh) * row_bytes;
}

// Q rows of the workgroup, staged through LDS a block of up to kQBlockBytes
// at a time: every load of a block is issued before the first is waited on.
constexpr int kQBlockBytes = 70 * 1024;  // 16 chunks of 16 bf16 D=128 rows

template <int ROW_BYTES>
struct QBlock {
  static constexpr int VEC = ROW_BYTES / 16;     // 16-byte pieces per row
  static constexpr int STRIDE = ROW_BYTES + 16;  // padded LDS row
  static constexpr int CHUNKS = kQBlockBytes / (16 * STRIDE) > 0 ? kQBlockBytes / (16 * STRIDE) : 1;
  static constexpr int BYTES = CHUNKS * 16 * STRIDE;

  static constexpr int PPT = (CHUNKS * 16 * VEC + 255) / 256;  // pieces per thread

  // Stage chunks first, first+step, ... (at most CHUNKS of them, all < nchunks)
  // into lds; returns how many were staged. Loads use clamped, always-valid
  // addresses and are all issued before the first store.
  __device__ __forceinline__ static int stage(uint8_t* lds, const uint8_t* q, int b, int g, int first,
                                              int step, int nchunks, const ScoreDims& d) {
    const int n = min(CHUNKS, (nchunks - first + step - 1) / step);
    const int pieces = n * 16 * VEC;
    uint4 reg[PPT];
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
      const int v = min((int)threadIdx.x + 256 * j, pieces - 1);
      const int row = v / VEC, piece = v - row * VEC;  // row within the staged block
      const int r = min((first + (row >> 4) * step) * 16 + (row & 15), d.R - 1);
      reg[j] = *reinterpret_cast<const uint4*>(text_row(q, b, g, r, d, ROW_BYTES) + piece * 16);
    }
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
      const int v = threadIdx.x + 256 * j;
      const int row = v / VEC, piece = v - row * VEC;
      const int r = (first + (row >> 4) * step) * 16 + (row & 15);
      if (v < pieces)
        *reinterpret_cast<uint4*>(lds + row * STRIDE + piece * 16) =
            r < d.R ? reg[j] : make_uint4(0, 0, 0, 0);
    }
    return n;
  }
};

// ---------------------------------------------------------------- sweep 1
// grid (n_kt, Hkv, B*rs1). Wave w holds keys [kt*128 + 32w, +32). Every wave
// runs over the workgroup's row chunks (chunk = rs, rs + rs1, ...); the four
// waves' per-row (max, sum) are combined in LDS in wave order.

template <int DT, int D>
__global__ void __launch_bounds__(256)
score_rowstats_kernel(ScoreDims d, const void* __restrict__ qv, const void* __restrict__ kv,
                      const uint8_t* __restrict__ token_keep, float2* __restrict__ rowpart) {
  using Tile = typename TileOf<DT, D>::T;
  using E = typename TileOf<DT, D>::E;
  using QB = QBlock<Tile::ROW_BYTES>;
  __shared__ __attribute__((aligned(16))) uint8_t qlds[QB::BYTES];
  __shared__ float2 part[QB::CHUNKS][kScoreWaves][16];

  const uint8_t* q = static_cast<const uint8_t*>(qv);
  const E* k = static_cast<const E*>(kv);
  const int kt = blockIdx.x, g = blockIdx.y;
  const int b = blockIdx.z / d.rs1, rs = blockIdx.z - b * d.rs1;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c = lane & 15, g4 = lane >> 4;
  const int key0 = kt * KT + w * KW;
  const uint8_t* keep_row = token_keep ? token_keep + (size_t)b * d.S : nullptr;
  const int nchunks = (d.R + 15) / 16;
  float2* out = rowpart + (((size_t)b * d.Hkv + g) * d.n_kt + kt) * d.R;

  // A tile of dropped-view keys only (no text key) contributes (-inf, 0).
  bool any = false;
  if (tid < KT) {
    const int key = kt * KT + tid;
    any = key < d.S && (key >= d.V_full || keep_row == nullptr || keep_row[key]);
  }
  if (!__syncthreads_or(any)) {
    for (int ch = rs; ch < nchunks; ch += d.rs1)
      if (tid < 16 && ch * 16 + tid < d.R) out[ch * 16 + tid] = make_float2(-INFINITY, 0.f);
    return;
  }

  Tile tile;
  tile.load_keys(k + (((size_t)b * d.S + min(key0, d.S)) * d.Hkv + g) * D, (size_t)d.Hkv * D,
                 max(0, min(KW, d.S - key0)), lane);
  // Per accumulator key: visible to text token t iff t >= lim (kept visual
  // keys: -1; text key V_full+t': t'; dropped or past the end: never).
  int lim[8];
  bool need_mask = false;
  {
    const uint32_t vis = kept_visual_mask(keep_row, key0, d.V_full, d.S, lane);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = kb * 4 + e;
        const int key = key0 + kb * 16 + 4 * g4 + e;
        int l;
        if (key >= d.S) l = INT_MAX;
        else if (key >= d.V_full) l = key - d.V_full;
        else l = ((vis >> i) & 1u) ? -1 : INT_MAX;
        lim[i] = l;
        need_mask |= l != -1;
      }
  }
  need_mask = __any(need_mask);
  const float sc = d.scale_log2;

  for (int first = rs; first < nchunks; first += d.rs1 * QB::CHUNKS) {
    const int n = QB::stage(qlds, q, b, g, first, d.rs1, nchunks, d);
    __syncthreads();
    for (int i = 0; i < n; ++i) {
      const int r = (first + i * d.rs1) * 16 + c;
      f32x4 acc[2];
      tile.logits(qlds + (i * 16 + c) * QB::STRIDE, lane, acc);
      float x[8];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) x[kb * 4 + e] = acc[kb][e];
      if (need_mask) {
        const int t = r < d.R ? r / d.G : -1;
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = t >= lim[j] ? x[j] : -INFINITY;
      }
      // raw logits: the scale is positive, so the max commutes with it
      float mx = x[0];
#pragma unroll
      for (int j = 1; j < 8; ++j) mx = fmaxf(mx, x[j]);
      mx = max_xor32(max_xor16(mx));
      float z = 0.f;
      if (mx != -INFINITY) {
        const float ms = -mx * sc;
#pragma unroll
        for (int j = 0; j < 8; ++j) z += __builtin_amdgcn_exp2f(fmaf(x[j], sc, ms));
      }
      z = sum_xor32(sum_xor16(z));
      if (g4 == 0) part[i][w][c] = make_float2(mx == -INFINITY ? -INFINITY : mx * sc, z);
    }
    __syncthreads();
    // combine the four waves per row, in wave order
    for (int v = tid; v < n * 16; v += 256) {
      const int i = v >> 4, rr = v & 15;
      const int r = (first + i * d.rs1) * 16 + rr;
      if (r < d.R) {
        float m = -INFINITY;
#pragma unroll
        for (int ww = 0; ww < kScoreWaves; ++ww) m = fmaxf(m, part[i][ww][rr].x);
        float zz = 0.f;
#pragma unroll
        for (int ww = 0; ww < kScoreWaves; ++ww) {
          const float2 p = part[i][ww][rr];
          if (p.x != -INFINITY) zz += p.y * exp2f(p.x - m);
        }
        out[r] = make_float2(m, zz);
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------- merge
// One row per (thread % 64), the key tiles split over 4 thread slices and
// combined in slice order.

__global__ void __launch_bounds__(256)
score_rowmerge_kernel(int rows_total, int R, int n_kt, const float2* __restrict__ rowpart,
                      float2* __restrict__ rowstat) {
  __shared__ float red[4][64];
  const int tid = threadIdx.x, slot = tid & 63, slice = tid >> 6;
  const int idx = blockIdx.x * 64 + slot;
  const bool ok = idx < rows_total;
  const int bg = ok ? idx / R : 0, r = ok ? idx - bg * R : 0;
  const float2* p = rowpart + (size_t)bg * n_kt * R + r;
  float m = -INFINITY;
  if (ok) {
#pragma unroll 4
    for (int kt = slice; kt < n_kt; kt += 4) m = fmaxf(m, p[(size_t)kt * R].x);
  }
  red[slice][slot] = m;
  __syncthreads();
  m = fmaxf(fmaxf(red[0][slot], red[1][slot]), fmaxf(red[2][slot], red[3][slot]));
  __syncthreads();
  float z = 0.f;
  if (ok) {
#pragma unroll 4
    for (int kt = slice; kt < n_kt; kt += 4) {
      const float2 v = p[(size_t)kt * R];
      if (v.x != -INFINITY) z += v.y * exp2f(v.x - m);
    }
  }
  red[slice][slot] = z;
  __syncthreads();
  if (slice == 0 && ok) {
    const float zt = ((red[0][slot] + red[1][slot]) + red[2][slot]) + red[3][slot];
    rowstat[idx] = make_float2(m, 1.0f / zt);
  }
}

// ---------------------------------------------------------------- sweep 2
// grid (n_vt, Hkv, B*rs2) over visual key tiles. Each wave owns 32 keys and
// accumulates exp2(logit - m)/Z over the workgroup's rows per lane, then sums
// the 16 rows of a lane group by DPP. Output: colpart[b][g][rs][V_full].

template <int DT, int D>
__global__ void __launch_bounds__(256)
score_colmass_kernel(ScoreDims d, const void* __restrict__ qv, const void* __restrict__ kv,
                     const uint8_t* __restrict__ token_keep, const float2* __restrict__ rowstat,
                     float* __restrict__ colpart) {
  using Tile = typename TileOf<DT, D>::T;
  using E = typename TileOf<DT, D>::E;
  using QB = QBlock<Tile::ROW_BYTES>;
  __shared__ __attribute__((aligned(16))) uint8_t qlds[QB::BYTES];
  __shared__ float2 rs_lds[QB::CHUNKS * 16];

  const uint8_t* q = static_cast<const uint8_t*>(qv);
  const E* k = static_cast<const E*>(kv);
  const int vt = blockIdx.x, g = blockIdx.y;
  const int b = blockIdx.z / d.rs2, rs = blockIdx.z - b * d.rs2;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c = lane & 15, g4 = lane >> 4;
  const int key0 = vt * KT + w * KW;
  const uint8_t* keep_row = token_keep ? token_keep + (size_t)b * d.S : nullptr;
  float* out = colpart + (((size_t)b * d.Hkv + g) * d.rs2 + rs) * d.V_full;
  const int nchunks = (d.R + 15) / 16;

  bool any = false;
  if (tid < KT) {
    const int key = vt * KT + tid;
    any = key < d.V_full && (keep_row == nullptr || keep_row[key]);
  }
  if (!__syncthreads_or(any)) {
    if (tid < KT && vt * KT + tid < d.V_full) out[vt * KT + tid] = 0.f;
    return;
  }

  Tile tile;
  tile.load_keys(k + (((size_t)b * d.S + min(key0, d.V_full)) * d.Hkv + g) * D, (size_t)d.Hkv * D,
                 max(0, min(KW, d.V_full - key0)), lane);
  const uint32_t vis = kept_visual_mask(keep_row, key0, d.V_full, d.S, lane);
  const float2* rstat = rowstat + ((size_t)b * d.Hkv + g) * d.R;
  const float sc = d.scale_log2;

  float col[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) col[i] = 0.f;
  for (int first = rs; first < nchunks; first += d.rs2 * QB::CHUNKS) {
    const int n = QB::stage(qlds, q, b, g, first, d.rs2, nchunks, d);
    for (int v = tid; v < n * 16; v += 256) {
      const int r = (first + (v >> 4) * d.rs2) * 16 + (v & 15);
      // rows past R get m = +inf so that their terms vanish
      rs_lds[v] = r < d.R ? rstat[r] : make_float2(INFINITY, 0.f);
    }
    __syncthreads();
    for (int i = 0; i < n; ++i) {
      const float2 rsv = rs_lds[i * 16 + c];
      f32x4 acc[2];
      tile.logits(qlds + (i * 16 + c) * QB::STRIDE, lane, acc);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          col[kb * 4 + e] += __builtin_amdgcn_exp2f(fmaf(acc[kb][e], sc, -rsv.x)) * rsv.y;
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) col[i] = row16_sum(col[i]);
  if (c == 0) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = key0 + kb * 16 + 4 * g4 + e;
        // dropped keys were summed over too; their column is forced to 0
        if (key < d.V_full) out[key] = ((vis >> (kb * 4 + e)) & 1u) ? col[kb * 4 + e] : 0.f;
      }
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

__device__ __forceinline__ int wave_sum_int(int v) {
  float f;  // exact: counts stay far below 2^24
  f = (float)v;
  f = row16_sum(f);
  f = sum_xor32(sum_xor16(f));
  return (int)f;
}

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
  if (threadIdx.x < 64) {
    // scan of the 16 wave totals in one wave
    const int l = threadIdx.x;
    const int t = l < kTopkWaves ? wsum[l] : 0;
    int y = t;
#pragma unroll
    for (int off = 1; off < kTopkWaves; off <<= 1) {
      const int u = __shfl_up(y, off, kWave);
      if (l >= off) y += u;
    }
    if (l < kTopkWaves) wsum[kTopkWaves + 1 + l] = y - t;
    if (l == kTopkWaves - 1) wsum[kTopkWaves] = y;
  }
  __syncthreads();
  const int excl = wsum[kTopkWaves + 1 + wave] + x - v;
  *total = wsum[kTopkWaves];
  __syncthreads();
  return excl;
}

__device__ __forceinline__ int block_sum(int v, int* wsum) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int s = wave_sum_int(v);
  if (lane == 0) wsum[wave] = s;
  __syncthreads();
  int t = 0;
#pragma unroll
  for (int w = 0; w < kTopkWaves; ++w) t += wsum[w];
  __syncthreads();
  return t;
}

// One workgroup per sample: V_b and the compacted offset, scores from the
// column-mass partials, radix select of the k_b-th largest order key, then
// the stable compaction.
__global__ void __launch_bounds__(kTopkThreads)
topk_compact_kernel(int S, int V_full, int Hkv, int rs2, float count, double keep_ratio,
                    const float* __restrict__ colpart, const uint8_t* __restrict__ token_keep,
                    float* __restrict__ scores, int32_t* __restrict__ kept_index,
                    int32_t* __restrict__ cu_seqlens) {
  __shared__ uint32_t keys[LITEVLM_MAX_VISUAL];
  __shared__ int hist[kTopkWaves][257];
  __shared__ int tot[256];
  __shared__ int wsum[2 * kTopkWaves + 2];
  __shared__ uint32_t red_u[2][kTopkWaves];
  __shared__ int sel_digit, sel_above;
  const int b = blockIdx.x;
  const int T = S - V_full;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  // Compacted offsets: every sample's length is k_b + T with k_b from its own
  // kept-visual count, so the prefix is recomputed here from token_keep.
  int cu_b = 0, V_b = V_full;
  for (int bb = 0; bb <= b; ++bb) {
    int Vbb = V_full;
    if (token_keep) {
      int cnt = 0;
      const uint8_t* row = token_keep + (size_t)bb * S;
      if ((reinterpret_cast<uintptr_t>(row) & 15) == 0) {
        // 16 flags (0/1 bytes) per load, summed with a byte-wise multiply
        const uint4* r4 = reinterpret_cast<const uint4*>(row);
        for (int j = tid; j < V_full / 16; j += kTopkThreads) {
          const uint4 u = r4[j];
          cnt += (int)((((u.x & 0x01010101u) * 0x01010101u) >> 24) + (((u.y & 0x01010101u) * 0x01010101u) >> 24) +
                       (((u.z & 0x01010101u) * 0x01010101u) >> 24) + (((u.w & 0x01010101u) * 0x01010101u) >> 24));
        }
        for (int j = (V_full & ~15) + tid; j < V_full; j += kTopkThreads) cnt += row[j] != 0;
      } else {
        for (int j = tid; j < V_full; j += kTopkThreads) cnt += row[j] != 0;
      }
      Vbb = block_sum(cnt, wsum);
    }
    if (bb < b) cu_b += keep_count(keep_ratio, Vbb) + T;
    else V_b = Vbb;
  }
  const int kb_ = keep_count(keep_ratio, V_b);

  // Scores: fixed-order sum over KV groups and row splits, then the mean over
  // Hq*T rows. Kept keys are >= 0x80000000; dropped tokens get key 0. Each
  // thread takes 4 consecutive keys so that all partial loads are in flight.
  const uint8_t* keep_row = token_keep ? token_keep + (size_t)b * S : nullptr;
  const float* cp = colpart + (size_t)b * Hkv * rs2 * V_full;
  const int nparts = Hkv * rs2;
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
  for (int j4 = tid * 4; j4 < V_full; j4 += kTopkThreads * 4) {
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    const int nk = min(4, V_full - j4);
    if (nk == 4 && (V_full & 3) == 0) {
      int i = 0;
      for (; i + 4 <= nparts; i += 4) {
        float4 p[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) p[u] = *reinterpret_cast<const float4*>(cp + (size_t)(i + u) * V_full + j4);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          acc[0] += p[u].x; acc[1] += p[u].y; acc[2] += p[u].z; acc[3] += p[u].w;
        }
      }
      for (; i < nparts; ++i) {
        const float4 p = *reinterpret_cast<const float4*>(cp + (size_t)i * V_full + j4);
        acc[0] += p.x; acc[1] += p.y; acc[2] += p.z; acc[3] += p.w;
      }
    } else {
      for (int i = 0; i < nparts; ++i)
        for (int u = 0; u < nk; ++u) acc[u] += cp[(size_t)i * V_full + j4 + u];
    }
    for (int u = 0; u < nk; ++u) {
      const int j = j4 + u;
      float s = -INFINITY;
      uint32_t key = 0u;
      if (keep_row == nullptr || keep_row[j]) {
        s = acc[u] / count;
        key = order_key(s);
        kmin = min(kmin, key);
        kmax = max(kmax, key);
      }
      scores[(size_t)b * V_full + j] = s;
      keys[j] = key;
    }
  }
  // block min / max of the kept keys
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, off, kWave));
    kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, off, kWave));
  }
  if (lane == 0) {
    red_u[0][wave] = kmin;
    red_u[1][wave] = kmax;
  }
  __syncthreads();
  kmin = 0xFFFFFFFFu;
  kmax = 0u;
#pragma unroll
  for (int w = 0; w < kTopkWaves; ++w) {
    kmin = min(kmin, red_u[0][w]);
    kmax = max(kmax, red_u[1][w]);
  }

  // Radix select of the kb_-th largest key. Bits above the highest bit where
  // kmin and kmax differ are common to every kept key and are skipped.
  const uint32_t diff = kmin ^ kmax;
  int bits_left = diff ? 32 - __clz((int)diff) : 0;
  uint32_t pmask = bits_left == 32 ? 0u : ~((1u << bits_left) - 1u);
  uint32_t prefix = kmax & pmask;
  int krem = kb_;
  if (kb_ > 0) {
    while (bits_left > 0) {
      const int width = bits_left < 8 ? bits_left : 8;
      const int shift = bits_left - width;
      const uint32_t dmask = (1u << width) - 1u;
      for (int i = tid; i < kTopkWaves * 257; i += kTopkThreads) (&hist[0][0])[i] = 0;
      __syncthreads();
      for (int j0 = 0; j0 < V_full; j0 += kTopkThreads) {
        const int j = j0 + tid;
        const uint32_t kk = j < V_full ? keys[j] : 0u;
        const bool cand = j < V_full && kk != 0u && (kk & pmask) == prefix;
        const int digit = (int)((kk >> shift) & dmask);
        // wave-aggregated count of the most common case: lanes sharing the
        // first candidate lane's digit add with one atomic
        const uint64_t active = __ballot(cand);
        if (active) {
          const int leader = __ffsll((unsigned long long)active) - 1;
          const int d0 = __builtin_amdgcn_readlane(digit, leader);
          const uint64_t same = __ballot(cand && digit == d0);
          if (lane == leader) atomicAdd(&hist[wave][d0], __popcll(same));
          if (cand && digit != d0) atomicAdd(&hist[wave][digit], 1);
        }
      }
      __syncthreads();
      if (tid < 256) {
        int t = 0;
#pragma unroll
        for (int w = 0; w < kTopkWaves; ++w) t += hist[w][tid];
        tot[tid] = t;
      }
      __syncthreads();
      if (tid < 64) {
        // lane l owns bins 4l..4l+3; suffix sums over lanes find the bin that
        // holds the krem-th largest candidate
        const int l = tid;
        const int c0 = tot[4 * l], c1 = tot[4 * l + 1], c2 = tot[4 * l + 2], c3 = tot[4 * l + 3];
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
      pmask |= dmask << shift;
      krem -= sel_above;
      bits_left -= width;
      __syncthreads();
    }
  }
  // prefix is now the kb_-th largest key; take every larger key plus the first
  // krem equal keys in position order.
  const uint32_t thr = prefix;
  const int per = (V_full + kTopkThreads - 1) / kTopkThreads;
  const int j0 = min(V_full, tid * per), j1 = min(V_full, j0 + per);
  int neq = 0, ngt = 0;
  if (kb_ > 0)
    for (int j = j0; j < j1; ++j) {
      const uint32_t kk = keys[j];
      neq += kk == thr;
      ngt += kk > thr;
    }
  int tot_eq;
  const int eq_before = block_exclusive_scan(neq, wsum, &tot_eq);
  const int nsel = ngt + max(0, min(neq, krem - eq_before));
  int tot_sel;
  const int sel_before = block_exclusive_scan(nsel, wsum, &tot_sel);
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
// Each workgroup copies kGatherRows packed rows per iteration: the source
// rows are resolved first, then every 16-byte load of the group is issued
// (from clamped, always-valid addresses) before the predicated stores.

constexpr int kGatherRows = 4;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int QPT, int KPT>
__global__ void __launch_bounds__(256)
gather_rows_kernel(int B, int S, const int32_t* __restrict__ kept_index,
                   const int32_t* __restrict__ cu_seqlens, const u32x4* __restrict__ q,
                   const u32x4* __restrict__ k, const u32x4* __restrict__ v, u32x4* __restrict__ qc,
                   u32x4* __restrict__ kc, u32x4* __restrict__ vc, int qvec, int kvvec) {
  __shared__ int cu[LITEVLM_MAX_BATCH + 1];
  for (int i = threadIdx.x; i <= B; i += blockDim.x) cu[i] = cu_seqlens[i];
  __syncthreads();
  const int total = cu[B];
  const int tid = threadIdx.x;
  for (int base = blockIdx.x * kGatherRows; base < total; base += gridDim.x * kGatherRows) {
    size_t src[kGatherRows];
#pragma unroll
    for (int r = 0; r < kGatherRows; ++r) {
      const int i = min(base + r, total - 1);
      // last b with cu[b] <= i, by a fixed 8-step search (B <= 256)
      int lo = 0;
#pragma unroll
      for (int step = 128; step >= 1; step >>= 1)
        if (lo + step <= B - 1 && cu[lo + step] <= i) lo += step;
      src[r] = (size_t)lo * S + kept_index[i];
    }
    u32x4 qv[kGatherRows * QPT], kv[kGatherRows * KPT], vv[kGatherRows * KPT];
#pragma unroll
    for (int r = 0; r < kGatherRows; ++r) {
      // kernel-uniform guards: an input is only read when its copy is requested
#pragma unroll
      for (int j = 0; j < QPT; ++j) {
        const int c = min(tid + 256 * j, qvec - 1);
        if (qc) qv[r * QPT + j] = q[src[r] * qvec + c];
      }
#pragma unroll
      for (int j = 0; j < KPT; ++j) {
        const int c = min(tid + 256 * j, kvvec - 1);
        if (kc) kv[r * KPT + j] = k[src[r] * kvvec + c];
        if (vc) vv[r * KPT + j] = v[src[r] * kvvec + c];
      }
    }
#pragma unroll
    for (int r = 0; r < kGatherRows; ++r) {
      const int i = base + r;
      const bool row_ok = i < total;
#pragma unroll
      for (int j = 0; j < QPT; ++j) {
        const int c = tid + 256 * j;
        if (qc && row_ok && c < qvec) qc[(size_t)i * qvec + c] = qv[r * QPT + j];
      }
#pragma unroll
      for (int j = 0; j < KPT; ++j) {
        const int c = tid + 256 * j;
        if (kc && row_ok && c < kvvec) kc[(size_t)i * kvvec + c] = kv[r * KPT + j];
        if (vc && row_ok && c < kvvec) vc[(size_t)i * kvvec + c] = vv[r * KPT + j];
      }
    }
  }
}

// ---------------------------------------------------------------- host launch

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

ScoreSplit score_split(int B, int S, int V_full, int Hq, int Hkv) {
  // Row chunks are split over workgroups until a sweep has ~2 workgroups per
  // CU (256 CUs); sweep 2 splits less since every split multiplies the
  // column partials top-k must read.
  ScoreSplit p;
  const int T = S - V_full;
  const int R = (Hq / Hkv) * T;
  p.n_kt = (S + KT - 1) / KT;
  p.n_vt = (V_full + KT - 1) / KT;
  p.nchunks = (R + 15) / 16;
  const long long w1 = (long long)p.n_kt * Hkv * B, w2 = (long long)p.n_vt * Hkv * B;
  p.rs1 = (int)std::min<long long>(p.nchunks, std::max<long long>(1, (512 + w1 - 1) / w1));
  p.rs2 = w2 == 0 ? 1 : (int)std::min<long long>(std::min(p.nchunks, 4),
                                                std::max<long long>(1, (256 + w2 - 1) / w2));
  return p;
}

ScoreWorkspace score_workspace_layout(int B, int S, int V_full, int Hq, int Hkv) {
  const ScoreSplit sp = score_split(B, S, V_full, Hq, Hkv);
  const size_t R = (size_t)(Hq / Hkv) * (S - V_full);
  ScoreWorkspace w;
  w.rowpart_off = 0;
  w.rowstat_off = align256(w.rowpart_off + sizeof(float2) * B * Hkv * (size_t)sp.n_kt * R);
  w.colpart_off = align256(w.rowstat_off + sizeof(float2) * B * Hkv * R);
  w.total = align256(w.colpart_off + sizeof(float) * B * Hkv * (size_t)sp.rs2 * V_full);
  return w;
}

template <int DT, int D>
static void launch_sweeps(const ScoreArgs& a, const ScoreDims& d, const ScoreSplit& sp,
                          float2* rowpart, float2* rowstat, float* colpart, hipStream_t stream) {
  hipLaunchKernelGGL((score_rowstats_kernel<DT, D>), dim3(sp.n_kt, a.Hkv, a.B * sp.rs1), dim3(256), 0,
                     stream, d, a.q, a.k, a.token_keep, rowpart);
  const int rows_total = a.B * a.Hkv * d.R;
  hipLaunchKernelGGL(score_rowmerge_kernel, dim3((rows_total + 63) / 64), dim3(256), 0, stream,
                     rows_total, d.R, d.n_kt, rowpart, rowstat);
  if (sp.n_vt > 0)
    hipLaunchKernelGGL((score_colmass_kernel<DT, D>), dim3(sp.n_vt, a.Hkv, a.B * sp.rs2), dim3(256), 0,
                       stream, d, a.q, a.k, a.token_keep, rowstat, colpart);
}

hipError_t launch_token_score_topk(const ScoreArgs& a, hipStream_t stream) {
  const ScoreWorkspace w = score_workspace_layout(a.B, a.S, a.V_full, a.Hq, a.Hkv);
  const ScoreSplit sp = score_split(a.B, a.S, a.V_full, a.Hq, a.Hkv);
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
  d.n_kt = sp.n_kt;
  d.rs1 = sp.rs1;
  d.rs2 = sp.rs2;
  d.scale_log2 = a.logit_scale_log2;

#define LITEVLM_SWEEPS(DT)                                                             \
  (a.D == 128 ? launch_sweeps<DT, 128>(a, d, sp, rowpart, rowstat, colpart, stream) \
              : launch_sweeps<DT, 64>(a, d, sp, rowpart, rowstat, colpart, stream))
  if (a.dtype == LITEVLM_BF16) LITEVLM_SWEEPS(LITEVLM_BF16);
  else if (a.dtype == LITEVLM_FP8_E4M3) LITEVLM_SWEEPS(LITEVLM_FP8_E4M3);
  else LITEVLM_SWEEPS(LITEVLM_F32);
#undef LITEVLM_SWEEPS

  hipLaunchKernelGGL(topk_compact_kernel, dim3(a.B), dim3(kTopkThreads), 0, stream, a.S, a.V_full,
                     a.Hkv, sp.rs2, (float)a.Hq * (float)d.T, a.keep_ratio, colpart, a.token_keep,
                     a.scores, a.kept_index, a.cu_seqlens);
  if (a.qc || a.kc || a.vc) {
    const int esz = a.dtype == LITEVLM_F32 ? 4 : (a.dtype == LITEVLM_BF16 ? 2 : 1);
    const int qvec = a.Hq * a.D * esz / 16, kvvec = a.Hkv * a.D * esz / 16;
    const int rows = a.B * a.S;
    const int grid = std::max(1, std::min(2048, (rows + kGatherRows - 1) / kGatherRows));
    // pieces per thread: Q rows up to 4096 x 16 B, K/V rows up to 1024 x 16 B
    auto launch = [&](auto kernel) {
      hipLaunchKernelGGL(kernel, dim3(grid), dim3(256), 0, stream, a.B, a.S, a.kept_index,
                         a.cu_seqlens, static_cast<const u32x4*>(a.q), static_cast<const u32x4*>(a.k),
                         static_cast<const u32x4*>(a.v), static_cast<u32x4*>(a.qc),
                         static_cast<u32x4*>(a.kc), static_cast<u32x4*>(a.vc), qvec, kvvec);
    };
    const int qpt = (qvec + 255) / 256, kpt = (kvvec + 255) / 256;
    if (qpt <= 1 && kpt <= 1) launch(gather_rows_kernel<1, 1>);
    else if (qpt <= 2 && kpt <= 1) launch(gather_rows_kernel<2, 1>);
    else if (qpt <= 4 && kpt <= 1) launch(gather_rows_kernel<4, 1>);
    else if (qpt <= 4 && kpt <= 2) launch(gather_rows_kernel<4, 2>);
    else if (qpt <= 8 && kpt <= 2) launch(gather_rows_kernel<8, 2>);
    else launch(gather_rows_kernel<16, 4>);
  }
  return hipGetLastError();
}

}  // namespace litevlm
