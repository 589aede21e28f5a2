// Text-guided visual-token scoring (Design section, Token Selection Module
// paragraph): the attention mass that the text rows of the first decoder layer
// put on each visual token, averaged over query heads and text rows.
//
// For KV group g the R = G*T text query rows (row r = t*G + hh is query head
// g*G+hh of text token t) attend causally over the patch-selected sequence.
// In original positions that is: kept visual keys (token_keep = 1) and text
// keys V_full+t' with t' <= t. Exact column mass needs each row's softmax
// normaliser first, so the work is two sweeps over K:
//   sweep 1  per (key split, row): max m and sum Z of exp2(logit) over the split
//   sweep 2  per row (merged at the start of each workgroup): m = max over
//            splits, Z = sum Z_split * exp2(m_split - m); then per visual key:
//            sum over rows of exp2(logit - m) / Z
// Both sweeps form logits on 32x32 MFMAs. Sweep 1 keeps 32 query rows per wave
// in registers and streams key tiles through LDS (a lane owns one query row of
// the transposed block, so its row statistics stay in the lane). Sweep 2 keeps
// 64 keys per wave in registers and streams query rows through LDS (a lane owns
// one key column, so its column mass accumulates in the lane). Every reduction
// runs in a fixed order, and the column partials of the workgroups are added
// as fixed-point integers, so results are deterministic.
#include <algorithm>
#include <cmath>
#include <type_traits>

#include "common.hpp"
#include "launch.hpp"
#include "viewsel.hpp"

namespace litevlm {

// sweep 1
constexpr int KB = 64;                      // keys per key tile
constexpr int kSweepWaves = 16;             // waves per sweep-1 workgroup, 32 query rows each
constexpr int kSweepThreads = 64 * kSweepWaves;
constexpr int RBLK = 32 * kSweepWaves;      // query rows per sweep-1 workgroup
constexpr int kMaxSplitTiles = 64;          // key tiles per split (one 64-bit live mask)
constexpr int kBalMaxBatch = kSweepWaves;   // balanced sweep-1 split: one wave per sample
constexpr int kBalWords = 4;                // ... and at most 256 key tiles per sample
constexpr int kLdsBytes = 160 * 1024;       // LDS of a workgroup (gfx950)
// sweep 2
constexpr int KW = 64;                      // keys per wave: 2 blocks of 32
constexpr int kColWaves = 4;                // waves per sweep-2 workgroup
constexpr int KT = KW * kColWaves;          // keys per sweep-2 workgroup
constexpr int CH = 32;                      // query rows per chunk

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Column sum of a visual key of a dropped view when the scoring takes the view
// selection itself: sweep 2 stores it (no sum reaches 2^62), so that the top-k
// reads the keep flags with the sums instead of evaluating the selection per key.
constexpr unsigned long long kDroppedCol = ~0ull;

// Work split of the sweeps (a function of the shape only, so that the
// workspace size is too).
struct ScoreSplit {
  int n_rb, n_kt, ns1;      // sweep 1: row blocks of RBLK rows, key tiles of KB keys, key splits
  int n_vt, nchunks, rs2;   // sweep 2: visual key tiles of KT keys, row chunks of CH rows, row splits
  int ns1_slots;            // sweep-1 partials per (sample, KV group, row): ns1, or 2*ns1 where a
                            // balanced split may give a sample more splits than ns1
};

struct ScoreDims {
  int B, S, V_full, T, Hq, Hkv, G, R;
  int tq0;  // the query rows are text tokens tq0 .. tq0 + T - 1 (the last T of them)
  // ns1: partials per (sample, KV group, row), the split count unless bal.
  // bal: sweep 1 splits each sample's live key tiles, ns1u splits per column
  // on average (the grid), at most ns1 for one sample.
  int n_rb, n_kt, ns1, n_vt, nchunks, rs2;
  int bal, ns1u;
  float scale_log2;
  float fx;  // fixed-point scale of the column sums (a power of two)
  // in-call patch selection (the kernels' VSEL instances): keep flags from the
  // view scores instead of a token mask
  ViewSel vs;
};

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier for LDS hand-over between the waves, with the waits
// spelled out: this wave's LDS reads have completed (its direct copies are
// waited for by the caller). The memory clobber keeps the compiler from moving
// LDS accesses across it; unlike __syncthreads it carries no fence, whose
// lowering here adds a wait for every copy in flight.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until at most n (0..7; larger n waits for 7) vector-memory operations
// of this wave are outstanding.
__device__ __forceinline__ void wait_vmcnt_upto(int n) {
  switch (n) {
    case 0: wait_vmcnt<0>(); break;
    case 1: wait_vmcnt<1>(); break;
    case 2: wait_vmcnt<2>(); break;
    case 3: wait_vmcnt<3>(); break;
    case 4: wait_vmcnt<4>(); break;
    case 5: wait_vmcnt<5>(); break;
    case 6: wait_vmcnt<6>(); break;
    default: wait_vmcnt<7>(); break;
  }
}

// Flat, XCD-aware work decode. Workgroup L runs on XCD L % 8; XCD x takes the
// contiguous column range [x*ncol/8, (x+1)*ncol/8), every column with all of
// its splits, so the query rows of a (sample, KV group) are read into one
// XCD's L2. Returns false for the padding workgroups of the grid.
__device__ __forceinline__ bool decode_column(int ncol, int nsplit, int& col, int& split) {
  const int L = blockIdx.x, x = L & 7, j = L >> 3;
  const int c0 = (int)(((long long)x * ncol) >> 3), c1 = (int)(((long long)(x + 1) * ncol) >> 3);
  if (j >= (c1 - c0) * nsplit) return false;
  const int cj = j / nsplit;
  col = c0 + cj;
  split = j - cj * nsplit;
  return true;
}

// (sample, KV group) pair at position i of an order that deals the pairs to
// the 8 XCDs round-robin: the XCD-contiguous column ranges then hold pairs x,
// x+8, x+16, ..., so every XCD gets a share of every sample.
__device__ __forceinline__ int pair_at(int i, int npair) {
  const int q = npair >> 3, m = npair & 7;
  if (i < m * (q + 1)) {
    const int r = i / (q + 1);
    return r + 8 * (i - r * (q + 1));
  }
  const int i2 = i - m * (q + 1), r = m + i2 / q;
  return r + 8 * (i2 - (r - m) * q);
}

// First key tile of split `split` of n tiles in ns splits: the first n % ns
// splits take one tile more, so the last split (text keys, masked) is never
// the long one.
__device__ __forceinline__ int split_begin(int split, int n, int ns) {
  const int base = n / ns, rem = n - base * ns;
  return split * base + min(split, rem);
}

template <int CTRL>
__device__ __forceinline__ int dpp_i(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, false);
}

// Balanced sweep-1 split over samples with unequal numbers of live key tiles
// (tiles holding a key that some row sees: a key of a kept view, or a text
// key), with the view selection inside the call.
//  1. Wave b evaluates sample b's view mask and marks its live tiles.
//  2. Wave 0 gives sample b ns_b = max(1, ceil(nl_b / tau)) splits per column
//     (nl_b live tiles), for the smallest tau in [1, 64] whose splits fit the
//     grid's B*ns1u per column, with at most ns1 for one sample, and takes the
//     workgroup's unit from the order (sample, KV group, row block, split),
//     each XCD a contiguous range of it.
//  3. Split s of a column takes the live tiles of ranks [a, a + ntl) (the
//     first nl_b % ns_b splits one more), and lane j of `list` returns the
//     j-th of them.
// LDS `tmp` (1 KB) is free for the workgroup on entry and again on return.
// Returns false for a workgroup without a unit; every thread returns the same.
struct BalUnit {
  int b, g, rb, split, ntl, ns;
  int list;
};

__device__ bool bal_unit(const ScoreDims& d, uint8_t* tmp, int w, int lane, BalUnit& u) {
  uint64_t* lm = reinterpret_cast<uint64_t*>(tmp);                      // [kBalMaxBatch][kBalWords]
  int* nl = reinterpret_cast<int*>(tmp + 8 * kBalMaxBatch * kBalWords);  // [kBalMaxBatch]
  int* res = nl + kBalMaxBatch;                                          // b, g, rb, split, ntl, ns, -, valid
  int* lst = res + 8;                                                    // [64]
  if (w < d.B) {
    const uint32_t vm = (uint32_t)view_keep_mask<kFusedViews>(view_load(d.vs.logit, d.vs.lexical, d.vs.N, w, lane),
                                                               d.vs.lexical != nullptr, d.vs.w, d.vs.tau, d.vs.N,
                                                               lane);
    int cnt = 0;
#pragma unroll
    for (int wd = 0; wd < kBalWords; ++wd) {
      const int t = 64 * wd + lane, k0 = KB * t, k1 = k0 + KB;
      uint32_t live = k1 > d.V_full ? 1u : 0u;  // holds a text key
#pragma unroll
      for (int v = 0; v < kFusedViews; ++v)  // bitwise, no branches: a kept view overlaps the tile
        live |= (v < d.vs.N ? 1u : 0u) & ((vm >> v) & 1u) & (d.vs.off[v] < k1 ? 1u : 0u) &
                (d.vs.off[v + 1] > k0 ? 1u : 0u);
      const uint64_t bits = __ballot((live & (t < d.n_kt ? 1u : 0u)) != 0u);
      cnt += __popcll(bits);
      if (lane == 0) lm[w * kBalWords + wd] = bits;
    }
    if (lane == 0) nl[w] = cnt;
  }
  __syncthreads();
  if (w == 0) {
    // lane b < B (all in the wave's first row of 16 lanes): sample b's live
    // tiles and splits per column; sums, maxima and prefixes over the samples
    // by row-of-16 DPP, read back with readlane (no LDS round trips)
    const int nlb = lane < d.B ? nl[lane] : 0;
    const int budget = d.B * d.ns1u;
    // ceil(n / t) for 0 <= n <= 256, 1 <= t <= 256: the float quotient is within
    // an ulp of the exact one, so its ceiling is off by at most one, corrected
    auto ceil_div = [](int n, int t) {
      int q = (int)ceilf(__fdividef((float)n, (float)t));
      q -= (q - 1) * t >= n ? 1 : 0;
      q += q * t < n ? 1 : 0;
      return q;
    };
    auto splits = [&](int tau) { return lane < d.B ? max(1, ceil_div(nlb, tau)) : 0; };
    auto samples_sum = [](int x) {
      x += dpp_i<0xB1>(x);   // quad_perm [1,0,3,2]
      x += dpp_i<0x4E>(x);   // quad_perm [2,3,0,1]
      x += dpp_i<0x141>(x);  // row_half_mirror
      x += dpp_i<0x140>(x);  // row_mirror
      return __builtin_amdgcn_readfirstlane(x);
    };
    auto samples_max = [](int x) {
      x = max(x, dpp_i<0xB1>(x));
      x = max(x, dpp_i<0x4E>(x));
      x = max(x, dpp_i<0x141>(x));
      x = max(x, dpp_i<0x140>(x));
      return __builtin_amdgcn_readfirstlane(x);
    };
    // tau >= ceil(nl_b / ns1) keeps every sample within ns1 splits; tau = 64
    // fits the budget, since ns1u >= ceil(n_kt / 64) >= ceil(nl_b / 64)
    int lo = samples_max(lane < d.B ? ceil_div(nlb, d.ns1) : 1);
    int hi = 64;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (samples_sum(splits(mid)) <= budget) hi = mid;
      else lo = mid + 1;
    }
    const int nsb = splits(lo);
    const int C = d.Hkv * d.n_rb;  // columns per sample
    // inclusive prefix of the units C*ns_b over the samples (row_shr 1, 2, 4, 8)
    int incl = C * nsb;
    incl += dpp_i<0x111>(incl);
    incl += dpp_i<0x112>(incl);
    incl += dpp_i<0x114>(incl);
    incl += dpp_i<0x118>(incl);
    const int total = __builtin_amdgcn_readlane(incl, 15);
    const int L = blockIdx.x, x = L & 7, j = L >> 3;
    const int u0 = (int)(((long long)x * total) >> 3), u1 = (int)(((long long)(x + 1) * total) >> 3);
    const bool valid = j < u1 - u0;
    const int unit = u0 + j;
    // sample b: the lane whose prefix range holds the unit
    const uint64_t hit = __ballot(valid && lane < d.B && unit < incl && unit >= incl - C * nsb);
    const int b = hit ? (int)__builtin_ctzll(hit) : 0;
    const int ns = __builtin_amdgcn_readlane(nsb, b), base = __builtin_amdgcn_readlane(incl, b) - C * ns;
    const int nlv = __builtin_amdgcn_readlane(nlb, b);
    const int r = unit - base, col = r / max(ns, 1), split = r - col * ns;
    const int a = split_begin(split, nlv, ns), ntl = split_begin(split + 1, nlv, ns) - a;
    if (lane == 0) {
      res[0] = b;
      res[1] = col / d.n_rb;
      res[2] = col - (col / d.n_rb) * d.n_rb;
      res[3] = split;
      res[4] = ntl;
      res[5] = ns;
      res[7] = valid && hit ? 1 : 0;
    }
    // the split's tiles: the live tile of rank a + i goes to entry i (ranks
    // from the lanes below in the same word plus the words before)
    lst[lane] = 0;
    int rank0 = 0;
#pragma unroll
    for (int wd = 0; wd < kBalWords; ++wd) {
      const uint64_t m = lm[b * kBalWords + wd];
      const int rank = rank0 + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
      if (((m >> lane) & 1ull) && rank >= a && rank < a + ntl) lst[rank - a] = 64 * wd + lane;
      rank0 += __popcll(m);
    }
  }
  __syncthreads();
  u.b = res[0];
  u.g = res[1];
  u.rb = res[2];
  u.split = res[3];
  u.ntl = res[4];
  u.ns = res[5];
  const bool valid = res[7] != 0;
  u.list = lst[lane];
  __syncthreads();  // tmp is read by every wave before the caller reuses it
  return valid;
}

// ---------------------------------------------------------------- sweep-1 logit tiles
// A sweep-1 workgroup keeps 32 query rows per wave in registers and streams
// 64-key tiles of K through LDS (row-major, 16-byte pieces XOR-swizzled per
// row, copied global -> LDS directly). A tile policy forms the transposed
// 64 x 32 block of a wave on 32x32 MFMAs, s[nb][r] = S^T[key 32*nb +
// acc_row(r)][row lane % 32] (a lane owns one query row), with acc_row(r) =
// 8*(r/4) + 4*(lane/32) + r%4, the 32x32 accumulator layout.

__device__ __forceinline__ int acc_row(int r, int hl) { return 8 * (r >> 2) + 4 * hl + (r & 3); }

// Query row r (0 <= r < R) of KV group g is query head g*G + r%G of text token r/G.
// Rows past R are read as row R-1 (their results are never used).
struct QRows {
  const uint8_t* base;  // text token 0, query head g*G of this sample
  int G, Hq, RB, R;
  __device__ __forceinline__ const uint8_t* row(int r) const {
    r = min(r, R - 1);
    const int t = r / G;
    return base + ((size_t)t * Hq + (r - t * G)) * RB;
  }
};

template <int D>
struct RowTileBf16 {
  static constexpr int RB = D * 2;        // bytes per row
  static constexpr int NP = RB / 16;      // 16-byte pieces per row
  static constexpr int KS = D / 16;       // k-steps of v_mfma_f32_32x32x16_bf16
  static constexpr int TILE = KB * RB;
  static constexpr int NBUF = 4;          // key-tile buffers: copies run NBUF-1 tiles ahead
  static_assert(NP == 2 * KS && (NP & (NP - 1)) == 0, "piece index 2*ks + hl must fit the XOR swizzle");
  bf16x8 q[KS];
  // LDS offset of the lane's k-step 0 piece within a tile (key lane % 32); the
  // piece of k-step ks is at kbase ^ (32*ks), since piece 2*ks + hl equals
  // (2*ks) ^ hl and the swizzle is an XOR below bit 4 of the row offset
  uint32_t kbase;
  // each 16-lane group reads 16 rows x 1 piece: conflict-free
  __device__ __forceinline__ static int swz(int key) { return key & (NP - 1); }

  static constexpr bool QSTAGE = true;  // query rows arrive through an LDS stage

  // k-step ks of lane half hl holds head dims 16*ks + 8*hl .. +7, read from a
  // staged row (pieces swizzled by swz of the row's index in the stage)
  __device__ __forceinline__ void init_lds(const uint8_t* stage, int srow, int lane) {
    const int lq = lane & 31, hl = lane >> 5;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      q[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(stage + srow * RB + ((2 * ks + hl) ^ swz(srow)) * 16));
    kbase = lq * RB + (hl ^ swz(lq)) * 16;  // key 32*nb + lq adds 32*nb*RB
  }

  // s[nb][r] = S^T[key 32*nb + acc_row(r)][row lane % 32]
  __device__ __forceinline__ void logits(const uint8_t* kl, f32x16 s[2], const QRows&, int, int) const {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[nb][r] = 0.f;
    // re-derived per tile, so that the compiler does not keep all KS offsets live
    uint32_t kb = kbase;
    asm volatile("" : "+v"(kb));
    auto kread = [&](int ks, int nb) __attribute__((always_inline)) {
      return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(kl + nb * 32 * RB + (kb ^ (32u * ks))));
    };
    bf16x8 ka[2][2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) ka[0][nb] = kread(0, nb);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ks + 1 < KS) {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) ka[(ks + 1) & 1][nb] = kread(ks + 1, nb);
      }
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        s[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[ks & 1][nb], q[ks], s[nb], 0, 0, 0);
    }
  }
};

template <int D>
struct RowTileFp8 {
  // v_mfma_f32_32x32x64_f8f6f4: a lane supplies 32 consecutive E4M3 bytes per k-step
  static constexpr int RB = D;
  static constexpr int NP = RB / 16;
  static constexpr int KS = D / 64;
  static constexpr int TILE = KB * RB;
  static constexpr int NBUF = 4;
  i32x8 q[KS];
  uint32_t koff[2 * KS];
  // rows 2i, 2i+1 fill 16 banks-groups between them: conflict-free
  __device__ __forceinline__ static int swz(int key) { return (key >> 1) & (NP - 1); }

  static constexpr bool QSTAGE = true;  // query rows arrive through an LDS stage

  // k-step ks of lane half hl holds bytes 64*ks + 32*hl .. +31 of a staged row
  __device__ __forceinline__ void init_lds(const uint8_t* stage, int srow, int lane) {
    const int lq = lane & 31, hl = lane >> 5;
    const uint8_t* p = stage + srow * RB;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int piece = 4 * ks + 2 * hl;
      const u32x4 lo = *reinterpret_cast<const u32x4*>(p + ((piece ^ swz(srow)) * 16));
      const u32x4 hi = *reinterpret_cast<const u32x4*>(p + (((piece + 1) ^ swz(srow)) * 16));
      q[ks] = i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
#pragma unroll
      for (int hp = 0; hp < 2; ++hp) koff[2 * ks + hp] = lq * RB + ((piece + hp) ^ swz(lq)) * 16;
    }
  }

  // s[nb][r] = S^T[key 32*nb + acc_row(r)][row lane % 32]
  __device__ __forceinline__ void logits(const uint8_t* kl, f32x16 s[2], const QRows&, int, int) const {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[nb][r] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const u32x4 lo = *reinterpret_cast<const u32x4*>(kl + nb * 32 * RB + koff[2 * ks]);
        const u32x4 hi = *reinterpret_cast<const u32x4*>(kl + nb * 32 * RB + koff[2 * ks + 1]);
        const i32x8 kb = {(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
        // format 0 = E4M3 for both operands; zero scale operands select the unscaled instruction
        s[nb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kb, q[ks], s[nb], 0, 0, 0, 0, 0, 0);
      }
    }
  }
};

template <int D>
struct RowTileF32 {
  // Plain fp32 FMAs; fp32 inputs are only used at small sizes. Query rows are
  // read from global memory, keys from the LDS tile (unswizzled).
  static constexpr int RB = D * 4;
  static constexpr int NP = RB / 16;
  static constexpr int TILE = KB * RB;
  static constexpr int NBUF = TILE >= 32768 ? 3 : 4;  // LDS budget of the 32 KB fp32 tiles
  static constexpr bool QSTAGE = false;  // query rows are read from global memory in logits
  __device__ __forceinline__ static int swz(int) { return 0; }
  __device__ __forceinline__ void init_lds(const uint8_t*, int, int) {}

  // row0: the wave's first query row
  __device__ __forceinline__ void logits(const uint8_t* kl, f32x16 s[2], const QRows& qr, int row0, int lane) const {
    const int lq = lane & 31, hl = lane >> 5;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * nb + acc_row(r, hl);
        const float* qf = reinterpret_cast<const float*>(qr.row(row0 + lq));
        const float* kf = reinterpret_cast<const float*>(kl + key * RB);
        float acc = 0.f;
        for (int dd = 0; dd < D; ++dd) acc = fmaf(qf[dd], kf[dd], acc);
        s[nb][r] = acc;
      }
  }
};

template <int DT, int D>
struct RowTileOf;
template <int D> struct RowTileOf<LITEVLM_BF16, D> { using T = RowTileBf16<D>; };
template <int D> struct RowTileOf<LITEVLM_FP8_E4M3, D> { using T = RowTileFp8<D>; };
template <int D> struct RowTileOf<LITEVLM_F32, D> { using T = RowTileF32<D>; };

// Key tiles of one split, streamed through a ring of NBUF LDS buffers with
// direct global -> LDS copies (1 KB per wave instruction, keys clamped to
// klim - 1, pieces swizzled by the tile policy). Every tile of the split is
// copied, live or not, so that each wave's count of copies in flight is known.
template <class Tile>
struct KeyPipe {
  static constexpr int IPC = Tile::TILE / 1024;  // wave copies per tile
  static constexpr int NB = Tile::NBUF;
  static_assert(Tile::TILE % 1024 == 0, "a key tile must split into whole wave copies");
  uint8_t* ring;
  const uint8_t* kg;  // key 0 of this sample and KV head
  size_t kvrow;
  int tile0, ntl, klim, w, lane, cpw;
  int list;  // with a balanced split: lane j holds the split's j-th key tile
  bool bal;

  __device__ __forceinline__ KeyPipe(uint8_t* r, const uint8_t* k, size_t kv, int t0, int n, int lim, int w_, int l,
                                     int list_, bool bal_)
      : ring(r), kg(k), kvrow(kv), tile0(t0), ntl(n), klim(lim), w(w_), lane(l), list(list_), bal(bal_) {
    cpw = w < IPC ? (IPC - 1 - w) / kSweepWaves + 1 : 0;  // this wave's copies per tile
  }
  // key tile of step t (0 <= t < ntl <= 64)
  __device__ __forceinline__ int tile(int t) const { return bal ? __builtin_amdgcn_readlane(list, t) : tile0 + t; }
  __device__ __forceinline__ const uint8_t* buf(int t) const { return ring + (t % NB) * Tile::TILE; }
  __device__ __forceinline__ void issue(int t) {
    if (t >= ntl) return;
    uint8_t* dst = ring + (t % NB) * Tile::TILE;
    const int key0 = tile(t) * KB;
    for (int sub = w; sub < IPC; sub += kSweepWaves) {
      const int slot = sub * 64 + lane;
      const int row = slot / Tile::NP, ph = slot - row * Tile::NP;
      const int key = min(key0 + row, klim - 1);
      __builtin_amdgcn_global_load_lds((const void*)(kg + key * kvrow + (ph ^ Tile::swz(row)) * 16),
                                       (__attribute__((address_space(3))) void*)(dst + sub * 1024), 16, 0, 0);
    }
  }
  // Wait until this wave's copies of tile t have landed; the copies of the
  // tiles after it (at most NB-2 of them) may stay in flight. Loads complete
  // in order, and nothing else is issued between the copies.
  __device__ __forceinline__ void wait_for(int t) const {
    const int pend = max(0, min(NB - 2, ntl - 1 - t)) * cpw;
    switch (pend) {
      case 0: wait_vmcnt<0>(); break;
      case 1: wait_vmcnt<1>(); break;
      case 2: wait_vmcnt<2>(); break;
      case 3: wait_vmcnt<3>(); break;
      default: wait_vmcnt<4>(); break;
    }
  }
};

// Live and plain flags of the split's key tiles (bit j for tile tile0 + j):
// live = some key visible to some row (limit = S: kept visual or text key;
// limit = V_full: kept visual key), plain = all 64 keys kept visual. The keep
// bytes (kf, loaded by the caller: f[i] for tile w + 16*i, key lane) are also
// stored to keepl[tile][key] for the per-element masks.
constexpr int kFlagsPer = kMaxSplitTiles / kSweepWaves;

__device__ __forceinline__ void load_keep_bytes(const uint8_t* keep_row, int tile0, int V_full, int w, int lane,
                                                uint8_t f[kFlagsPer]) {
  // unconditional loads (of valid bytes when there is no mask): a branch here
  // would make the compiler wait for every load in flight
  const bool masked = keep_row && V_full > 0;
#pragma unroll
  for (int i = 0; i < kFlagsPer; ++i) {
    const int key = (tile0 + w + kSweepWaves * i) * KB + lane;
    const uint8_t* fp = masked ? keep_row + min(key, V_full - 1) : nullptr;
    f[i] = masked ? *fp : 1;
  }
}

template <class Pipe>
__device__ __forceinline__ void tile_flags(uint64_t* mw, uint8_t* keepl, const uint8_t f[kFlagsPer], const Pipe& pipe,
                                           int ntl, int V_full, int limit, int w, int lane, uint64_t& live,
                                           uint64_t& plain) {
  // each wave writes the bits of its own tiles into its own words; no atomics
  uint64_t lv_w = 0, pl_w = 0;
#pragma unroll
  for (int i = 0; i < kFlagsPer; ++i) {
    const int j = w + kSweepWaves * i;
    const int key = pipe.tile(j) * KB + lane;
    const bool vis = key < V_full && f[i] != 0;
    const bool txt = key >= V_full && key < limit;
    const uint64_t lv = __ballot(vis || txt), pl = __ballot(vis);
    if (j < ntl) {
      keepl[j * KB + lane] = vis ? 1 : 0;
      lv_w |= (lv != 0ull ? 1ull : 0ull) << j;
      pl_w |= (pl == ~0ull ? 1ull : 0ull) << j;
    }
  }
  if (lane == 0) {
    mw[w] = lv_w;
    mw[kSweepWaves + w] = pl_w;
  }
  __syncthreads();
  live = 0;
  plain = 0;
#pragma unroll
  for (int ww = 0; ww < kSweepWaves; ++ww) {
    live |= mw[ww];
    plain |= mw[kSweepWaves + ww];
  }
}

// Bit j (j = 16*nb + r) of the lane's 32 accumulator keys 32*nb + acc_row(r,
// lane/32) of tile j0 set where the key is a kept visual key (from the LDS keep
// bytes, 4 consecutive keys per word). Keys ascend with j.
__device__ __forceinline__ uint32_t lane_kept_bits(const uint8_t* keepl_tile, int lane) {
  const int hl = lane >> 5;
  uint32_t m = 0;
#pragma unroll
  for (int q4 = 0; q4 < 8; ++q4) {
    const uint32_t wd = *reinterpret_cast<const uint32_t*>(keepl_tile + 8 * q4 + 4 * hl);
#pragma unroll
    for (int e = 0; e < 4; ++e) m |= ((wd >> (8 * e)) & 1u) << (4 * q4 + e);
  }
  return m;
}

// Number of the lane's 32 accumulator keys that are <= key0 + 4*(lane/32) + L;
// they form a prefix of the bit order above.
__device__ __forceinline__ int keys_upto(int L) {
  int n = 0;
#pragma unroll
  for (int q4 = 0; q4 < 8; ++q4) n += min(max(L - 8 * q4 + 1, 0), 4);  // quad q4 holds offsets 8*q4 + 0..3
  return n;
}

// ---------------------------------------------------------------- sweep 1
// Flat grid over (b, g, row block rb) x ns1 key splits. Wave w owns query
// rows rb*512 + 32w .. +31 (one per lane, S^T layout) and keeps an exact
// running (max, sum) of exp2(logit) over the split's visible keys; the key
// tiles stream through a ring of LDS buffers, dead tiles (dropped views only) are
// not computed. Output: rowpart[b][g][split][row] = (max, sum), max in log2
// units. With d.bal (the view selection inside the call, 2..16 samples) the
// same grid takes units of the balanced split instead (bal_unit): a split is
// a list of live tiles, a sample has up to ns1 of them per column, and split 0
// fills the slots its sample does not use with (-inf, 0).

template <int DT, int D, bool VSEL>
__global__ void __launch_bounds__(kSweepThreads)
score_rowstats_kernel(ScoreDims d, const void* __restrict__ qv, const void* __restrict__ kv,
                      const uint8_t* __restrict__ token_keep, float2* __restrict__ rowpart,
                      unsigned long long* __restrict__ acc) {
  using Tile = typename RowTileOf<DT, D>::T;
  // LDS: key-tile ring buffers j at j*TILE, then the query stage, which starts
  // after the first two buffers: buffers 2.. overlap the stage and are first
  // filled once every wave has read its query rows from it. The workgroup's
  // query rows pass through the stage in rounds of QRR rows (whole rows per
  // 1 KB direct copy, so that every copy reads contiguous bytes; one round
  // where the rows fit), and each wave then reads its operand registers from
  // it. The keep bytes and flag words sit after the ring, inside the stage.
  constexpr int NPRE = Tile::NBUF < 3 ? Tile::NBUF - 1 : 2;  // key tiles in flight while the stage is in use
  constexpr int QOFF = Tile::QSTAGE ? NPRE * Tile::TILE : Tile::NBUF * Tile::TILE;
  constexpr int QROWS_MAX = Tile::QSTAGE ? (kLdsBytes - QOFF) / (32 * Tile::RB) * 32 : 32;
  constexpr int QRR = Tile::QSTAGE ? (RBLK < QROWS_MAX ? RBLK : QROWS_MAX) : 1;
  constexpr int QST = Tile::QSTAGE ? QRR * Tile::RB : 0;
  constexpr int NQR = Tile::QSTAGE ? (RBLK + QRR - 1) / QRR : 0;
  constexpr int FOFF = Tile::NBUF * Tile::TILE;  // keep bytes, then flag words
  constexpr int FEND = FOFF + kMaxSplitTiles * KB + 2 * kSweepWaves * 8;
  constexpr int LDS_BYTES = FEND > QOFF + QST ? FEND : QOFF + QST;
  static_assert(!Tile::QSTAGE || (QRR % 32 == 0 && QST % 1024 == 0), "stage rounds must hold whole waves and copies");
  static_assert(LDS_BYTES <= kLdsBytes, "sweep-1 LDS layout exceeds the workgroup limit");
  // One LDS object (key ring, query stage, keep bytes, flag words): with a
  // single object the compiler adds no vmcnt wait of its own before reads of
  // one buffer while direct copies into another are in flight; the explicit
  // waits and barriers order copies before reads.
  __shared__ __attribute__((aligned(1024))) uint8_t lds[LDS_BYTES];
  uint8_t* qstage = lds + QOFF;
  uint8_t* keepl = lds + FOFF;
  uint64_t* mw = reinterpret_cast<uint64_t*>(keepl + kMaxSplitTiles * KB);

  // the column sums of sweep 2 start from zero (this grid runs before it);
  // after the work decode: loads wait for the stores issued before them
  auto zero_acc = [&]() {
    for (int i = blockIdx.x * kSweepThreads + threadIdx.x; i < d.B * d.V_full; i += gridDim.x * kSweepThreads)
      acc[i] = 0ull;
  };

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int b, g, rb, split, tile0 = 0, ntl, list = 0, nsb = 0;
  bool bal = false;
  if constexpr (VSEL) bal = d.bal != 0;
  if (bal) {
    BalUnit u;
    if (!bal_unit(d, lds, w, lane, u)) {
      zero_acc();
      return;
    }
    b = u.b;
    g = u.g;
    rb = u.rb;
    split = u.split;
    ntl = u.ntl;
    nsb = u.ns;
    list = u.list;
  } else {
    int col;
    if (!decode_column(d.B * d.Hkv * d.n_rb, d.ns1, col, split)) {
      zero_acc();
      return;
    }
    const int bg = col / d.n_rb;
    rb = col - bg * d.n_rb;
    b = bg / d.Hkv;
    g = bg - b * d.Hkv;
    tile0 = split_begin(split, d.n_kt, d.ns1);
    ntl = split_begin(split + 1, d.n_kt, d.ns1) - tile0;
  }
  zero_acc();
  const int lq = lane & 31, hl = lane >> 5;
  const uint8_t* keep_row = token_keep ? token_keep + (size_t)b * d.S : nullptr;
  const uint8_t* q = static_cast<const uint8_t*>(qv);
  const uint8_t* k = static_cast<const uint8_t*>(kv);
  const QRows qr{q + (((size_t)b * d.S + d.V_full + d.tq0) * d.Hq + (size_t)g * d.G) * Tile::RB, d.G, d.Hq,
                 Tile::RB, d.R};
  const int row0 = rb * RBLK + 32 * w;
  const int row = row0 + lq;
  const bool wave_active = row0 < d.R;

  // copies of query-row round `round` into the stage: row rr of the round,
  // 16-byte piece ph at stage slot ph ^ swz(rr)
  auto q_round = [&](int round) {
    const int ncopy = min(QRR, RBLK - round * QRR) * Tile::RB / 1024;
    for (int sub = w; sub < ncopy; sub += kSweepWaves) {
      const int slot = sub * 64 + lane;
      const int rr = slot / Tile::NP, ph = slot - rr * Tile::NP;
      __builtin_amdgcn_global_load_lds((const void*)(qr.row(rb * RBLK + round * QRR + rr) + (ph ^ Tile::swz(rr)) * 16),
                                       (__attribute__((address_space(3))) void*)(qstage + sub * 1024), 16, 0, 0);
    }
  };
  const int my_round = (32 * w) / QRR, srow = 32 * w + lq - my_round * QRR;

  // The first key tiles, the first query round and the keep bytes, all in
  // flight together: the key tiles (not shared with other workgroups, so
  // mostly from HBM) go first, their latency hidden behind the query copies;
  // the keep bytes go last, since their first use waits for them (and, loads
  // completing in order, for everything before them).
  Tile tile;
  KeyPipe<Tile> pipe(lds, k + ((size_t)b * d.S * d.Hkv + g) * Tile::RB, (size_t)d.Hkv * Tile::RB, tile0, ntl,
                     d.S, w, lane, list, bal);
#pragma unroll
  for (int t = 0; t < (Tile::QSTAGE ? NPRE : Tile::NBUF - 1); ++t) pipe.issue(t);
  if (Tile::QSTAGE) q_round(0);
  asm volatile("" ::: "memory");  // keep the copies ahead of the keep-byte loads
  uint8_t kf[kFlagsPer];
  ViewIn vin;
  if constexpr (VSEL) vin = view_load(d.vs.logit, d.vs.lexical, d.vs.N, b, lane);
  else load_keep_bytes(keep_row, tile0, d.V_full, w, lane, kf);
  if (Tile::QSTAGE) {
    wait_vmcnt<0>();  // round 0, the first key tiles and the keep bytes have landed
    __syncthreads();
    if (wave_active && my_round == 0) tile.init_lds(qstage, srow, lane);
    for (int round = 1; round < NQR; ++round) {
      __syncthreads();  // every read of the previous round is done
      q_round(round);
      wait_vmcnt<0>();
      __syncthreads();
      if (wave_active && my_round == round) tile.init_lds(qstage, srow, lane);
    }
    __syncthreads();  // every read of the stage is done: buffers 2.. may be filled
#pragma unroll
    for (int t = NPRE; t < Tile::NBUF - 1; ++t) pipe.issue(t);
  }
  pipe.wait_for(0);
  __syncthreads();  // tile 0 and the keep bytes have landed
  if constexpr (VSEL) {
    // the keep flags of the lane's keys from the sample's view selection
    const uint32_t vm = (uint32_t)view_keep_mask<kFusedViews>(vin, d.vs.lexical != nullptr, d.vs.w, d.vs.tau, d.vs.N, lane);
#pragma unroll
    for (int i = 0; i < kFlagsPer; ++i) {
      const int key = pipe.tile(w + kSweepWaves * i) * KB + lane;
      kf[i] = d.V_full > 0 ? (uint8_t)view_token_flag(d.vs, vm, min(key, d.V_full - 1)) : 1;
    }
  }
  uint64_t live, plain;
  tile_flags(mw, keepl, kf, pipe, ntl, d.V_full, d.S, w, lane, live, plain);

  // token of the lane's row for the causal text mask (-1: a row past R sees no text)
  const int t_row = row < d.R ? d.tq0 + row / d.G : -1;
  const float c = d.scale_log2;
  float m_run = -INFINITY, z_run = 0.f;

  // Statistics of one tile held in s (masking as needed).
  auto stats = [&](int t, f32x16* s) __attribute__((always_inline)) {
    if (!((plain >> t) & 1ull)) {
      // visible: kept visual keys, and text keys V_full + t' with t' <= the row's token
      const int key0 = pipe.tile(t) * KB;
      const int ns = keys_upto(d.S - 1 - key0 - 4 * hl);        // keys < S
      const int n1 = min(keys_upto(d.V_full + t_row - key0 - 4 * hl), ns);
      const uint32_t below_n1 = n1 >= 32 ? 0xFFFFFFFFu : ((1u << n1) - 1u);
      uint32_t vis;
      if (key0 >= d.V_full) {
        vis = below_n1;  // text keys only: the causal limit alone
      } else {
        const uint32_t kept = lane_kept_bits(keepl + t * KB, lane);
        const int nv = keys_upto(d.V_full - 1 - key0 - 4 * hl);   // keys < V_full
        const uint32_t below_nv = nv >= 32 ? 0xFFFFFFFFu : ((1u << nv) - 1u);
        vis = kept | (below_n1 & ~below_nv);
      }
#pragma unroll
      for (int j = 0; j < 32; ++j) s[j >> 4][j & 15] = ((vis >> j) & 1u) ? s[j >> 4][j & 15] : -INFINITY;
    }
    // raw logits: the scale is positive, so the max commutes with it
    float mx = __builtin_elementwise_maximum(s[0][0], s[1][0]);
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = __builtin_elementwise_maximum(mx, __builtin_elementwise_maximum(s[0][r], s[1][r]));
    mx = max_xor32(mx);
    const float m_new = fmaxf(m_run, mx);
    // exact running max: the sum so far is rescaled whenever the max grows
    const float ms = m_new == -INFINITY ? 0.f : -m_new * c;
    const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(fmaf(m_run, c, ms));
    float z4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) z4[r & 3] += __builtin_amdgcn_exp2f(fmaf(s[nb][r], c, ms));
    z_run = fmaf(z_run, alpha, (z4[0] + z4[1]) + (z4[2] + z4[3]));
    m_run = m_new;
  };

  // Waves w and w+4 share a SIMD. Group 0 (w & 4 == 0) forms the logits of
  // tile t and then its statistics within step t; group 1 first finishes the
  // statistics of tile t-1 and then forms the logits of tile t, keeping them
  // across the barrier. On each SIMD one group's VALU work overlaps the other
  // group's MFMAs.
  const bool lag = (w & 4) != 0;
  f32x16 s[2];
  for (int t = 0; t < ntl; ++t) {
    // the buffer of tile t+NBUF-1 was last read in step t-1
    pipe.issue(t + Tile::NBUF - 1);
    if (wave_active) {
      if (lag) {
        if (t > 0 && ((live >> (t - 1)) & 1ull)) stats(t - 1, s);
        if ((live >> t) & 1ull) tile.logits(pipe.buf(t), s, qr, row0, lane);
      } else if ((live >> t) & 1ull) {
        tile.logits(pipe.buf(t), s, qr, row0, lane);
        stats(t, s);
      }
    }
    pipe.wait_for(t + 1);
    __syncthreads();
  }
  if (wave_active && lag && ((live >> (ntl - 1)) & 1ull)) stats(ntl - 1, s);
  // both lane halves share the running max; their sums cover different keys
  const float z = sum_xor32(z_run);
  if (hl == 0 && row < d.R) {
    float2* rp = rowpart + ((size_t)b * d.Hkv + g) * d.ns1 * d.R + row;
    rp[(size_t)split * d.R] = make_float2(m_run == -INFINITY ? -INFINITY : m_run * c, z);
    // a balanced split fills the partials of the splits its sample does not use
    if (bal && split == 0)
      for (int sl = nsb; sl < d.ns1; ++sl) rp[(size_t)sl * d.R] = make_float2(-INFINITY, 0.f);
  }
}

// ---------------------------------------------------------------- sweep-2 logit tiles
// A sweep-2 tile policy holds one wave's 64 keys of one KV head in registers
// (the B operand of S = Q K^T) and forms, for the 32 query rows of a chunk
// staged in LDS, s[nb][r] = q(acc_row(r)) . k(32*nb + lane % 32) in fp32: a
// lane owns one key column of each 32-key block. ro[] are the lane's byte
// offsets of its A-operand pieces within a chunk.

template <int D>
struct ColTileBf16 {
  static constexpr int RB = D * 2;        // bytes per row
  static constexpr int NP = RB / 16;      // 16-byte pieces per row
  static constexpr int KS = D / 16;       // k-steps of v_mfma_f32_32x32x16_bf16
  static_assert(NP == 2 * KS && (NP & (NP - 1)) == 0, "piece index 2*ks + hl must fit the XOR swizzle");
  bf16x8 kreg[2][KS];
  // LDS offset of the lane's k-step 0 piece within a chunk (row lane % 32); the
  // piece of k-step ks is at rbase ^ (32*ks) (piece 2*ks + hl = (2*ks) ^ hl,
  // and the swizzle is an XOR below bit 4 of the row offset)
  uint32_t rbase;
  // LDS piece swizzle of Q rows: each 16-lane group reads 16 rows x 1 piece
  __device__ __forceinline__ static int qswz(int r) { return r & (NP - 1); }

  __device__ __forceinline__ void init(int lane) {
    const int lq = lane & 31, hl = lane >> 5;
    rbase = lq * RB + (hl ^ qswz(lq)) * 16;
  }

  __device__ __forceinline__ void load_keys(const uint8_t* kbase, size_t kstride, int nvalid, int lane) {
    const int lq = lane & 31, hl = lane >> 5;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int key = min(nb * 32 + lq, max(nvalid - 1, 0));
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        kreg[nb][ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                                                      kbase + key * kstride + (ks * 16 + 8 * hl) * 2));
    }
  }

  __device__ __forceinline__ void logits(const uint8_t* buf, int, f32x16 s[2]) const {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[nb][r] = 0.f;
    // re-derived per chunk, so that the compiler does not keep all KS offsets live
    uint32_t rb = rbase;
    asm volatile("" : "+v"(rb));
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 qb = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(buf + (rb ^ (32u * ks))));
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        s[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qb, kreg[nb][ks], s[nb], 0, 0, 0);
    }
  }
};

template <int D>
struct ColTileFp8 {
  // v_mfma_f32_32x32x64_f8f6f4: a lane supplies 32 consecutive E4M3 bytes per k-step
  static constexpr int RB = D;
  static constexpr int NP = RB / 16;
  static constexpr int KS = D / 64;
  i32x8 kreg[2][KS];
  uint32_t ro[2 * KS];
  __device__ __forceinline__ static int qswz(int r) { return (r >> 1) & (NP - 1); }

  __device__ __forceinline__ void init(int lane) {
    const int lq = lane & 31, hl = lane >> 5;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int hp = 0; hp < 2; ++hp) ro[2 * ks + hp] = lq * RB + ((4 * ks + 2 * hl + hp) ^ qswz(lq)) * 16;
  }

  __device__ __forceinline__ void load_keys(const uint8_t* kbase, size_t kstride, int nvalid, int lane) {
    const int lq = lane & 31, hl = lane >> 5;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int key = min(nb * 32 + lq, max(nvalid - 1, 0));
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const uint8_t* p = kbase + key * kstride + ks * 64 + 32 * hl;
        const u32x4 lo = *reinterpret_cast<const u32x4*>(p);
        const u32x4 hi = *reinterpret_cast<const u32x4*>(p + 16);
        kreg[nb][ks] = i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
      }
    }
  }

  __device__ __forceinline__ void logits(const uint8_t* buf, int, f32x16 s[2]) const {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[nb][r] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const u32x4 lo = *reinterpret_cast<const u32x4*>(buf + ro[2 * ks]);
      const u32x4 hi = *reinterpret_cast<const u32x4*>(buf + ro[2 * ks + 1]);
      const i32x8 qb = {(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        // format 0 = E4M3 for both operands; zero scale operands select the unscaled instruction
        s[nb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(qb, kreg[nb][ks], s[nb], 0, 0, 0, 0, 0, 0);
    }
  }
};

template <int D>
struct ColTileF32 {
  // Plain fp32 FMAs; fp32 inputs are only used at small sizes. The lane's two
  // keys are read from global memory, its 16 accumulator rows from LDS.
  static constexpr int RB = D * 4;
  static constexpr int NP = RB / 16;
  const uint8_t* kbase;
  size_t kstride;
  int nvalid;
  __device__ __forceinline__ static int qswz(int) { return 0; }
  __device__ __forceinline__ void init(int) {}

  __device__ __forceinline__ void load_keys(const uint8_t* kb_, size_t ks_, int nv, int) {
    kbase = kb_;
    kstride = ks_;
    nvalid = nv;
  }

  __device__ __forceinline__ void logits(const uint8_t* buf, int lane, f32x16 s[2]) const {
    const int lq = lane & 31, hl = lane >> 5;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int key = nb * 32 + lq;
      const float* kr = reinterpret_cast<const float*>(kbase + min(key, max(nvalid - 1, 0)) * kstride);
      for (int r = 0; r < 16; ++r) {
        const float* qf = reinterpret_cast<const float*>(buf + acc_row(r, hl) * RB);
        float acc = 0.f;
        if (key < nvalid)
          for (int dd = 0; dd < D; ++dd) acc = fmaf(qf[dd], kr[dd], acc);
        s[nb][r] = acc;
      }
    }
  }
};

template <int DT, int D>
struct ColTileOf;
template <int D> struct ColTileOf<LITEVLM_BF16, D> { using T = ColTileBf16<D>; };
template <int D> struct ColTileOf<LITEVLM_FP8_E4M3, D> { using T = ColTileFp8<D>; };
template <int D> struct ColTileOf<LITEVLM_F32, D> { using T = ColTileF32<D>; };

// Text query rows of a workgroup pass through three chunk buffers in LDS,
// filled with direct global -> LDS copies (16-byte pieces, XOR-swizzled per
// row) two chunks ahead of use. Row r of KV group g is query head g*G + r%G
// of text token r/G; each lane tracks (token, head) of its copies and steps
// them by the row distance between the workgroup's chunks. Rows past R repeat
// a valid row; their statistics make their terms vanish.
template <class Tile>
struct QRing {
  static constexpr int RB = Tile::RB;
  static constexpr int NP = Tile::NP;
  static constexpr int CB = CH * RB;                            // bytes per chunk
  static constexpr int IPC = CB / 1024;                         // wave copies per chunk
  static constexpr int CPW = (IPC + kColWaves - 1) / kColWaves;
  static constexpr int NBUF = 3;
  static constexpr int BYTES = NBUF * CB;
  static_assert(CB % 1024 == 0, "a chunk must split into whole wave copies");
  static_assert(IPC % kColWaves == 0 || IPC < kColWaves, "copies must split evenly over waves");

  const uint8_t* qbase;  // row (text token 0, head g*G) of this sample and group
  int G, Hq, T, dt, dh;
  int t[CPW], hh[CPW];
  uint32_t src[CPW];     // byte offset of the lane's piece within its row

  __device__ __forceinline__ void init(const uint8_t* q, int b, int g, const ScoreDims& d, int w, int lane,
                                       int row0, int cstep) {
    qbase = q + (((size_t)b * d.S + d.V_full + d.tq0) * d.Hq + (size_t)g * d.G) * RB;
    G = d.G;
    Hq = d.Hq;
    T = d.T;
    dt = cstep / d.G;
    dh = cstep - dt * d.G;
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
      const int slot = (w + kColWaves * j) * 64 + lane;
      const int row = slot / NP;
      src[j] = ((slot % NP) ^ Tile::qswz(row)) * 16;
      const int r = row0 + row;
      t[j] = r / G;
      hh[j] = r - t[j] * G;
    }
  }

  // number of copies that issue() makes for wave w
  __device__ __forceinline__ static int copies(int w) {
    int n = 0;
#pragma unroll
    for (int j = 0; j < CPW; ++j) n += (w + kColWaves * j < IPC) ? 1 : 0;
    return n;
  }

  // copies of the current chunk into buf, then step to the workgroup's next chunk
  __device__ __forceinline__ void issue(uint8_t* buf, int w) {
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
      const int sub = w + kColWaves * j;
      if (sub < IPC) {
        const int tt = min(t[j], T - 1);
        __builtin_amdgcn_global_load_lds((const void*)(qbase + ((size_t)tt * Hq + hh[j]) * RB + src[j]),
                                         (__attribute__((address_space(3))) void*)(buf + sub * 1024),
                                         16, 0, 0);
      }
      hh[j] += dh;
      t[j] += dt;
      if (hh[j] >= G) {
        hh[j] -= G;
        t[j] += 1;
      }
    }
  }
};

// One float2 store to LDS (ds_write_b64), opaque to the compiler's wait
// insertion; the caller orders it with an LDS wait and a barrier.
__device__ __forceinline__ void lds_store_f2(float2* p, float2 v) {
  const uint32_t a = (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) float2*)p);
  asm volatile("ds_write_b64 %0, %1" ::"v"(a), "v"(v) : "memory");
}

// Workgroup-wide OR through four per-wave words of the kernel's own LDS
// array (the runtime's block reduction would add an LDS object of its own).
// The store and the barriers wait for LDS accesses only (direct copies into
// other LDS buffers may stay in flight).
__device__ __forceinline__ bool block_any(bool v, uint32_t* slots) {
  const uint64_t m = __ballot(v);
  if ((threadIdx.x & 63) == 0) {
    const uint32_t a = (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint32_t*)(slots + (threadIdx.x >> 6)));
    const uint32_t x = m != 0 ? 1u : 0u;
    asm volatile("ds_write_b32 %0, %1" ::"v"(a), "v"(x) : "memory");
  }
  lds_barrier();
  const bool r = (slots[0] | slots[1] | slots[2] | slots[3]) != 0;
  lds_barrier();
  return r;
}

// ---------------------------------------------------------------- sweep 2
// Flat grid over columns (b, g, visual key tile vt of KT keys) x rs2 row splits.
// A workgroup first merges the sweep-1 partials of its rows into per-row
// (-max, 1/sum) in LDS: m = max over splits, Z = sum Z_split * exp2(m_split -
// m). Each wave owns 64 keys; a lane accumulates exp2(logit - m)/Z of its key
// column over the 16 accumulator rows it holds of each chunk, so only the two
// lane halves (disjoint rows) are summed at the end. The workgroup's column
// partials go into acc[b][key] as fixed-point integers (value * fx, rounded
// to nearest): integer addition is associative, so the sums do not depend on
// the order in which the workgroups add them.

constexpr int kMaxChunksPerSplit = 32;  // row chunks of one sweep-2 workgroup (table of 8 KB)

template <int DT, int D, bool VSEL>
__global__ void __launch_bounds__(256, DT == LITEVLM_F32 ? 2 : 3)  // fp32 chunks: 16 KB each
score_colmass_kernel(ScoreDims d, const void* __restrict__ qv, const void* __restrict__ kv,
                     const uint8_t* __restrict__ token_keep, const float2* __restrict__ rowpart,
                     unsigned long long* __restrict__ acc) {
  using Tile = typename ColTileOf<DT, D>::T;
  using Ring = QRing<Tile>;
  // one LDS object (see sweep 1): the chunk buffers, the row statistics of
  // the workgroup's rows, four flag words
  constexpr int TAB = Ring::BYTES;
  constexpr int FLG = TAB + kMaxChunksPerSplit * CH * 8;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[FLG + 16];
  float2* table = reinterpret_cast<float2*>(lds + TAB);

  int col, rs;
  if (!decode_column(d.B * d.Hkv * d.n_vt, d.rs2, col, rs)) return;
  const int bgi = col / d.n_vt, vt = col - bgi * d.n_vt;
  const int bg = pair_at(bgi, d.B * d.Hkv);
  const int b = bg / d.Hkv, g = bg - b * d.Hkv;
  const uint8_t* q = static_cast<const uint8_t*>(qv);
  const uint8_t* k = static_cast<const uint8_t*>(kv);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int hl = lane >> 5;
  const int key0 = vt * KT + w * KW;
  const uint8_t* keep_row = token_keep ? token_keep + (size_t)b * d.S : nullptr;
  const int nch = (d.nchunks - rs + d.rs2 - 1) / d.rs2;
  const int cstep = d.rs2 * CH;
  const int row0 = rs * CH;
  if (nch > kMaxChunksPerSplit) return;  // the host split keeps nch within the table

  // Row statistics of local row lr = i*CH + j (global row row0 + i*cstep + j):
  // P consecutive threads share a row, each taking every P-th split, and
  // combine their (max, sum) by shuffles in fixed order. The first 2*8 splits
  // of a thread's first row are loaded before everything else, so that they
  // return while the keys are still in flight (loads complete in order).
  const int nrows = nch * CH;
  const int P = nrows >= 256 ? 1 : (nrows >= 128 ? 2 : (nrows >= 64 ? 4 : 8));
  const float2* rp0 = rowpart + ((size_t)b * d.Hkv + g) * d.ns1 * d.R;
  auto row_of = [&](int lr) { return lr < nrows ? row0 + (lr / CH) * cstep + (lr % CH) : d.R; };
  float2 pre[2][8];
  {
    const int p = tid % P;
    const float2* rp = rp0 + min(row_of(tid / P), d.R - 1);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int j = 0; j < 8; ++j) pre[h][j] = rp[(size_t)min(p + (8 * h + j) * P, d.ns1 - 1) * d.R];
  }

  // The keep byte of the thread's key, the keys and the first two query
  // chunks are in flight while the row statistics are merged (loads complete
  // in order: the keep byte first, since the merge is followed by its use).
  const int tkey = vt * KT + tid;
  // an unconditional load (of a valid byte when there is no mask), so that no
  // branch makes the compiler wait for every load in flight here
  const uint8_t* tkp = keep_row ? keep_row + min(tkey, d.V_full - 1) : static_cast<const uint8_t*>(kv);
  uint8_t tkraw = 1;
  ViewIn vin;
  if constexpr (VSEL) vin = view_load(d.vs.logit, d.vs.lexical, d.vs.N, b, lane);
  else tkraw = *tkp;
  Ring ring;
  ring.init(q, b, g, d, w, lane, row0, cstep);
  Tile tile;
  tile.init(lane);
  tile.load_keys(k + (((size_t)b * d.S + min(key0, d.V_full - 1)) * d.Hkv + g) * Tile::RB,
                 (size_t)d.Hkv * Tile::RB, max(0, min(KW, d.V_full - key0)), lane);
  ring.issue(lds, w);
  if (nch > 1) ring.issue(lds + Ring::CB, w);

  // fold splits s0 + j*P (j < 8; those past ns1 ignored) into a running (max, sum)
  auto fold8 = [&](float2 (&u)[8], int s0, float& m, float& z) {
    float mg = m;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (s0 + j * P >= d.ns1) u[j] = make_float2(-INFINITY, 0.f);
      mg = fmaxf(mg, u[j].x);
    }
    if (mg != -INFINITY) {
      // exp2(-inf - mg) = 0 for splits without a visible key (their sum is 0)
      z = m == -INFINITY ? 0.f : z * __builtin_amdgcn_exp2f(m - mg);
#pragma unroll
      for (int j = 0; j < 8; ++j) z += u[j].y * __builtin_amdgcn_exp2f(u[j].x - mg);
      m = mg;
    }
  };
  for (int base = 0; base < nrows * P; base += 256) {
    const int idx = base + tid, lr = idx / P, p = idx - lr * P;
    const int r = row_of(lr);
    float m = -INFINITY, z = 0.f;
    int s0 = p;
    if (base == 0) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        fold8(pre[h], s0, m, z);
        s0 += 8 * P;
      }
    }
    if (r < d.R) {
      const float2* rp = rp0 + r;
      for (; s0 < d.ns1; s0 += 8 * P) {
        float2 u[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) u[j] = rp[(size_t)min(s0 + j * P, d.ns1 - 1) * d.R];
        fold8(u, s0, m, z);
      }
    }
    for (int off = 1; off < P; off <<= 1) {
      const float mo = __shfl_xor(m, off), zo = __shfl_xor(z, off);
      const float mn = fmaxf(m, mo);
      z = (m == -INFINITY ? 0.f : z * __builtin_amdgcn_exp2f(m - mn)) +
          (mo == -INFINITY ? 0.f : zo * __builtin_amdgcn_exp2f(mo - mn));
      m = mn;
    }
    // rows past R: exp2(-inf) = 0 and a zero weight. The store is written as
    // inline assembly: the table and the chunk buffers being filled by the
    // direct copies are disjoint, but the compiler cannot tell and would make
    // the store wait for every copy in flight.
    if (p == 0 && lr < nrows) {
      const float2 e = r < d.R ? make_float2(-m, 1.0f / z) : make_float2(-INFINITY, 0.f);
      lds_store_f2(table + lr, e);
    }
  }
  uint32_t vm = 0;
  if constexpr (VSEL) vm = (uint32_t)view_keep_mask<kFusedViews>(vin, d.vs.lexical != nullptr, d.vs.w, d.vs.tau, d.vs.N, lane);
  const uint8_t tkb = VSEL ? (uint8_t)view_token_flag(d.vs, vm, min(tkey, d.V_full - 1)) : (keep_row ? tkraw : 1);
  const bool tkept = tkey < d.V_full && tkb != 0;
  // the mark of a dropped key's column, from one workgroup per key tile (no
  // other workgroup writes a dropped key's column)
  if (VSEL && g == 0 && rs == 0 && tkey < d.V_full && tkb == 0) acc[(size_t)b * d.V_full + tkey] = kDroppedCol;
  if (!block_any(tkept, reinterpret_cast<uint32_t*>(lds + FLG))) {
    // no kept key in the tile: nothing to add (the copies into LDS land
    // before the workgroup ends)
    wait_vmcnt<0>();
    return;
  }
  const float c = d.scale_log2;
  const int cpw = __builtin_amdgcn_readfirstlane(Ring::copies(w));  // wave-uniform: scalar branches

  // four partial sums per key column (accumulator rows r with r % 4 = j)
  float cm[2][4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};

  // Chunk i sits in buffer i % 3. Step i waits for its copies (those of chunk
  // i+1 may stay in flight; loads complete in order), and its barrier also
  // marks the end of every read of chunk i-1, whose buffer then takes chunk i+2.
  auto body = [&](auto bufc, int i) {
    constexpr int BUF = decltype(bufc)::value;
    const uint8_t* buf = lds + BUF * Ring::CB;
    wait_vmcnt_upto(i + 1 < nch ? cpw : 0);
    lds_barrier();
    if (i + 2 < nch) ring.issue(lds + ((BUF + 2) % Ring::NBUF) * Ring::CB, w);
    f32x16 s[2];
    tile.logits(buf, lane, s);
    // (-max, 1/sum) of the lane's accumulator rows 8*j + 4*hl + 0..3
    f32x4 st[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x4* sp = reinterpret_cast<const f32x4*>(table + i * CH + 8 * j + 4 * hl);
      st[2 * j] = sp[0];
      st[2 * j + 1] = sp[1];
    }
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float ms = (r & 1) ? st[r >> 1].z : st[r >> 1].x;
        const float iz = (r & 1) ? st[r >> 1].w : st[r >> 1].y;
        cm[nb][r & 3] = fmaf(__builtin_amdgcn_exp2f(fmaf(s[nb][r], c, ms)), iz, cm[nb][r & 3]);
      }
  };
  for (int i = 0; i < nch; i += 3) {
    body(std::integral_constant<int, 0>{}, i);
    if (i + 1 < nch) body(std::integral_constant<int, 1>{}, i + 1);
    if (i + 2 < nch) body(std::integral_constant<int, 2>{}, i + 2);
  }
  // the lane's key column over its rows, then the other lane half's rows:
  // lane L ends with key key0 + L
  float tot[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) tot[nb] = (cm[nb][0] + cm[nb][1]) + (cm[nb][2] + cm[nb][3]);
  const float give = hl ? tot[0] : tot[1];
  const float got = __shfl_xor(give, 32);
  const float colmass = (hl ? tot[1] : tot[0]) + got;
  const int key = key0 + lane;
  // dropped keys were summed over too; their column stays 0
  if (key < d.V_full && (VSEL ? view_token_flag(d.vs, vm, key) != 0 : (keep_row == nullptr || keep_row[key])))
    __hip_atomic_fetch_add(acc + (size_t)b * d.V_full + key, (unsigned long long)__float2ll_rn(colmass * d.fx),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
constexpr int kDigitBits = 12;              // radix digit width of the selection
constexpr int kBins = 1 << kDigitBits;
constexpr int kBinsPer = kBins / kTopkThreads;  // histogram bins owned by each thread
static_assert(kBins == kBinsPer * kTopkThreads, "the threads own whole runs of histogram bins");
static_assert(LITEVLM_MAX_VISUAL % (4 * kTopkThreads) == 0, "key loads come in whole rounds of float4");

__device__ __forceinline__ int wave_sum_int(int v) {
  float f;  // exact: counts stay far below 2^24
  f = (float)v;
  f = row16_sum(f);
  f = sum_xor32(sum_xor16(f));
  return (int)f;
}

// Nonzero bytes of a 32-bit word.
__device__ __forceinline__ int nonzero_bytes(uint32_t u) {
  u |= u >> 4;
  u |= u >> 2;
  u |= u >> 1;
  return __popc(u & 0x01010101u);
}

// Nonzero flags among row[0..n), counted by one wave (result on every lane).
__device__ __forceinline__ int wave_count_flags(const uint8_t* row, int n, int lane) {
  int cnt = 0;
  if ((reinterpret_cast<uintptr_t>(row) & 15) == 0) {
    const uint4* r4 = reinterpret_cast<const uint4*>(row);
    for (int j = lane; j < n / 16; j += 64) {
      const uint4 u = r4[j];
      cnt += nonzero_bytes(u.x) + nonzero_bytes(u.y) + nonzero_bytes(u.z) + nonzero_bytes(u.w);
    }
    for (int j = (n & ~15) + lane; j < n; j += 64) cnt += row[j] != 0;
  } else {
    for (int j = lane; j < n; j += 64) cnt += row[j] != 0;
  }
  return wave_sum_int(cnt);
}

// Block-wide exclusive scan of one int per thread with a single barrier; the
// 16 wave totals go to wsum, which the caller must not reuse before another
// barrier. Returns the exclusive prefix; *total gets the block total.
__device__ __forceinline__ int block_scan_excl(int v, int* wsum, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // inclusive wave scan on DPP: within rows of 16 (row_shr 1, 2, 4, 8), then
  // row 0's last lane into row 1 and row 2's into row 3 (row_bcast:15), then
  // lane 31 into rows 2 and 3 (row_bcast:31)
  int x = v;
  x += dpp_i<0x111>(x);
  x += dpp_i<0x112>(x);
  x += dpp_i<0x114>(x);
  x += dpp_i<0x118>(x);
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kTopkWaves; ++w) {
    const int t = wsum[w];
    tot += t;
    before += w < wave ? t : 0;
  }
  *total = tot;
  return before + x - v;
}

// One workgroup per sample: the compacted offset from every earlier sample's
// kept-visual count, the scores (fixed-point column sums times inv: the mean
// over the Hq*T text rows; -inf for dropped tokens), their order keys, radix
// select of the k_b-th largest key (12-bit digits below the common prefix of
// the kept keys), then the stable compaction.
// VSEL: the keep flags come from the view selection (vs), and the selection's
// outputs are written here: view_keep [B, N], the token mask [B, S] and the
// kept-visual counts [B] (each may be NULL).
template <bool VSEL>
__global__ void __launch_bounds__(kTopkThreads)
topk_compact_kernel(int S, int V_full, double keep_ratio, const uint8_t* __restrict__ token_keep,
                    const unsigned long long* __restrict__ acc, double inv, float* __restrict__ scores,
                    int32_t* __restrict__ kept_index, int32_t* __restrict__ cu_seqlens, ViewSel vs,
                    uint8_t* __restrict__ view_keep_out, uint8_t* __restrict__ token_keep_out,
                    int32_t* __restrict__ n_visual_out) {
  __shared__ uint32_t keys[LITEVLM_MAX_VISUAL];
  __shared__ int hist[kBins];
  __shared__ int vcnt[LITEVLM_MAX_BATCH];
  __shared__ int wsum[4][kTopkWaves];  // [0] batch offset, [1], [2] radix passes, [3] compaction
  __shared__ uint32_t red_u[2][kTopkWaves];
  __shared__ int sel_digit, sel_above;
  const int b = blockIdx.x;
  const int T = S - V_full;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  // Order keys of the kept tokens' scores (dropped tokens: key 0; kept keys
  // are >= 0x80000000 since scores are >= 0). The column sums and keep bytes
  // of this sample are requested first, from clamped addresses, so that a
  // thread's rounds are all in flight at once, together with the loads of the
  // kept-visual counts below.
  const uint8_t* keep_row = token_keep ? token_keep + (size_t)b * S : nullptr;
  // the sample's view selection, requested first (its mask gives every keep flag)
  // and the view scores of sample `wave` (<= b), whose kept-visual count
  // enters this sample's offset
  ViewIn vin, vinw;
  if constexpr (VSEL) {
    vin = view_load(vs.logit, vs.lexical, vs.N, b, lane);
    vinw = view_load(vs.logit, vs.lexical, vs.N, min(wave, b), lane);
  }
  const unsigned long long* ac = acc + (size_t)b * V_full;
  float* sc = scores + (size_t)b * V_full;
  auto score_of = [&](unsigned long long v, bool kept) { return kept ? (float)((double)v * inv) : -INFINITY; };
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
  const bool vec = V_full >= 4 && (V_full & 3) == 0 && (reinterpret_cast<uintptr_t>(sc) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(ac) & 15) == 0 &&
                   (keep_row == nullptr || (reinterpret_cast<uintptr_t>(keep_row) & 3) == 0);
  typedef unsigned long long u64x2 __attribute__((ext_vector_type(2)));
  constexpr int R4 = LITEVLM_MAX_VISUAL / (4 * kTopkThreads);
  u64x2 a4[R4][2];
  uint32_t f4[R4];
  if (vec) {
#pragma unroll
    for (int i = 0; i < R4; ++i) {
      const int j4 = min(4 * (tid + i * kTopkThreads), V_full - 4);
      a4[i][0] = *reinterpret_cast<const u64x2*>(ac + j4);
      a4[i][1] = *reinterpret_cast<const u64x2*>(ac + j4 + 2);
      if constexpr (!VSEL) {
        // unconditional load (of valid bytes when there is no mask): no branch
        const uint32_t* fp = keep_row ? reinterpret_cast<const uint32_t*>(keep_row + j4)
                                      : reinterpret_cast<const uint32_t*>(ac + j4);
        const uint32_t fraw = *fp;
        f4[i] = keep_row ? fraw : 0x01010101u;
      }
    }
  }
  if constexpr (VSEL) {
    // keep flags from the column sums (dropped keys carry kDroppedCol), and
    // the selection's outputs for this sample
    const uint32_t vm = (uint32_t)view_keep_mask<kFusedViews>(vin, vs.lexical != nullptr, vs.w, vs.tau, vs.N, lane);
    if (view_keep_out && tid < vs.N) view_keep_out[(size_t)b * vs.N + tid] = (uint8_t)((vm >> tid) & 1u);
    uint8_t* row = token_keep_out ? token_keep_out + (size_t)b * S : nullptr;
    const bool row4 = (reinterpret_cast<uintptr_t>(row) & 3) == 0;  // 4 flags per store
    if (vec) {
#pragma unroll
      for (int i = 0; i < R4; ++i) {
        const unsigned long long av[4] = {a4[i][0].x, a4[i][0].y, a4[i][1].x, a4[i][1].y};
        uint32_t f = 0;
#pragma unroll
        for (int u = 0; u < 4; ++u) f |= (uint32_t)(av[u] != kDroppedCol) << (8 * u);
        f4[i] = f;
        const int j4 = 4 * (tid + i * kTopkThreads);
        if (row && j4 < V_full) {
          if (row4) {
            *reinterpret_cast<uint32_t*>(row + j4) = f;
          } else {
#pragma unroll
            for (int u = 0; u < 4; ++u) row[j4 + u] = (uint8_t)((f >> (8 * u)) & 1u);
          }
        }
      }
    } else if (row) {
      for (int j = tid; j < V_full; j += kTopkThreads) row[j] = (uint8_t)(ac[j] != kDroppedCol);
    }
    if (row)
      for (int j = V_full + tid; j < S; j += kTopkThreads) row[j] = 1;
  }

  // Kept-visual counts of samples 0..b, one sample per wave at a time.
  for (int bb = wave; bb <= b; bb += kTopkWaves) {
    int c;
    if constexpr (VSEL) {
      const ViewIn vi = bb == wave ? vinw : view_load(vs.logit, vs.lexical, vs.N, bb, lane);
      const uint32_t m = (uint32_t)view_keep_mask<kFusedViews>(vi, vs.lexical != nullptr, vs.w, vs.tau, vs.N, lane);
      c = 0;
      for (int v = 0; v < vs.N; ++v) c += ((m >> v) & 1u) ? vs.off[v + 1] - vs.off[v] : 0;
    } else {
      c = token_keep ? wave_count_flags(token_keep + (size_t)bb * S, V_full, lane) : V_full;
    }
    if (lane == 0) vcnt[bb] = c;
  }
  for (int i = tid; i < kBins; i += kTopkThreads) hist[i] = 0;

  if (vec) {
#pragma unroll
    for (int i = 0; i < R4; ++i) {
      const int j4 = 4 * (tid + i * kTopkThreads);
      if (j4 < V_full) {
        const unsigned long long av[4] = {a4[i][0].x, a4[i][0].y, a4[i][1].x, a4[i][1].y};
        float sv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const bool kept = ((f4[i] >> (8 * u)) & 0xFFu) != 0u;
          sv[u] = score_of(av[u], kept);
          const uint32_t key = kept ? order_key(sv[u]) : 0u;
          if (kept) {
            kmin = min(kmin, key);
            kmax = max(kmax, key);
          }
          keys[j4 + u] = key;
        }
        *reinterpret_cast<float4*>(sc + j4) = make_float4(sv[0], sv[1], sv[2], sv[3]);
      }
    }
  } else {
    for (int j = tid; j < V_full; j += kTopkThreads) {
      const bool kept = VSEL ? ac[j] != kDroppedCol : (keep_row == nullptr || keep_row[j]);
      const float sv = score_of(ac[j], kept);
      sc[j] = sv;
      const uint32_t key = kept ? order_key(sv) : 0u;
      if (kept) {
        kmin = min(kmin, key);
        kmax = max(kmax, key);
      }
      keys[j] = key;
    }
  }
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
  // compacted offset of this sample: sum over earlier samples of k_bb + T
  int cu_b;
  {
    const int term = tid < b ? keep_count(keep_ratio, vcnt[tid]) + T : 0;
    const int wsm = wave_sum_int(term);
    if (lane == 0) wsum[0][wave] = wsm;
    __syncthreads();
    cu_b = 0;
#pragma unroll
    for (int w = 0; w < kTopkWaves; ++w) cu_b += wsum[0][w];
  }
  const int kb_ = keep_count(keep_ratio, vcnt[b]);
  if (VSEL && n_visual_out && tid == 0) n_visual_out[b] = vcnt[b];

  // Radix select of the kb_-th largest key. Bits above the highest bit where
  // kmin and kmax differ are common to every kept key and are skipped.
  const uint32_t diff = kmin ^ kmax;
  int bits_left = diff ? 32 - __clz((int)diff) : 0;
  uint32_t pmask = bits_left == 32 ? 0u : ~((1u << bits_left) - 1u);
  uint32_t prefix = kmax & pmask;
  int krem = kb_;
  constexpr int KPT = LITEVLM_MAX_VISUAL / kTopkThreads;
  int pass = 0;
  if (kb_ > 0) {
    while (bits_left > 0) {
      const int width = bits_left < kDigitBits ? bits_left : kDigitBits;
      const int shift = bits_left - width;
      const uint32_t dmask = (1u << width) - 1u;
#pragma unroll
      for (int i = 0; i < KPT; ++i) {
        const int j = tid + i * kTopkThreads;
        if (j < V_full) {
          const uint32_t kk = keys[j];
          if (kk != 0u && (kk & pmask) == prefix) atomicAdd(&hist[(kk >> shift) & dmask], 1);
        }
      }
      __syncthreads();
      // thread t owns bins kBinsPer*t ..; "above" counts candidates in higher bins
      int cb[kBinsPer];
      int csum = 0;
#pragma unroll
      for (int u = 0; u < kBinsPer; ++u) {
        cb[u] = hist[kBinsPer * tid + u];
        csum += cb[u];
      }
      int total;
      const int excl = block_scan_excl(csum, wsum[1 + (pass & 1)], &total);
      const int above = total - excl - csum;
      // bins are cleared for the next pass by their owners
#pragma unroll
      for (int u = 0; u < kBinsPer; ++u) hist[kBinsPer * tid + u] = 0;
      if (above < krem && above + csum >= krem) {
        // the bin holding the krem-th largest candidate, from the top bin down
        int a = above, dsel = kBinsPer * tid;
        bool found = false;
#pragma unroll
        for (int u = kBinsPer - 1; u >= 0; --u) {
          if (!found && a + cb[u] >= krem) {
            dsel = kBinsPer * tid + u;
            found = true;
          } else if (!found) {
            a += cb[u];
          }
        }
        sel_digit = dsel;
        sel_above = a;
      }
      __syncthreads();
      prefix |= ((uint32_t)sel_digit) << shift;
      pmask |= dmask << shift;
      krem -= sel_above;
      bits_left -= width;
      ++pass;
    }
  }
  // prefix is now the kb_-th largest key; take every larger key plus the first
  // krem equal keys in position order. One scan of (larger, equal) counts
  // packed as 16-bit halves gives both prefixes.
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
  int tot_packed;
  const int before = block_scan_excl((ngt << 16) | neq, wsum[3], &tot_packed);
  int32_t* out = kept_index + cu_b;
  if (kb_ > 0) {
    int gtr = before >> 16, eqr = before & 0xFFFF;
    for (int j = j0; j < j1; ++j) {
      const uint32_t kk = keys[j];
      if (kk > thr) {
        out[gtr + min(eqr, krem)] = j;
        ++gtr;
      } else if (kk == thr) {
        if (eqr < krem) out[gtr + eqr] = j;
        ++eqr;
      }
    }
  }
  for (int t = tid; t < T; t += kTopkThreads) out[kb_ + t] = V_full + t;
  if (tid == 0) {
    cu_seqlens[b + 1] = cu_b + kb_ + T;
    if (b == 0) cu_seqlens[0] = 0;
  }
}

// ---------------------------------------------------------------- gather
// Each packed row is one token's Q, K and V rows, W = qvec + 2*kvvec 16-byte
// pieces; thread t copies pieces t, t+256, ... of every row, so no thread idles
// on the short K/V rows. A workgroup takes RPI rows per iteration: the
// kept indices are loaded together with cu_seqlens (they need no offset), the
// sample of each row is found by a search of cu_seqlens in LDS, then every
// 16-byte load of the group is issued (from clamped, always-valid addresses)
// before the predicated stores.

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int PPT, int RPI>
__global__ void __launch_bounds__(256)
gather_rows_kernel(int B, int S, const int32_t* __restrict__ kept_index,
                   const int32_t* __restrict__ cu_seqlens, const u32x4* __restrict__ q,
                   const u32x4* __restrict__ k, const u32x4* __restrict__ v, u32x4* __restrict__ qc,
                   u32x4* __restrict__ kc, u32x4* __restrict__ vc, int qvec, int kvvec) {
  __shared__ int cu[LITEVLM_MAX_BATCH + 1];
  const int tid = threadIdx.x;
  const int cap = B * S;
  // segment and offset of this thread's pieces (the same for every row)
  int seg[PPT], off[PPT];
#pragma unroll
  for (int j = 0; j < PPT; ++j) {
    const int p = tid + 256 * j;
    seg[j] = p < qvec ? 0 : (p < qvec + kvvec ? 1 : (p < qvec + 2 * kvvec ? 2 : 3));
    off[j] = seg[j] == 0 ? p : (seg[j] == 1 ? p - qvec : p - qvec - kvvec);
    if ((seg[j] == 0 && !qc) || (seg[j] == 1 && !kc) || (seg[j] == 2 && !vc)) seg[j] = 3;  // not requested
  }
  int base = blockIdx.x * RPI;
  int idx[RPI];
#pragma unroll
  for (int r = 0; r < RPI; ++r) idx[r] = kept_index[min(base + r, cap - 1)];
  for (int i = tid; i <= B; i += blockDim.x) cu[i] = cu_seqlens[i];
  __syncthreads();
  const int total = cu[B];
  for (; base < total; base += gridDim.x * RPI) {
    size_t src[RPI];
#pragma unroll
    for (int r = 0; r < RPI; ++r) {
      const int i = min(base + r, total - 1);
      // last b with cu[b] <= i, by a fixed 8-step search (B <= 256)
      int lo = 0;
#pragma unroll
      for (int step = 128; step >= 1; step >>= 1)
        if (lo + step <= B - 1 && cu[lo + step] <= i) lo += step;
      src[r] = (size_t)lo * S + (base + r < total ? idx[r] : idx[0]);
    }
    // indices of the next iteration, in flight with this one's rows
    const int nbase = base + gridDim.x * RPI;
    if (nbase < total) {
#pragma unroll
      for (int r = 0; r < RPI; ++r) idx[r] = kept_index[min(nbase + r, cap - 1)];
    }
    u32x4 val[RPI][PPT];
#pragma unroll
    for (int r = 0; r < RPI; ++r)
#pragma unroll
      for (int j = 0; j < PPT; ++j) {
        const u32x4* sp = seg[j] == 0 ? q + src[r] * qvec : (seg[j] == 1 ? k + src[r] * kvvec : v + src[r] * kvvec);
        if (seg[j] != 3) val[r][j] = sp[off[j]];
      }
#pragma unroll
    for (int r = 0; r < RPI; ++r) {
      const int i = base + r;
      if (i >= total) continue;
#pragma unroll
      for (int j = 0; j < PPT; ++j) {
        if (seg[j] == 0) qc[(size_t)i * qvec + off[j]] = val[r][j];
        else if (seg[j] == 1) kc[(size_t)i * kvvec + off[j]] = val[r][j];
        else if (seg[j] == 2) vc[(size_t)i * kvvec + off[j]] = val[r][j];
      }
    }
  }
}


// ---------------------------------------------------------------- host launch

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Shapes where sweep 1 may split unevenly over the samples (with the view
// selection inside the call): more than one sample, at most one per wave of
// the workgroup, at least two splits per column to move, and every sample's
// live tiles in kBalWords words.
static bool bal_shape(int B, int ns1, int n_kt) {
  return B > 1 && B <= kBalMaxBatch && ns1 >= 2 && n_kt <= 64 * kBalWords;
}

static ScoreSplit score_split(int B, int S, int V_full, int Hq, int Hkv, int n_query) {
  // Sweep 1: one 16-wave workgroup per CU (256 CUs); the key tiles of each
  // (sample, KV group, row block) are split until the grid has ~256
  // workgroups, at most kMaxSplitTiles tiles to one split. Sweep 2: row chunks
  // are split over workgroups while the grid fits one pass of the chip at
  // three 4-wave workgroups per CU, at most 4 ways (every split merges its
  // rows' statistics again and adds its own column partials), and at least
  // as many ways as keep a workgroup within kMaxChunksPerSplit chunks.
  ScoreSplit p;
  const int R = (Hq / Hkv) * n_query;
  p.n_rb = (R + RBLK - 1) / RBLK;
  p.n_kt = (S + KB - 1) / KB;
  const long long cols = std::max<long long>(1, (long long)B * Hkv * p.n_rb);
  const int want = (int)std::max<long long>(1, 256 / cols);
  p.ns1 = std::max((p.n_kt + kMaxSplitTiles - 1) / kMaxSplitTiles, std::min(p.n_kt, want));
  p.ns1_slots = bal_shape(B, p.ns1, p.n_kt) ? 2 * p.ns1 : p.ns1;
  p.n_vt = (V_full + KT - 1) / KT;
  p.nchunks = (R + CH - 1) / CH;
  const long long c2 = (long long)p.n_vt * Hkv * B;
  const int fit = c2 == 0 ? 1 : (int)std::min<long long>(std::min(p.nchunks, 4), std::max<long long>(1, 768 / c2));
  p.rs2 = std::max(fit, (p.nchunks + kMaxChunksPerSplit - 1) / kMaxChunksPerSplit);
  if (c2 > 768) p.rs2 = std::max(p.rs2, std::min(p.nchunks, 2));
  return p;
}

ScoreWorkspace score_workspace_layout(int B, int S, int V_full, int Hq, int Hkv, int n_query) {
  const ScoreSplit sp = score_split(B, S, V_full, Hq, Hkv, n_query);
  const size_t R = (size_t)(Hq / Hkv) * n_query;
  ScoreWorkspace w;
  w.rowpart_off = 0;
  w.acc_off = align256(w.rowpart_off + sizeof(float2) * B * Hkv * (size_t)sp.ns1_slots * R);
  w.total = align256(w.acc_off + sizeof(unsigned long long) * B * (size_t)V_full);
  return w;
}

// Flat XCD-aware grids: 8 XCDs x (columns per XCD, rounded up) x splits.
static int sweep_grid(long long ncol, int nsplit) { return (int)(8 * ((ncol + 7) / 8) * nsplit); }

template <int DT, int D, bool VSEL>
static void launch_sweeps_v(const ScoreArgs& a, const ScoreDims& d, const ScoreSplit& sp, float2* rowpart,
                            unsigned long long* acc, hipStream_t stream) {
  hipLaunchKernelGGL((score_rowstats_kernel<DT, D, VSEL>),
                     dim3(sweep_grid((long long)a.B * a.Hkv * sp.n_rb, sp.ns1)), dim3(kSweepThreads), 0, stream, d,
                     a.q, a.k, a.token_keep, rowpart, acc);
  if (sp.n_vt > 0)
    hipLaunchKernelGGL((score_colmass_kernel<DT, D, VSEL>),
                       dim3(sweep_grid((long long)a.B * a.Hkv * sp.n_vt, sp.rs2)), dim3(64 * kColWaves), 0, stream,
                       d, a.q, a.k, a.token_keep, rowpart, acc);
}

template <int DT, int D>
static void launch_sweeps(const ScoreArgs& a, const ScoreDims& d, const ScoreSplit& sp, float2* rowpart,
                          unsigned long long* acc, hipStream_t stream) {
  if (d.vs.N > 0) launch_sweeps_v<DT, D, true>(a, d, sp, rowpart, acc, stream);
  else launch_sweeps_v<DT, D, false>(a, d, sp, rowpart, acc, stream);
}

hipError_t launch_token_score_topk(const ScoreArgs& a, hipStream_t stream) {
  const ScoreWorkspace w = score_workspace_layout(a.B, a.S, a.V_full, a.Hq, a.Hkv, a.query_rows);
  const ScoreSplit sp = score_split(a.B, a.S, a.V_full, a.Hq, a.Hkv, a.query_rows);
  char* ws = static_cast<char*>(a.workspace);
  float2* rowpart = reinterpret_cast<float2*>(ws + w.rowpart_off);
  unsigned long long* acc = reinterpret_cast<unsigned long long*>(ws + w.acc_off);
  ScoreDims d;
  d.B = a.B;
  d.S = a.S;
  d.V_full = a.V_full;
  d.T = a.query_rows;
  d.tq0 = a.S - a.V_full - a.query_rows;
  d.Hq = a.Hq;
  d.Hkv = a.Hkv;
  d.G = a.Hq / a.Hkv;
  d.R = d.G * d.T;
  d.n_rb = sp.n_rb;
  d.n_kt = sp.n_kt;
  // with the view selection inside the call, every workgroup can find the
  // live tiles of every sample, and sweep 1 splits them evenly
  d.bal = a.vs.N > 0 && bal_shape(a.B, sp.ns1, sp.n_kt) ? 1 : 0;
  d.ns1u = sp.ns1;
  d.ns1 = d.bal ? sp.ns1_slots : sp.ns1;
  d.n_vt = sp.n_vt;
  d.nchunks = sp.nchunks;
  d.rs2 = sp.rs2;
  d.scale_log2 = a.logit_scale_log2;
  d.vs = a.vs;
  // A text row adds at most 1 to a column, so a column sum is at most Hq*T:
  // with Hq*T <= 2^e, fx = 2^(62-e) keeps every sum below 2^62.
  const double rows = (double)a.Hq * (double)d.T;
  int e = 0;
  while (std::ldexp(1.0, e) < rows) ++e;
  d.fx = std::ldexp(1.0f, 62 - e);
  const double inv = 1.0 / ((double)d.fx * rows);

#define LITEVLM_SWEEPS(DT)                                           \
  (a.D == 128 ? launch_sweeps<DT, 128>(a, d, sp, rowpart, acc, stream) \
              : launch_sweeps<DT, 64>(a, d, sp, rowpart, acc, stream))
  if (a.dtype == LITEVLM_BF16) LITEVLM_SWEEPS(LITEVLM_BF16);
  else if (a.dtype == LITEVLM_FP8_E4M3) LITEVLM_SWEEPS(LITEVLM_FP8_E4M3);
  else LITEVLM_SWEEPS(LITEVLM_F32);
#undef LITEVLM_SWEEPS

  if (a.vs.N > 0)
    hipLaunchKernelGGL(topk_compact_kernel<true>, dim3(a.B), dim3(kTopkThreads), 0, stream, a.S, a.V_full,
                       a.keep_ratio, a.token_keep, acc, inv, a.scores, a.kept_index, a.cu_seqlens, a.vs,
                       a.view_keep, a.token_keep_out, a.n_visual_kept);
  else
    hipLaunchKernelGGL(topk_compact_kernel<false>, dim3(a.B), dim3(kTopkThreads), 0, stream, a.S, a.V_full,
                       a.keep_ratio, a.token_keep, acc, inv, a.scores, a.kept_index, a.cu_seqlens, a.vs,
                       nullptr, nullptr, nullptr);
  if (a.qc || a.kc || a.vc) {
    const int esz = a.dtype == LITEVLM_F32 ? 4 : (a.dtype == LITEVLM_BF16 ? 2 : 1);
    launch_gather(a.B, a.S, a.kept_index, a.cu_seqlens, a.q, a.k, a.v, a.qc, a.kc, a.vc,
                  a.Hq * a.D * esz / 16, a.Hkv * a.D * esz / 16, stream);
  }

  return hipGetLastError();
}

void launch_gather(int B, int S, const int32_t* kept_index, const int32_t* cu_seqlens, const void* q,
                   const void* k, const void* v, void* qc, void* kc, void* vc, int qvec, int kvvec,
                   hipStream_t stream) {
  const int rows = B * S;
  auto launch = [&](auto kernel, int rpi) {
    const int grid = std::max(1, std::min(1024, (rows + rpi - 1) / rpi));
    hipLaunchKernelGGL(kernel, dim3(grid), dim3(256), 0, stream, B, S, kept_index, cu_seqlens,
                       static_cast<const u32x4*>(q), static_cast<const u32x4*>(k), static_cast<const u32x4*>(v),
                       static_cast<u32x4*>(qc), static_cast<u32x4*>(kc), static_cast<u32x4*>(vc), qvec, kvvec);
  };
  // 16-byte pieces per thread and row, (Q + K + V pieces) / 256: at most
  // (4096 + 2*4096) / 256 = 48 with Hq <= LITEVLM_MAX_HEADS (or a hidden-state
  // row of up to 196 KB); about 12-24 loads in flight per thread. At 3 pieces
  // (the 32/8-head, D = 128 bf16 rows) 4 rows per workgroup spread the rows
  // over more workgroups than 8 did and measured faster (6 us at the batch-8
  // workload, equal at batch 1).
  const int ppt = (qvec + 2 * kvvec + 255) / 256;
  if (ppt <= 1) launch(gather_rows_kernel<1, 8>, 8);
  else if (ppt <= 2) launch(gather_rows_kernel<2, 8>, 8);
  else if (ppt <= 3) launch(gather_rows_kernel<3, 4>, 4);
  else if (ppt <= 4) launch(gather_rows_kernel<4, 6>, 6);
  else if (ppt <= 6) launch(gather_rows_kernel<6, 4>, 4);
  else if (ppt <= 12) launch(gather_rows_kernel<12, 2>, 2);
  else if (ppt <= 24) launch(gather_rows_kernel<24, 1>, 1);
  else launch(gather_rows_kernel<48, 1>, 1);
}

hipError_t launch_gather_hidden(int B, int S, int row_bytes, const void* hidden, const int32_t* kept_index,
                                const int32_t* cu_seqlens, void* out, hipStream_t stream) {
  launch_gather(B, S, kept_index, cu_seqlens, hidden, nullptr, nullptr, out, nullptr, nullptr, row_bytes / 16, 0,
                stream);
  return hipGetLastError();
}

}  // namespace litevlm
