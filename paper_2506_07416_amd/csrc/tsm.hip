// Token Selection Module front end: the scoring queries and keys of the
// standalone first decoder layer, from the layer's input hidden states.
//
//   k[b, j]   = rope(r_j * x[b, j] W_k'^T, pos_j)   for every kept token j
//   q[b, t]   = rope(r_t * x[b, t] W_q'^T, pos_t)   for the text tokens t
//   r_j       = 1 / sqrt(mean_c x[b, j, c]^2 + eps)  (RMS normalisation)
//   pos_j     = number of kept tokens before j (positions of the patch-selected sequence)
//
// W' carries the normalisation gain (W'[n, c] = W[n, c] * gamma[c],
// tsm_fold_gain_kernel), so the projection is a plain bf16 GEMM on MFMA with
// fp32 accumulation, and the RMS factor and the rotary embedding are applied
// in its epilogue:
//   - the sum of squares of each row comes from the A operands the waves
//     already hold for the MFMAs (no second pass over x);
//   - a wave owns two column blocks that are rotary partners (elements d and
//     d + D/2 of one head), so the rotation is lane-local in the accumulators.
//
// Tiling (the defaults below): a workgroup (4 waves) computes 128 rows x 128
// output features; wave (wr, wc) holds rows 64*wr .. +64 and the column blocks
// c0 and c0 + D/64. A and B tiles of 64 columns of the model width stream
// global -> LDS directly (global_load_lds_dwordx4) through a double buffer
// (66 KB, two workgroups per CU) into 128-byte rows whose 16-byte pieces are
// XOR-swizzled so that operand reads are free of bank conflicts. Measured
// alternatives (256-row or 256-feature tiles, 3- to 6-stage rings, 32-column
// stages, four workgroups per CU with 32-column stages) were slower or equal on
// both the batch-1 and the batch-8 shapes.
//
// Epilogue: the rotation angle is reduced to [-1/2, 1/2] turns in double and
// taken by the hardware sine and cosine (which work in turns), and the rotated
// tile is staged through the free ring as bf16 rows so that it leaves in
// 16-byte stores of whole rows; the accumulators hold one feature per lane.
#include <type_traits>

#include "common.hpp"
#include "launch.hpp"

namespace litevlm {
namespace {

// Staging: 64 columns of the model width per stage, double buffered.
constexpr int kKT = 64, kStages = 2;  // Dm % kKT == 0 (host check)
constexpr int kPieces = kKT / 8;      // 16-byte pieces per staged row
constexpr int kRowB = kKT * 2;        // bytes per staged row

// Workgroup tile MT rows x NT features over NW waves; each wave holds 64 rows
// (two 32-row blocks) and NT / (NW / (MT / 64)) features.
template <int MT, int NT, int NW>
struct TsmTile {
  static constexpr int kAB = MT * kRowB;  // A tile bytes per stage
  static constexpr int kBB = NT * kRowB;  // B tile bytes per stage
  static constexpr int kStageB = kAB + kBB;
  static constexpr int kRingB = kStages * kStageB;
  static constexpr int kLdsB =
      kRingB + MT * 4 /* row factors */ + MT * 4 /* positions */ + 128 /* reductions */ + MT /* keep flags */;
  static constexpr int kWgPerCu = (160 * 1024 / kLdsB) >= 2 ? 2 : 1;
  static constexpr int kThreads = 64 * NW;
  static constexpr int kNWR = MT / 64;       // waves along the rows
  static constexpr int kNWC = NW / kNWR;     // waves along the features (share rows)
  static constexpr int kCBW = NT / kNWC / 32;  // 32-feature blocks per wave
  static_assert(kNWR * kNWC == NW && (kCBW == 2 || kCBW == 4), "tile shape");
};

struct TsmParams {
  const uint8_t* x;     // bf16 [B, S, Dm]
  const uint8_t* keep;  // uint8 [B, S] or NULL
  const uint8_t* wq;    // bf16 [Hq*D, Dm]
  const uint8_t* wk;    // bf16 [Hkv*D, Dm]
  uint16_t* q;          // bf16 [B, S, Hq, D]
  uint16_t* k;          // bf16 [B, S, Hkv, D]
  int B, S, V_full, Dm, Hq, Hkv;
  int mk, nk, mq, nq, gk, gq, per_xcd;  // gk, gq: key and query row tiles (B*mk, B*mq)
  int compact;                          // deal the working key row tiles by rank (kMT = 256 only)
  float eps;
  double log2_theta;
};

template <int N>
__device__ __forceinline__ void vm_wait() {
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// XOR swizzle of a staged row's pieces. The LDS serves a 16-byte read for 16
// lanes per cycle across 64 banks (256 bytes): the 16 consecutive rows such a
// group reads must put their pieces in distinct 16-byte bank slots. A 256-byte
// bank window holds 256 / (2*kKT) rows, so rows that share a window position
// get distinct pieces.
__device__ __forceinline__ int swz(int row) { return kPieces == 4 ? (row >> 2) & 3 : (row >> 1) & 7; }

// Workgroup barrier that waits only for this wave's LDS operations: the
// __syncthreads fence would also wait for every direct copy still in flight,
// which would drain the ring each stage.
__device__ __forceinline__ void ring_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ __forceinline__ int acc_row(int r, int hl) { return 8 * (r >> 2) + 4 * hl + (r & 3); }

typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));

// x.lo*y.lo + x.hi*y.hi + c on packed bf16 pairs (fp32 accumulate).
__device__ __forceinline__ float dot2_bf16(uint32_t x, uint32_t y, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2v, x), __builtin_bit_cast(bf16x2v, y), c, false);
}

template <int D, int MT, int NT, int NW>
__global__ __launch_bounds__(64 * NW, (TsmTile<MT, NT, NW>::kWgPerCu)) void tsm_proj_kernel(TsmParams p) {
  using Tl = TsmTile<MT, NT, NW>;
  constexpr int kMT = MT, kNT = NT, kAB = Tl::kAB, kBB = Tl::kBB, kStageB = Tl::kStageB, kRingB = Tl::kRingB;
  constexpr int kTh = Tl::kThreads, NWR = Tl::kNWR, NWC = Tl::kNWC;
  constexpr int PB = D / 64;     // column-block distance of rotary partners
  constexpr int RB = 2;          // 32-row blocks per wave
  constexpr int CBW = Tl::kCBW;  // 32-column blocks per wave
  __shared__ __attribute__((aligned(1024))) uint8_t lds[Tl::kLdsB];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  bool isq;
  int b, mt, nt;
  if (MT == 256 && p.compact) {
    // Only the key row tiles that hold a kept row produce anything. Every
    // workgroup finds them from the keep bytes (one wave per tile in turn,
    // four bytes a lane) and deals them, with their feature tiles, to the
    // XCDs round robin by rank: each XCD gets the same number of working
    // items whatever the dropped views, and a row tile's feature tiles stay on
    // one XCD (they share its rows of x in that L2). The query items follow,
    // continuing the rotation. The flags go into the ring, unused until the
    // stage copies start.
    uint8_t* gf = lds;
    for (int g0 = 0; g0 < p.gk; g0 += 8 * NW) {
      uint32_t any8 = 0;
      uint8_t kb[8][4];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int g = g0 + u * NW + w;
        const int gb = g / p.mk, r0 = (g % p.mk) * kMT;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = r0 + lane + 64 * e;  // kMT = 256 rows: 64 lanes x 4
          kb[u][e] = (g < p.gk && r < p.S) ? p.keep[(size_t)gb * p.S + r] : 0;
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const bool kept = (kb[u][0] | kb[u][1] | kb[u][2] | kb[u][3]) != 0;
        any8 |= (__ballot(kept) != 0ull ? 1u : 0u) << u;
      }
      if (lane == 0) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int g = g0 + u * NW + w;
          if (g < p.gk) gf[g] = (uint8_t)((any8 >> u) & 1u);
        }
      }
    }
    __syncthreads();
    // the working tile of rank x + 8*(j / nk), and the number of working tiles
    // (every wave computes the same values)
    const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
    const int rk = x + 8 * (j / p.nk);
    int nwork = 0, grp = 0;
    for (int c0 = 0; c0 < p.gk; c0 += 64) {
      const bool f = c0 + lane < p.gk && gf[c0 + lane] != 0;
      const uint64_t m = __ballot(f);
      const int cnt = __popcll(m);
      if (rk >= nwork && rk < nwork + cnt) {
        const int before = __popcll(m & ((1ull << lane) - 1ull));
        const uint64_t sel = __ballot(f && before == rk - nwork);
        grp = c0 + __ffsll((unsigned long long)sel) - 1;
      }
      nwork += cnt;
    }
    const int ck = nwork > x ? (nwork - x + 7) / 8 : 0;  // working key tiles of this XCD
    if (j < ck * p.nk) {
      isq = false;
      b = grp / p.mk;
      mt = grp % p.mk;
      nt = j % p.nk;
    } else {
      const int qi = (x - nwork % 8 + 8) % 8 + 8 * (j - ck * p.nk);
      if (qi >= p.gq * p.nq) return;
      isq = true;
      b = qi / (p.mq * p.nq);
      const int r = qi % (p.mq * p.nq);
      mt = r / p.nq;
      nt = r % p.nq;
    }
  } else {
    // an XCD takes a contiguous item range
    const int item = (blockIdx.x & 7) * p.per_xcd + (blockIdx.x >> 3);
    const int n_k_items = p.gk * p.nk;
    if (item >= n_k_items + p.gq * p.nq) return;
    if (item < n_k_items) {
      isq = false;
      b = item / (p.mk * p.nk);
      const int r = item % (p.mk * p.nk);
      mt = r / p.nk;
      nt = r % p.nk;
    } else {
      const int jq = item - n_k_items;
      isq = true;
      b = jq / (p.mq * p.nq);
      const int r = jq % (p.mq * p.nq);
      mt = r / p.nq;
      nt = r % p.nq;
    }
  }
  const int row0 = (isq ? p.V_full : 0) + mt * kMT;  // first row of the tile within the sample
  const int nrows = min(kMT, p.S - row0);
  const int n0 = nt * kNT;
  const uint8_t* W = isq ? p.wq : p.wk;
  const int H = isq ? p.Hq : p.Hkv;
  const int Dm = p.Dm;

  float* rs = reinterpret_cast<float*>(lds + kRingB);
  int* pos = reinterpret_cast<int*>(lds + kRingB + kMT * 4);
  int* red = reinterpret_cast<int*>(lds + kRingB + kMT * 8);
  uint8_t* kflag = lds + kRingB + kMT * 8 + 128;

  const int wr = w % NWR, wc = w / NWR, hl = lane >> 5, l32 = lane & 31;

  // ---- positions of the tile's rows in the patch-selected sequence
  {
    const uint8_t* kr = p.keep ? p.keep + (size_t)b * p.S : nullptr;
    int cnt = 0;
    if (kr)
      for (int j = tid; j < row0; j += kTh) cnt += kr[j];
#pragma unroll
    for (int x = 1; x < kWave; x <<= 1) cnt += __shfl_xor(cnt, x, kWave);
    if (lane == 0) red[w] = cnt;
    __syncthreads();
    int base = row0;
    if (kr) {
      base = 0;
      for (int x = 0; x < NW; ++x) base += red[x];
    }
    for (int t0 = 0; t0 < kMT; t0 += kTh) {
      const int t = t0 + tid;
      int f = 0;
      if (t < nrows) f = kr ? kr[row0 + t] : 1;
      int incl = f;
#pragma unroll
      for (int x = 1; x < kWave; x <<= 1) {
        const int y = __shfl_up(incl, x, kWave);
        if (lane >= x) incl += y;
      }
      __syncthreads();
      if (lane == kWave - 1) red[NW + w] = incl;
      __syncthreads();
      int before = t0 == 0 ? 0 : red[2 * NW];  // kept rows of the earlier chunks
      for (int x = 0; x < w; ++x) before += red[NW + x];
      if (t < kMT) {
        pos[t] = base + before + (incl - f);
        kflag[t] = (uint8_t)f;
      }
      __syncthreads();
      if (tid == 0) {
        int c = t0 == 0 ? 0 : red[2 * NW];
        for (int x = 0; x < NW; ++x) c += red[NW + x];
        red[2 * NW] = c;
      }
    }
  }

  // ---- a key tile whose rows are all dropped tokens produces nothing: the
  // keys of dropped views are never scored
  if (!isq && p.keep) {
    __syncthreads();
    if (red[2 * NW] == 0) return;
  }

  // ---- per-lane copy sources (fixed) and operand offsets (fixed)
  // copy j of a wave fills LDS pieces (w + 4j)*64 + lane of the A (resp. B) tile
  constexpr int CA = kAB / (1024 * NW), CB = kBB / (1024 * NW);  // copies per thread per stage
  size_t asrc[CA], bsrc[CB];
#pragma unroll
  for (int j = 0; j < CA; ++j) {
    const int slot = (w + NW * j) * 64 + lane;
    const int row = slot / kPieces, logical = (slot % kPieces) ^ swz(row);
    asrc[j] = ((size_t)((size_t)b * p.S + row0 + min(row, nrows - 1)) * Dm + logical * 8) * 2;
  }
#pragma unroll
  for (int j = 0; j < CB; ++j) {
    const int slot = (w + NW * j) * 64 + lane;
    const int row = slot / kPieces, logical = (slot % kPieces) ^ swz(row);
    bsrc[j] = ((size_t)(n0 + row) * Dm + logical * 8) * 2;
  }
  const uint32_t lds_w = __builtin_amdgcn_readfirstlane((uint32_t)w * 1024u);
  // this wave's column blocks: rotary partners (blocks PB apart) always together
  int cbl[CBW];
  if constexpr (CBW == 4) {
#pragma unroll
    for (int i = 0; i < 4; ++i) cbl[i] = 4 * wc + i;
  } else {  // two waves share a 128-feature span: blocks {c0, c0 + PB}
    cbl[0] = (D == 128) ? wc : 2 * wc;
    cbl[1] = cbl[0] + PB;
  }
  constexpr int KS = kKT / 16;          // k16 steps per stage
  uint32_t aoff[RB][KS], boff[CBW][KS];  // [block][k16 step]
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const int logical = 2 * ks + hl;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int row = 64 * wr + 32 * rb + l32;
      aoff[rb][ks] = row * kRowB + ((logical ^ swz(row)) * 16);
    }
#pragma unroll
    for (int c = 0; c < CBW; ++c) {
      const int nrow = 32 * cbl[c] + l32;
      boff[c][ks] = kAB + nrow * kRowB + ((logical ^ swz(nrow)) * 16);
    }
  }

  auto copy_stage = [&](int s) __attribute__((always_inline)) {
    const size_t kb = (size_t)s * kKT * 2;
    uint8_t* st = lds + (s % kStages) * kStageB;
#pragma unroll
    for (int j = 0; j < CA; ++j)
      __builtin_amdgcn_global_load_lds((const void*)(p.x + asrc[j] + kb),
                                       (__attribute__((address_space(3))) void*)(st + lds_w + NW * j * 1024), 16, 0, 0);
#pragma unroll
    for (int j = 0; j < CB; ++j)
      __builtin_amdgcn_global_load_lds((const void*)(W + bsrc[j] + kb),
                                       (__attribute__((address_space(3))) void*)(st + kAB + lds_w + NW * j * 1024), 16,
                                       0, 0);
  };

  f32x16 acc[RB][CBW];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int c = 0; c < CBW; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[rb][c][r] = 0.f;
  float ssq[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) ssq[rb] = 0.f;

  const int nK = Dm / kKT;
  constexpr int CS = CA + CB;  // copies per thread per stage
  static_assert(CS * (kStages - 2) <= 63 && kStages >= 2 && kStages <= 6, "vmcnt range");
  for (int s = 0; s < kStages - 1 && s < nK; ++s) copy_stage(s);
  for (int s = 0; s < nK; ++s) {
    // stage s has landed once at most the copies of the stages issued after it remain
    const int later = min(nK - 1, s + kStages - 2) - s;
    if (later >= 4) vm_wait<4 * CS>();
    else if (later == 3) vm_wait<3 * CS>();
    else if (later == 2) vm_wait<2 * CS>();
    else if (later == 1) vm_wait<CS>();
    else vm_wait<0>();
    ring_barrier();  // every wave's copies of stage s are visible; ring slot (s-1)%kStages is free
    if (s + kStages - 1 < nK) copy_stage(s + kStages - 1);
    const uint8_t* st = lds + (s % kStages) * kStageB;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      bf16x8 a[RB], bo[CBW];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) a[rb] = *reinterpret_cast<const bf16x8*>(st + aoff[rb][ks]);
#pragma unroll
      for (int c = 0; c < CBW; ++c) bo[c] = *reinterpret_cast<const bf16x8*>(st + boff[c][ks]);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int c = 0; c < CBW; ++c)
          acc[rb][c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[rb], bo[c], acc[rb][c], 0, 0, 0);
      // Row sums of squares from the A operands on the packed bf16 dot unit. The
      // two waves holding the same rows take alternate k16 steps, so every SIMD
      // carries the same vector work.
      if ((ks % NWC) == wc) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const u32x4v u = __builtin_bit_cast(u32x4v, a[rb]);
#pragma unroll
          for (int e = 0; e < 4; ++e) ssq[rb] = dot2_bf16(u[e], u[e], ssq[rb]);
        }
      }
    }
  }

  // ---- epilogue: RMS factor per row, rotary embedding, bf16 store
  // (the ring is free now: its first bytes hold the wc = 1 waves' partial sums)
  float* part = reinterpret_cast<float*>(lds);  // [NWC][kMT]
  __syncthreads();
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const float tot = sum_xor32(ssq[rb]);
    if (hl == 0) part[wc * kMT + 64 * wr + 32 * rb + l32] = tot;
  }
  __syncthreads();
  if (wc == 0 && hl == 0) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int row = 64 * wr + 32 * rb + l32;
      float tot = 0.f;
      for (int x = 0; x < NWC; ++x) tot += part[x * kMT + row];
      rs[row] = 1.f / sqrtf(tot / (float)Dm + p.eps);
    }
  }
  __syncthreads();
  // The rotated tile goes through the (now free) ring as bf16 rows of kNT
  // features, 16-byte pieces XOR-swizzled by row, and leaves it in 16-byte
  // stores of whole rows (the accumulators hold one feature per lane).
  static_assert(kMT * kNT * 2 <= kRingB, "output tile exceeds the ring");
  constexpr int kOutRowB = kNT * 2;
  auto out_slot = [&](int row, int col) {
    return row * kOutRowB + ((((col * 2) >> 4) ^ (row & 7)) << 4) + ((col * 2) & 15);
  };
  // rotary pairs of this wave's column list: slots c (a first-half block) and
  // cp (its partner, PB blocks on)
  auto rotate_pair = [&](auto ic) __attribute__((always_inline)) {
    constexpr int i = decltype(ic)::value;
    constexpr int c = CBW == 2 ? 0 : (D == 128 ? i : 2 * i);
    constexpr int cp = CBW == 2 ? 1 : c + PB;
    const int col = 32 * cbl[c] + l32;  // tile feature of the first-half element; its partner is D/2 on
    const int d = (32 * cbl[c]) % D + l32;  // element of the first half of its head (d < D/2)
    const double turns_per_pos = exp2(-(2.0 * d / D) * p.log2_theta) * 0.15915494309189535;  // / (2 pi)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 64 * wr + 32 * rb + acc_row(r, hl);
        const float f = rs[row];
        const float x1 = acc[rb][c][r] * f, x2 = acc[rb][cp][r] * f;
        // angle pos * theta^(-2d/D) in turns, reduced to [-1/2, 1/2] in double;
        // the hardware sine and cosine take turns
        double t = (double)pos[row] * turns_per_pos;
        t -= rint(t);
        const float sn = __builtin_amdgcn_sinf((float)t), cs = __builtin_amdgcn_cosf((float)t);
        *reinterpret_cast<uint16_t*>(lds + out_slot(row, col)) = f32_to_bf16_bits(x1 * cs - x2 * sn);
        *reinterpret_cast<uint16_t*>(lds + out_slot(row, col + D / 2)) = f32_to_bf16_bits(x2 * cs + x1 * sn);
        __builtin_amdgcn_sched_barrier(0);  // one row at a time: bounded live ranges
      }
  };
  rotate_pair(std::integral_constant<int, 0>{});
  if constexpr (CBW == 4) rotate_pair(std::integral_constant<int, 1>{});
  __syncthreads();
  // rows of the tile that exist and are kept (queries: every text row)
  uint16_t* out = isq ? p.q : p.k;
  constexpr int kPiecesPerRow = kOutRowB / 16;
#pragma unroll
  for (int j = 0; j < kMT * kPiecesPerRow / kTh; ++j) {
    const int q = tid + kTh * j;
    const int row = q / kPiecesPerRow, pc = q % kPiecesPerRow;
    if (row < nrows && (isq || kflag[row])) {
      const u32x4v v = *reinterpret_cast<const u32x4v*>(lds + row * kOutRowB + ((pc ^ (row & 7)) << 4));
      *reinterpret_cast<u32x4v*>(out + ((size_t)b * p.S + row0 + row) * H * D + n0 + 8 * pc) = v;
    }
  }
}

// w_out[n, c] = bf16(w[n, c] * gamma[c]): the RMS normalisation gain folded
// into the projection that follows it (done once per set of weights).
__global__ __launch_bounds__(256) void tsm_fold_gain_kernel(const uint16_t* __restrict__ w,
                                                            const float* __restrict__ gamma,
                                                            uint16_t* __restrict__ w_out, int64_t rows, int cols) {
  const int64_t n = rows * cols;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    w_out[i] = f32_to_bf16_bits(bf16_bits_to_f32(w[i]) * gamma[i % cols]);
}

}  // namespace

hipError_t launch_tsm_qk(const TsmArgs& a, hipStream_t stream) {
  TsmParams p;
  p.x = static_cast<const uint8_t*>(a.hidden);
  p.keep = a.token_keep;
  p.wq = static_cast<const uint8_t*>(a.w_q);
  p.wk = static_cast<const uint8_t*>(a.w_k);
  p.q = static_cast<uint16_t*>(a.q);
  p.k = static_cast<uint16_t*>(a.k);
  p.B = a.B;
  p.S = a.S;
  p.V_full = a.V_full;
  p.Dm = a.Dm;
  p.Hq = a.Hq;
  p.Hkv = a.Hkv;
  p.eps = a.eps;
  p.log2_theta = log2((double)a.rope_theta);
  const int T = a.S - a.V_full;
  auto setup = [&](int MT, int NT) {
    p.mk = (a.S + MT - 1) / MT;
    p.nk = a.Hkv * a.D / NT;
    p.mq = (T + MT - 1) / MT;
    p.nq = a.Hq * a.D / NT;
    p.gk = a.B * p.mk;
    p.gq = a.B * p.mq;
    p.compact = 0;
    p.per_xcd = (p.gk * p.nk + p.gq * p.nq + 7) / 8;
    return dim3(8 * p.per_xcd);
  };
  // 256 x 256 tiles (8 waves, one workgroup per CU) halve the L2 traffic per
  // flop; they are used when they still give every CU a workgroup.
  const bool big = (a.Hkv * a.D) % 256 == 0 && (a.Hq * a.D) % 256 == 0 &&
                   (int64_t)a.B * ((a.S + 255) / 256) * (a.Hkv * a.D / 256) >= 256;
  if (big) {
    dim3 grid = setup(256, 256);
    // the dealing workgroups keep one flag byte per key row tile in the stage
    // ring: longer batches take the contiguous ranges
    if (a.token_keep && p.gk <= TsmTile<256, 256, 8>::kRingB) {
      // at most (gk+7)/8 working key row tiles per XCD, and (gq*nq+7)/8 query items
      p.compact = 1;
      p.per_xcd = (p.gk + 7) / 8 * p.nk + (p.gq * p.nq + 7) / 8;
      grid = dim3(8 * p.per_xcd);
    }
    if (a.D == 128) hipLaunchKernelGGL((tsm_proj_kernel<128, 256, 256, 8>), grid, dim3(512), 0, stream, p);
    else hipLaunchKernelGGL((tsm_proj_kernel<64, 256, 256, 8>), grid, dim3(512), 0, stream, p);
  } else {
    const dim3 grid = setup(128, 128);
    if (a.D == 128) hipLaunchKernelGGL((tsm_proj_kernel<128, 128, 128, 4>), grid, dim3(256), 0, stream, p);
    else hipLaunchKernelGGL((tsm_proj_kernel<64, 128, 128, 4>), grid, dim3(256), 0, stream, p);
  }
  return hipGetLastError();
}

hipError_t launch_tsm_fold_gain(const void* w, const float* gamma, void* w_out, int rows, int cols,
                                hipStream_t stream) {
  const int64_t n = (int64_t)rows * cols;
  const int64_t blocks = (n + 255) / 256;
  const dim3 grid((unsigned)(blocks < 4096 ? blocks : 4096));
  hipLaunchKernelGGL(tsm_fold_gain_kernel, grid, dim3(256), 0, stream, static_cast<const uint16_t*>(w), gamma,
                     static_cast<uint16_t*>(w_out), (int64_t)rows, cols);
  return hipGetLastError();
}

}  // namespace litevlm
