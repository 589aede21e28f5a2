// Causal GQA prefill attention over packed variable-length sequences: the
// quadratic part of the LLM prefill that token compression shrinks
// (Introduction; Related Work, Visual Token Compression; Figure 3b; FP8 from
// the Experiments section, Deployment paragraph).
//
// Flash-style forward with fp32 accumulation and an online softmax in the
// exp2 domain. A workgroup owns 128 query rows of one query head (4 waves x 32
// rows) and streams the keys of its KV head in 64-key tiles through LDS.
//
// Both products are formed transposed so that a lane owns one query row
// throughout: S^T = K Q^T puts query (lane % 32) in the accumulator columns,
// and O^T = V^T P^T keeps the same ownership for the output, so the running
// max / sum / rescale of a row never leave the two lanes (lane, lane ^ 32)
// that hold it. Q stays in registers as the B operand. K rows are read as the
// A operand in a permuted order chosen so that the exponentiated accumulator
// of S^T is already the B operand of the P.V product; V stays row-major in LDS
// and the LDS transpose reads (ds_read_b64_tr_b16 / _b8) build its A operand.
#include <type_traits>

#include "common.hpp"
#include "launch.hpp"

namespace litevlm {

struct AttnParams {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* cu;
  void* o;
  int B, Hq, Hkv, G, n_mtiles, n_work, per_xcd;
  int Hw, P;  // pipelined bf16 path: query heads per workgroup, 32-position blocks per workgroup
  float scale_log2, out_scale;
};

// max(a, b, c): the NaN-propagating maximum, which folds into one
// v_maximum3_f32 (no canonicalisation).
__device__ __forceinline__ float max3f(float a, float b, float c) {
  return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}

// Maximum of the 32 accumulator values s[0][0..15], s[1][0..15] as a tree of
// 16 three-input maxima, depth 4.
__device__ __forceinline__ float max32(const f32x16 s[2]) {
  float t[11];
#pragma unroll
  for (int i = 0; i < 10; ++i) {
    const int a = 3 * i, b = 3 * i + 1, c = 3 * i + 2;
    t[i] = max3f(s[a >> 4][a & 15], s[b >> 4][b & 15], s[c >> 4][c & 15]);
  }
  t[10] = max3f(s[1][14], s[1][15], t[9]);
  const float u0 = max3f(t[0], t[1], t[2]), u1 = max3f(t[3], t[4], t[5]), u2 = max3f(t[6], t[7], t[8]);
  return max3f(u0, u1, __builtin_elementwise_maximum(u2, t[10]));
}

// Row of the 32x32 accumulator held in register r by lane half hl.
__device__ __forceinline__ int acc_row32(int r, int hl) { return 8 * (r >> 2) + 4 * hl + (r & 3); }
// Swap bits 2 and 3: the K-row order that lines S^T up with the P.V operand.
__device__ __forceinline__ int swap23(int x) { return (x & ~12) | ((x & 4) << 1) | ((x & 8) >> 1); }

template <int OUT>
__device__ __forceinline__ void store_out(void* o, size_t idx, float x) {
  if (OUT == LITEVLM_BF16) static_cast<uint16_t*>(o)[idx] = f32_to_bf16_bits(x);
  else static_cast<float*>(o)[idx] = x;
}

// Key (within the 64-key tile) held by S^T block nb, accumulator row rho.
// bf16: P.V k-steps of 16 keys, lane half hl holding keys 8*hl..8*hl+7 of a
// step, so row rho of block nb is key 32*nb + swap23(rho).
// fp8: one P.V k-step of 64 keys, lane half hl holding keys 32*hl..32*hl+31,
// so row rho of block nb is key 32*bit2(rho) + 16*nb + 4*(rho>>3) + (rho&3).
template <bool FP8>
__device__ __forceinline__ int tile_key(int nb, int rho) {
  if (FP8) return 32 * ((rho >> 2) & 1) + 16 * nb + 4 * (rho >> 3) + (rho & 3);
  return 32 * nb + swap23(rho);
}

// Work item of a flat grid. Items are ordered (KV head, query tile heaviest
// first, sample, head in group) and dealt to the 8 XCDs in contiguous ranges:
// an XCD owns whole KV heads across the batch, so workgroups sharing K/V sit
// behind the same L2 while ragged samples spread evenly over the XCDs, and
// within an XCD the longest causal tiles start first.
__device__ __forceinline__ bool decode_work(const AttnParams& p, int& b, int& h, int& mt) {
  const int L = blockIdx.x;
  const int w = (L & 7) * p.per_xcd + (L >> 3);
  if (w >= p.n_work) return false;
  const int hh = w % p.G;
  int rest = w / p.G;
  b = rest % p.B;
  rest /= p.B;
  const int mrev = rest % p.n_mtiles;
  const int g = rest / p.n_mtiles;
  h = g * p.G + hh;
  mt = p.n_mtiles - 1 - mrev;
  return true;
}

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Output of a wave's 32 query rows: o[db][r] holds element db*32 +
// acc_row32(r, hl) of row lane % 32 (the O^T accumulators). The block goes
// through the wave's 32 rows of free LDS at ob (2*D bytes a row) as bf16,
// 16-byte pieces XOR-swizzled by row, and leaves in 16-byte stores of whole
// rows, 2*D/16 lanes a row (rather than 8-byte pieces scattered over 32 rows):
// row i < nrows goes to out + i*stride. LDS operations of one wave complete in
// order, so the reads see the writes without a wait of their own; the caller
// guarantees that no other wave uses these LDS rows meanwhile and that no copy
// into them is in flight.
template <int D>
__device__ __forceinline__ void store_rows_bf16(const f32x16 (&o)[D / 32], float inv, uint8_t* ob, int lane, int nrows,
                                                uint16_t* out, size_t stride) {
  constexpr int ORB = 2 * D, OP = ORB / 16;  // bytes and 16-byte pieces per output row
  const int lq = lane & 31, hl = lane >> 5;
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      // accumulator rows 4*q4 .. 4*q4+3: elements db*32 + 8*q4 + 4*hl + 0..3
      const u32x2 v = {(uint32_t)f32_to_bf16_bits(o[db][4 * q4] * inv) |
                           ((uint32_t)f32_to_bf16_bits(o[db][4 * q4 + 1] * inv) << 16),
                       (uint32_t)f32_to_bf16_bits(o[db][4 * q4 + 2] * inv) |
                           ((uint32_t)f32_to_bf16_bits(o[db][4 * q4 + 3] * inv) << 16)};
      const int piece = 4 * db + q4;
      *reinterpret_cast<u32x2*>(ob + lq * ORB + ((piece ^ (lq & (OP - 1))) * 16) + 8 * hl) = v;
    }
#pragma unroll
  for (int i = 0; i < 32 * OP / 64; ++i) {
    const int pc = lane + 64 * i, row = pc / OP, col = pc % OP;
    const u32x4 v = *reinterpret_cast<const u32x4*>(ob + row * ORB + ((col ^ (row & (OP - 1))) * 16));
    if (row < nrows) *reinterpret_cast<u32x4*>(out + (size_t)row * stride + col * 8) = v;
  }
}

// ---------------------------------------------------------------------------
// bf16 path: 4 waves x 32 query rows of one head per workgroup, 64-key tiles
// double-buffered in LDS. Tiles are copied global -> LDS directly
// (global_load_lds_dwordx4, no VGPR staging) into XOR-swizzled rows so that
// the MFMA operand reads are bank-conflict free; V stays row-major and is read
// transposed with ds_read_b64_tr_b16. Every per-lane offset is computed once,
// outside the key loop. Under 256 VGPRs, so two waves share each SIMD and one
// wave's softmax overlaps the other's matrix work.

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// s_waitcnt immediate: wait until at most n vector-memory operations remain
// (expcnt and lgkmcnt left unconstrained).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier with only the LDS wait spelled out (the copies in flight
// are waited for explicitly by the caller; the fence of __syncthreads would
// wait for all of them). The memory clobber keeps LDS accesses on their side.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int D, bool CAUSAL, int OUT>
__global__ void __launch_bounds__(256, 2)
attn_bf16_kernel(AttnParams p) {
  constexpr int BN = 64, NW = 4, BM = 128;
  constexpr int RB = D * 2;                 // bytes per key row
  constexpr int NP = RB / 16;               // 16-byte pieces per row
  constexpr int TB = BN * RB;               // bytes per tile
  constexpr int LI = TB / 1024 / NW;        // direct-copy instructions per wave per tile
  constexpr int KS = D / 16, DB = D / 32;
  constexpr float RS_MAX = 256.f;  // 2^TAU, TAU = 8: bound on a lane's 32 probabilities
  static_assert(LI >= 1 && TB % (1024 * NW) == 0, "tile must split into whole wave copies");
  // V swizzle: piece ^ 4*(row & 3) keeps the 4 rows x 4 pieces of a transposed
  // read distinct (D = 64 has only 8 pieces per row: piece ^ 4*(row & 1)).
  constexpr int VSW = NP >= 16 ? 3 : 1;
  // One LDS object holds both K and V double buffers (K at buf*TB, V at
  // (2+buf)*TB). With a single object the compiler adds no vmcnt wait of its
  // own between a direct copy into one buffer and reads of the other; the
  // explicit wait + barrier below orders each buffer's copy before its reads.
  __shared__ __attribute__((aligned(1024))) uint8_t kvl[4 * TB];

  int b, h, mt;
  if (!decode_work(p, b, h, mt)) return;
  const int seq0 = p.cu[b];
  const int len = p.cu[b + 1] - seq0;
  const int m0 = mt * BM;
  if (m0 >= len) return;
  const int g = h / p.G;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lq = lane & 31, hl = lane >> 5;
  const int g16 = lane >> 4, s16 = lane & 15;
  const uint32_t kvrow = (uint32_t)p.Hkv * RB;
  const uint8_t* kbase = static_cast<const uint8_t*>(p.k) + ((size_t)seq0 * p.Hkv + g) * RB;
  const uint8_t* vbase = static_cast<const uint8_t*>(p.v) + ((size_t)seq0 * p.Hkv + g) * RB;
  const int qi = m0 + w * 32 + lq;
  const int wave_q0 = m0 + w * 32;

  // ---- per-lane constants
  // Copy j of a wave moves 16-byte pieces of tile row ld_row[j]; its source
  // is (tile base, wave-uniform) + ld_koff[j] / ld_voff[j] (per lane, fixed).
  int ld_row[LI];
  uint32_t ld_koff[LI], ld_voff[LI];
#pragma unroll
  for (int j = 0; j < LI; ++j) {
    const int slot = (w + NW * j) * 64 + lane;
    const int r = slot / NP, ph = slot % NP;
    ld_row[j] = r;
    ld_koff[j] = (uint32_t)r * kvrow + (uint32_t)(ph ^ (r & (NP - 1))) * 16;
    ld_voff[j] = (uint32_t)r * kvrow + (uint32_t)(ph ^ (4 * (r & VSW))) * 16;
  }
  const uint32_t lds_w = __builtin_amdgcn_readfirstlane((uint32_t)w * 1024u);  // this wave's copy slot
  // K operand of S^T block nb: row 32*nb + swap23(lq), logical piece 2*ks + hl
  const int rho = swap23(lq);
  uint32_t koff[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) koff[ks] = rho * RB + (((2 * ks + hl) ^ (rho & (NP - 1))) * 16);
  // (block nb adds 32 rows; row & (NP-1) is unchanged for NP <= 32, so the
  // swizzle of row 32*nb + rho equals that of rho)
  // V operand by transposed reads: lane reads row 16*kk + 8*(g16>>1) + 4*hf + (s16>>2),
  // head-dim block c0 = 8*db + 4*(g16&1) + (s16&3) of 4 elements.
  const int vrow0 = 8 * (g16 >> 1) + (s16 >> 2);
  uint32_t voff[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const int c0 = 8 * db + 4 * (g16 & 1) + (s16 & 3);
    voff[db] = vrow0 * RB + (((c0 >> 1) ^ (4 * (vrow0 & VSW))) * 16) + (c0 & 1) * 8;
  }

  auto copy_tile = [&](int tile, auto bufc) __attribute__((always_inline)) {
    constexpr int BUF = decltype(bufc)::value;
    const int k0 = tile * BN;
    const uint8_t* kt = kbase + (size_t)k0 * kvrow;
    const uint8_t* vt = vbase + (size_t)k0 * kvrow;
    const bool full = k0 + BN <= len;
#pragma unroll
    for (int j = 0; j < LI; ++j) {
      // rows past the sequence end repeat its last key
      const uint32_t fix = full ? 0u : (uint32_t)(min(k0 + ld_row[j], len - 1) - (k0 + ld_row[j])) * kvrow;
      __builtin_amdgcn_global_load_lds((const void*)(kt + (ld_koff[j] + fix)),
                                       (__attribute__((address_space(3))) void*)(kvl + BUF * TB + lds_w + NW * j * 1024),
                                       16, 0, 0);
      __builtin_amdgcn_global_load_lds((const void*)(vt + (ld_voff[j] + fix)),
                                       (__attribute__((address_space(3))) void*)(kvl + (2 + BUF) * TB + lds_w + NW * j * 1024),
                                       16, 0, 0);
    }
  };

  // ---- queries: the wave's 32 rows are copied whole (NP lanes a row, so each
  // copy reads 1 KB of contiguous rows) into its quarter of the second K/V
  // buffers, free until step 0 refills them, with 16-byte pieces XOR-swizzled
  // by row; each lane then reads its operand registers (row lq, pieces
  // 2*ks + hl) from there. Read straight from memory, every load of the
  // operand layout would touch 32 rows at 32 bytes each.
  uint8_t* qst = kvl + (w < 2 ? TB : 3 * TB) + (w & 1) * (32 * RB);  // 32 rows of this wave
  {
    constexpr int QRI = 1024 / RB;  // rows per 1 KB copy
    const int r_in = lane / NP, ph = lane % NP;
    const uint32_t lds_q = __builtin_amdgcn_readfirstlane((uint32_t)(qst - kvl));
#pragma unroll
    for (int j = 0; j < 32 / QRI; ++j) {
      const int r = QRI * j + r_in;
      const uint8_t* src = static_cast<const uint8_t*>(p.q) +
                           ((size_t)(seq0 + min(wave_q0 + r, len - 1)) * p.Hq + h) * RB + ((ph ^ (r & (NP - 1))) * 16);
      __builtin_amdgcn_global_load_lds((const void*)src,
                                       (__attribute__((address_space(3))) void*)(kvl + lds_q + j * 1024), 16, 0, 0);
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float c = p.scale_log2;
  const int kend = CAUSAL ? min(len, m0 + BM) : len;
  const int nt = (kend + BN - 1) / BN;

  copy_tile(0, std::integral_constant<int, 0>{});
  wait_vmcnt<0>();  // this wave's copies have landed: its own query rows may be read
  bf16x8 qreg[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    qreg[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(qst + lq * RB + (((2 * ks + hl) ^ (lq & (NP - 1))) * 16)));
  __builtin_amdgcn_sched_barrier(0);
  __syncthreads();  // tile 0 has landed for every wave, and every wave has its queries (step 0 refills the second buffers)

  // step t (K, V of tile t in buffers BUF = t & 1); instantiated per buffer so
  // that every LDS offset is an immediate
  auto step = [&](int t, auto bufc) __attribute__((always_inline)) {
    constexpr int BUF = decltype(bufc)::value;
    const int k0 = t * BN;
    if (t + 1 < nt) copy_tile(t + 1, std::integral_constant<int, BUF ^ 1>{});  // buffer last read in step t-1
    if (!(CAUSAL && k0 > wave_q0 + 31)) {
      // ---- S^T blocks: 2 x (32 keys x 32 queries). K operands are read from
      // LDS two k-steps ahead of their MFMAs (a ring of three).
      const uint8_t* kl = kvl + BUF * TB;
      const uint8_t* vl = kvl + (2 + BUF) * TB;
      f32x16 s[2];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[nb][r] = 0.f;
      auto kread = [&](int ks, int nb) __attribute__((always_inline)) {
        return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(kl + nb * 32 * RB + koff[ks]));
      };
      bf16x8 ka[3][2];
#pragma unroll
      for (int ks = 0; ks < 2 && ks < KS; ++ks)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) ka[ks][nb] = kread(ks, nb);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if (ks + 2 < KS) {
#pragma unroll
          for (int nb = 0; nb < 2; ++nb) ka[(ks + 2) % 3][nb] = kread(ks + 2, nb);
        }
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) s[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[ks % 3][nb], qreg[ks], s[nb], 0, 0, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if (ks + 2 < KS) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      }
      // V operands of the first P.V k-step, read while the softmax runs
      auto vread = [&](int kk, int db, int hf) __attribute__((always_inline)) {
        return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vl + voff[db] + (16 * kk + 4 * hf) * RB));
      };
      s16x4 vr[2][DB][2];
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) vr[0][db][hf] = vread(0, db, hf);
      // ---- mask (edge tiles only), tile max in raw logit units
      const bool need_mask = (k0 + BN > len) || (CAUSAL && k0 + BN - 1 > wave_q0);
      if (need_mask) {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = k0 + 32 * nb + swap23(acc_row32(r, hl));
            if (key >= len || (CAUSAL && key > qi)) s[nb][r] = -INFINITY;
          }
      }
      // ---- P = exp2(s*c - m*c) under the running max m, as the B operand of
      // O^T += V^T P^T. A lane sum above 2^TAU (so some p may exceed 2^TAU) or
      // the first visible keys of a row send the wave through the exact path:
      // m becomes the row max, the output so far is rescaled and P is formed
      // again. Rows whose max grows by less than TAU keep m (lazy rescale).
      float rsk[4];
      bf16x8 pb[4];
      auto form_p = [&](float mc) __attribute__((always_inline)) {
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          float e[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) e[i] = __builtin_amdgcn_exp2f(fmaf(s[kk >> 1][8 * (kk & 1) + i], c, -mc));
          pb[kk] = bf16x8{(__bf16)e[0], (__bf16)e[1], (__bf16)e[2], (__bf16)e[3],
                          (__bf16)e[4], (__bf16)e[5], (__bf16)e[6], (__bf16)e[7]};
          rsk[kk] = ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
        }
        return (rsk[0] + rsk[1]) + (rsk[2] + rsk[3]);
      };
      float rs = form_p(m_run == -INFINITY ? 0.f : m_run * c);
      const bool exact = rs > RS_MAX || (m_run == -INFINITY && rs > 0.f);
      if (__any(exact)) {
        float mx = max32(s);
        {
          const float2 pr = pair_xor32(mx);
          mx = __builtin_elementwise_maximum(pr.x, pr.y);
        }
        const float m_new = fmaxf(m_run, mx);
        const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f((m_run - m_new) * c);
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
        m_run = m_new;
        rs = form_p(m_run == -INFINITY ? 0.f : m_run * c);
      }
      l_run += rs;
      // ---- O^T += V^T P^T; V operands one k-step ahead of their MFMAs
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        if (kk + 1 < 4) {
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) vr[(kk + 1) & 1][db][hf] = vread(kk + 1, db, hf);
        }
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const bf16x8 va = __builtin_bit_cast(bf16x8, __builtin_shufflevector(vr[kk & 1][db][0], vr[kk & 1][db][1], 0, 1, 2, 3, 4, 5, 6, 7));
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[kk], o[db], 0, 0, 0);
        }
      }
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        if (kk + 1 < 4) __builtin_amdgcn_sched_group_barrier(0x100, 2 * DB, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, DB, 0);
      }
    }
    wait_vmcnt<0>();
    __syncthreads();
  };
  for (int t = 0; t < nt; t += 2) {
    step(t, std::integral_constant<int, 0>{});
    if (t + 1 < nt) step(t + 1, std::integral_constant<int, 1>{});
  }

  const float l = sum_xor32(l_run);
  const float inv = (l > 0.f) ? p.out_scale / l : 0.f;
  if constexpr (OUT == LITEVLM_BF16) {
    static_assert(sizeof(kvl) >= 4 * 32 * 2 * D, "the output rows of the 4 waves fit the tile buffers");
    int lane_e = lane;  // opaque: the epilogue's offsets are not shared with (kept live from) the prologue's
    asm volatile("" : "+v"(lane_e));
    store_rows_bf16<D>(o, inv, kvl + w * 32 * (2 * D), lane_e, len - wave_q0,
                       static_cast<uint16_t*>(p.o) + ((size_t)(seq0 + wave_q0) * p.Hq + h) * D, (size_t)p.Hq * D);
  } else if (qi < len) {
    const size_t obase = ((size_t)(seq0 + qi) * p.Hq + h) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) store_out<OUT>(p.o, obase + db * 32 + acc_row32(r, hl), o[db][r] * inv);
  }
}

// ---------------------------------------------------------------------------
// bf16 path for grids that fit one pass of the chip (at most two workgroups
// per CU): a software-pipelined tile loop, for when one workgroup's chain of
// key tiles is the critical path rather than the chip's throughput.
//
// A workgroup is 4 waves and covers 128 (query position, head) rows of one KV
// head: Hw query heads (the largest of 4, 2, 1 dividing G) times 32*(4/Hw)
// consecutive positions. Wave w takes head w % Hw and the 32 positions of
// block w / Hw; at the GQA shapes (G = 4) the four waves are the four query
// heads of one 32-position block, so they share one causal extent and every
// K/V tile is staged once for all of them.
//
// K and V tiles of 64 keys are copied global -> LDS directly into rings of two
// slots each, one tile ahead of use. A wave keeps its 32 query rows in
// registers and computes, per key tile t:
//   (a) the mask (edge tiles only) and the row max of S_t = K_t Q^T, formed in
//       the previous step; the output is rescaled only when a row's max grows
//       by more than 2^8 (so every p <= 2^8);
//   (b) the exponentials P_t = exp2(S_t*c - m*c), packed to bf16 as they are
//       formed and issued between the MFMAs of S_{t+1} = K_{t+1} Q^T, so the
//       matrix pipe runs the next tile's logits under this tile's vector work
//       (the last tile also forms the logits of a stale slot, discarded, so the
//       loop needs no separate tail);
//   (c) O^T += V_t^T P_t^T, the transposed V reads two 16-key steps ahead.
// One barrier per tile hands the ring slots over. About 240 VGPRs: two waves
// per SIMD.

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Transposed LDS read (ds_read_b64_tr_b16) as inline assembly: the builtin
// makes the compiler wait for every direct copy in flight before it, which
// would drain the copies issued ahead. The caller waits (lgkmcnt) before use.
template <int OFF>
__device__ __forceinline__ s16x4 ds_read_tr16(uint32_t addr) {
  s16x4 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}

// The V operands of one key tile: va[kk][db] = V^T rows 32*db.., keys 16*kk..
// (two transposed reads of 4 keys each per lane, rows 4 apart).
template <int RB, int DB, int KK>
__device__ __forceinline__ void vread_kk(bf16x8 (&va)[DB], const uint32_t (&vaddr)[DB]) {
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const s16x4 lo = ds_read_tr16<(16 * KK) * RB>(vaddr[db]);
    const s16x4 hi = ds_read_tr16<(16 * KK + 4) * RB>(vaddr[db]);
    va[db] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  }
}

// Wait until at most N LDS accesses of the wave remain; the operands pass
// through the wait, so that nothing reading them is placed before it.
template <int N, int DB>
__device__ __forceinline__ void lds_wait_n(bf16x8 (&a)[DB]) {
  if constexpr (DB == 4)
    asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]) : "i"(N));
  else
    asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(a[0]), "+v"(a[1]) : "i"(N));
}

// Work item (KV head g, head group hgrp of Hw heads, query block mt from the
// last, sample b), dealt to the 8 XCDs in contiguous ranges: an XCD owns whole
// KV heads across the batch, so workgroups sharing K/V sit behind the same L2,
// and within an XCD the longest causal blocks start first.
__device__ __forceinline__ bool decode_work_hg(const AttnParams& p, int& b, int& g, int& hgrp, int& mt) {
  const int L = blockIdx.x;
  const int w = (L & 7) * p.per_xcd + (L >> 3);
  if (w >= p.n_work) return false;
  const int ng = p.G / p.Hw;
  b = w % p.B;
  int rest = w / p.B;
  const int mrev = rest % p.n_mtiles;
  rest /= p.n_mtiles;
  hgrp = rest % ng;
  g = rest / ng;
  mt = p.n_mtiles - 1 - mrev;
  return true;
}


template <int D, bool CAUSAL, int OUT>
__global__ void __launch_bounds__(256, 2)
attn_bf16_pipe_kernel(AttnParams p) {
  constexpr int BN = 64, NW = 4, NS = 2;    // keys per tile, waves, ring slots
  constexpr int RB = D * 2;                 // bytes per key row
  constexpr int NP = RB / 16;               // 16-byte pieces per row
  constexpr int TB = BN * RB;               // bytes per tile
  constexpr int LI = TB / 1024 / NW;        // direct-copy instructions per wave per tile (K or V)
  constexpr int KS = D / 16, DB = D / 32;
  constexpr int EPK = 32 / KS;              // exponentials per QK k-step
  constexpr float TAU = 8.f;                // log2 bound on p under a lagging max
  static_assert(LI >= 1 && TB % (1024 * NW) == 0, "tile must split into whole wave copies");
  static_assert(LI <= 4, "the wait below counts at most 8 copies in flight");
  // V swizzle: piece ^ 4*(row & 3) keeps the 4 rows x 4 pieces of a transposed
  // read distinct (D = 64 has only 8 pieces per row: piece ^ 4*(row & 1)).
  constexpr int VSW = NP >= 16 ? 3 : 1;
  // One LDS object: K slots at s*TB, V slots at (NS+s)*TB. With a single
  // object the compiler adds no wait of its own between a direct copy into one
  // slot and reads of another.
  __shared__ __attribute__((aligned(1024))) uint8_t kvl[2 * NS * TB];

  int b, g, hgrp, mt;
  if (!decode_work_hg(p, b, g, hgrp, mt)) return;
  const int seq0 = p.cu[b];
  const int len = p.cu[b + 1] - seq0;
  const int bmw = 32 * p.P;                 // positions per workgroup
  const int m0 = mt * bmw;
  if (m0 >= len) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: scalar branches
  const int lq = lane & 31, hl = lane >> 5;
  const int g16 = lane >> 4, s16 = lane & 15;
  const int h = g * p.G + hgrp * p.Hw + w % p.Hw;
  const int wave_q0 = m0 + 32 * (w / p.Hw);
  const int qi = wave_q0 + lq;
  const uint32_t kvrow = (uint32_t)p.Hkv * RB;
  const uint8_t* kbase = static_cast<const uint8_t*>(p.k) + ((size_t)seq0 * p.Hkv + g) * RB;
  const uint8_t* vbase = static_cast<const uint8_t*>(p.v) + ((size_t)seq0 * p.Hkv + g) * RB;

  // ---- per-lane constants
  // Copy j of a wave moves 16-byte pieces of tile row ld_row[j]; its source
  // is (tile base, wave-uniform) + ld_koff[j] / ld_voff[j] (per lane, fixed).
  int ld_row[LI];
  uint32_t ld_koff[LI], ld_voff[LI];
#pragma unroll
  for (int j = 0; j < LI; ++j) {
    const int slot = (w + NW * j) * 64 + lane;
    const int r = slot / NP, ph = slot % NP;
    ld_row[j] = r;
    ld_koff[j] = (uint32_t)r * kvrow + (uint32_t)(ph ^ (r & (NP - 1))) * 16;
    ld_voff[j] = (uint32_t)r * kvrow + (uint32_t)(ph ^ (4 * (r & VSW))) * 16;
  }
  const uint32_t lds_w = __builtin_amdgcn_readfirstlane((uint32_t)w * 1024u);  // this wave's copy slot
  // K operand of S^T block nb: row 32*nb + swap23(lq), logical piece 2*ks + hl
  // (block nb adds 32 rows; row & (NP-1) is unchanged for NP <= 32, so the
  // swizzle of row 32*nb + rho equals that of rho)
  const int rho = swap23(lq);
  uint32_t koff[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) koff[ks] = rho * RB + (((2 * ks + hl) ^ (rho & (NP - 1))) * 16);
  // V operand by transposed reads: lane reads row 16*kk + 8*(g16>>1) + 4*hf + (s16>>2),
  // head-dim block c0 = 8*db + 4*(g16&1) + (s16&3) of 4 elements.
  // (LDS byte addresses: the reads are inline assembly)
  const int vrow0 = 8 * (g16 >> 1) + (s16 >> 2);
  uint32_t voff[DB];
  const uint32_t kvl_base =
      (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint8_t*)kvl);
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const int c0 = 8 * db + 4 * (g16 & 1) + (s16 & 3);
    voff[db] = kvl_base + vrow0 * RB + (((c0 >> 1) ^ (4 * (vrow0 & VSW))) * 16) + (c0 & 1) * 8;
  }

  const int kend = CAUSAL ? min(len, m0 + bmw) : len;
  const int nt = (kend + BN - 1) / BN;

  auto copy_rows = [&](const uint8_t* src, int tile, uint8_t* dst, const uint32_t* off) __attribute__((always_inline)) {
    const int k0 = tile * BN;
    const uint8_t* st = src + (size_t)k0 * kvrow;
    // rows past the sequence end repeat its last key (no branch: the row
    // shift is zero inside the sequence)
    const int last = len - 1 - k0;
#pragma unroll
    for (int j = 0; j < LI; ++j) {
      const uint32_t fix = (uint32_t)(min(ld_row[j], last) - ld_row[j]) * kvrow;
      __builtin_amdgcn_global_load_lds((const void*)(st + (off[j] + fix)),
                                       (__attribute__((address_space(3))) void*)(dst + lds_w + NW * j * 1024),
                                       16, 0, 0);
    }
  };
  auto copy_k = [&](int tile, auto slotc) __attribute__((always_inline)) {
    copy_rows(kbase, tile, kvl + decltype(slotc)::value * TB, ld_koff);
  };
  auto copy_v = [&](int tile, auto slotc) __attribute__((always_inline)) {
    copy_rows(vbase, tile, kvl + (NS + decltype(slotc)::value) * TB, ld_voff);
  };
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;

  bf16x8 qreg[KS];
  {
    const uint8_t* qr = static_cast<const uint8_t*>(p.q) + ((size_t)(seq0 + min(qi, len - 1)) * p.Hq + h) * RB;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qreg[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(qr + (ks * 16 + 8 * hl) * 2));
  }
  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float c = p.scale_log2;
  const float tau_raw = TAU / c;  // TAU in raw logit units (c > 0)

  // S^T blocks of a tile in a K slot: 2 x (32 keys x 32 queries),
  // s[nb][r] = q(lane%32) . k(32*nb + swap23(acc_row32(r, hl))).
  auto kread = [&](const uint8_t* kl, int ks, int nb) __attribute__((always_inline)) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(kl + nb * 32 * RB + koff[ks]));
  };

  // ---- prologue: Q, then K0, K1 and V0 landed
  copy_k(0, S0{});
  if (nt > 1) copy_k(1, S1{});
  copy_v(0, S0{});
  wait_vmcnt<0>();
  lds_barrier();
  f32x16 s[2];
  {
    const uint8_t* kl = kvl;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[nb][r] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        s[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kread(kl, ks, nb), qreg[ks], s[nb], 0, 0, 0);
  }
  lds_barrier();  // every wave has read K0: its slot may be refilled

  // step t: S_t in s; K_{t+1} in K slot (U+1)%2, V_t in V slot U (U = t % 2);
  // MORE: a tile t+1 exists (every step but the last)
  auto step = [&](int t, auto uc, auto morec) __attribute__((always_inline)) {
    constexpr int U = decltype(uc)::value;
    constexpr bool MORE = decltype(morec)::value;
    constexpr int UK1 = (U + 1) % NS;
    const int k0 = t * BN;
    // copies one step ahead of use: K_{t+2} into K_t's slot (read in step
    // t-1), V_{t+1} into V_{t-1}'s slot
    if (t + 2 < nt) copy_k(t + 2, std::integral_constant<int, U>{});
    if (t + 1 < nt) copy_v(t + 1, std::integral_constant<int, UK1>{});
    // ---- (a) mask (edge tiles only), row max, lazy rescale
    const bool need_mask = (k0 + BN > len) || (CAUSAL && k0 + BN - 1 > wave_q0);
    if (need_mask) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k0 + 32 * nb + swap23(acc_row32(r, hl));
          if (key >= len || (CAUSAL && key > qi)) s[nb][r] = -INFINITY;
        }
    }
    {
      float mx = max32(s);
      const float2 pr = pair_xor32(mx);
      mx = __builtin_elementwise_maximum(pr.x, pr.y);
      const bool grow = mx > m_run + tau_raw;
      if (__any(grow)) {
        const float m_new = grow ? mx : m_run;
        const float alpha = (!grow) ? 1.f : (m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((m_run - m_new) * c));
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
        m_run = m_new;
      }
    }
    const float mc = m_run == -INFINITY ? 0.f : m_run * c;
    // ---- (b) P_t = exp2(S_t*c - m*c), packed to bf16 as it is formed, with
    // its row sum, under the MFMAs of S_{t+1}
    uint32_t pk[16];  // bf16 pairs: pk[i] holds values 2i, 2i+1 of the lane's 32
    float rsum[4] = {0.f, 0.f, 0.f, 0.f};
    auto expo2 = [&](int i) __attribute__((always_inline)) {  // values 2i, 2i+1
      const float e0 = __builtin_amdgcn_exp2f(fmaf(s[(2 * i) >> 4][(2 * i) & 15], c, -mc));
      const float e1 = __builtin_amdgcn_exp2f(fmaf(s[(2 * i + 1) >> 4][(2 * i + 1) & 15], c, -mc));
      pk[i] = __builtin_bit_cast(uint32_t, bf16x2{(__bf16)e0, (__bf16)e1});
      rsum[i & 3] += e0 + e1;
    };
    f32x16 sn[2];
    if constexpr (MORE) {
      const uint8_t* kl = kvl + UK1 * TB;
      bf16x8 ka[2][2];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) ka[0][nb] = kread(kl, 0, nb);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if (ks + 1 < KS) {
#pragma unroll
          for (int nb = 0; nb < 2; ++nb) ka[(ks + 1) & 1][nb] = kread(kl, ks + 1, nb);
        }
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          sn[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[ks & 1][nb], qreg[ks],
                                                           ks == 0 ? f32x16{} : sn[nb], 0, 0, 0);
#pragma unroll
          for (int j = 0; j < EPK / 4; ++j) expo2((ks * EPK + nb * (EPK / 2)) / 2 + j);
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) expo2(i);
    }
    l_run += (rsum[0] + rsum[1]) + (rsum[2] + rsum[3]);
    // ---- (c) O^T += V_t^T P_t^T. The transposed V reads of keys 0-31 are
    // issued here, those of keys 32-63 once the first are in registers; each
    // half is waited for before its MFMAs (the registers pass through the
    // wait, so that no MFMA is placed before it).
    uint32_t vaddr[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) vaddr[db] = voff[db] + (NS + U) * TB;
    bf16x8 va0[DB], va1[DB];
    auto pv = [&](int kk, bf16x8 (&va)[DB]) __attribute__((always_inline)) {
      const bf16x8 pb = __builtin_bit_cast(bf16x8, u32x4{pk[4 * kk], pk[4 * kk + 1], pk[4 * kk + 2], pk[4 * kk + 3]});
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[db], pb, o[db], 0, 0, 0);
    };
    vread_kk<RB, DB, 0>(va0, vaddr);
    vread_kk<RB, DB, 1>(va1, vaddr);
    lds_wait_n<2 * DB>(va0);
    pv(0, va0);
    vread_kk<RB, DB, 2>(va0, vaddr);
    lds_wait_n<2 * DB>(va1);
    pv(1, va1);
    vread_kk<RB, DB, 3>(va1, vaddr);
    lds_wait_n<2 * DB>(va0);
    pv(2, va0);
    lds_wait_n<0>(va1);
    pv(3, va1);
    // K_{t+2} and V_{t+1} have landed
    wait_vmcnt<0>();
    lds_barrier();
    if constexpr (MORE) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) s[nb] = sn[nb];
    }
  };
  using Y = std::true_type;
  // steps in pairs (ring slots 0, 1). The final step also forms the logits
  // of a next tile from a stale slot; they are discarded.
  for (int t = 0;; t += 2) {
    step(t, S0{}, Y{});
    if (t + 1 == nt) break;
    step(t + 1, S1{}, Y{});
    if (t + 2 == nt) break;
  }

  const float l = sum_xor32(l_run);
  const float inv = (l > 0.f) ? p.out_scale / l : 0.f;
  if constexpr (OUT == LITEVLM_BF16) {
    static_assert(sizeof(kvl) >= 4 * 32 * 2 * D, "the output rows of the 4 waves fit the tile buffers");
    store_rows_bf16<D>(o, inv, kvl + w * 32 * (2 * D), lane, len - wave_q0,
                       static_cast<uint16_t*>(p.o) + ((size_t)(seq0 + wave_q0) * p.Hq + h) * D, (size_t)p.Hq * D);
  } else if (qi < len) {
    const size_t obase = ((size_t)(seq0 + qi) * p.Hq + h) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) store_out<OUT>(p.o, obase + db * 32 + acc_row32(r, hl), o[db][r] * inv);
  }
}


// ---------------------------------------------------------------------------
// E4M3 path: the bf16 kernel's structure on v_mfma_f32_32x32x64_f8f6f4. S^T
// block nb holds keys 32*bit2(rho) + 16*nb + 4*(rho>>3) + (rho&3) in row rho, so
// that a lane half's 32 accumulator values are keys 32*hl .. 32*hl+31, the B
// operand of one P.V k-step. K rows are 16-byte pieces read directly; V is
// row-major and read transposed with ds_read_b64_tr_b8 (8 keys per read).
// P is quantised as p*2^8 under a running max that may lag the row max by at
// most half a binade: every p is then <= 2^0.5, so p*2^8 <= 362 stays inside
// the E4M3 range (448), and the 2^8 shift keeps p >= 2^-14 out of the E4M3
// subnormal range. The output is rescaled only when a row's max grows by more
// than that half binade, which after the first tiles of a row is rare.

typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) i32x2 lds_i32x2;

template <int D, bool CAUSAL, int OUT>
__global__ void __launch_bounds__(256, 3)
attn_fp8_kernel(AttnParams p) {
  constexpr int BN = 64, NW = 4, BM = 128;
  constexpr int RB = D;                     // bytes per key row
  constexpr int NP = RB / 16;               // 16-byte pieces per row
  constexpr int TB = BN * RB;
  constexpr int LI = (TB / 1024 + NW - 1) / NW;
  constexpr int NI = TB / 1024;             // wave copies per tile
  constexpr int QKS = D / 64, DB = D / 32;
  constexpr int PSHIFT = 8;
  constexpr float TAU = 0.5f;               // log2 lag allowed between the running and the row max
  static_assert(TB % 1024 == 0, "tile must split into whole wave copies");
  // One LDS object holds both K and V double buffers (K at buf*TB, V at
  // (2+buf)*TB). With a single object the compiler adds no vmcnt wait of its
  // own between a direct copy into one buffer and reads of the other; the
  // explicit wait + barrier below orders each buffer's copy before its reads.
  __shared__ __attribute__((aligned(1024))) uint8_t kvl[4 * TB];

  int b, h, mt;
  if (!decode_work(p, b, h, mt)) return;
  const int seq0 = p.cu[b];
  const int len = p.cu[b + 1] - seq0;
  const int m0 = mt * BM;
  if (m0 >= len) return;
  const int g = h / p.G;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: scalar branches
  const int lq = lane & 31, hl = lane >> 5;
  const int g16 = lane >> 4, s16 = lane & 15;
  const uint32_t kvrow = (uint32_t)p.Hkv * RB;
  const uint8_t* kbase = static_cast<const uint8_t*>(p.k) + ((size_t)seq0 * p.Hkv + g) * RB;
  const uint8_t* vbase = static_cast<const uint8_t*>(p.v) + ((size_t)seq0 * p.Hkv + g) * RB;
  const int qi = m0 + w * 32 + lq;
  const int wave_q0 = m0 + w * 32;

  // piece swizzles (involutions): K reads hit 16 rows x 1 piece per 16 lanes;
  // V transposed reads (8 bytes a lane, 32 lanes a cycle) hit 8 rows x the 2
  // pieces 2*db, 2*db+1 per 32 lanes. With 128-byte rows, rows r and r^1 fill
  // the two halves of the 256-byte bank window, and piece p of row r sits at
  // p ^ (r & 6): pieces (2*db + e) ^ 2i = 2*(db ^ i) + e are distinct over the
  // 4 row pairs i and both halves e, so the 32 lanes hit 32 distinct 8-byte
  // slots.
  auto kswz = [](int r) {
    return NP >= 8 ? (((r >> 1) & 3) | (((r >> 5) & 1) << 2)) : (((r >> 2) & 1) | (((r >> 5) & 1) << 1));
  };
  auto vswz = [](int r) { return NP >= 8 ? (r & 6) : ((r >> 1) & (NP - 1) & 3); };

  // Copy j of a wave moves 16-byte pieces of tile row ld_row[j]; its source
  // is (tile base, wave-uniform) + ld_koff[j] / ld_voff[j] (per lane, fixed).
  int ld_row[LI];
  uint32_t ld_koff[LI], ld_voff[LI];
#pragma unroll
  for (int j = 0; j < LI; ++j) {
    const int slot = min(w + NW * j, NI - 1) * 64 + lane;
    const int r = slot / NP, ph = slot % NP;
    ld_row[j] = r;
    ld_koff[j] = (uint32_t)r * kvrow + (uint32_t)(ph ^ kswz(r)) * 16;
    ld_voff[j] = (uint32_t)r * kvrow + (uint32_t)(ph ^ vswz(r)) * 16;
  }
  const uint32_t lds_w = __builtin_amdgcn_readfirstlane((uint32_t)w * 1024u);  // this wave's copy slot
  // K operand: rows tile_key<fp8>(nb, lq), pieces 4*ks + 2*hl and +1
  uint32_t koff[2][QKS][2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int row = tile_key<true>(nb, lq);
#pragma unroll
    for (int ks = 0; ks < QKS; ++ks)
#pragma unroll
      for (int u = 0; u < 2; ++u) koff[nb][ks][u] = row * RB + (((4 * ks + 2 * hl + u) ^ kswz(row)) * 16);
  }
  // V operand: read j covers keys 32*(g16>>1) + 8*j + 0..7 at head dim 32*db + lq;
  // source lane s16 addresses row 32*(g16>>1) + 8*j + (s16>>1), piece 2*db + (g16&1), half s16&1
  uint32_t voff[DB];
  const int vrow0 = 32 * (g16 >> 1) + (s16 >> 1);
#pragma unroll
  for (int db = 0; db < DB; ++db)
    voff[db] = vrow0 * RB + (((2 * db + (g16 & 1)) ^ vswz(vrow0)) * 16) + (s16 & 1) * 8;
  // rows vrow0 + 8*j share vswz: it depends on bits 1, 2 of the row only

  auto copy_tile = [&](int tile, auto bufc) __attribute__((always_inline)) {
    constexpr int BUF = decltype(bufc)::value;
    const int k0 = tile * BN;
    const uint8_t* kt = kbase + (size_t)k0 * kvrow;
    const uint8_t* vt = vbase + (size_t)k0 * kvrow;
    const bool full = k0 + BN <= len;
#pragma unroll
    for (int j = 0; j < LI; ++j) {
      if (w + NW * j >= NI) break;
      // rows past the sequence end repeat its last key
      const uint32_t fix = full ? 0u : (uint32_t)(min(k0 + ld_row[j], len - 1) - (k0 + ld_row[j])) * kvrow;
      __builtin_amdgcn_global_load_lds((const void*)(kt + (ld_koff[j] + fix)),
                                       (__attribute__((address_space(3))) void*)(kvl + BUF * TB + lds_w + NW * j * 1024),
                                       16, 0, 0);
      __builtin_amdgcn_global_load_lds((const void*)(vt + (ld_voff[j] + fix)),
                                       (__attribute__((address_space(3))) void*)(kvl + (2 + BUF) * TB + lds_w + NW * j * 1024),
                                       16, 0, 0);
    }
  };

  i32x8 qreg[QKS];
  {
    const uint8_t* qr = static_cast<const uint8_t*>(p.q) + ((size_t)(seq0 + min(qi, len - 1)) * p.Hq + h) * RB;
#pragma unroll
    for (int ks = 0; ks < QKS; ++ks) {
      const u32x4 lo = *reinterpret_cast<const u32x4*>(qr + ks * 64 + 32 * hl);
      const u32x4 hi = *reinterpret_cast<const u32x4*>(qr + ks * 64 + 32 * hl + 16);
      qreg[ks] = i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
    }
  }
  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float m_run = -INFINITY;
  // row sums by the matrix core: ones^T P^T puts the row sum of the quantised
  // p in every accumulator row
  f32x16 lsum;
#pragma unroll
  for (int r = 0; r < 16; ++r) lsum[r] = 0.f;
  const i32x8 ones = {0x38383838, 0x38383838, 0x38383838, 0x38383838,
                      0x38383838, 0x38383838, 0x38383838, 0x38383838};  // E4M3 1.0
  const float c = p.scale_log2;
  const float tau_raw = TAU / c;  // TAU in raw logit units (c > 0)
  const int kend = CAUSAL ? min(len, m0 + BM) : len;
  const int nt = (kend + BN - 1) / BN;

  copy_tile(0, std::integral_constant<int, 0>{});
  wait_vmcnt<0>();
  __syncthreads();

  // step t (K, V of tile t in buffers BUF = t & 1); instantiated per buffer so
  // that every LDS offset is an immediate
  auto step = [&](int t, auto bufc) __attribute__((always_inline)) {
    constexpr int BUF = decltype(bufc)::value;
    const int k0 = t * BN;
    if (t + 1 < nt) copy_tile(t + 1, std::integral_constant<int, BUF ^ 1>{});
    if (!(CAUSAL && k0 > wave_q0 + 31)) {
      const uint8_t* kl = kvl + BUF * TB;
      f32x16 s[2];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[nb][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < QKS; ++ks) {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          const u32x4 lo = *reinterpret_cast<const u32x4*>(kl + koff[nb][ks][0]);
          const u32x4 hi = *reinterpret_cast<const u32x4*>(kl + koff[nb][ks][1]);
          const i32x8 a = {(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
          s[nb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, qreg[ks], s[nb], 0, 0, 0, 0, 0, 0);
        }
      }
      const bool need_mask = (k0 + BN > len) || (CAUSAL && k0 + BN - 1 > wave_q0);
      if (need_mask) {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = k0 + tile_key<true>(nb, acc_row32(r, hl));
            if (key >= len || (CAUSAL && key > qi)) s[nb][r] = -INFINITY;
          }
      }
      float mx = max32(s);
      {
        const float2 pr = pair_xor32(mx);
        mx = __builtin_elementwise_maximum(pr.x, pr.y);
      }
      // lazy running max: rescale only when a row's max grows past m + TAU
      const bool grow = mx > m_run + tau_raw;
      if (__any(grow)) {
        const float m_new = grow ? mx : m_run;
        const float alpha = grow ? __builtin_amdgcn_exp2f((m_run - m_new) * c) : 1.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) lsum[r] *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
        m_run = m_new;
      }
      // p * 2^PSHIFT = exp2(s*c - m*c + PSHIFT)
      const float mc = (m_run == -INFINITY) ? 0.f : m_run * c - (float)PSHIFT;
      int pw[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int nb = i >> 2, r0 = (i & 3) * 4;
        float e[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) e[u] = __builtin_amdgcn_exp2f(fmaf(s[nb][r0 + u], c, -mc));
        int wd = __builtin_amdgcn_cvt_pk_fp8_f32(e[0], e[1], 0, false);
        pw[i] = __builtin_amdgcn_cvt_pk_fp8_f32(e[2], e[3], wd, true);
      }
      const i32x8 pb = {pw[0], pw[1], pw[2], pw[3], pw[4], pw[5], pw[6], pw[7]};
      lsum = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(ones, pb, lsum, 0, 0, 0, 0, 0, 0);
      const uint8_t* vl = kvl + (2 + BUF) * TB;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        i32x2 part[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          part[j] = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2*)(vl + voff[db] + (8 * j) * RB));
        const i32x8 va = {part[0][0], part[0][1], part[1][0], part[1][1],
                          part[2][0], part[2][1], part[3][0], part[3][1]};
        o[db] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(va, pb, o[db], 0, 0, 0, 0, 0, 0);
      }
    }
    wait_vmcnt<0>();
    __syncthreads();
  };
  for (int t = 0; t < nt; t += 2) {
    step(t, std::integral_constant<int, 0>{});
    if (t + 1 < nt) step(t + 1, std::integral_constant<int, 1>{});
  }

  const float l = lsum[0];
  const float inv = (l > 0.f) ? p.out_scale / l : 0.f;   // l already carries 2^PSHIFT
  if constexpr (OUT == LITEVLM_BF16 && CAUSAL) {  // (the non-causal instance would spill)
    static_assert(sizeof(kvl) >= 4 * 32 * 2 * D, "the output rows of the 4 waves fit the tile buffers");
    int lane_e = lane;  // opaque: the epilogue's offsets are not shared with (kept live from) the prologue's
    asm volatile("" : "+v"(lane_e));
    store_rows_bf16<D>(o, inv, kvl + w * 32 * (2 * D), lane_e, len - wave_q0,
                       static_cast<uint16_t*>(p.o) + ((size_t)(seq0 + wave_q0) * p.Hq + h) * D, (size_t)p.Hq * D);
  } else if (qi < len) {
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
  int b, h, mt;
  if (!decode_work(p, b, h, mt)) return;
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
  // bf16 grids of at most two 128-row workgroups per CU (256 CUs) take the
  // pipelined loop: there the longest workgroup's chain of tiles sets the time
  if (a.in_dtype == LITEVLM_BF16 &&
      (long long)((a.max_seqlen + 127) / 128) * a.Hq * a.B <= 2LL * 256) {
    p.Hw = p.G % 4 == 0 ? 4 : (p.G % 2 == 0 ? 2 : 1);
    p.P = 4 / p.Hw;
    const int bmp = 32 * p.P;
    p.n_mtiles = (a.max_seqlen + bmp - 1) / bmp;
    p.n_work = p.n_mtiles * (a.Hq / p.Hw) * a.B;
    p.per_xcd = (p.n_work + 7) / 8;
    hipLaunchKernelGGL((attn_bf16_pipe_kernel<D, CAUSAL, OUT>), dim3(8 * p.per_xcd), dim3(256), 0, stream, p);
    return;
  }
  const int bm = a.in_dtype == LITEVLM_F32 ? 64 : 128;
  p.n_mtiles = (a.max_seqlen + bm - 1) / bm;
  p.n_work = p.n_mtiles * a.Hq * a.B;
  p.per_xcd = (p.n_work + 7) / 8;
  const dim3 grid(8 * p.per_xcd);
  if (a.in_dtype == LITEVLM_BF16)
    hipLaunchKernelGGL((attn_bf16_kernel<D, CAUSAL, OUT>), grid, dim3(256), 0, stream, p);
  else if (a.in_dtype == LITEVLM_FP8_E4M3)
    hipLaunchKernelGGL((attn_fp8_kernel<D, CAUSAL, OUT>), grid, dim3(256), 0, stream, p);
  else
    hipLaunchKernelGGL((attn_fwd_f32_kernel<D, CAUSAL, OUT>), grid, dim3(64), 0, stream, p);
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
