// Token Selection Module front end: the scoring queries and keys of the
// standalone first decoder layer, from the layer's input hidden states.
//
//   k[b, j]   = rope(r_j * x[b, j] W_k'^T, pos_j)   for every token j
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
// Tiling: a workgroup (4 waves) computes 128 rows x 128 output features; wave
// (wr, wc) holds rows 64*wr .. +64 and the column blocks c0 and c0 + D/64.
// A and B tiles of 32 columns of the model width stream global -> LDS directly
// (global_load_lds_dwordx4) through a 4-stage ring, three stages ahead of the
// MFMAs, into 64-byte rows whose four 16-byte pieces are XOR-swizzled by
// (row >> 1) & 3 so that each quarter-wave's operand reads hit distinct banks.
#include "common.hpp"
#include "launch.hpp"

namespace litevlm {
namespace {

constexpr int kMT = 128, kNT = 128, kKT = 32, kStages = 4;
constexpr int kRowB = kKT * 2;        // bytes per staged row
constexpr int kAB = kMT * kRowB;      // A tile bytes per stage
constexpr int kBB = kNT * kRowB;      // B tile bytes per stage
constexpr int kStageB = kAB + kBB;
constexpr int kRingB = kStages * kStageB;
constexpr int kLdsB = kRingB + kMT * 4 /* row factors */ + kMT * 4 /* positions */ + 64 /* reductions */;

struct TsmParams {
  const uint8_t* x;     // bf16 [B, S, Dm]
  const uint8_t* keep;  // uint8 [B, S] or NULL
  const uint8_t* wq;    // bf16 [Hq*D, Dm]
  const uint8_t* wk;    // bf16 [Hkv*D, Dm]
  uint16_t* q;          // bf16 [B, S, Hq, D]
  uint16_t* k;          // bf16 [B, S, Hkv, D]
  int B, S, V_full, Dm, Hq, Hkv;
  int mk, nk, mq, nq, n_k_items, n_items, per_xcd;
  float eps;
  double log2_theta;
};

template <int N>
__device__ __forceinline__ void vm_wait() {
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

__device__ __forceinline__ int swz(int row) { return (row >> 1) & 3; }

// Workgroup barrier that waits only for this wave's LDS operations: the
// __syncthreads fence would also wait for every direct copy still in flight,
// which would drain the ring each stage.
__device__ __forceinline__ void ring_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ __forceinline__ int acc_row(int r, int hl) { return 8 * (r >> 2) + 4 * hl + (r & 3); }

typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));

template <int D>
__global__ __launch_bounds__(256, 2) void tsm_proj_kernel(TsmParams p) {
  constexpr int PB = D / 64;  // column-block distance of rotary partners
  const int L = blockIdx.x;
  const int item = (L & 7) * p.per_xcd + (L >> 3);  // an XCD takes a contiguous item range
  if (item >= p.n_items) return;
  bool isq;
  int b, mt, nt;
  if (item < p.n_k_items) {
    isq = false;
    b = item / (p.mk * p.nk);
    const int r = item % (p.mk * p.nk);
    mt = r / p.nk;
    nt = r % p.nk;
  } else {
    const int j = item - p.n_k_items;
    isq = true;
    b = j / (p.mq * p.nq);
    const int r = j % (p.mq * p.nq);
    mt = r / p.nq;
    nt = r % p.nq;
  }
  const int row0 = (isq ? p.V_full : 0) + mt * kMT;  // first row of the tile within the sample
  const int nrows = min(kMT, p.S - row0);
  const int n0 = nt * kNT;
  const uint8_t* W = isq ? p.wq : p.wk;
  const int H = isq ? p.Hq : p.Hkv;
  const int Dm = p.Dm;

  __shared__ __attribute__((aligned(1024))) uint8_t lds[kLdsB];
  float* rs = reinterpret_cast<float*>(lds + kRingB);
  int* pos = reinterpret_cast<int*>(lds + kRingB + kMT * 4);
  int* red = reinterpret_cast<int*>(lds + kRingB + kMT * 8);

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wr = w & 1, wc = w >> 1, hl = lane >> 5, l32 = lane & 31;

  // ---- positions of the tile's rows in the patch-selected sequence
  {
    const uint8_t* kr = p.keep ? p.keep + (size_t)b * p.S : nullptr;
    int cnt = 0;
    if (kr)
      for (int j = tid; j < row0; j += 256) cnt += kr[j];
#pragma unroll
    for (int x = 1; x < kWave; x <<= 1) cnt += __shfl_xor(cnt, x, kWave);
    int f = 0;
    if (tid < kMT && tid < nrows) f = kr ? kr[row0 + tid] : 1;
    int incl = f;
#pragma unroll
    for (int x = 1; x < kWave; x <<= 1) {
      const int y = __shfl_up(incl, x, kWave);
      if (lane >= x) incl += y;
    }
    if (lane == 0) red[w] = cnt;
    if (lane == kWave - 1) red[4 + w] = incl;
    __syncthreads();
    if (tid < kMT) {
      const int base = kr ? red[0] + red[1] + red[2] + red[3] : row0;
      pos[tid] = base + (incl - f) + (w == 1 ? red[4] : 0);
    }
  }

  // ---- per-lane copy sources (fixed) and operand offsets (fixed)
  // copy j of a wave fills LDS pieces (w + 4j)*64 + lane of the A (resp. B) tile
  size_t asrc[2], bsrc[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int slot = (w + 4 * j) * 64 + lane;
    const int row = slot >> 2, logical = (slot & 3) ^ swz(slot >> 2);
    asrc[j] = ((size_t)((size_t)b * p.S + row0 + min(row, nrows - 1)) * Dm + logical * 8) * 2;
    bsrc[j] = ((size_t)(n0 + row) * Dm + logical * 8) * 2;
  }
  const uint32_t lds_w = __builtin_amdgcn_readfirstlane((uint32_t)w * 1024u);
  const int c0 = (D == 128) ? wc : 2 * wc;  // this wave's column blocks: c0 and c0 + PB
  uint32_t aoff[2][2], boff[2][2];          // [block][k16 step]
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const int logical = 2 * ks + hl;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const int row = 64 * wr + 32 * rb + l32;
      aoff[rb][ks] = row * kRowB + ((logical ^ swz(row)) * 16);
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int nrow = 32 * (c0 + c * PB) + l32;
      boff[c][ks] = kAB + nrow * kRowB + ((logical ^ swz(nrow)) * 16);
    }
  }

  auto copy_stage = [&](int s) __attribute__((always_inline)) {
    const size_t kb = (size_t)s * kKT * 2;
    uint8_t* st = lds + (s % kStages) * kStageB;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      __builtin_amdgcn_global_load_lds((const void*)(p.x + asrc[j] + kb),
                                       (__attribute__((address_space(3))) void*)(st + lds_w + 4 * j * 1024), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((const void*)(W + bsrc[j] + kb),
                                       (__attribute__((address_space(3))) void*)(st + kAB + lds_w + 4 * j * 1024), 16,
                                       0, 0);
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[rb][c][r] = 0.f;
  float ssq[2] = {0.f, 0.f};

  const int nK = Dm / kKT;
  for (int s = 0; s < kStages - 1 && s < nK; ++s) copy_stage(s);
  for (int s = 0; s < nK; ++s) {
    // stage s has landed once at most the copies of the later issued stages remain
    if (s + 2 < nK) vm_wait<8>();
    else if (s + 1 < nK) vm_wait<4>();
    else vm_wait<0>();
    ring_barrier();  // every wave's copies of stage s are visible; ring slot (s-1)%4 is free
    if (s + kStages - 1 < nK) copy_stage(s + kStages - 1);
    const uint8_t* st = lds + (s % kStages) * kStageB;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 a[2], bo[2];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) a[rb] = *reinterpret_cast<const bf16x8*>(st + aoff[rb][ks]);
#pragma unroll
      for (int c = 0; c < 2; ++c) bo[c] = *reinterpret_cast<const bf16x8*>(st + boff[c][ks]);
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int c = 0; c < 2; ++c) acc[rb][c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[rb], bo[c], acc[rb][c], 0, 0, 0);
      if (wc == 0) {  // row sums of squares, from the A operands (one wave per row half)
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
          const u32x4v u = __builtin_bit_cast(u32x4v, a[rb]);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float lo = __uint_as_float(u[e] << 16), hi = __uint_as_float(u[e] & 0xFFFF0000u);
            ssq[rb] = fmaf(lo, lo, ssq[rb]);
            ssq[rb] = fmaf(hi, hi, ssq[rb]);
          }
        }
      }
    }
  }

  // ---- epilogue: RMS factor per row, rotary embedding, bf16 store
  if (wc == 0) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const float tot = sum_xor32(ssq[rb]);
      if (hl == 0) rs[64 * wr + 32 * rb + l32] = 1.f / sqrtf(tot / (float)Dm + p.eps);
    }
  }
  __syncthreads();
  const int d = (32 * c0) % D + l32;  // element of the first half of its head (d < D/2)
  const int head = (n0 + 32 * c0) / D;
  const double inv_freq = exp2(-(2.0 * d / D) * p.log2_theta);
  uint16_t* out = isq ? p.q : p.k;
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 64 * wr + 32 * rb + acc_row(r, hl);
      if (row < nrows) {
        const float f = rs[row];
        const float x1 = acc[rb][0][r] * f, x2 = acc[rb][1][r] * f;
        // angle pos * theta^(-2d/D), reduced to [-pi, pi] in double
        double a = (double)pos[row] * inv_freq;
        a -= 6.283185307179586 * rint(a * 0.15915494309189535);
        float sn, cs;
        sincosf((float)a, &sn, &cs);
        uint16_t* o = out + (((size_t)b * p.S + row0 + row) * H + head) * D;
        o[d] = f32_to_bf16_bits(x1 * cs - x2 * sn);
        o[d + D / 2] = f32_to_bf16_bits(x2 * cs + x1 * sn);
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
  const int T = a.S - a.V_full;
  p.mk = (a.S + kMT - 1) / kMT;
  p.nk = a.Hkv * a.D / kNT;
  p.mq = (T + kMT - 1) / kMT;
  p.nq = a.Hq * a.D / kNT;
  p.n_k_items = a.B * p.mk * p.nk;
  p.n_items = p.n_k_items + a.B * p.mq * p.nq;
  p.per_xcd = (p.n_items + 7) / 8;
  p.eps = a.eps;
  p.log2_theta = log2((double)a.rope_theta);
  const dim3 grid(8 * p.per_xcd);
  if (a.D == 128) hipLaunchKernelGGL((tsm_proj_kernel<128>), grid, dim3(256), 0, stream, p);
  else hipLaunchKernelGGL((tsm_proj_kernel<64>), grid, dim3(256), 0, stream, p);
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
