// GEMMs of the MMDiT block (QKV, output projection, MLP), with the bias,
// GELU and gated-residual epilogues fused.
//
// bf16 path (MFMA):
//  - Macro tile 256 x BN (BN in {256, 192, 128}) x 64, one 512-thread
//    workgroup of 8 waves (2 x 4, or 4 x 2 for BN = 192), each wave a
//    128 x 64 (64 x 96) block of v_mfma_f32_32x32x16_bf16 tiles; two
//    waves per SIMD hide each other's LDS and barrier waits.  The 256-wide
//    tile runs the ping-pong form (gemm_bf16_pp_kernel): the two halves of
//    the workgroup alternate compute and memory phases.
//  - The MFMA computes C^T = W A^T, so each lane owns groups of four
//    consecutive output columns of one row (8-byte stores in the epilogue).
//  - k-tiles are staged global -> registers -> LDS through two LDS buffers,
//    one barrier per k-tile: while tile t is multiplied, tile t+1 is in
//    flight (and, for the 128-wide tile, tile t+2 too).  LDS rows are 128 bytes (64 bf16) with the 16-byte chunk index
//    XOR-swizzled by (row / 2) mod 8, which makes both the staging writes and
//    the 16-byte fragment reads of 16 consecutive rows bank-conflict free.
//  - The epilogue goes through LDS wave by wave so that every store covers
//    whole row segments (or, for the transposed store, column runs).
//  - Small-N GEMMs (the N = D projections) are split along K when the tile
//    grid would leave most of the 256 CUs idle: each split writes fp32
//    partials and a reduce kernel sums them in split order (deterministic)
//    and applies the epilogue.  When the 256-wide tiles overrun the last
//    full wave of workgroups by a few (the MLP-in projection of the FLUX
//    block: 336 tiles on 256 CUs), only those last tiles are split (the
//    split tail): they run after the whole tiles, in 2-4 k splits, and a
//    small reduce sums their partials, so the partial wave takes a fraction
//    of a tile's time instead of a whole one.
// fp32 path: 64x64 tiles on the VALU (the exactness path).
#include <stdio.h>
#include <stdlib.h>

#include "kernels.h"

namespace avits {
namespace {

constexpr int kBM = 256, kBK = 64;
constexpr int kCUs = 256;

// GELU with the tanh approximation written through the logistic function:
// 0.5 (1 + tanh(u)) = 1 / (1 + exp(-2u)), on the hardware exp2 and
// reciprocal (about 1 ulp each; the result is rounded to bf16).  Large |x|
// saturate to x and -0.
__device__ __forceinline__ float gelu_fast(float x) {
  const float u = 0.7978845608028654f * (x + 0.044715f * x * x * x);
  const float e = __builtin_amdgcn_exp2f(-2.f * 1.4426950408889634f * u);
  return x * __builtin_amdgcn_rcpf(1.f + e);
}

__device__ __forceinline__ f32x16 mfma32x32x16(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// The fused scatter: region 0's final row m (columns from col, stored as
// the vector w) also goes to its canvas row, when the problem has one.
template <typename T, typename V>
__device__ __forceinline__ void scatter_copy(const GemmProblem& p, int64_t m, int64_t col, const V& w) {
  if (!p.scat || m < p.scat_row0) return;
  const int64_t q = p.scat_idx[m - p.scat_row0];
  if (q < 0 || q >= p.scat_n) return;
  *reinterpret_cast<V*>(static_cast<T*>(p.scat) + q * p.scat_ld + col) = w;
}

// Epilogue for four consecutive columns n..n+3 of row m of problem p (the
// four columns never straddle a region boundary: region starts are
// multiples of 4).
template <typename T>
__device__ __forceinline__ void epilogue4(const GemmArgs& a, const GemmProblem& p, int64_t m, int64_t n,
                                          float v0, float v1, float v2, float v3) {
  float v[4] = {v0, v1, v2, v3};
  if (p.bias) {
    const T* b = static_cast<const T*>(p.bias);
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] += ld(b, n + r);
  }
  int mode;
  T* out;
  int64_t col, ldo;
  if (n < a.n_split) {
    mode = a.mode0; out = static_cast<T*>(p.out0); col = n; ldo = p.ld0;
  } else if (n < a.n_split2) {
    mode = a.mode1; out = static_cast<T*>(p.out1); col = n - a.n_split; ldo = p.ld1;
  } else {
    mode = a.mode2; out = static_cast<T*>(p.out2); col = n - a.n_split2; ldo = p.ld2;
  }
  if (mode == EPI_GELU) {
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = gelu_fast(v[r]);
  } else if (mode == EPI_RESID_GATE) {
    const T* res = static_cast<const T*>(p.resid);
    const T* gt = static_cast<const T*>(p.gate);
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = ld(res, m * p.ldr + col + r) + ld(gt, n + r) * v[r];
  } else if (mode == EPI_STORE_T) {
#pragma unroll
    for (int r = 0; r < 4; ++r) st(out, (col + r) * ldo + m, v[r]);
    return;
  }
  T* dst = out + m * ldo + col;
  if constexpr (sizeof(T) == 2) {
    u32x2 w = {pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3])};
    *reinterpret_cast<u32x2*>(dst) = w;
    if (n < a.n_split) scatter_copy<T>(p, m, col, w);
  } else {
    const float4 w = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4*>(dst) = w;
    if (n < a.n_split) scatter_copy<T>(p, m, col, w);
  }
}

// Eight consecutive columns of one row (bf16 output): 16-byte loads of the
// bias, gate and residual and one 16-byte store when the eight columns share
// one output region with a row-major mode and aligned strides; otherwise two
// epilogue4 calls.  Same arithmetic, in the same order, as epilogue4.
__device__ __forceinline__ void epilogue8(const GemmArgs& a, const GemmProblem& p, int64_t m, int64_t n,
                                          const float (&v)[8]) {
  const bool r0 = n < a.n_split, r1 = n < a.n_split2;
  int mode;
  bf16_t* out;
  int64_t col, ldo;
  if (r0) { mode = a.mode0; out = static_cast<bf16_t*>(p.out0); col = n; ldo = p.ld0; }
  else if (r1) { mode = a.mode1; out = static_cast<bf16_t*>(p.out1); col = n - a.n_split; ldo = p.ld1; }
  else { mode = a.mode2; out = static_cast<bf16_t*>(p.out2); col = n - a.n_split2; ldo = p.ld2; }
  const bool same = r0 == (n + 7 < a.n_split) && r1 == (n + 7 < a.n_split2);
  const bool aligned = ((col | ldo) & 7) == 0 && (mode != EPI_RESID_GATE || (p.ldr & 7) == 0);
  if (!same || !aligned || mode == EPI_STORE_T) {
    epilogue4<bf16_t>(a, p, m, n, v[0], v[1], v[2], v[3]);
    epilogue4<bf16_t>(a, p, m, n + 4, v[4], v[5], v[6], v[7]);
    return;
  }
  float x[8];
  if (p.bias) {
    const u32x4 b = *reinterpret_cast<const u32x4*>(static_cast<const bf16_t*>(p.bias) + n);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = v[2 * e] + __uint_as_float(b[e] << 16);
      x[2 * e + 1] = v[2 * e + 1] + __uint_as_float(b[e] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = v[e];
  }
  if (mode == EPI_GELU) {
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = gelu_fast(x[e]);
  } else if (mode == EPI_RESID_GATE) {
    const u32x4 r = *reinterpret_cast<const u32x4*>(static_cast<const bf16_t*>(p.resid) + m * p.ldr + col);
    const u32x4 g = *reinterpret_cast<const u32x4*>(static_cast<const bf16_t*>(p.gate) + n);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = __uint_as_float(r[e] << 16) + __uint_as_float(g[e] << 16) * x[2 * e];
      x[2 * e + 1] = __uint_as_float(r[e] & 0xffff0000u) + __uint_as_float(g[e] & 0xffff0000u) * x[2 * e + 1];
    }
  }
  const u32x4 w = {pack_bf2(x[0], x[1]), pack_bf2(x[2], x[3]), pack_bf2(x[4], x[5]), pack_bf2(x[6], x[7])};
  *reinterpret_cast<u32x4*>(out + m * ldo + col) = w;
  if (r0) scatter_copy<bf16_t>(p, m, col, w);
}

// Split-K reduce fused with the modulated layer norm that follows the
// output projection: one wave per output row (N = D columns, 8 per chunk,
// chunk c of lane l at columns 8 (l + 64 c)).  The row's partials are summed
// in split order, the bias and gated residual applied as epilogue4 does, the
// result rounded to bf16 and stored; the layer norm then reads those bf16
// values with the chunk layout and summation order of ln_mod_kernel, so both
// routes give the same bits.
constexpr int kRlnChunks = 8;  // rows up to 64 * 8 * 8 = 4096 columns
template <int SPLITS>
__global__ __launch_bounds__(256) void splitk_reduce_ln_kernel(const GemmArgs a, const float* __restrict__ partial,
                                                               const GemmPostLN post) {
  const int lane = threadIdx.x % kWave;
  const int64_t rows = a.p[0].M + (a.nprob > 1 ? a.p[1].M : 0);
  const int64_t grow = int64_t(blockIdx.x) * 4 + threadIdx.x / kWave;
  if (grow >= rows) return;
  const bool second = grow >= a.p[0].M;
  const int64_t m = second ? grow - a.p[0].M : grow;
  const GemmProblem& p = second ? a.p[1] : a.p[0];
  const int64_t nchunk = a.N / 8;
  // This row's image's gate and LN modulation (one set when a.mod.B == 0).
  const int64_t moff = mod_offset(a.mod, p.row0 + m);
  const bf16_t* bias = static_cast<const bf16_t*>(p.bias);
  const bf16_t* gate = static_cast<const bf16_t*>(p.gate) + moff;
  const bf16_t* res = static_cast<const bf16_t*>(p.resid) + m * p.ldr;
  bf16_t* y = static_cast<bf16_t*>(p.out0) + m * p.ld0;
  u32x4 yv[kRlnChunks];
#pragma unroll
  for (int c = 0; c < kRlnChunks; ++c) {
    const int64_t idx = lane + kWave * c;
    if (idx >= nchunk) continue;
    const int64_t n = 8 * idx;
    float v[8];
#pragma unroll
    for (int k = 0; k < SPLITS; ++k) {
      const float* src = partial + (int64_t(k) * rows + grow) * a.N + n;
      const float4 x0 = *reinterpret_cast<const float4*>(src), x1 = *reinterpret_cast<const float4*>(src + 4);
      const float t[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = k == 0 ? t[e] : v[e] + t[e];
    }
    const u32x4 rw = *reinterpret_cast<const u32x4*>(res + n);
    const u32x4 gw = *reinterpret_cast<const u32x4*>(gate + n);
    const u32x4 bw = bias ? *reinterpret_cast<const u32x4*>(bias + n) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = __uint_as_float(rw[e] << 16) +
                       __uint_as_float(gw[e] << 16) * (v[2 * e] + __uint_as_float(bw[e] << 16));
      const float hi = __uint_as_float(rw[e] & 0xffff0000u) +
                       __uint_as_float(gw[e] & 0xffff0000u) * (v[2 * e + 1] + __uint_as_float(bw[e] & 0xffff0000u));
      yv[c][e] = pack_bf2(lo, hi);
    }
    *reinterpret_cast<u32x4*>(y + n) = yv[c];
    scatter_copy<bf16_t>(p, m, n, yv[c]);
  }
  // Modulated layer norm of the bf16 row.
  const bf16_t* sc = static_cast<const bf16_t*>(post.scale[second ? 1 : 0]) + moff;
  const bf16_t* sh = static_cast<const bf16_t*>(post.shift[second ? 1 : 0]) + moff;
  bf16_t* hr = static_cast<bf16_t*>(post.out) + grow * post.ld;
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kRlnChunks; ++c) {
    if (lane + kWave * c >= nchunk) continue;
#pragma unroll
    for (int e = 0; e < 4; ++e) s += __uint_as_float(yv[c][e] << 16) + __uint_as_float(yv[c][e] & 0xffff0000u);
  }
  const float mean = wave_sum(s) / float(a.N);
  float q = 0.f;
#pragma unroll
  for (int c = 0; c < kRlnChunks; ++c) {
    if (lane + kWave * c >= nchunk) continue;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float x0 = __uint_as_float(yv[c][e] << 16) - mean, x1 = __uint_as_float(yv[c][e] & 0xffff0000u) - mean;
      q = fmaf(x0, x0, fmaf(x1, x1, q));
    }
  }
  const float rstd = rsqrtf(wave_sum(q) / float(a.N) + 1e-6f);
#pragma unroll
  for (int c = 0; c < kRlnChunks; ++c) {
    const int64_t idx = lane + kWave * c;
    if (idx >= nchunk) continue;
    const u32x4 g = reinterpret_cast<const u32x4*>(sc)[idx], t = reinterpret_cast<const u32x4*>(sh)[idx];
    u32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = (__uint_as_float(yv[c][e] << 16) - mean) * rstd * (1.f + __uint_as_float(g[e] << 16)) +
                       __uint_as_float(t[e] << 16);
      const float hi = (__uint_as_float(yv[c][e] & 0xffff0000u) - mean) * rstd *
                           (1.f + __uint_as_float(g[e] & 0xffff0000u)) +
                       __uint_as_float(t[e] & 0xffff0000u);
      o[e] = pack_bf2(lo, hi);
    }
    reinterpret_cast<u32x4*>(hr)[idx] = o;
  }
}

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own
// L2).  Renumber them so that XCD x runs a contiguous range of logical ids:
// neighbouring logical tiles share weight / activation tiles in one L2.
__device__ __forceinline__ int64_t xcd_logical_id(int64_t bid, int64_t grid) {
  constexpr int kXcds = 8;
  const int64_t per = grid / kXcds, rem = grid % kXcds;
  const int64_t x = bid % kXcds, i = bid / kXcds;
  return x < rem ? x * (per + 1) + i : rem * (per + 1) + (x - rem) * per + i;
}

// Logical tile -> (problem, tile origin).  Tiles of one problem come first;
// within a problem, consecutive tiles walk down the rows of one column block
// so neighbouring workgroups share the weight tile.
__device__ __forceinline__ bool decode_tile(const GemmArgs& a, int bm, int bn, int64_t tile, int& prob, int64_t& m0,
                                            int64_t& n0) {
  const int64_t tn = (a.N + bn - 1) / bn;
  const int64_t tm0 = (a.p[0].M + bm - 1) / bm;
  const int64_t t0 = tm0 * tn;
  prob = 0;
  int64_t tm = tm0;
  if (tile >= t0) {
    tile -= t0;
    prob = 1;
    if (a.nprob < 2) return false;
    tm = (a.p[1].M + bm - 1) / bm;
  }
  if (tm == 0) return false;
  m0 = (tile % tm) * bm;
  n0 = (tile / tm) * bn;
  return m0 < a.p[prob].M && n0 < a.N;
}

__device__ __forceinline__ int64_t tiles_total(const GemmArgs& a, int bm, int bn) {
  const int64_t tn = (a.N + bn - 1) / bn;
  return ((a.p[0].M + bm - 1) / bm + (a.nprob > 1 ? (a.p[1].M + bm - 1) / bm : 0)) * tn;
}

// Workgroup -> (problem, tile origin, k split): the k splits of a tile are
// adjacent logical ids.
__device__ __forceinline__ bool map_tile(const GemmArgs& a, int bm, int bn, int splits, int& prob, int64_t& m0,
                                         int64_t& n0, int& ks) {
  const int64_t bid = xcd_logical_id(blockIdx.x, gridDim.x);
  ks = int(bid % splits);
  return decode_tile(a, bm, bn, bid / splits, prob, m0, n0);
}

// Split tail.  When the tiles overrun the last full wave of workgroups on the
// chip by a few, the first F = tiles - tail tiles run whole (workgroups
// 0 .. F - 1) and the last `tail` tiles run in `tsp` k splits each
// (workgroups F onwards, dispatched after the whole tiles): the partial wave
// takes 1 / tsp of a tile's time instead of a whole one.  The two classes are
// renumbered for the XCDs separately.  tidx is the tile's index in the tail
// (-1 for a whole tile).
__device__ __forceinline__ bool map_tile_tail(const GemmArgs& a, int bm, int bn, int64_t tail, int tsp, int& prob,
                                              int64_t& m0, int64_t& n0, int& ks, int64_t& tidx) {
  const int64_t F = tiles_total(a, bm, bn) - tail;
  const int64_t bid = blockIdx.x;
  if (bid < F) {
    ks = 0;
    tidx = -1;
    return decode_tile(a, bm, bn, xcd_logical_id(bid, F), prob, m0, n0);
  }
  const int64_t u = xcd_logical_id(bid - F, int64_t(gridDim.x) - F);
  tidx = u / tsp;
  ks = int(u % tsp);
  return decode_tile(a, bm, bn, F + tidx, prob, m0, n0);
}

// Epilogue through LDS, wave by wave.  The MFMA layout gives each lane four
// consecutive columns of one row, so storing straight from the accumulators
// would send every store instruction to 32 different rows.  Instead each wave
// turns its block around in its own LDS region, 32 rows at a time (no
// workgroup barrier: a wave's LDS operations complete in order): it writes
// the 32 x WN fp32 accumulators, reads them back row-major (WN / 4 lanes per
// row, four columns each) and stores whole row segments; the columns of a
// transposed region are read down the rows instead (four lanes per column,
// eight rows each), so each column's 32 rows go out as one 64-byte run.  A
// lane keeps the same columns for all rows, so its bias, gate, output region
// and mode are loaded once.  The LDS column of a value is XOR-swizzled by 8
// times its 8-row group (WN is a multiple of 32), so the down-the-rows reads
// of a half-wave hit 32 distinct banks and 4-column groups stay aligned.  Split-K
// partials take the row-major path without the epilogue.  The caller passes
// the main loop's LDS once every wave is done with it.
template <int WM, int WN, int TM, int TN>
__device__ __forceinline__ void staged_epilogue(const GemmArgs& a, const GemmProblem& p, int64_t m0, int64_t n0,
                                                bool part, float* __restrict__ pbase, int64_t pld,
                                                const f32x16 (&acc)[TM][TN], float* sm, int wave, int wm, int wn,
                                                int lane) {
  constexpr int P = WN + 4;                  // LDS row pitch (floats)
  constexpr int kLPR = WN / 4;               // lanes per row
  constexpr int kRPI = kWave / kLPR;         // rows per row-major sweep
  constexpr int kIt = 32 / kRPI;             // row-major sweeps per 32-row block
  constexpr int kTIt = WN * 4 / kWave;       // down-the-rows sweeps per 32-row block
  static_assert(32 % kRPI == 0 && (WN * 4) % kWave == 0, "epilogue lane layout");
  float* reg = sm + wave * 32 * P;
  const int l32 = lane % 32, hi = lane / 32;
  auto swz_col = [](int row, int col) { return col ^ (((row >> 3) & 3) << 3); };
  auto mode_of = [&](int64_t n) { return n < a.n_split ? a.mode0 : n < a.n_split2 ? a.mode1 : a.mode2; };

  // Row-major role of this lane: columns n .. n + 3, rows r0 + kRPI * it.
  const int c4 = lane % kLPR, r0 = lane / kLPR;
  const int64_t nb = n0 + wn * WN, n = nb + 4 * c4;
  const bool lane_ok = r0 < kRPI && n < a.N;
  const int mode = lane_ok ? mode_of(n) : EPI_STORE;
  bf16_t* out = nullptr;
  int64_t col = 0, ldo = 0;
  if (n < a.n_split) { out = static_cast<bf16_t*>(p.out0); col = n; ldo = p.ld0; }
  else if (n < a.n_split2) { out = static_cast<bf16_t*>(p.out1); col = n - a.n_split; ldo = p.ld1; }
  else { out = static_cast<bf16_t*>(p.out2); col = n - a.n_split2; ldo = p.ld2; }
  float bias[4] = {0.f, 0.f, 0.f, 0.f}, gate[4] = {0.f, 0.f, 0.f, 0.f};
  if (lane_ok && !part) {
    if (p.bias) {
#pragma unroll
      for (int r = 0; r < 4; ++r) bias[r] = ld(static_cast<const bf16_t*>(p.bias), n + r);
    }
    if (mode == EPI_RESID_GATE) {
#pragma unroll
      for (int r = 0; r < 4; ++r) gate[r] = ld(static_cast<const bf16_t*>(p.gate), n + r);
    }
  }
  const bool row_major = lane_ok && (part || mode != EPI_STORE_T);
  const bool has_t = !part && (a.mode0 == EPI_STORE_T || a.mode1 == EPI_STORE_T || a.mode2 == EPI_STORE_T);

#pragma unroll
  for (int i = 0; i < TM; ++i) {
    // acc[i][j][4q + r] = C[row 32 i + l32][col 32 j + 8 q + 4 hi + r] of this wave's block.
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x16& c = acc[i][j];
        *reinterpret_cast<float4*>(reg + l32 * P + swz_col(l32, 32 * j + 8 * q + 4 * hi)) =
            make_float4(c[4 * q], c[4 * q + 1], c[4 * q + 2], c[4 * q + 3]);
      }
    const int64_t mb = m0 + wm * WM + 32 * i;  // first output row of the block
    if (row_major) {
      float4 u[kIt];
#pragma unroll
      for (int it = 0; it < kIt; ++it) {
        const int rr = r0 + kRPI * it;
        u[it] = *reinterpret_cast<const float4*>(reg + rr * P + swz_col(rr, 4 * c4));
      }
      if (part) {
#pragma unroll
        for (int it = 0; it < kIt; ++it) {
          const int64_t m = mb + r0 + kRPI * it;
          if (m < p.M) *reinterpret_cast<float4*>(pbase + (m - m0) * pld + (n - n0)) = u[it];
        }
      } else {
        float res[kIt][4];
        if (mode == EPI_RESID_GATE) {
          const bf16_t* rp = static_cast<const bf16_t*>(p.resid);
#pragma unroll
          for (int it = 0; it < kIt; ++it) {
            const int64_t m = std::min<int64_t>(mb + r0 + kRPI * it, p.M - 1);
            const u32x2 w = *reinterpret_cast<const u32x2*>(rp + m * p.ldr + col);
            res[it][0] = __uint_as_float(w[0] << 16);
            res[it][1] = __uint_as_float(w[0] & 0xffff0000u);
            res[it][2] = __uint_as_float(w[1] << 16);
            res[it][3] = __uint_as_float(w[1] & 0xffff0000u);
          }
        }
#pragma unroll
        for (int it = 0; it < kIt; ++it) {
          const int64_t m = mb + r0 + kRPI * it;
          if (m >= p.M) continue;
          float v[4] = {u[it].x + bias[0], u[it].y + bias[1], u[it].z + bias[2], u[it].w + bias[3]};
          if (mode == EPI_GELU) {
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = gelu_fast(v[r]);
          } else if (mode == EPI_RESID_GATE) {
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = res[it][r] + gate[r] * v[r];
          }
          const u32x2 w = {pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3])};
          *reinterpret_cast<u32x2*>(out + m * ldo + col) = w;
          if (n < a.n_split) scatter_copy<bf16_t>(p, m, col, w);
        }
      }
    }
    if (has_t) {
#pragma unroll
      for (int it = 0; it < kTIt; ++it) {
        const int item = it * kWave + lane;
        const int tc = item / 4, mc = item % 4;   // column of the block, 8-row group
        const int64_t nt = nb + tc, m = mb + 8 * mc;
        if (nt >= a.N || m >= p.M || mode_of(nt) != EPI_STORE_T) continue;
        const bf16_t* bp = static_cast<const bf16_t*>(p.bias);
        const float b = bp ? ld(bp, nt) : 0.f;
        bf16_t* o;
        int64_t c0, lo;
        if (nt < a.n_split) { o = static_cast<bf16_t*>(p.out0); c0 = nt; lo = p.ld0; }
        else if (nt < a.n_split2) { o = static_cast<bf16_t*>(p.out1); c0 = nt - a.n_split; lo = p.ld1; }
        else { o = static_cast<bf16_t*>(p.out2); c0 = nt - a.n_split2; lo = p.ld2; }
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = reg[(8 * mc + e) * P + swz_col(8 * mc + e, tc)] + b;
        bf16_t* dst = o + c0 * lo + m;
        if (m + 8 <= p.M) {
          const u32x4 w = {pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[4], v[5]), pack_bf2(v[6], v[7])};
          *reinterpret_cast<u32x4*>(dst) = w;
        } else {
          for (int e = 0; m + e < p.M; ++e) st(dst, e, v[e]);
        }
      }
    }
  }
}

// Swizzled 16-byte chunk slot of (row, chunk) in a 128-byte LDS row.
__device__ __forceinline__ int swz(int row, int chunk) { return row * 8 + (chunk ^ ((row >> 1) & 7)); }

template <int BN, int WAVES_M, int WAVES_N, int STAGES>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N) void gemm_bf16_kernel(const GemmArgs a,
                                                                           float* __restrict__ partial, int splits) {
  constexpr int NT = 64 * WAVES_M * WAVES_N;
  constexpr int WM = kBM / WAVES_M, WN = BN / WAVES_N;
  constexpr int TM = WM / 32, TN = WN / 32;  // 32x32 MFMA tiles per wave
  constexpr int CA = kBM * 8 / NT;           // 16-byte A chunks staged per thread per k-tile
  constexpr int CW = BN * 8 / NT;
  constexpr int RS = NT / 8;                 // rows between a thread's chunks
  static_assert(WM % 32 == 0 && WN % 32 == 0 && (BN * 8) % NT == 0 && RS % 16 == 0, "tile shape");
  __shared__ u32x4 lds[2][(kBM + BN) * 8];

  int prob, ks;
  int64_t m0, n0;
  if (!map_tile(a, kBM, BN, splits, prob, m0, n0, ks)) return;
  const GemmProblem p = prob ? a.p[1] : a.p[0];  // by value: a select, no indexed copy of the arguments
  const bf16_t* A = static_cast<const bf16_t*>(p.A);
  const bf16_t* W = static_cast<const bf16_t*>(p.W);
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int l32 = lane % 32, hi = lane / 32;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;

  const int64_t nk = a.K / kBK;
  const int64_t kt0 = nk * ks / splits, kt1 = nk * (ks + 1) / splits;

  // Staging: thread t moves 16-byte chunk (t % 8) of rows t / 8 + RS j, so all
  // of its chunks share one column offset and one swizzle (RS j / 2 = 0 mod 8).
  // Loads are raw buffer loads with loop-invariant per-thread offsets; the
  // k-advance moves the scalar resource base.  The resource covers only the
  // rows that exist, so the range check returns zeros past the end of A or W.
  constexpr int LPT = CA + CW;  // loads per thread per k-tile
  const int row_t = tid / 8, kc_t = tid % 8;
  const int slot_t = row_t * 8 + (kc_t ^ ((row_t >> 1) & 7));
  uint32_t a_off[CA], w_off[CW];
#pragma unroll
  for (int j = 0; j < CA; ++j) a_off[j] = uint32_t(((row_t + RS * j) * p.lda + kc_t * 8) * 2);
#pragma unroll
  for (int j = 0; j < CW; ++j) w_off[j] = uint32_t(((row_t + RS * j) * a.K + kc_t * 8) * 2);
  const char* a_base = reinterpret_cast<const char*>(A + m0 * p.lda);
  const char* w_base = reinterpret_cast<const char*>(W + n0 * a.K);
  const int64_t a_bytes = (p.M - m0) * p.lda * 2, w_bytes = (a.N - n0) * a.K * 2;
  struct Stage {
    u32x4 a[CA], w[CW];
  };
  auto load_tile = [&](Stage& st, int64_t kt) {
    const int64_t koff = kt * kBK * 2;
    const u32x4 ra = buffer_rsrc(a_base + koff, range32(a_bytes - koff));
    const u32x4 rw = buffer_rsrc(w_base + koff, range32(w_bytes - koff));
#pragma unroll
    for (int j = 0; j < CA; ++j) buffer_load16(st.a[j], ra, a_off[j]);
#pragma unroll
    for (int j = 0; j < CW; ++j) buffer_load16(st.w[j], rw, w_off[j]);
  };
  auto ready = [&](Stage& st) {
#pragma unroll
    for (int j = 0; j < CA; ++j) vm_ready(st.a[j]);
#pragma unroll
    for (int j = 0; j < CW; ++j) vm_ready(st.w[j]);
  };
  auto store_tile = [&](const Stage& st, int buf) {
#pragma unroll
    for (int j = 0; j < CA; ++j) lds[buf][slot_t + RS * 8 * j] = st.a[j];
#pragma unroll
    for (int j = 0; j < CW; ++j) lds[buf][kBM * 8 + slot_t + RS * 8 * j] = st.w[j];
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Fragments are double-buffered across the 16-wide k steps: the LDS reads
  // of step kk + 1 are in flight while the MFMAs of step kk run, so a wave
  // rarely stalls on LDS latency.
  auto compute = [&](int buf) {
    const u32x4* L = lds[buf];
    bf16x8 af[2][TM], wf[2][TN];
    auto read = [&](int kk, int slot) {
      const int chunk = 2 * kk + hi;
#pragma unroll
      for (int i = 0; i < TM; ++i) af[slot][i] = as_bf16x8(L[swz(wm * WM + 32 * i + l32, chunk)]);
#pragma unroll
      for (int j = 0; j < TN; ++j) wf[slot][j] = as_bf16x8(L[kBM * 8 + swz(wn * WN + 32 * j + l32, chunk)]);
    };
    read(0, 0);
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      if (kk + 1 < kBK / 16) read(kk + 1, (kk + 1) & 1);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32x32x16(wf[kk & 1][j], af[kk & 1][i], acc[i][j]);
    }
  };

  const int64_t n_t = kt1 - kt0;
  if constexpr (STAGES == 2) {
    // Software pipeline, two register stages and two LDS buffers: while
    // k-tile t is multiplied from LDS, tile t + 1 (loaded one step earlier)
    // is stored to the other buffer and tile t + 2 is in flight.  Loads
    // complete in issue order, so "the older stage is ready" is
    // vmcnt <= LPT while the newer stage is in flight, else vmcnt == 0.
    Stage s0, s1;
    if (n_t > 0) {
      load_tile(s0, kt0);
      if (n_t > 1) {
        load_tile(s1, kt0 + 1);
        vm_wait<LPT>();
      } else {
        vm_wait<0>();
      }
      ready(s0);
      store_tile(s0, 0);
    }
    lds_barrier();
    for (int64_t t = 0; t < n_t; t += 2) {
      // even step: compute buffer 0; s1 holds tile t + 1.
      const bool next2 = t + 2 < n_t;
      if (next2) load_tile(s0, kt0 + t + 2);
      compute(0);
      if (t + 1 < n_t) {
        if (next2) vm_wait<LPT>(); else vm_wait<0>();
        ready(s1);
        store_tile(s1, 1);
      }
      lds_barrier();
      if (t + 1 >= n_t) break;
      // odd step: compute buffer 1; s0 holds tile t + 2.
      const bool next3 = t + 3 < n_t;
      if (next3) load_tile(s1, kt0 + t + 3);
      compute(1);
      if (next2) {
        if (next3) vm_wait<LPT>(); else vm_wait<0>();
        ready(s0);
        store_tile(s0, 0);
      }
      lds_barrier();
    }
  } else {
    // One register stage, two LDS buffers: tile t + 1 is in flight while
    // tile t is multiplied.
    Stage st;
    if (n_t > 0) {
      load_tile(st, kt0);
      vm_wait<0>();
      ready(st);
      store_tile(st, 0);
    }
    lds_barrier();
    for (int64_t t = 0; t < n_t; ++t) {
      const int buf = int(t & 1);
      const bool next = t + 1 < n_t;
      if (next) load_tile(st, kt0 + t + 1);
      compute(buf);
      if (next) {
        vm_wait<0>();
        ready(st);
        store_tile(st, buf ^ 1);
      }
      lds_barrier();
    }
  }

  // The last barrier of the main loop has passed: LDS is free.
  const int64_t rows_all = a.p[0].M + (a.nprob > 1 ? a.p[1].M : 0);
  float* pbase = splits > 1 ? partial + (int64_t(ks) * rows_all + (prob ? a.p[0].M : 0) + m0) * a.N + n0 : nullptr;
  staged_epilogue<WM, WN, TM, TN>(a, p, m0, n0, splits > 1, pbase, a.N, acc,
                                  reinterpret_cast<float*>(&lds[0][0]), wave, wm, wn, lane);
}

// Ping-pong form of the 256 x 256 x 64 kernel.  The 8 waves form two groups
// of four (one wave of each group per SIMD); group g owns output rows
// [128 g, 128 g + 128) and each of its waves a 128 x 64 block.  The groups
// alternate between a compute phase (the 32 MFMAs of one k-tile, fragments
// read from LDS) and a memory phase (stage half of a later k-tile into LDS
// and issue the global loads of the half after it), one workgroup barrier
// per phase, offset by one phase: while one group's waves issue MFMAs the
// other group's waves on the same SIMDs do the memory work, so the matrix
// pipe of each SIMD is fed from one wave or the other in every phase.
//   phase 2t:     group 0 computes k-tile t;  group 1 stages its half of
//                 tile t + 1 and loads its half of tile t + 2;
//   phase 2t + 1: group 1 computes k-tile t;  group 0 stages / loads the same.
// Tile t lives in LDS buffer t mod 2: it is read in phases 2t and 2t + 1 and
// written in phases 2t - 2 and 2t - 1, after tile t - 2 left that buffer.
__global__ __launch_bounds__(512) void gemm_bf16_pp_kernel(const GemmArgs a, float* __restrict__ partial,
                                                          int splits, int64_t tail, int tsp) {
  constexpr int BN = 256, WM = 128, WN = 64;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int HALF = 4;                    // 16-byte chunks per thread per half-tile operand
  __shared__ u32x4 lds[2][(kBM + BN) * 8];

  int prob, ks;
  int64_t m0, n0, tidx = -1;
  if (tail > 0 ? !map_tile_tail(a, kBM, BN, tail, tsp, prob, m0, n0, ks, tidx)
               : !map_tile(a, kBM, BN, splits, prob, m0, n0, ks))
    return;
  const GemmProblem p = prob ? a.p[1] : a.p[0];  // by value: a select, no indexed copy of the arguments
  const bf16_t* A = static_cast<const bf16_t*>(p.A);
  const bf16_t* W = static_cast<const bf16_t*>(p.W);
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int l32 = lane % 32, hi = lane / 32;
  const int grp = __builtin_amdgcn_readfirstlane(wave / 4);
  const int wm = grp, wn = wave % 4;

  const int nsp = tidx >= 0 ? tsp : splits;
  const int64_t nk = a.K / kBK;
  const int64_t kt0 = nk * ks / nsp, kt1 = nk * (ks + 1) / nsp;
  const int64_t n_t = kt1 - kt0;

  // Staging of this group's half: A rows and W rows [128 grp, 128 grp + 128),
  // thread tg moves chunk tg % 8 of rows tg / 8 + 32 j (one swizzle for all j).
  const int tg = tid % 256;
  const int row_t = tg / 8, kc_t = tg % 8;
  const int slot_t = (128 * grp + row_t) * 8 + (kc_t ^ ((row_t >> 1) & 7));
  uint32_t a_off[HALF], w_off[HALF];
#pragma unroll
  for (int j = 0; j < HALF; ++j) {
    a_off[j] = uint32_t(((128 * grp + row_t + 32 * j) * p.lda + kc_t * 8) * 2);
    w_off[j] = uint32_t(((128 * grp + row_t + 32 * j) * a.K + kc_t * 8) * 2);
  }
  const char* a_base = reinterpret_cast<const char*>(A + m0 * p.lda);
  const char* w_base = reinterpret_cast<const char*>(W + n0 * a.K);
  const int64_t a_bytes = (p.M - m0) * p.lda * 2, w_bytes = (a.N - n0) * a.K * 2;
  // The staged loads stay in flight across the group's next compute phase
  // (a loop-carried value), so they are compiler-visible buffer loads: the
  // compiler places the vmcnt wait before the LDS store that consumes them.
  u32x4 sa[HALF], sw[HALF];
  auto load_half = [&](int64_t kt) {
    const int64_t koff = kt * kBK * 2;
    const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(a_base + koff), 0, int(range32(a_bytes - koff)), 0x00020000);
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(w_base + koff), 0, int(range32(w_bytes - koff)), 0x00020000);
#pragma unroll
    for (int j = 0; j < HALF; ++j) sa[j] = __builtin_amdgcn_raw_buffer_load_b128(ra, int(a_off[j]), 0, 0);
#pragma unroll
    for (int j = 0; j < HALF; ++j) sw[j] = __builtin_amdgcn_raw_buffer_load_b128(rw, int(w_off[j]), 0, 0);
  };
  auto store_half = [&](int buf) {
#pragma unroll
    for (int j = 0; j < HALF; ++j) lds[buf][slot_t + 256 * j] = sa[j];
#pragma unroll
    for (int j = 0; j < HALF; ++j) lds[buf][kBM * 8 + slot_t + 256 * j] = sw[j];
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto compute = [&](int buf) {
    const u32x4* L = lds[buf];
    bf16x8 af[2][TM], wf[2][TN];
    // Fragments are read in the order the next k step's MFMAs (i-major)
    // consume them, so the first MFMAs wait on the oldest reads.
    auto read = [&](int kk, int slot) {
      const int chunk = 2 * kk + hi;
      wf[slot][0] = as_bf16x8(L[kBM * 8 + swz(wn * WN + l32, chunk)]);
      af[slot][0] = as_bf16x8(L[swz(wm * WM + l32, chunk)]);
#pragma unroll
      for (int j = 1; j < TN; ++j) wf[slot][j] = as_bf16x8(L[kBM * 8 + swz(wn * WN + 32 * j + l32, chunk)]);
#pragma unroll
      for (int i = 1; i < TM; ++i) af[slot][i] = as_bf16x8(L[swz(wm * WM + 32 * i + l32, chunk)]);
    };
    read(0, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, TM + TN, 0);
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      if (kk + 1 < kBK / 16) read(kk + 1, (kk + 1) & 1);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32x32x16(wf[kk & 1][j], af[kk & 1][i], acc[i][j]);
      if (kk + 1 < kBK / 16) {
#pragma unroll
        for (int r = 0; r < TM + TN; ++r) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, TM * TN - (TM + TN), 0);
      } else {
        __builtin_amdgcn_sched_group_barrier(0x008, TM * TN, 0);
      }
    }
  };

  if (n_t > 0) {
    load_half(kt0);
    store_half(0);
    if (n_t > 1) load_half(kt0 + 1);
  }
  lds_barrier();
  // Memory phase of k-tile t: stage this group's half of tile t + 1, then
  // issue its loads of tile t + 2.
  auto memory = [&](int64_t t) {
    if (t + 1 < n_t) {
      store_half(int((t + 1) & 1));
      if (t + 2 < n_t) load_half(kt0 + t + 2);
    }
  };
  // Each group runs its own straight loop; both pass the same barriers.
  if (grp == 0) {
    for (int64_t t = 0; t < n_t; ++t) {
      compute(int(t & 1));
      lds_barrier();
      memory(t);
      lds_barrier();
    }
  } else {
    for (int64_t t = 0; t < n_t; ++t) {
      memory(t);
      lds_barrier();
      compute(int(t & 1));
      lds_barrier();
    }
  }

  // Split partials: a tail tile's go to its own 256 x 256 block (split-major),
  // a fully split launch's to rows of the [split][row][N] array.
  float* pbase = nullptr;
  int64_t pld = a.N;
  if (tidx >= 0) {
    pbase = partial + (tidx * tsp + ks) * int64_t(kBM * BN);
    pld = BN;
  } else if (splits > 1) {
    const int64_t rows_all = a.p[0].M + (a.nprob > 1 ? a.p[1].M : 0);
    pbase = partial + (int64_t(ks) * rows_all + (prob ? a.p[0].M : 0) + m0) * a.N + n0;
  }
  staged_epilogue<WM, WN, TM, TN>(a, p, m0, n0, pbase != nullptr, pbase, pld, acc,
                                  reinterpret_cast<float*>(&lds[0][0]), wave, wm, wn, lane);
}

// Sum the k splits of each tail tile in split order and apply the epilogue.
// Block b covers rows 8 (b mod 32) .. + 7 of tail tile b / 32, one thread per
// eight columns.
__global__ __launch_bounds__(256) void tail_reduce_kernel(const GemmArgs a, const float* __restrict__ partial,
                                                          int64_t tail, int tsp) {
  constexpr int BN = 256;
  const int64_t t = blockIdx.x / (kBM / 8);
  const int r = int(blockIdx.x % (kBM / 8)) * 8 + int(threadIdx.x) / 32;
  const int c = (int(threadIdx.x) % 32) * 8;
  int prob;
  int64_t m0, n0;
  if (!decode_tile(a, kBM, BN, tiles_total(a, kBM, BN) - tail + t, prob, m0, n0)) return;
  const GemmProblem p = prob ? a.p[1] : a.p[0];
  const int64_t m = m0 + r, n = n0 + c;
  if (m >= p.M || n >= a.N) return;
  const float* src = partial + t * tsp * int64_t(kBM * BN) + r * BN + c;
  float v[8];
  {
    const float4 x0 = *reinterpret_cast<const float4*>(src), x1 = *reinterpret_cast<const float4*>(src + 4);
    v[0] = x0.x; v[1] = x0.y; v[2] = x0.z; v[3] = x0.w; v[4] = x1.x; v[5] = x1.y; v[6] = x1.z; v[7] = x1.w;
  }
  for (int k = 1; k < tsp; ++k) {
    const float* q = src + int64_t(k) * kBM * BN;
    const float4 x0 = *reinterpret_cast<const float4*>(q), x1 = *reinterpret_cast<const float4*>(q + 4);
    v[0] += x0.x; v[1] += x0.y; v[2] += x0.z; v[3] += x0.w; v[4] += x1.x; v[5] += x1.y; v[6] += x1.z; v[7] += x1.w;
  }
  epilogue8(a, p, m, n, v);
}

// Sum the split-K partials in split order and apply the epilogue: one thread
// per eight columns of a row.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const GemmArgs a, const float* __restrict__ partial,
                                                            int splits) {
  const int64_t rows = a.p[0].M + (a.nprob > 1 ? a.p[1].M : 0);
  const int64_t groups = a.N / 8;
  const int64_t g = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (g >= rows * groups) return;
  const int64_t grow = g / groups, n = (g % groups) * 8;
  const float* src = partial + grow * a.N + n;
  float v[8];
  {
    const float4 x0 = *reinterpret_cast<const float4*>(src), x1 = *reinterpret_cast<const float4*>(src + 4);
    v[0] = x0.x; v[1] = x0.y; v[2] = x0.z; v[3] = x0.w; v[4] = x1.x; v[5] = x1.y; v[6] = x1.z; v[7] = x1.w;
  }
  for (int k = 1; k < splits; ++k) {
    const float* q = src + int64_t(k) * rows * a.N;
    const float4 x0 = *reinterpret_cast<const float4*>(q), x1 = *reinterpret_cast<const float4*>(q + 4);
    v[0] += x0.x; v[1] += x0.y; v[2] += x0.z; v[3] += x0.w; v[4] += x1.x; v[5] += x1.y; v[6] += x1.z; v[7] += x1.w;
  }
  const bool second = grow >= a.p[0].M;
  GemmProblem p = second ? a.p[1] : a.p[0];
  const int64_t m = second ? grow - a.p[0].M : grow;
  if (a.mod.B) p.gate = static_cast<const bf16_t*>(p.gate) + mod_offset(a.mod, p.row0 + m);  // this row's image
  epilogue8(a, p, m, n, v);
}

// fp32 VALU GEMM: 64x64 tile, 16x16 threads, 4x4 outputs per thread.
constexpr int kFB = 64, kFK = 16;
__global__ __launch_bounds__(256) void gemm_f32_kernel(const GemmArgs a) {
  __shared__ float As[kFK][kFB + 4];
  __shared__ float Ws[kFK][kFB + 4];
  int prob, ks;
  int64_t m0, n0;
  if (!map_tile(a, kFB, kFB, 1, prob, m0, n0, ks)) return;
  const GemmProblem p = prob ? a.p[1] : a.p[0];  // by value: a select, no indexed copy of the arguments
  const float* A = static_cast<const float*>(p.A);
  const float* W = static_cast<const float*>(p.W);
  const int tid = threadIdx.x, tx = tid % 16, ty = tid / 16;
  const int lrow = tid / 4, lk = (tid % 4) * 4;
  float acc[4][4] = {};
  for (int64_t k0 = 0; k0 < a.K; k0 += kFK) {
    const int64_t m = m0 + lrow, n = n0 + lrow;
    float4 va = make_float4(0.f, 0.f, 0.f, 0.f), vw = va;
    if (m < p.M) va = *reinterpret_cast<const float4*>(A + m * p.lda + k0 + lk);
    if (n < a.N) vw = *reinterpret_cast<const float4*>(W + n * a.K + k0 + lk);
    __syncthreads();
    As[lk + 0][lrow] = va.x; As[lk + 1][lrow] = va.y; As[lk + 2][lrow] = va.z; As[lk + 3][lrow] = va.w;
    Ws[lk + 0][lrow] = vw.x; Ws[lk + 1][lrow] = vw.y; Ws[lk + 2][lrow] = vw.z; Ws[lk + 3][lrow] = vw.w;
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kFK; ++kk) {
      float av[4], wv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) wv[j] = Ws[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], wv[j], acc[i][j]);
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = m0 + ty * 4 + i, n = n0 + tx * 4;
    if (m < p.M && n < a.N) epilogue4<float>(a, p, m, n, acc[i][0], acc[i][1], acc[i][2], acc[i][3]);
  }
}

int64_t tiles_of(const GemmArgs& a, int bm, int bn) {
  int64_t t = 0;
  for (int i = 0; i < a.nprob; ++i) t += ceil_div64(a.p[i].M, bm) * ceil_div64(a.N, bn);
  return t;
}

}  // namespace

GemmPlan plan_gemm(const GemmArgs& a, int dtype, size_t partial_bytes, const char* family) {
  GemmPlan pl;
  if (dtype != AVITS_BF16) {
    pl.bn = kFB;
    pl.tiles = tiles_of(a, kFB, kFB);
    return pl;
  }
  // Score every (column tile, K split) pair: busy fraction of the last wave
  // of work units on the 256 CUs, times a per-tile factor (the 256-wide tile
  // runs the ping-pong kernel and moves less L2 data per FLOP; the factors
  // are measured on MI355X at the FLUX block shapes), times a factor for the
  // extra fp32 partial traffic of a split.
  const int cands[3] = {256, 192, 128};
  const double eff[3] = {1.0, 0.74, 0.65};
  const int64_t nk = a.K / kBK;
  const int64_t rows = a.p[0].M + (a.nprob > 1 ? a.p[1].M : 0);
  double best = -1.0;
  for (int c = 0; c < 3; ++c) {
    const int64_t t = tiles_of(a, kBM, cands[c]);
    if (t == 0) continue;
    for (int sp = 1; sp <= 4; ++sp) {
      if (sp > 1 && (nk / sp < 4 || size_t(sp) * size_t(rows) * size_t(a.N) * sizeof(float) > partial_bytes)) break;
      const int64_t units = t * sp;
      const double fill = double(units) / double(ceil_div64(units, kCUs) * kCUs);
      const double score = fill * eff[c] * (sp > 1 ? 0.95 : 1.0);
      if (score > best + 1e-9) {
        best = score;
        pl.bn = cands[c];
        pl.tiles = t;
        pl.splits = sp;
        pl.tail = 0;
        pl.tail_splits = 1;
      }
    }
    // The 256-wide tile may instead split only the tiles that overrun the
    // last full wave (the tail): the partial wave then takes 1 / tsp of a
    // tile's time.
    const int64_t full = t / kCUs, rem = t % kCUs;
    if (cands[c] != 256 || full == 0 || rem == 0) continue;
    for (int tsp = 2; tsp <= 4; ++tsp) {
      if (rem * tsp > kCUs || nk / tsp < 4 || size_t(rem * tsp) * kBM * 256 * sizeof(float) > partial_bytes) break;
      const double fill = double(t) / double(kCUs) / (double(full) + 1.0 / tsp);
      const double score = fill * eff[c] * 0.95;
      if (score > best + 1e-9) {
        best = score;
        pl.bn = 256;
        pl.tiles = t;
        pl.splits = 1;
        pl.tail = rem;
        pl.tail_splits = tsp;
      }
    }
  }
  pl.waves = 8;
  // Two register stages fit the registers of the 128-wide tile only.  The staged
  // loads are asynchronous inline assembly, so an instance that spilled a
  // destination register would read it before the load lands: every
  // instance must build without scratch (the build checks it).
  pl.stages = pl.bn == 128 ? 2 : 1;
  // Tuning override "BN,SPLITS[,8[,STAGES[,TAIL,TSP]]]" (e.g. AVITS_GEMM_TILE=256,3,8,1),
  // for one launch family with AVITS_GEMM_TILE_<family> (e.g. _gemm_o).  TAIL > 0
  // (256-wide tile, SPLITS 1) runs the last min(TAIL, tiles) tiles in TSP k splits.
  const char* env = nullptr;
  if (family) {
    char name[64];
    snprintf(name, sizeof(name), "AVITS_GEMM_TILE_%s", family);
    env = getenv(name);
  }
  if (!env) env = getenv("AVITS_GEMM_TILE");
  if (env) {
    int bn = 0, sp = 0, wv = 8, stg = 2, tail = 0, tsp = 1;
    const int got = sscanf(env, "%d,%d,%d,%d,%d,%d", &bn, &sp, &wv, &stg, &tail, &tsp);
    if (got >= 2 && (bn == 256 || bn == 192 || bn == 128) && sp >= 1 && sp <= 4 && wv == 8 &&
        (stg == 1 || stg == 2)) {
      pl.bn = bn;
      pl.splits = sp;
      pl.waves = wv;
      pl.stages = bn == 128 ? stg : 1;  // the wider tiles have one register stage only
      pl.tiles = tiles_of(a, kBM, bn);
      pl.tail = 0;
      pl.tail_splits = 1;
      if (got == 6 && bn == 256 && sp == 1 && tail > 0 && tsp >= 2 && tsp <= 4 && nk / tsp >= 1) {
        pl.tail = std::min<int64_t>(tail, pl.tiles);
        pl.tail_splits = tsp;
      }
    }
  }
  return pl;
}

size_t gemm_partial_bytes(const GemmArgs& a, const GemmPlan& pl) {
  if (pl.tail > 0) return size_t(pl.tail) * size_t(pl.tail_splits) * kBM * size_t(pl.bn) * sizeof(float);
  if (pl.splits <= 1) return 0;
  const int64_t rows = a.p[0].M + (a.nprob > 1 ? a.p[1].M : 0);
  return size_t(pl.splits) * size_t(rows) * size_t(a.N) * sizeof(float);
}

int launch_gemm(const GemmArgs& a, int dtype, hipStream_t s, const char* family, float* partial,
                size_t partial_bytes, GemmPostLN* post_ln) {
  GemmPlan pl = plan_gemm(a, dtype, partial ? partial_bytes : 0, family);
  if (pl.tiles == 0) return AVITS_OK;
  // Per-image gates are applied by the split-K reduce (the GEMM's own
  // epilogue has one gate per launch): such a projection always runs split.
  const bool per_image_gate = a.mod.B > 0 && a.mode0 == EPI_RESID_GATE;
  if (per_image_gate && (pl.splits < 2 || pl.tail > 0)) {
    pl.splits = 2;
    pl.tail = 0;
    pl.tail_splits = 1;
  }
  // The reduce kernels take eight columns per thread.
  if ((pl.splits > 1 || pl.tail > 0) && (!partial || partial_bytes < gemm_partial_bytes(a, pl) || a.N % 8 != 0)) {
    if (per_image_gate)
      return set_error(AVITS_ERR_UNSUPPORTED, "gemm %s: per-image gates need a split-K scratch of %zu bytes and N %% 8 == 0",
                       family ? family : "", gemm_partial_bytes(a, pl));
    pl.splits = 1;
    pl.tail = 0;
  }
  if (per_image_gate && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "gemm %s: per-image gates need bf16", family ? family : "");
  if (dtype == AVITS_BF16) {
    const dim3 grid(unsigned(pl.tiles * pl.splits + pl.tail * (pl.tail_splits - 1)));
    {
    TimedLaunch timed(family, s);  // the GEMM kernel alone; the reduce is its own family
    switch (pl.bn * 100 + pl.waves * 10 + pl.stages) {
      case 25681:
        hipLaunchKernelGGL(gemm_bf16_pp_kernel, grid, dim3(512), 0, s, a, partial, pl.splits, pl.tail,
                           pl.tail_splits);
        break;
      case 19281: hipLaunchKernelGGL((gemm_bf16_kernel<192, 4, 2, 1>), grid, dim3(512), 0, s, a, partial, pl.splits); break;
      case 12881: hipLaunchKernelGGL((gemm_bf16_kernel<128, 2, 4, 1>), grid, dim3(512), 0, s, a, partial, pl.splits); break;
      default: hipLaunchKernelGGL((gemm_bf16_kernel<128, 2, 4, 2>), grid, dim3(512), 0, s, a, partial, pl.splits); break;
    }
    }
    if (post_ln) post_ln->done = false;
    if (pl.tail > 0) {
      TimedLaunch timed_reduce("splitk_reduce", s);
      hipLaunchKernelGGL(tail_reduce_kernel, dim3(unsigned(pl.tail * (kBM / 8))), dim3(256), 0, s, a,
                         (const float*)partial, pl.tail, pl.tail_splits);
    }
    const int64_t rows_all = a.p[0].M + (a.nprob > 1 ? a.p[1].M : 0);
    if (pl.splits > 1 && post_ln && a.mode0 == EPI_RESID_GATE && a.n_split >= a.N && a.N % 8 == 0 &&
        a.N <= int64_t(kWave) * 8 * kRlnChunks) {
      TimedLaunch timed_reduce("splitk_reduce", s);
      const dim3 rgrid(unsigned(ceil_div64(rows_all, 4)));
      if (pl.splits == 2) hipLaunchKernelGGL(splitk_reduce_ln_kernel<2>, rgrid, dim3(256), 0, s, a, partial, *post_ln);
      else if (pl.splits == 3) hipLaunchKernelGGL(splitk_reduce_ln_kernel<3>, rgrid, dim3(256), 0, s, a, partial, *post_ln);
      else hipLaunchKernelGGL(splitk_reduce_ln_kernel<4>, rgrid, dim3(256), 0, s, a, partial, *post_ln);
      post_ln->done = true;
    } else if (pl.splits > 1) {
      TimedLaunch timed_reduce("splitk_reduce", s);
      const int64_t rows = rows_all;
      const int64_t work = rows * (a.N / 8);
      hipLaunchKernelGGL(splitk_reduce_kernel, dim3(unsigned(ceil_div64(work, 256))), dim3(256), 0, s, a,
                         (const float*)partial, pl.splits);
    }
  } else {
    TimedLaunch timed(family, s);
    hipLaunchKernelGGL(gemm_f32_kernel, dim3(unsigned(pl.tiles)), dim3(256), 0, s, a);
  }
  return launch_status("gemm");
}

}  // namespace avits
