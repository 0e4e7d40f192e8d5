// GEMMs of the MMDiT block (QKV, output projection, MLP), with the bias,
// GELU and gated-residual epilogues fused.
//
// bf16: 128x128 output tile per 256-thread workgroup, k-tiles of 64 staged
// through padded LDS rows (conflict-free 16-byte fragment reads), each wave a
// 64x64 quadrant of 4x4 v_mfma_f32_16x16x32_bf16 tiles.  The MFMA computes
// C^T = W A^T so that each lane ends up owning four consecutive output
// columns of one row: the epilogue stores 8 contiguous bytes per lane.
// fp32: 64x64 tiles on the VALU (the fp32 path exists for exactness checks).
#include "kernels.h"

namespace avits {
namespace {

constexpr int kBM = 128, kBN = 128, kBK = 64;
constexpr int kLdsRow = kBK + 8;  // padded row, bf16 elements

__device__ __forceinline__ float gelu_tanh(float x) {
  const float u = 0.7978845608028654f * (x + 0.044715f * x * x * x);
  return 0.5f * x * (1.f + tanhf(u));
}

// Epilogue for four consecutive columns n..n+3 of row m (n % 4 == 0, n < N).
template <typename T>
__device__ __forceinline__ void epilogue4(const GemmArgs& a, const GemmProblem& p, int64_t m, int64_t n,
                                          float v0, float v1, float v2, float v3) {
  float v[4] = {v0, v1, v2, v3};
  if (p.bias) {
    const T* b = static_cast<const T*>(p.bias);
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] += ld(b, n + r);
  }
  const bool first = n < a.n_split;
  const int mode = first ? a.mode0 : a.mode1;
  T* out = static_cast<T*>(first ? p.out0 : p.out1);
  const int64_t col = first ? n : n - a.n_split;
  const int64_t ldo = first ? p.ld0 : p.ld1;
  if (mode == EPI_GELU) {
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = gelu_tanh(v[r]);
  } else if (mode == EPI_RESID_GATE) {
    const T* res = static_cast<const T*>(p.resid);
    const T* gt = static_cast<const T*>(p.gate);
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = ld(res, m * p.ldr + col + r) + ld(gt, n + r) * v[r];
  }
  T* dst = out + m * ldo + col;
  if constexpr (sizeof(T) == 2) {
    u32x2 w = {pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3])};
    *reinterpret_cast<u32x2*>(dst) = w;
  } else {
    *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
  }
}

// Map the flat workgroup id onto (problem, tile row, tile col).
__device__ __forceinline__ bool map_tile(const GemmArgs& a, int bm, int bn, int& prob, int64_t& m0, int64_t& n0) {
  const int64_t tn = (a.N + bn - 1) / bn;
  int64_t bid = blockIdx.x;
  const int64_t t0 = ((a.p[0].M + bm - 1) / bm) * tn;
  prob = 0;
  if (bid >= t0) {
    bid -= t0;
    prob = 1;
    if (a.nprob < 2) return false;
  }
  m0 = (bid / tn) * bm;
  n0 = (bid % tn) * bn;
  return m0 < a.p[prob].M;
}

__global__ __launch_bounds__(256) void gemm_bf16_kernel(const GemmArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t As[kBM * kLdsRow];
  __shared__ __attribute__((aligned(16))) bf16_t Ws[kBN * kLdsRow];
  int prob;
  int64_t m0, n0;
  if (!map_tile(a, kBM, kBN, prob, m0, n0)) return;
  const GemmProblem& p = a.p[prob];
  const bf16_t* A = static_cast<const bf16_t*>(p.A);
  const bf16_t* W = static_cast<const bf16_t*>(p.W);
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int g = lane / 16, r16 = lane % 16;
  const int wm = wave / 2, wn = wave % 2;

  // Global -> register staging: 4 16-byte pieces of each operand per thread.
  u32x4 ra[4], rw[4];
  auto load_tile = [&](int64_t k0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int piece = tid + 256 * j;
      const int row = piece / 8, kc = (piece % 8) * 8;
      const int64_t m = m0 + row, n = n0 + row;
      u32x4 z = {0u, 0u, 0u, 0u};
      ra[j] = m < p.M ? *reinterpret_cast<const u32x4*>(A + m * p.lda + k0 + kc) : z;
      rw[j] = n < a.N ? *reinterpret_cast<const u32x4*>(W + n * a.K + k0 + kc) : z;
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int piece = tid + 256 * j;
      const int row = piece / 8, kc = (piece % 8) * 8;
      *reinterpret_cast<u32x4*>(&As[row * kLdsRow + kc]) = ra[j];
      *reinterpret_cast<u32x4*>(&Ws[row * kLdsRow + kc]) = rw[j];
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  load_tile(0);
  store_tile();
  __syncthreads();
  for (int64_t k0 = 0; k0 < a.K; k0 += kBK) {
    const bool more = k0 + kBK < a.K;
    if (more) load_tile(k0 + kBK);
#pragma unroll
    for (int c = 0; c < kBK / 32; ++c) {
      bf16x8 af[4], wf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = as_bf16x8(*reinterpret_cast<const u32x4*>(&As[(wm * 64 + 16 * i + r16) * kLdsRow + 32 * c + 8 * g]));
#pragma unroll
      for (int j = 0; j < 4; ++j)
        wf[j] = as_bf16x8(*reinterpret_cast<const u32x4*>(&Ws[(wn * 64 + 16 * j + r16) * kLdsRow + 32 * c + 8 * g]));
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma16x16x32(wf[j], af[i], acc[i][j]);
    }
    __syncthreads();
    if (more) {
      store_tile();
      __syncthreads();
    }
  }
  // acc[i][j][r] = C[m0 + wm*64 + 16i + r16][n0 + wn*64 + 16j + 4g + r].
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = m0 + wm * 64 + 16 * i + r16;
    if (m >= p.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t n = n0 + wn * 64 + 16 * j + 4 * g;
      if (n < a.N) epilogue4<bf16_t>(a, p, m, n, acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
    }
  }
}

// fp32 VALU GEMM: 64x64 tile, 16x16 threads, 4x4 outputs per thread.
constexpr int kFB = 64, kFK = 16;
__global__ __launch_bounds__(256) void gemm_f32_kernel(const GemmArgs a) {
  __shared__ float As[kFK][kFB + 4];
  __shared__ float Ws[kFK][kFB + 4];
  int prob;
  int64_t m0, n0;
  if (!map_tile(a, kFB, kFB, prob, m0, n0)) return;
  const GemmProblem& p = a.p[prob];
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

}  // namespace

int launch_gemm(const GemmArgs& a, int dtype, hipStream_t s) {
  const int bm = dtype == AVITS_BF16 ? kBM : kFB, bn = bm;
  const int64_t tn = ceil_div64(a.N, bn);
  int64_t tiles = 0;
  for (int i = 0; i < a.nprob; ++i) tiles += ceil_div64(a.p[i].M, bm) * tn;
  if (tiles == 0) return AVITS_OK;
  TimedLaunch timed("gemm", s);
  if (dtype == AVITS_BF16)
    hipLaunchKernelGGL(gemm_bf16_kernel, dim3(unsigned(tiles)), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(gemm_f32_kernel, dim3(unsigned(tiles)), dim3(256), 0, s, a);
  return launch_status("gemm");
}

}  // namespace avits
