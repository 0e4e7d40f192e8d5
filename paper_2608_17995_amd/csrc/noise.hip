// Coordinate-bound noise re-injection (Section 3.2: into the mixed-resolution
// sequence when Stage 2 starts and into the full grid when Stage 3 starts).
//
// The noise is one fixed standard-normal field over the high-resolution
// grid: eps(p, c) at raster pixel p and latent channel c.  A low-resolution
// token (a 2x2 block of pixels) takes the sum of its four children's noise
// halved (unit variance, consistent with the children).  eps comes from the
// counter-based generator Philox-4x32-10 (Salmon, Moraes, Dror and Shaw,
// SC 2011): counter (p, c / 4, 0, 0), key (seed low word, seed high word);
// the four output words are turned into four normals by the Box-Muller
// transform of uniform pairs u = (w >> 8 + 1/2) 2^-24.  Any row's noise is
// produced on its own, so the same pixel receives the same noise in every
// stage and in any row order.
//
// One thread per (row, 4 channels): the row's coordinate (a pixel or a
// block) from its index (raster rows) or its position (half units, as the
// mixed sequence carries them), one Philox call per pixel, and the mix
// x <- (1 - t) x + t eps in fp32 with one rounding to the storage type.
#include "common.h"

namespace avits {
namespace {

constexpr uint32_t kPhiloxM0 = 0xD2511F53u, kPhiloxM1 = 0xCD9E8D57u;
constexpr uint32_t kPhiloxW0 = 0x9E3779B9u, kPhiloxW1 = 0xBB67AE85u;

__device__ __forceinline__ u32x4 philox4x32_10(u32x4 x, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += kPhiloxW0;
      k1 += kPhiloxW1;
    }
    const uint32_t hi0 = __umulhi(kPhiloxM0, x[0]), lo0 = kPhiloxM0 * x[0];
    const uint32_t hi1 = __umulhi(kPhiloxM1, x[2]), lo1 = kPhiloxM1 * x[2];
    x = u32x4{hi1 ^ x[1] ^ k0, lo1, hi0 ^ x[3] ^ k1, lo0};
  }
  return x;
}

__device__ __forceinline__ float uniform24(uint32_t w) {
  return (float(w >> 8) + 0.5f) * 5.9604644775390625e-08f;  // 2^-24; exact in fp32
}

// Four standard normals of pixel p, channels 4j .. 4j + 3.
__device__ __forceinline__ float4 pixel_normals(int64_t p, uint32_t j, uint32_t k0, uint32_t k1) {
  const u32x4 w = philox4x32_10(u32x4{uint32_t(p), j, 0u, 0u}, k0, k1);
  float4 z;
  {
    const float r = sqrtf(-2.f * logf(uniform24(w[0])));
    float s, c;
    sincosf(6.283185307179586f * uniform24(w[1]), &s, &c);
    z.x = r * c;
    z.y = r * s;
  }
  {
    const float r = sqrtf(-2.f * logf(uniform24(w[2])));
    float s, c;
    sincosf(6.283185307179586f * uniform24(w[3]), &s, &c);
    z.z = r * c;
    z.w = r * s;
  }
  return z;
}

enum { kRowsRaster = 0, kRowsHalfUnits = 1, kRowsLowRes = 2 };

template <typename T>
__global__ __launch_bounds__(256) void noise_reinject_kernel(T* __restrict__ x, int64_t rows, int64_t C,
                                                             const int32_t* __restrict__ pos, int kind, int W_hr,
                                                             float t, uint32_t k0, uint32_t k1) {
  const int64_t g = int64_t(blockIdx.x) * 256 + threadIdx.x;
  const int64_t groups = C / 4;
  if (g >= rows * groups) return;
  const int64_t r = g / groups;
  const uint32_t j = uint32_t(g % groups);
  // The row's pixel (block = false) or the top-left pixel of its 2x2 block.
  int64_t y, xx;
  bool block;
  if (kind == kRowsRaster) {
    y = r / W_hr;
    xx = r % W_hr;
    block = false;
  } else if (kind == kRowsLowRes) {
    const int W_lr = W_hr / 2;
    y = 2 * (r / W_lr);
    xx = 2 * (r % W_lr);
    block = true;
  } else {
    const int Y = pos[3 * r + 1], X = pos[3 * r + 2];
    block = (Y & 1) != 0;  // odd half-unit coordinates: a block centre (4 r + 1, 4 c + 1)
    y = block ? (Y - 1) / 2 : Y / 2;
    xx = block ? (X - 1) / 2 : X / 2;
  }
  float4 e;
  if (block) {
    const float4 a = pixel_normals(y * W_hr + xx, j, k0, k1);
    const float4 b = pixel_normals(y * W_hr + xx + 1, j, k0, k1);
    const float4 c = pixel_normals((y + 1) * W_hr + xx, j, k0, k1);
    const float4 d = pixel_normals((y + 1) * W_hr + xx + 1, j, k0, k1);
    e = make_float4(0.5f * (a.x + b.x + c.x + d.x), 0.5f * (a.y + b.y + c.y + d.y),
                    0.5f * (a.z + b.z + c.z + d.z), 0.5f * (a.w + b.w + c.w + d.w));
  } else {
    e = pixel_normals(y * W_hr + xx, j, k0, k1);
  }
  T* row = x + r * C + 4 * int64_t(j);
  const float ev[4] = {e.x, e.y, e.z, e.w};
  if (t == 1.f) {  // pure noise: x is not read
#pragma unroll
    for (int q = 0; q < 4; ++q) st(row, q, ev[q]);
  } else {
    const float keep = 1.f - t;
#pragma unroll
    for (int q = 0; q < 4; ++q) st(row, q, fmaf(t, ev[q], keep * ld(row, q)));
  }
}

__global__ __launch_bounds__(256) void noise_bits_kernel(int64_t first, int64_t n, int64_t C, uint32_t k0,
                                                         uint32_t k1, uint32_t* __restrict__ out) {
  const int64_t g = int64_t(blockIdx.x) * 256 + threadIdx.x;
  const int64_t groups = C / 4;
  if (g >= n * groups) return;
  const int64_t p = first + g / groups;
  const uint32_t j = uint32_t(g % groups);
  const u32x4 w = philox4x32_10(u32x4{uint32_t(p), j, 0u, 0u}, k0, k1);
  *reinterpret_cast<u32x4*>(out + g * 4) = w;
}

}  // namespace
}  // namespace avits

using namespace avits;

extern "C" int avits_noise_reinject(void* x, int64_t rows, int64_t C, const int32_t* pos, int32_t rows_kind,
                                    int32_t H_hr, int32_t W_hr, float t, uint64_t seed, int dtype, void* stream) {
  AVITS_REQUIRE(rows >= 0 && C >= 4 && C % 4 == 0, "noise_reinject: rows=%lld C=%lld (C a positive multiple of 4)",
                (long long)rows, (long long)C);
  AVITS_REQUIRE(H_hr >= 2 && W_hr >= 2 && H_hr % 2 == 0 && W_hr % 2 == 0,
                "noise_reinject: grid %d x %d must be even and at least 2 x 2", H_hr, W_hr);
  AVITS_REQUIRE(int64_t(H_hr) * W_hr <= (int64_t(1) << 32), "noise_reinject: grid of %lld pixels beyond 2^32",
                (long long)(int64_t(H_hr) * W_hr));
  AVITS_REQUIRE(t >= 0.f && t <= 1.f, "noise_reinject: t=%g outside [0, 1]", t);
  AVITS_REQUIRE(rows_kind == kRowsRaster || rows_kind == kRowsHalfUnits || rows_kind == kRowsLowRes,
                "noise_reinject: rows_kind %d unknown", rows_kind);
  const int64_t grid_rows = rows_kind == kRowsLowRes ? int64_t(H_hr / 2) * (W_hr / 2) : int64_t(H_hr) * W_hr;
  AVITS_REQUIRE(rows_kind == kRowsHalfUnits || rows <= grid_rows,
                "noise_reinject: %lld rows beyond the %lld of the grid", (long long)rows, (long long)grid_rows);
  AVITS_REQUIRE(rows_kind != kRowsHalfUnits || pos || rows == 0, "noise_reinject: positions required");
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "noise_reinject: dtype %d unsupported", dtype);
  if (rows == 0) return AVITS_OK;
  AVITS_REQUIRE(x, "noise_reinject: null x");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t threads = rows * (C / 4);
  const dim3 grid(unsigned((threads + 255) / 256));
  const uint32_t k0 = uint32_t(seed), k1 = uint32_t(seed >> 32);
  TimedLaunch timed("noise", s);
  if (dtype == AVITS_F32)
    hipLaunchKernelGGL(noise_reinject_kernel<float>, grid, dim3(256), 0, s, static_cast<float*>(x), rows, C, pos,
                       rows_kind, W_hr, t, k0, k1);
  else
    hipLaunchKernelGGL(noise_reinject_kernel<bf16_t>, grid, dim3(256), 0, s, static_cast<bf16_t*>(x), rows, C, pos,
                       rows_kind, W_hr, t, k0, k1);
  return launch_status("noise_reinject");
}

extern "C" int avits_noise_bits(int64_t first_pixel, int64_t n_pixels, int64_t C, uint64_t seed, uint32_t* bits,
                                void* stream) {
  AVITS_REQUIRE(first_pixel >= 0 && n_pixels >= 0 && first_pixel + n_pixels <= (int64_t(1) << 32),
                "noise_bits: pixels [%lld, %lld) outside [0, 2^32)", (long long)first_pixel,
                (long long)(first_pixel + n_pixels));
  AVITS_REQUIRE(C >= 4 && C % 4 == 0, "noise_bits: C=%lld must be a positive multiple of 4", (long long)C);
  if (n_pixels == 0) return AVITS_OK;
  AVITS_REQUIRE(bits, "noise_bits: null bits");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t threads = n_pixels * (C / 4);
  TimedLaunch timed("noise", s);
  hipLaunchKernelGGL(noise_bits_kernel, dim3(unsigned((threads + 255) / 256)), dim3(256), 0, s, first_pixel,
                     n_pixels, C, uint32_t(seed), uint32_t(seed >> 32), bits);
  return launch_status("noise_bits");
}
