// The modulated layer norm of one bf16 row held by a wavefront in registers
// (h = LN(x)(1 + scale) + shift: layer norm without affine, eps 1e-6,
// biased variance), shared by the block's LN kernel and the gather that
// produces the block's input rows, so both give the same bits.
#pragma once

#include "common.h"

namespace avits {
namespace {

constexpr float kLnEps = 1e-6f;
constexpr int kLnMaxChunks = 8;  // bf16 rows up to 64 * 8 * 8 = 4096 elements in registers

// Lane l holds the row's 16-byte chunks l + 64 c (eight elements each) in
// v[c] for l + 64 c < nchunk = D / 8.  The sums run over the lane's chunks
// in order and then across the wave.  PRELOAD issues every scale and shift
// load before the reductions (a kernel that does nothing else); without it
// each chunk's scale and shift are loaded where they are used, which keeps
// the register count of a kernel that also does other work low.  Same
// arithmetic either way.
template <bool PRELOAD>
__device__ __forceinline__ void ln_mod_row_bf16(const u32x4 (&v)[kLnMaxChunks], int64_t nchunk, int64_t D,
                                                int lane, const bf16_t* __restrict__ sh,
                                                const bf16_t* __restrict__ sc, bf16_t* __restrict__ hr) {
  u32x4 g[kLnMaxChunks], t[kLnMaxChunks];
  if constexpr (PRELOAD) {
#pragma unroll
    for (int c = 0; c < kLnMaxChunks; ++c) {
      const int64_t idx = lane + kWave * c;
      if (idx < nchunk) {
        g[c] = reinterpret_cast<const u32x4*>(sc)[idx];
        t[c] = reinterpret_cast<const u32x4*>(sh)[idx];
      }
    }
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kLnMaxChunks; ++c) {
    if (lane + kWave * c < nchunk) {
#pragma unroll
      for (int e = 0; e < 4; ++e) s += __uint_as_float(v[c][e] << 16) + __uint_as_float(v[c][e] & 0xffff0000u);
    }
  }
  const float mean = wave_sum(s) / float(D);
  float q = 0.f;
#pragma unroll
  for (int c = 0; c < kLnMaxChunks; ++c) {
    if (lane + kWave * c < nchunk) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a = __uint_as_float(v[c][e] << 16) - mean, b = __uint_as_float(v[c][e] & 0xffff0000u) - mean;
        q = fmaf(a, a, fmaf(b, b, q));
      }
    }
  }
  const float rstd = rsqrtf(wave_sum(q) / float(D) + kLnEps);
  float mean_out = mean;
  if constexpr (!PRELOAD) {
    // The same value through an empty asm: the output loop recomputes
    // x - mean instead of keeping 64 differences live across the reduction.
    asm volatile("" : "+v"(mean_out));
  }
#pragma unroll
  for (int c = 0; c < kLnMaxChunks; ++c) {
    const int64_t idx = lane + kWave * c;
    if (idx < nchunk) {
      if constexpr (!PRELOAD) {
        g[c] = reinterpret_cast<const u32x4*>(sc)[idx];
        t[c] = reinterpret_cast<const u32x4*>(sh)[idx];
      }
      u32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a = (__uint_as_float(v[c][e] << 16) - mean_out) * rstd * (1.f + __uint_as_float(g[c][e] << 16)) +
                        __uint_as_float(t[c][e] << 16);
        const float b = (__uint_as_float(v[c][e] & 0xffff0000u) - mean_out) * rstd *
                            (1.f + __uint_as_float(g[c][e] & 0xffff0000u)) +
                        __uint_as_float(t[c][e] & 0xffff0000u);
        o[e] = pack_bf2(a, b);
      }
      reinterpret_cast<u32x4*>(hr)[idx] = o;
    }
  }
}

}  // namespace
}  // namespace avits
