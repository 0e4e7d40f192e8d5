// The modulated layer norm of one bf16 row held by a wavefront in registers
// (h = LN(x)(1 + scale) + shift: layer norm without affine, eps 1e-6,
// biased variance), shared by the block's LN kernel and the gather that
// produces the block's input rows, so both give the same bits.
#pragma once

#include <algorithm>

#include "common.h"

namespace avits {
namespace {

constexpr float kLnEps = 1e-6f;
constexpr int kLnMaxChunks = 8;  // bf16 rows up to 64 * 8 * 8 = 4096 elements in registers

// Lane l holds the row's 16-byte chunks l + 64 c (eight elements each) in
// v[c] for l + 64 c < nchunk = D / 8, and the same chunks of the scale and
// shift vectors in g[c] and t[c] (ln_mod_vectors).  The sums run over the
// lane's chunks in order and then across the wave.
__device__ __forceinline__ void ln_mod_row_bf16(const u32x4 (&v)[kLnMaxChunks], const u32x4 (&g)[kLnMaxChunks],
                                                const u32x4 (&t)[kLnMaxChunks], int64_t nchunk, int64_t D, int lane,
                                                bf16_t* __restrict__ hr) {
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
#pragma unroll
  for (int c = 0; c < kLnMaxChunks; ++c) {
    const int64_t idx = lane + kWave * c;
    if (idx < nchunk) {
      u32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a = (__uint_as_float(v[c][e] << 16) - mean) * rstd * (1.f + __uint_as_float(g[c][e] << 16)) +
                        __uint_as_float(t[c][e] << 16);
        const float b = (__uint_as_float(v[c][e] & 0xffff0000u) - mean) * rstd *
                            (1.f + __uint_as_float(g[c][e] & 0xffff0000u)) +
                        __uint_as_float(t[c][e] & 0xffff0000u);
        o[e] = pack_bf2(a, b);
      }
      reinterpret_cast<u32x4*>(hr)[idx] = o;
    }
  }
}

// The lane's chunks of the scale and shift vectors, with unconditional
// loads (lanes past the end read the last chunk again; never used), so a
// caller can issue them together with the row's own loads.
__device__ __forceinline__ void ln_mod_vectors(const bf16_t* __restrict__ sh, const bf16_t* __restrict__ sc,
                                               int64_t nchunk, int lane, u32x4 (&g)[kLnMaxChunks],
                                               u32x4 (&t)[kLnMaxChunks]) {
#pragma unroll
  for (int c = 0; c < kLnMaxChunks; ++c) {
    const int64_t idx = std::min<int64_t>(lane + kWave * c, nchunk - 1);
    g[c] = reinterpret_cast<const u32x4*>(sc)[idx];
    t[c] = reinterpret_cast<const u32x4*>(sh)[idx];
  }
}

}  // namespace
}  // namespace avits
