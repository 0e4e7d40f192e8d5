// One-workgroup radix selection of the top k of N <= 16384 fp32 values held
// in registers (Eq. topk): order-preserving uint32 keys, four 8-bit digit
// passes with per-wave LDS histograms, and an index-ordered emission so ties
// go to the lowest index and the output is ascending.  Shared by the
// selection entry points and the fused score + selection.
#pragma once

#include "common.h"

namespace avits {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;

__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;  // NaN ranks lowest
  if (u == 0x80000000u) u = 0u;                     // -0.0 == +0.0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Key of element i: of scores[i], or of the fp32 sum scores[i] + delta[i]
// when a perturbation is given (the seeded tie-break of Eq. topk).
__device__ __forceinline__ uint32_t key_at(const float* __restrict__ scores, const float* __restrict__ delta,
                                           int64_t i) {
  return order_key(delta ? scores[i] + delta[i] : scores[i]);
}

// Integer wave scans without the LDS pipe: DPP row shifts inside each
// 16-lane row (lanes shifted in from outside the row read 0), then the row
// totals by readlane.  Integer sums, so any order gives the same result.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), CTRL, 0xf, 0xf, true));
}
constexpr int kDppShr1 = 0x111, kDppShl1 = 0x101;  // row_shr:n = 0x110 + n, row_shl:n = 0x100 + n
// Inclusive prefix sum over the wave (lane l gets the sum of lanes 0 .. l).
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v) {
  v += dpp_u32<kDppShr1>(v);
  v += dpp_u32<kDppShr1 + 1>(v);
  v += dpp_u32<kDppShr1 + 3>(v);
  v += dpp_u32<kDppShr1 + 7>(v);
  const uint32_t t0 = __builtin_amdgcn_readlane(v, 15), t1 = __builtin_amdgcn_readlane(v, 31),
                 t2 = __builtin_amdgcn_readlane(v, 47);
  const int row = int(threadIdx.x % kWave) / 16;
  return v + (row > 0 ? t0 : 0u) + (row > 1 ? t1 : 0u) + (row > 2 ? t2 : 0u);
}
// Inclusive suffix sum over the wave (lane l gets the sum of lanes l .. 63).
__device__ __forceinline__ uint32_t wave_incl_suffix_u32(uint32_t v) {
  v += dpp_u32<kDppShl1>(v);
  v += dpp_u32<kDppShl1 + 1>(v);
  v += dpp_u32<kDppShl1 + 3>(v);
  v += dpp_u32<kDppShl1 + 7>(v);
  const uint32_t r1 = __builtin_amdgcn_readlane(v, 16), r2 = __builtin_amdgcn_readlane(v, 32),
                 r3 = __builtin_amdgcn_readlane(v, 48);
  const int row = int(threadIdx.x % kWave) / 16;
  return v + (row < 1 ? r1 : 0u) + (row < 2 ? r2 : 0u) + (row < 3 ? r3 : 0u);
}
// Sum over the wave, every lane receiving it.
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
  return __builtin_amdgcn_readlane(wave_incl_scan_u32(v), kWave - 1);
}

// Exclusive prefix sum over the workgroup; returns the total in *total.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* wsum, uint32_t* total) {
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const uint32_t incl = wave_incl_scan_u32(v);
  __syncthreads();
  if (lane == kWave - 1) wsum[wave] = incl;
  __syncthreads();
  uint32_t before = 0, all = 0;
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t s = wsum[w];
    before += w < wave ? s : 0u;
    all += s;
  }
  *total = all;
  return before + incl - v;
}

// kRegKeys keys per thread stay in registers: N <= 16384.
constexpr int kRegKeys = 16;

// The selection of one workgroup of kThreads threads over N <= 16384 keys
// held in registers: thread t holds the q = ceil(N / kThreads) consecutive
// elements t q .. t q + q - 1 in keys[0 .. q) (so the final emission needs a
// single workgroup scan); keys past N are ignored.  Writes the indices of
// the k largest keys (ties: lowest index) to idx in ascending order.
__device__ __forceinline__ void select_block_keys(const uint32_t (&keys)[kRegKeys], int N, int k,
                                                  int32_t* __restrict__ idx) {
  // Per-wave histograms (atomics contend only inside a wave), two sets: pass
  // p counts into set p mod 2 while the other set is cleared for pass p + 1,
  // so a pass needs two workgroup barriers (after the counts, after the
  // digit pick), not five.
  __shared__ __attribute__((aligned(16))) uint32_t hist[2][kWaves][256];
  __shared__ uint32_t wsum[kWaves];
  __shared__ uint32_t s_digit, s_above;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int q = (N + kThreads - 1) / kThreads;

  for (int b = tid; b < kWaves * 256; b += kThreads) (&hist[0][0][0])[b] = 0u;
  __syncthreads();
  uint32_t prefix = 0u, mask = 0u;
  uint32_t remaining = uint32_t(k);  // rank of the k-th largest among the current candidates
#pragma unroll 1
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass, cur = pass & 1;
    if (pass < 3)
      for (int b = tid; b < kWaves * 256; b += kThreads) (&hist[cur ^ 1][0][0])[b] = 0u;
    // Scores of one exponent share their top digits, so a wave first adds
    // its most frequent-looking digit(s) with one ballot-counted atomic
    // (two rounds in the first pass, one later), then the rest one by one.
    const int rounds = pass == 0 ? 2 : 1;
#pragma unroll
    for (int j = 0; j < kRegKeys; ++j) {
      if (j >= q) break;  // uniform
      const int i = tid * q + j;
      const uint32_t key = keys[j];
      bool pending = i < N && (key & mask) == prefix;
      const uint32_t digit = (key >> shift) & 255u;
      for (int it = 0; it < rounds; ++it) {
        const uint64_t act = __ballot(pending);
        if (act == 0) break;
        const int leader = __ffsll(static_cast<unsigned long long>(act)) - 1;
        const uint32_t d0 = __builtin_amdgcn_readlane(digit, leader);  // leader is wave-uniform
        const uint64_t same = __ballot(pending && digit == d0);
        if (lane == leader) atomicAdd(&hist[cur][wave][d0], uint32_t(__popcll(same)));
        pending = pending && digit != d0;
      }
      if (pending) atomicAdd(&hist[cur][wave][digit], 1u);
    }
    __syncthreads();
    // Wave 0 picks the digit: lane l owns digits 4 l .. 4 l + 3 (their
    // counts over the per-wave histograms), the suffix sum over the lanes
    // above it gives the candidates above its digits, and the selected
    // digit b has (candidates above b) < remaining <= (candidates at or
    // above b).
    if (wave == 0) {
      u32x4 c = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int w = 0; w < kWaves; ++w) c += *reinterpret_cast<const u32x4*>(&hist[cur][w][4 * lane]);
      const uint32_t own = c[0] + c[1] + c[2] + c[3];
      uint32_t above = wave_incl_suffix_u32(own) - own;
#pragma unroll
      for (int e = 3; e >= 0; --e) {
        if (above < remaining && above + c[e] >= remaining) {
          s_digit = uint32_t(4 * lane + e);
          s_above = above;
        }
        above += c[e];
      }
    }
    __syncthreads();
    prefix |= s_digit << shift;
    mask |= 255u << shift;
    remaining -= s_above;
  }
  // T = prefix; `remaining` elements equal to T are still needed.  One
  // workgroup scan of the per-thread counts of keys > T and == T gives each
  // thread its output offset; the threads' element ranges are consecutive,
  // so the output is in index order and the first `need` keys equal to T
  // (lowest indices) are the ones taken.
  const uint32_t T = prefix, need = remaining;
  uint32_t gt_c = 0u, eq_c = 0u;
#pragma unroll
  for (int j = 0; j < kRegKeys; ++j) {
    if (j < q && tid * q + j < N) {
      gt_c += keys[j] > T;
      eq_c += keys[j] == T;
    }
  }
  uint32_t tot;
  // Packed counts: low 16 bits equal-to-T, high 16 bits greater-than-T (N <= 16384).
  const uint32_t ex = block_exclusive_scan(eq_c | (gt_c << 16), wsum, &tot);
  uint32_t eq_seen = ex & 0xffffu;
  uint32_t at = (ex >> 16) + min(eq_seen, need);
#pragma unroll
  for (int j = 0; j < kRegKeys; ++j) {
    const int i = tid * q + j;
    if (j < q && i < N) {
      const uint32_t key = keys[j];
      if (key > T) {
        idx[at++] = i;
      } else if (key == T) {
        if (eq_seen < need) idx[at++] = i;
        ++eq_seen;
      }
    }
  }
}

__device__ __forceinline__ void select_block(const float* __restrict__ scores, const float* __restrict__ delta,
                                             int N, int k, int32_t* __restrict__ idx) {
  const int q = (N + kThreads - 1) / kThreads;
  uint32_t keys[kRegKeys];
#pragma unroll
  for (int j = 0; j < kRegKeys; ++j) {
    const int i = int(threadIdx.x) * q + j;
    keys[j] = j < q && i < N ? key_at(scores, delta, i) : 0u;
  }
  select_block_keys(keys, N, k, idx);
}

}  // namespace
}  // namespace avits
