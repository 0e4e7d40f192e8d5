// Deterministic top-K selection (Eq. topk) by radix select over fp32 scores.
//
// Scores map to order-preserving uint32 keys (larger score -> larger key;
// -0.0 folded into +0.0; every NaN -> key 0, below -inf).  Four 8-bit digit
// passes, most significant first, narrow the candidates down to the exact key
// T of the k-th largest element and the number `need` of elements equal to T
// that still belong to the top-k.  A final pass in index order emits every
// element with key > T and the first `need` elements with key == T (lowest
// indices win), so the output is ascending and independent of atomic order:
// the only atomics are histogram increments, whose sums are order-free.
//
// One 1024-thread workgroup does the whole selection: at the sizes of a
// resolution transition (N = 4096 .. 16384 scores, 16-64 KiB) the cost is
// latency, not bandwidth; the scores stay in L2 between passes.
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

// Exclusive prefix sum over the workgroup; returns the total in *total.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* wsum, uint32_t* total) {
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  uint32_t incl = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t t = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += t;
  }
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

// Up to kRegKeys keys per thread stay in registers (N <= 16384); larger N
// re-reads the scores (L2-resident) on every pass.
constexpr int kRegKeys = 16;

// Calls f(j, i, key) for every element i = tid + kThreads * j < N.
template <bool IN_REGS, typename F>
__device__ __forceinline__ void for_each_key(const uint32_t (&keys)[IN_REGS ? kRegKeys : 1],
                                             const float* __restrict__ scores, int N, F&& f) {
  if constexpr (IN_REGS) {
#pragma unroll
    for (int j = 0; j < kRegKeys; ++j) {
      const int i = threadIdx.x + kThreads * j;
      if (i < N) f(i, keys[j]);
    }
  } else {
    for (int i = threadIdx.x; i < N; i += kThreads) f(i, order_key(scores[i]));
  }
}

template <bool IN_REGS>
__global__ __launch_bounds__(kThreads) void radix_select_kernel(const float* __restrict__ scores, int N, int k,
                                                                int32_t* __restrict__ idx) {
  __shared__ uint32_t hist[kWaves][256];   // per-wave histograms: atomics contend only inside a wave
  __shared__ uint32_t tot_s[256], suf_s[256];
  __shared__ uint32_t wsum[kWaves];
  __shared__ uint32_t s_digit, s_above;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;

  uint32_t keys[IN_REGS ? kRegKeys : 1] = {};
  if constexpr (IN_REGS) {
#pragma unroll
    for (int j = 0; j < kRegKeys; ++j) {
      const int i = tid + kThreads * j;
      keys[j] = i < N ? order_key(scores[i]) : 0u;
    }
  }

  uint32_t prefix = 0u, mask = 0u;
  uint32_t remaining = uint32_t(k);  // rank of the k-th largest among the current candidates
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int b = tid; b < kWaves * 256; b += kThreads) (&hist[0][0])[b] = 0u;
    __syncthreads();
    for_each_key<IN_REGS>(keys, scores, N, [&](int, uint32_t key) {
      if ((key & mask) == prefix) atomicAdd(&hist[wave][(key >> shift) & 255u], 1u);
    });
    __syncthreads();
    // Waves 0..3 own digits 64w .. 64w + 63: the count per digit and its
    // suffix sum inside the wave (shuffle scan from the high lanes down).
    if (wave < 4) {
      const int b = 64 * wave + lane;
      uint32_t c = 0u;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) c += hist[w][b];
      uint32_t suf = c;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t t = __shfl_down(suf, o, kWave);
        if (lane + o < kWave) suf += t;
      }
      tot_s[b] = c;
      suf_s[b] = suf;
      if (lane == 0) wsum[wave] = suf;  // this wave's 64 digits in total
    }
    __syncthreads();
    // The selected digit b has (candidates above b) < remaining <= (candidates at or above b).
    if (wave < 4) {
      const int b = 64 * wave + lane;
      uint32_t higher = 0u;
      for (int w = wave + 1; w < 4; ++w) higher += wsum[w];
      const uint32_t c = tot_s[b];
      const uint32_t above = suf_s[b] - c + higher;
      if (above < remaining && above + c >= remaining) {
        s_digit = uint32_t(b);
        s_above = above;
      }
    }
    __syncthreads();
    prefix |= s_digit << shift;
    mask |= 255u << shift;
    remaining -= s_above;
    __syncthreads();
  }
  // T = prefix; `remaining` elements equal to T are still needed.  Emit in
  // index order, one 1024-element chunk per block-wide scan.
  const uint32_t T = prefix, need = remaining;
  uint32_t eq_before = 0u, out_before = 0u;
  const int nchunks = (N + kThreads - 1) / kThreads;
  auto emit_chunk = [&](int i, uint32_t key) {
    uint32_t gt = 0u, eq = 0u;
    if (i < N) {
      gt = key > T;
      eq = key == T;
    }
    uint32_t tot;
    // Pack both counts: low 16 bits equal-to-T, high 16 bits greater-than-T.
    const uint32_t ex = block_exclusive_scan(eq | (gt << 16), wsum, &tot);
    const uint32_t eq_ex = ex & 0xffffu, gt_ex = ex >> 16;
    const uint32_t eq_tot = tot & 0xffffu, gt_tot = tot >> 16;
    const uint32_t eq_quota = need > eq_before ? need - eq_before : 0u;  // eq still to take
    const bool sel = gt || (eq && eq_ex < eq_quota);
    const uint32_t at = out_before + gt_ex + min(eq_ex, eq_quota);
    if (sel && at < uint32_t(k)) idx[at] = i;
    out_before += gt_tot + min(eq_tot, eq_quota);
    eq_before += eq_tot;
  };
  if constexpr (IN_REGS) {
#pragma unroll
    for (int j = 0; j < kRegKeys; ++j)
      if (j < nchunks) emit_chunk(tid + kThreads * j, keys[j]);
  } else {
    for (int j = 0; j < nchunks; ++j) {
      const int i = tid + kThreads * j;
      emit_chunk(i, i < N ? order_key(scores[i]) : 0u);
    }
  }
}

}  // namespace
}  // namespace avits

using namespace avits;

extern "C" size_t avits_select_workspace_bytes(int64_t N) {
  (void)N;
  return 0;
}

extern "C" int avits_select(const float* scores, int64_t N, int64_t k, int32_t* idx, void* workspace,
                            size_t workspace_bytes, void* stream) {
  (void)workspace;
  (void)workspace_bytes;
  AVITS_REQUIRE(N >= 1 && N <= INT32_MAX, "select: N=%lld outside [1, 2^31)", (long long)N);
  AVITS_REQUIRE(k >= 0 && k <= N, "select: k=%lld outside [0, N=%lld]", (long long)k, (long long)N);
  if (k == 0) return AVITS_OK;
  AVITS_REQUIRE(scores && idx, "select: null scores/idx");
  hipStream_t s = static_cast<hipStream_t>(stream);
  TimedLaunch timed("select", s);
  if (N <= int64_t(kThreads) * kRegKeys)
    hipLaunchKernelGGL(radix_select_kernel<true>, dim3(1), dim3(kThreads), 0, s, scores, int(N), int(k), idx);
  else
    hipLaunchKernelGGL(radix_select_kernel<false>, dim3(1), dim3(kThreads), 0, s, scores, int(N), int(k), idx);
  return launch_status("select");
}
