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

__global__ __launch_bounds__(kThreads) void radix_select_kernel(const float* __restrict__ scores, int N, int k,
                                                                int32_t* __restrict__ idx) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t wsum[kWaves];
  __shared__ uint32_t s_digit, s_above;
  const int tid = threadIdx.x;

  uint32_t prefix = 0u, mask = 0u;
  uint32_t remaining = uint32_t(k);  // rank of T among the current candidates
  for (int shift = 24; shift >= 0; shift -= 8) {
    if (tid < 256) hist[tid] = 0u;
    __syncthreads();
    for (int i = tid; i < N; i += kThreads) {
      const uint32_t key = order_key(scores[i]);
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    // Suffix sums over digits: above[b] = candidates with digit > b.
    if (tid < 256) {
      // Count of candidates whose digit is strictly greater than this bin.
      uint32_t above = 0u;
      for (int b = 255; b > tid; --b) above += hist[b];
      const uint32_t here = hist[tid];
      if (above < remaining && above + here >= remaining) {
        s_digit = uint32_t(tid);
        s_above = above;
      }
    }
    __syncthreads();
    prefix |= s_digit << shift;
    mask |= 255u << shift;
    remaining -= s_above;
    __syncthreads();
  }
  // T = prefix; `remaining` elements equal to T are still needed.
  const uint32_t T = prefix, need = remaining;
  uint32_t eq_before = 0u, out_before = 0u;
  for (int base = 0; base < N; base += kThreads) {
    const int i = base + tid;
    uint32_t gt = 0u, eq = 0u;
    if (i < N) {
      const uint32_t key = order_key(scores[i]);
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
  TimedLaunch timed("select", static_cast<hipStream_t>(stream));
  hipLaunchKernelGGL(radix_select_kernel, dim3(1), dim3(kThreads), 0, static_cast<hipStream_t>(stream), scores,
                     int(N), int(k), idx);
  return launch_status("select");
}
