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
// Up to N = 16384 one 1024-thread workgroup does the whole selection: at the
// sizes of a resolution transition (N = 4096 .. 16384 scores, 16-64 KiB) the
// cost is latency, not bandwidth, and the keys stay in registers between
// passes (each thread holds consecutive elements, so the emission is one
// workgroup scan).  Larger N runs the same passes grid-wide (below).
#include <mutex>

#include "common.h"
#include "select_block.h"

namespace avits {
namespace {

__global__ __launch_bounds__(kThreads) void radix_select_kernel(const float* __restrict__ scores,
                                                                const float* __restrict__ delta, int N, int k,
                                                                int32_t* __restrict__ idx) {
  select_block(scores, delta, N, k, idx);
}

// B independent selections, one workgroup each: element b selects the top
// k[b] of scores[off[b] .. off[b + 1]) and writes local indices at
// idx + out[b].
constexpr int kMaxBatch = 64;
struct SelBatch {
  int64_t off[kMaxBatch + 1];
  int64_t out[kMaxBatch];
  int32_t k[kMaxBatch];
};

__global__ __launch_bounds__(kThreads) void radix_select_batched_kernel(const float* __restrict__ scores,
                                                                        const float* __restrict__ delta,
                                                                        const SelBatch bt, int32_t* __restrict__ idx) {
  const int b = blockIdx.x;
  const int64_t o = bt.off[b];
  const int N = int(bt.off[b + 1] - o), k = bt.k[b];
  if (k == 0) return;
  select_block(scores + o, delta ? delta + o : nullptr, N, k, idx + bt.out[b]);
}

// ---------------------------------------------------------------------------
// Grid-wide radix select for N above what one workgroup holds in registers:
// the same four digit passes and index-order emission, spread over the GPU.
//   init            state: prefix 0, need k, histograms zeroed
//   4 x hist, scan  every workgroup histograms the current digit of the keys
//                   that match the prefix (LDS, then one atomic per bin: the
//                   sums are order-free); one workgroup picks the digit
//   count           per 4096-element chunk: keys > T and keys == T
//   offsets         one workgroup scans the chunk counts in index order:
//                   each chunk's output offset and its quota of keys == T
//   emit            each chunk writes its selected indices in index order
// Scores are read with 16-byte loads; every pass streams them once.
constexpr int kGT = 256;               // threads per workgroup of the grid passes
constexpr int kGWaves = kGT / kWave;
constexpr int kHistBlocks = 2048;      // histogram workgroups (grid-stride)
constexpr int kChunk = 16 * kGT;       // elements per count / emit workgroup (16 per thread)

struct SelState {
  uint32_t prefix;                     // digits chosen so far, in place
  uint32_t need;                       // rank of the k-th largest among keys matching the prefix
  uint32_t pad[62];
  uint32_t hist[4][256];               // global digit histograms, one per pass
};

__global__ __launch_bounds__(kGT) void select_init_kernel(SelState* __restrict__ st, uint32_t k) {
  for (int b = threadIdx.x; b < 4 * 256; b += kGT) (&st->hist[0][0])[b] = 0u;
  if (threadIdx.x == 0) {
    st->prefix = 0u;
    st->need = k;
  }
}

// Keys of elements i0 .. i0 + 3; live[e] is false past the end of the scores.
__device__ __forceinline__ void load_keys4(const float* __restrict__ scores, const float* __restrict__ delta,
                                           int64_t N, int64_t i0, uint32_t (&key)[4], bool (&live)[4]) {
  if (i0 + 3 < N && (reinterpret_cast<uintptr_t>(scores + i0) & 15) == 0 &&
      (!delta || (reinterpret_cast<uintptr_t>(delta + i0) & 15) == 0)) {
    float4 v = *reinterpret_cast<const float4*>(scores + i0);
    if (delta) {
      const float4 d = *reinterpret_cast<const float4*>(delta + i0);
      v.x += d.x; v.y += d.y; v.z += d.z; v.w += d.w;
    }
    key[0] = order_key(v.x); key[1] = order_key(v.y); key[2] = order_key(v.z); key[3] = order_key(v.w);
    live[0] = live[1] = live[2] = live[3] = true;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      live[e] = i0 + e < N;
      key[e] = live[e] ? key_at(scores, delta, i0 + e) : 0u;
    }
  }
}

constexpr int kSubHist = 4;  // LDS histogram copies per wave (lane % 4): spreads atomics on one bin

__global__ __launch_bounds__(kGT) void select_hist_kernel(const float* __restrict__ scores,
    const float* __restrict__ delta, int64_t N, int pass,
                                                          SelState* __restrict__ st) {
  __shared__ uint32_t hs[kGWaves * kSubHist][256];
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  uint32_t* h = hs[wave * kSubHist + (lane & (kSubHist - 1))];
  for (int b = tid; b < kGWaves * kSubHist * 256; b += kGT) (&hs[0][0])[b] = 0u;
  __syncthreads();
  const int shift = 24 - 8 * pass;
  const uint32_t mask = pass ? 0xffffffffu << (32 - 8 * pass) : 0u;
  const uint32_t prefix = st->prefix & mask;
  // The top digit of similar scores coincides (one exponent covers most of a
  // min-max-normalised score range), so in the first pass a wave adds its two
  // most frequent-looking digits with one atomic each (ballot) before the
  // remaining lanes add one by one; later passes, whose digits are spread,
  // aggregate only one (which also bounds the cost of heavily tied scores).
  // A thread's four keys go through each round together: one leader digit,
  // one ballot per key, one atomic for all of them.
  const int rounds = pass == 0 ? 2 : 1;
  auto count4 = [&](const uint32_t (&key)[4], const bool (&ok)[4]) {
    bool pending[4];
    uint32_t digit[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      pending[e] = ok[e] && (key[e] & mask) == prefix;
      digit[e] = (key[e] >> shift) & 255u;
    }
    for (int it = 0; it < rounds; ++it) {
      const uint64_t act = __ballot(pending[0] || pending[1] || pending[2] || pending[3]);
      if (act == 0) break;
      const int leader = __ffsll(static_cast<unsigned long long>(act)) - 1;
      const uint32_t first = pending[0] ? digit[0] : pending[1] ? digit[1] : pending[2] ? digit[2] : digit[3];
      const uint32_t d0 = __builtin_amdgcn_readlane(first, leader);  // leader is wave-uniform
      uint32_t total = 0u;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        total += uint32_t(__popcll(__ballot(pending[e] && digit[e] == d0)));
        pending[e] = pending[e] && digit[e] != d0;
      }
      if (lane == leader) atomicAdd(&h[d0], total);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (pending[e]) atomicAdd(&h[digit[e]], 1u);
  };
  // Grid-stride over groups of four keys, the next group's 16-byte loads in
  // flight while the current group is counted (groups that are not whole
  // or not 16-byte aligned take load_keys4's element path instead).
  const int64_t groups = (N + 3) / 4, stride = int64_t(gridDim.x) * kGT;
  const bool al = (reinterpret_cast<uintptr_t>(scores) & 15) == 0 &&
                  (!delta || (reinterpret_cast<uintptr_t>(delta) & 15) == 0);
  float4 rv = make_float4(0.f, 0.f, 0.f, 0.f), rd = rv;
  auto issue = [&](int64_t i0) {
    if (al && i0 + 3 < N) {
      rv = *reinterpret_cast<const float4*>(scores + i0);
      if (delta) rd = *reinterpret_cast<const float4*>(delta + i0);
    }
  };
  int64_t g = int64_t(blockIdx.x) * kGT + tid;
  issue(4 * g);
  for (; g - tid < groups; g += stride) {
    uint32_t key[4];
    bool live[4];
    const int64_t i0 = 4 * g;
    if (al && i0 + 3 < N) {
      float4 v = rv;
      if (delta) {
        v.x += rd.x; v.y += rd.y; v.z += rd.z; v.w += rd.w;
      }
      key[0] = order_key(v.x); key[1] = order_key(v.y); key[2] = order_key(v.z); key[3] = order_key(v.w);
      live[0] = live[1] = live[2] = live[3] = true;
    } else {
      load_keys4(scores, delta, N, i0, key, live);  // past the end: live = false
    }
    issue(4 * (g + stride));
    count4(key, live);
  }
  __syncthreads();
  for (int b = tid; b < 256; b += kGT) {
    uint32_t c = 0u;
#pragma unroll
    for (int w = 0; w < kGWaves * kSubHist; ++w) c += hs[w][b];
    if (c) atomicAdd(&st->hist[pass][b], c);
  }
}

// One workgroup: the digit b of this pass with (matching keys above b) <
// need <= (matching keys at or above b).
__global__ __launch_bounds__(256) void select_scan_kernel(int pass, SelState* __restrict__ st) {
  __shared__ uint32_t wsum[4];
  const int b = threadIdx.x, wave = b / kWave, lane = b % kWave;
  const uint32_t c = st->hist[pass][b];
  const uint32_t suf = wave_incl_suffix_u32(c);  // suffix sum inside the wave, high lanes down
  if (lane == 0) wsum[wave] = suf;
  __syncthreads();
  uint32_t higher = 0u;
  for (int w = wave + 1; w < 4; ++w) higher += wsum[w];
  const uint32_t above = suf - c + higher, need = st->need;
  __syncthreads();
  if (above < need && above + c >= need) {
    st->prefix |= uint32_t(b) << (24 - 8 * pass);
    st->need = need - above;
  }
}

// Sixteen consecutive elements of thread t of chunk `chunk`: t * 16 ..
__device__ __forceinline__ void chunk_keys(const float* __restrict__ scores, const float* __restrict__ delta,
                                           int64_t N, int64_t i0, uint32_t (&key)[16], bool (&live)[16]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t k4[4];
    bool l4[4];
    load_keys4(scores, delta, N, i0 + 4 * q, k4, l4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      key[4 * q + e] = k4[e];
      live[4 * q + e] = l4[e];
    }
  }
}

// Exclusive scan over a kGT-thread workgroup; *total gets the sum.
__device__ __forceinline__ uint32_t grid_block_scan(uint32_t v, uint32_t* wsum, uint32_t* total) {
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const uint32_t incl = wave_incl_scan_u32(v);
  __syncthreads();
  if (lane == kWave - 1) wsum[wave] = incl;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kGWaves; ++w) {
    before += w < wave ? wsum[w] : 0u;
    all += wsum[w];
  }
  *total = all;
  return before + incl - v;
}

__global__ __launch_bounds__(kGT) void select_count_kernel(const float* __restrict__ scores,
    const float* __restrict__ delta, int64_t N,
                                                           const SelState* __restrict__ st,
                                                           uint32_t* __restrict__ cnt) {
  __shared__ uint32_t wsum[kGWaves];
  const uint32_t T = st->prefix;
  const int64_t i0 = int64_t(blockIdx.x) * kChunk + 16 * threadIdx.x;
  uint32_t key[16];
  bool live[16];
  chunk_keys(scores, delta, N, i0, key, live);
  uint32_t packed = 0u;  // keys > T in the high 16 bits, keys == T in the low
#pragma unroll
  for (int e = 0; e < 16; ++e) packed += live[e] ? ((key[e] > T) << 16) | uint32_t(key[e] == T) : 0u;
  uint32_t tot;
  grid_block_scan(packed, wsum, &tot);
  if (threadIdx.x == 0) {
    cnt[2 * blockIdx.x] = tot >> 16;
    cnt[2 * blockIdx.x + 1] = tot & 0xffffu;
  }
}

// One workgroup of 1024 threads walks the chunks in index order, four
// consecutive chunks per thread per step (two 16-byte loads), with two
// block-wide scans per step: every chunk's quota of keys == T (the first
// `need` of them in index order) and its output offset.
__global__ __launch_bounds__(kThreads) void select_offsets_kernel(const uint32_t* __restrict__ cnt, int nchunks,
                                                                  const SelState* __restrict__ st,
                                                                  uint32_t* __restrict__ off) {
  constexpr int kPer = 4;
  __shared__ uint32_t wsum[kWaves];
  const uint32_t need = st->need;
  uint32_t eq_before = 0u, out_before = 0u;
  for (int c0 = 0; c0 < nchunks; c0 += kThreads * kPer) {
    const int cb = c0 + kPer * threadIdx.x;
    uint32_t gt[kPer], eq[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      gt[j] = cb + j < nchunks ? cnt[2 * (cb + j)] : 0u;
      eq[j] = cb + j < nchunks ? cnt[2 * (cb + j) + 1] : 0u;
    }
    const uint32_t eq_run = eq[0] + eq[1] + eq[2] + eq[3];
    uint32_t eq_tot;
    uint32_t eb = eq_before + block_exclusive_scan(eq_run, wsum, &eq_tot);
    uint32_t take[kPer], sel_run = 0u;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      take[j] = eb < need ? min(eq[j], need - eb) : 0u;
      eb += eq[j];
      sel_run += gt[j] + take[j];
    }
    uint32_t sel_tot;
    uint32_t ob = out_before + block_exclusive_scan(sel_run, wsum, &sel_tot);
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      if (cb + j < nchunks) {
        off[2 * (cb + j)] = ob;
        off[2 * (cb + j) + 1] = take[j];
      }
      ob += gt[j] + take[j];
    }
    eq_before += eq_tot;
    out_before += sel_tot;
  }
}

// Chunk = 4 waves x 4 rounds x 256 consecutive elements (4 per lane, one
// 16-byte load).  Counts per wave first (keys stay in registers), a 4-entry
// scan in LDS, then each round ranks its lanes with a wave scan, so
// neighbouring lanes store neighbouring output positions.
__global__ __launch_bounds__(kGT) void select_emit_kernel(const float* __restrict__ scores,
    const float* __restrict__ delta, int64_t N,
                                                          const SelState* __restrict__ st,
                                                          const uint32_t* __restrict__ off, int64_t k,
                                                          int32_t* __restrict__ idx) {
  constexpr int kRounds = kChunk / kGT / 4;  // 4
  __shared__ uint32_t wcnt[kGWaves];
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const uint32_t T = st->prefix;
  const int64_t w0 = int64_t(blockIdx.x) * kChunk + int64_t(wave) * kRounds * 4 * kWave;
  uint32_t key[kRounds][4];
  bool live[kRounds][4];
  uint32_t packed = 0u;  // keys > T in the high 16 bits, keys == T in the low
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    load_keys4(scores, delta, N, w0 + 4 * (r * kWave + lane), key[r], live[r]);
#pragma unroll
    for (int e = 0; e < 4; ++e) packed += live[r][e] ? ((key[r][e] > T) << 16) | uint32_t(key[r][e] == T) : 0u;
  }
  packed = wave_sum_u32(packed);
  if (lane == 0) wcnt[wave] = packed;
  __syncthreads();
  uint32_t before = 0u;  // this chunk's keys before this wave, packed
  for (int w = 0; w < wave; ++w) before += wcnt[w];
  uint32_t gt_b = before >> 16, eq_b = before & 0xffffu;
  const uint32_t base = off[2 * blockIdx.x], take = off[2 * blockIdx.x + 1];
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    uint32_t mine = 0u;
#pragma unroll
    for (int e = 0; e < 4; ++e) mine += live[r][e] ? ((key[r][e] > T) << 16) | uint32_t(key[r][e] == T) : 0u;
    const uint32_t incl = wave_incl_scan_u32(mine);  // wave inclusive scan of the packed counts
    const uint32_t ex = incl - mine, all = __builtin_amdgcn_readlane(incl, kWave - 1);
    uint32_t g = gt_b + (ex >> 16), q = eq_b + (ex & 0xffffu);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool gt = live[r][e] && key[r][e] > T, eq = live[r][e] && key[r][e] == T;
      const bool sel = gt || (eq && q < take);
      const uint32_t at = base + g + min(q, take);
      if (sel && at < uint64_t(k)) idx[at] = int32_t(w0 + 4 * (r * kWave + lane) + e);
      g += gt;
      q += eq;
    }
    gt_b += all >> 16;
    eq_b += all & 0xffffu;
  }
}

inline size_t align256(size_t v) { return (v + 255) / 256 * 256; }

struct SelWs {
  SelState* st;
  uint32_t* cnt;  // [nchunks][2]
  uint32_t* off;  // [nchunks][2]
  size_t bytes;
};
SelWs select_ws_layout(char* base, int64_t N) {
  SelWs w{};
  const int64_t nchunks = (N + kChunk - 1) / kChunk;
  size_t o = 0;
  w.st = reinterpret_cast<SelState*>(base + o); o += align256(sizeof(SelState));
  w.cnt = reinterpret_cast<uint32_t*>(base + o); o += align256(size_t(nchunks) * 8);
  w.off = reinterpret_cast<uint32_t*>(base + o); o += align256(size_t(nchunks) * 8);
  w.bytes = o;
  return w;
}

// Workspace bytes of the grid path for N scores (select_ws_layout's size,
// usable in constant expressions).
constexpr size_t select_ws_bytes(int64_t N) {
  return (sizeof(SelState) + 255) / 256 * 256 + 2 * ((size_t((N + kChunk - 1) / kChunk) * 8 + 255) / 256 * 256);
}

// Allocation-free selection: the grid path's state lives in this file-scope
// device array instead of a caller workspace.  Each GPU holds its own copy
// until the process ends; its address on a device comes from
// hipGetSymbolAddress (the array's name is not a device address in host
// code).
constexpr int64_t kNoAllocMaxN = int64_t(1) << 26;
constexpr size_t kNoAllocBytes = select_ws_bytes(kNoAllocMaxN);
__device__ __align__(256) unsigned char scratch[kNoAllocBytes];

constexpr int64_t kOneBlockMax = int64_t(kThreads) * kRegKeys;  // 16384: one workgroup, keys in registers

}  // namespace
}  // namespace avits

using namespace avits;

extern "C" size_t avits_select_workspace_bytes(int64_t N) {
  if (N <= kOneBlockMax) return 0;
  return select_ws_layout(nullptr, N).bytes;
}

static int select_impl(const float* scores, const float* delta, int64_t N, int64_t k, int32_t* idx, void* workspace,
                       size_t workspace_bytes, void* stream) {
  AVITS_REQUIRE(N >= 1 && N <= INT32_MAX, "select: N=%lld outside [1, 2^31)", (long long)N);
  AVITS_REQUIRE(k >= 0 && k <= N, "select: k=%lld outside [0, N=%lld]", (long long)k, (long long)N);
  if (k == 0) return AVITS_OK;
  AVITS_REQUIRE(scores && idx, "select: null scores/idx");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (N <= kOneBlockMax) {
    TimedLaunch timed("select", s);
    hipLaunchKernelGGL(radix_select_kernel, dim3(1), dim3(kThreads), 0, s, scores, delta, int(N), int(k), idx);
    return launch_status("select");
  }
  const SelWs need = select_ws_layout(nullptr, N);
  if (!workspace || workspace_bytes < need.bytes)
    return set_error(AVITS_ERR_WORKSPACE, "select: workspace of %zu bytes, need %zu for N=%lld", workspace_bytes,
                     need.bytes, (long long)N);
  const SelWs ws = select_ws_layout(static_cast<char*>(workspace), N);
  const int nchunks = int((N + kChunk - 1) / kChunk);
  const int hblocks = int(std::min<int64_t>(kHistBlocks, (N + 4 * kGT * 8 - 1) / (4 * kGT * 8)));
  TimedLaunch timed("select", s);
  hipLaunchKernelGGL(select_init_kernel, dim3(1), dim3(kGT), 0, s, ws.st, uint32_t(k));
  for (int pass = 0; pass < 4; ++pass) {
    hipLaunchKernelGGL(select_hist_kernel, dim3(hblocks), dim3(kGT), 0, s, scores, delta, N, pass, ws.st);
    hipLaunchKernelGGL(select_scan_kernel, dim3(1), dim3(256), 0, s, pass, ws.st);
  }
  hipLaunchKernelGGL(select_count_kernel, dim3(nchunks), dim3(kGT), 0, s, scores, delta, N, ws.st, ws.cnt);
  hipLaunchKernelGGL(select_offsets_kernel, dim3(1), dim3(kThreads), 0, s, ws.cnt, nchunks, ws.st, ws.off);
  hipLaunchKernelGGL(select_emit_kernel, dim3(nchunks), dim3(kGT), 0, s, scores, delta, N, ws.st, ws.off, k, idx);
  return launch_status("select");
}

extern "C" int avits_select(const float* scores, int64_t N, int64_t k, int32_t* idx, void* workspace,
                            size_t workspace_bytes, void* stream) {
  return select_impl(scores, nullptr, N, k, idx, workspace, workspace_bytes, stream);
}

extern "C" int avits_select_perturbed(const float* scores, const float* delta, int64_t N, int64_t k, int32_t* idx,
                                      void* workspace, size_t workspace_bytes, void* stream) {
  AVITS_REQUIRE(k == 0 || delta, "select_perturbed: null delta");
  return select_impl(scores, delta, N, k, idx, workspace, workspace_bytes, stream);
}

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of `scratch` on the calling thread's current device,
// looked up once per device.
int scratch_on_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return set_error(AVITS_ERR_HIP, "select_noalloc: hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return set_error(AVITS_ERR_UNSUPPORTED, "select_noalloc: device %d outside [0, %d)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return set_error(AVITS_ERR_HIP, "select_noalloc: hipGetSymbolAddress on device %d: %s", dev,
                       hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return AVITS_OK;
}
}  // namespace

extern "C" size_t avits_select_noalloc_max_n(void) { return size_t(kNoAllocMaxN); }

extern "C" int avits_select_noalloc(const float* scores, int64_t N, int64_t k, int32_t* idx, void* stream) {
  AVITS_REQUIRE(N >= 1 && N <= kNoAllocMaxN, "select_noalloc: N=%lld outside [1, %lld]", (long long)N,
                (long long)kNoAllocMaxN);
  AVITS_REQUIRE(k >= 0 && k <= N, "select_noalloc: k=%lld outside [0, N=%lld]", (long long)k, (long long)N);
  if (k == 0) return AVITS_OK;
  AVITS_REQUIRE(scores && idx, "select_noalloc: null scores/idx");
  if (N <= kOneBlockMax) return select_impl(scores, nullptr, N, k, idx, nullptr, 0, stream);
  void* ws = nullptr;
  const int rc = scratch_on_current_device(&ws);
  if (rc != AVITS_OK) return rc;
  static_assert(kNoAllocBytes >= select_ws_bytes(kNoAllocMaxN), "scratch holds the largest grid-path state");
  return select_impl(scores, nullptr, N, k, idx, ws, kNoAllocBytes, stream);
}

extern "C" int avits_select_batched(const float* scores, const float* delta, int32_t B, const int64_t* offsets,
                                    const int64_t* k, int32_t* idx, void* stream) {
  AVITS_REQUIRE(B >= 1 && B <= kMaxBatch, "select_batched: B=%d outside [1, %d]", B, kMaxBatch);
  AVITS_REQUIRE(offsets && k, "select_batched: null offsets/k");
  SelBatch bt{};
  int64_t out = 0;
  AVITS_REQUIRE(offsets[0] == 0, "select_batched: offsets[0]=%lld must be 0", (long long)offsets[0]);
  for (int b = 0; b < B; ++b) {
    const int64_t n = offsets[b + 1] - offsets[b];
    AVITS_REQUIRE(n >= 1 && n <= kOneBlockMax, "select_batched: element %d has N=%lld outside [1, %d]", b,
                  (long long)n, kOneBlockMax);
    AVITS_REQUIRE(k[b] >= 0 && k[b] <= n, "select_batched: element %d has k=%lld outside [0, N=%lld]", b,
                  (long long)k[b], (long long)n);
    bt.off[b] = offsets[b];
    bt.k[b] = int32_t(k[b]);
    bt.out[b] = out;
    out += k[b];
  }
  bt.off[B] = offsets[B];
  if (out == 0) return AVITS_OK;
  AVITS_REQUIRE(scores && idx, "select_batched: null scores/idx");
  hipStream_t s = static_cast<hipStream_t>(stream);
  TimedLaunch timed("select", s);
  hipLaunchKernelGGL(radix_select_batched_kernel, dim3(unsigned(B)), dim3(kThreads), 0, s, scores, delta, bt, idx);
  return launch_status("select_batched");
}
