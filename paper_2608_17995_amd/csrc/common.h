// Shared device helpers for the gfx950 kernels: storage types, bf16
// conversion, wavefront reductions and the MFMA operand types.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "avits.h"

namespace avits {

constexpr int kWave = 64;  // CDNA wavefront width

typedef uint16_t bf16_t;  // bf16 storage (bit pattern)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float(uint32_t(b) << 16); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32; NaN stays NaN).
__device__ __forceinline__ bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, static_cast<__bf16>(f)); }

// Two floats -> packed bf16 pair (low half = a), one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf2(float a, float b) {
  const bf16x2_t v = {static_cast<__bf16>(a), static_cast<__bf16>(b)};
  return __builtin_bit_cast(uint32_t, v);
}

// Element access for the two storage types.
template <typename T> struct Elem;
template <> struct Elem<float> {
  static __device__ __forceinline__ float load(const float* p, int64_t i) { return p[i]; }
  static __device__ __forceinline__ void store(float* p, int64_t i, float v) { p[i] = v; }
};
template <> struct Elem<bf16_t> {
  static __device__ __forceinline__ float load(const bf16_t* p, int64_t i) { return bf2f(p[i]); }
  static __device__ __forceinline__ void store(bf16_t* p, int64_t i, float v) { p[i] = f2bf(v); }
};

template <typename T> __device__ __forceinline__ float ld(const T* p, int64_t i) { return Elem<T>::load(p, i); }
template <typename T> __device__ __forceinline__ void st(T* p, int64_t i, float v) { Elem<T>::store(p, i, v); }

// Cross-lane exchanges that stay off the LDS pipe (a shuffle through
// ds_bpermute waits on it for each step): DPP moves inside 16-lane rows,
// v_permlane32_swap between the two halves of the wave, readlane.
template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141; // lane i <- 7 - i in each group of 8
constexpr int kDppMirror = 0x140;     // lane i <- 15 - i in each row of 16

// Lane l % 32 of each half: lo = v[l % 32], hi = v[l % 32 + 32].
__device__ __forceinline__ void wave_halves(float v, float& lo, float& hi) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  lo = __uint_as_float(p[0]);
  hi = __uint_as_float(p[1]);
}
// v + v[l ^ 32] and max(v, v[l ^ 32]) (the same bits as the shuffle forms).
__device__ __forceinline__ float sum_xor32(float v) {
  float lo, hi;
  wave_halves(v, lo, hi);
  return lo + hi;
}
__device__ __forceinline__ float max_xor32(float v) {
  float lo, hi;
  wave_halves(v, lo, hi);
  return fmaxf(lo, hi);
}

// Sum over aligned groups of n lanes (n = 1, 2, 4, 8 or 16), every lane of a
// group receiving it: the butterfly over lane bits 0, 1, 2, 3 in that
// order.  Once bits below b are summed a group of 2^b lanes holds one
// value, so the mirror moves pair the same groups as lane ^ 2^b, and the
// result is bit for bit the xor-shuffle butterfly's.
__device__ __forceinline__ float group_sum(float v, int n) {
  if (n > 1) v += dpp_move<kDppXor1>(v);
  if (n > 2) v += dpp_move<kDppXor2>(v);
  if (n > 4) v += dpp_move<kDppHalfMirror>(v);
  if (n > 8) v += dpp_move<kDppMirror>(v);
  return v;
}

// Wavefront reductions (all 64 lanes receive the result): each 16-lane row
// by DPP, then the four row values, read once each, combined as
// (row 0 + row 1) + (row 2 + row 3).
__device__ __forceinline__ float wave_sum(float v) {
  v = group_sum(v, 16);
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (r0 + r1) + (r2 + r3);
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_move<kDppXor1>(v));
  v = fmaxf(v, dpp_move<kDppXor2>(v));
  v = fmaxf(v, dpp_move<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_move<kDppMirror>(v));
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}
__device__ __forceinline__ float wave_min(float v) {
  v = fminf(v, dpp_move<kDppXor1>(v));
  v = fminf(v, dpp_move<kDppXor2>(v));
  v = fminf(v, dpp_move<kDppHalfMirror>(v));
  v = fminf(v, dpp_move<kDppMirror>(v));
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return fminf(fminf(r0, r1), fminf(r2, r3));
}

// Block-wide sum of one float per thread; `red` holds >= blockDim.x/64 floats.
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x / kWave, l = threadIdx.x % kWave, nw = blockDim.x / kWave;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

__device__ __forceinline__ f32x4 mfma16x16x32(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const u32x4& v) { return __builtin_bit_cast(bf16x8, v); }

// Workgroup barrier for LDS producer/consumer hand-offs: waits for this
// wave's own LDS operations (lgkmcnt) and meets the other waves, but leaves
// its global loads in flight.  __syncthreads() also carries a release fence,
// which drains every outstanding global load at each barrier; a software
// pipeline that keeps the next tiles' loads in flight across the barrier
// needs this narrower form.  The memory clobber keeps the compiler from
// moving LDS accesses across it.
// Raw (untyped, stride 0) buffer resource for the bytes [base, base + bytes):
// loads at offsets >= bytes return zeros.
__device__ __forceinline__ u32x4 buffer_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  return u32x4{uint32_t(b), uint32_t(b >> 32) & 0xffffu, bytes, 0x00020000u};
}

// The 32-bit range of a buffer resource over `bytes` bytes from its base.
// Ranges of 4 GiB or more are capped at 2^32 - 1: every offset a kernel
// issues against a resource is a tile's (far below 4 GiB), so only a range
// that ends within reach of those offsets must be exact, and it then is.
__device__ __forceinline__ uint32_t range32(int64_t bytes) {
  return bytes >= int64_t(0xffffffffu) ? 0xffffffffu : uint32_t(bytes);
}

// 16-byte buffer load whose completion the caller waits for explicitly with
// vm_wait<N>() followed by vm_ready() on the destination (the compiler does
// not track the load, so it neither drains nor reorders around it).
__device__ __forceinline__ void buffer_load16(u32x4& dst, const u32x4& rsrc, uint32_t voff) {
  asm volatile("buffer_load_dwordx4 %0, %1, %2, 0 offen" : "=v"(dst) : "v"(voff), "s"(rsrc) : "memory");
}

// Wait until at most N vector-memory operations of this wave are in flight
// (they complete in issue order).
template <int N>
__device__ __forceinline__ void vm_wait() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Marks a register as (re)defined here, so no use of it moves above the
// preceding vm_wait.
__device__ __forceinline__ void vm_ready(u32x4& v) { asm volatile("" : "+v"(v)); }

__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

}  // namespace avits

// Host-side error plumbing and launch timing (abi.hip).
namespace avits {
int set_error(int code, const char* fmt, ...);
int launch_status(const char* what);

// Brackets the launches made during its lifetime with timing events when
// timing is enabled (avits_timing_enable); a no-op otherwise.
class TimedLaunch {
 public:
  TimedLaunch(const char* family, hipStream_t stream);
  ~TimedLaunch();
  TimedLaunch(const TimedLaunch&) = delete;
  TimedLaunch& operator=(const TimedLaunch&) = delete;

 private:
  int family_;
  hipStream_t stream_;
  hipEvent_t start_ = nullptr;
};
}  // namespace avits

#define AVITS_REQUIRE(cond, ...)                                            \
  do {                                                                      \
    if (!(cond)) return ::avits::set_error(AVITS_ERR_INVALID_ARG, __VA_ARGS__); \
  } while (0)
