// Non-causal flash attention with log-sum-exp output (the joint attention of
// Section 3.3.1, Eqs. joint_qk and dit_attn), and its LSE-only form.
//
// bf16: one 256-thread workgroup per (128 query rows, head), 32 rows per
// wave.  Key tiles of 64 rows and the matching V^T tile are staged in padded
// LDS.  Both products run on v_mfma_f32_16x16x32_bf16 in transposed form:
//   S^T = K Q^T   -> each lane holds 4 keys x 1 query row (row = lane % 16),
//   O^T = V^T P^T -> each lane holds 4 head-dim values of the same row,
// so the online-softmax statistics of a row never leave its lane group, and
// the probabilities produced by the first product are, register for
// register, the B operand of the second (the contraction order over keys is
// the same permutation on both operands).  Softmax runs in the log2 domain
// with fp32 statistics.
// fp32: one thread per query row on the VALU (exactness path).
#include "kernels.h"

namespace avits {
namespace {

constexpr int kRows = 128;       // query rows per workgroup
constexpr int kKT = kAttnKeyTile; // keys per tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <int DH, bool WITH_V>
__global__ __launch_bounds__(256) void attn_bf16_kernel(const AttnArgs a) {
  constexpr int kC = DH / 32;       // head-dim chunks of 32
  constexpr int kKL = DH + 8;       // padded K row (elements)
  constexpr int kVL = kKT + 8;      // padded V^T row (elements)
  __shared__ __attribute__((aligned(16))) bf16_t Ks[kKT * kKL];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[WITH_V ? DH * kVL : 8];

  const int h = blockIdx.y;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int g = lane / 16, r16 = lane % 16;
  const int64_t row_base = int64_t(blockIdx.x) * kRows + wave * 32;
  const bf16_t* Q = static_cast<const bf16_t*>(a.q);
  const bf16_t* K = static_cast<const bf16_t*>(a.k);
  const bf16_t* VT = static_cast<const bf16_t*>(a.vt);

  bf16x8 qf[2][kC];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const int64_t row = row_base + 16 * rt + r16;
    const bf16_t* src = Q + row * a.q_tok + h * a.q_head + 8 * g;
#pragma unroll
    for (int c = 0; c < kC; ++c) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (row < a.Sq) v = *reinterpret_cast<const u32x4*>(src + 32 * c);
      qf[rt][c] = as_bf16x8(v);
    }
  }
  const float scale2 = kLog2e * rsqrtf(float(DH));
  float mrow[2] = {-INFINITY, -INFINITY};
  float lrow[2] = {0.f, 0.f};
  f32x4 oacc[2][WITH_V ? DH / 16 : 1];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int dt = 0; dt < (WITH_V ? DH / 16 : 1); ++dt) oacc[rt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int64_t k0 = 0; k0 < a.Sk; k0 += kKT) {
    __syncthreads();
    for (int p = tid; p < kKT * DH / 8; p += 256) {
      const int key = p / (DH / 8), col = (p % (DH / 8)) * 8;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (k0 + key < a.Sk) v = *reinterpret_cast<const u32x4*>(K + (k0 + key) * a.k_tok + h * a.k_head + col);
      *reinterpret_cast<u32x4*>(&Ks[key * kKL + col]) = v;
    }
    if constexpr (WITH_V) {
      const bf16_t* vsrc = VT + int64_t(h) * DH * a.ldvt + k0;
      for (int p = tid; p < DH * kKT / 8; p += 256) {
        const int dv = p / (kKT / 8), kc = (p % (kKT / 8)) * 8;
        *reinterpret_cast<u32x4*>(&Vs[dv * kVL + kc]) =
            *reinterpret_cast<const u32x4*>(vsrc + int64_t(dv) * a.ldvt + kc);
      }
    }
    __syncthreads();

    // Logits: s[rt][t][i] = q_row . k_(16t + 4g + i), log2-scaled.
    f32x4 s[2][kKT / 16];
#pragma unroll
    for (int t = 0; t < kKT / 16; ++t) {
      bf16x8 kf[kC];
#pragma unroll
      for (int c = 0; c < kC; ++c)
        kf[c] = as_bf16x8(*reinterpret_cast<const u32x4*>(&Ks[(16 * t + r16) * kKL + 32 * c + 8 * g]));
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < kC; ++c) acc = mfma16x16x32(kf[c], qf[rt][c], acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool valid = k0 + 16 * t + 4 * g + i < a.Sk;
          acc[i] = valid ? acc[i] * scale2 : -INFINITY;
        }
        s[rt][t] = acc;
      }
    }
    // Online softmax per row (the row's four lane groups share statistics).
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      float mx = -INFINITY;
#pragma unroll
      for (int t = 0; t < kKT / 16; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) mx = fmaxf(mx, s[rt][t][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
      mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
      const float mnew = fmaxf(mrow[rt], mx);
      const float corr = exp2f(mrow[rt] - mnew);
      mrow[rt] = mnew;
      float ls = 0.f;
#pragma unroll
      for (int t = 0; t < kKT / 16; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = exp2f(s[rt][t][i] - mnew);
          s[rt][t][i] = e;
          ls += e;
        }
      lrow[rt] = lrow[rt] * corr + ls;
      if constexpr (WITH_V) {
#pragma unroll
        for (int dt = 0; dt < DH / 16; ++dt) oacc[rt][dt] *= corr;
      }
    }
    if constexpr (WITH_V) {
      // P^T operand for key chunk c2: keys {32c2 + 4g + i} then {32c2 + 16 + 4g + i}.
      bf16x8 pf[2][2];
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int c2 = 0; c2 < 2; ++c2) {
          const f32x4 lo = s[rt][2 * c2], hi = s[rt][2 * c2 + 1];
          u32x4 v = {pack_bf2(lo[0], lo[1]), pack_bf2(lo[2], lo[3]), pack_bf2(hi[0], hi[1]), pack_bf2(hi[2], hi[3])};
          pf[rt][c2] = as_bf16x8(v);
        }
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt) {
#pragma unroll
        for (int c2 = 0; c2 < 2; ++c2) {
          const bf16_t* vr = &Vs[(16 * dt + r16) * kVL + 32 * c2 + 4 * g];
          const u32x2 lo = *reinterpret_cast<const u32x2*>(vr);
          const u32x2 hi = *reinterpret_cast<const u32x2*>(vr + 16);
          const u32x4 v = {lo[0], lo[1], hi[0], hi[1]};
          const bf16x8 vf = as_bf16x8(v);
#pragma unroll
          for (int rt = 0; rt < 2; ++rt) oacc[rt][dt] = mfma16x16x32(vf, pf[rt][c2], oacc[rt][dt]);
        }
      }
    }
  }

#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    float l = lrow[rt];
    l += __shfl_xor(l, 16, kWave);
    l += __shfl_xor(l, 32, kWave);
    const int64_t row = row_base + 16 * rt + r16;
    if (row >= a.Sq) continue;
    if (a.lse && g == 0) a.lse[int64_t(h) * a.Sq + row] = (mrow[rt] + log2f(l)) * kLn2;
    if constexpr (WITH_V) {
      const float inv = 1.f / l;
      bf16_t* dst = static_cast<bf16_t*>(a.o) + row * a.ldo + int64_t(h) * DH + 4 * g;
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt) {
        const f32x4 o = oacc[rt][dt];
        const u32x2 w = {pack_bf2(o[0] * inv, o[1] * inv), pack_bf2(o[2] * inv, o[3] * inv)};
        *reinterpret_cast<u32x2*>(dst + 16 * dt) = w;
      }
    }
  }
}

// fp32 VALU attention: one thread per query row, 32-key tiles in LDS.
constexpr int kFRows = 64, kFKT = 32;
template <int DH, bool WITH_V>
__global__ __launch_bounds__(kFRows) void attn_f32_kernel(const AttnArgs a) {
  __shared__ float Ks[kFKT * DH];
  __shared__ float Vs[WITH_V ? kFKT * DH : 1];
  const int h = blockIdx.y;
  const int64_t row = int64_t(blockIdx.x) * kFRows + threadIdx.x;
  const bool ok = row < a.Sq;
  const float* Q = static_cast<const float*>(a.q);
  const float* K = static_cast<const float*>(a.k);
  const float* VT = static_cast<const float*>(a.vt);
  float q[DH], o[WITH_V ? DH : 1];
#pragma unroll
  for (int c = 0; c < DH; ++c) q[c] = ok ? Q[row * a.q_tok + h * a.q_head + c] : 0.f;
#pragma unroll
  for (int c = 0; c < (WITH_V ? DH : 1); ++c) o[c] = 0.f;
  const float scale = rsqrtf(float(DH));
  float m = -INFINITY, l = 0.f;
  for (int64_t k0 = 0; k0 < a.Sk; k0 += kFKT) {
    __syncthreads();
    for (int p = threadIdx.x; p < kFKT * DH; p += kFRows) {
      const int key = p / DH, c = p % DH;
      const bool kv = k0 + key < a.Sk;
      Ks[p] = kv ? K[(k0 + key) * a.k_tok + h * a.k_head + c] : 0.f;
      if constexpr (WITH_V) Vs[p] = kv ? VT[(int64_t(h) * DH + c) * a.ldvt + k0 + key] : 0.f;
    }
    __syncthreads();
    const int nk = int(std::min<int64_t>(kFKT, a.Sk - k0));
    float s[kFKT];
    float mx = m;
    for (int j = 0; j < kFKT; ++j) {
      float acc = 0.f;
#pragma unroll
      for (int c = 0; c < DH; ++c) acc = fmaf(q[c], Ks[j * DH + c], acc);
      s[j] = j < nk ? acc * scale : -INFINITY;
      mx = fmaxf(mx, s[j]);
    }
    const float corr = expf(m - mx);
    m = mx;
    l *= corr;
    if constexpr (WITH_V) {
#pragma unroll
      for (int c = 0; c < DH; ++c) o[c] *= corr;
    }
    for (int j = 0; j < nk; ++j) {
      const float e = expf(s[j] - m);
      l += e;
      if constexpr (WITH_V) {
#pragma unroll
        for (int c = 0; c < DH; ++c) o[c] = fmaf(e, Vs[j * DH + c], o[c]);
      }
    }
  }
  if (!ok) return;
  if (a.lse) a.lse[int64_t(h) * a.Sq + row] = m + logf(l);
  if constexpr (WITH_V) {
    float* dst = static_cast<float*>(a.o) + row * a.ldo + int64_t(h) * DH;
#pragma unroll
    for (int c = 0; c < DH; ++c) dst[c] = o[c] / l;
  }
}

template <int DH>
void launch_dh(const AttnArgs& a, int dtype, hipStream_t s) {
  const bool with_v = a.vt != nullptr;
  if (dtype == AVITS_BF16) {
    const dim3 grid(unsigned(ceil_div64(a.Sq, kRows)), unsigned(a.H));
    if (with_v) hipLaunchKernelGGL((attn_bf16_kernel<DH, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((attn_bf16_kernel<DH, false>), grid, dim3(256), 0, s, a);
  } else {
    const dim3 grid(unsigned(ceil_div64(a.Sq, kFRows)), unsigned(a.H));
    if (with_v) hipLaunchKernelGGL((attn_f32_kernel<DH, true>), grid, dim3(kFRows), 0, s, a);
    else hipLaunchKernelGGL((attn_f32_kernel<DH, false>), grid, dim3(kFRows), 0, s, a);
  }
}

}  // namespace

int launch_attention(const AttnArgs& a, int dtype, hipStream_t s) {
  if (a.Sq == 0) return AVITS_OK;
  TimedLaunch timed(a.vt ? "attention" : "joint_lse", s);
  if (a.d == 128) launch_dh<128>(a, dtype, s);
  else launch_dh<64>(a, dtype, s);
  return launch_status("attention");
}

}  // namespace avits

using namespace avits;

extern "C" int avits_joint_lse(const void* q, const void* k_all, int64_t N, int64_t Nk, int32_t H, int32_t d,
                               int dtype, float* lse, void* stream) {
  AVITS_REQUIRE(N >= 1 && Nk >= 1 && H >= 1, "joint_lse: N=%lld Nk=%lld H=%d must be >= 1", (long long)N,
                (long long)Nk, H);
  if (d != 64 && d != 128) return set_error(AVITS_ERR_UNSUPPORTED, "joint_lse: head dim %d (need 64 or 128)", d);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "joint_lse: dtype %d unsupported", dtype);
  AVITS_REQUIRE(q && k_all && lse, "joint_lse: null pointer");
  AttnArgs a{};
  a.q = q;
  a.q_tok = int64_t(H) * d;
  a.q_head = d;
  a.k = k_all;
  a.k_tok = int64_t(H) * d;
  a.k_head = d;
  a.lse = lse;
  a.Sq = N;
  a.Sk = Nk;
  a.H = H;
  a.d = d;
  return launch_attention(a, dtype, static_cast<hipStream_t>(stream));
}
