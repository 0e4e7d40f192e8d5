// Spatiotemporal importance (Section 3.3; Eqs. spatial, dit_attn, step_var,
// joint).
//
// Three launches on the caller's stream:
//  1. spatial partials P[h, i] = sum_{j<L} exp(q_ih . k_jh / sqrt(d) - lse[h, i]).
//     bf16: one workgroup per (128 image rows, head); text keys staged through
//     LDS in 64-key tiles; q.k^T on v_mfma_f32_16x16x32_bf16 computed as
//     K Q^T so that each lane owns one query row and four keys, which keeps
//     the exp-and-sum in registers.  fp32: the same tiling on the VALU.
//  2. per row i: A_i = mean_h P[h, i], V_i = sum_c (f_t - f_prev)^2 / (2 D_f)
//     (one wavefront per row, streaming both feature rows), plus one min/max
//     partial of A and V per workgroup.
//  3. finalize: every workgroup reduces the same partials in the same order
//     (deterministic global min/max) and writes S for its slice of rows.
#include "common.h"

namespace avits {
namespace {

constexpr int kSpRows = 128;     // image rows per spatial workgroup (4 waves x 32)
constexpr int kSpKeys = 64;      // text keys per LDS tile
constexpr int kTmpBlocks = 512;  // max workgroups of the temporal pass
constexpr float kLog2e = 1.4426950408889634f;

// ---------------------------------------------------------------------------
// 1. spatial partials, bf16 MFMA.
template <int DH>
__global__ __launch_bounds__(256) void spatial_bf16_kernel(const bf16_t* __restrict__ q,
                                                           const bf16_t* __restrict__ ktxt,
                                                           const float* __restrict__ lse, int N, int L,
                                                           int H, float* __restrict__ part) {
  constexpr int kChunks = DH / 32;      // 32-wide slices of the head dim
  constexpr int kLds = DH + 8;          // padded LDS row (bf16 elements)
  __shared__ __attribute__((aligned(16))) bf16_t ks[kSpKeys * kLds];

  const int h = blockIdx.y;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int g = lane / 16, r16 = lane % 16;
  const int row_base = blockIdx.x * kSpRows + wave * 32;
  const int64_t qstride = int64_t(H) * DH;  // elements between consecutive tokens

  // Query fragments (B operand): lane holds row r16 of each 16-row tile,
  // head-dim elements 32c + 8g .. 32c + 8g + 7.
  bf16x8 qf[2][kChunks];
  float lse2[2];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const int row = row_base + rt * 16 + r16;
    const bool ok = row < N;
    const bf16_t* src = q + int64_t(row) * qstride + int64_t(h) * DH + 8 * g;
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (ok) v = *reinterpret_cast<const u32x4*>(src + 32 * c);
      qf[rt][c] = as_bf16x8(v);
    }
    lse2[rt] = ok ? lse[int64_t(h) * N + row] * kLog2e : 0.f;
  }
  const float scale2 = kLog2e * rsqrtf(float(DH));
  float acc_sum[2] = {0.f, 0.f};

  for (int k0 = 0; k0 < L; k0 += kSpKeys) {
    __syncthreads();
    // Stage 64 keys x DH into LDS (16-byte pieces), zero beyond L.
    constexpr int kPieces = kSpKeys * DH / 8;
    for (int p = threadIdx.x; p < kPieces; p += 256) {
      const int key = p / (DH / 8), col = (p % (DH / 8)) * 8;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (k0 + key < L) v = *reinterpret_cast<const u32x4*>(ktxt + (int64_t(k0 + key) * H + h) * DH + col);
      *reinterpret_cast<u32x4*>(&ks[key * kLds + col]) = v;
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < kSpKeys / 16; ++t) {
      bf16x8 kf[kChunks];
#pragma unroll
      for (int c = 0; c < kChunks; ++c)
        kf[c] = as_bf16x8(*reinterpret_cast<const u32x4*>(&ks[(16 * t + r16) * kLds + 32 * c + 8 * g]));
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < kChunks; ++c) s = mfma16x16x32(kf[c], qf[rt][c], s);
        // s[i] = logit of key 16t + 4g + i against this lane's row.
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = k0 + 16 * t + 4 * g + i;
          const float e = exp2f(s[i] * scale2 - lse2[rt]);
          acc_sum[rt] += key < L ? e : 0.f;
        }
      }
    }
  }
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    float v = acc_sum[rt];
    v += __shfl_xor(v, 16, kWave);
    v += __shfl_xor(v, 32, kWave);
    const int row = row_base + rt * 16 + r16;
    if (g == 0 && row < N) part[int64_t(h) * N + row] = v;
  }
}

// 1'. spatial partials, fp32 on the VALU: one thread per image row.
template <int DH>
__global__ __launch_bounds__(128) void spatial_f32_kernel(const float* __restrict__ q,
                                                          const float* __restrict__ ktxt,
                                                          const float* __restrict__ lse, int N, int L, int H,
                                                          float* __restrict__ part) {
  __shared__ float ks[kSpKeys * DH];
  const int h = blockIdx.y;
  const int row = blockIdx.x * 128 + threadIdx.x;
  const bool ok = row < N;
  float qr[DH];
#pragma unroll
  for (int c = 0; c < DH; ++c) qr[c] = ok ? q[(int64_t(row) * H + h) * DH + c] : 0.f;
  const float l = ok ? lse[int64_t(h) * N + row] : 0.f;
  const float scale = rsqrtf(float(DH));
  float acc = 0.f;
  for (int k0 = 0; k0 < L; k0 += kSpKeys) {
    __syncthreads();
    for (int p = threadIdx.x; p < kSpKeys * DH; p += 128) {
      const int key = p / DH, c = p % DH;
      ks[p] = k0 + key < L ? ktxt[(int64_t(k0 + key) * H + h) * DH + c] : 0.f;
    }
    __syncthreads();
    const int nk = min(kSpKeys, L - k0);
    for (int j = 0; j < nk; ++j) {
      float s = 0.f;
#pragma unroll
      for (int c = 0; c < DH; ++c) s = fmaf(qr[c], ks[j * DH + c], s);
      acc += expf(s * scale - l);
    }
  }
  if (ok) part[int64_t(h) * N + row] = acc;
}

// ---------------------------------------------------------------------------
// 2. temporal variance and head-mean of the spatial partials.
template <typename T>
__global__ __launch_bounds__(256) void temporal_kernel(const T* __restrict__ ft, const T* __restrict__ fp,
                                                       const float* __restrict__ part, int64_t N, int H,
                                                       int64_t Df, float* __restrict__ a_out,
                                                       float* __restrict__ v_out, float4* __restrict__ mm) {
  __shared__ float4 red[4];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t wstep = int64_t(gridDim.x) * 4;
  float amin = INFINITY, amax = -INFINITY, vmin = INFINITY, vmax = -INFINITY;
  constexpr int kVec = 16 / sizeof(T);
  const bool vec = (Df % kVec) == 0;
  for (int64_t i = int64_t(blockIdx.x) * 4 + wave; i < N; i += wstep) {
    const T* a = ft + i * Df;
    const T* b = fp + i * Df;
    float s = 0.f;
    if (vec) {
      const u32x4* av = reinterpret_cast<const u32x4*>(a);
      const u32x4* bv = reinterpret_cast<const u32x4*>(b);
      for (int64_t c = lane; c < Df / kVec; c += kWave) {
        const u32x4 x = av[c], y = bv[c];
        if constexpr (sizeof(T) == 2) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float d0 = __uint_as_float(x[e] << 16) - __uint_as_float(y[e] << 16);
            const float d1 = __uint_as_float(x[e] & 0xffff0000u) - __uint_as_float(y[e] & 0xffff0000u);
            s = fmaf(d0, d0, s);
            s = fmaf(d1, d1, s);
          }
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float d0 = __uint_as_float(x[e]) - __uint_as_float(y[e]);
            s = fmaf(d0, d0, s);
          }
        }
      }
    } else {
      for (int64_t c = lane; c < Df; c += kWave) {
        const float d0 = ld(a, c) - ld(b, c);
        s = fmaf(d0, d0, s);
      }
    }
    s = wave_sum(s);
    float ah = 0.f;
    for (int h = lane; h < H; h += kWave) ah += part[int64_t(h) * N + i];
    ah = wave_sum(ah);
    const float A = ah / float(H);
    const float V = s / (2.f * float(Df));
    if (lane == 0) {
      a_out[i] = A;
      v_out[i] = V;
    }
    amin = fminf(amin, A); amax = fmaxf(amax, A);
    vmin = fminf(vmin, V); vmax = fmaxf(vmax, V);
  }
  if (lane == 0) red[wave] = make_float4(amin, amax, vmin, vmax);
  __syncthreads();
  if (threadIdx.x == 0) {
    float4 r = red[0];
    for (int w = 1; w < 4; ++w) {
      r.x = fminf(r.x, red[w].x); r.y = fmaxf(r.y, red[w].y);
      r.z = fminf(r.z, red[w].z); r.w = fmaxf(r.w, red[w].w);
    }
    mm[blockIdx.x] = r;
  }
}

// ---------------------------------------------------------------------------
// 3. global min/max and the fused score.
__global__ __launch_bounds__(256) void finalize_kernel(const float* __restrict__ a, const float* __restrict__ v,
                                                       const float4* __restrict__ mm, int n_mm, int64_t N,
                                                       float alpha, float eps, float* __restrict__ scores) {
  __shared__ float4 red[256];
  float4 r = make_float4(INFINITY, -INFINITY, INFINITY, -INFINITY);
  for (int i = threadIdx.x; i < n_mm; i += 256) {
    const float4 m = mm[i];
    r.x = fminf(r.x, m.x); r.y = fmaxf(r.y, m.y); r.z = fminf(r.z, m.z); r.w = fmaxf(r.w, m.w);
  }
  red[threadIdx.x] = r;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s) {
      const float4 o = red[threadIdx.x + s];
      float4 m = red[threadIdx.x];
      m.x = fminf(m.x, o.x); m.y = fmaxf(m.y, o.y); m.z = fminf(m.z, o.z); m.w = fmaxf(m.w, o.w);
      red[threadIdx.x] = m;
    }
    __syncthreads();
  }
  const float4 t = red[0];
  const float ia = 1.f / (t.y - t.x + eps), iv = 1.f / (t.w - t.z + eps);
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < N; i += int64_t(gridDim.x) * 256) {
    const float an = (a[i] - t.x) * ia, vn = (v[i] - t.z) * iv;
    scores[i] = alpha * an + (1.f - alpha) * vn;
  }
}

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

struct ScoreWs {
  float* part;  // [H, N]
  float* a;     // [N]
  float* v;     // [N]
  float4* mm;   // [kTmpBlocks]
  size_t bytes;
};

ScoreWs score_ws_layout(char* base, int64_t N, int32_t H) {
  ScoreWs w;
  size_t off = 0;
  w.part = reinterpret_cast<float*>(base + off); off += align256(sizeof(float) * size_t(N) * H);
  w.a = reinterpret_cast<float*>(base + off); off += align256(sizeof(float) * size_t(N));
  w.v = reinterpret_cast<float*>(base + off); off += align256(sizeof(float) * size_t(N));
  w.mm = reinterpret_cast<float4*>(base + off); off += align256(sizeof(float4) * kTmpBlocks);
  w.bytes = off;
  return w;
}

}  // namespace
}  // namespace avits

using namespace avits;

extern "C" size_t avits_score_workspace_bytes(int64_t N, int32_t H) {
  if (N < 1 || H < 1) return 0;
  return score_ws_layout(nullptr, N, H).bytes;
}

extern "C" int avits_score(const void* latent_q, const void* text_k, const float* row_lse, const void* feat_t,
                           const void* feat_prev, int64_t N, int64_t L, int32_t H, int32_t d, int64_t D_f,
                           float alpha, float eps, int dtype, float* scores, float* a_raw, float* v_raw,
                           void* workspace, size_t workspace_bytes, void* stream) {
  AVITS_REQUIRE(N >= 1 && N <= INT32_MAX, "score: N=%lld outside [1, 2^31)", (long long)N);
  AVITS_REQUIRE(L >= 1 && L <= INT32_MAX, "score: L=%lld outside [1, 2^31)", (long long)L);
  AVITS_REQUIRE(H >= 1 && D_f >= 1, "score: H=%d and D_f=%lld must be >= 1", H, (long long)D_f);
  AVITS_REQUIRE(alpha >= 0.f && alpha <= 1.f, "score: alpha=%g outside [0, 1]", alpha);
  AVITS_REQUIRE(eps >= 0.f, "score: eps=%g < 0", eps);
  if (d != 64 && d != 128) return set_error(AVITS_ERR_UNSUPPORTED, "score: head dim %d (need 64 or 128)", d);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "score: dtype %d unsupported", dtype);
  AVITS_REQUIRE(latent_q && text_k && row_lse && feat_t && feat_prev && scores, "score: null input/output pointer");
  const ScoreWs need = score_ws_layout(nullptr, N, H);
  if (!workspace || workspace_bytes < need.bytes)
    return set_error(AVITS_ERR_WORKSPACE, "score: workspace of %zu bytes, need %zu", workspace_bytes, need.bytes);
  ScoreWs ws = score_ws_layout(static_cast<char*>(workspace), N, H);
  float* a_dst = a_raw ? a_raw : ws.a;
  float* v_dst = v_raw ? v_raw : ws.v;
  hipStream_t s = static_cast<hipStream_t>(stream);

  const int n = int(N), l = int(L);
  {
  TimedLaunch timed("score_spatial", s);
  if (dtype == AVITS_BF16) {
    const dim3 grid(unsigned((N + kSpRows - 1) / kSpRows), unsigned(H));
    if (d == 128)
      hipLaunchKernelGGL(spatial_bf16_kernel<128>, grid, dim3(256), 0, s, (const bf16_t*)latent_q,
                         (const bf16_t*)text_k, row_lse, n, l, H, ws.part);
    else
      hipLaunchKernelGGL(spatial_bf16_kernel<64>, grid, dim3(256), 0, s, (const bf16_t*)latent_q,
                         (const bf16_t*)text_k, row_lse, n, l, H, ws.part);
  } else {
    const dim3 grid(unsigned((N + 127) / 128), unsigned(H));
    if (d == 128)
      hipLaunchKernelGGL(spatial_f32_kernel<128>, grid, dim3(128), 0, s, (const float*)latent_q,
                         (const float*)text_k, row_lse, n, l, H, ws.part);
    else
      hipLaunchKernelGGL(spatial_f32_kernel<64>, grid, dim3(128), 0, s, (const float*)latent_q,
                         (const float*)text_k, row_lse, n, l, H, ws.part);
  }
  }
  const int tblocks = int(std::min<int64_t>(kTmpBlocks, (N + 3) / 4));
  {
  TimedLaunch timed("score_temporal", s);
  if (dtype == AVITS_BF16)
    hipLaunchKernelGGL(temporal_kernel<bf16_t>, dim3(tblocks), dim3(256), 0, s, (const bf16_t*)feat_t,
                       (const bf16_t*)feat_prev, ws.part, N, H, D_f, a_dst, v_dst, ws.mm);
  else
    hipLaunchKernelGGL(temporal_kernel<float>, dim3(tblocks), dim3(256), 0, s, (const float*)feat_t,
                       (const float*)feat_prev, ws.part, N, H, D_f, a_dst, v_dst, ws.mm);
  }
  const int fblocks = int(std::min<int64_t>(256, (N + 255) / 256));
  TimedLaunch timed("score_finalize", s);
  hipLaunchKernelGGL(finalize_kernel, dim3(fblocks), dim3(256), 0, s, a_dst, v_dst, ws.mm, tblocks, N, alpha, eps,
                     scores);
  return launch_status("score");
}
