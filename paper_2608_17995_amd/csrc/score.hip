// Spatiotemporal importance (Section 3.3; Eqs. spatial, dit_attn, step_var,
// joint).
//
// Three launches on the caller's stream:
//  1. per (head h, image row i): the spatial partial
//       P[h, i] = sum_{j<L} exp(q_ih . k_jh / sqrt(d) - lse[h, i])
//     and, for bf16, the temporal partial over the head's channel slice
//       Q[h, i] = sum_{c in slice h} (f_t[i, c] - f_prev[i, c])^2
//     in one fused kernel (MFMA q.k^T with the feature stream overlapped);
//     fp32 runs the spatial partials on the VALU.
//  2. combine: A_i = mean_h P[h, i], V_i = sum_h Q[h, i] / (2 D_f) (fp32: the
//     variance is streamed here), plus one min/max partial of A and V per
//     workgroup.
//  3. finalize: every workgroup reduces the same partials (min and max are
//     exact in any order) and writes S for its slice of rows.
#include "common.h"
#include "select_block.h"

namespace avits {
namespace {

constexpr int kSpRows = 128;     // image rows per spatial workgroup (4 waves x 32)
constexpr int kSpKeys = 64;      // text keys per LDS tile
constexpr int kTmpBlocks = 512;  // max workgroups of the temporal pass
constexpr int kMaxScoreImages = 4096;  // images of one batched launch (grid y / z)
constexpr int kOneGroupMax = kThreads * kRegKeys;  // 16384: fused score + selection in one workgroup
constexpr float kLog2e = 1.4426950408889634f;

// ---------------------------------------------------------------------------
// 1. bf16: spatial partials on MFMA fused with the temporal partials.
//
// Workgroup = (128 image rows, head h), 4 waves x 32 rows.  Spatial part:
// S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (lane = one query row, 16 keys per
// 32-key sub-tile), text-key tiles of 64 double-buffered in LDS with the next
// tile prefetched into registers (one barrier per tile); exp2(logit - lse)
// summed per row.
// Temporal part: the workgroup streams channel slice [h D_f / H, (h+1) D_f / H)
// of both feature rows of its 128 rows, one (row, 16-byte chunk) pair per lane
// per key tile, software-pipelined: the pair consumed in tile t was loaded
// during tile t - 1, so the 2 N D_f-element stream is in flight while the
// MFMAs run; per-(head, row) partial sums of squared differences go to
// part_v.
template <int DH>
__global__ __launch_bounds__(256, 3) void spatial_temporal_bf16_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ ktxt, const float* __restrict__ lse,
    const bf16_t* __restrict__ ft, const bf16_t* __restrict__ fp, int N, int L, int H, int64_t Df,
    float* __restrict__ part_a, float* __restrict__ part_v) {
  constexpr int kC = DH / 16;                 // 16-wide head-dim chunks (MFMA k)
  constexpr int kLds = DH + 8;                // padded LDS row (bf16 elements)
  constexpr int kKP = kSpKeys * DH / 8 / 256; // 16-byte K pieces per thread per tile
  __shared__ __attribute__((aligned(16))) bf16_t ks[2][kSpKeys * kLds];

  // Workgroup b of an image's n = row blocks x heads runs on XCD b mod 8;
  // renumber so that each XCD takes a contiguous range of (head, row block)
  // ids, head-major: the row blocks of a head share one L2, which then
  // fetches that head's text keys once.
  int h, rb;
  {
    const int n_rb = int(gridDim.x), n = n_rb * int(gridDim.y);
    const int b = int(blockIdx.x) + n_rb * int(blockIdx.y);
    const int x = b % 8;
    int start = 0;
    for (int y = 0; y < x; ++y) start += (n - y + 7) / 8;
    const int u = start + b / 8;
    h = u / n_rb;
    rb = u % n_rb;
  }
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int l32 = lane % 32, hi = lane / 32;
  const int wrow0 = rb * kSpRows + wave * 32;  // this wave's 32 rows
  const int row = wrow0 + l32;
  const int64_t qstride = int64_t(H) * DH;
  {  // image blockIdx.z of a stack of equally shaped images
    const int64_t img = blockIdx.z;
    q += img * N * qstride;
    ktxt += img * L * qstride;
    lse += img * H * N;
    ft += img * N * Df;
    fp += img * N * Df;
    part_a += img * H * N;
    part_v += img * H * N;
  }

  // ---- temporal slice: lane pairs j = 0 .. npairs - 1 cover row
  // wrow0 + j rpi + lane / nch, chunk lane % nch (rpi = 64 / nch rows per
  // instruction). ----
  const int64_t c0 = Df * h / H, c1 = Df * (h + 1) / H;
  const int64_t nch = (c1 - c0) / 8;  // 16-byte chunks per row in the slice
  const bool vec = (c0 % 8 == 0) && ((c1 - c0) % 8 == 0) && nch > 0 && nch <= 64 && (64 % nch == 0);
  const int rpi = vec ? int(64 / nch) : 1;
  const int npairs = vec ? int(32 / rpi) : 0;
  const int r_in = vec ? lane / int(nch) : 0, cc = vec ? lane % int(nch) : 0;
  auto issue_pair = [&](int j, u32x4& x, u32x4& y) {
    x = u32x4{0u, 0u, 0u, 0u};
    y = x;
    const int rr = wrow0 + j * rpi + r_in;
    if (j < npairs && rr < N) {
      x = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(ft + int64_t(rr) * Df + c0 + 8 * cc));
      y = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(fp + int64_t(rr) * Df + c0 + 8 * cc));
    }
  };
  auto consume_pair = [&](int j, const u32x4& x, const u32x4& y) {
    if (j >= npairs) return;  // uniform across the wave
    float acc = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float d0 = __uint_as_float(x[e] << 16) - __uint_as_float(y[e] << 16);
      const float d1 = __uint_as_float(x[e] & 0xffff0000u) - __uint_as_float(y[e] & 0xffff0000u);
      acc = fmaf(d0, d0, fmaf(d1, d1, acc));
    }
    if (nch <= 16) {
      acc = group_sum(acc, int(nch));
    } else {
      for (int o = 1; o < nch; o <<= 1) acc += __shfl_xor(acc, o, kWave);
    }
    const int rr = wrow0 + j * rpi + r_in;
    if (cc == 0 && rr < N) part_v[int64_t(h) * N + rr] = acc;
  };
  u32x4 cx, cy;  // the feature pair of the current key tile

  // ---- spatial: Q^T fragments (B operand), lane = row l32, dims 16c + 8hi .. +7 ----
  // Each load reads 32 bytes from each of 32 rows, so the eight loads share
  // every cache line: plain loads, which keep the lines for the next ones (a
  // streaming hint here makes the query read markedly slower).
  bf16x8 qf[kC];
  {
    const bf16_t* src = q + int64_t(min(row, N - 1)) * qstride + int64_t(h) * DH + 8 * hi;
#pragma unroll
    for (int c = 0; c < kC; ++c) qf[c] = as_bf16x8(*reinterpret_cast<const u32x4*>(src + 16 * c));
  }
  const float lse2 = row < N ? lse[int64_t(h) * N + row] * kLog2e : 0.f;
  const float scale2 = kLog2e * rsqrtf(float(DH));
  float psum = 0.f;

  // Text keys: tile t + 2 is loaded into registers while tile t is
  // multiplied and stored to LDS at the end of tile t + 1 (two LDS buffers,
  // two register sets, one barrier per tile that waits for LDS only), so a
  // key load has two tiles of work to arrive in.
  auto load_k = [&](u32x4 (&kr)[kKP], int k0) {
#pragma unroll
    for (int j = 0; j < kKP; ++j) {
      const int p = tid + 256 * j, key = p / (DH / 8), col = (p % (DH / 8)) * 8;
      const int krow = min(k0 + key, L - 1);
      kr[j] = *reinterpret_cast<const u32x4*>(ktxt + (int64_t(krow) * H + h) * DH + col);
    }
  };
  auto store_k = [&](const u32x4 (&kr)[kKP], int buf) {
#pragma unroll
    for (int j = 0; j < kKP; ++j) {
      const int p = tid + 256 * j, key = p / (DH / 8), col = (p % (DH / 8)) * 8;
      *reinterpret_cast<u32x4*>(&ks[buf][key * kLds + col]) = kr[j];
    }
  };
  int jt = 0;  // key tiles done = temporal pairs consumed
  // The two 32-key sub-tiles of a tile are two independent MFMA chains,
  // both issued before any exp2, and four partial sums per lane break the
  // chain of adds.  acc[t][r] = logit of key 32t + 8(r/4) + 4hi + r%4
  // against this lane's row; exp2 is the hardware instruction (about 1 ulp;
  // terms below 2^-126 flush to zero); only the last tile masks keys past L.
  float ps[4] = {0.f, 0.f, 0.f, 0.f};
  static_assert(kSpKeys == 64, "two 32-key sub-tiles per tile");
  // One key tile from ks[buf] at k0; knext1 holds tile k0 + 64 (in flight),
  // knext2 receives tile k0 + 128.  The tile's feature pair is issued first
  // and consumed at the end of the tile.
  auto tile = [&](int buf, int k0, u32x4 (&knext2)[kKP], const u32x4 (&knext1)[kKP]) {
    issue_pair(jt, cx, cy);
    if (k0 + 2 * kSpKeys < L) load_k(knext2, k0 + 2 * kSpKeys);
    f32x16 acc[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;
#pragma unroll
    for (int c = 0; c < kC; ++c)
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const bf16x8 kf =
            as_bf16x8(*reinterpret_cast<const u32x4*>(&ks[buf][(32 * t + l32) * kLds + 16 * c + 8 * hi]));
        acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[c], acc[t], 0, 0, 0);
      }
    if (k0 + kSpKeys <= L) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) ps[r & 3] += __builtin_amdgcn_exp2f(fmaf(acc[t][r], scale2, -lse2));
    } else {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k0 + 32 * t + 8 * (r / 4) + 4 * hi + (r % 4);
          const float e = __builtin_amdgcn_exp2f(fmaf(acc[t][r], scale2, -lse2));
          ps[r & 3] += key < L ? e : 0.f;
        }
    }
    consume_pair(jt, cx, cy);
    ++jt;
    // The other buffer was last read one tile ago, before the barrier that
    // ended that tile, so it can be refilled now.  The barrier waits for
    // LDS only: the key loads in flight stay in flight.
    if (k0 + kSpKeys < L) store_k(knext1, buf ^ 1);
    lds_barrier();
  };
  u32x4 ka[kKP], kb[kKP];
  load_k(ka, 0);
  if (kSpKeys < L) load_k(kb, kSpKeys);
  store_k(ka, 0);
  __syncthreads();
  for (int k0 = 0; k0 < L; k0 += 2 * kSpKeys) {
    tile(0, k0, ka, kb);
    if (k0 + kSpKeys >= L) break;
    tile(1, k0 + kSpKeys, kb, ka);
  }
  psum = (ps[0] + ps[1]) + (ps[2] + ps[3]);
  psum = sum_xor32(psum);
  if (hi == 0 && row < N) part_a[int64_t(h) * N + row] = psum;
  // Pairs left when the slice has more pairs than there are key tiles:
  // issued in batches so their loads overlap instead of waiting one after
  // another.
  constexpr int kBatch = 8;
  while (jt < npairs) {
    u32x4 bx[kBatch], by[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) issue_pair(jt + u, bx[u], by[u]);
#pragma unroll
    for (int u = 0; u < kBatch; ++u) consume_pair(jt + u, bx[u], by[u]);
    jt += kBatch;
  }

  if (!vec) {
    for (int r = 0; r < 32; ++r) {
      const int rr = wrow0 + r;
      if (rr >= N) break;
      float acc = 0.f;
      for (int64_t c = c0 + lane; c < c1; c += kWave) {
        const float d0 = bf2f(ft[int64_t(rr) * Df + c]) - bf2f(fp[int64_t(rr) * Df + c]);
        acc = fmaf(d0, d0, acc);
      }
      acc = wave_sum(acc);
      if (lane == 0) part_v[int64_t(h) * N + rr] = acc;
    }
  }
}

// 1b. bf16: per row, A = mean_h part_a, V = sum_h part_v / (2 D_f), with
// every head's load in flight at once; one min/max partial of A and V per
// 64-row workgroup.
constexpr int kCombineHeads = 32;  // heads summed with every load issued up front

__global__ __launch_bounds__(64) void combine_kernel(const float* __restrict__ part_a,
                                                     const float* __restrict__ part_v, int64_t N, int H, int64_t Df,
                                                     float* __restrict__ a_out, float* __restrict__ v_out,
                                                     float4* __restrict__ mm) {
  const int64_t i = int64_t(blockIdx.x) * kWave + threadIdx.x;
  {  // image blockIdx.y: its partials, outputs and min/max slots
    const int64_t img = blockIdx.y;
    part_a += img * H * N;
    part_v += img * H * N;
    a_out += img * N;
    v_out += img * N;
    mm += img * gridDim.x;
  }
  float amin = INFINITY, amax = -INFINITY, vmin = INFINITY, vmax = -INFINITY;
  if (i < N) {
    float sa = 0.f, sv = 0.f;
    if (H <= kCombineHeads) {
      float pa[kCombineHeads], pv[kCombineHeads];
#pragma unroll
      for (int h = 0; h < kCombineHeads; ++h) {
        pa[h] = h < H ? part_a[int64_t(h) * N + i] : 0.f;
        pv[h] = h < H ? part_v[int64_t(h) * N + i] : 0.f;
      }
#pragma unroll
      for (int h = 0; h < kCombineHeads; ++h) {
        sa += pa[h];
        sv += pv[h];
      }
    } else {
      for (int h = 0; h < H; ++h) {
        sa += part_a[int64_t(h) * N + i];
        sv += part_v[int64_t(h) * N + i];
      }
    }
    const float A = sa / float(H), V = sv / (2.f * float(Df));
    a_out[i] = A;
    v_out[i] = V;
    amin = amax = A;
    vmin = vmax = V;
  }
  amin = wave_min(amin); amax = wave_max(amax);
  vmin = wave_min(vmin); vmax = wave_max(vmax);
  if (threadIdx.x == 0) mm[blockIdx.x] = make_float4(amin, amax, vmin, vmax);
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
  {  // image blockIdx.z
    const int64_t img = blockIdx.z;
    q += img * N * H * DH;
    ktxt += img * L * H * DH;
    lse += img * H * N;
    part += img * H * N;
  }
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
// 2'. fp32: temporal variance and head-mean of the spatial partials.
template <typename T>
__global__ __launch_bounds__(256) void temporal_kernel(const T* __restrict__ ft, const T* __restrict__ fp,
                                                       const float* __restrict__ part, int64_t N, int H,
                                                       int64_t Df, float* __restrict__ a_out,
                                                       float* __restrict__ v_out, float4* __restrict__ mm) {
  __shared__ float4 red[4];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t wstep = int64_t(gridDim.x) * 4;
  {  // image blockIdx.y
    const int64_t img = blockIdx.y;
    ft += img * N * Df;
    fp += img * N * Df;
    part += img * H * N;
    a_out += img * N;
    v_out += img * N;
    mm += img * gridDim.x;
  }
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
// 2''. From precomputed attention masses and N_T snapshots: A_i = sum_h
// mass[h, i] * inv (inv = 1 / (H * count) averages heads and the `count`
// accumulated probes), V_i = (1 / D_f) sum_c var_k(z[k, i, c]) with the
// unbiased variance over the N_T snapshots, formed from the deviations
// d_k = z_k - z_0 (sum d and sum d^2 in fp32; the shift keeps the sums small
// for slowly changing features).  One wave per row; per-workgroup min/max
// partials as temporal_kernel.
constexpr int kMaxSnapshots = 16;
struct Snapshots {
  const void* p[kMaxSnapshots];  // n_t device pointers, each [N, D_f]
};

template <typename T>
__global__ __launch_bounds__(256) void mass_temporal_kernel(const float* __restrict__ mass, int64_t mass_ld, int H,
                                                            float inv,
                                                            const Snapshots zs, int n_t, int64_t N, int64_t Df,
                                                            float* __restrict__ a_out, float* __restrict__ v_out,
                                                            float4* __restrict__ mm) {
  __shared__ float4 red[4];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t wstep = int64_t(gridDim.x) * 4;
  const float nt = float(n_t), inv_nm1 = 1.f / float(n_t - 1);
  float amin = INFINITY, amax = -INFINITY, vmin = INFINITY, vmax = -INFINITY;
  constexpr int kVec = 16 / sizeof(T);
  const bool vec = (Df % kVec) == 0;
  for (int64_t i = int64_t(blockIdx.x) * 4 + wave; i < N; i += wstep) {
    const T* z0 = static_cast<const T*>(zs.p[0]) + i * Df;
    float acc = 0.f;
    if (vec) {
      for (int64_t c = lane; c < Df / kVec; c += kWave) {
        float base[kVec], s1[kVec], s2[kVec];
        const u32x4 b = reinterpret_cast<const u32x4*>(z0)[c];
#pragma unroll
        for (int e = 0; e < kVec; ++e) {
          if constexpr (sizeof(T) == 2) base[e] = __uint_as_float(e % 2 ? b[e / 2] & 0xffff0000u : b[e / 2] << 16);
          else base[e] = __uint_as_float(b[e]);
          s1[e] = 0.f;
          s2[e] = 0.f;
        }
        for (int k = 1; k < n_t; ++k) {
          const u32x4 v = reinterpret_cast<const u32x4*>(static_cast<const T*>(zs.p[k]) + i * Df)[c];
#pragma unroll
          for (int e = 0; e < kVec; ++e) {
            float x;
            if constexpr (sizeof(T) == 2) x = __uint_as_float(e % 2 ? v[e / 2] & 0xffff0000u : v[e / 2] << 16);
            else x = __uint_as_float(v[e]);
            const float d = x - base[e];
            s1[e] += d;
            s2[e] = fmaf(d, d, s2[e]);
          }
        }
#pragma unroll
        for (int e = 0; e < kVec; ++e) acc += (s2[e] - s1[e] * s1[e] / nt) * inv_nm1;
      }
    } else {
      for (int64_t c = lane; c < Df; c += kWave) {
        const float b0 = ld(z0, c);
        float s1 = 0.f, s2 = 0.f;
        for (int k = 1; k < n_t; ++k) {
          const float d = ld(static_cast<const T*>(zs.p[k]) + i * Df, c) - b0;
          s1 += d;
          s2 = fmaf(d, d, s2);
        }
        acc += (s2 - s1 * s1 / nt) * inv_nm1;
      }
    }
    acc = wave_sum(acc);
    float ah = 0.f;
    for (int h = lane; h < H; h += kWave) ah += mass[int64_t(h) * mass_ld + i];
    ah = wave_sum(ah);
    const float A = ah * inv;
    const float V = acc / float(Df);
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
  {  // image blockIdx.y: its raw terms, min/max partials and scores
    const int64_t img = blockIdx.y;
    a += img * N;
    v += img * N;
    mm += img * n_mm;
    scores += img * N;
  }
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

// 3'. The fused score and the top-k selection in one workgroup (N <= 16384):
// the min/max partials reduced, each thread's consecutive scores computed
// (the arithmetic of finalize_kernel, so the scores are the same bits) and
// written, then selected from registers (Eq. topk, lowest-index ties).
__global__ __launch_bounds__(kThreads) void finalize_select_kernel(const float* __restrict__ a,
                                                                   const float* __restrict__ v,
                                                                   const float4* __restrict__ mm, int n_mm, int N,
                                                                   float alpha, float eps, float* __restrict__ scores,
                                                                   int k, int32_t* __restrict__ idx) {
  __shared__ float4 red[kWaves];
  float4 r = make_float4(INFINITY, -INFINITY, INFINITY, -INFINITY);
  for (int i = threadIdx.x; i < n_mm; i += kThreads) {
    const float4 m = mm[i];
    r.x = fminf(r.x, m.x); r.y = fmaxf(r.y, m.y); r.z = fminf(r.z, m.z); r.w = fmaxf(r.w, m.w);
  }
  r.x = wave_min(r.x); r.y = wave_max(r.y); r.z = wave_min(r.z); r.w = wave_max(r.w);
  if (threadIdx.x % kWave == 0) red[threadIdx.x / kWave] = r;
  __syncthreads();
  float4 t = red[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) {
    t.x = fminf(t.x, red[w].x); t.y = fmaxf(t.y, red[w].y); t.z = fminf(t.z, red[w].z); t.w = fmaxf(t.w, red[w].w);
  }
  const float ia = 1.f / (t.y - t.x + eps), iv = 1.f / (t.w - t.z + eps);
  const int q = (N + kThreads - 1) / kThreads;
  uint32_t keys[kRegKeys];
#pragma unroll
  for (int j = 0; j < kRegKeys; ++j) {
    const int i = int(threadIdx.x) * q + j;
    const bool live = j < q && i < N;
    const int ic = live ? i : 0;
    const float an = (a[ic] - t.x) * ia, vn = (v[ic] - t.z) * iv;
    const float sc = alpha * an + (1.f - alpha) * vn;
    if (live) scores[i] = sc;
    keys[j] = live ? order_key(sc) : 0u;
  }
  if (k > 0) select_block_keys(keys, N, k, idx);
}

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

struct ScoreWs {
  float* part;  // [H, N] spatial partials
  float* part_v;  // [H, N] temporal partials (bf16 path)
  float* a;     // [N]
  float* v;     // [N]
  float4* mm;   // min/max partials, one per combine workgroup
  size_t bytes;
};

// B images' buffers, image-major: part / part_v [B][H][N], a / v [B][N],
// mm [B][max(kTmpBlocks, ceil(N / 64))].
ScoreWs score_ws_layout(char* base, int64_t N, int32_t H, int64_t B = 1) {
  ScoreWs w;
  size_t off = 0;
  const size_t nb = size_t(N) * size_t(B);
  w.part = reinterpret_cast<float*>(base + off); off += align256(sizeof(float) * nb * H);
  w.part_v = reinterpret_cast<float*>(base + off); off += align256(sizeof(float) * nb * H);
  w.a = reinterpret_cast<float*>(base + off); off += align256(sizeof(float) * nb);
  w.v = reinterpret_cast<float*>(base + off); off += align256(sizeof(float) * nb);
  w.mm = reinterpret_cast<float4*>(base + off);
  off += align256(sizeof(float4) * size_t(B) * size_t(std::max<int64_t>(kTmpBlocks, (N + kWave - 1) / kWave)));
  w.bytes = off;
  return w;
}

// B >= 1 equally shaped images, stacked image-major; each is scored with
// its own min/max.  Every kernel takes the image from its last grid index.
int score_launch(const char* who, const void* latent_q, const void* text_k, const float* row_lse,
                 const void* feat_t, const void* feat_prev, int64_t B, int64_t N, int64_t L, int32_t H, int32_t d,
                 int64_t D_f, float alpha, float eps, int dtype, float* scores, float* a_raw, float* v_raw,
                 void* workspace, size_t workspace_bytes, void* stream, int64_t sel_k = -1,
                 int32_t* sel_idx = nullptr) {
  AVITS_REQUIRE(B >= 1 && B <= kMaxScoreImages, "%s: B=%lld images outside [1, %d]", who, (long long)B,
                kMaxScoreImages);
  AVITS_REQUIRE(N >= 1 && N <= INT32_MAX, "%s: N=%lld outside [1, 2^31)", who, (long long)N);
  AVITS_REQUIRE(L >= 1 && L <= INT32_MAX, "%s: L=%lld outside [1, 2^31)", who, (long long)L);
  AVITS_REQUIRE(H >= 1 && D_f >= 1, "%s: H=%d and D_f=%lld must be >= 1", who, H, (long long)D_f);
  AVITS_REQUIRE(alpha >= 0.f && alpha <= 1.f, "%s: alpha=%g outside [0, 1]", who, alpha);
  AVITS_REQUIRE(eps >= 0.f, "%s: eps=%g < 0", who, eps);
  if (d != 64 && d != 128) return set_error(AVITS_ERR_UNSUPPORTED, "%s: head dim %d (need 64 or 128)", who, d);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "%s: dtype %d unsupported", who, dtype);
  AVITS_REQUIRE(latent_q && text_k && row_lse && feat_t && feat_prev && scores, "%s: null input/output pointer",
                who);
  const ScoreWs need = score_ws_layout(nullptr, N, H, B);
  if (!workspace || workspace_bytes < need.bytes)
    return set_error(AVITS_ERR_WORKSPACE, "%s: workspace of %zu bytes, need %zu", who, workspace_bytes, need.bytes);
  ScoreWs ws = score_ws_layout(static_cast<char*>(workspace), N, H, B);
  float* a_dst = a_raw ? a_raw : ws.a;
  float* v_dst = v_raw ? v_raw : ws.v;
  hipStream_t s = static_cast<hipStream_t>(stream);

  const int n = int(N), l = int(L);
  const unsigned nimg = unsigned(B);
  int nmm;
  if (dtype == AVITS_BF16) {
    {
      TimedLaunch timed("score_spatial", s);
      const dim3 grid(unsigned((N + kSpRows - 1) / kSpRows), unsigned(H), nimg);
      if (d == 128)
        hipLaunchKernelGGL(spatial_temporal_bf16_kernel<128>, grid, dim3(256), 0, s, (const bf16_t*)latent_q,
                           (const bf16_t*)text_k, row_lse, (const bf16_t*)feat_t, (const bf16_t*)feat_prev, n, l, H,
                           D_f, ws.part, ws.part_v);
      else
        hipLaunchKernelGGL(spatial_temporal_bf16_kernel<64>, grid, dim3(256), 0, s, (const bf16_t*)latent_q,
                           (const bf16_t*)text_k, row_lse, (const bf16_t*)feat_t, (const bf16_t*)feat_prev, n, l, H,
                           D_f, ws.part, ws.part_v);
    }
    nmm = int((N + kWave - 1) / kWave);
    TimedLaunch timed("score_combine", s);
    hipLaunchKernelGGL(combine_kernel, dim3(nmm, nimg), dim3(kWave), 0, s, ws.part, ws.part_v, N, H, D_f, a_dst,
                       v_dst, ws.mm);
  } else {
    {
      TimedLaunch timed("score_spatial", s);
      const dim3 grid(unsigned((N + 127) / 128), unsigned(H), nimg);
      if (d == 128)
        hipLaunchKernelGGL(spatial_f32_kernel<128>, grid, dim3(128), 0, s, (const float*)latent_q,
                           (const float*)text_k, row_lse, n, l, H, ws.part);
      else
        hipLaunchKernelGGL(spatial_f32_kernel<64>, grid, dim3(128), 0, s, (const float*)latent_q,
                           (const float*)text_k, row_lse, n, l, H, ws.part);
    }
    nmm = int(std::min<int64_t>(kTmpBlocks, (N + 3) / 4));
    TimedLaunch timed("score_combine", s);
    hipLaunchKernelGGL(temporal_kernel<float>, dim3(nmm, nimg), dim3(256), 0, s, (const float*)feat_t,
                       (const float*)feat_prev, ws.part, N, H, D_f, a_dst, v_dst, ws.mm);
  }
  if (sel_k >= 0) {
    // One image, N <= kOneGroupMax: the score and the selection in one workgroup.
    TimedLaunch timed("score_finalize", s);
    hipLaunchKernelGGL(finalize_select_kernel, dim3(1), dim3(kThreads), 0, s, a_dst, v_dst, ws.mm, nmm, n, alpha,
                       eps, scores, int(sel_k), sel_idx);
    return launch_status(who);
  }
  const int fblocks = int(std::min<int64_t>(256, (N + 255) / 256));
  TimedLaunch timed("score_finalize", s);
  hipLaunchKernelGGL(finalize_kernel, dim3(fblocks, nimg), dim3(256), 0, s, a_dst, v_dst, ws.mm, nmm, N, alpha,
                     eps, scores);
  return launch_status(who);
}

}  // namespace
}  // namespace avits

using namespace avits;

extern "C" size_t avits_score_workspace_bytes(int64_t N, int32_t H) {
  if (N < 1 || H < 1) return 0;
  return score_ws_layout(nullptr, N, H).bytes;
}

extern "C" size_t avits_score_batched_workspace_bytes(int64_t B, int64_t N, int32_t H) {
  if (B < 1 || B > kMaxScoreImages || N < 1 || H < 1) return 0;
  return score_ws_layout(nullptr, N, H, B).bytes;
}

extern "C" int avits_score(const void* latent_q, const void* text_k, const float* row_lse, const void* feat_t,
                           const void* feat_prev, int64_t N, int64_t L, int32_t H, int32_t d, int64_t D_f,
                           float alpha, float eps, int dtype, float* scores, float* a_raw, float* v_raw,
                           void* workspace, size_t workspace_bytes, void* stream) {
  return score_launch("score", latent_q, text_k, row_lse, feat_t, feat_prev, 1, N, L, H, d, D_f, alpha, eps, dtype,
                      scores, a_raw, v_raw, workspace, workspace_bytes, stream);
}

extern "C" int avits_score_select(const void* latent_q, const void* text_k, const float* row_lse,
                                  const void* feat_t, const void* feat_prev, int64_t N, int64_t L, int32_t H,
                                  int32_t d, int64_t D_f, float alpha, float eps, int dtype, float* scores,
                                  float* a_raw, float* v_raw, int64_t k, int32_t* idx, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  AVITS_REQUIRE(N >= 1 && N <= kOneGroupMax, "score_select: N=%lld outside [1, %d] (use avits_score + avits_select)",
                (long long)N, kOneGroupMax);
  AVITS_REQUIRE(k >= 0 && k <= N, "score_select: k=%lld outside [0, N=%lld]", (long long)k, (long long)N);
  AVITS_REQUIRE(k == 0 || idx, "score_select: null idx");
  return score_launch("score_select", latent_q, text_k, row_lse, feat_t, feat_prev, 1, N, L, H, d, D_f, alpha, eps,
                      dtype, scores, a_raw, v_raw, workspace, workspace_bytes, stream, k, idx);
}

extern "C" int avits_score_batched(const void* latent_q, const void* text_k, const float* row_lse,
                                   const void* feat_t, const void* feat_prev, int64_t B, int64_t N, int64_t L,
                                   int32_t H, int32_t d, int64_t D_f, float alpha, float eps, int dtype,
                                   float* scores, float* a_raw, float* v_raw, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  return score_launch("score_batched", latent_q, text_k, row_lse, feat_t, feat_prev, B, N, L, H, d, D_f, alpha, eps,
                      dtype, scores, a_raw, v_raw, workspace, workspace_bytes, stream);
}

extern "C" int avits_score_from_mass(const float* mass, int64_t mass_ld, int32_t H, int32_t count,
                                     const void* const* snapshots,
                                     int32_t n_t,
                                     int64_t N, int64_t D_f, float alpha, float eps, int dtype, float* scores,
                                     float* a_raw, float* v_raw, void* workspace, size_t workspace_bytes,
                                     void* stream) {
  AVITS_REQUIRE(N >= 1 && N <= INT32_MAX, "score_from_mass: N=%lld outside [1, 2^31)", (long long)N);
  AVITS_REQUIRE(mass_ld >= N, "score_from_mass: mass_ld=%lld < N=%lld", (long long)mass_ld, (long long)N);
  AVITS_REQUIRE(H >= 1 && count >= 1 && D_f >= 1, "score_from_mass: H=%d count=%d D_f=%lld must be >= 1", H, count,
                (long long)D_f);
  AVITS_REQUIRE(n_t >= 2 && n_t <= kMaxSnapshots, "score_from_mass: n_t=%d snapshots outside [2, %d]", n_t,
                kMaxSnapshots);
  AVITS_REQUIRE(alpha >= 0.f && alpha <= 1.f, "score_from_mass: alpha=%g outside [0, 1]", alpha);
  AVITS_REQUIRE(eps >= 0.f, "score_from_mass: eps=%g < 0", eps);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "score_from_mass: dtype %d unsupported", dtype);
  AVITS_REQUIRE(mass && snapshots && scores, "score_from_mass: null input/output pointer");
  Snapshots zs{};
  for (int k = 0; k < n_t; ++k) {
    AVITS_REQUIRE(snapshots[k], "score_from_mass: snapshot %d is null", k);
    zs.p[k] = snapshots[k];
  }
  const ScoreWs need = score_ws_layout(nullptr, N, H);
  if (!workspace || workspace_bytes < need.bytes)
    return set_error(AVITS_ERR_WORKSPACE, "score_from_mass: workspace of %zu bytes, need %zu", workspace_bytes,
                     need.bytes);
  ScoreWs ws = score_ws_layout(static_cast<char*>(workspace), N, H);
  float* a_dst = a_raw ? a_raw : ws.a;
  float* v_dst = v_raw ? v_raw : ws.v;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int nmm = int(std::min<int64_t>(kTmpBlocks, (N + 3) / 4));
  const float inv = 1.f / (float(H) * float(count));
  {
    TimedLaunch timed("score_combine", s);
    if (dtype == AVITS_BF16)
      hipLaunchKernelGGL(mass_temporal_kernel<bf16_t>, dim3(nmm), dim3(256), 0, s, mass, mass_ld, H, inv, zs, n_t, N, D_f,
                         a_dst, v_dst, ws.mm);
    else
      hipLaunchKernelGGL(mass_temporal_kernel<float>, dim3(nmm), dim3(256), 0, s, mass, mass_ld, H, inv, zs, n_t, N, D_f,
                         a_dst, v_dst, ws.mm);
  }
  const int fblocks = int(std::min<int64_t>(256, (N + 255) / 256));
  TimedLaunch timed("score_finalize", s);
  hipLaunchKernelGGL(finalize_kernel, dim3(fblocks), dim3(256), 0, s, a_dst, v_dst, ws.mm, nmm, N, alpha, eps,
                     scores);
  return launch_status("score_from_mass");
}
