// Non-causal flash attention with log-sum-exp output (the joint attention of
// Section 3.3.1, Eqs. joint_qk and dit_attn), and its LSE-only form.
//
// bf16: one 256-thread workgroup per (128 query rows, head), 32 rows per
// wave, two workgroups per CU, the row blocks of one head on one XCD.  Key
// tiles of 64 rows and the matching V^T tile are prefetched into registers
// one tile ahead and staged in padded LDS.
// Both products run on v_mfma_f32_32x32x16_bf16 in transposed form:
//   S^T = K Q^T   -> each lane holds 16 keys x 1 query row (row = lane % 32),
//   O^T = V^T P^T -> each lane holds 16 head-dim values of the same row,
// so a row's online-softmax statistics live in two lanes (l, l ^ 32), and the
// probabilities produced by the first product are, register for register,
// the B operand of the second (the contraction over keys uses the same key
// permutation on both operands).  Softmax runs in the log2 domain with fp32
// statistics.
// Load balance: 128-row units of one head each take one of the two workgroup
// slots of a CU, so a grid that overruns the first slot of every CU by a few
// units leaves most CUs with one unit and some with two.  The launcher then
// splits the overrun units (or, for small grids, every unit) along the keys:
// each piece writes its unnormalised output and (max, sum) per row, and a
// combine kernel merges the pieces in key order.
// fp32: one thread per query row on the VALU (exactness path).
#include <stdio.h>
#include <stdlib.h>

#include <type_traits>

#include "kernels.h"

namespace avits {
namespace {

constexpr int kRows = 128;        // query rows per workgroup (4 waves x 32)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// One workgroup's work: a head, its query rows [q_lo, q_hi) and up to two key
// ranges [ks[r], ks[r] + kn[r]).
struct AttnUnit {
  int h;
  int64_t q_lo, q_hi;
  int64_t ks[2], kn[2];
};

// Number of row blocks of `rows` query rows per head.
__host__ __device__ inline int64_t attn_row_blocks(const AttnArgs& a, int rows) {
  if (a.segs.n == 0) return (a.Sq + rows - 1) / rows;
  int64_t v = 0;
#pragma unroll
  for (int b = 0; b < kMaxSeqs; ++b)  // static indices: no private copy of the arguments
#pragma unroll
    for (int r = 0; r < 2; ++r) v += b < a.segs.n ? (a.segs.len[b][r] + rows - 1) / rows : 0;
  return v;
}

// Workgroup b of a class of n runs on XCD b mod 8: renumber so that each
// XCD takes a contiguous range of the class's logical ids.
__device__ __forceinline__ int64_t attn_xcd_id(int64_t b, int64_t n) {
  const int64_t x = b % 8;
  int64_t start = 0;
  for (int64_t y = 0; y < x; ++y) start += (n - y + 7) / 8;
  return start + b / 8;
}

// Unit u -> its head, query rows [q_lo, q_hi) and key ranges.  With
// sequences, the row blocks of a head enumerate each sequence's two row
// ranges in turn, and the keys are that sequence's rows.
__device__ __forceinline__ AttnUnit attn_decode(const AttnArgs& a, int rows, int64_t u) {
  const int64_t n_rb = attn_row_blocks(a, rows);
  AttnUnit w;
  w.h = int(u / n_rb);
  int64_t rb = u % n_rb;
  if (a.segs.n == 0) {
    w.q_lo = rb * rows;
    w.q_hi = std::min<int64_t>(a.Sq, w.q_lo + rows);
    w.ks[0] = 0; w.kn[0] = a.Sk;
    w.ks[1] = 0; w.kn[1] = 0;
    return w;
  }
  // Static indices throughout (a dynamically indexed argument array would be
  // copied to private memory).
  w.q_lo = w.q_hi = 0;
  w.ks[0] = w.ks[1] = 0;
  w.kn[0] = w.kn[1] = 0;
  bool found = false;
#pragma unroll
  for (int b = 0; b < kMaxSeqs; ++b) {
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int64_t nb = b < a.segs.n ? (a.segs.len[b][r] + rows - 1) / rows : 0;
      if (!found && rb < nb) {
        found = true;
        w.q_lo = a.segs.start[b][r] + rb * rows;
        w.q_hi = std::min<int64_t>(a.segs.start[b][r] + a.segs.len[b][r], w.q_lo + rows);
        w.ks[0] = a.segs.start[b][0];
        w.kn[0] = a.segs.len[b][0];
        w.ks[1] = a.segs.start[b][1];
        w.kn[1] = a.segs.len[b][1];
      }
      if (!found) rb -= nb;
    }
  }
  return w;  // every unit of the grid (n_rb * H of them) finds its range
}

// Workgroup -> unit, with the units of one XCD contiguous and head-major, so
// the row blocks of a head share one L2.  Split tail: units below split_from
// take workgroups 0 .. split_from - 1; each later unit runs in ksp pieces
// (workgroups split_from onwards, dispatched after the whole units), piece p
// over key tiles [T p / ksp, T (p + 1) / ksp) of the unit's T key tiles (the
// tiles of its first key range, then of its second); `piece` is the piece's
// slot in the partial buffer (-1 for a whole unit).
__device__ __forceinline__ AttnUnit attn_unit(const AttnArgs& a, int rows, int64_t& piece) {
  const int64_t U = attn_row_blocks(a, rows) * a.H;
  const int64_t bid = blockIdx.x;
  int64_t u;
  int p = 0;
  piece = -1;
  if (bid < a.split_from) {
    u = attn_xcd_id(bid, std::min<int64_t>(a.split_from, U));
  } else {
    const int64_t v = attn_xcd_id(bid - a.split_from, int64_t(gridDim.x) - a.split_from);
    u = a.split_from + v / a.ksp;
    p = int(v % a.ksp);
    piece = v;
  }
  AttnUnit w = attn_decode(a, rows, u);
  if (piece >= 0) {
    const int64_t t0 = (w.kn[0] + 63) / 64, T = t0 + (w.kn[1] + 63) / 64;
    const int64_t t_lo = T * p / a.ksp, t_hi = T * (p + 1) / a.ksp;
    // The piece's share of each range (either may be empty).
    const int64_t a0 = std::min(t_lo, t0), b0 = std::min(t_hi, t0);
    const int64_t a1 = std::max(t_lo, t0) - t0, b1 = std::max(t_hi, t0) - t0;
    const int64_t n0 = std::max<int64_t>(0, std::min<int64_t>(w.kn[0], 64 * b0) - 64 * a0);
    const int64_t n1 = std::max<int64_t>(0, std::min<int64_t>(w.kn[1], 64 * b1) - 64 * a1);
    w.ks[0] += 64 * a0;
    w.kn[0] = n0;
    w.ks[1] += 64 * a1;
    w.kn[1] = n1;
  }
  return w;
}

// Lane l of a 32x32 MFMA output tile holds row 8*(r/4) + 4*(l/32) + r%4 of
// column l%32 in register r.  With S^T = K Q^T the column is the query row
// and the row is the LDS key row.  Key rows are stored in LDS with bits 2 and
// 3 of their index within the tile swapped, so register r of lane half h
// holds key 16*(r/8) + 8h + 4*((r/4)%2) + r%4 of its 32-key sub-tile: for
// the 16-key chunk c of the P^T operand, lane half h then holds the
// contiguous keys 16c + 8h .. +7, and each V^T operand is a single 16-byte
// LDS read (V^T rows padded to a 16-byte multiple).  The last, partial key
// tile runs through its own instance of the tile body (key masking, V^T
// zeroing), so full tiles carry no tail arithmetic; the text-mass sum is
// compiled in only when MASS is set.
template <int DH, bool WITH_V, bool MASS>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(const AttnArgs a) {
  constexpr int NW = kRows / 32;             // waves
  constexpr int kKT = 64;                    // keys per tile
  constexpr int kT = 64 * NW;                // threads
  constexpr int kC = DH / 16;
  constexpr int kKL = DH + 8;                // padded K row (elements), 16-byte multiple
  constexpr int kVL = kKT + 8;               // padded V^T row (elements), 16-byte multiple
  constexpr int kKP = kKT * DH / 8 / kT;     // 16-byte K pieces per thread per tile
  constexpr int kVP = DH * kKT / 8 / kT;     // 16-byte V^T pieces per thread per tile
  static_assert(kKP >= 1 && kVP >= 1, "tile too small for the workgroup");
  __shared__ __attribute__((aligned(16))) bf16_t Ks[2][kKT * kKL];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[2][WITH_V ? DH * kVL : 8];

  int64_t piece;
  const AttnUnit un = attn_unit(a, 32 * NW, piece);
  const int h = un.h;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int l32 = lane % 32, hi = lane / 32;
  const int64_t row = un.q_lo + wave * 32 + l32;
  const bf16_t* Q = static_cast<const bf16_t*>(a.q);
  const bf16_t* K = static_cast<const bf16_t*>(a.k) + int64_t(h) * a.k_head;
  const bf16_t* VT = static_cast<const bf16_t*>(a.vt) + int64_t(h) * DH * a.ldvt;

  bf16x8 qf[kC];
  {
    const bf16_t* src = Q + std::min<int64_t>(row, un.q_hi - 1) * a.q_tok + h * a.q_head + 8 * hi;
#pragma unroll
    for (int c = 0; c < kC; ++c) qf[c] = as_bf16x8(*reinterpret_cast<const u32x4*>(src + 16 * c));
  }
  const float scale2 = kLog2e * rsqrtf(float(DH));
  float mrow = -INFINITY, lrow = 0.f, trow = 0.f;
  f32x16 oacc[WITH_V ? DH / 32 : 1];
#pragma unroll
  for (int dt = 0; dt < (WITH_V ? DH / 32 : 1); ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[dt][r] = 0.f;

  // Per-thread piece coordinates (fixed over the tiles).
  int k_key[kKP], k_dst[kKP], v_dv[kVP], v_kc[kVP];
  const bf16_t* k_src[kKP];
  const bf16_t* v_src[kVP];
#pragma unroll
  for (int j = 0; j < kKP; ++j) {
    const int p = tid + kT * j;
    const int kk = p / (DH / 8), col = (p % (DH / 8)) * 8;
    k_key[j] = kk;
    const int rowp = (kk & ~12) | ((kk & 4) << 1) | ((kk & 8) >> 1);
    k_dst[j] = rowp * kKL + col;
    k_src[j] = K + int64_t(kk) * a.k_tok + col;
  }
#pragma unroll
  for (int j = 0; j < kVP; ++j) {
    const int p = tid + kT * j;
    v_dv[j] = p / (kKT / 8);
    v_kc[j] = (p % (kKT / 8)) * 8;
    v_src[j] = VT + int64_t(v_dv[j]) * a.ldvt + v_kc[j];
  }
  // Register prefetch of the next tile.
  u32x4 kreg[kKP], vreg[WITH_V ? kVP : 1];
  // Tile of key rows k0 .. k0 + rem - 1 (rem < kKT: the partial tile at the
  // end of a key range).
  auto load_tile = [&](int64_t k0, int rem) {
    if (rem == kKT) {
#pragma unroll
      for (int j = 0; j < kKP; ++j) kreg[j] = *reinterpret_cast<const u32x4*>(k_src[j] + k0 * a.k_tok);
      if constexpr (WITH_V) {
#pragma unroll
        for (int j = 0; j < kVP; ++j) vreg[j] = *reinterpret_cast<const u32x4*>(v_src[j] + k0);
      }
    } else {
      // Clamp key rows; zero V^T beyond the end so that 0-probability keys
      // contribute exactly 0.
#pragma unroll
      for (int j = 0; j < kKP; ++j) {
        const int kk = std::min(k_key[j], rem - 1);
        kreg[j] = *reinterpret_cast<const u32x4*>(k_src[j] + (k0 + kk - k_key[j]) * a.k_tok);
      }
      if constexpr (WITH_V) {
#pragma unroll
        for (int j = 0; j < kVP; ++j) {
          vreg[j] = *reinterpret_cast<const u32x4*>(v_src[j] + k0);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int kk = v_kc[j] + 2 * e;
            vreg[j][e] = (kk < rem ? vreg[j][e] & 0xffffu : 0u) | (kk + 1 < rem ? vreg[j][e] & 0xffff0000u : 0u);
          }
        }
      }
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int j = 0; j < kKP; ++j) *reinterpret_cast<u32x4*>(&Ks[buf][k_dst[j]]) = kreg[j];
    if constexpr (WITH_V) {
#pragma unroll
      for (int j = 0; j < kVP; ++j) *reinterpret_cast<u32x4*>(&Vs[buf][v_dv[j] * kVL + v_kc[j]]) = vreg[j];
    }
  };
  // Key (within the tile) of accumulator register r of sub-tile t, less 8 h.
  auto key_of = [](int t, int r) { return 32 * t + 16 * (r / 8) + 4 * ((r / 4) & 1) + (r % 4); };

  // Key tiles: ceil(kn[0] / kKT) over the first range, then the second's.
  const int64_t t0 = (un.kn[0] + kKT - 1) / kKT;
  const int64_t n_tiles = t0 + (un.kn[1] + kKT - 1) / kKT;
  auto tile_at = [&](int64_t it, int64_t& base, int& rem) {
    const bool first = it < t0;  // selects, not a dynamic index into un.ks / un.kn
    const int64_t local = (first ? it : it - t0) * kKT;
    base = (first ? un.ks[0] : un.ks[1]) + local;
    rem = int(std::min<int64_t>(kKT, (first ? un.kn[0] : un.kn[1]) - local));
  };
  int buf = 0;
  // Key tile `it` (rows k0 .. k0 + rem - 1; its key index within a range
  // starting at 0 is k0 - ks[0] for the text-mass test): prefetch tile it + 1
  // into registers, consume tile it from LDS, stage tile it + 1 in the other
  // LDS buffer.
  auto tile = [&](int64_t it, int64_t k0, int rem, auto tail_tag) {
    constexpr bool kTail = decltype(tail_tag)::value;
    const bool more = it + 1 < n_tiles;
    if (more) {
      int64_t nb;
      int nr;
      tile_at(it + 1, nb, nr);
      load_tile(nb, nr);
    }

    f32x16 s[kKT / 32];
#pragma unroll
    for (int t = 0; t < kKT / 32; ++t) {
      f32x16 acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
      for (int c = 0; c < kC; ++c) {
        const bf16x8 kf = as_bf16x8(*reinterpret_cast<const u32x4*>(&Ks[buf][(32 * t + l32) * kKL + 16 * c + 8 * hi]));
        acc = mfma32(kf, qf[c], acc);
      }
      s[t] = acc;
    }
    if constexpr (kTail) {
      const int lim = rem - 8 * hi;
#pragma unroll
      for (int t = 0; t < kKT / 32; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (key_of(t, r) >= lim) s[t][r] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < kKT / 32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[t][r]);
    mx = max_xor32(mx) * scale2;
    const bool raise = mx > mrow + 8.f;
    float corr = 1.f;
    if (raise) {
      corr = __builtin_amdgcn_exp2f(mrow - mx);
      mrow = mx;
    }
    float ls = 0.f;
#pragma unroll
    for (int t = 0; t < kKT / 32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = __builtin_amdgcn_exp2f(fmaf(s[t][r], scale2, -mrow));
        s[t][r] = e;
        ls += e;
      }
    lrow = lrow * corr + ls;
    if constexpr (MASS) {
      if (k0 < a.mass_keys) {
        float ts = ls;
        if (k0 + kKT > a.mass_keys) {
          ts = 0.f;
          const int lim = int(a.mass_keys - k0) - 8 * hi;
#pragma unroll
          for (int t = 0; t < kKT / 32; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) ts += key_of(t, r) < lim ? s[t][r] : 0.f;
        }
        trow = trow * corr + ts;
      } else {
        trow *= corr;
      }
    }
    if constexpr (WITH_V) {
      if (__any(raise)) {
        // Rare (the max rises by more than 8): keep it a branch, not a
        // multiply by 1 on every tile.
        asm volatile("" ::: "memory");
#pragma unroll
        for (int dt = 0; dt < DH / 32; ++dt) oacc[dt] *= corr;
      }
#pragma unroll
      for (int c = 0; c < kKT / 16; ++c) {
        const f32x16& st = s[c / 2];
        const int b = 8 * (c % 2);
        const u32x4 pv = {pack_bf2(st[b + 0], st[b + 1]), pack_bf2(st[b + 2], st[b + 3]),
                          pack_bf2(st[b + 4], st[b + 5]), pack_bf2(st[b + 6], st[b + 7])};
        const bf16x8 pf = as_bf16x8(pv);
#pragma unroll
        for (int dt = 0; dt < DH / 32; ++dt) {
          const u32x4 vv = *reinterpret_cast<const u32x4*>(&Vs[buf][(32 * dt + l32) * kVL + 16 * c + 8 * hi]);
          oacc[dt] = mfma32(as_bf16x8(vv), pf, oacc[dt]);
        }
      }
    }
    if (more) store_tile(buf ^ 1);
    lds_barrier();
    buf ^= 1;
  };

  {
    int64_t b0;
    int r0;
    tile_at(0, b0, r0);
    load_tile(b0, r0);
  }
  store_tile(0);
  lds_barrier();
  // Per key range: its full tiles, then its partial tile through the tail
  // instance of the body (so the hot loop holds the full-tile body only).
  int64_t it = 0;
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int64_t n_full = un.kn[r] / kKT;
    const int rem_last = int(un.kn[r] % kKT);
    for (int64_t f = 0; f < n_full; ++f, ++it) tile(it, un.ks[r] + f * kKT, kKT, std::integral_constant<bool, false>());
    if (rem_last) {
      tile(it, un.ks[r] + n_full * kKT, rem_last, std::integral_constant<bool, true>());
      ++it;
    }
  }

  float l = sum_xor32(lrow);
  const float tm = sum_xor32(trow);
  if (row >= un.q_hi) return;
  if constexpr (WITH_V) {
    if (piece >= 0) {
      // A key piece: its unnormalised output and (max, sum, text sum) per
      // row, in the output's column order, for the combine kernel.
      const int64_t lr = row - un.q_lo;
      float* po = a.part + (piece * kRows + lr) * DH + 4 * hi;
#pragma unroll
      for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f32x16& o = oacc[dt];
          *reinterpret_cast<float4*>(po + 32 * dt + 8 * q) = make_float4(o[4 * q], o[4 * q + 1], o[4 * q + 2], o[4 * q + 3]);
        }
      if (hi == 0) {
        float* pm = a.part_ml + (piece * kRows + lr) * 4;
        *reinterpret_cast<float4*>(pm) = make_float4(mrow, l, MASS ? tm : 0.f, 0.f);
      }
      return;
    }
  }
  if (a.lse && hi == 0) a.lse[int64_t(h) * a.Sq + row] = (mrow + log2f(l)) * kLn2;
  if (MASS && hi == 0) {
    float* dst = a.mass + int64_t(h) * a.Sq + row;
    *dst = (a.mass_accumulate ? *dst : 0.f) + tm / l;
  }
  if constexpr (WITH_V) {
    const float inv = 1.f / l;
    bf16_t* dst = static_cast<bf16_t*>(a.o) + row * a.ldo + int64_t(h) * DH + 4 * hi;
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x16& o = oacc[dt];
        const u32x2 w = {pack_bf2(o[4 * q] * inv, o[4 * q + 1] * inv), pack_bf2(o[4 * q + 2] * inv, o[4 * q + 3] * inv)};
        *reinterpret_cast<u32x2*>(dst + 32 * dt + 8 * q) = w;
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
  float m = -INFINITY, l = 0.f, tl = 0.f;  // tl: the part of l from keys < a.mass_keys
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
    tl *= corr;
    if constexpr (WITH_V) {
#pragma unroll
      for (int c = 0; c < DH; ++c) o[c] *= corr;
    }
    for (int j = 0; j < nk; ++j) {
      const float e = expf(s[j] - m);
      l += e;
      tl += k0 + j < a.mass_keys ? e : 0.f;
      if constexpr (WITH_V) {
#pragma unroll
        for (int c = 0; c < DH; ++c) o[c] = fmaf(e, Vs[j * DH + c], o[c]);
      }
    }
  }
  if (!ok) return;
  if (a.lse) a.lse[int64_t(h) * a.Sq + row] = m + logf(l);
  if (a.mass) {
    float* dst = a.mass + int64_t(h) * a.Sq + row;
    *dst = (a.mass_accumulate ? *dst : 0.f) + tl / l;
  }
  if constexpr (WITH_V) {
    float* dst = static_cast<float*>(a.o) + row * a.ldo + int64_t(h) * DH;
#pragma unroll
    for (int c = 0; c < DH; ++c) dst[c] = o[c] / l;
  }
}

// Combine the key pieces of each split unit: 16 lanes per query row, eight
// output columns per lane (DH = 128; four for DH = 64), every piece's loads
// issued together.  With m_p, l_p the piece's running max (log2 domain) and
// sum, and O_p its unnormalised output, the row's output is
// sum_p 2^(m_p - m) O_p / sum_p 2^(m_p - m) l_p with m = max_p m_p, and its
// log-sum-exp (m + log2 of the denominator) ln 2: the single-pass result up
// to rounding.  With a text mass, the pieces' text sums t_p merge the same
// way: mass = sum_p 2^(m_p - m) t_p / sum_p 2^(m_p - m) l_p.  Pieces are
// summed in key order.
constexpr int kMaxPieces = 4;
template <int DH>
__global__ __launch_bounds__(256) void attn_combine_kernel(const AttnArgs a) {
  constexpr int kLPR = 16, kCols = DH / kLPR;  // lanes per row, columns per lane
  const int sub = threadIdx.x % kLPR;
  const int64_t n_rb = attn_row_blocks(a, kRows);
  const int64_t n_split = n_rb * a.H - a.split_from;
  const int64_t g = int64_t(blockIdx.x) * (256 / kLPR) + threadIdx.x / kLPR;  // split unit * kRows + row
  if (g >= n_split * kRows) return;
  const int64_t su = g / kRows, lr = g % kRows;
  const AttnUnit un = attn_decode(a, kRows, a.split_from + su);
  const int h = un.h;
  const int64_t row = un.q_lo + lr;
  if (row >= un.q_hi) return;
  float4 ml[kMaxPieces];
  float o[kMaxPieces][kCols];
#pragma unroll
  for (int p = 0; p < kMaxPieces; ++p) {
    if (p < a.ksp) {
      const int64_t pc = (su * a.ksp + p) * kRows + lr;
      ml[p] = *reinterpret_cast<const float4*>(a.part_ml + pc * 4);
      const float* po = a.part + pc * DH + sub * kCols;
#pragma unroll
      for (int e = 0; e < kCols; e += 4) {
        const float4 v = *reinterpret_cast<const float4*>(po + e);
        o[p][e] = v.x; o[p][e + 1] = v.y; o[p][e + 2] = v.z; o[p][e + 3] = v.w;
      }
    }
  }
  float m = -INFINITY;
#pragma unroll
  for (int p = 0; p < kMaxPieces; ++p)
    if (p < a.ksp) m = fmaxf(m, ml[p].x);
  float den = 0.f, tden = 0.f, acc[kCols];
#pragma unroll
  for (int e = 0; e < kCols; ++e) acc[e] = 0.f;
#pragma unroll
  for (int p = 0; p < kMaxPieces; ++p) {
    if (p < a.ksp) {
      const float wgt = __builtin_amdgcn_exp2f(ml[p].x - m);
      den = fmaf(wgt, ml[p].y, den);
      tden = fmaf(wgt, ml[p].z, tden);
#pragma unroll
      for (int e = 0; e < kCols; ++e) acc[e] = fmaf(wgt, o[p][e], acc[e]);
    }
  }
  const float inv = 1.f / den;
  bf16_t* dst = static_cast<bf16_t*>(a.o) + row * a.ldo + int64_t(h) * DH + sub * kCols;
  if constexpr (kCols == 8) {
    *reinterpret_cast<u32x4*>(dst) = u32x4{pack_bf2(acc[0] * inv, acc[1] * inv), pack_bf2(acc[2] * inv, acc[3] * inv),
                                           pack_bf2(acc[4] * inv, acc[5] * inv), pack_bf2(acc[6] * inv, acc[7] * inv)};
  } else {
    *reinterpret_cast<u32x2*>(dst) = u32x2{pack_bf2(acc[0] * inv, acc[1] * inv), pack_bf2(acc[2] * inv, acc[3] * inv)};
  }
  if (a.lse && sub == 0) a.lse[int64_t(h) * a.Sq + row] = (m + log2f(den)) * kLn2;
  if (a.mass && sub == 1) {
    float* dst = a.mass + int64_t(h) * a.Sq + row;
    *dst = (a.mass_accumulate ? *dst : 0.f) + tden * inv;
  }
}

// Split-tail plan for the bf16 kernel with V (one sequence or packed ones): whole units
// fill the first workgroup slot of every CU, and the units beyond it run in
// key pieces (or, with fewer units than CUs, every unit is split so that
// the CUs are busy).  Returns ksp (1: no split) and sets split_from and the
// partial pointers.
constexpr int kAttnCUs = 256;
int plan_attn_split(AttnArgs& a, int DH) {
  a.split_from = INT64_MAX;
  a.ksp = 1;
  a.part_ml = nullptr;
  if (!a.part || !a.vt) return 1;
  const int64_t U = attn_row_blocks(a, kRows) * a.H;
  // Fewest key tiles of any unit (every piece must get at least one).
  int64_t T = (a.Sk + 63) / 64;
  if (a.segs.n > 0) {
    T = INT64_MAX;
    for (int b = 0; b < a.segs.n; ++b)
      T = std::min<int64_t>(T, (a.segs.len[b][0] + 63) / 64 + (a.segs.len[b][1] + 63) / 64);
  }
  int64_t from, ksp;
  // Measured on MI355X at S = 1741 (28 key tiles): with at most 128 units,
  // pieces one per CU are fastest; up to 256 units, two per CU; for 336
  // units, 256 whole and the rest in two pieces each (finer pieces lose more
  // to the combine than they gain).
  if (2 * U <= kAttnCUs) {
    from = 0;
    ksp = std::min<int64_t>(kMaxPieces, kAttnCUs / U);
  } else if (U <= kAttnCUs) {
    from = 0;
    ksp = std::min<int64_t>(kMaxPieces, 2 * kAttnCUs / U);
  } else {
    // Both slots of every CU make a round of 2 * 256 units.  A last round of
    // at most 256 units runs in two pieces each; one of up to 384 keeps one
    // whole unit per CU and splits the rest; a fuller one is balanced enough
    // already (984 units at S = 5171: 403 us unsplit, 415 split).
    const int64_t rem = U % (2 * kAttnCUs), base = U - rem;
    if (rem == 0 || rem > kAttnCUs + kAttnCUs / 2) return 1;
    from = rem <= kAttnCUs ? base : base + kAttnCUs;
    ksp = 2;
  }
  // Tuning override "FROM,KSP" (e.g. AVITS_ATTN_SPLIT=256,3; KSP 1 disables).
  if (const char* env = getenv("AVITS_ATTN_SPLIT")) {
    long long f = 0, k = 0;
    if (sscanf(env, "%lld,%lld", &f, &k) == 2 && f >= 0 && f <= U && k >= 1 && k <= kMaxPieces) {
      from = f;
      ksp = k;
    }
  }
  if (from >= U) return 1;
  ksp = std::min<int64_t>(ksp, T);  // at least one key tile per piece
  auto need = [&](int64_t k) { return size_t((U - from) * k) * kRows * (DH + 4) * sizeof(float); };
  while (ksp >= 2 && need(ksp) > a.part_bytes) --ksp;
  if (ksp < 2) return 1;
  const int64_t pieces = (U - from) * ksp;
  a.split_from = from;
  a.ksp = int(ksp);
  a.part_ml = a.part + pieces * kRows * DH;
  return int(ksp);
}

template <int DH>
void launch_dh(AttnArgs a, int dtype, hipStream_t s) {
  const bool with_v = a.vt != nullptr;
  if (dtype == AVITS_BF16) {
    const int64_t U = attn_row_blocks(a, kRows) * a.H;
    const int ksp = plan_attn_split(a, DH);
    const dim3 grid(static_cast<unsigned>(ksp > 1 ? a.split_from + (U - a.split_from) * ksp : U));
    if (with_v) {
      if (a.mass) hipLaunchKernelGGL((attn_bf16_kernel<DH, true, true>), grid, dim3(256), 0, s, a);
      else hipLaunchKernelGGL((attn_bf16_kernel<DH, true, false>), grid, dim3(256), 0, s, a);
      if (ksp > 1) {
        const int64_t rows = (U - a.split_from) * kRows;
        hipLaunchKernelGGL((attn_combine_kernel<DH>), dim3(unsigned(ceil_div64(rows, 16))), dim3(256), 0, s, a);
      }
    } else if (a.mass) {
      hipLaunchKernelGGL((attn_bf16_kernel<DH, false, true>), grid, dim3(256), 0, s, a);
    } else {
      hipLaunchKernelGGL((attn_bf16_kernel<DH, false, false>), grid, dim3(256), 0, s, a);
    }
  } else {
    const dim3 grid(unsigned(ceil_div64(a.Sq, kFRows)), unsigned(a.H));
    if (with_v) hipLaunchKernelGGL((attn_f32_kernel<DH, true>), grid, dim3(kFRows), 0, s, a);
    else hipLaunchKernelGGL((attn_f32_kernel<DH, false>), grid, dim3(kFRows), 0, s, a);
  }
}

}  // namespace

int launch_attention(const AttnArgs& a, int dtype, hipStream_t s) {
  if (a.Sq == 0) return AVITS_OK;
  if (a.segs.n > 0 && (dtype != AVITS_BF16 || a.mass))
    return set_error(AVITS_ERR_UNSUPPORTED, "attention: packed sequences need bf16 and no text mass");
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

extern "C" int avits_joint_attention_stats(const void* q, const void* k_all, int64_t N, int64_t Nk, int64_t L,
                                           int32_t H, int32_t d, int dtype, float* lse, float* mass, int accumulate,
                                           void* stream) {
  AVITS_REQUIRE(N >= 1 && Nk >= 1 && H >= 1, "joint_attention_stats: N=%lld Nk=%lld H=%d must be >= 1",
                (long long)N, (long long)Nk, H);
  AVITS_REQUIRE(L >= 0 && L <= Nk, "joint_attention_stats: L=%lld outside [0, Nk=%lld]", (long long)L,
                (long long)Nk);
  if (d != 64 && d != 128)
    return set_error(AVITS_ERR_UNSUPPORTED, "joint_attention_stats: head dim %d (need 64 or 128)", d);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "joint_attention_stats: dtype %d unsupported", dtype);
  AVITS_REQUIRE(q && k_all && mass, "joint_attention_stats: null q/k_all/mass");
  AttnArgs a{};
  a.q = q;
  a.q_tok = int64_t(H) * d;
  a.q_head = d;
  a.k = k_all;
  a.k_tok = int64_t(H) * d;
  a.k_head = d;
  a.lse = lse;
  a.mass = mass;
  a.mass_keys = L;
  a.mass_accumulate = accumulate != 0;
  a.Sq = N;
  a.Sk = Nk;
  a.H = H;
  a.d = d;
  return launch_attention(a, dtype, static_cast<hipStream_t>(stream));
}
