// One MMDiT joint-attention block on the compacted sequence (Section 3.3.1).
//
// Launch sequence (double-stream; each GEMM is one grouped launch covering
// the text rows with the text weights and the image rows with the image
// weights):
//   ln_mod(x, shift1, scale1)             -> h                 [S, D]
//   h W_qkv^T + b                         -> qk [S, 2D] (q | k, token-major)
//                                            v^T [H, d, S_pad] (transposed epilogue)
//   qk_norm_rope(qk) in place             -> RMSNorm * g, RoPE at pos
//   attention(q, k, v^T)                  -> o [S, D], lse [H, S]
//   x + gate1 (o W_o^T + b)               -> x_mid             (fused epilogue)
//   ln_mod(x_mid, shift2, scale2)         -> h
//   GELU(h W_1^T + b)                     -> m [S, F]          (fused epilogue)
//   x_mid + gate2 (m W_2^T + b)           -> x_out             (fused epilogue)
// Single-stream: ln_mod -> one GEMM whose epilogue writes q | k, v^T, and
// GELU(m) beside the attention output (cat = [o, GELU(m)], [S, D + F]) ->
// qk_norm_rope -> attention into cat -> x + gate (cat W_out^T + b).
#include "kernels.h"
#include "ln_row.h"

namespace avits {
namespace {

constexpr float kRmsEps = 1e-6f;
constexpr float kLog2Theta = 13.287712379549449f;  // log2(10000)

// h = LN(x) (1 + scale) + shift, one wavefront per row; rows [0, n_a) use
// (shift_a, scale_a), the rest (shift_b, scale_b).  bf16 rows of up to 4096
// elements are held in registers (one read, one write); other rows take the
// generic three-pass form.
template <typename T>
__global__ __launch_bounds__(256) void ln_mod_kernel(const T* __restrict__ x, T* __restrict__ h, int64_t S,
                                                     int64_t D, int64_t n_a, const T* __restrict__ shift_a,
                                                     const T* __restrict__ scale_a, const T* __restrict__ shift_b,
                                                     const T* __restrict__ scale_b, const ModRows mods) {
  const int lane = threadIdx.x % kWave;
  const int64_t row = int64_t(blockIdx.x) * 4 + threadIdx.x / kWave;
  if (row >= S) return;
  const T* xr = x + row * D;
  const int64_t moff = mod_offset(mods, row);  // this row's image (several images in one pass)
  const T* sh = (row < n_a ? shift_a : shift_b) + moff;
  const T* sc = (row < n_a ? scale_a : scale_b) + moff;
  T* hr = h + row * D;
  if constexpr (sizeof(T) == 2) {
    const int64_t nchunk = D / 8;
    if (D % 8 == 0 && nchunk <= int64_t(kWave) * kLnMaxChunks) {
      u32x4 v[kLnMaxChunks];
#pragma unroll
      for (int c = 0; c < kLnMaxChunks; ++c) {
        const int64_t idx = lane + kWave * c;
        if (idx < nchunk) v[c] = reinterpret_cast<const u32x4*>(xr)[idx];
      }
      u32x4 g[kLnMaxChunks], t[kLnMaxChunks];
      ln_mod_vectors(sh, sc, nchunk, lane, g, t);
      ln_mod_row_bf16(v, g, t, nchunk, D, lane, hr);
      return;
    }
  }
  float s = 0.f;
  for (int64_t c = lane; c < D; c += kWave) s += ld(xr, c);
  const float mean = wave_sum(s) / float(D);
  float v = 0.f;
  for (int64_t c = lane; c < D; c += kWave) {
    const float t = ld(xr, c) - mean;
    v = fmaf(t, t, v);
  }
  const float rstd = rsqrtf(wave_sum(v) / float(D) + kLnEps);
  for (int64_t c = lane; c < D; c += kWave) st(hr, c, (ld(xr, c) - mean) * rstd * (1.f + ld(sc, c)) + ld(sh, c));
}

// Eight consecutive elements (16 bytes of bf16, 32 of fp32) to / from fp32.
__device__ __forceinline__ void load8(const bf16_t* p, int64_t off, float (&x)[8]) {
  const u32x4 v = *reinterpret_cast<const u32x4*>(p + off);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[2 * e] = __uint_as_float(v[e] << 16);
    x[2 * e + 1] = __uint_as_float(v[e] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load8(const float* p, int64_t off, float (&x)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p + off), b = *reinterpret_cast<const float4*>(p + off + 4);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}
__device__ __forceinline__ void store8(bf16_t* p, const float (&x)[8]) {
  *reinterpret_cast<u32x4*>(p) =
      u32x4{pack_bf2(x[0], x[1]), pack_bf2(x[2], x[3]), pack_bf2(x[4], x[5]), pack_bf2(x[6], x[7])};
}
__device__ __forceinline__ void store8(float* p, const float (&x)[8]) {
  *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(x[4], x[5], x[6], x[7]);
}

// In-place RMSNorm (times the gain) and RoPE of q [S, ld] and k [S, ld]
// (head-major within a row: the block passes q | k of one [S, 2D] buffer,
// ld = 2D; the probe passes two [S, D] arrays, ld = D).  Each lane owns 8 consecutive elements
// (4 rotation pairs) of one head, so a d-wide head spans d/8 lanes and the
// RMS reduction stays inside that lane group.  Rows [0, n_a) use the gains
// of stream a.  A wavefront takes kQkPasses passes of 64*8/d heads of one
// row (a row's 2H heads are split over `parts` wavefronts, so that short
// sequences still put several wavefronts on every SIMD); all its loads are
// in flight before its first store.
constexpr int kQkPasses = 3;
template <typename T, int DH>
__global__ __launch_bounds__(256) void qk_norm_rope_kernel(T* __restrict__ q, T* __restrict__ k, int64_t ld,
                                                           const int32_t* __restrict__ pos, float pos_scale,
                                                           int64_t S, int H, int parts, int64_t n_a,
                                                           const T* __restrict__ gq_a, const T* __restrict__ gk_a,
                                                           const T* __restrict__ gq_b, const T* __restrict__ gk_b) {
  constexpr int kLanesPerHead = DH / 8;
  constexpr int kHeadsPerPass = kWave / kLanesPerHead;
  constexpr int p0 = DH / 16, p1 = 7 * DH / 32;  // rotation pairs per axis: (p0, p1, p1)
  const int lane = threadIdx.x % kWave;
  const int64_t gw = int64_t(blockIdx.x) * 4 + threadIdx.x / kWave;
  const int64_t row = gw / parts;
  if (row >= S) return;
  const int h0 = int(gw % parts) * kQkPasses * kHeadsPerPass;
  const int sub = lane % kLanesPerHead;           // position of the lane inside its head
  const int hoff = lane / kLanesPerHead;          // head slot within a pass
  const bool a_rows = row < n_a;
  // Angles of this lane's four pairs m = 4 sub + j.
  float cs[4], sn[4];
  const int32_t pr[3] = {pos[3 * row], pos[3 * row + 1], pos[3 * row + 2]};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int m = 4 * sub + j;
    const int axis = m < p0 ? 0 : (m < p0 + p1 ? 1 : 2);
    const int mi = axis == 0 ? m : (axis == 1 ? m - p0 : m - p0 - p1);
    const int na = axis == 0 ? 2 * p0 : 2 * p1;
    const float freq = exp2f(-2.f * float(mi) / float(na) * kLog2Theta);
    sincosf(float(pr[axis]) * pos_scale * freq, &sn[j], &cs[j]);
  }
  T* const qrow = q + row * ld;
  T* const krow = k + row * ld;
  // Both gain vectors of this lane's 8 elements, loaded once per row.
  float gq[8], gk[8];
  load8(a_rows ? gq_a : gq_b, 8 * sub, gq);
  load8(a_rows ? gk_a : gk_b, 8 * sub, gk);
  // Head slots 0..H-1 are query heads, H..2H-1 key heads; a slot past the
  // end loads head 0 and is not stored.
  auto at = [&](int head) {
    return (head < H ? qrow + int64_t(head) * DH : krow + int64_t(head - H) * DH) + 8 * sub;
  };
  {
    float x[kQkPasses][8];
#pragma unroll
    for (int i = 0; i < kQkPasses; ++i) {
      const int head = h0 + i * kHeadsPerPass + hoff;
      load8(at(head < 2 * H ? head : 0), 0, x[i]);
    }
#pragma unroll
    for (int i = 0; i < kQkPasses; ++i) {
      const int head = h0 + i * kHeadsPerPass + hoff;
      float ss = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) ss = fmaf(x[i][e], x[i][e], ss);
      ss = group_sum(ss, kLanesPerHead);
      const float r = rsqrtf(ss / float(DH) + kRmsEps);
      const float* g = head < H ? gq : gk;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float y0 = x[i][2 * j] * r * g[2 * j];
        const float y1 = x[i][2 * j + 1] * r * g[2 * j + 1];
        x[i][2 * j] = y0 * cs[j] - y1 * sn[j];
        x[i][2 * j + 1] = y0 * sn[j] + y1 * cs[j];
      }
      if (head < 2 * H) store8(at(head), x[i]);
    }
  }
}

struct BlockWs {
  char* h;      // [S, D]
  char* qk;     // [S, 2D]
  char* vt;     // [H, d, ldvt]
  char* o;      // double: [S, D]; single: cat [S, D + F]
  char* xmid;   // double only
  char* mlp;    // double only: [S, F]
  float* partial;  // split-K partial sums of the N = D projections
  size_t partial_bytes;
  int64_t ldvt;
  size_t bytes;
};

BlockWs block_ws_layout(char* base, int kind, int64_t S, int64_t H, int64_t d, int64_t F, int64_t esz) {
  BlockWs w{};
  const int64_t D = H * d;
  w.ldvt = ceil_div64(std::max<int64_t>(S, 1), kAttnKeyTile) * kAttnKeyTile;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = base ? base + off : nullptr;
    off += align_up(bytes, 256);
    return p;
  };
  w.h = take(size_t(S * D * esz));
  w.qk = take(size_t(S * 2 * D * esz));
  w.vt = take(size_t(H * d * w.ldvt * esz));
  if (kind == AVITS_BLOCK_DOUBLE) {
    w.o = take(size_t(S * D * esz));
    w.xmid = take(size_t(S * D * esz));
    w.mlp = take(size_t(S * F * esz));
  } else {
    w.o = take(size_t(S * (D + F) * esz));
  }
  w.partial_bytes = gemm_partial_reserve(S, D);
  w.partial = reinterpret_cast<float*>(take(w.partial_bytes));
  w.bytes = off;
  return w;
}

// Per-stream views of a block call: (row offset, row count, weights).
struct Stream { int64_t r0, rows; const avits_double_stream_weights* dw; };

template <typename T>
const T* mod_row(const void* mod, int r, int64_t D) { return static_cast<const T*>(mod) + r * D; }

// h = LN(x)(1 + scale) + shift with the modulation rows (r_shift, r_scale) of
// each stream (the single kind has one set for every row).
template <typename T>
int launch_ln_mod(const T* x, T* h, int64_t S, int64_t D, int64_t n_txt, const avits_block_weights* w, int r_shift,
                  hipStream_t s, const ModRows& mods = ModRows{}) {
  const dim3 rows_grid(unsigned(ceil_div64(S, 4))), blk(256);
  TimedLaunch timed("ln_mod", s);
  if (w->kind == AVITS_BLOCK_DOUBLE) {
    const avits_double_stream_weights& wa = n_txt ? w->txt : w->img;
    const avits_double_stream_weights& wb = n_txt < S ? w->img : w->txt;
    hipLaunchKernelGGL(ln_mod_kernel<T>, rows_grid, blk, 0, s, x, h, S, D, n_txt, mod_row<T>(wa.mod, r_shift, D),
                       mod_row<T>(wa.mod, r_shift + 1, D), mod_row<T>(wb.mod, r_shift, D),
                       mod_row<T>(wb.mod, r_shift + 1, D), mods);
  } else {
    const void* m = w->single.mod;
    hipLaunchKernelGGL(ln_mod_kernel<T>, rows_grid, blk, 0, s, x, h, S, D, S, mod_row<T>(m, 0, D),
                       mod_row<T>(m, 1, D), mod_row<T>(m, 0, D), mod_row<T>(m, 1, D), mods);
  }
  return launch_status("block ln_mod");
}

// RMSNorm * g and RoPE of q and k in place, with each stream's gains.
template <typename T>
int launch_qk_norm_rope(T* q, T* k, int64_t ld, const int32_t* pos, float pos_scale, int64_t S, int64_t n_txt, int H,
                        int d, const avits_block_weights* w, hipStream_t s) {
  const T *gqa, *gka, *gqb, *gkb;
  int64_t na;
  if (w->kind == AVITS_BLOCK_DOUBLE) {
    const avits_double_stream_weights& wa = n_txt ? w->txt : w->img;
    const avits_double_stream_weights& wb = n_txt < S ? w->img : w->txt;
    gqa = static_cast<const T*>(wa.g_q); gka = static_cast<const T*>(wa.g_k);
    gqb = static_cast<const T*>(wb.g_q); gkb = static_cast<const T*>(wb.g_k);
    na = n_txt;
  } else {
    gqa = gqb = static_cast<const T*>(w->single.g_q);
    gka = gkb = static_cast<const T*>(w->single.g_k);
    na = S;
  }
  const int parts = int(ceil_div64(2 * int64_t(H), int64_t(kQkPasses) * (kWave * 8 / d)));
  const dim3 grid(unsigned(ceil_div64(S * parts, 4))), blk(256);
  TimedLaunch timed("qk_rope", s);
  if (d == 128)
    hipLaunchKernelGGL((qk_norm_rope_kernel<T, 128>), grid, blk, 0, s, q, k, ld, pos, pos_scale, S, H, parts, na,
                       gqa, gka, gqb, gkb);
  else
    hipLaunchKernelGGL((qk_norm_rope_kernel<T, 64>), grid, blk, 0, s, q, k, ld, pos, pos_scale, S, H, parts, na,
                       gqa, gka, gqb, gkb);
  return launch_status("block qk_norm_rope");
}

// The block's first stage alone: LN + modulation, the q and k projections,
// RMSNorm and RoPE, written to q_out [S, D] and k_out [S, D].
template <typename T>
int run_block_qk(const void* x_in, const int32_t* pos, float pos_scale, int64_t n_txt, int64_t n_img,
                 const avits_block_weights* w, int H, int d, int dtype, void* q_out, void* k_out, void* h_ws,
                 hipStream_t s) {
  const int64_t S = n_txt + n_img, D = int64_t(H) * d;
  T* h = static_cast<T*>(h_ws);
  T* q = static_cast<T*>(q_out);
  T* k = static_cast<T*>(k_out);
  int rc;
  if ((rc = launch_ln_mod<T>(static_cast<const T*>(x_in), h, S, D, n_txt, w, 0, s)) != AVITS_OK) return rc;
  GemmArgs g{};
  g.N = 2 * D;          // the first 2D output rows of W_qkv (or W_in): q then k
  g.K = D;
  g.n_split = D;
  g.n_split2 = 2 * D;
  g.mode0 = EPI_STORE;
  g.mode1 = EPI_STORE;
  if (w->kind == AVITS_BLOCK_DOUBLE) {
    const Stream st2[2] = {{0, n_txt, &w->txt}, {n_txt, n_img, &w->img}};
    for (const Stream& t : st2) {
      if (t.rows == 0) continue;
      GemmProblem& p = g.p[g.nprob++];
      p.A = h + t.r0 * D; p.lda = D; p.W = t.dw->w_qkv; p.bias = t.dw->b_qkv; p.M = t.rows;
      p.out0 = q + t.r0 * D; p.ld0 = D;
      p.out1 = k + t.r0 * D; p.ld1 = D;
    }
  } else {
    GemmProblem& p = g.p[g.nprob++];
    p.A = h; p.lda = D; p.W = w->single.w_in; p.bias = w->single.b_in; p.M = S;
    p.out0 = q; p.ld0 = D;
    p.out1 = k; p.ld1 = D;
  }
  if ((rc = launch_gemm(g, dtype, s, w->kind == AVITS_BLOCK_DOUBLE ? "gemm_qkv" : "gemm_single_in", nullptr, 0)) !=
      AVITS_OK)
    return rc;
  return launch_qk_norm_rope<T>(q, k, D, pos, pos_scale, S, n_txt, H, d, w, s);
}

template <typename T>
int run_block(const void* x_in, void* x_out, const int32_t* pos, float pos_scale, int64_t n_txt, int64_t n_img,
              const avits_block_weights* w, int H, int d, int dtype, float* lse_out, const BlockWs& ws,
              hipStream_t s, const AttnSegs* segs = nullptr, float* mass_out = nullptr, int mass_accumulate = 0,
              const avits_block_outputs* sc = nullptr, const ModRows& mods = ModRows{}) {
  const int64_t S = n_txt + n_img, D = int64_t(H) * d, F = w->mlp_hidden;
  const bool dbl = w->kind == AVITS_BLOCK_DOUBLE;
  const T* x = static_cast<const T*>(x_in);
  T* h = reinterpret_cast<T*>(ws.h);
  T* qk = reinterpret_cast<T*>(ws.qk);
  T* vt = reinterpret_cast<T*>(ws.vt);
  int rc;

  // The non-empty streams (double kind).
  const Stream st2[2] = {{0, n_txt, &w->txt}, {n_txt, n_img, &w->img}};
  int nst = 0;
  Stream streams[2];
  if (dbl) {
    for (const Stream& t : st2)
      if (t.rows > 0) streams[nst++] = t;
  }
  auto mod_row = [&](const void* mod, int r) { return static_cast<const T*>(mod) + r * D; };

  // 1. modulated layer norm (or the caller's, computed as it gathered x).
  const T* hq = h;
  if (sc && sc->h_in) hq = static_cast<const T*>(sc->h_in);
  else if ((rc = launch_ln_mod<T>(x, h, S, D, n_txt, w, 0, s, mods)) != AVITS_OK) return rc;

  // 2. QKV projection: q | k token-major, v transposed per head
  //    (+ the single block's MLP input, GELU'd beside o).
  {
    GemmArgs g{};
    g.K = D;
    g.n_split = 2 * D;
    g.n_split2 = 3 * D;
    g.mode0 = EPI_STORE;
    g.mode1 = EPI_STORE_T;
    g.mode2 = EPI_GELU;
    if (dbl) {
      g.N = 3 * D;
      for (int i = 0; i < nst; ++i) {
        GemmProblem& p = g.p[i];
        const int64_t r0 = streams[i].r0;
        p.A = hq + r0 * D; p.lda = D;
        p.W = streams[i].dw->w_qkv; p.bias = streams[i].dw->b_qkv; p.M = streams[i].rows;
        p.out0 = qk + r0 * 2 * D; p.ld0 = 2 * D;
        p.out1 = vt + r0; p.ld1 = ws.ldvt;
      }
      g.nprob = nst;
    } else {
      g.N = 3 * D + F;
      GemmProblem& p = g.p[0];
      p.A = hq; p.lda = D; p.W = w->single.w_in; p.bias = w->single.b_in; p.M = S;
      p.out0 = qk; p.ld0 = 2 * D;
      p.out1 = vt; p.ld1 = ws.ldvt;
      p.out2 = reinterpret_cast<T*>(ws.o) + D; p.ld2 = D + F;
      g.nprob = 1;
    }
    if ((rc = launch_gemm(g, dtype, s, dbl ? "gemm_qkv" : "gemm_single_in", ws.partial, ws.partial_bytes)) != AVITS_OK)
      return rc;
  }

  // 3. q/k RMSNorm + RoPE in place.
  if ((rc = launch_qk_norm_rope<T>(qk, qk + D, 2 * D, pos, pos_scale, S, n_txt, H, d, w, s)) != AVITS_OK) return rc;

  // 4. joint attention over all S rows (or within each packed sequence).
  {
    AttnArgs a{};
    if (segs) a.segs = *segs;
    a.q = qk; a.q_tok = 2 * D; a.q_head = d;
    a.k = qk + D; a.k_tok = 2 * D; a.k_head = d;
    a.vt = vt; a.ldvt = ws.ldvt;
    a.o = ws.o; a.ldo = dbl ? D : D + F;
    a.lse = lse_out;
    // The text mass of Eq. spatial under the same running maximum: the
    // softmax share of the keys [0, n_txt) (the text rows lead the sequence).
    a.mass = mass_out;
    a.mass_keys = n_txt;
    a.mass_accumulate = mass_accumulate;
    a.Sq = S; a.Sk = S; a.H = H; a.d = d;
    a.part = ws.partial; a.part_bytes = ws.partial_bytes;  // no GEMM partials are live here
    if ((rc = launch_attention(a, dtype, s)) != AVITS_OK) return rc;
  }

  T* out = static_cast<T*>(x_out);
  // The next block's first stage (its LN + modulation of this block's
  // output) rides on the last projection's split-K reduce when the GEMM is
  // split and each problem's rows take one set of the next block's vectors;
  // otherwise the LN kernel runs on x_out.
  const bool want_next = sc && sc->h_next && sc->next_w;
  auto finish_next = [&](const T* y, const GemmPostLN& nl, bool fused) -> int {
    if (!want_next || (fused && sizeof(T) == 2 && nl.done)) return AVITS_OK;
    return launch_ln_mod<T>(y, static_cast<T*>(sc->h_next), S, D, n_txt, sc->next_w, 0, s, mods);
  };
  // The Stage-3 scatter rides on the last projection: the output rows of the
  // last scatter_k image rows also go to their canvas rows.
  auto set_scatter = [&](GemmProblem& p, int64_t rows) {
    if (!sc || !sc->canvas || sc->scatter_k == 0) return;
    p.scat = sc->canvas;
    p.scat_idx = sc->scatter_idx;
    p.scat_row0 = rows - sc->scatter_k;
    p.scat_ld = D;
    p.scat_n = sc->n_canvas;
  };
  if (!dbl) {
    GemmArgs g{};
    g.N = D; g.K = D + F; g.n_split = g.n_split2 = g.N; g.mode0 = EPI_RESID_GATE; g.nprob = 1;
    g.mod = mods;
    GemmProblem& p = g.p[0];
    p.A = ws.o; p.lda = D + F; p.W = w->single.w_out; p.bias = w->single.b_out; p.M = S;
    p.out0 = out; p.ld0 = D; p.resid = x; p.ldr = D; p.gate = mod_row(w->single.mod, 2);
    set_scatter(p, S);
    // The next block's first stage on the reduce when that block is single
    // too (one set of vectors for the launch's one problem).
    GemmPostLN nl{};
    const bool fuse_next = want_next && sc->next_w->kind == AVITS_BLOCK_SINGLE;
    if (fuse_next) {
      nl.out = sc->h_next;
      nl.ld = D;
      nl.shift[0] = mod_row(sc->next_w->single.mod, 0);
      nl.scale[0] = mod_row(sc->next_w->single.mod, 1);
    }
    if ((rc = launch_gemm(g, dtype, s, "gemm_single_out", ws.partial, ws.partial_bytes,
                          sizeof(T) == 2 && fuse_next ? &nl : nullptr)) != AVITS_OK)
      return rc;
    return finish_next(out, nl, fuse_next);
  }

  // 5. output projection + gated residual.
  T* xmid = reinterpret_cast<T*>(ws.xmid);
  {
    GemmArgs g{};
    g.N = D; g.K = D; g.n_split = g.n_split2 = g.N; g.mode0 = EPI_RESID_GATE; g.nprob = nst;
    g.mod = mods;
    for (int i = 0; i < nst; ++i) {
      GemmProblem& p = g.p[i];
      const int64_t r0 = streams[i].r0;
      p.row0 = r0;
      p.A = reinterpret_cast<T*>(ws.o) + r0 * D; p.lda = D;
      p.W = streams[i].dw->w_o; p.bias = streams[i].dw->b_o; p.M = streams[i].rows;
      p.out0 = xmid + r0 * D; p.ld0 = D; p.resid = x + r0 * D; p.ldr = D;
      p.gate = mod_row(streams[i].dw->mod, 2);
    }
    // 6. the second modulated layer norm rides on the split-K reduce when
    //    the projection is split (bf16), else runs on its own.
    GemmPostLN ln{};
    ln.out = h;
    ln.ld = D;
    for (int i = 0; i < nst; ++i) {
      ln.shift[i] = mod_row(streams[i].dw->mod, 3);
      ln.scale[i] = mod_row(streams[i].dw->mod, 4);
    }
    if ((rc = launch_gemm(g, dtype, s, "gemm_o", ws.partial, ws.partial_bytes,
                          sizeof(T) == 2 ? &ln : nullptr)) != AVITS_OK)
      return rc;
    if (!(sizeof(T) == 2 && ln.done) && (rc = launch_ln_mod<T>(xmid, h, S, D, n_txt, w, 3, s, mods)) != AVITS_OK)
      return rc;
  }
  // 7. MLP in + GELU.
  T* mlp = reinterpret_cast<T*>(ws.mlp);
  {
    GemmArgs g{};
    g.N = F; g.K = D; g.n_split = g.n_split2 = g.N; g.mode0 = EPI_GELU; g.nprob = nst;
    for (int i = 0; i < nst; ++i) {
      GemmProblem& p = g.p[i];
      const int64_t r0 = streams[i].r0;
      p.A = h + r0 * D; p.lda = D; p.W = streams[i].dw->w_mlp1; p.bias = streams[i].dw->b_mlp1;
      p.M = streams[i].rows; p.out0 = mlp + r0 * F; p.ld0 = F;
    }
    if ((rc = launch_gemm(g, dtype, s, "gemm_mlp_in", ws.partial, ws.partial_bytes)) != AVITS_OK) return rc;
  }
  // 8. MLP out + gated residual.
  {
    GemmArgs g{};
    g.N = D; g.K = F; g.n_split = g.n_split2 = g.N; g.mode0 = EPI_RESID_GATE; g.nprob = nst;
    g.mod = mods;
    for (int i = 0; i < nst; ++i) {
      GemmProblem& p = g.p[i];
      const int64_t r0 = streams[i].r0;
      p.row0 = r0;
      p.A = mlp + r0 * F; p.lda = F; p.W = streams[i].dw->w_mlp2; p.bias = streams[i].dw->b_mlp2;
      p.M = streams[i].rows; p.out0 = out + r0 * D; p.ld0 = D; p.resid = xmid + r0 * D; p.ldr = D;
      p.gate = mod_row(streams[i].dw->mod, 5);
      if (r0 == n_txt && n_img > 0) set_scatter(p, n_img);   // the image stream
    }
    GemmPostLN nl{};
    if (want_next) {
      nl.out = sc->h_next;
      nl.ld = D;
      for (int i = 0; i < nst; ++i) {
        const avits_block_weights* nw = sc->next_w;
        const void* m = nw->kind == AVITS_BLOCK_SINGLE ? nw->single.mod
                        : streams[i].r0 < n_txt       ? nw->txt.mod
                                                      : nw->img.mod;
        nl.shift[i] = mod_row(m, 0);
        nl.scale[i] = mod_row(m, 1);
      }
    }
    if ((rc = launch_gemm(g, dtype, s, "gemm_mlp_out", ws.partial, ws.partial_bytes,
                          sizeof(T) == 2 && want_next ? &nl : nullptr)) != AVITS_OK)
      return rc;
    return finish_next(out, nl, want_next);
  }
}

bool all_set(const avits_double_stream_weights& w) {
  return w.mod && w.w_qkv && w.b_qkv && w.g_q && w.g_k && w.w_o && w.b_o && w.w_mlp1 && w.b_mlp1 && w.w_mlp2 &&
         w.b_mlp2;
}

}  // namespace
}  // namespace avits

using namespace avits;

extern "C" size_t avits_block_workspace_bytes(int32_t kind, int64_t S, int32_t H, int32_t d, int32_t mlp_hidden,
                                              int dtype) {
  if (S < 0 || H < 1 || d < 1 || mlp_hidden < 1) return 0;
  if (kind != AVITS_BLOCK_DOUBLE && kind != AVITS_BLOCK_SINGLE) return 0;
  if (dtype != AVITS_F32 && dtype != AVITS_BF16) return 0;
  return block_ws_layout(nullptr, kind, S, H, d, mlp_hidden, dtype == AVITS_F32 ? 4 : 2).bytes;
}

namespace avits {
namespace {
// Host-side checks shared by avits_block_forward and avits_block_qk; returns
// AVITS_OK or the error code (with the message set).
int check_block_args(const char* fn, const void* x_in, const int32_t* pos, float pos_scale, int64_t n_txt,
                     int64_t n_img, const avits_block_weights* w, int32_t H, int32_t d, int dtype) {
  AVITS_REQUIRE(w, "%s: null weights", fn);
  AVITS_REQUIRE(n_txt >= 0 && n_img >= 0, "%s: n_txt=%lld n_img=%lld must be >= 0", fn, (long long)n_txt,
                (long long)n_img);
  AVITS_REQUIRE(H >= 1, "%s: H=%d < 1", fn, H);
  AVITS_REQUIRE(pos_scale > 0.f && pos_scale <= 1.f, "%s: pos_scale=%g outside (0, 1]", fn, pos_scale);
  if (d != 64 && d != 128) return set_error(AVITS_ERR_UNSUPPORTED, "%s: head dim %d (need 64 or 128)", fn, d);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "%s: dtype %d unsupported", fn, dtype);
  AVITS_REQUIRE(w->kind == AVITS_BLOCK_DOUBLE || w->kind == AVITS_BLOCK_SINGLE, "%s: bad kind %d", fn, w->kind);
  AVITS_REQUIRE(w->mlp_hidden >= 64 && w->mlp_hidden % 64 == 0,
                "%s: mlp_hidden=%d must be a positive multiple of 64", fn, w->mlp_hidden);
  const int64_t S = n_txt + n_img;
  AVITS_REQUIRE(S <= INT32_MAX, "%s: S=%lld too large", fn, (long long)S);
  if (S == 0) return AVITS_OK;
  AVITS_REQUIRE(x_in && pos, "%s: null x_in/pos", fn);
  if (w->kind == AVITS_BLOCK_DOUBLE) {
    AVITS_REQUIRE(n_txt == 0 || all_set(w->txt), "%s: missing text-stream weight", fn);
    AVITS_REQUIRE(n_img == 0 || all_set(w->img), "%s: missing image-stream weight", fn);
  } else {
    const avits_single_weights& sw = w->single;
    AVITS_REQUIRE(sw.mod && sw.w_in && sw.b_in && sw.g_q && sw.g_k && sw.w_out && sw.b_out,
                  "%s: missing single-block weight", fn);
  }
  return AVITS_OK;
}
}  // namespace
}  // namespace avits

extern "C" size_t avits_block_qk_workspace_bytes(int64_t S, int32_t H, int32_t d, int dtype) {
  if (S < 0 || H < 1 || d < 1 || (dtype != AVITS_F32 && dtype != AVITS_BF16)) return 0;
  return align_up(size_t(S) * size_t(H) * size_t(d) * (dtype == AVITS_F32 ? 4 : 2), 256);
}

extern "C" int avits_block_qk(const void* x_in, const int32_t* pos, float pos_scale, int64_t n_txt, int64_t n_img,
                              const avits_block_weights* w, int32_t H, int32_t d, int dtype, void* q_out, void* k_out,
                              void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_block_args("block_qk", x_in, pos, pos_scale, n_txt, n_img, w, H, d, dtype);
  if (rc != AVITS_OK) return rc;
  const int64_t S = n_txt + n_img;
  if (S == 0) return AVITS_OK;
  AVITS_REQUIRE(q_out && k_out && q_out != k_out, "block_qk: q_out and k_out must be distinct non-null buffers");
  const size_t need = avits_block_qk_workspace_bytes(S, H, d, dtype);
  if (!workspace || workspace_bytes < need)
    return set_error(AVITS_ERR_WORKSPACE, "block_qk: workspace of %zu bytes, need %zu", workspace_bytes, need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == AVITS_BF16)
    return run_block_qk<bf16_t>(x_in, pos, pos_scale, n_txt, n_img, w, H, d, dtype, q_out, k_out, workspace, s);
  return run_block_qk<float>(x_in, pos, pos_scale, n_txt, n_img, w, H, d, dtype, q_out, k_out, workspace, s);
}

extern "C" int avits_block_forward(const void* x_in, void* x_out, const int32_t* pos, float pos_scale,
                                   int64_t n_txt, int64_t n_img, const avits_block_weights* w, int32_t H, int32_t d,
                                   int dtype, float* lse_out, void* workspace, size_t workspace_bytes,
                                   void* stream) {
  avits_block_outputs o{};
  o.lse = lse_out;
  return avits_block_forward_ex(x_in, x_out, pos, pos_scale, n_txt, n_img, w, H, d, dtype, &o, workspace,
                                workspace_bytes, stream);
}

extern "C" int avits_block_forward_ex(const void* x_in, void* x_out, const int32_t* pos, float pos_scale,
                                      int64_t n_txt, int64_t n_img, const avits_block_weights* w, int32_t H,
                                      int32_t d, int dtype, const avits_block_outputs* outs, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  const avits_block_outputs none{};
  if (!outs) outs = &none;
  int rc = check_block_args("block_forward", x_in, pos, pos_scale, n_txt, n_img, w, H, d, dtype);
  if (rc != AVITS_OK) return rc;
  const int64_t S = n_txt + n_img;
  if (S == 0) return AVITS_OK;
  AVITS_REQUIRE(x_out, "block_forward: null x_out");
  AVITS_REQUIRE(x_in != x_out, "block_forward: x_out must not alias x_in");
  const int64_t esz = dtype == AVITS_F32 ? 4 : 2;
  const BlockWs need = block_ws_layout(nullptr, w->kind, S, H, d, w->mlp_hidden, esz);
  if (!workspace || workspace_bytes < need.bytes)
    return set_error(AVITS_ERR_WORKSPACE, "block_forward: workspace of %zu bytes, need %zu", workspace_bytes,
                     need.bytes);
  const BlockWs ws = block_ws_layout(static_cast<char*>(workspace), w->kind, S, H, d, w->mlp_hidden, esz);
  if (outs->canvas || outs->scatter_k) {
    AVITS_REQUIRE(outs->scatter_k >= 0 && outs->scatter_k <= n_img,
                  "block_forward_ex: scatter_k=%lld outside [0, n_img=%lld]", (long long)outs->scatter_k,
                  (long long)n_img);
    AVITS_REQUIRE(outs->scatter_k == 0 || (outs->canvas && outs->scatter_idx && outs->n_canvas >= 1),
                  "block_forward_ex: scatter needs canvas, scatter_idx and n_canvas >= 1");
    AVITS_REQUIRE(outs->canvas != x_in && outs->canvas != x_out, "block_forward_ex: canvas must not alias x_in/x_out");
  }
  const char* wb = static_cast<const char*>(workspace);
  if (outs->h_in) {
    const char* hb = static_cast<const char*>(outs->h_in);
    AVITS_REQUIRE(outs->h_in != x_in && outs->h_in != x_out && !(hb >= wb && hb < wb + need.bytes),
                  "block_forward_ex: h_in must not alias x_in, x_out or the workspace");
  }
  if (outs->h_next || outs->next_w) {
    AVITS_REQUIRE(outs->h_next && outs->next_w, "block_forward_ex: h_next and next_w go together");
    const avits_block_weights* nw = outs->next_w;
    AVITS_REQUIRE(nw->kind == AVITS_BLOCK_DOUBLE ? (nw->txt.mod || n_txt == 0) && (nw->img.mod || n_img == 0)
                                                 : nw->kind == AVITS_BLOCK_SINGLE && nw->single.mod != nullptr,
                  "block_forward_ex: next_w lacks the modulation its rows need");
    const char* hb = static_cast<const char*>(outs->h_next);
    AVITS_REQUIRE(outs->h_next != x_in && outs->h_next != x_out && outs->h_next != outs->h_in &&
                      !(hb >= wb && hb < wb + need.bytes),
                  "block_forward_ex: h_next must not alias x_in, x_out, h_in or the workspace");
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == AVITS_BF16)
    return run_block<bf16_t>(x_in, x_out, pos, pos_scale, n_txt, n_img, w, H, d, dtype, outs->lse, ws, s, nullptr,
                             outs->mass, outs->mass_accumulate, outs);
  return run_block<float>(x_in, x_out, pos, pos_scale, n_txt, n_img, w, H, d, dtype, outs->lse, ws, s, nullptr,
                          outs->mass, outs->mass_accumulate, outs);
}

extern "C" int avits_block_forward_batched(const void* x_in, void* x_out, const int32_t* pos, float pos_scale,
                                           int32_t B, const int64_t* txt_off, const int64_t* img_off,
                                           const avits_block_weights* w, int32_t H, int32_t d, int dtype,
                                           float* lse_out, void* workspace, size_t workspace_bytes,
                                           void* stream) {
  return avits_block_forward_batched_ex(x_in, x_out, pos, pos_scale, B, txt_off, img_off, w, 0, H, d, dtype, lse_out,
                                        workspace, workspace_bytes, stream);
}

extern "C" int avits_block_forward_batched_ex(const void* x_in, void* x_out, const int32_t* pos, float pos_scale,
                                              int32_t B, const int64_t* txt_off, const int64_t* img_off,
                                              const avits_block_weights* w, int64_t mod_stride, int32_t H,
                                              int32_t d, int dtype, float* lse_out, void* workspace,
                                              size_t workspace_bytes, void* stream) {
  AVITS_REQUIRE(B >= 1 && B <= kMaxSeqs, "block_forward_batched: B=%d outside [1, %d]", B, kMaxSeqs);
  AVITS_REQUIRE(mod_stride >= 0, "block_forward_batched: mod_stride=%lld < 0", (long long)mod_stride);
  AVITS_REQUIRE(txt_off && img_off, "block_forward_batched: null txt_off/img_off");
  AVITS_REQUIRE(txt_off[0] == 0 && img_off[0] == 0, "block_forward_batched: offsets must start at 0");
  AttnSegs segs{};
  segs.n = B;
  const int64_t n_txt = txt_off[B], n_img = img_off[B];
  for (int b = 0; b < B; ++b) {
    const int64_t lt = txt_off[b + 1] - txt_off[b], li = img_off[b + 1] - img_off[b];
    AVITS_REQUIRE(lt >= 0 && li >= 0 && lt + li >= 1,
                  "block_forward_batched: sequence %d has %lld text and %lld image rows", b, (long long)lt,
                  (long long)li);
    segs.start[b][0] = txt_off[b];
    segs.len[b][0] = lt;
    segs.start[b][1] = n_txt + img_off[b];
    segs.len[b][1] = li;
  }
  int rc = check_block_args("block_forward_batched", x_in, pos, pos_scale, n_txt, n_img, w, H, d, dtype);
  if (rc != AVITS_OK) return rc;
  if (dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "block_forward_batched: packed sequences need bf16 (dtype %d)", dtype);
  const int64_t S = n_txt + n_img;
  AVITS_REQUIRE(x_out, "block_forward_batched: null x_out");
  AVITS_REQUIRE(x_in != x_out, "block_forward_batched: x_out must not alias x_in");
  const BlockWs need = block_ws_layout(nullptr, w->kind, S, H, d, w->mlp_hidden, 2);
  if (!workspace || workspace_bytes < need.bytes)
    return set_error(AVITS_ERR_WORKSPACE, "block_forward_batched: workspace of %zu bytes, need %zu",
                     workspace_bytes, need.bytes);
  const BlockWs ws = block_ws_layout(static_cast<char*>(workspace), w->kind, S, H, d, w->mlp_hidden, 2);
  // Per-image modulation: segment b ends at image b's last text row,
  // segment B + b at its last image row (rows packed by stream).
  ModRows mods{};
  if (mod_stride > 0 && B > 1) {
    mods.B = B;
    mods.stride = mod_stride;
    for (int b = 0; b < B; ++b) {
      mods.end[b] = txt_off[b + 1];
      mods.end[B + b] = n_txt + img_off[b + 1];
    }
  }
  return run_block<bf16_t>(x_in, x_out, pos, pos_scale, n_txt, n_img, w, H, d, dtype, lse_out, ws,
                           static_cast<hipStream_t>(stream), &segs, nullptr, 0, nullptr, mods);
}

// ---------------------------------------------------------------------------
// Around the path, for the Stage-2 steps of Section 3.2 run on the selected
// tokens alone: the model's latent embedder (a linear map into the hidden
// width), its output layer (modulated layer norm, then a linear map back to
// the latent channels), and the Euler update of Eq. euler on those tokens.
namespace avits {
namespace {

// z = z + dt v, computed in fp32 and rounded once; 8 elements per thread.
template <typename T>
__global__ __launch_bounds__(256) void euler_kernel(T* __restrict__ z, const T* __restrict__ v, int64_t n,
                                                    float dt) {
  const int64_t i0 = (int64_t(blockIdx.x) * 256 + threadIdx.x) * 8;
  if (i0 >= n) return;
  if (i0 + 8 <= n) {
    float a[8], b[8];
    load8(z, i0, a);
    load8(v, i0, b);
#pragma unroll
    for (int e = 0; e < 8; ++e) a[e] = fmaf(dt, b[e], a[e]);
    store8(z + i0, a);
  } else {
    for (int64_t i = i0; i < n; ++i) st(z, i, fmaf(dt, ld(v, i), ld(z, i)));
  }
}

int check_linear(const char* fn, int64_t M, int64_t K, int64_t N, int dtype) {
  AVITS_REQUIRE(M >= 0 && M <= INT32_MAX, "%s: M=%lld outside [0, 2^31)", fn, (long long)M);
  AVITS_REQUIRE(K >= 64 && K % 64 == 0, "%s: K=%lld must be a positive multiple of 64", fn, (long long)K);
  AVITS_REQUIRE(N >= 8 && N % 8 == 0, "%s: N=%lld must be a positive multiple of 8", fn, (long long)N);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16) return set_error(AVITS_ERR_UNSUPPORTED, "%s: dtype %d", fn, dtype);
  return AVITS_OK;
}

// out = x W^T + b (plain store epilogue, no split).
int run_linear(const void* x, int64_t M, int64_t K, const void* w, const void* b, int64_t N, int dtype, void* out,
               hipStream_t s, const char* family) {
  GemmArgs g{};
  g.nprob = 1;
  g.N = N;
  g.K = K;
  g.n_split = g.n_split2 = N;
  g.mode0 = g.mode1 = g.mode2 = EPI_STORE;
  GemmProblem& p = g.p[0];
  p.A = x; p.lda = K; p.W = w; p.bias = b; p.M = M;
  p.out0 = out; p.ld0 = N;
  return launch_gemm(g, dtype, s, family, nullptr, 0);
}

}  // namespace
}  // namespace avits

extern "C" int avits_linear(const void* x, int64_t M, int64_t K, const void* w, const void* b, int64_t N, int dtype,
                            void* out, void* stream) {
  int rc = check_linear("linear", M, K, N, dtype);
  if (rc != AVITS_OK) return rc;
  if (M == 0) return AVITS_OK;
  AVITS_REQUIRE(x && w && out, "linear: null x/w/out");
  rc = run_linear(x, M, K, w, b, N, dtype, out, static_cast<hipStream_t>(stream), "linear");
  return rc != AVITS_OK ? rc : launch_status("linear");
}

extern "C" size_t avits_final_layer_workspace_bytes(int64_t M, int64_t D, int dtype) {
  if (M < 0 || D < 1 || (dtype != AVITS_F32 && dtype != AVITS_BF16)) return 0;
  return align_up(size_t(M) * size_t(D) * (dtype == AVITS_F32 ? 4 : 2), 256);
}

extern "C" int avits_final_layer(const void* x, int64_t M, int64_t D, const void* mod, const void* w, const void* b,
                                 int64_t C, int dtype, void* out, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  int rc = check_linear("final_layer", M, D, C, dtype);
  if (rc != AVITS_OK) return rc;
  if (M == 0) return AVITS_OK;
  AVITS_REQUIRE(x && mod && w && out, "final_layer: null x/mod/w/out");
  const size_t need = avits_final_layer_workspace_bytes(M, D, dtype);
  if (!workspace || workspace_bytes < need)
    return set_error(AVITS_ERR_WORKSPACE, "final_layer: workspace of %zu bytes, need %zu", workspace_bytes, need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 rows_grid(unsigned(ceil_div64(M, 4))), blk(256);
  {
    TimedLaunch timed("ln_mod", s);
    if (dtype == AVITS_BF16) {
      const bf16_t *sh = static_cast<const bf16_t*>(mod), *sc = sh + D;
      hipLaunchKernelGGL(ln_mod_kernel<bf16_t>, rows_grid, blk, 0, s, static_cast<const bf16_t*>(x),
                         static_cast<bf16_t*>(workspace), M, D, M, sh, sc, sh, sc, ModRows{});
    } else {
      const float *sh = static_cast<const float*>(mod), *sc = sh + D;
      hipLaunchKernelGGL(ln_mod_kernel<float>, rows_grid, blk, 0, s, static_cast<const float*>(x),
                         static_cast<float*>(workspace), M, D, M, sh, sc, sh, sc, ModRows{});
    }
  }
  if ((rc = launch_status("final_layer ln_mod")) != AVITS_OK) return rc;
  rc = run_linear(workspace, M, D, w, b, C, dtype, out, s, "final_linear");
  return rc != AVITS_OK ? rc : launch_status("final_layer");
}

extern "C" int avits_euler_update(void* z, const void* v, int64_t n, float dt, int dtype, void* stream) {
  AVITS_REQUIRE(n >= 0, "euler_update: n=%lld < 0", (long long)n);
  AVITS_REQUIRE(std::isfinite(dt), "euler_update: dt=%g is not finite", dt);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "euler_update: dtype %d unsupported", dtype);
  if (n == 0) return AVITS_OK;
  AVITS_REQUIRE(z && v, "euler_update: null z/v");
  AVITS_REQUIRE(reinterpret_cast<uintptr_t>(z) % 16 == 0 && reinterpret_cast<uintptr_t>(v) % 16 == 0,
                "euler_update: z and v must be 16-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 grid(unsigned(ceil_div64(ceil_div64(n, 8), 256)));
  TimedLaunch timed("euler", s);
  if (dtype == AVITS_BF16)
    hipLaunchKernelGGL(euler_kernel<bf16_t>, grid, dim3(256), 0, s, static_cast<bf16_t*>(z),
                       static_cast<const bf16_t*>(v), n, dt);
  else
    hipLaunchKernelGGL(euler_kernel<float>, grid, dim3(256), 0, s, static_cast<float*>(z),
                       static_cast<const float*>(v), n, dt);
  return launch_status("euler_update");
}
