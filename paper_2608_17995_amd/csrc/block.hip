// One MMDiT joint-attention block on the compacted sequence (Section 3.3.1).
//
// Launch sequence (double-stream; each GEMM is one grouped launch covering
// the text rows with the text weights and the image rows with the image
// weights):
//   ln_mod(x, shift1, scale1) -> h
//   h W_qkv^T + b                       -> qkv          [S, 3D]
//   qk_rope_relayout(qkv)               -> q, k [H, S, d] (RMSNorm * g, RoPE at pos),
//                                          v^T [H, d, S padded to 64]
//   attention(q, k, v^T)                -> o [S, D], lse [H, S]
//   x + gate1 (o W_o^T + b)             -> x_mid        (fused epilogue)
//   ln_mod(x_mid, shift2, scale2)       -> h
//   GELU(h W_1^T + b)                   -> m [S, F]     (fused epilogue)
//   x_mid + gate2 (m W_2^T + b)         -> x_out        (fused epilogue)
// Single-stream: ln_mod -> one GEMM whose epilogue writes q|k|v to qkv and
// GELU(m) beside the attention output (cat = [o, GELU(m)], [S, D + F]) ->
// relayout -> attention into cat -> x + gate (cat W_out^T + b).
#include "kernels.h"

namespace avits {
namespace {

constexpr float kLnEps = 1e-6f, kRmsEps = 1e-6f;
constexpr float kLog2Theta = 13.287712379549449f;  // log2(10000)

// h = LN(x) (1 + scale) + shift, one wavefront per row; rows [0, n_a) use
// (shift_a, scale_a), the rest (shift_b, scale_b).
template <typename T>
__global__ __launch_bounds__(256) void ln_mod_kernel(const T* __restrict__ x, T* __restrict__ h, int64_t S,
                                                     int64_t D, int64_t n_a, const T* __restrict__ shift_a,
                                                     const T* __restrict__ scale_a, const T* __restrict__ shift_b,
                                                     const T* __restrict__ scale_b) {
  const int lane = threadIdx.x % kWave;
  const int64_t row = int64_t(blockIdx.x) * 4 + threadIdx.x / kWave;
  if (row >= S) return;
  const T* xr = x + row * D;
  float s = 0.f;
  for (int64_t c = lane; c < D; c += kWave) s += ld(xr, c);
  const float mean = wave_sum(s) / float(D);
  float v = 0.f;
  for (int64_t c = lane; c < D; c += kWave) {
    const float t = ld(xr, c) - mean;
    v = fmaf(t, t, v);
  }
  const float rstd = rsqrtf(wave_sum(v) / float(D) + kLnEps);
  const T* sh = row < n_a ? shift_a : shift_b;
  const T* sc = row < n_a ? scale_a : scale_b;
  T* hr = h + row * D;
  for (int64_t c = lane; c < D; c += kWave) st(hr, c, (ld(xr, c) - mean) * rstd * (1.f + ld(sc, c)) + ld(sh, c));
}

// RMSNorm + RoPE of q and k, and the per-head transpose of v.
// Workgroup: 64 sequence rows x one head.  Rows [0, n_a) use the gains of
// stream a.  q, k: [H, S, d]; vt: [H, d, ldvt], zero beyond S.
template <typename T, int DH>
__global__ __launch_bounds__(256) void qk_rope_relayout_kernel(
    const T* __restrict__ qkv, int64_t ld_qkv, const int32_t* __restrict__ pos, int64_t S, int H, int64_t n_a,
    const T* __restrict__ gq_a, const T* __restrict__ gk_a, const T* __restrict__ gq_b,
    const T* __restrict__ gk_b, T* __restrict__ q, T* __restrict__ k, T* __restrict__ vt, int64_t ldvt) {
  constexpr int kPairs = DH / 2;
  __shared__ float vs[64][DH + 1];
  const int h = blockIdx.y;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t row0 = int64_t(blockIdx.x) * 64;
  const int64_t D = int64_t(H) * DH;

  // Pair m = lane (d = 128) or lane < 32 (d = 64): axis and in-axis index.
  const int m = lane;
  const bool live = m < kPairs;
  constexpr int p0 = DH / 16, p1 = 7 * DH / 32;  // pairs per axis: (p0, p1, p1)
  const int axis = m < p0 ? 0 : (m < p0 + p1 ? 1 : 2);
  const int mi = axis == 0 ? m : (axis == 1 ? m - p0 : m - p0 - p1);
  const int na = axis == 0 ? 2 * p0 : 2 * p1;  // axis width in dims
  const float freq = exp2f(-2.f * float(mi) / float(na) * kLog2Theta);

  for (int r = wave; r < 64; r += 4) {
    const int64_t row = row0 + r;
    if (row >= S) break;
    const T* src = qkv + row * ld_qkv + int64_t(h) * DH;
    const float ang = float(pos[3 * row + axis]) * freq;
    float sn, cs;
    sincosf(ang, &sn, &cs);
    const bool a = row < n_a;
#pragma unroll
    for (int which = 0; which < 2; ++which) {
      const T* x = src + which * D;
      const T* gain = which == 0 ? (a ? gq_a : gq_b) : (a ? gk_a : gk_b);
      const float x0 = live ? ld(x, 2 * m) : 0.f, x1 = live ? ld(x, 2 * m + 1) : 0.f;
      const float ms = wave_sum(x0 * x0 + x1 * x1) / float(DH);
      const float r_ = rsqrtf(ms + kRmsEps);
      if (live) {
        const float y0 = x0 * r_ * ld(gain, 2 * m), y1 = x1 * r_ * ld(gain, 2 * m + 1);
        T* dst = (which == 0 ? q : k) + (int64_t(h) * S + row) * DH + 2 * m;
        st(dst, 0, y0 * cs - y1 * sn);
        st(dst, 1, y0 * sn + y1 * cs);
      }
    }
  }
  // v^T through LDS: read rows coalesced, write keys coalesced.
  for (int p = threadIdx.x; p < 64 * DH; p += 256) {
    const int r = p / DH, c = p % DH;
    const int64_t row = row0 + r;
    vs[r][c] = row < S ? ld(qkv + row * ld_qkv + 2 * D + int64_t(h) * DH, c) : 0.f;
  }
  __syncthreads();
  for (int p = threadIdx.x; p < 64 * DH; p += 256) {
    const int c = p / 64, r = p % 64;
    if (row0 + r < ldvt) st(vt + (int64_t(h) * DH + c) * ldvt + row0, r, vs[r][c]);
  }
}

struct BlockWs {
  char* h;
  char* qkv;
  char* q;
  char* k;
  char* vt;
  char* o;      // double: [S, D]; single: cat [S, D + F]
  char* xmid;   // double only
  char* mlp;    // double only: [S, F]
  int64_t ldvt;
  size_t bytes;
};

BlockWs block_ws_layout(char* base, int kind, int64_t S, int64_t H, int64_t d, int64_t F, int64_t esz) {
  BlockWs w{};
  const int64_t D = H * d;
  w.ldvt = ceil_div64(std::max<int64_t>(S, 1), kAttnKeyTile) * kAttnKeyTile;
  size_t off = 0;
  auto take = [&](int64_t elems) {
    char* p = base ? base + off : nullptr;
    off += align_up(size_t(elems) * size_t(esz), 256);
    return p;
  };
  w.h = take(S * D);
  w.qkv = take(S * 3 * D);
  w.q = take(H * S * d);
  w.k = take(H * S * d);
  w.vt = take(H * d * w.ldvt);
  if (kind == AVITS_BLOCK_DOUBLE) {
    w.o = take(S * D);
    w.xmid = take(S * D);
    w.mlp = take(S * F);
  } else {
    w.o = take(S * (D + F));
  }
  w.bytes = off;
  return w;
}

template <typename T>
int run_block(const void* x_in, void* x_out, const int32_t* pos, int64_t n_txt, int64_t n_img,
              const avits_block_weights* w, int H, int d, int dtype, float* lse_out, const BlockWs& ws,
              hipStream_t s) {
  const int64_t S = n_txt + n_img, D = int64_t(H) * d, F = w->mlp_hidden;
  const int64_t esz = sizeof(T);
  const bool dbl = w->kind == AVITS_BLOCK_DOUBLE;
  const T* x = static_cast<const T*>(x_in);
  T* h = reinterpret_cast<T*>(ws.h);
  T* qkv = reinterpret_cast<T*>(ws.qkv);
  const dim3 rows_grid(unsigned(ceil_div64(S, 4))), blk(256);
  int rc;

  // Per-stream views: (row offset, row count, weights) for up to two streams.
  struct Stream { int64_t r0, rows; const avits_double_stream_weights* dw; };
  Stream st2[2] = {{0, n_txt, &w->txt}, {n_txt, n_img, &w->img}};
  int nst = 0;
  Stream streams[2];
  if (dbl) {
    for (auto& t : st2)
      if (t.rows > 0) streams[nst++] = t;
  }
  auto mod_row = [&](const void* mod, int r) { return static_cast<const T*>(mod) + r * D; };

  // 1. modulated layer norm.
  if (dbl) {
    const void* ma = n_txt ? w->txt.mod : w->img.mod;
    const void* mb = n_img ? w->img.mod : w->txt.mod;
    TimedLaunch timed("ln_mod", s);
    hipLaunchKernelGGL(ln_mod_kernel<T>, rows_grid, blk, 0, s, x, h, S, D, n_txt, mod_row(ma, 0), mod_row(ma, 1),
                       mod_row(mb, 0), mod_row(mb, 1));
  } else {
    const void* mm = w->single.mod;
    TimedLaunch timed("ln_mod", s);
    hipLaunchKernelGGL(ln_mod_kernel<T>, rows_grid, blk, 0, s, x, h, S, D, S, mod_row(mm, 0), mod_row(mm, 1),
                       mod_row(mm, 0), mod_row(mm, 1));
  }
  if ((rc = launch_status("block ln_mod")) != AVITS_OK) return rc;

  // 2. QKV projection (+ the single block's MLP input, GELU'd beside o).
  {
    GemmArgs g{};
    g.K = D;
    if (dbl) {
      g.N = 3 * D;
      g.n_split = g.N;
      g.mode0 = g.mode1 = EPI_STORE;
      for (int i = 0; i < nst; ++i) {
        GemmProblem& p = g.p[i];
        p.A = h + streams[i].r0 * D; p.lda = D;
        p.W = streams[i].dw->w_qkv; p.bias = streams[i].dw->b_qkv; p.M = streams[i].rows;
        p.out0 = qkv + streams[i].r0 * 3 * D; p.ld0 = 3 * D;
      }
      g.nprob = nst;
    } else {
      g.N = 3 * D + F;
      g.n_split = 3 * D;
      g.mode0 = EPI_STORE;
      g.mode1 = EPI_GELU;
      GemmProblem& p = g.p[0];
      p.A = h; p.lda = D; p.W = w->single.w_in; p.bias = w->single.b_in; p.M = S;
      p.out0 = qkv; p.ld0 = 3 * D;
      p.out1 = reinterpret_cast<T*>(ws.o) + D; p.ld1 = D + F;
      g.nprob = 1;
    }
    if ((rc = launch_gemm(g, dtype, s)) != AVITS_OK) return rc;
  }

  // 3. q/k RMSNorm + RoPE, v transpose.
  {
    const T *gqa, *gka, *gqb, *gkb;
    int64_t na;
    if (dbl) {
      const avits_double_stream_weights& ta = n_txt ? w->txt : w->img;
      const avits_double_stream_weights& tb = n_img ? w->img : w->txt;
      gqa = static_cast<const T*>(ta.g_q); gka = static_cast<const T*>(ta.g_k);
      gqb = static_cast<const T*>(tb.g_q); gkb = static_cast<const T*>(tb.g_k);
      na = n_txt;
    } else {
      gqa = gqb = static_cast<const T*>(w->single.g_q);
      gka = gkb = static_cast<const T*>(w->single.g_k);
      na = S;
    }
    const dim3 grid(unsigned(ceil_div64(S, 64)), unsigned(H));
    TimedLaunch timed("qk_rope", s);
    if (d == 128)
      hipLaunchKernelGGL((qk_rope_relayout_kernel<T, 128>), grid, blk, 0, s, qkv, 3 * D, pos, S, H, na, gqa, gka,
                         gqb, gkb, reinterpret_cast<T*>(ws.q), reinterpret_cast<T*>(ws.k),
                         reinterpret_cast<T*>(ws.vt), ws.ldvt);
    else
      hipLaunchKernelGGL((qk_rope_relayout_kernel<T, 64>), grid, blk, 0, s, qkv, 3 * D, pos, S, H, na, gqa, gka,
                         gqb, gkb, reinterpret_cast<T*>(ws.q), reinterpret_cast<T*>(ws.k),
                         reinterpret_cast<T*>(ws.vt), ws.ldvt);
    if ((rc = launch_status("block qk_rope_relayout")) != AVITS_OK) return rc;
  }

  // 4. joint attention over all S rows.
  {
    AttnArgs a{};
    a.q = ws.q; a.q_tok = d; a.q_head = S * d;
    a.k = ws.k; a.k_tok = d; a.k_head = S * d;
    a.vt = ws.vt; a.ldvt = ws.ldvt;
    a.o = ws.o; a.ldo = dbl ? D : D + F;
    a.lse = lse_out;
    a.Sq = S; a.Sk = S; a.H = H; a.d = d;
    if ((rc = launch_attention(a, dtype, s)) != AVITS_OK) return rc;
  }

  T* out = static_cast<T*>(x_out);
  if (!dbl) {
    GemmArgs g{};
    g.N = D; g.K = D + F; g.n_split = g.N; g.mode0 = g.mode1 = EPI_RESID_GATE; g.nprob = 1;
    GemmProblem& p = g.p[0];
    p.A = ws.o; p.lda = D + F; p.W = w->single.w_out; p.bias = w->single.b_out; p.M = S;
    p.out0 = out; p.ld0 = D; p.resid = x; p.ldr = D; p.gate = mod_row(w->single.mod, 2);
    return launch_gemm(g, dtype, s);
  }

  // 5. output projection + gated residual.
  T* xmid = reinterpret_cast<T*>(ws.xmid);
  {
    GemmArgs g{};
    g.N = D; g.K = D; g.n_split = g.N; g.mode0 = g.mode1 = EPI_RESID_GATE; g.nprob = nst;
    for (int i = 0; i < nst; ++i) {
      GemmProblem& p = g.p[i];
      const int64_t r0 = streams[i].r0;
      p.A = reinterpret_cast<T*>(ws.o) + r0 * D; p.lda = D;
      p.W = streams[i].dw->w_o; p.bias = streams[i].dw->b_o; p.M = streams[i].rows;
      p.out0 = xmid + r0 * D; p.ld0 = D; p.resid = x + r0 * D; p.ldr = D;
      p.gate = mod_row(streams[i].dw->mod, 2);
    }
    if ((rc = launch_gemm(g, dtype, s)) != AVITS_OK) return rc;
  }
  // 6. second modulated layer norm.
  {
    const void* ma = n_txt ? w->txt.mod : w->img.mod;
    const void* mb = n_img ? w->img.mod : w->txt.mod;
    TimedLaunch timed("ln_mod", s);
    hipLaunchKernelGGL(ln_mod_kernel<T>, rows_grid, blk, 0, s, xmid, h, S, D, n_txt, mod_row(ma, 3), mod_row(ma, 4),
                       mod_row(mb, 3), mod_row(mb, 4));
  }
  if ((rc = launch_status("block ln_mod2")) != AVITS_OK) return rc;
  // 7. MLP in + GELU.
  T* mlp = reinterpret_cast<T*>(ws.mlp);
  {
    GemmArgs g{};
    g.N = F; g.K = D; g.n_split = g.N; g.mode0 = g.mode1 = EPI_GELU; g.nprob = nst;
    for (int i = 0; i < nst; ++i) {
      GemmProblem& p = g.p[i];
      const int64_t r0 = streams[i].r0;
      p.A = h + r0 * D; p.lda = D; p.W = streams[i].dw->w_mlp1; p.bias = streams[i].dw->b_mlp1;
      p.M = streams[i].rows; p.out0 = mlp + r0 * F; p.ld0 = F;
    }
    if ((rc = launch_gemm(g, dtype, s)) != AVITS_OK) return rc;
  }
  // 8. MLP out + gated residual.
  {
    GemmArgs g{};
    g.N = D; g.K = F; g.n_split = g.N; g.mode0 = g.mode1 = EPI_RESID_GATE; g.nprob = nst;
    for (int i = 0; i < nst; ++i) {
      GemmProblem& p = g.p[i];
      const int64_t r0 = streams[i].r0;
      p.A = mlp + r0 * F; p.lda = F; p.W = streams[i].dw->w_mlp2; p.bias = streams[i].dw->b_mlp2;
      p.M = streams[i].rows; p.out0 = out + r0 * D; p.ld0 = D; p.resid = xmid + r0 * D; p.ldr = D;
      p.gate = mod_row(streams[i].dw->mod, 5);
    }
    if ((rc = launch_gemm(g, dtype, s)) != AVITS_OK) return rc;
  }
  (void)esz;
  return AVITS_OK;
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

extern "C" int avits_block_forward(const void* x_in, void* x_out, const int32_t* pos, int64_t n_txt,
                                   int64_t n_img, const avits_block_weights* w, int32_t H, int32_t d, int dtype,
                                   float* lse_out, void* workspace, size_t workspace_bytes, void* stream) {
  AVITS_REQUIRE(w, "block_forward: null weights");
  AVITS_REQUIRE(n_txt >= 0 && n_img >= 0, "block_forward: n_txt=%lld n_img=%lld must be >= 0", (long long)n_txt,
                (long long)n_img);
  AVITS_REQUIRE(H >= 1, "block_forward: H=%d < 1", H);
  if (d != 64 && d != 128) return set_error(AVITS_ERR_UNSUPPORTED, "block_forward: head dim %d (need 64 or 128)", d);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "block_forward: dtype %d unsupported", dtype);
  AVITS_REQUIRE(w->kind == AVITS_BLOCK_DOUBLE || w->kind == AVITS_BLOCK_SINGLE, "block_forward: bad kind %d",
                w->kind);
  AVITS_REQUIRE(w->mlp_hidden >= 64 && w->mlp_hidden % 64 == 0, "block_forward: mlp_hidden=%d must be a positive multiple of 64",
                w->mlp_hidden);
  const int64_t S = n_txt + n_img;
  AVITS_REQUIRE(S <= INT32_MAX, "block_forward: S=%lld too large", (long long)S);
  if (S == 0) return AVITS_OK;
  AVITS_REQUIRE(x_in && x_out && pos, "block_forward: null x_in/x_out/pos");
  AVITS_REQUIRE(x_in != x_out, "block_forward: x_out must not alias x_in");
  if (w->kind == AVITS_BLOCK_DOUBLE) {
    AVITS_REQUIRE(n_txt == 0 || all_set(w->txt), "block_forward: missing text-stream weight");
    AVITS_REQUIRE(n_img == 0 || all_set(w->img), "block_forward: missing image-stream weight");
  } else {
    const avits_single_weights& sw = w->single;
    AVITS_REQUIRE(sw.mod && sw.w_in && sw.b_in && sw.g_q && sw.g_k && sw.w_out && sw.b_out,
                  "block_forward: missing single-block weight");
  }
  const int64_t esz = dtype == AVITS_F32 ? 4 : 2;
  const BlockWs need = block_ws_layout(nullptr, w->kind, S, H, d, w->mlp_hidden, esz);
  if (!workspace || workspace_bytes < need.bytes)
    return set_error(AVITS_ERR_WORKSPACE, "block_forward: workspace of %zu bytes, need %zu", workspace_bytes,
                     need.bytes);
  const BlockWs ws = block_ws_layout(static_cast<char*>(workspace), w->kind, S, H, d, w->mlp_hidden, esz);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == AVITS_BF16) return run_block<bf16_t>(x_in, x_out, pos, n_txt, n_img, w, H, d, dtype, lse_out, ws, s);
  return run_block<float>(x_in, x_out, pos, n_txt, n_img, w, H, d, dtype, lse_out, ws, s);
}
