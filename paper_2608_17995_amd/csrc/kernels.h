// Internal launchers shared between the translation units of libavits.
#pragma once

#include <algorithm>

#include "common.h"

namespace avits {

// ----------------------------------------------------------------------------
// GEMM: C[m, n] = sum_k A[m, k] * W[n, k] + bias[n], followed by an epilogue.
// Up to two independent problems (the text and image streams of a double
// block) share one launch; they share N, K and the epilogue modes.
enum EpiMode : int {
  EPI_STORE = 0,       // out = C
  EPI_GELU = 1,        // out = GELU_tanh(C)
  EPI_RESID_GATE = 2,  // out = resid + gate[n] * C
};

struct GemmProblem {
  const void* A;       // [M, lda]
  int64_t lda;
  const void* W;       // [N, K]
  const void* bias;    // [N] or null
  int64_t M;
  // Output columns n < n_split go to out0 (row stride ld0, column n),
  // the others to out1 (row stride ld1, column n - n_split).
  void* out0;
  int64_t ld0;
  void* out1;
  int64_t ld1;
  const void* resid;   // EPI_RESID_GATE: [M, ldr], same columns as out0
  int64_t ldr;
  const void* gate;    // EPI_RESID_GATE: [N]
};

struct GemmArgs {
  GemmProblem p[2];
  int nprob;
  int64_t N, K;
  int64_t n_split;     // >= N when the output is not split
  int mode0, mode1;
};

int launch_gemm(const GemmArgs& a, int dtype, hipStream_t s);

// ----------------------------------------------------------------------------
// Flash attention over one sequence, all heads.  q/k are addressed as
// base + token * tok_stride + head * head_stride (elements); v is given
// transposed per head, vt[h][c][key] with row stride ldvt >= Sk rounded up to
// the key tile (the padding must hold finite values); o is [Sq, H*d] with row
// stride ldo.  Without v (vt == null) only the log-sum-exp is produced.
struct AttnArgs {
  const void* q;
  int64_t q_tok, q_head;
  const void* k;
  int64_t k_tok, k_head;
  const void* vt;      // [H, d, ldvt] or null
  int64_t ldvt;
  void* o;             // [Sq, ldo] or null
  int64_t ldo;
  float* lse;          // [H, Sq] or null
  int64_t Sq, Sk;
  int H, d;
};

constexpr int kAttnKeyTile = 64;  // key padding unit expected for vt

int launch_attention(const AttnArgs& a, int dtype, hipStream_t s);

inline int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace avits
