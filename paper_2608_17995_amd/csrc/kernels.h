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
  EPI_STORE_T = 3,     // out[col * ld + m] = C (transposed store)
};

// Several images packed in one block pass (rows packed by stream: the text
// rows of images 0..B-1, then their image rows), each with its own
// modulation vectors: rows [end[i-1], end[i]) of the packed sequence form
// segment i (end[-1] = 0), segments 0..B-1 hold the images' text rows and
// B..2B-1 their image rows, and segment i's rows use the modulation block of
// image i mod B, `stride` elements after the previous image's.  B == 0: one
// modulation for every row.
constexpr int kMaxSeqs = 16;
struct ModRows {
  int32_t B;
  int64_t stride;
  int64_t end[2 * kMaxSeqs];
};

// Element offset of packed row `row`'s modulation block.  The loop is
// unrolled over the whole array so every index is static (a dynamically
// indexed kernel-argument array would be copied to private memory).
__device__ __forceinline__ int64_t mod_offset(const ModRows& m, int64_t row) {
  if (m.B == 0) return 0;
  int seg = 0;
#pragma unroll
  for (int i = 0; i < 2 * kMaxSeqs - 1; ++i) seg += (i < 2 * m.B - 1 && row >= m.end[i]) ? 1 : 0;
  return int64_t(seg < m.B ? seg : seg - m.B) * m.stride;
}

// Output columns are split into up to three regions, [0, n_split),
// [n_split, n_split2) and [n_split2, N); region r writes out_r with row
// stride ld_r at column (n - region start) and applies mode_r.
struct GemmProblem {
  const void* A;       // [M, lda]
  int64_t lda;
  const void* W;       // [N, K]
  const void* bias;    // [N] or null
  int64_t M;
  void* out0;
  int64_t ld0;
  void* out1;
  int64_t ld1;
  void* out2;
  int64_t ld2;
  const void* resid;   // EPI_RESID_GATE: [M, ldr], same columns as the region
  int64_t ldr;
  const void* gate;    // EPI_RESID_GATE: [N]
  // Optional second destination of region 0's final rows (the Stage-3
  // scatter fused into a block's last projection): row m >= scat_row0 also
  // goes to scat[scat_idx[m - scat_row0] * scat_ld + column] when that index
  // lies in [0, scat_n).
  void* scat;
  const int32_t* scat_idx;
  int64_t scat_row0, scat_ld, scat_n;
  int64_t row0;        // packed row of the problem's row 0 (for `mod` below)
};

struct GemmArgs {
  GemmProblem p[2];
  int nprob;
  int64_t N, K;
  int64_t n_split, n_split2;  // region starts; >= N when unused
  int mode0, mode1, mode2;
  // Per-image gates (EPI_RESID_GATE) and post-LN modulation: row m of
  // problem p takes gate + mod_offset(mod, p.row0 + m).  Applied by the
  // split-K reduce kernels, so launch_gemm runs such a projection split.
  ModRows mod;
};

struct GemmPlan {
  int bn = 0;          // column tile
  int splits = 1;      // K splits (fp32 partials + reduce when > 1)
  int waves = 8;       // waves per workgroup
  int stages = 2;      // register staging depth of the k-tile pipeline (1 or 2)
  int64_t tiles = 0;   // output tiles
  int64_t tail = 0;    // last tiles run in tail_splits k splits (256-wide tile, splits == 1)
  int tail_splits = 1;
};
GemmPlan plan_gemm(const GemmArgs& a, int dtype, size_t partial_bytes, const char* family = nullptr);
size_t gemm_partial_bytes(const GemmArgs& a, const GemmPlan& pl);
// `partial` is scratch for split-K partial sums; when it is null or smaller
// than the plan needs, the GEMM runs unsplit.
// `family` names the timing family of the launch (see avits_timing_read).
// Optional modulated layer norm of the GEMM's output rows, fused into the
// split-K reduce when the GEMM is split: out = LN(y) * (1 + scale[p]) +
// shift[p] for the rows of problem p (offset per image by the launch's
// ModRows), y the bf16 result rows (layer norm
// without affine, eps 1e-6, biased variance, as the block's other LN).
// `done` reports whether it ran; when not, the caller normalises itself.
struct GemmPostLN {
  void* out;
  int64_t ld;
  const void* shift[2];
  const void* scale[2];
  bool done;
};

int launch_gemm(const GemmArgs& a, int dtype, hipStream_t s, const char* family, float* partial = nullptr,
                size_t partial_bytes = 0, GemmPostLN* post_ln = nullptr);

// Bytes of split-K scratch the block reserves: up to 4 splits of an [S, D] fp32 output.
inline size_t gemm_partial_reserve(int64_t S, int64_t D) { return size_t(4) * size_t(S) * size_t(D) * sizeof(float); }

// ----------------------------------------------------------------------------
// Flash attention over one sequence, all heads.  q/k are addressed as
// base + token * tok_stride + head * head_stride (elements); v is given
// transposed per head, vt[h][c][key] with row stride ldvt >= Sk rounded up to
// the key tile (the padding keys are read but masked, whatever they hold);
// o is [Sq, H*d] with row stride ldo.  Without v (vt == null) only the
// log-sum-exp is produced.
// Block-diagonal attention over packed sequences: sequence b is the union
// of two row ranges (its text rows and its image rows when the rows are
// packed by stream); its rows attend to its own rows only.
struct AttnSegs {
  int n;                        // 0: one sequence, all rows (no segments)
  int64_t start[kMaxSeqs][2];
  int64_t len[kMaxSeqs][2];
};

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
  float* mass;         // [H, Sq] or null: softmax mass of keys [0, mass_keys) (the text keys)
  int64_t mass_keys;
  int mass_accumulate; // add to `mass` instead of overwriting it
  int64_t Sq, Sk;
  int H, d;
  AttnSegs segs;       // n > 0: queries and keys per sequence (Sq == Sk == packed rows)
  // Scratch for the split tail (bf16 with V, one sequence): the last units of
  // the grid may run in key pieces whose unnormalised partial outputs are
  // combined by a second kernel.  Null: never split.
  float* part;
  size_t part_bytes;
  float* part_ml;      // set by the launcher: (max, sum, text sum, 0) per piece row, after the outputs
  int64_t split_from;  // set by the launcher: units >= split_from run in ksp pieces
  int ksp;
};

constexpr int kAttnKeyTile = 64;  // key padding unit expected for vt

int launch_attention(const AttnArgs& a, int dtype, hipStream_t s);

inline int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace avits
