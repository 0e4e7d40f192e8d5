// Stage-2 gather / 2x upsample and Stage-3 scatter (Section 3.2).
//
// Pure data movement, HBM-bound.  Each wavefront moves one token row at a time
// with 16-byte vector accesses; a row is D elements (6 KiB for D = 3072 bf16).
// One launch covers every row job of the gather so small grids never idle the
// chip: prefix copies, selected-row copies (+ their positions) and the
// upsampled fill of unselected canvas rows (nearest: one job per low-res
// token, which reads its row once and writes its unselected 2x2 children;
// bilinear: one job per high-res pixel).
#include "common.h"
#include "ln_row.h"

namespace avits {
namespace {

constexpr int kRowsPerBlock = 4;  // one wavefront per row job

// Row copies by the 64 lanes of a wave: every lane loads up to kCopyBatch
// 16-byte chunks (lane + 64 u) before storing any, so a row of up to 8 KB is
// one round trip.  `n` counts 16-byte chunks; i0 is the batch's first chunk.
constexpr int kCopyBatch = 8;
__device__ __forceinline__ void load_chunks(const u32x4* __restrict__ s, int n, int i0, int lane,
                                            u32x4 (&r)[kCopyBatch]) {
  const u32x4* sl = s + (i0 + lane);  // one 64-bit base; chunk u at +1 KiB u
  const int left = n - (i0 + lane);
#pragma unroll
  for (int u = 0; u < kCopyBatch; ++u)
    if (u * kWave < left) r[u] = sl[u * kWave];
}
__device__ __forceinline__ void store_chunks(u32x4* __restrict__ d, int n, int i0, int lane,
                                             const u32x4 (&r)[kCopyBatch]) {
  u32x4* dl = d + (i0 + lane);
  const int left = n - (i0 + lane);
#pragma unroll
  for (int u = 0; u < kCopyBatch; ++u)
    if (u * kWave < left) dl[u * kWave] = r[u];
}

// A row of n <= 64 kCopyBatch chunks into registers with unconditional
// loads: lanes past the row's end read its last chunk again (the value is
// never used), so there is no branch per chunk and the compiler keeps one
// copy of the array.
__device__ __forceinline__ void load_row_clamped(const u32x4* __restrict__ s, int n, int lane,
                                                 u32x4 (&r)[kCopyBatch]) {
#pragma unroll
  for (int u = 0; u < kCopyBatch; ++u) r[u] = s[min(lane + u * kWave, n - 1)];
}

// Copy `bytes` (multiple of 16) from src to dst; chunks from `from` on.
__device__ __forceinline__ void wave_copy_row(const char* __restrict__ src, char* __restrict__ dst,
                                              int64_t bytes, int lane, int64_t from = 0) {
  const u32x4* s = reinterpret_cast<const u32x4*>(src);
  u32x4* d = reinterpret_cast<u32x4*>(dst);
  const int n = int(bytes / 16);
#pragma unroll 1
  for (int i0 = int(from); i0 < n; i0 += kCopyBatch * kWave) {
    u32x4 r[kCopyBatch];
    load_chunks(s, n, i0, lane, r);
    store_chunks(d, n, i0, lane, r);
  }
}

// First position in the ascending idx[0..k) not below p.
// Number of entries of the ascending idx[0, k) below p, by the whole wave
// (p uniform): each round samples 64 evenly spaced entries of the remaining
// range [lo, hi] in one load and keeps the stretch between the last sample
// below p and the first at or above it, so k <= 4096 takes two dependent
// loads instead of a binary search's twelve.
__device__ __forceinline__ int64_t wave_lower_bound(const int32_t* idx, int64_t k, int64_t p, int lane) {
  int64_t lo = 0, hi = k;  // the answer lies in [lo, hi]
  while (hi - lo > kWave) {
    const int64_t step = (hi - lo + kWave - 1) / kWave;
    const int64_t at = lo + int64_t(lane) * step;
    const int c = __popcll(__ballot(at < hi && idx[at] < p));  // samples below p
    if (c == 0) return lo;
    const int64_t nhi = std::min<int64_t>(hi, lo + int64_t(c) * step);
    lo += int64_t(c - 1) * step + 1;
    hi = nhi;
  }
  const int64_t at = lo + lane;
  return lo + __popcll(__ballot(at < hi && idx[at] < p));
}

template <typename T>
__device__ __forceinline__ void bilinear_row(const T* __restrict__ low, T* __restrict__ dst, int64_t p,
                                             int H_lr, int W_lr, int64_t D, int lane) {
  const int W_hr = 2 * W_lr;
  const int r = int(p / W_hr), c = int(p % W_hr);
  // Source coordinate (o + 0.5)/2 - 0.5 clamped at 0; taps clamped to the grid.
  auto taps = [](int o, int n, int& i0, int& i1, float& w1) {
    float src = fmaxf((o + 0.5f) * 0.5f - 0.5f, 0.f);
    i0 = min(int(floorf(src)), n - 1);
    i1 = min(i0 + 1, n - 1);
    w1 = src - float(i0);
  };
  int r0, r1, c0, c1;
  float wr1, wc1;
  taps(r, H_lr, r0, r1, wr1);
  taps(c, W_lr, c0, c1, wc1);
  const float wr0 = 1.f - wr1, wc0 = 1.f - wc1;
  const T* a = low + (int64_t(r0) * W_lr + c0) * D;
  const T* b = low + (int64_t(r0) * W_lr + c1) * D;
  const T* e = low + (int64_t(r1) * W_lr + c0) * D;
  const T* f = low + (int64_t(r1) * W_lr + c1) * D;
  for (int64_t i = lane; i < D; i += kWave) {
    // Rows first, then columns (the order of the separable definition).
    float left = wr0 * ld(a, i) + wr1 * ld(e, i);
    float right = wr0 * ld(b, i) + wr1 * ld(f, i);
    st(dst, i, wc0 * left + wc1 * right);
  }
}

// Where image b of a stack finds its selection and puts its rows: idx
// entries [idx_off[b], idx_off[b + 1]), compact rows from row_off[b], pos
// rows from pos_off[b].  A single image is the stack of one.
constexpr int kMaxRelayoutImages = 64;
struct ImageRows {
  int64_t idx_off[kMaxRelayoutImages + 1];
  int64_t row_off[kMaxRelayoutImages];
  int64_t pos_off[kMaxRelayoutImages];
};

// Optional output of the gather (one image, bf16): the modulated layer norm
// of every compact row, h = LN(row)(1 + scale) + shift, with (shift_a,
// scale_a) for rows [0, n_a) and (shift_b, scale_b) for the others: the
// first stage of the block that takes the compact rows, computed while the
// row is in registers.
struct LnOut {
  bf16_t* h;  // [n_prefix + k, D], or null: no layer norm
  int64_t n_a;
  const bf16_t *shift_a, *scale_a, *shift_b, *scale_b;
};
static_assert(kCopyBatch == kLnMaxChunks, "a fused row must fit the layer norm's register layout");

// Compact row `row`: its scale and shift chunks (issued right after the
// row's own loads, so both latencies overlap), then its LN once the row is
// in r (lane + 64 u).
__device__ __forceinline__ void ln_vectors_of_row(const LnOut& ln, int64_t row, int64_t D, int lane,
                                                  u32x4 (&g)[kLnMaxChunks], u32x4 (&t)[kLnMaxChunks]) {
  const bool a = row < ln.n_a;
  ln_mod_vectors(a ? ln.shift_a : ln.shift_b, a ? ln.scale_a : ln.scale_b, D / 8, lane, g, t);
}
__device__ __forceinline__ void ln_of_row(const LnOut& ln, int64_t row, int64_t D, int lane,
                                          const u32x4 (&r)[kCopyBatch], const u32x4 (&g)[kLnMaxChunks],
                                          const u32x4 (&t)[kLnMaxChunks]) {
  ln_mod_row_bf16(r, g, t, D / 8, D, lane, ln.h + row * D);
}

// Image blockIdx.y of a stack of equally shaped images (lowres [B, N/4, D],
// highres / canvas [B, N, D], prefix [B, n_prefix, D]).
template <typename T>
__global__ __launch_bounds__(kWave * kRowsPerBlock) void gather_upsample_kernel(
    const T* __restrict__ lowres, const T* highres, const T* __restrict__ prefix,
    const int32_t* __restrict__ idx, const ImageRows im, int H_lr, int W_lr, int64_t n_prefix, int64_t D,
    int mode, T* __restrict__ compact, int32_t* __restrict__ pos_sel, T* canvas, int canvas_aliases,
    const LnOut ln) {
  const int lane = threadIdx.x % kWave;
  const int64_t job = int64_t(blockIdx.x) * kRowsPerBlock + threadIdx.x / kWave;
  const int W_hr = 2 * W_lr;
  const int64_t N = int64_t(4) * H_lr * W_lr;
  const int64_t row_bytes = D * int64_t(sizeof(T));
  const int b = blockIdx.y;
  const int64_t k = im.idx_off[b + 1] - im.idx_off[b];
  lowres += int64_t(b) * (N / 4) * D;
  highres += int64_t(b) * N * D;
  canvas += int64_t(b) * N * D;
  if (prefix) prefix += int64_t(b) * n_prefix * D;
  idx += im.idx_off[b];
  compact += im.row_off[b] * D;
  pos_sel += im.pos_off[b] * 3;
  if (job < n_prefix) {
    if constexpr (sizeof(T) == 2) {
      if (ln.h) {  // the row fits one batch (the host checks D)
        const int n = int(row_bytes / 16);
        u32x4 r[kCopyBatch], g[kLnMaxChunks], t[kLnMaxChunks];
        load_row_clamped(reinterpret_cast<const u32x4*>(prefix + job * D), n, lane, r);
        ln_vectors_of_row(ln, job, D, lane, g, t);
        store_chunks(reinterpret_cast<u32x4*>(compact + job * D), n, 0, lane, r);
        ln_of_row(ln, job, D, lane, r, g, t);
        return;
      }
    }
    wave_copy_row(reinterpret_cast<const char*>(prefix + job * D),
                  reinterpret_cast<char*>(compact + job * D), row_bytes, lane);
    return;
  }
  int64_t j = job - n_prefix;
  if (j < k) {
    const int64_t p = idx[j];
    if (p < 0 || p >= N) return;  // outside the grid: nothing is read or written for it
    // One read of the high-resolution row feeds the compact row and, when
    // the canvas is a separate buffer, the canvas row.
    const u32x4* src = reinterpret_cast<const u32x4*>(highres + p * D);
    u32x4* to_compact = reinterpret_cast<u32x4*>(compact + (n_prefix + j) * D);
    u32x4* to_canvas = reinterpret_cast<u32x4*>(canvas + p * D);
    const int n = int(row_bytes / 16);
    bool done = false;
    if constexpr (sizeof(T) == 2) {
      if (ln.h) {  // one batch holds the row
        u32x4 r[kCopyBatch], g[kLnMaxChunks], t[kLnMaxChunks];
        load_row_clamped(src, n, lane, r);
        ln_vectors_of_row(ln, n_prefix + j, D, lane, g, t);
        store_chunks(to_compact, n, 0, lane, r);
        if (!canvas_aliases) store_chunks(to_canvas, n, 0, lane, r);
        ln_of_row(ln, n_prefix + j, D, lane, r, g, t);
        done = true;
      }
    }
#pragma unroll 1
    for (int i0 = 0; !done && i0 < n; i0 += kCopyBatch * kWave) {
      u32x4 r[kCopyBatch];
      load_chunks(src, n, i0, lane, r);
      store_chunks(to_compact, n, i0, lane, r);
      if (!canvas_aliases) store_chunks(to_canvas, n, i0, lane, r);
    }
    if (lane == 0) {
      pos_sel[3 * j + 0] = 0;
      pos_sel[3 * j + 1] = int32_t(p / W_hr);
      pos_sel[3 * j + 2] = int32_t(p % W_hr);
    }
    return;
  }
  if (mode == AVITS_UP_NEAREST) {
    // Low-res token q: its children p00, p00 + 1 (row 2r) and p10, p10 + 1
    // (row 2r + 1) all take its row; the selected ones (idx ascending and
    // unique, so p00 + 1 follows p00 there if both are in it) are skipped.
    const int64_t q = j - k;
    if (q >= N / 4) return;
    const int64_t p00 = 2 * (q / W_lr) * W_hr + 2 * (q % W_lr), p10 = p00 + W_hr;
    const int64_t a0 = wave_lower_bound(idx, k, p00, lane), a1 = wave_lower_bound(idx, k, p10, lane);
    const bool s00 = a0 < k && idx[a0] == p00;
    const bool s01 = a0 + s00 < k && idx[a0 + s00] == p00 + 1;
    const bool s10 = a1 < k && idx[a1] == p10;
    const bool s11 = a1 + s10 < k && idx[a1 + s10] == p10 + 1;
    const u32x4* src = reinterpret_cast<const u32x4*>(lowres + q * D);
    u32x4* const dst[4] = {reinterpret_cast<u32x4*>(canvas + p00 * D), reinterpret_cast<u32x4*>(canvas + (p00 + 1) * D),
                           reinterpret_cast<u32x4*>(canvas + p10 * D), reinterpret_cast<u32x4*>(canvas + (p10 + 1) * D)};
    const bool keep[4] = {!s00, !s01, !s10, !s11};
    const int n = int(row_bytes / 16);
#pragma unroll 1
    for (int i0 = 0; i0 < n; i0 += kCopyBatch * kWave) {
      u32x4 r[kCopyBatch];
      load_chunks(src, n, i0, lane, r);
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (keep[c]) store_chunks(dst[c], n, i0, lane, r);
    }
    return;
  }
  const int64_t p = j - k;
  if (p >= N) return;
  const int64_t at = wave_lower_bound(idx, k, p, lane);
  if (at < k && idx[at] == p) return;  // selected: handled by its own job
  bilinear_row(lowres, canvas + p * D, p, H_lr, W_lr, D, lane);
}

// Image blockIdx.y: its selection idx[idx_off[b] ..), its rows of `out`
// from row_off[b], its canvas at b N D.
template <typename T>
__global__ __launch_bounds__(kWave * kRowsPerBlock) void scatter_kernel(
    const T* __restrict__ out, const int32_t* __restrict__ idx, const ImageRows im, int64_t N,
    int64_t D, T* __restrict__ canvas) {
  const int lane = threadIdx.x % kWave;
  const int64_t j = int64_t(blockIdx.x) * kRowsPerBlock + threadIdx.x / kWave;
  const int b = blockIdx.y;
  const int64_t k = im.idx_off[b + 1] - im.idx_off[b];
  if (j >= k) return;
  idx += im.idx_off[b];
  const int64_t row_offset = im.row_off[b];
  canvas += int64_t(b) * N * D;
  const int64_t p = idx[j];
  if (p < 0 || p >= N) return;  // outside the canvas: skipped
  wave_copy_row(reinterpret_cast<const char*>(out + (row_offset + j) * D),
                reinterpret_cast<char*>(canvas + p * D), D * int64_t(sizeof(T)), lane);
}

// ---------------------------------------------------------------------------
// The mixed-resolution sequence of Stage 2 (Section 3.2): the K selected
// low-res tokens are expanded to their four high-res children, the other
// M' - K stay at low resolution, all in one sequence behind the prefix.
// Rows: parent idx[j]'s children at 4j + 2 dr + dc (raster order inside the
// 2x2 block), then the kept parents in ascending order.  Positions are in
// half units (twice the high-res coordinate): a child (2r+dr, 2c+dc) sits at
// (0, 2(2r+dr), 2(2c+dc)), a kept token at its block centre (0, 4r+1, 4c+1).
//
// One wave per low-res parent.  A selected parent's four rows are written
// from one read of its low-res row (nearest) or interpolated per child
// (bilinear); a kept parent is one row copy.  Row slots are derived from the
// parent's rank in idx, and are bounds-checked so that an idx that is not
// ascending and unique cannot write outside the buffers.

// Copy one row of `bytes` (multiple of 16) to four destinations.
__device__ __forceinline__ void wave_fan_row(const char* __restrict__ src, char* d0, char* d1, char* d2,
                                             char* d3, int64_t bytes, int lane) {
  const u32x4* s = reinterpret_cast<const u32x4*>(src);
  const int64_t n = bytes / 16;
  for (int64_t i = lane; i < n; i += kWave) {
    const u32x4 v = s[i];
    reinterpret_cast<u32x4*>(d0)[i] = v;
    reinterpret_cast<u32x4*>(d1)[i] = v;
    reinterpret_cast<u32x4*>(d2)[i] = v;
    reinterpret_cast<u32x4*>(d3)[i] = v;
  }
}

template <typename T>
__global__ __launch_bounds__(kWave * kRowsPerBlock) void gather_mixed_kernel(
    const T* __restrict__ lowres, const T* __restrict__ prefix, const int32_t* __restrict__ idx, int64_t k,
    int H_lr, int W_lr, int64_t n_prefix, int64_t D, int mode, T* __restrict__ compact,
    int32_t* __restrict__ pos, int32_t* __restrict__ children) {
  const int lane = threadIdx.x % kWave;
  const int64_t job = int64_t(blockIdx.x) * kRowsPerBlock + threadIdx.x / kWave;
  const int64_t Mp = int64_t(H_lr) * W_lr;
  const int64_t row_bytes = D * int64_t(sizeof(T));
  if (job < n_prefix) {
    wave_copy_row(reinterpret_cast<const char*>(prefix + job * D),
                  reinterpret_cast<char*>(compact + job * D), row_bytes, lane);
    return;
  }
  const int64_t p = job - n_prefix;
  if (p >= Mp) return;
  const int r = int(p / W_lr), c = int(p % W_lr);
  const int64_t at = wave_lower_bound(idx, k, p, lane);
  T* body = compact + n_prefix * D;
  if (at < k && idx[at] == p) {
    const int W_hr = 2 * W_lr;
    T* dst[4];
    for (int ch = 0; ch < 4; ++ch) dst[ch] = body + (4 * at + ch) * D;
    if (mode == AVITS_UP_NEAREST) {
      wave_fan_row(reinterpret_cast<const char*>(lowres + p * D), reinterpret_cast<char*>(dst[0]),
                   reinterpret_cast<char*>(dst[1]), reinterpret_cast<char*>(dst[2]),
                   reinterpret_cast<char*>(dst[3]), row_bytes, lane);
    } else {
      for (int ch = 0; ch < 4; ++ch)
        bilinear_row(lowres, dst[ch], int64_t(2 * r + (ch >> 1)) * W_hr + 2 * c + (ch & 1), H_lr, W_lr, D, lane);
    }
    // Selected parents of low-res rows before r, and before r + 1.
    const int64_t row0 = children ? wave_lower_bound(idx, k, int64_t(r) * W_lr, lane) : 0;
    const int64_t row1 = children ? wave_lower_bound(idx, k, int64_t(r + 1) * W_lr, lane) : 0;
    if (lane < 4) {
      const int dr = lane >> 1, dc = lane & 1;
      int32_t* ps = pos + 3 * (4 * at + lane);
      ps[0] = 0;
      ps[1] = 2 * (2 * r + dr);
      ps[2] = 2 * (2 * c + dc);
      if (children) {
        // Rank of child (2r+dr, 2c+dc) among all children in high-res raster
        // order: the children of earlier low-res rows, then row 2r+dr's
        // share of this row's selected parents, then the parents to the left.
        const int64_t rank = 4 * row0 + dr * 2 * (row1 - row0) + 2 * (at - row0) + dc;
        if (rank >= 0 && rank < 4 * k) children[rank] = int32_t(int64_t(2 * r + dr) * W_hr + 2 * c + dc);
      }
    }
    return;
  }
  const int64_t slot = p - at;  // kept parents before p
  if (slot < 0 || slot >= Mp - k) return;
  wave_copy_row(reinterpret_cast<const char*>(lowres + p * D),
                reinterpret_cast<char*>(body + (4 * k + slot) * D), row_bytes, lane);
  if (lane == 0) {
    int32_t* ps = pos + 3 * (4 * k + slot);
    ps[0] = 0;
    ps[1] = 4 * r + 1;
    ps[2] = 4 * c + 1;
  }
}

template <typename T>
__global__ __launch_bounds__(kWave * kRowsPerBlock) void scatter_mixed_kernel(
    const T* __restrict__ out, const int32_t* __restrict__ idx, int64_t k, int H_lr, int W_lr,
    int64_t row_offset, int64_t D, T* __restrict__ canvas_hr, T* __restrict__ state_lr) {
  const int lane = threadIdx.x % kWave;
  const int64_t p = int64_t(blockIdx.x) * kRowsPerBlock + threadIdx.x / kWave;
  const int64_t Mp = int64_t(H_lr) * W_lr;
  if (p >= Mp) return;
  const int64_t row_bytes = D * int64_t(sizeof(T));
  const int64_t at = wave_lower_bound(idx, k, p, lane);
  const T* body = out + row_offset * D;
  if (at < k && idx[at] == p) {
    const int r = int(p / W_lr), c = int(p % W_lr), W_hr = 2 * W_lr;
    for (int ch = 0; ch < 4; ++ch) {
      const int64_t q = int64_t(2 * r + (ch >> 1)) * W_hr + 2 * c + (ch & 1);
      wave_copy_row(reinterpret_cast<const char*>(body + (4 * at + ch) * D),
                    reinterpret_cast<char*>(canvas_hr + q * D), row_bytes, lane);
    }
    return;
  }
  const int64_t slot = p - at;
  if (slot < 0 || slot >= Mp - k) return;
  wave_copy_row(reinterpret_cast<const char*>(body + (4 * k + slot) * D),
                reinterpret_cast<char*>(state_lr + p * D), row_bytes, lane);
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace
}  // namespace avits

using namespace avits;

namespace {

// One launch over the B images of `im`; k_max is the largest selection.
int launch_gather(const void* lowres, const void* highres_prev, const void* prefix, const int32_t* idx,
                  const ImageRows& im, int B, int64_t k_max, int32_t H_lr, int32_t W_lr, int64_t n_prefix,
                  int64_t D, int mode, int dtype, void* compact, int32_t* pos_sel, void* canvas, void* stream,
                  const char* who, const LnOut& ln = LnOut{}) {
  const int64_t N = int64_t(4) * H_lr * W_lr;
  const int64_t jobs = n_prefix + k_max + (mode == AVITS_UP_NEAREST ? N / 4 : N);
  const dim3 grid(unsigned(ceil_div(jobs, kRowsPerBlock)), unsigned(B)), block(kWave * kRowsPerBlock);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int alias = canvas == highres_prev;
  TimedLaunch timed("gather_upsample", s);
  if (dtype == AVITS_F32)
    hipLaunchKernelGGL(gather_upsample_kernel<float>, grid, block, 0, s, (const float*)lowres,
                       (const float*)highres_prev, (const float*)prefix, idx, im, H_lr, W_lr, n_prefix, D,
                       mode, (float*)compact, pos_sel, (float*)canvas, alias, LnOut{});
  else
    hipLaunchKernelGGL(gather_upsample_kernel<bf16_t>, grid, block, 0, s, (const bf16_t*)lowres,
                       (const bf16_t*)highres_prev, (const bf16_t*)prefix, idx, im, H_lr, W_lr, n_prefix, D,
                       mode, (bf16_t*)compact, pos_sel, (bf16_t*)canvas, alias, ln);
  return launch_status(who);
}

int launch_scatter(const void* out, const int32_t* idx, const ImageRows& im, int B, int64_t k_max, int64_t N,
                   int64_t D, int dtype, void* canvas, void* stream, const char* who) {
  const dim3 grid(unsigned(ceil_div(k_max, kRowsPerBlock)), unsigned(B)), block(kWave * kRowsPerBlock);
  hipStream_t s = static_cast<hipStream_t>(stream);
  TimedLaunch timed("scatter", s);
  if (dtype == AVITS_F32)
    hipLaunchKernelGGL(scatter_kernel<float>, grid, block, 0, s, (const float*)out, idx, im, N, D, (float*)canvas);
  else
    hipLaunchKernelGGL(scatter_kernel<bf16_t>, grid, block, 0, s, (const bf16_t*)out, idx, im, N, D,
                       (bf16_t*)canvas);
  return launch_status(who);
}

__global__ __launch_bounds__(256) void grid_positions_kernel(int32_t* __restrict__ pos, int64_t rows, int W,
                                                             int frame, int scale, int offset) {
  const int64_t r = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (r >= rows) return;
  pos[3 * r + 0] = frame;
  pos[3 * r + 1] = int32_t(r / W) * scale + offset;
  pos[3 * r + 2] = int32_t(r % W) * scale + offset;
}

__global__ __launch_bounds__(256) void scale_positions_kernel(const int32_t* src, int64_t n, int scale,
                                                              int32_t* dst) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) dst[i] = src[i] * scale;
}

}  // namespace

extern "C" int avits_grid_positions(int32_t* pos, int64_t rows, int32_t W, int32_t frame, int32_t scale,
                                    int32_t offset, void* stream) {
  AVITS_REQUIRE(rows >= 0 && W >= 1, "grid_positions: rows=%lld W=%d", (long long)rows, W);
  AVITS_REQUIRE(rows <= INT32_MAX, "grid_positions: rows=%lld beyond 2^31", (long long)rows);
  if (rows == 0) return AVITS_OK;
  AVITS_REQUIRE(pos, "grid_positions: null pos");
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(grid_positions_kernel, dim3(unsigned(ceil_div(rows, 256))), dim3(256), 0, s, pos, rows, W, frame,
                     scale, offset);
  return launch_status("grid_positions");
}

extern "C" int avits_scale_positions(const int32_t* src, int64_t rows, int32_t scale, int32_t* dst, void* stream) {
  AVITS_REQUIRE(rows >= 0 && rows <= INT32_MAX / 3, "scale_positions: rows=%lld", (long long)rows);
  if (rows == 0) return AVITS_OK;
  AVITS_REQUIRE(src && dst, "scale_positions: null src/dst");
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(scale_positions_kernel, dim3(unsigned(ceil_div(3 * rows, 256))), dim3(256), 0, s, src, 3 * rows,
                     scale, dst);
  return launch_status("scale_positions");
}

extern "C" int avits_gather_upsample(const void* lowres, const void* highres_prev, const void* prefix,
                                     const int32_t* idx, int64_t k, int32_t H_lr, int32_t W_lr,
                                     int64_t n_prefix, int64_t D, int mode, int dtype, void* compact,
                                     int32_t* pos_sel, void* canvas, void* stream) {
  AVITS_REQUIRE(H_lr >= 1 && W_lr >= 1, "gather_upsample: H_lr=%d W_lr=%d must be >= 1", H_lr, W_lr);
  const int64_t N = int64_t(4) * H_lr * W_lr;
  AVITS_REQUIRE(k >= 0 && k <= N, "gather_upsample: k=%lld outside [0, N=%lld]", (long long)k, (long long)N);
  AVITS_REQUIRE(n_prefix >= 0, "gather_upsample: n_prefix=%lld < 0", (long long)n_prefix);
  AVITS_REQUIRE(D >= 1, "gather_upsample: D=%lld < 1", (long long)D);
  AVITS_REQUIRE(mode == AVITS_UP_NEAREST || mode == AVITS_UP_BILINEAR, "gather_upsample: bad mode %d", mode);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "gather_upsample: dtype %d unsupported", dtype);
  const int64_t esz = dtype == AVITS_F32 ? 4 : 2;
  AVITS_REQUIRE((D * esz) % 16 == 0, "gather_upsample: a row of D=%lld elements must be a multiple of 16 bytes", (long long)D);
  AVITS_REQUIRE(lowres && highres_prev && canvas, "gather_upsample: null lowres/highres_prev/canvas");
  AVITS_REQUIRE(n_prefix == 0 || prefix, "gather_upsample: null prefix with n_prefix=%lld", (long long)n_prefix);
  AVITS_REQUIRE(n_prefix + k == 0 || compact, "gather_upsample: null compact");
  AVITS_REQUIRE(k == 0 || (idx && pos_sel), "gather_upsample: null idx/pos_sel with k=%lld", (long long)k);
  ImageRows im{};
  im.idx_off[1] = k;
  return launch_gather(lowres, highres_prev, prefix, idx, im, 1, k, H_lr, W_lr, n_prefix, D, mode, dtype, compact,
                       pos_sel, canvas, stream, "gather_upsample");
}

extern "C" int avits_gather_upsample_ln(const void* lowres, const void* highres_prev, const void* prefix,
                                        const int32_t* idx, int64_t k, int32_t H_lr, int32_t W_lr,
                                        int64_t n_prefix, int64_t D, int mode, int dtype, void* compact,
                                        int32_t* pos_sel, void* canvas, int64_t n_txt, const void* shift_txt,
                                        const void* scale_txt, const void* shift_img, const void* scale_img,
                                        void* h_out, void* stream) {
  if (dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "gather_upsample_ln: dtype %d unsupported (bf16 only)", dtype);
  AVITS_REQUIRE(D >= 8 && D % 8 == 0 && D <= int64_t(kWave) * kCopyBatch * 8,
                "gather_upsample_ln: D=%lld must be a multiple of 8 in [8, %d]", (long long)D, kWave * kCopyBatch * 8);
  AVITS_REQUIRE(n_txt >= 0 && n_txt <= n_prefix, "gather_upsample_ln: n_txt=%lld outside [0, n_prefix=%lld]",
                (long long)n_txt, (long long)n_prefix);
  AVITS_REQUIRE(n_prefix + k == 0 || h_out, "gather_upsample_ln: null h_out");
  AVITS_REQUIRE(h_out == nullptr || h_out != compact, "gather_upsample_ln: h_out must not alias compact");
  AVITS_REQUIRE(n_txt == 0 || (shift_txt && scale_txt), "gather_upsample_ln: null text-stream shift/scale");
  AVITS_REQUIRE(n_prefix + k == n_txt || (shift_img && scale_img), "gather_upsample_ln: null image-stream shift/scale");
  AVITS_REQUIRE(H_lr >= 1 && W_lr >= 1, "gather_upsample_ln: H_lr=%d W_lr=%d must be >= 1", H_lr, W_lr);
  const int64_t N = int64_t(4) * H_lr * W_lr;
  AVITS_REQUIRE(k >= 0 && k <= N, "gather_upsample_ln: k=%lld outside [0, N=%lld]", (long long)k, (long long)N);
  AVITS_REQUIRE(n_prefix >= 0, "gather_upsample_ln: n_prefix=%lld < 0", (long long)n_prefix);
  AVITS_REQUIRE(mode == AVITS_UP_NEAREST || mode == AVITS_UP_BILINEAR, "gather_upsample_ln: bad mode %d", mode);
  AVITS_REQUIRE(lowres && highres_prev && canvas, "gather_upsample_ln: null lowres/highres_prev/canvas");
  AVITS_REQUIRE(n_prefix == 0 || prefix, "gather_upsample_ln: null prefix with n_prefix=%lld", (long long)n_prefix);
  AVITS_REQUIRE(n_prefix + k == 0 || compact, "gather_upsample_ln: null compact");
  AVITS_REQUIRE(k == 0 || (idx && pos_sel), "gather_upsample_ln: null idx/pos_sel with k=%lld", (long long)k);
  ImageRows im{};
  im.idx_off[1] = k;
  LnOut ln{};
  ln.h = static_cast<bf16_t*>(h_out);
  ln.n_a = n_txt;
  ln.shift_a = static_cast<const bf16_t*>(shift_txt);
  ln.scale_a = static_cast<const bf16_t*>(scale_txt);
  ln.shift_b = static_cast<const bf16_t*>(shift_img);
  ln.scale_b = static_cast<const bf16_t*>(scale_img);
  return launch_gather(lowres, highres_prev, prefix, idx, im, 1, k, H_lr, W_lr, n_prefix, D, mode, dtype, compact,
                       pos_sel, canvas, stream, "gather_upsample_ln", ln);
}

extern "C" int avits_scatter(const void* out, const int32_t* idx, int64_t k, int64_t row_offset, int64_t D,
                             int64_t n_canvas, int dtype, void* canvas, void* stream) {
  AVITS_REQUIRE(k >= 0 && row_offset >= 0 && D >= 1, "scatter: bad k=%lld row_offset=%lld D=%lld",
                (long long)k, (long long)row_offset, (long long)D);
  AVITS_REQUIRE(n_canvas >= 1, "scatter: n_canvas=%lld must be >= 1", (long long)n_canvas);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "scatter: dtype %d unsupported", dtype);
  const int64_t esz = dtype == AVITS_F32 ? 4 : 2;
  AVITS_REQUIRE((D * esz) % 16 == 0, "scatter: a row of D=%lld elements must be a multiple of 16 bytes", (long long)D);
  if (k == 0) return AVITS_OK;
  AVITS_REQUIRE(out && idx && canvas, "scatter: null pointer");
  ImageRows im{};
  im.idx_off[1] = k;
  im.row_off[0] = row_offset;
  return launch_scatter(out, idx, im, 1, k, n_canvas, D, dtype, canvas, stream, "scatter");
}

extern "C" int avits_gather_upsample_batched(const void* lowres, const void* highres_prev, const void* prefix,
                                             const int32_t* idx, const int64_t* idx_off, int32_t B,
                                             int32_t H_lr, int32_t W_lr, int64_t n_prefix, int64_t D, int mode,
                                             int dtype, void* compact, const int64_t* row_off, int32_t* pos,
                                             void* canvas, void* stream) {
  AVITS_REQUIRE(B >= 1 && B <= kMaxRelayoutImages, "gather_upsample_batched: B=%d outside [1, %d]", B,
                kMaxRelayoutImages);
  AVITS_REQUIRE(idx_off && row_off, "gather_upsample_batched: null idx_off/row_off");
  AVITS_REQUIRE(H_lr >= 1 && W_lr >= 1, "gather_upsample_batched: H_lr=%d W_lr=%d must be >= 1", H_lr, W_lr);
  const int64_t N = int64_t(4) * H_lr * W_lr;
  AVITS_REQUIRE(n_prefix >= 0, "gather_upsample_batched: n_prefix=%lld < 0", (long long)n_prefix);
  AVITS_REQUIRE(D >= 1, "gather_upsample_batched: D=%lld < 1", (long long)D);
  AVITS_REQUIRE(mode == AVITS_UP_NEAREST || mode == AVITS_UP_BILINEAR, "gather_upsample_batched: bad mode %d",
                mode);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "gather_upsample_batched: dtype %d unsupported", dtype);
  const int64_t esz = dtype == AVITS_F32 ? 4 : 2;
  AVITS_REQUIRE((D * esz) % 16 == 0,
                "gather_upsample_batched: a row of D=%lld elements must be a multiple of 16 bytes", (long long)D);
  AVITS_REQUIRE(idx_off[0] == 0, "gather_upsample_batched: idx_off[0]=%lld, must be 0", (long long)idx_off[0]);
  ImageRows im{};
  int64_t k_max = 0;
  for (int b = 0; b < B; ++b) {
    const int64_t k = idx_off[b + 1] - idx_off[b];
    AVITS_REQUIRE(k >= 0 && k <= N, "gather_upsample_batched: image %d selects k=%lld outside [0, N=%lld]", b,
                  (long long)k, (long long)N);
    AVITS_REQUIRE(row_off[b] >= 0, "gather_upsample_batched: row_off[%d]=%lld < 0", b, (long long)row_off[b]);
    im.idx_off[b] = idx_off[b];
    im.row_off[b] = row_off[b];
    im.pos_off[b] = row_off[b] + n_prefix;
    k_max = std::max(k_max, k);
  }
  im.idx_off[B] = idx_off[B];
  AVITS_REQUIRE(lowres && highres_prev && canvas, "gather_upsample_batched: null lowres/highres_prev/canvas");
  AVITS_REQUIRE(n_prefix == 0 || prefix, "gather_upsample_batched: null prefix with n_prefix=%lld",
                (long long)n_prefix);
  AVITS_REQUIRE(n_prefix + k_max == 0 || compact, "gather_upsample_batched: null compact");
  AVITS_REQUIRE(k_max == 0 || (idx && pos), "gather_upsample_batched: null idx/pos");
  return launch_gather(lowres, highres_prev, prefix, idx, im, B, k_max, H_lr, W_lr, n_prefix, D, mode, dtype,
                       compact, pos, canvas, stream, "gather_upsample_batched");
}

extern "C" int avits_scatter_batched(const void* out, const int32_t* idx, const int64_t* idx_off, int32_t B,
                                     const int64_t* row_off, int64_t N, int64_t D, int dtype, void* canvas,
                                     void* stream) {
  AVITS_REQUIRE(B >= 1 && B <= kMaxRelayoutImages, "scatter_batched: B=%d outside [1, %d]", B,
                kMaxRelayoutImages);
  AVITS_REQUIRE(idx_off && row_off, "scatter_batched: null idx_off/row_off");
  AVITS_REQUIRE(N >= 1 && D >= 1, "scatter_batched: N=%lld and D=%lld must be >= 1", (long long)N, (long long)D);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "scatter_batched: dtype %d unsupported", dtype);
  const int64_t esz = dtype == AVITS_F32 ? 4 : 2;
  AVITS_REQUIRE((D * esz) % 16 == 0, "scatter_batched: a row of D=%lld elements must be a multiple of 16 bytes",
                (long long)D);
  AVITS_REQUIRE(idx_off[0] == 0, "scatter_batched: idx_off[0]=%lld, must be 0", (long long)idx_off[0]);
  ImageRows im{};
  int64_t k_max = 0;
  for (int b = 0; b < B; ++b) {
    const int64_t k = idx_off[b + 1] - idx_off[b];
    AVITS_REQUIRE(k >= 0 && k <= N, "scatter_batched: image %d selects k=%lld outside [0, N=%lld]", b,
                  (long long)k, (long long)N);
    AVITS_REQUIRE(row_off[b] >= 0, "scatter_batched: row_off[%d]=%lld < 0", b, (long long)row_off[b]);
    im.idx_off[b] = idx_off[b];
    im.row_off[b] = row_off[b];
    k_max = std::max(k_max, k);
  }
  im.idx_off[B] = idx_off[B];
  if (k_max == 0) return AVITS_OK;
  AVITS_REQUIRE(out && idx && canvas, "scatter_batched: null pointer");
  return launch_scatter(out, idx, im, B, k_max, N, D, dtype, canvas, stream, "scatter_batched");
}

extern "C" int avits_gather_mixed(const void* lowres, const void* prefix, const int32_t* idx, int64_t k,
                                  int32_t H_lr, int32_t W_lr, int64_t n_prefix, int64_t D, int mode, int dtype,
                                  void* compact, int32_t* pos, int32_t* children, void* stream) {
  AVITS_REQUIRE(H_lr >= 1 && W_lr >= 1, "gather_mixed: H_lr=%d W_lr=%d must be >= 1", H_lr, W_lr);
  const int64_t Mp = int64_t(H_lr) * W_lr;
  AVITS_REQUIRE(k >= 0 && k <= Mp, "gather_mixed: k=%lld outside [0, M'=%lld]", (long long)k, (long long)Mp);
  AVITS_REQUIRE(n_prefix >= 0, "gather_mixed: n_prefix=%lld < 0", (long long)n_prefix);
  AVITS_REQUIRE(D >= 1, "gather_mixed: D=%lld < 1", (long long)D);
  AVITS_REQUIRE(mode == AVITS_UP_NEAREST || mode == AVITS_UP_BILINEAR, "gather_mixed: bad mode %d", mode);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "gather_mixed: dtype %d unsupported", dtype);
  const int64_t esz = dtype == AVITS_F32 ? 4 : 2;
  AVITS_REQUIRE((D * esz) % 16 == 0, "gather_mixed: a row of D=%lld elements must be a multiple of 16 bytes", (long long)D);
  AVITS_REQUIRE(lowres && compact && pos, "gather_mixed: null lowres/compact/pos");
  AVITS_REQUIRE(n_prefix == 0 || prefix, "gather_mixed: null prefix with n_prefix=%lld", (long long)n_prefix);
  AVITS_REQUIRE(k == 0 || idx, "gather_mixed: null idx with k=%lld", (long long)k);
  const int64_t jobs = n_prefix + Mp;
  const dim3 grid(unsigned(ceil_div(jobs, kRowsPerBlock))), block(kWave * kRowsPerBlock);
  hipStream_t s = static_cast<hipStream_t>(stream);
  TimedLaunch timed("gather_mixed", s);
  if (dtype == AVITS_F32)
    hipLaunchKernelGGL(gather_mixed_kernel<float>, grid, block, 0, s, (const float*)lowres, (const float*)prefix,
                       idx, k, H_lr, W_lr, n_prefix, D, mode, (float*)compact, pos, children);
  else
    hipLaunchKernelGGL(gather_mixed_kernel<bf16_t>, grid, block, 0, s, (const bf16_t*)lowres,
                       (const bf16_t*)prefix, idx, k, H_lr, W_lr, n_prefix, D, mode, (bf16_t*)compact, pos,
                       children);
  return launch_status("gather_mixed");
}

extern "C" int avits_scatter_mixed(const void* out, const int32_t* idx, int64_t k, int32_t H_lr, int32_t W_lr,
                                   int64_t row_offset, int64_t D, int dtype, void* canvas_hr, void* state_lr,
                                   void* stream) {
  AVITS_REQUIRE(H_lr >= 1 && W_lr >= 1, "scatter_mixed: H_lr=%d W_lr=%d must be >= 1", H_lr, W_lr);
  const int64_t Mp = int64_t(H_lr) * W_lr;
  AVITS_REQUIRE(k >= 0 && k <= Mp, "scatter_mixed: k=%lld outside [0, M'=%lld]", (long long)k, (long long)Mp);
  AVITS_REQUIRE(row_offset >= 0 && D >= 1, "scatter_mixed: bad row_offset=%lld D=%lld", (long long)row_offset,
                (long long)D);
  if (dtype != AVITS_F32 && dtype != AVITS_BF16)
    return set_error(AVITS_ERR_UNSUPPORTED, "scatter_mixed: dtype %d unsupported", dtype);
  const int64_t esz = dtype == AVITS_F32 ? 4 : 2;
  AVITS_REQUIRE((D * esz) % 16 == 0, "scatter_mixed: a row of D=%lld elements must be a multiple of 16 bytes", (long long)D);
  AVITS_REQUIRE(out, "scatter_mixed: null out");
  AVITS_REQUIRE(k == 0 || (idx && canvas_hr), "scatter_mixed: null idx/canvas_hr with k=%lld", (long long)k);
  AVITS_REQUIRE(k == Mp || state_lr, "scatter_mixed: null state_lr with %lld kept tokens", (long long)(Mp - k));
  const dim3 grid(unsigned(ceil_div(Mp, kRowsPerBlock))), block(kWave * kRowsPerBlock);
  hipStream_t s = static_cast<hipStream_t>(stream);
  TimedLaunch timed("scatter_mixed", s);
  if (dtype == AVITS_F32)
    hipLaunchKernelGGL(scatter_mixed_kernel<float>, grid, block, 0, s, (const float*)out, idx, k, H_lr, W_lr,
                       row_offset, D, (float*)canvas_hr, (float*)state_lr);
  else
    hipLaunchKernelGGL(scatter_mixed_kernel<bf16_t>, grid, block, 0, s, (const bf16_t*)out, idx, k, H_lr, W_lr,
                       row_offset, D, (bf16_t*)canvas_hr, (bf16_t*)state_lr);
  return launch_status("scatter_mixed");
}
