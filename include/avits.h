/*
 * avits.h — C ABI of the AViTS selective-upsampling step on AMD MI355X (gfx950).
 *
 * The library implements the hot path of spatiotemporal token selection for
 * dynamic-resolution diffusion transformers (AViTS, Section 3): score every
 * high-resolution latent token, select the top-K, gather them with the text
 * (and reference) tokens into a compacted sequence while the other tokens are
 * upsampled from the low-resolution latent, run one MMDiT joint-attention
 * block on the compacted sequence, and scatter the result back.
 *
 * Conventions shared by every entry point:
 *  - Every tensor argument is a DEVICE pointer owned by the caller, row-major
 *    and contiguous, 16-byte aligned.  The library never allocates device
 *    memory; scratch space comes through a caller-provided workspace whose
 *    size the matching *_workspace_bytes() query returns.
 *  - `stream` is a hipStream_t (NULL = the null stream).  Calls are
 *    asynchronous: they enqueue kernels and return; no host<->device copy and
 *    no synchronisation happens inside.
 *  - Return value: AVITS_OK, or a negative error code.  Validation uses the
 *    host-side arguments only (shapes, pointers, sizes); the contents of
 *    device buffers are never inspected.  After an error nothing was
 *    enqueued, except for AVITS_ERR_HIP, which reports a launch failure.
 *    avits_last_error() returns the message of the calling thread's last
 *    failure.
 *  - `dtype` selects the storage type of every non-index tensor of a call:
 *    AVITS_F32 or AVITS_BF16.  Scores, log-sum-exps and all accumulation are
 *    fp32; indices and positions are int32.
 *  - Calls that overlap on one stream are ordered; calls on different
 *    streams that share a workspace race.
 */
#ifndef AVITS_H
#define AVITS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  AVITS_OK = 0,
  AVITS_ERR_INVALID_ARG = -1, /* bad shape, null pointer, k out of range, ... */
  AVITS_ERR_UNSUPPORTED = -2, /* dtype / head dim / device not supported    */
  AVITS_ERR_WORKSPACE = -3,   /* workspace missing or smaller than required */
  AVITS_ERR_HIP = -4          /* a kernel launch failed                      */
};

enum { AVITS_F32 = 0, AVITS_BF16 = 1 };
enum { AVITS_UP_NEAREST = 0, AVITS_UP_BILINEAR = 1 };
enum { AVITS_BLOCK_DOUBLE = 0, AVITS_BLOCK_SINGLE = 1 };

/* Version string "major.minor.patch". */
const char* avits_version(void);

/* Message of the calling thread's last failed call ("" if none). */
const char* avits_last_error(void);

/* ------------------------------------------------------------------------
 * avits_score — spatiotemporal importance (Section 3.3; Eqs. spatial,
 * dit_attn, zbar, step_var and joint).
 *
 * For each of the N scored image tokens i:
 *   A_i = (1/H) sum_h sum_{j<L} exp(q_ih . k_jh / sqrt(d) - row_lse[h, i])
 *       (the text share of the joint image->text attention of Eq. dit_attn;
 *        row_lse is the log-sum-exp of token i's logits over the joint key
 *        set, e.g. from avits_joint_lse),
 *   V_i = (1/D_f) sum_c (feat_t[i,c] - feat_prev[i,c])^2 / 2
 *       (Eq. step_var with the two consecutive steps as the snapshots),
 *   S_i = alpha * (A_i - min A)/(max A - min A + eps)
 *       + (1 - alpha) * (V_i - min V)/(max V - min V + eps).
 *
 * latent_q  [N, H, d]   image queries after QK-norm and RoPE   (dtype)
 * text_k    [L, H, d]   text keys after QK-norm                (dtype)
 * row_lse   [H, N]      fp32
 * feat_t, feat_prev [N, D_f]                                   (dtype)
 * scores    [N]         fp32 output S
 * a_raw, v_raw [N]      fp32 outputs A and V; each may be NULL
 * Requires N >= 1, L >= 1, H >= 1, d in {64, 128}, D_f >= 1,
 * 0 <= alpha <= 1, eps >= 0.
 * ---------------------------------------------------------------------- */
size_t avits_score_workspace_bytes(int64_t N, int32_t H);
int avits_score(const void* latent_q, const void* text_k, const float* row_lse,
                const void* feat_t, const void* feat_prev,
                int64_t N, int64_t L, int32_t H, int32_t d, int64_t D_f,
                float alpha, float eps, int dtype,
                float* scores, float* a_raw, float* v_raw,
                void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * avits_score_select — avits_score followed by avits_select(scores, k) in
 * one call (Section 3.3: Eq. joint, then Eq. topk), for N <= 16384: the
 * normalisation and the selection run in one workgroup, one launch less.
 * scores, a_raw, v_raw and idx [k] are exactly what the two calls write.
 * Arguments as avits_score, plus k (0 <= k <= N; k == 0 writes scores only)
 * and idx (device int32 [k]).  N > 16384 -> AVITS_ERR_INVALID_ARG (use the
 * two calls).  Other errors as avits_score.
 * ---------------------------------------------------------------------- */
int avits_score_select(const void* latent_q, const void* text_k, const float* row_lse,
                       const void* feat_t, const void* feat_prev,
                       int64_t N, int64_t L, int32_t H, int32_t d, int64_t D_f,
                       float alpha, float eps, int dtype,
                       float* scores, float* a_raw, float* v_raw, int64_t k, int32_t* idx,
                       void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * avits_score_batched — avits_score over B equally shaped images in one
 * pass (Section 3.3, applied per image: a CFG pair, or several prompts at
 * one resolution).  Image b's min-max normalisation (Eq. joint) uses its own
 * A and V only, so its scores equal avits_score on image b alone.
 *
 * Inputs are stacked image-major, each image laid out as in avits_score:
 * latent_q [B, N, H, d], text_k [B, L, H, d] (every image has L text keys),
 * row_lse [B, H, N], feat_t and feat_prev [B, N, D_f]; outputs scores, and
 * a_raw / v_raw when not NULL, [B, N] fp32.  All device pointers, owned by
 * the caller.  workspace >= avits_score_batched_workspace_bytes(B, N, H)
 * (which returns 0 for arguments outside the limits).  Requires
 * 1 <= B <= 4096 and the limits of avits_score; errors as avits_score.
 * ---------------------------------------------------------------------- */
size_t avits_score_batched_workspace_bytes(int64_t B, int64_t N, int32_t H);
int avits_score_batched(const void* latent_q, const void* text_k, const float* row_lse,
                        const void* feat_t, const void* feat_prev,
                        int64_t B, int64_t N, int64_t L, int32_t H, int32_t d, int64_t D_f,
                        float alpha, float eps, int dtype,
                        float* scores, float* a_raw, float* v_raw,
                        void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * avits_select — top-K selection (Eq. topk).
 *
 * Writes the indices of the k largest scores to idx[0..k) in strictly
 * ascending order.  Order is (score descending, index ascending): among equal
 * scores the lowest index wins, so the result is deterministic; -0.0 equals
 * +0.0 and NaN ranks below every number.  k == 0 enqueues nothing.
 * scores [N] fp32; idx [k] int32.  Requires N >= 1 and 0 <= k <= N.
 * ---------------------------------------------------------------------- */
size_t avits_select_workspace_bytes(int64_t N);
int avits_select(const float* scores, int64_t N, int64_t k, int32_t* idx,
                 void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * avits_select_perturbed — Eq. topk with the paper's tie-break by a small
 * perturbation applied before the selection (Section 3.3): the keys are the
 * fp32 sums scores[i] + delta[i] (one rounding), then as avits_select
 * (ties of the sums still go to the lowest index).  delta [N] fp32 is the
 * caller's seeded perturbation (e.g. 1e-6 times standard normal draws).
 * Other arguments, workspace and errors as avits_select.
 * ---------------------------------------------------------------------- */
int avits_select_perturbed(const float* scores, const float* delta, int64_t N, int64_t k,
                           int32_t* idx, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * avits_select_noalloc — avits_select for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same selection, bit for bit, with
 * no workspace argument.  The state of the grid path (N > 16384) lives in
 * one fixed array of about 260 KiB in the library's device memory, one copy
 * per GPU, held until the process ends; the call makes no hipMalloc,
 * hipFree or other allocating call (the first call on a device looks the
 * array's address up once).  Every call on one GPU shares that GPU's array:
 * calls that overlap on one GPU (other streams, other threads) race;
 * calls on one stream are ordered and safe.  The array is re-initialised by
 * every call, so nothing carries over between calls.
 * scores [N] fp32, idx [k] int32: device pointers of the calling thread's
 * current device, owned by the caller.  Requires 1 <= N <=
 * avits_select_noalloc_max_n() (2^26) and 0 <= k <= N; otherwise
 * AVITS_ERR_INVALID_ARG and nothing is enqueued.  Other errors as
 * avits_select.
 * ---------------------------------------------------------------------- */
size_t avits_select_noalloc_max_n(void);
int avits_select_noalloc(const float* scores, int64_t N, int64_t k, int32_t* idx, void* stream);

/* ------------------------------------------------------------------------
 * avits_select_batched — B independent selections in one launch (images of
 * a batch with their own token counts and budgets).  Element b selects the
 * top k[b] of scores[offsets[b] .. offsets[b + 1]) (perturbed by delta over
 * the same range when delta is not NULL) and writes its indices, local to
 * the element and ascending, to idx[sum_{c<b} k[c] ..].  offsets [B + 1] and
 * k [B] are host arrays (int64); scores, delta, idx device arrays.
 * Requires 1 <= B <= 64, offsets[0] == 0, 1 <= N_b <= 16384 and
 * 0 <= k[b] <= N_b.  No workspace.
 * ---------------------------------------------------------------------- */
int avits_select_batched(const float* scores, const float* delta, int32_t B, const int64_t* offsets,
                         const int64_t* k, int32_t* idx, void* stream);

/* ------------------------------------------------------------------------
 * avits_gather_upsample — Stage-2 re-layout (Section 3.2).
 *
 * With N = 4*H_lr*W_lr high-res tokens in raster order on a (2H_lr)x(2W_lr)
 * grid and the selected indices idx[0..k) (ascending, unique, < N):
 *   compact[0 .. n_prefix)        = prefix rows (text, then reference)
 *   compact[n_prefix + j]         = highres_prev[idx[j]]
 *   pos_sel[j]                    = (0, idx[j] / W_hr, idx[j] % W_hr)
 *   canvas[p]                     = highres_prev[p]      if p is selected
 *                                   upsample2x(lowres)[p] otherwise
 * mode AVITS_UP_NEAREST copies the low-res cell (p's row/2, col/2);
 * AVITS_UP_BILINEAR interpolates with half-pixel centres and edge clamping
 * (fp32 arithmetic).  canvas may alias highres_prev (selected rows are then
 * left in place); it may not overlap any other argument.
 * lowres [H_lr*W_lr, D], highres_prev [N, D], prefix [n_prefix, D] (may be
 * NULL when n_prefix == 0), compact [n_prefix + k, D], pos_sel [k, 3] int32,
 * canvas [N, D].  The caller writes the prefix rows' positions itself.
 * An idx entry outside [0, N) is skipped on the device (its compact row
 * and position are left unwritten), so no access leaves the buffers.
 * ---------------------------------------------------------------------- */
int avits_gather_upsample(const void* lowres, const void* highres_prev, const void* prefix,
                          const int32_t* idx, int64_t k, int32_t H_lr, int32_t W_lr,
                          int64_t n_prefix, int64_t D, int mode, int dtype,
                          void* compact, int32_t* pos_sel, void* canvas, void* stream);

/* ------------------------------------------------------------------------
 * avits_gather_upsample_batched — the Stage-2 re-layout of Section 3.2 for
 * B equally shaped images in one launch, each with its own selection, its
 * rows placed anywhere in one packed compact buffer (e.g. the image rows of
 * avits_block_forward_batched).  For image b, with idx_b = idx[idx_off[b] ..
 * idx_off[b + 1]) (ascending, unique, < N) and k_b its length, it does what
 * avits_gather_upsample does with
 *   lowres + b*(N/4)*D, highres_prev + b*N*D, prefix + b*n_prefix*D,
 *   compact rows from row_off[b], canvas + b*N*D,
 * and writes pos[row_off[b] + n_prefix + j] = (0, idx_b[j] / W_hr,
 * idx_b[j] % W_hr): pos is indexed like compact's rows (the prefix rows'
 * positions are the caller's).  lowres [B, H_lr*W_lr, D], highres_prev and
 * canvas [B, N, D] (canvas may alias highres_prev, as one stack), prefix
 * [B, n_prefix, D] or NULL when n_prefix == 0; idx_off [B + 1] and row_off
 * [B] are host int64 arrays (idx_off[0] == 0); device buffers are the
 * caller's.  1 <= B <= 64; each k_b in [0, N]; rows of different images must
 * not overlap in compact.  Errors as avits_gather_upsample.
 * ---------------------------------------------------------------------- */
int avits_gather_upsample_batched(const void* lowres, const void* highres_prev, const void* prefix,
                                  const int32_t* idx, const int64_t* idx_off, int32_t B,
                                  int32_t H_lr, int32_t W_lr, int64_t n_prefix, int64_t D, int mode,
                                  int dtype, void* compact, const int64_t* row_off, int32_t* pos,
                                  void* canvas, void* stream);

/* ------------------------------------------------------------------------
 * avits_gather_upsample_ln — avits_gather_upsample (one image, bf16) that
 * also writes the first stage of the double block the compacted rows feed
 * (Section 3.3.1, the block on the compacted sequence): for every compact
 * row r < n_prefix + k,
 *   h[r] = LN(compact[r]) (1 + scale) + shift
 * (layer norm without affine, eps 1e-6, biased variance, fp32 arithmetic,
 * rounded to bf16), with (shift_txt, scale_txt) for rows r < n_txt (the
 * text rows leading the prefix) and (shift_img, scale_img) for the others
 * (the reference rows and the selected rows: the image stream).  The
 * shift / scale vectors are [D] bf16: rows 0 and 1 of each stream's
 * modulation.  h is bit-identical to the block's own first stage, so
 * avits_block_forward_ex with h_in = h_out gives the block output bit for
 * bit.  h_out [n_prefix + k, D] bf16, not aliasing compact.  D a multiple
 * of 8 in [8, 4096]; 0 <= n_txt <= n_prefix.  Other arguments, outputs
 * and errors as avits_gather_upsample; dtype other than bf16 ->
 * AVITS_ERR_UNSUPPORTED.
 * ---------------------------------------------------------------------- */
int avits_gather_upsample_ln(const void* lowres, const void* highres_prev, const void* prefix,
                             const int32_t* idx, int64_t k, int32_t H_lr, int32_t W_lr, int64_t n_prefix,
                             int64_t D, int mode, int dtype, void* compact, int32_t* pos_sel, void* canvas,
                             int64_t n_txt, const void* shift_txt, const void* scale_txt,
                             const void* shift_img, const void* scale_img, void* h_out, void* stream);

/* ------------------------------------------------------------------------
 * avits_block_forward — one MMDiT joint-attention block on the compacted
 * sequence (Section 3.3.1: joint self-attention over [C; Z], Eq. joint_qk,
 * with the model's QK-normalisation), FLUX-style:
 *
 * double (per stream s; rows [0, n_txt) use `txt`, the rest `img`):
 *   h = LN(x)(1 + scale1) + shift1;  q,k,v = h W_qkv^T + b_qkv;
 *   q,k = RMSNorm_d(.) * g;  RoPE(q, k) at pos;  o = softmax(q k^T/sqrt d) v
 *   over all S rows;  x += gate1 (o W_o^T + b_o);
 *   x += gate2 (GELU_tanh((LN(x)(1 + scale2) + shift2) W_1^T + b_1) W_2^T + b_2)
 * single (one weight set):
 *   h = LN(x)(1 + scale) + shift;  [q k v m] = h W_in^T + b_in;
 *   q,k normalised and rotated;  x += gate ([attn(q,k,v); GELU_tanh(m)] W_out^T + b_out)
 * LN has no affine and eps 1e-6; RMSNorm eps 1e-6.  RoPE: three axes
 * (frame, row, col) over head-dim slices (d/8, 7d/16, 7d/16), theta 10000,
 * adjacent pairs (2m, 2m+1) rotated by pos * theta^(-2m/n).
 * Modulation rows: double (shift1, scale1, gate1, shift2, scale2, gate2);
 * single (shift, scale, gate).  Weights use the [out, in] layout.
 *
 * x_in, x_out [S, D] with S = n_txt + n_img, D = H*d (x_out must not alias
 * x_in); pos [S, 3] int32, RoPE position = pos * pos_scale with pos_scale in
 * (0, 1] (1: integer grid positions; 0.5: positions given in half units, as
 * the mixed-resolution sequence of avits_gather_mixed has them); lse_out
 * [H, S] fp32 or NULL.  For the single kind
 * n_txt only splits the count (both parts use the same weights).  S == 0 is a
 * no-op.  Requires d in {64, 128}; all weight pointers of the used kind
 * non-NULL.
 * ---------------------------------------------------------------------- */
typedef struct avits_double_stream_weights {
  const void* mod;     /* [6, D]        */
  const void* w_qkv;   /* [3D, D]       */
  const void* b_qkv;   /* [3D]          */
  const void* g_q;     /* [d]           */
  const void* g_k;     /* [d]           */
  const void* w_o;     /* [D, D]        */
  const void* b_o;     /* [D]           */
  const void* w_mlp1;  /* [F, D], F = mlp_hidden */
  const void* b_mlp1;  /* [F]           */
  const void* w_mlp2;  /* [D, F]        */
  const void* b_mlp2;  /* [D]           */
} avits_double_stream_weights;

typedef struct avits_single_weights {
  const void* mod;     /* [3, D]        */
  const void* w_in;    /* [3D + F, D]   */
  const void* b_in;    /* [3D + F]      */
  const void* g_q;     /* [d]           */
  const void* g_k;     /* [d]           */
  const void* w_out;   /* [D, D + F]    */
  const void* b_out;   /* [D]           */
} avits_single_weights;

typedef struct avits_block_weights {
  int32_t kind;        /* AVITS_BLOCK_DOUBLE or AVITS_BLOCK_SINGLE */
  int32_t mlp_hidden;  /* F (4*D for FLUX)                         */
  avits_double_stream_weights txt, img;  /* kind == DOUBLE */
  avits_single_weights single;           /* kind == SINGLE */
} avits_block_weights;

size_t avits_block_workspace_bytes(int32_t kind, int64_t S, int32_t H, int32_t d,
                                   int32_t mlp_hidden, int dtype);
int avits_block_forward(const void* x_in, void* x_out, const int32_t* pos, float pos_scale,
                        int64_t n_txt, int64_t n_img, const avits_block_weights* w,
                        int32_t H, int32_t d, int dtype, float* lse_out,
                        void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * avits_block_forward_ex — avits_block_forward with optional statistics of
 * its joint attention, taken inside the same pass (Section 3.3.1: the
 * attention maps of the backbone's own blocks are the spatial signal, Eq.
 * spatial with the softmax of Eq. dit_attn):
 *   lse[h, r]   = log sum_j exp(q_rh . k_jh / sqrt d)          (natural log)
 *   mass[h, r] (+)= sum_{j < n_txt} softmax_j(q_rh . k_jh / sqrt d)
 * over all S keys, j < n_txt being the text rows that lead the sequence.
 * The text mass is tracked beside the softmax normaliser under the same
 * running maximum, so it costs no second Q K^T pass.  With
 * mass_accumulate != 0 it is added to what `mass` holds (the aggregation
 * over blocks and collection steps of Section 3.3.1; avits_score_from_mass
 * divides by their count).
 * The Stage-3 scatter of Section 3.2 can ride on the block's last
 * projection: with scatter_k > 0, the output rows of the last scatter_k
 * image rows (x_out rows S - scatter_k + j) are also written to
 * canvas[scatter_idx[j]] (bit-identical to avits_scatter after the block;
 * an index outside [0, n_canvas) is skipped).  canvas [n_canvas, D] of
 * dtype, not aliasing x_in or x_out; scatter_idx [scatter_k] int32; 0 <=
 * scatter_k <= n_img.
 * The block's first stage can come in precomputed: h_in [S, D] of dtype
 * holds h = LN(x_in)(1 + scale1) + shift1 of every row with its stream's
 * first two modulation rows (the single kind: its own), e.g. written by
 * avits_gather_upsample_ln as it gathers x_in; the block then starts from
 * it and skips its own layer norm (x_in still supplies the residual).  Not
 * aliasing x_in, x_out or the workspace.
 * And the next block's first stage can go out: with h_next and next_w set,
 * h_next [S, D] of dtype receives LN(x_out)(1 + scale1) + shift1 with the
 * next block's first two modulation rows (double: its text-stream rows for
 * rows < n_txt, its image-stream rows after; single: its own), bit for bit
 * what that block computes first; pass it there as h_in.  In a stack of
 * blocks this replaces one layer-norm launch per block (it rides on the
 * split-K reduce of the last projection, as the block's second layer norm
 * rides on the output projection's).  Not aliasing x_in, x_out, h_in or the
 * workspace; next_w is read on the host only.
 * outs may be NULL (= avits_block_forward without lse).  lse and mass
 * [H, S] fp32 device buffers or NULL; other arguments and errors as
 * avits_block_forward.
 * ---------------------------------------------------------------------- */
typedef struct avits_block_outputs {
  float* lse;                  /* [H, S] or NULL */
  float* mass;                 /* [H, S] or NULL */
  int32_t mass_accumulate;     /* nonzero: mass += this block's mass */
  const int32_t* scatter_idx;  /* [scatter_k] or NULL */
  int64_t scatter_k;           /* 0: no fused scatter */
  void* canvas;                /* [n_canvas, D] or NULL */
  int64_t n_canvas;
  const void* h_in;            /* [S, D]: the first modulated layer norm, precomputed; or NULL */
  void* h_next;                /* [S, D]: the next block's first stage, or NULL */
  const struct avits_block_weights* next_w;  /* that block's weights (host struct), or NULL */
} avits_block_outputs;

int avits_block_forward_ex(const void* x_in, void* x_out, const int32_t* pos, float pos_scale,
                           int64_t n_txt, int64_t n_img, const avits_block_weights* w,
                           int32_t H, int32_t d, int dtype, const avits_block_outputs* outs,
                           void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * avits_block_forward_batched — B images through one block in one pass: the
 * rows of all images are packed by stream, the text rows of images 0..B-1
 * first (image b's at [txt_off[b], txt_off[b+1])), then their image rows
 * (image b's at txt_off[B] + [img_off[b], img_off[b+1])).  Every row-wise
 * stage runs over all rows at once; the joint attention is block diagonal:
 * image b's rows attend to image b's rows only (Eq. joint_qk per image), so
 * each image's output equals avits_block_forward on that image alone.
 * txt_off, img_off [B + 1] host int64 arrays starting at 0; each image has
 * at least one row; 1 <= B <= 16.  bf16 only (AVITS_ERR_UNSUPPORTED
 * otherwise).  Workspace: avits_block_workspace_bytes(kind, S, H, d, F,
 * dtype) with S = txt_off[B] + img_off[B].  lse_out [H, S] is per packed row.
 * Other arguments and errors as avits_block_forward.
 * ---------------------------------------------------------------------- */
int avits_block_forward_batched(const void* x_in, void* x_out, const int32_t* pos, float pos_scale,
                                int32_t B, const int64_t* txt_off, const int64_t* img_off,
                                const avits_block_weights* w, int32_t H, int32_t d, int dtype,
                                float* lse_out, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * avits_block_forward_batched_ex — avits_block_forward_batched with one set
 * of modulation vectors per image, for images at different timesteps in
 * one pass (Section 3.2: every image of a batch runs its own denoising
 * schedule; with a diffusion transformer the timestep enters each block
 * through its modulation vectors).  Image b's rows (its text rows with the
 * text stream, its image rows with the image stream; every row with the
 * single kind) use the modulation rows at mod + b * mod_stride elements,
 * where mod is the stream's `mod` pointer in w: the caller lays the images'
 * [6, D] (double) or [3, D] (single) blocks out mod_stride elements apart,
 * e.g. as [B, 6, D] with mod_stride = 6 D.  mod_stride == 0 shares one set
 * across the images (exactly avits_block_forward_batched).  Every other
 * weight is shared.  The gated projections apply their per-image gates in
 * their split-K reduce, so they always run split (the workspace of
 * avits_block_workspace_bytes covers it).  Errors as
 * avits_block_forward_batched; AVITS_ERR_INVALID_ARG for mod_stride < 0.
 * ---------------------------------------------------------------------- */
int avits_block_forward_batched_ex(const void* x_in, void* x_out, const int32_t* pos, float pos_scale,
                                   int32_t B, const int64_t* txt_off, const int64_t* img_off,
                                   const avits_block_weights* w, int64_t mod_stride, int32_t H, int32_t d,
                                   int dtype, float* lse_out, void* workspace, size_t workspace_bytes,
                                   void* stream);

/* ------------------------------------------------------------------------
 * avits_block_qk — the first stage of a block alone (the attention probe of
 * Section 3.3.1: the queries and keys whose joint softmax defines the
 * image-to-text attention mass of Eq. spatial): for each row,
 *   h = LN(x)(1 + scale1) + shift1;  q = h W_q^T + b_q;  k = h W_k^T + b_k;
 *   q, k = RMSNorm_d(.) * g;  RoPE(q, k) at pos
 * exactly as avits_block_forward computes them (W_q, W_k = the first 2D
 * output rows of W_qkv, or of W_in for the single kind; stream weights per
 * row as there).
 * x_in [S, D], pos [S, 3] int32; q_out, k_out [S, D] = [S, H, d] (distinct,
 * not aliasing x_in), which is the layout avits_score and avits_joint_lse
 * take: the image queries are q_out + n_txt * D, the text keys k_out, the
 * joint key set k_out itself.  workspace >= avits_block_qk_workspace_bytes(S,
 * H, d, dtype) bytes (S*D elements).  S == 0 is a no-op.  Other arguments
 * and errors as avits_block_forward.
 * ---------------------------------------------------------------------- */
size_t avits_block_qk_workspace_bytes(int64_t S, int32_t H, int32_t d, int dtype);
int avits_block_qk(const void* x_in, const int32_t* pos, float pos_scale, int64_t n_txt, int64_t n_img,
                   const avits_block_weights* w, int32_t H, int32_t d, int dtype,
                   void* q_out, void* k_out, void* workspace, size_t workspace_bytes,
                   void* stream);

/* ------------------------------------------------------------------------
 * avits_scatter — Stage-3 re-layout (Section 3.2): canvas[idx[j]] =
 * out[row_offset + j] for j < k.  out [row_offset + k, D], idx [k] int32
 * (unique, in [0, n_canvas)), canvas [n_canvas, D].  An index outside
 * [0, n_canvas) is skipped on the device (its row is not written), so no
 * access leaves the canvas.  k == 0 enqueues nothing.  Requires
 * n_canvas >= 1.
 * ---------------------------------------------------------------------- */
int avits_scatter(const void* out, const int32_t* idx, int64_t k, int64_t row_offset,
                  int64_t D, int64_t n_canvas, int dtype, void* canvas, void* stream);

/* ------------------------------------------------------------------------
 * avits_scatter_batched — the Stage-3 re-layout for B images in one launch:
 * for image b and j < k_b = idx_off[b + 1] - idx_off[b],
 *   canvas[b*N + idx[idx_off[b] + j]] = out[row_off[b] + j].
 * out [*, D] (the packed block output), idx the concatenated selections
 * (each unique, < N), canvas [B, N, D]; idx_off [B + 1] and row_off [B] are
 * host int64 arrays (idx_off[0] == 0).  1 <= B <= 64, each k_b in [0, N];
 * nothing is enqueued when every k_b is 0.  Errors as avits_scatter.
 * ---------------------------------------------------------------------- */
int avits_scatter_batched(const void* out, const int32_t* idx, const int64_t* idx_off, int32_t B,
                          const int64_t* row_off, int64_t N, int64_t D, int dtype, void* canvas,
                          void* stream);

/* ------------------------------------------------------------------------
 * avits_grid_positions / avits_scale_positions — RoPE positions of grid
 * tokens (Section 3.1: token i sits at spatial coordinate p_i = (r_i, c_i)):
 *   avits_grid_positions:  pos[r] = (frame, (r / W) scale + offset,
 *                                            (r % W) scale + offset)
 *   for raster rows r < rows of a grid W wide (e.g. scale 1, offset 0: a
 *   grid's own integer positions; scale 4, offset 1: low-res block centres
 *   in half units of the 2x grid);
 *   avits_scale_positions: dst[r] = src[r] * scale, all three coordinates
 *   (e.g. scale 2: positions in half units).
 * pos, src, dst [rows, 3] int32 device pointers (src and dst may be the
 * same).  Requires W >= 1 and rows >= 0; rows == 0 enqueues nothing.
 * ---------------------------------------------------------------------- */
int avits_grid_positions(int32_t* pos, int64_t rows, int32_t W, int32_t frame, int32_t scale, int32_t offset,
                         void* stream);
int avits_scale_positions(const int32_t* src, int64_t rows, int32_t scale, int32_t* dst, void* stream);

/* ------------------------------------------------------------------------
 * avits_gather_mixed — the mixed-resolution sequence of Stage 2 (Section
 * 3.2): the tokens selected at low-res granularity are expanded to their four
 * high-res children by 2x upsampling; the other M' - K low-res tokens stay in
 * the sequence at low resolution.
 *   compact rows [0, n_prefix)          = prefix
 *   compact row n_prefix + 4j + 2dr + dc = up(lowres) at high-res pixel
 *       (2r + dr, 2c + dc), (r, c) = divmod(idx[j], W_lr), dr, dc in {0, 1}
 *   compact row n_prefix + 4K + m       = lowres[p_m], p_m the m-th
 *       unselected low-res index in ascending order
 * up() is nearest (the parent's row) or bilinear (as avits_gather_upsample).
 * pos [4K + M' - K, 3] int32 is written for the rows after the prefix, in
 * half units (twice the high-res coordinate, so a low-res token at its 2x2
 * block centre stays integral): a child (0, 2(2r+dr), 2(2c+dc)); a kept
 * token (0, 4r + 1, 4c + 1).  Run the block with pos_scale = 0.5 on these
 * and with the prefix positions doubled.  children [4K] int32, if not NULL,
 * receives the children's high-res raster indices in ascending order (the
 * idx avits_gather_upsample and avits_scatter take for the Stage-3 full
 * expansion).
 * lowres [M', D] with M' = H_lr * W_lr; prefix [n_prefix, D] (may be NULL if
 * n_prefix == 0); idx [K] int32, ascending and unique in [0, M') (as
 * avits_select writes it; other contents give unspecified rows but no access
 * outside the buffers); compact [n_prefix + 3K + M', D], not aliasing the
 * inputs.  Requires D * elem_size % 16 == 0.  0 <= K <= M'.
 * ---------------------------------------------------------------------- */
int avits_gather_mixed(const void* lowres, const void* prefix, const int32_t* idx, int64_t k,
                       int32_t H_lr, int32_t W_lr, int64_t n_prefix, int64_t D, int mode, int dtype,
                       void* compact, int32_t* pos, int32_t* children, void* stream);

/* ------------------------------------------------------------------------
 * avits_scatter_mixed — the inverse re-layout after the Stage-2 blocks: each
 * expanded row goes to its high-res pixel, each kept row to its low-res slot.
 *   canvas_hr[(2r+dr) * 2W_lr + 2c+dc] = out[row_offset + 4j + 2dr + dc]
 *   state_lr[p_m]                       = out[row_offset + 4K + m]
 * with the layout of avits_gather_mixed.  out [row_offset + 3K + M', D];
 * canvas_hr [4M', D] (may be NULL if K == 0); state_lr [M', D] (may be NULL
 * if K == M'; may alias the gather's lowres).  Other rows of canvas_hr and
 * state_lr are left as they are.  idx and errors as avits_gather_mixed.
 * ---------------------------------------------------------------------- */
int avits_scatter_mixed(const void* out, const int32_t* idx, int64_t k, int32_t H_lr, int32_t W_lr,
                        int64_t row_offset, int64_t D, int dtype, void* canvas_hr, void* state_lr,
                        void* stream);

/* ------------------------------------------------------------------------
 * avits_joint_lse — log-sum-exp of each image query's logits over the joint
 * key set (the softmax normaliser of Eq. dit_attn):
 *   lse[h, i] = log sum_{j < Nk} exp(q_ih . k_jh / sqrt(d))   (natural log)
 * q [N, H, d], k_all [Nk, H, d] (dtype); lse [H, N] fp32.
 * Requires N >= 1, Nk >= 1, d in {64, 128}.
 * ---------------------------------------------------------------------- */
int avits_joint_lse(const void* q, const void* k_all, int64_t N, int64_t Nk,
                    int32_t H, int32_t d, int dtype, float* lse, void* stream);

/* ------------------------------------------------------------------------
 * avits_joint_attention_stats — the joint softmax statistics of each image
 * query in one pass over the joint key set (Eq. dit_attn), with the
 * image-to-text attention mass of Eq. spatial per head tracked inside the
 * online softmax under the same running maximum:
 *   lse[h, i]   = log sum_{j < Nk} exp(q_ih . k_jh / sqrt(d))      (natural log)
 *   mass[h, i] (+)= sum_{j < L} exp(q_ih . k_jh / sqrt(d) - lse[h, i])
 * The first L rows of k_all are the text keys.  With accumulate != 0 the
 * mass is added to what `mass` holds, so the probes of several blocks or
 * steps sum into one buffer (the aggregation over selected blocks and
 * steps of Section 3.3.1; avits_score_from_mass divides by their count).
 * q [N, H, d], k_all [Nk, H, d] (dtype); lse [H, N] fp32 or NULL; mass
 * [H, N] fp32.  Requires N, Nk, H >= 1, 0 <= L <= Nk, d in {64, 128}.
 * ---------------------------------------------------------------------- */
int avits_joint_attention_stats(const void* q, const void* k_all, int64_t N, int64_t Nk,
                                int64_t L, int32_t H, int32_t d, int dtype, float* lse,
                                float* mass, int accumulate, void* stream);

/* ------------------------------------------------------------------------
 * avits_score_from_mass — the fused importance score from precomputed
 * attention masses (Eq. spatial, aggregated) and N_T feature snapshots
 * (Eqs. zbar and step_var for general N_T):
 *   A_i = (1 / (H count)) sum_h mass[h, i]
 *   V_i = (1 / D_f) sum_c sum_k (z_k[i, c] - zbar[i, c])^2 / (N_T - 1)
 *   S_i = alpha (A_i - min A) / (max A - min A + eps)
 *       + (1 - alpha) (V_i - min V) / (max V - min V + eps)
 * mass [H, N] fp32 with row stride mass_ld >= N (the sum of `count`
 * probes; e.g. the image-row columns of a block's [H, S] mass, mass_ld = S
 * and the pointer advanced by the text rows); snapshots: a host array of
 * n_t device pointers, snapshot k [N, D_f] (dtype), consecutive steps in
 * order; scores, a_raw, v_raw as avits_score.  workspace >=
 * avits_score_workspace_bytes(N, H).  Requires 2 <= n_t <= 16, count >= 1.  With one probe and n_t = 2 it computes what avits_score
 * computes, from the mass instead of the query/key recomputation.
 * ---------------------------------------------------------------------- */
int avits_score_from_mass(const float* mass, int64_t mass_ld, int32_t H, int32_t count,
                          const void* const* snapshots, int32_t n_t, int64_t N, int64_t D_f, float alpha, float eps,
                          int dtype, float* scores, float* a_raw, float* v_raw,
                          void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Around the path: the Stage-2 denoising steps of Section 3.2 advance only
 * the selected tokens, with the Euler rule of Eq. euler applied to their
 * latents.  Kept in compact form ([k, C], the selected rows in ascending
 * token order), one Stage-2 step is
 *     h = avits_linear(z_sel)                 latent -> hidden rows
 *     blocks on [text; ref; h]                (avits_block_forward ...)
 *     v = avits_final_layer(image rows)       hidden -> velocity [k, C]
 *     avits_euler_update(z_sel, v, dt)        z_sel += dt * v
 * and avits_scatter puts z_sel into the canvas when Stage 2 ends.  The
 * embedder and the output layer are the model's (FLUX-style: a linear map;
 * a modulated layer norm and a linear map), not the paper's.
 *
 * avits_linear: out[m, n] = sum_k x[m, k] w[n, k] + b[n] (b may be NULL).
 * x [M, K], w [N, K], b [N], out [M, N], all of dtype, row-major, device
 * pointers owned by the caller; fp32 accumulation, one rounding.  Requires
 * 0 <= M < 2^31 (M == 0 enqueues nothing), K a positive multiple of 64, N a
 * positive multiple of 8.
 *
 * avits_final_layer: out = avits_linear(LN(x) * (1 + scale) + shift, w, b)
 * with LN the layer norm without affine parameters (eps 1e-6, biased
 * variance, as in the block), mod [2, D] = (shift; scale).  x [M, D],
 * w [C, D], b [C] or NULL, out [M, C]; D a positive multiple of 64, C of 8.
 * The normalised rows are rounded to dtype in the workspace
 * (>= avits_final_layer_workspace_bytes(M, D, dtype)) before the GEMM.
 *
 * avits_euler_update: z[i] = z[i] + dt * v[i] for i < n, in fp32, rounded
 * once to dtype; z updated in place.  z and v 16-byte aligned device
 * pointers, not overlapping; dt finite (negative when integrating from
 * t = 1 towards t = 0); n == 0 enqueues nothing.
 *
 * Errors: AVITS_ERR_INVALID_ARG for shapes outside the limits or null
 * pointers, AVITS_ERR_UNSUPPORTED for a dtype other than F32 / BF16,
 * AVITS_ERR_WORKSPACE for a short workspace.
 * ---------------------------------------------------------------------- */
int avits_linear(const void* x, int64_t M, int64_t K, const void* w, const void* b, int64_t N, int dtype,
                 void* out, void* stream);
size_t avits_final_layer_workspace_bytes(int64_t M, int64_t D, int dtype);
int avits_final_layer(const void* x, int64_t M, int64_t D, const void* mod, const void* w, const void* b,
                      int64_t C, int dtype, void* out, void* workspace, size_t workspace_bytes, void* stream);
int avits_euler_update(void* z, const void* v, int64_t n, float dt, int dtype, void* stream);

/* ------------------------------------------------------------------------
 * avits_noise_reinject — coordinate-bound noise re-injection (Section 3.2:
 * into the mixed-resolution sequence when Stage 2 starts, into the full
 * grid when Stage 3 starts): for each of `rows` rows of x [rows, C],
 *   x[r] <- (1 - t) x[r] + t eps(row r's coordinate)
 * in fp32, rounded once to dtype (t == 1 writes eps without reading x).
 * eps is one fixed standard-normal field over the H_hr x W_hr high-res grid:
 * channel c of pixel p (raster index) is the Box-Muller normal of word c % 4
 * of Philox-4x32-10 (Salmon et al., SC 2011) at counter (p, c / 4, 0, 0)
 * and key (seed low 32 bits, seed high 32 bits), uniforms
 * (w >> 8 + 1/2) 2^-24, words (0, 1) -> channels (4j, 4j + 1) as
 * (r cos 2 pi u1, r sin 2 pi u1) with r = sqrt(-2 ln u0), words (2, 3) ->
 * (4j + 2, 4j + 3).  A low-res token (a 2x2 block) takes the sum of its four
 * children's noise halved.  A row's coordinate, by rows_kind:
 *   0  raster rows of the high-res grid (row r = pixel r; rows <= H_hr W_hr)
 *   1  positions in half units, pos [rows, 3] int32 (frame, Y, X), as
 *      avits_gather_mixed writes them: even (Y, X) = pixel (Y/2, X/2), odd
 *      (Y, X) = (4r+1, 4c+1) = low-res block (r, c)
 *   2  raster rows of the low-res grid (row r = block r; rows <=
 *      H_hr W_hr / 4): the downsampled noise, e.g. Stage 1's initial latent
 * x device pointer [rows, C] (dtype), C a positive multiple of 4; pos device
 * pointer (kind 1) or NULL.  Requires even H_hr, W_hr >= 2, 0 <= t <= 1.
 * rows == 0 enqueues nothing.
 *
 * avits_noise_bits — the generator's raw stream for the parity checks:
 * bits[i, c] = word c % 4 of Philox-4x32-10 at counter (first_pixel + i,
 * c / 4, 0, 0), key as above; bits [n_pixels, C] uint32 device pointer.
 * ---------------------------------------------------------------------- */
int avits_noise_reinject(void* x, int64_t rows, int64_t C, const int32_t* pos, int32_t rows_kind,
                         int32_t H_hr, int32_t W_hr, float t, uint64_t seed, int dtype, void* stream);
int avits_noise_bits(int64_t first_pixel, int64_t n_pixels, int64_t C, uint64_t seed, uint32_t* bits,
                     void* stream);

/* ------------------------------------------------------------------------
 * Launch timing (instrumentation for benchmarks; not part of the method).
 * While enabled, every kernel the library enqueues is bracketed by a pair of
 * HIP events on the caller's stream.  avits_timing_read() waits for the
 * recorded events and returns the accumulated time and launch count of one
 * launch family: "score_spatial", "score_combine", "score_finalize",
 * "select", "gather_upsample", "scatter", "ln_mod", "gemm_qkv", "gemm_o",
 * "gemm_mlp_in", "gemm_mlp_out", "gemm_single_in", "gemm_single_out",
 * "splitk_reduce", "qk_rope", "attention", "joint_lse" (also the
 * statistics pass of avits_joint_attention_stats), "gather_mixed",
 * "scatter_mixed", "linear", "final_linear" (the GEMM of avits_final_layer;
 * its layer norm counts as "ln_mod"), "euler", "noise"; "gemm" returns the
 * sum of the six GEMM families (the GEMM kernels alone: the split-K
 * reduction that follows a split launch is "splitk_reduce").  Unknown
 * family -> AVITS_ERR_INVALID_ARG.
 * avits_timing_reset() waits for pending events and zeroes every total.
 * Not thread-safe: use from one host thread.
 * ---------------------------------------------------------------------- */
int avits_timing_enable(int on);
void avits_timing_reset(void);
int avits_timing_read(const char* family, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif
#endif /* AVITS_H */
