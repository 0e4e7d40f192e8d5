"""One selective-upsampling step on one GPU: score -> select -> gather/upsample
-> joint-attention block -> scatter (Section 3.2 Stage 2 with the importance
estimator of Section 3.3), as a fixed launch sequence on one stream.

All buffers are allocated once at construction (torch device memory); run()
only enqueues the five library calls, so a step does no allocation and no
host<->device traffic.
"""
from __future__ import annotations

import dataclasses

from . import _binding as B


@dataclasses.dataclass
class StepShape:
    N: int          # high-res tokens scored (4 * H_lr * W_lr)
    H_lr: int
    W_lr: int
    L: int          # text tokens
    R: int          # reference tokens (always kept)
    k: int          # tokens selected
    D: int
    H: int
    D_f: int        # temporal-feature channels
    mlp_hidden: int

    @property
    def S(self):
        return self.L + self.R + self.k


def run_chain(blocks, cur, out_of, hbuf, pos, L: int, S: int, H: int, ws, stream=None, pos_scale=1.0,
              on_block=None, mass=None, n_mass: int = 0):
    """The blocks in order on the rows cur [S, D]: block i writes out_of(i);
    each block's first stage (LN + modulation) comes from the block before
    it, written by that block's last split-K reduce into hbuf[i % 2]
    (avits_block_forward_ex h_next -> h_in), so a stack of n blocks runs one
    layer-norm launch instead of n.  mass (with n_mass) accumulates the text
    mass of the first n_mass blocks.  Returns the last output."""
    n = len(blocks)
    for i, w in enumerate(blocks):
        nxt = out_of(i)
        nw = blocks[i + 1] if i + 1 < n else None
        B.avits_block_forward_ex(cur, nxt, pos, L, S - L, w, H, mass_out=mass if i < n_mass else None,
                                 mass_accumulate=True, workspace=ws, stream=stream, pos_scale=pos_scale,
                                 h_in=hbuf[i % 2][:S] if i else None,
                                 h_next=hbuf[(i + 1) % 2][:S] if nw is not None else None, next_weights=nw)
        if on_block is not None:
            on_block(i, cur, nxt)
        cur = nxt
    return cur


class SelectiveStep:
    def __init__(self, shape: StepShape, weights: B.BlockWeights, prefix_pos, dtype, device="cuda",
                 alpha=0.5, eps=1e-8, mode=B.UP_NEAREST, canvas=None, keep_lse=False):
        import torch
        s = shape
        self.shape, self.weights, self.alpha, self.eps, self.mode = s, weights, alpha, eps, mode
        f32, i32 = torch.float32, torch.int32
        self.scores = torch.empty(s.N, dtype=f32, device=device)
        self.a_raw = torch.empty(s.N, dtype=f32, device=device)
        self.v_raw = torch.empty(s.N, dtype=f32, device=device)
        self.idx = torch.empty(s.k, dtype=i32, device=device)
        self.compact = torch.empty(s.S, s.D, dtype=dtype, device=device)
        self.pos = torch.empty(s.S, 3, dtype=i32, device=device)
        self.pos[: s.L + s.R].copy_(prefix_pos)
        self.x_out = torch.empty(s.S, s.D, dtype=dtype, device=device)
        self.canvas = canvas  # None: the canvas aliases highres_prev (in-place update)
        self._step_canvas = canvas
        self.lse = torch.empty(s.H, s.S, dtype=f32, device=device) if keep_lse else None
        d = s.D // s.H
        self.ws_score = torch.empty(max(B.avits_score_workspace_bytes(s.N, s.H), 1), dtype=torch.uint8, device=device)
        self.ws_select = torch.empty(max(B.avits_select_workspace_bytes(s.N), 1), dtype=torch.uint8, device=device)
        code = B.BF16 if dtype == torch.bfloat16 else B.F32
        self.ws_block = torch.empty(
            max(B.avits_block_workspace_bytes(weights.kind, s.S, s.H, d, s.mlp_hidden, code), 1),
            dtype=torch.uint8, device=device)
        # bf16 double block: the gather also writes the block's first stage
        # (the modulated layer norm of every compact row) while each row is
        # in registers, and the block starts from it.
        self.ln_vectors = None
        if code == B.BF16 and weights.kind == B.BLOCK_DOUBLE and s.D % 8 == 0 and s.D <= 4096:
            mt, mi = weights.tensors["txt"].get("mod"), weights.tensors["img"].get("mod")
            if mi is not None:
                mt = mi if mt is None else mt
                self.ln_vectors = (mt[0], mt[1], mi[0], mi[1])
                self.h = torch.empty(s.S, s.D, dtype=dtype, device=device)

    # Up to 8192 scored tokens the selection runs inside the scoring call
    # (avits_score_select, one launch less); select() then has nothing left
    # to do.  At 16384 the one-workgroup normalisation costs more than the
    # launch it saves (measured on MI355X), so the two calls stay separate.
    FUSED_MAX_N = 8192

    def score(self, latent_q, text_k, row_lse, feat_t, feat_prev, stream=None):
        if self.shape.N <= self.FUSED_MAX_N:
            B.avits_score_select(latent_q, text_k, row_lse, feat_t, feat_prev, self.alpha, self.eps, self.scores,
                                 self.shape.k, self.idx, self.a_raw, self.v_raw, self.ws_score, stream)
        else:
            B.avits_score(latent_q, text_k, row_lse, feat_t, feat_prev, self.alpha, self.eps, self.scores,
                          self.a_raw, self.v_raw, self.ws_score, stream)

    def select(self, stream=None):
        if self.shape.k and self.shape.N > self.FUSED_MAX_N:
            B.avits_select(self.scores, self.shape.k, self.idx, self.ws_select, stream)

    def gather(self, lowres, highres_prev, prefix, stream=None):
        s = self.shape
        canvas = highres_prev if self.canvas is None else self.canvas
        if self.ln_vectors is not None:
            B.avits_gather_upsample_ln(lowres, highres_prev, prefix, self.idx, s.H_lr, s.W_lr, self.compact,
                                       self.pos[s.L + s.R:], canvas, s.L, *self.ln_vectors, self.h, self.mode,
                                       stream)
        else:
            B.avits_gather_upsample(lowres, highres_prev, prefix, self.idx, s.H_lr, s.W_lr, self.compact,
                                    self.pos[s.L + s.R:], canvas, self.mode, stream)
        self._step_canvas = canvas

    # The scatter rides on the block's last projection (the image rows'
    # outputs go to their canvas rows from the same epilogue); scatter()
    # then has nothing left to do.
    def block(self, stream=None):
        s = self.shape
        B.avits_block_forward_ex(self.compact, self.x_out, self.pos, s.L, s.R + s.k, self.weights, s.H,
                                 lse_out=self.lse, workspace=self.ws_block, stream=stream,
                                 scatter_idx=self.idx if s.k else None,
                                 canvas=self._step_canvas if s.k else None,
                                 h_in=self.h if self.ln_vectors is not None else None)

    def scatter(self, highres_prev, stream=None):
        pass

    def run(self, latent_q, text_k, row_lse, feat_t, feat_prev, lowres, highres_prev, prefix, stream=None):
        self.score(latent_q, text_k, row_lse, feat_t, feat_prev, stream)
        self.select(stream)
        self.gather(lowres, highres_prev, prefix, stream)
        self.block(stream)
        self.scatter(highres_prev, stream)


class StackStep:
    """One denoising step of a selective block stack (Section 3.2 Stage 2 over
    the whole backbone, the importance taken from its first double block):

      probe    double block 0's first stage on [prefix; X_prev] -> q, k
      lse      joint log-sum-exp of the image queries over [prefix; image] keys
      score    spatial (text mass) + temporal (X_prev vs X_prev2) -> S
      select   top-k of S
      gather   compact = [prefix; X_prev[idx]], canvas = X_prev on idx, else up(lowres)
      blocks   the double blocks, then the single blocks, on the compacted rows
      scatter  canvas[idx] = last block's image rows  -> X_new

    Buffers are allocated once; run() enqueues library calls only.  The
    prefix rows ([text; ref]) use the text weights for the text rows and the
    image weights for the reference rows, as in the block.  ``on_block(i, x_in,
    x_out)``, if given, is called after block i is enqueued (for inspection).

    ``fused=True`` takes the spatial importance from the joint-softmax pass
    itself (avits_joint_attention_stats, the text mass tracked beside the
    normaliser) and scores with avits_score_from_mass; ``probe_blocks`` lists
    the double blocks whose first stages are probed, their masses averaged
    (fused only; the default probes block 0).
    """

    def __init__(self, shape: StepShape, doubles: list, singles: list, prefix_pos, dtype, device="cuda",
                 alpha=0.5, eps=1e-8, mode=B.UP_NEAREST, fused=False, probe_blocks=(0,)):
        import torch
        s = shape
        if not doubles:
            raise ValueError("the probe needs at least one double block")
        self.shape, self.doubles, self.singles = s, list(doubles), list(singles)
        self.alpha, self.eps, self.mode = alpha, eps, mode
        self.fused, self.probe_blocks = fused, tuple(probe_blocks)
        if not self.probe_blocks or any(b < 0 or b >= len(self.doubles) for b in self.probe_blocks):
            raise ValueError("probe_blocks must name double blocks")
        if not fused and self.probe_blocks != (0,):
            raise ValueError("several probe blocks need fused=True")
        f32, i32 = torch.float32, torch.int32
        d = s.D // s.H
        code = B.BF16 if dtype == torch.bfloat16 else B.F32
        LR = s.L + s.R
        self.q_prefix = torch.empty(max(LR, 1), s.D, dtype=dtype, device=device)
        self.q_img = torch.empty(s.N, s.D, dtype=dtype, device=device)
        self.k_all = torch.empty(LR + s.N, s.D, dtype=dtype, device=device)
        self.lse = torch.empty(s.H, s.N, dtype=f32, device=device)
        self.mass = torch.empty(s.H, s.N, dtype=f32, device=device)
        self.prefix_pos = torch.as_tensor(prefix_pos, dtype=i32).to(device)
        self.img_pos = torch.empty(s.N, 3, dtype=i32, device=device)
        B.avits_grid_positions(self.img_pos, 2 * s.W_lr)      # (0, r, c) on the high-res grid
        self.scores = torch.empty(s.N, dtype=f32, device=device)
        self.a_raw = torch.empty(s.N, dtype=f32, device=device)
        self.v_raw = torch.empty(s.N, dtype=f32, device=device)
        self.idx = torch.empty(s.k, dtype=i32, device=device)
        self.compact = torch.empty(s.S, s.D, dtype=dtype, device=device)
        self.pos = torch.empty(s.S, 3, dtype=i32, device=device)
        self.pos[:LR].copy_(self.prefix_pos)
        self.x = [torch.empty(s.S, s.D, dtype=dtype, device=device) for _ in range(2)]
        self.hbuf = [torch.empty(s.S, s.D, dtype=dtype, device=device) for _ in range(2)]
        self.ws_score = torch.empty(max(B.avits_score_workspace_bytes(s.N, s.H), 1), dtype=torch.uint8, device=device)
        self.ws_select = torch.empty(max(B.avits_select_workspace_bytes(s.N), 1), dtype=torch.uint8, device=device)
        need = max(B.avits_block_qk_workspace_bytes(max(LR, s.N), s.H, d, code),
                   B.avits_block_workspace_bytes(B.BLOCK_DOUBLE, s.S, s.H, d, s.mlp_hidden, code),
                   B.avits_block_workspace_bytes(B.BLOCK_SINGLE, s.S, s.H, d, s.mlp_hidden, code) if singles else 0)
        self.ws_block = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
        self.out = None

    def _qk(self, w, x_prev, prefix, stream):
        s = self.shape
        LR = s.L + s.R
        if LR:
            B.avits_block_qk(prefix, self.prefix_pos, s.L, s.R, w, s.H, self.q_prefix[:LR], self.k_all[:LR],
                             self.ws_block, stream)
        B.avits_block_qk(x_prev, self.img_pos, 0, s.N, w, s.H, self.q_img, self.k_all[LR:], self.ws_block, stream)

    def probe(self, x_prev, prefix, stream=None):
        """The probe blocks' queries and keys, then the joint LSE (and, fused,
        the text mass summed over the probe blocks)."""
        s = self.shape
        LR = s.L + s.R
        d = s.D // s.H
        q, k = self.q_img.view(s.N, s.H, d), self.k_all.view(LR + s.N, s.H, d)
        for n, b in enumerate(self.probe_blocks):
            self._qk(self.doubles[b], x_prev, prefix, stream)
            if self.fused:
                B.avits_joint_attention_stats(q, k, s.L, self.mass, lse=self.lse, accumulate=n > 0, stream=stream)
            else:
                B.avits_joint_lse(q, k, self.lse, stream)

    def run(self, x_prev, x_prev2, lowres, prefix, canvas, stream=None, on_block=None):
        """X_new (written to ``canvas``, which must not alias x_prev) from X_prev and X_prev2."""
        s = self.shape
        LR = s.L + s.R
        d = s.D // s.H
        if canvas.data_ptr() == x_prev.data_ptr():
            raise ValueError("canvas must not alias x_prev: X_prev is the next step's X_prev2")
        self.probe(x_prev, prefix, stream)
        if self.fused:
            B.avits_score_from_mass(self.mass, len(self.probe_blocks), [x_prev2, x_prev], self.alpha, self.eps,
                                    self.scores, self.a_raw, self.v_raw, self.ws_score, stream)
        else:
            B.avits_score(self.q_img.view(s.N, s.H, d), self.k_all[:s.L].view(s.L, s.H, d), self.lse, x_prev,
                          x_prev2, self.alpha, self.eps, self.scores, self.a_raw, self.v_raw, self.ws_score, stream)
        if s.k:
            B.avits_select(self.scores, s.k, self.idx, self.ws_select, stream)
        B.avits_gather_upsample(lowres, x_prev, prefix if LR else None, self.idx, s.H_lr, s.W_lr, self.compact,
                                self.pos[LR:], canvas, self.mode, stream)
        cur = run_chain(self.doubles + self.singles, self.compact, lambda i: self.x[i % 2], self.hbuf, self.pos, s.L,
                        s.S, s.H, self.ws_block, stream, on_block=on_block)
        self.out = cur
        if s.k:
            B.avits_scatter(cur, self.idx, LR, canvas, stream)
        return canvas


class MixedStage2:
    """The paper's Stage 2 on one GPU (Section 3.2): score the M' low-res
    tokens from Stage 1's signals, keep the top K = floor(rho M'), expand them
    2x2 and keep the rest at low resolution in one mixed sequence, then run the
    block stack on that sequence for each Stage-2 step, and finally send the
    rows back (children to the high-res canvas, kept tokens to the low-res
    state).

      transition  probe (first stage of the probe double blocks on [prefix;
                  Z_lr] at low-res grid positions) -> text mass -> score from
                  the mass and the N_T low-res snapshots -> select K ->
                  gather_mixed
      step        the double blocks, then the single blocks, on the mixed
                  sequence with half-unit positions (pos_scale 0.5)
      leave       scatter_mixed into (canvas_hr, state_lr)

    ``children`` holds the expanded tokens' high-res indices in ascending
    order, the idx the Stage-3 expansion (avits_gather_upsample) takes.
    Buffers are allocated once; the three calls enqueue library calls only.
    """

    def __init__(self, H_lr: int, W_lr: int, L: int, R: int, K: int, D: int, H: int, mlp_hidden: int,
                 doubles: list, singles: list, prefix_pos, dtype, device="cuda", alpha=0.5, eps=1e-8,
                 mode=B.UP_NEAREST, probe_blocks=(0,)):
        import torch
        if not doubles:
            raise ValueError("the probe needs at least one double block")
        Mp = H_lr * W_lr
        if not 0 <= K <= Mp:
            raise ValueError(f"K={K} outside [0, {Mp}]")
        self.H_lr, self.W_lr, self.L, self.R, self.K, self.D, self.H = H_lr, W_lr, L, R, K, D, H
        self.Mp, self.LR = Mp, L + R
        self.S = self.LR + 4 * K + Mp - K
        self.doubles, self.singles = list(doubles), list(singles)
        self.alpha, self.eps, self.mode, self.probe_blocks = alpha, eps, mode, tuple(probe_blocks)
        if not self.probe_blocks or any(b < 0 or b >= len(self.doubles) for b in self.probe_blocks):
            raise ValueError("probe_blocks must name double blocks")
        f32, i32 = torch.float32, torch.int32
        d = D // H
        code = B.BF16 if dtype == torch.bfloat16 else B.F32
        LR = self.LR
        prefix_pos = torch.as_tensor(prefix_pos, dtype=i32).to(device)
        self.prefix_pos = prefix_pos
        self.lr_pos = torch.empty(Mp, 3, dtype=i32, device=device)
        B.avits_grid_positions(self.lr_pos, W_lr)             # (0, r, c) on the low-res grid
        self.q_prefix = torch.empty(max(LR, 1), D, dtype=dtype, device=device)
        self.q_img = torch.empty(Mp, D, dtype=dtype, device=device)
        self.k_all = torch.empty(LR + Mp, D, dtype=dtype, device=device)
        self.lse = torch.empty(H, Mp, dtype=f32, device=device)
        self.mass = torch.empty(H, Mp, dtype=f32, device=device)
        self.scores = torch.empty(Mp, dtype=f32, device=device)
        self.idx = torch.empty(K, dtype=i32, device=device)
        self.children = torch.empty(4 * K, dtype=i32, device=device)
        self.x = torch.empty(self.S, D, dtype=dtype, device=device)
        self.pos = torch.empty(self.S, 3, dtype=i32, device=device)
        if LR:
            B.avits_scale_positions(prefix_pos, 2, self.pos[:LR])   # half units
        self.buf = [torch.empty(self.S, D, dtype=dtype, device=device) for _ in range(2)]
        self.hbuf = [torch.empty(self.S, D, dtype=dtype, device=device) for _ in range(2)]
        self.ws_score = torch.empty(max(B.avits_score_workspace_bytes(Mp, H), 1), dtype=torch.uint8, device=device)
        self.ws_select = torch.empty(max(B.avits_select_workspace_bytes(Mp), 1), dtype=torch.uint8, device=device)
        need = max(B.avits_block_qk_workspace_bytes(max(LR, Mp), H, d, code),
                   B.avits_block_workspace_bytes(B.BLOCK_DOUBLE, self.S, H, d, mlp_hidden, code),
                   B.avits_block_workspace_bytes(B.BLOCK_SINGLE, self.S, H, d, mlp_hidden, code) if singles else 0)
        self.ws_block = torch.empty(max(need, 1), dtype=torch.uint8, device=device)

    def transition(self, z_lr, snapshots, prefix, stream=None):
        """Select and build the mixed sequence from the low-res latent z_lr
        [M', D], Stage 1's N_T >= 2 low-res snapshots (oldest first) and the
        prefix rows [L + R, D]."""
        LR, Mp, H, D = self.LR, self.Mp, self.H, self.D
        d = D // H
        q, k = self.q_img.view(Mp, H, d), self.k_all.view(LR + Mp, H, d)
        for n, b in enumerate(self.probe_blocks):
            w = self.doubles[b]
            if LR:
                B.avits_block_qk(prefix, self.prefix_pos, self.L, self.R, w, H, self.q_prefix[:LR], self.k_all[:LR],
                                 self.ws_block, stream)
            B.avits_block_qk(z_lr, self.lr_pos, 0, Mp, w, H, self.q_img, self.k_all[LR:], self.ws_block, stream)
            B.avits_joint_attention_stats(q, k, self.L, self.mass, lse=self.lse, accumulate=n > 0, stream=stream)
        B.avits_score_from_mass(self.mass, len(self.probe_blocks), list(snapshots), self.alpha, self.eps,
                                self.scores, workspace=self.ws_score, stream=stream)
        if self.K:
            B.avits_select(self.scores, self.K, self.idx, self.ws_select, stream)
        B.avits_gather_mixed(z_lr, prefix if LR else None, self.idx if self.K else None, self.H_lr, self.W_lr,
                             self.x, self.pos[LR:], self.children if self.K else None, self.mode, stream)

    def step(self, stream=None, on_block=None):
        """One pass of the block stack over the mixed sequence; the result
        becomes the sequence the next step reads."""
        cur = run_chain(self.doubles + self.singles, self.x, lambda i: self.buf[i % 2], self.hbuf, self.pos, self.L,
                        self.S, self.H, self.ws_block, stream, pos_scale=0.5, on_block=on_block)
        self.x, self.buf[(len(self.doubles) + len(self.singles) - 1) % 2] = cur, self.x
        return self.x

    def leave(self, canvas_hr, state_lr, stream=None):
        """Children rows to canvas_hr [4M', D], kept rows to state_lr [M', D]."""
        B.avits_scatter_mixed(self.x, self.idx if self.K else None, self.H_lr, self.W_lr, self.LR,
                              canvas_hr if self.K else None, state_lr if self.K < self.Mp else None, stream)
        return canvas_hr, state_lr


class BatchedStep:
    """One selective-upsampling step for B images at once (a CFG pair, or
    several prompts): each image has its own scores, budget k_b, text rows
    and canvas; one selection launch covers all images, and one block pass
    runs every image's compacted sequence, rows packed by stream (the text
    rows of all images, then their [reference; selected] rows) with
    block-diagonal attention.

      score    S_b from image b's own q, text keys, LSE and features; one
               avits_score_batched launch when the inputs come stacked
      select   avits_select_batched over the B score vectors (k_b each)
      gather   the text rows into the text area (avits_scatter of the
               rows), [ref_b; X_prev,b[idx_b]] into image b's area and its
               canvas filled by upsampling (avits_gather_upsample, or one
               avits_gather_upsample_batched launch for stacked images)
      block    avits_block_forward_batched_ex over the packed rows (with
               mod_stride > 0 each image takes its own modulation block,
               images at different timesteps)
      scatter  canvas_b[idx_b] = image b's selected output rows (one
               avits_scatter_batched launch for stacked canvases)

    Buffers are allocated once; run() enqueues library calls only.
    """

    def __init__(self, shape: StepShape, ks: list, weights: B.BlockWeights, prefix_pos, dtype, device="cuda",
                 alpha=0.5, eps=1e-8, mode=B.UP_NEAREST, mod_stride: int = 0):
        import torch
        s = shape
        self.shape, self.ks, self.weights, self.alpha, self.eps, self.mode = s, list(ks), weights, alpha, eps, mode
        self.mod_stride = mod_stride
        Bn = len(self.ks)
        if not 1 <= Bn <= 16 or any(not 0 <= k <= s.N for k in self.ks):
            raise ValueError("1 <= B <= 16 images with 0 <= k_b <= N")
        i32, f32 = torch.int32, torch.float32
        self.txt_off = [s.L * b for b in range(Bn + 1)]
        self.img_off = [0]
        for k in self.ks:
            self.img_off.append(self.img_off[-1] + s.R + k)
        T = self.txt_off[-1]
        self.S_tot = T + self.img_off[-1]
        self.scores = torch.empty(Bn * s.N, dtype=f32, device=device)
        self.idx = torch.empty(max(sum(self.ks), 1), dtype=i32, device=device)
        self.out_off = [sum(self.ks[:b]) for b in range(Bn + 1)]
        self.x = torch.empty(self.S_tot, s.D, dtype=dtype, device=device)
        self.x_out = torch.empty(self.S_tot, s.D, dtype=dtype, device=device)
        self.pos = torch.zeros(self.S_tot, 3, dtype=i32, device=device)
        prefix_pos = torch.as_tensor(prefix_pos, dtype=i32).to(device)
        for b in range(Bn):
            self.pos[self.txt_off[b]:self.txt_off[b + 1]].copy_(prefix_pos[:s.L])
            a0 = T + self.img_off[b]
            self.pos[a0:a0 + s.R].copy_(prefix_pos[s.L:s.L + s.R])
        # Row indices of each image's text area in the packed rows (for the text-row copy).
        self.txt_rows = [torch.arange(self.txt_off[b], self.txt_off[b + 1], dtype=i32, device=device)
                         for b in range(Bn)]
        self.txt_rows_all = torch.arange(T, dtype=i32, device=device)
        d = s.D // s.H
        code = B.BF16 if dtype == torch.bfloat16 else B.F32
        self.ws_score = torch.empty(max(B.avits_score_batched_workspace_bytes(Bn, s.N, s.H), 1), dtype=torch.uint8,
                                    device=device)
        self.ws_block = torch.empty(
            max(B.avits_block_workspace_bytes(weights.kind, self.S_tot, s.H, d, s.mlp_hidden, code), 1),
            dtype=torch.uint8, device=device)

    def run(self, latent_q, text_k, row_lse, feat_t, feat_prev, lowres, highres_prev, text, ref, stream=None):
        """Per-image inputs, given either as lists over the images (one launch
        per image for that stage) or as tensors stacked over the images (one
        launch for all):

          score inputs   latent_q [B, N, H, d], text_k [B, L, H, d],
                         row_lse [B, H, N], feat_t, feat_prev [B, N, D_f]
          layout inputs  lowres [B, N/4, D], highres_prev [B, N, D] (the
                         canvases, updated in place), text [B, L, D],
                         ref [B, R, D] or None

        Lists hold the per-image tensors of the same shapes without the B."""
        import torch
        s = self.shape
        T = self.txt_off[-1]
        Bn = len(self.ks)
        if torch.is_tensor(latent_q):
            B.avits_score_batched(latent_q, text_k, row_lse, feat_t, feat_prev, self.alpha, self.eps,
                                  self.scores.view(Bn, s.N), workspace=self.ws_score, stream=stream)
        else:
            for b in range(Bn):
                B.avits_score(latent_q[b], text_k[b], row_lse[b], feat_t[b], feat_prev[b], self.alpha, self.eps,
                              self.scores[b * s.N:(b + 1) * s.N], workspace=self.ws_score, stream=stream)
        if sum(self.ks):
            B.avits_select_batched(self.scores, [b * s.N for b in range(Bn + 1)], self.ks, self.idx, stream=stream)
        img_rows = [T + a for a in self.img_off[:-1]]
        if torch.is_tensor(highres_prev):
            if s.L:
                B.avits_scatter(text.view(T, s.D), self.txt_rows_all, 0, self.x, stream)
            B.avits_gather_upsample_batched(lowres, highres_prev, ref if s.R else None, self.idx, self.out_off,
                                            s.H_lr, s.W_lr, self.x, img_rows, self.pos, highres_prev, self.mode,
                                            stream)
        else:
            for b in range(Bn):
                if s.L:
                    B.avits_scatter(text[b], self.txt_rows[b], 0, self.x, stream)
                a0 = img_rows[b]
                idx_b = self.idx[self.out_off[b]:self.out_off[b + 1]]
                B.avits_gather_upsample(lowres[b], highres_prev[b], ref[b] if s.R else None, idx_b, s.H_lr,
                                        s.W_lr, self.x[a0:a0 + s.R + self.ks[b]],
                                        self.pos[a0 + s.R:a0 + s.R + self.ks[b]], highres_prev[b], self.mode, stream)
        B.avits_block_forward_batched_ex(self.x, self.x_out, self.pos, self.txt_off, self.img_off, self.weights, s.H,
                                         self.mod_stride, workspace=self.ws_block, stream=stream)
        if torch.is_tensor(highres_prev):
            B.avits_scatter_batched(self.x_out, self.idx, self.out_off, [a + s.R for a in img_rows], highres_prev,
                                    stream)
        else:
            for b in range(Bn):
                if self.ks[b]:
                    idx_b = self.idx[self.out_off[b]:self.out_off[b + 1]]
                    B.avits_scatter(self.x_out, idx_b, img_rows[b] + s.R, highres_prev[b], stream)
        return highres_prev


class SelectedEuler:
    """Stage-2 denoising steps on the selected tokens alone (Section 3.2, with
    the Euler rule of Eq. euler): their latents stay compact, z_sel [k, C] in
    ascending token order, and each step runs

      embed    avits_linear: z_sel -> hidden rows behind the prefix
      blocks   the double blocks, then the single blocks, on [text; ref; rows]
      output   avits_final_layer on the selected rows -> velocity v [k, C]
      update   avits_euler_update: z_sel += dt v

    ``finish`` scatters z_sel into the latent canvas (avits_scatter).  The
    prefix rows (the text and reference hidden states) are rewritten at every
    step, since the blocks overwrite their buffers.  Buffers are allocated
    once; step() enqueues library calls only.
    """

    def __init__(self, k: int, L: int, R: int, C: int, D: int, H: int, mlp_hidden: int, doubles: list,
                 singles: list, embed_w, embed_b, final_mod, final_w, final_b, pos, dtype, device="cuda"):
        import torch
        if k < 1 or not (doubles or singles):
            raise ValueError("at least one selected token and one block")
        self.k, self.L, self.R, self.C, self.D, self.H = k, L, R, C, D, H
        self.doubles, self.singles = list(doubles), list(singles)
        self.embed_w, self.embed_b = embed_w, embed_b
        self.final_mod, self.final_w, self.final_b = final_mod, final_w, final_b
        S = L + R + k
        self.S = S
        self.pos = torch.as_tensor(pos, dtype=torch.int32).to(device)
        if tuple(self.pos.shape) != (S, 3):
            raise ValueError("pos must hold the positions of [text; ref; selected] rows")
        self.x = [torch.empty(S, D, dtype=dtype, device=device) for _ in range(2)]
        self.hbuf = [torch.empty(S, D, dtype=dtype, device=device) for _ in range(2)]
        self.v = torch.empty(k, C, dtype=dtype, device=device)
        self.prefix_rows = torch.arange(L + R, dtype=torch.int32, device=device)
        d = D // H
        code = B.BF16 if dtype == torch.bfloat16 else B.F32
        kinds = ([B.BLOCK_DOUBLE] if doubles else []) + ([B.BLOCK_SINGLE] if singles else [])
        self.ws_block = torch.empty(max(max(B.avits_block_workspace_bytes(kd, S, H, d, mlp_hidden, code)
                                            for kd in kinds), 1), dtype=torch.uint8, device=device)
        self.ws_final = torch.empty(max(B.avits_final_layer_workspace_bytes(k, D, code), 1), dtype=torch.uint8,
                                    device=device)
        self.last = None  # the buffer holding the last block's output after step()

    def step(self, z_sel, prefix, dt: float, stream=None, on_block=None):
        """One Euler step of the selected latents z_sel [k, C] (in place);
        prefix [L + R, D] holds the text and reference hidden rows."""
        s0 = self.L + self.R
        if s0:
            B.avits_scatter(prefix, self.prefix_rows, 0, self.x[0], stream)
        B.avits_linear(z_sel, self.embed_w, self.embed_b, self.x[0][s0:], stream)
        S = self.L + self.R + self.k
        last = run_chain(self.doubles + self.singles, self.x[0], lambda i: self.x[(i + 1) % 2], self.hbuf, self.pos,
                         self.L, S, self.H, self.ws_block, stream, on_block=on_block)
        self.last = last
        B.avits_final_layer(self.last[s0:], self.final_mod, self.final_w, self.final_b, self.v,
                            workspace=self.ws_final, stream=stream)
        B.avits_euler_update(z_sel, self.v, dt, stream)
        return z_sel

    def finish(self, z_sel, idx, canvas, stream=None):
        """canvas[idx[j]] = z_sel[j]: the selected latents back in place."""
        B.avits_scatter(z_sel, idx, 0, canvas, stream)
        return canvas


class ThreeStageSampler:
    """The three-stage dynamic-resolution sampler of Section 3.2 (Fig. 3a) on
    one GPU, every step a library call:

      stage 1      the low-res latent z1 [M', C] from the downsampled
                   coordinate-bound noise, n1 + nt Euler steps (Eq. euler) of
                   [text; embed(z1)] at the low-res grid positions; over the
                   last nt steps the snapshots of z1 and the text mass of the
                   image rows, taken inside every double block's own
                   attention (avits_block_forward_ex, accumulated)
      transition   scores from the mass and the snapshots (Eqs. spatial,
                   step_var, joint) -> top K = floor(rho M') (Eq. topk) ->
                   clean estimate z1 - t v -> the mixed sequence (selected
                   tokens expanded 2x2, the rest kept) -> coordinate-bound
                   noise re-injected at t
      stage 2      n2 Euler steps of the mixed sequence (half-unit positions,
                   pos_scale 0.5)
      transition   clean estimate -> expanded rows to their pixels, kept rows
                   upsampled around them -> noise re-injected at t; rows in
                   raster order
      stage 3      n3 Euler steps of the full grid

    Each step embeds the latents (avits_linear), runs the double then the
    single blocks on [text; rows], maps the image rows to the velocity
    (avits_final_layer) and updates the latents (avits_euler_update).  The
    time grid is uniform, t_i = 1 - i / (n1 + nt + n2 + n3).  Buffers are
    allocated once; the stage methods enqueue library calls only.  After a
    run, z1 / snaps / mass / scores / idx / z2 / z3 hold each stage's state.
    """

    def __init__(self, H_lr: int, W_lr: int, L: int, C: int, D: int, H: int, mlp_hidden: int, doubles: list,
                 singles: list, sampler_w: dict, prefix_pos, K: int, n1: int, nt: int, n2: int, n3: int, dtype,
                 seed: int, alpha=0.5, eps=1e-8, device="cuda"):
        import torch
        if not doubles:
            raise ValueError("the text mass needs at least one double block")
        Mp = H_lr * W_lr
        if not 0 <= K <= Mp or nt < 2 or min(n1, n2, n3) < 0:
            raise ValueError("0 <= K <= M', nt >= 2 snapshots, step counts >= 0")
        self.H_lr, self.W_lr, self.L, self.C, self.D, self.H = H_lr, W_lr, L, C, D, H
        self.Mp, self.N, self.K = Mp, 4 * Mp, K
        self.doubles, self.singles, self.sw = list(doubles), list(singles), sampler_w
        self.n1, self.nt, self.n2, self.n3 = n1, nt, n2, n3
        self.seed, self.alpha, self.eps = seed, alpha, eps
        n = n1 + nt + n2 + n3
        self.t = [1.0 - i / n for i in range(n + 1)]
        self.S1, self.S2, self.S3 = L + Mp, L + 4 * K + Mp - K, L + 4 * Mp
        f32, i32 = torch.float32, torch.int32
        mk = lambda *shape, dt=dtype: torch.empty(*shape, dtype=dt, device=device)  # noqa: E731
        self.z1, self.v1 = mk(Mp, C), mk(Mp, C)
        self.snaps = [mk(Mp, C) for _ in range(nt)]
        self.mass = mk(H, self.S1, dt=f32)
        self.scores = mk(Mp, dt=f32)
        self.idx = mk(max(K, 1), dt=i32)
        self.children = mk(max(4 * K, 1), dt=i32)
        self.z2, self.v2 = mk(self.S2 - L, C), mk(self.S2 - L, C)
        self.z3, self.v3 = mk(self.N, C), mk(self.N, C)
        self.state = mk(Mp, C)
        self.g_rows, self.g_pos = mk(max(4 * K, 1), C), mk(max(4 * K, 1), 3, dt=i32)
        self.x = [mk(self.S3, D) for _ in range(2)]
        self.hbuf = [mk(self.S3, D) for _ in range(2)]
        prefix_pos = torch.as_tensor(prefix_pos, dtype=i32).to(device)
        self.pos1, self.pos2, self.pos3 = mk(self.S1, 3, dt=i32), mk(self.S2, 3, dt=i32), mk(self.S3, 3, dt=i32)
        if L:
            self.pos1[:L].copy_(prefix_pos)
            self.pos3[:L].copy_(prefix_pos)
            B.avits_scale_positions(prefix_pos, 2, self.pos2[:L])       # half units
        B.avits_grid_positions(self.pos1[L:], W_lr)                     # (0, r, c) low-res
        B.avits_grid_positions(self.pos3[L:], 2 * W_lr)                 # (0, r, c) high-res
        self.prefix_rows = torch.arange(max(L, 1), dtype=i32, device=device)
        d = D // H
        code = B.BF16 if dtype == torch.bfloat16 else B.F32
        kinds = [B.BLOCK_DOUBLE] + ([B.BLOCK_SINGLE] if singles else [])
        self.ws_block = mk(max(B.avits_block_workspace_bytes(kd, self.S3, H, d, mlp_hidden, code) for kd in kinds),
                           dt=torch.uint8)
        self.ws_final = mk(max(B.avits_final_layer_workspace_bytes(self.N, D, code), 1), dt=torch.uint8)
        self.ws_score = mk(max(B.avits_score_workspace_bytes(Mp, H), 1), dt=torch.uint8)
        self.ws_select = mk(max(B.avits_select_workspace_bytes(Mp), 1), dt=torch.uint8)

    # One Euler step of latents z (rows behind the prefix) at positions pos.
    def _step(self, z, v, pos, S, dt, prefix, pos_scale=1.0, collect=False, stream=None):
        L = self.L
        x0, x1 = self.x[0][:S], self.x[1][:S]
        if L:
            B.avits_scatter(prefix, self.prefix_rows[:L], 0, x0, stream)
        B.avits_linear(z, self.sw["embed_w"], self.sw["embed_b"], x0[L:], stream)
        cur = run_chain(self.doubles + self.singles, x0, lambda i: (x1, x0)[i % 2], self.hbuf, pos, L, S, self.H,
                        self.ws_block, stream, pos_scale=pos_scale, mass=self.mass if collect else None,
                        n_mass=len(self.doubles))
        B.avits_final_layer(cur[L:], self.sw["final_mod"], self.sw["final_w"], self.sw["final_b"], v,
                            workspace=self.ws_final, stream=stream)
        B.avits_euler_update(z, v, dt, stream)

    def stage1(self, prefix, stream=None):
        B.avits_noise_reinject(self.z1, 1.0, self.seed, 2 * self.H_lr, 2 * self.W_lr, rows_kind=B.NOISE_LOWRES,
                               stream=stream)
        self.mass.zero_()
        for i in range(self.n1 + self.nt):
            self._step(self.z1, self.v1, self.pos1, self.S1, self.t[i + 1] - self.t[i], prefix,
                       collect=i >= self.n1, stream=stream)
            if i >= self.n1:
                self.snaps[i - self.n1].copy_(self.z1)

    def transition12(self, stream=None):
        L, K = self.L, self.K
        t_s = self.t[self.n1 + self.nt]
        B.avits_score_from_mass(self.mass[:, L:], self.nt * len(self.doubles), self.snaps, self.alpha, self.eps,
                                self.scores, workspace=self.ws_score, stream=stream)
        if K:
            B.avits_select(self.scores, K, self.idx[:K], self.ws_select, stream)
        B.avits_euler_update(self.z1, self.v1, -t_s, stream)          # clean estimate z1 - t v
        B.avits_gather_mixed(self.z1, None, self.idx[:K] if K else None, self.H_lr, self.W_lr, self.z2,
                             self.pos2[L:], self.children[:4 * K] if K else None, stream=stream)
        B.avits_noise_reinject(self.z2, t_s, self.seed, 2 * self.H_lr, 2 * self.W_lr, pos=self.pos2[L:],
                               stream=stream)

    def stage2(self, prefix, stream=None):
        i0 = self.n1 + self.nt
        for i in range(i0, i0 + self.n2):
            self._step(self.z2, self.v2, self.pos2, self.S2, self.t[i + 1] - self.t[i], prefix, pos_scale=0.5,
                       stream=stream)

    def transition23(self, stream=None):
        K, Mp = self.K, self.Mp
        t_s = self.t[self.n1 + self.nt + self.n2]
        B.avits_euler_update(self.z2, self.v2, -t_s, stream)          # clean estimate
        B.avits_scatter_mixed(self.z2, self.idx[:K] if K else None, self.H_lr, self.W_lr, 0,
                              self.z3 if K else None, self.state if K < Mp else None, stream)
        # The kept tokens expanded by 2x nearest upsampling around the expanded rows.
        B.avits_gather_upsample(self.state, self.z3, None, self.children[:4 * K], self.H_lr, self.W_lr,
                                self.g_rows[:4 * K], self.g_pos[:4 * K], self.z3, B.UP_NEAREST, stream)
        B.avits_noise_reinject(self.z3, t_s, self.seed, 2 * self.H_lr, 2 * self.W_lr, stream=stream)

    def stage3(self, prefix, stream=None):
        i0 = self.n1 + self.nt + self.n2
        for i in range(i0, i0 + self.n3):
            self._step(self.z3, self.v3, self.pos3, self.S3, self.t[i + 1] - self.t[i], prefix, stream=stream)

    def run(self, prefix, stream=None):
        """The whole sampler; returns z3 [N, C], the final latent in raster order."""
        self.stage1(prefix, stream)
        self.transition12(stream)
        self.stage2(prefix, stream)
        self.transition23(stream)
        self.stage3(prefix, stream)
        return self.z3
