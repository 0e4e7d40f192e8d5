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
        self.lse = torch.empty(s.H, s.S, dtype=f32, device=device) if keep_lse else None
        d = s.D // s.H
        self.ws_score = torch.empty(max(B.avits_score_workspace_bytes(s.N, s.H), 1), dtype=torch.uint8, device=device)
        self.ws_select = torch.empty(max(B.avits_select_workspace_bytes(s.N), 1), dtype=torch.uint8, device=device)
        code = B.BF16 if dtype == torch.bfloat16 else B.F32
        self.ws_block = torch.empty(
            max(B.avits_block_workspace_bytes(weights.kind, s.S, s.H, d, s.mlp_hidden, code), 1),
            dtype=torch.uint8, device=device)

    def score(self, latent_q, text_k, row_lse, feat_t, feat_prev, stream=None):
        B.avits_score(latent_q, text_k, row_lse, feat_t, feat_prev, self.alpha, self.eps, self.scores,
                      self.a_raw, self.v_raw, self.ws_score, stream)

    def select(self, stream=None):
        if self.shape.k:
            B.avits_select(self.scores, self.shape.k, self.idx, self.ws_select, stream)

    def gather(self, lowres, highres_prev, prefix, stream=None):
        s = self.shape
        canvas = highres_prev if self.canvas is None else self.canvas
        B.avits_gather_upsample(lowres, highres_prev, prefix, self.idx, s.H_lr, s.W_lr, self.compact,
                                self.pos[s.L + s.R:], canvas, self.mode, stream)

    def block(self, stream=None):
        s = self.shape
        B.avits_block_forward(self.compact, self.x_out, self.pos, s.L, s.R + s.k, self.weights, s.H,
                              self.lse, self.ws_block, stream)

    def scatter(self, highres_prev, stream=None):
        s = self.shape
        canvas = highres_prev if self.canvas is None else self.canvas
        if s.k:
            B.avits_scatter(self.x_out, self.idx, s.L + s.R, canvas, stream)

    def run(self, latent_q, text_k, row_lse, feat_t, feat_prev, lowres, highres_prev, prefix, stream=None):
        self.score(latent_q, text_k, row_lse, feat_t, feat_prev, stream)
        self.select(stream)
        self.gather(lowres, highres_prev, prefix, stream)
        self.block(stream)
        self.scatter(highres_prev, stream)
