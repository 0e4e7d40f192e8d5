"""Benchmark of one selective-upsampling step on one MI355X.

A step is one pass of the whole hot path over one synthetic input batch:
score (spatial + temporal + fuse) -> top-K select -> gather + 2x upsample ->
double-stream MMDiT block on the compacted sequence -> scatter, at the
FLUX-shaped 1024^2 workload (hidden 3072, 24x128 heads, 512 text tokens,
64x64 high-res latent, keep ratio 0.3 -> k = 1229, S = 1741), bf16 storage
with fp32 accumulation.  All inputs are resident in HBM before timing; the
timed steps rotate over four copies of the step's inputs (at different
addresses), so no step finds its inputs in the 256 MB last-level cache from
the step before.  The joint log-sum-exp the scorer consumes is produced
before timing (it is the previous step's attention by-product); a second
figure times the step with it included.

Further legs in the same run: the step at the Qwen-Image-Edit shape and at
FLUX 2048^2 over keep ratios 0.1 / 0.3 / 0.5 / 1.0, the FLUX stack (19
double + 38 single blocks, 4 denoising steps including the probe and the
joint log-sum-exp), the select sweep, fused scoring, the mixed-resolution
Stage 2 and the batched legs.

Prints one JSON line.  Usage: python bench.py [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "ms per selective DiT block step + attn MFMA util + score/select HBM GB/s"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


# HBM traffic of the dominant kernel, measured with the FETCH_SIZE and
# WRITE_SIZE counters (each in its own profiler pass) and scaled by what the
# same counters read for a plain copy of known size.  It is reported only while
# the GEMM sources hash to what they were when the counters were taken.
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "gemm_bf16_flux1024_hbm_traffic.md")
GEMM_SOURCES = ("gemm.hip", "kernels.h", "common.h")


def gemm_sources_sha256() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_17995_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic() -> dict | None:
    """{'bytes_per_launch': ..., ...} from the committed counter summary, or
    None when there is none or the GEMM sources changed since it was taken."""
    try:
        with open(TRAFFIC_PROFILE) as fh:
            for line in fh:
                if line.startswith("traffic_json: "):
                    rec = json.loads(line[len("traffic_json: "):])
                    return rec if rec.get("sources_sha256") == gemm_sources_sha256() else None
    except OSError:
        return None
    return None


# HBM traffic of the streaming stages (score, select, gather/upsample,
# scatter), from the same two counter passes over the step's kernels; reported
# only while the sources of those kernels hash to what they were then.
STAGE_TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "stages_flux1024_hbm_traffic.md")
STAGE_SOURCES = ("score.hip", "select.hip", "select_block.h", "relayout.hip", "common.h")

# Launch families (the library's per-launch timing names) of each streaming stage.
STAGE_FAMILIES = {"score": ("score_spatial", "score_combine", "score_finalize"), "select": ("select",),
                  "gather_upsample": ("gather_upsample",), "scatter": ("scatter",)}

LEGS = ("fused_scoring", "block_mass", "select_sweep", "mixed_stage2", "batched", "workloads", "stack",
        "three_stage")


def sources_sha256(files) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2608_17995_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_stage_traffic() -> dict | None:
    """Per-stage counter-measured HBM bytes of the FLUX 1024^2 step, or None
    when there is no summary or its kernels' sources changed since."""
    try:
        with open(STAGE_TRAFFIC_PROFILE) as fh:
            for line in fh:
                if line.startswith("traffic_json: "):
                    rec = json.loads(line[len("traffic_json: "):])
                    return rec if rec.get("sources_sha256") == sources_sha256(STAGE_SOURCES) else None
    except OSError:
        return None
    return None


# ---------------------------------------------------------------------------
# Algorithmic work (what the step must read, write and compute).

def block_flops(S: int, D: int, F: int | None = None) -> dict:
    """FLOPs of one double-stream block on S rows (MLP hidden F, default 4D)."""
    F = 4 * D if F is None else F
    gemm = 2 * S * D * (3 * D + D + F + F)       # QKV, O, MLP in, MLP out
    attn = 4 * S * S * D                          # Q K^T and P V, non-causal
    return {"gemm": gemm, "attention": attn, "total": gemm + attn}


def dense_model_flops(tokens: int, D: int = 3072, blocks: int = 57) -> float:
    """24 D^2 S + 4 S^2 D per block (F = 4D), summed over the blocks."""
    return blocks * (24 * D * D * tokens + 4 * tokens * tokens * D)


def gemm_min_bytes(S: int, D: int, F: int, e: int = 2) -> int:
    """Compulsory HBM bytes of the four GEMM launches of one double-stream
    block (both streams): each operand read once, each output written once.
    QKV: x_mod, W_qkv -> qkv; O: attn, W_o, residual -> x; MLP in: x_mod, W_1
    -> h; MLP out: h, W_2, residual -> x.  Biases and gates are negligible."""
    w = 2 * (3 * D * D + D * D + D * F + F * D)           # two streams' weights
    act = S * D + S * 3 * D                               # QKV
    act += S * D + 2 * S * D                              # O (in, resid, out)
    act += S * D + S * F                                  # MLP in
    act += S * F + 2 * S * D                              # MLP out (in, resid, out)
    return e * (w + act)


def stage_bytes(w, e: int = 2) -> dict:
    """Algorithmic HBM bytes per stage (canvas updated in place)."""
    N, D, Df, L, R, k, H = w.N, w.D, w.Df, w.L, w.R, w.k, w.H
    S = L + R + k
    score = N * D * e + L * D * e + 4 * H * N + 2 * N * Df * e + 12 * N
    select = 4 * N + 4 * k
    from paper_2608_17995_amd.step import SelectiveStep
    if N <= SelectiveStep.FUSED_MAX_N:      # the selection runs inside the scoring call (avits_score_select)
        score, select = score + select, 0
    gather = ((L + R) * D * e + k * D * e + w.N_lr * D * e + 4 * k          # reads
              + S * D * e + (N - k) * D * e + 12 * k)                       # writes
    if e == 2 and D % 8 == 0 and D <= 4096:
        # bf16: the gather also writes the block's first stage (the modulated
        # layer norm of every compact row; avits_gather_upsample_ln).
        gather += S * D * e
    scatter = 0         # the scatter rides on the block's last projection (the block stage's bytes)
    return {"score": score, "select": select, "gather_upsample": gather, "scatter": scatter}


# ---------------------------------------------------------------------------

def _cpu_baseline(w, host, row_lse, wt, wi):
    """Time the oracle (fp64 NumPy, untuned) on one full step of the same workload."""
    import numpy as np
    import oracle
    from synth import generator as G
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    t0 = time.perf_counter()
    s, _, _ = oracle.score(host["latent_q"], host["text_k"], row_lse, host["feat_t"], host["feat_prev"], w.alpha)
    idx = oracle.select_topk(s, w.k)
    compact, pos, canvas = oracle.gather_upsample(host["lowres"], host["highres_prev"],
                                                  np.concatenate([host["text"], host["ref"]]), idx, w.H_lr, w.W_lr)
    pos_all = np.concatenate([G.prefix_positions(w), pos])
    out, _ = oracle.double_block(compact, pos_all, w.L, wt, wi, w.H)
    oracle.scatter(out, idx, w.LR, canvas)
    dt = time.perf_counter() - t0
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [threads])
    except Exception:  # pragma: no cover
        pass
    return {"value": round(dt * 1e3, 1), "unit": "ms", "cores": int(threads), "kind": "oracle",
            "sample": f"one full step (score, select, gather/upsample, double block, scatter) of {w.name} "
                      f"in fp64 NumPy on the host; {os.cpu_count()} CPUs visible",
            "cpu_model": _cpu_model(), "cpus_visible": os.cpu_count(),
            "cpus_usable": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None,
            "blas": _blas_info()}


def _cpu_model() -> str | None:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def _blas_info() -> list:
    try:
        from threadpoolctl import threadpool_info
        return [{"api": i.get("internal_api"), "version": i.get("version"), "threads": i.get("num_threads"),
                 "library": os.path.basename(i.get("filepath", ""))} for i in threadpool_info()]
    except Exception:  # pragma: no cover
        return []


def _fused_scoring(avits, torch, w, q, k_all, kt, feat_t, feat_prev, lse, reps: int = 10) -> dict:
    """The scoring stage with the text mass taken inside the joint-softmax
    pass (avits_joint_attention_stats + avits_score_from_mass) beside the
    form the step uses (joint LSE, then the query/key scorer).  Both pairs run
    on the step's inputs; times are per call, from the library's events."""
    N, H = w.N, w.H
    mass = torch.empty(H, N, device="cuda")
    snaps = [feat_prev, feat_t]
    s1, s2 = torch.empty(N, device="cuda"), torch.empty(N, device="cuda")
    ws = torch.empty(avits.avits_score_workspace_bytes(N, H), dtype=torch.uint8, device="cuda")

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3

    out = {
        "stats_pass_us": timed(lambda: avits.avits_joint_attention_stats(q, k_all, w.L, mass, lse=lse)),
        "score_from_mass_us": timed(lambda: avits.avits_score_from_mass(mass, 1, snaps, w.alpha, w.eps_minmax, s1,
                                                                        workspace=ws)),
        "joint_lse_us": timed(lambda: avits.avits_joint_lse(q, k_all, lse)),
        "score_us": timed(lambda: avits.avits_score(q, kt, lse, feat_t, feat_prev, w.alpha, w.eps_minmax, s2,
                                                    workspace=ws)),
    }
    out = {k: round(v, 2) for k, v in out.items()}
    out["max_abs_score_diff"] = float((s1 - s2).abs().max().item())
    return out


def _select_sweep(avits, torch, reps: int = 10) -> list:
    """Top-k selection beyond the step's N: k = 0.3 N of N scores drawn as
    u^(1/4) (u uniform; the top exponent bits coincide, as for min-max
    normalised scores).  Above 16384 scores the selection makes six streaming
    passes over them (four digit histograms, count, emit); `hbm_gbs` counts
    those reads plus the 4k-byte index write."""
    out = []
    for lg in (14, 20, 22, 24, 26):
        N = 1 << lg
        k = int(0.3 * N + 0.5)
        g = torch.Generator(device="cuda")
        g.manual_seed(lg)
        s = torch.rand(N, device="cuda", generator=g) ** 0.25
        idx = torch.empty(k, dtype=torch.int32, device="cuda")
        ws = torch.empty(max(avits.avits_select_workspace_bytes(N), 1), dtype=torch.uint8, device="cuda")
        for _ in range(2):
            avits.avits_select(s, k, idx, workspace=ws)
        torch.cuda.synchronize()
        avits.avits_timing_reset()
        avits.avits_timing_enable(True)
        for _ in range(reps):
            avits.avits_select(s, k, idx, workspace=ws)
        torch.cuda.synchronize()
        avits.avits_timing_enable(False)
        ms, n = avits.avits_timing_read("select")
        t = ms / n / 1e3
        passes = 1 if N <= 16384 else 6
        gbs = (passes * 4 * N + 4 * k) / t / 1e9
        out.append({"N": N, "k": k, "us": round(t * 1e6, 1), "passes": passes, "hbm_gbs": round(gbs, 1),
                    "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)})
        del s, idx, ws
    return out


def _mixed_stage2(avits, torch, w, text, bw, reps: int = 10) -> dict:
    """The paper's own Stage 2 at the same shape (Section 3.2): selection over
    the M' low-res tokens, K = floor(rho M') expanded 2x2 and the rest kept at
    low resolution in one mixed sequence; one double block on it.  Times the
    transition (probe, text mass, score, select, gather_mixed), one step (the
    block, half-unit RoPE) and the re-layout back (scatter_mixed)."""
    import numpy as np
    from paper_2608_17995_amd.step import MixedStage2
    from synth import configs as C
    from synth import generator as G
    Mp = w.N_lr
    K = C.mixed_keep_count(w.rho, Mp)
    feat_t, feat_prev, _ = G.feature_pair(w.seed + 17, Mp, w.D, w.dtype)

    def cuda(a):
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16).cuda()

    z, z_prev = cuda(feat_t), cuda(feat_prev)
    m = MixedStage2(w.H_lr, w.W_lr, w.L, w.R, K, w.D, w.H, w.mlp_ratio * w.D, [bw], [],
                    G.prefix_positions(w), torch.bfloat16, alpha=w.alpha, eps=w.eps_minmax)
    canvas = torch.empty(w.N, w.D, dtype=torch.bfloat16, device="cuda")
    state = torch.empty_like(z)

    def timed(fn):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        e[0].record()
        for _ in range(reps):
            fn()
        e[1].record()
        torch.cuda.synchronize()
        return e[0].elapsed_time(e[1]) / reps

    t_trans = timed(lambda: m.transition(z, [z_prev, z], text))
    x0 = m.x.clone()

    def one_step():
        m.x.copy_(x0)      # restart from the transition's sequence (copy timed separately below)
        m.step()

    t_copy = timed(lambda: m.x.copy_(x0))
    t_step = timed(one_step) - t_copy
    t_leave = timed(lambda: m.leave(canvas, state))
    avits.avits_timing_reset()
    avits.avits_timing_enable(True)
    for _ in range(reps):
        m.transition(z, [z_prev, z], text)
        m.leave(canvas, state)
    torch.cuda.synchronize()
    avits.avits_timing_enable(False)
    g_ms, g_n = avits.avits_timing_read("gather_mixed")
    s_ms, s_n = avits.avits_timing_read("scatter_mixed")
    e, D, S = 2, w.D, m.S
    gather_bytes = (w.LR + Mp) * D * e + S * D * e + (S - w.LR) * 12 + 16 * K + 4 * K
    scatter_bytes = 2 * (S - w.LR) * D * e + 4 * K
    fl = block_flops(S, D, w.mlp_ratio * D)
    g_us, s_us = 1e3 * g_ms / max(g_n, 1), 1e3 * s_ms / max(s_n, 1)
    return {
        "lowres_tokens": Mp, "K": K, "seq_len": S,
        "seq_len_compacted_path": w.S,
        "transition_ms": round(t_trans, 4), "block_step_ms": round(t_step, 4), "leave_ms": round(t_leave, 4),
        "block_tflops": round(fl["total"] / (t_step / 1e3) / 1e12, 1),
        "gather_mixed_us": round(g_us, 2), "scatter_mixed_us": round(s_us, 2),
        "gather_mixed_gbs": round(gather_bytes / (g_us / 1e6) / 1e9, 1) if g_us > 0 else None,
        "scatter_mixed_gbs": round(scatter_bytes / (s_us / 1e6) / 1e9, 1) if s_us > 0 else None,
        "gather_mixed_bytes": gather_bytes, "scatter_mixed_bytes": scatter_bytes,
    }


def _block_mass(avits, torch, w, bw, x, pos, reps: int = 10) -> dict:
    """The block with the text attention mass taken inside its own joint
    attention (avits_block_forward_ex, Section 3.3.1) against the plain
    block, on the step's compacted rows: the cost of the spatial signal when
    it comes from the backbone's attention pass itself."""
    S = x.shape[0]
    out = torch.empty_like(x)
    mass = torch.zeros(w.H, S, device="cuda")
    ws = torch.empty(avits.avits_block_workspace_bytes(avits.BLOCK_DOUBLE, S, w.H, w.d, w.mlp_ratio * w.D,
                                                       avits.BF16), dtype=torch.uint8, device="cuda")

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        e[0].record()
        for _ in range(reps):
            fn()
        e[1].record()
        torch.cuda.synchronize()
        return e[0].elapsed_time(e[1]) / reps

    def plain():
        avits.avits_block_forward(x, out, pos, w.L, S - w.L, bw, w.H, workspace=ws)

    def with_mass():
        avits.avits_block_forward_ex(x, out, pos, w.L, S - w.L, bw, w.H, mass_out=mass, mass_accumulate=True,
                                     workspace=ws)

    t_p, t_m = float("inf"), float("inf")
    for _ in range(3):
        t_p = min(t_p, timed(plain))
        t_m = min(t_m, timed(with_mass))
    return {"plain_ms": round(t_p, 4), "with_mass_ms": round(t_m, 4), "overhead": round(t_m / t_p - 1.0, 4)}


def _batched_block(avits, torch, w, bw, x, reps: int = 10) -> dict:
    """Two images of the workload (a CFG pair: same weights, own text and own
    selection) through one double block in one pass, rows packed by stream
    and attention block-diagonal, against two single-image passes."""
    L, I = w.L, w.R + w.k
    S = 2 * (L + I)
    xb = torch.cat([x[:L], x[:L], x[L:], x[L:]]).contiguous()
    pos = torch.zeros(S, 3, dtype=torch.int32, device="cuda")
    pos1 = torch.zeros(L + I, 3, dtype=torch.int32, device="cuda")
    out = torch.empty_like(xb)
    out1 = torch.empty_like(x)
    ws = torch.empty(avits.avits_block_workspace_bytes(avits.BLOCK_DOUBLE, S, w.H, w.d, w.mlp_ratio * w.D,
                                                       avits.BF16), dtype=torch.uint8, device="cuda")

    def timed(fn):
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        e[0].record()
        for _ in range(reps):
            fn()
        e[1].record()
        torch.cuda.synchronize()
        return e[0].elapsed_time(e[1]) / reps

    def batched():
        avits.avits_block_forward_batched(xb, out, pos, [0, L, 2 * L], [0, I, 2 * I], bw, w.H, workspace=ws)

    def two():
        for _ in range(2):
            avits.avits_block_forward(x, out1, pos1, L, I, bw, w.H, workspace=ws)

    # The pair at two timesteps: each image with its own modulation vectors
    # ([2, 6, D] per stream, avits_block_forward_batched_ex).
    per = {}
    for part in ("txt", "img"):
        per[part] = dict(bw.tensors[part])
        m = per[part]["mod"]
        per[part]["mod"] = torch.cat([m, (m.float() * 1.01).to(m.dtype)]).contiguous()
    bw2 = avits.BlockWeights(avits.BLOCK_DOUBLE, txt=per["txt"], img=per["img"])

    def batched_mod():
        avits.avits_block_forward_batched_ex(xb, out, pos, [0, L, 2 * L], [0, I, 2 * I], bw2, w.H, 6 * w.D,
                                             workspace=ws)

    # Alternate the forms (each after its own warm-up) and keep the best of
    # three, so clock drift between the measurements does not decide the ratio.
    t_b, t_2, t_m = float("inf"), float("inf"), float("inf")
    for _ in range(3):
        t_2 = min(t_2, timed(two))
        t_b = min(t_b, timed(batched))
        t_m = min(t_m, timed(batched_mod))
    return {"images": 2, "rows": S, "batched_ms": round(t_b, 4), "two_single_ms": round(t_2, 4),
            "speedup": round(t_2 / t_b, 3), "per_image_modulation_ms": round(t_m, 4)}


def _batched_step(avits, torch, w, bw, shape, prefix_pos, q, kt, lse, feat, fp, low, text, ref, single_step,
                  reps: int = 10) -> dict:
    """A CFG pair through the whole step at once (BatchedStep on inputs stacked
    over the pair: one scoring launch, one selection, one gather, one block,
    one scatter) against two single-image steps.  The stacked inputs are
    resident before timing."""
    from paper_2608_17995_amd.step import BatchedStep
    bstep = BatchedStep(shape, [w.k, w.k], bw, prefix_pos, torch.bfloat16, alpha=w.alpha)
    q2, kt2, lse2, fp2, low2, text2 = (torch.stack([t, t]) for t in (q, kt, lse, fp, low, text))
    feat2, canv2 = torch.stack([feat, feat]), torch.stack([feat, feat])
    ref2 = torch.stack([ref, ref]) if w.R else None

    def batched():
        # feat_t of the pair: the canvases' contents before this step (equal
        # for both images of the pair here).
        bstep.run(q2, kt2, lse2, feat2, fp2, low2, canv2, text2, ref2)

    canvas1 = feat.clone()

    def two():
        for _ in range(2):
            single_step.run(q, kt, lse, canvas1, fp, low, canvas1, torch.cat([text, ref]) if w.R else text)

    def timed(fn):
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        e[0].record()
        for _ in range(reps):
            fn()
        e[1].record()
        torch.cuda.synchronize()
        return e[0].elapsed_time(e[1]) / reps

    t_b, t_2 = float("inf"), float("inf")
    for _ in range(3):
        t_2 = min(t_2, timed(two))
        t_b = min(t_b, timed(batched))
    return {"images": 2, "batched_ms": round(t_b, 4), "two_single_ms": round(t_2, 4), "speedup": round(t_2 / t_b, 3)}


def _gpu_block_weights(avits, torch, w, gen, kind):
    """Random-init bf16 weights of one block of the workload's architecture,
    drawn on the GPU (timing legs only: N(0, 0.02) projections, modulation
    shifts / scales N(0, 0.02), gates and RMSNorm gains 1 + N(0, 0.02))."""
    D, F, d = w.D, w.mlp_ratio * w.D, w.d

    def n(*shape, std=0.02, mean=0.0):
        return (torch.randn(*shape, generator=gen, device="cuda") * std + mean).to(torch.bfloat16)

    def mod(rows):
        m = torch.randn(rows, D, generator=gen, device="cuda") * 0.02
        m[2::3] += 1.0
        return m.to(torch.bfloat16)

    if kind == avits.BLOCK_SINGLE:
        return avits.BlockWeights(avits.BLOCK_SINGLE, single={
            "mod": mod(3), "w_in": n(3 * D + F, D), "b_in": n(3 * D + F), "g_q": n(d, mean=1.0),
            "g_k": n(d, mean=1.0), "w_out": n(D, D + F), "b_out": n(D)})

    def stream():
        return {"mod": mod(6), "w_qkv": n(3 * D, D), "b_qkv": n(3 * D), "g_q": n(d, mean=1.0), "g_k": n(d, mean=1.0),
                "w_o": n(D, D), "b_o": n(D), "w_mlp1": n(F, D), "b_mlp1": n(F), "w_mlp2": n(D, F), "b_mlp2": n(D)}
    return avits.BlockWeights(avits.BLOCK_DOUBLE, txt=stream(), img=stream())


def _timed_steps(torch, run, n_sets, steps, warmup, stages=None):
    """ms per step of run(i) over `steps` steps (input set i % n_sets), after
    `warmup` untimed steps; with `stages`, also ms per stage from events that
    run(i, events) records between its stages."""
    for i in range(warmup):
        run(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        run(i)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    if not stages:
        return ms, None
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)] for _ in range(steps)]
    for i in range(steps):
        run(i, evs[i])
    torch.cuda.synchronize()
    per = {st: sum(e[j].elapsed_time(e[j + 1]) for e in evs) / steps for j, st in enumerate(stages)}
    return ms, per


STEP_STAGES = ("score", "select", "gather_upsample", "block", "scatter")


def _input_sets(torch, base: dict, budget_bytes: float = 512e6, max_sets: int = 4) -> list:
    """The step's inputs plus copies at other addresses, enough that the
    inputs of one step are gone from the 256 MB last-level cache when that
    set comes round again (at most max_sets sets)."""
    import math
    nbytes = sum(t.numel() * t.element_size() for t in base.values())
    n = max(1, min(max_sets, math.ceil(budget_bytes / max(nbytes, 1))))
    return [base] + [{k: v.clone() for k, v in base.items()} for _ in range(n - 1)]


def _workload_legs(avits, torch, steps: int, warmup: int) -> list:
    """The selective step at the Qwen-Image-Edit shape and at FLUX 2048^2 over
    its keep ratios: the seeded scoring and layout inputs of the parity
    tests, random-init weights drawn on the GPU, the joint log-sum-exp made in
    set-up (and timed on its own).  One record per shape / keep ratio."""
    import numpy as np
    from paper_2608_17995_amd.step import SelectiveStep, StepShape
    from synth import configs as C
    from synth import generator as G

    out = []
    for base, rhos in ((C.QWEN_EDIT, (C.QWEN_EDIT.rho,)), (C.FLUX_2048, C.FLUX_2048_RHOS)):
        w0 = base
        si = G.score_inputs(w0)
        lay = G.layout_inputs(w0, si["feat_t"])

        def cuda(a):
            return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16).cuda()

        gen = torch.Generator(device="cuda")
        gen.manual_seed(w0.seed)
        bw = _gpu_block_weights(avits, torch, w0, gen, avits.BLOCK_DOUBLE)
        first = {"q": cuda(si["latent_q"]), "kt": cuda(si["text_k"]), "fp": cuda(si["feat_prev"]),
                 "high": cuda(lay["highres_prev"]), "low": cuda(lay["lowres"]),
                 "prefix": cuda(np.concatenate([lay["text"], lay["ref"]])),
                 "k_all": cuda(np.concatenate([si["text_k"], si["ref_k"], si["latent_k"]])),
                 "lse": torch.empty(w0.H, w0.N, device="cuda")}
        del si, lay
        avits.avits_joint_lse(first["q"], first["k_all"], first["lse"])
        sets = _input_sets(torch, first)
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        e[0].record()
        for _ in range(3):
            avits.avits_joint_lse(first["q"], first["k_all"], first["lse"])
        e[1].record()
        torch.cuda.synchronize()
        lse_ms = e[0].elapsed_time(e[1]) / 3
        prefix_pos = torch.from_numpy(G.prefix_positions(w0)).cuda()
        for rho in rhos:
            w = w0 if rho == w0.rho and base is C.QWEN_EDIT else w0.with_rho(rho)
            shape = StepShape(N=w.N, H_lr=w.H_lr, W_lr=w.W_lr, L=w.L, R=w.R, k=w.k, D=w.D, H=w.H, D_f=w.Df,
                              mlp_hidden=w.mlp_ratio * w.D)
            step = SelectiveStep(shape, bw, prefix_pos, torch.bfloat16, alpha=w.alpha)

            def run(i, ev=None, step=step):
                st = sets[i % len(sets)]
                if ev is not None:
                    ev[0].record()
                step.score(st["q"], st["kt"], st["lse"], st["high"], st["fp"])
                if ev is not None:
                    ev[1].record()
                step.select()
                if ev is not None:
                    ev[2].record()
                step.gather(st["low"], st["high"], st["prefix"])
                if ev is not None:
                    ev[3].record()
                step.block()
                if ev is not None:
                    ev[4].record()
                step.scatter(st["high"])
                if ev is not None:
                    ev[5].record()

            ms, per = _timed_steps(torch, run, len(sets), steps, warmup, STEP_STAGES)
            fl = block_flops(w.S, w.D, w.mlp_ratio * w.D)
            by = stage_bytes(w)
            out.append({
                "workload": w.name, "N": w.N, "L": w.L, "R": w.R, "k": w.k, "seq_len": w.S,
                "ms_per_step": round(ms, 4), "tokens_per_s": round(w.S / (ms / 1e3), 1),
                "canvas_tokens_per_s": round(w.N / (ms / 1e3), 1),
                "ms_per_step_with_joint_lse": round(ms + lse_ms, 4), "joint_lse_ms": round(lse_ms, 4),
                "stages_ms": {k: round(v, 4) for k, v in per.items()},
                "block_tflops": round(fl["total"] / (per["block"] / 1e3) / 1e12, 1),
                "block_mfma_frac": round(fl["total"] / (per["block"] / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                "hbm_gbs": {k: round(by[k] / (per[k] / 1e3) / 1e9, 1)
                            for k in ("score", "select", "gather_upsample", "scatter") if per[k] > 0 and by[k] > 0},
                "input_sets": len(sets)})
            del step
        del sets, first, bw
        torch.cuda.empty_cache()
    return out


def _stack_leg(avits, torch) -> dict:
    """The FLUX stack at the resolution transition (19 double + 38 single
    blocks, 512 text tokens, 32x32 -> 64x64, k = 1229): 4 denoising steps,
    each probe (double block 0's first stage on every image row) -> joint
    log-sum-exp -> score -> select -> gather -> 57 blocks -> scatter.
    Random-init weights drawn on the GPU; seeded features."""
    import numpy as np
    from paper_2608_17995_amd.step import StackStep, StepShape
    from synth import configs as C
    from synth import generator as G

    w = C.FLUX_STACK
    gen = torch.Generator(device="cuda")
    gen.manual_seed(w.seed)
    doubles = [_gpu_block_weights(avits, torch, w, gen, avits.BLOCK_DOUBLE) for _ in range(w.n_double)]
    singles = [_gpu_block_weights(avits, torch, w, gen, avits.BLOCK_SINGLE) for _ in range(w.n_single)]

    def cuda(a):
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16).cuda()

    x0, x_m1, _ = G.feature_pair(w.seed, w.N, w.D, w.dtype)
    lay = G.layout_inputs(w, x0)
    low, text = cuda(lay["lowres"]), cuda(lay["text"])
    shape = StepShape(N=w.N, H_lr=w.H_lr, W_lr=w.W_lr, L=w.L, R=w.R, k=w.k, D=w.D, H=w.H, D_f=w.Df,
                      mlp_hidden=w.mlp_ratio * w.D)
    st = StackStep(shape, doubles, singles, torch.from_numpy(G.prefix_positions(w)).cuda(), torch.bfloat16,
                   alpha=w.alpha)
    xs = [cuda(x_m1), cuda(x0)] + [torch.empty(w.N, w.D, dtype=torch.bfloat16, device="cuda")
                                   for _ in range(w.steps)]
    warm = torch.empty_like(xs[0])
    st.run(xs[1], xs[0], low, text, warm)           # warm-up step (untimed)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(w.steps + 1)]
    t0 = time.perf_counter()
    ev[0].record()
    for s in range(w.steps):
        st.run(xs[s + 1], xs[s], low, text, xs[s + 2])
        ev[s + 1].record()
    torch.cuda.synchronize()
    total = (time.perf_counter() - t0) * 1e3
    per = [ev[s].elapsed_time(ev[s + 1]) for s in range(w.steps)]
    fl_blocks = (w.n_double + w.n_single) * block_flops(w.S, w.D, w.mlp_ratio * w.D)["total"]
    fl_probe = 2 * (w.L + w.N) * w.D * 2 * w.D + 2 * w.N * (w.L + w.N) * w.D   # q/k projection + joint LSE
    mean = sum(per) / len(per)
    return {"workload": w.name, "blocks": w.n_double + w.n_single, "steps": w.steps, "k": w.k, "seq_len": w.S,
            "ms_per_denoise_step": [round(x, 3) for x in per], "ms_per_denoise_step_mean": round(mean, 3),
            "ms_total_4_steps": round(total, 3),
            "tflops": round((fl_blocks + fl_probe) / (mean / 1e3) / 1e12, 1),
            "includes": "probe (double block 0's q/k on all image rows), joint log-sum-exp, score, select, "
                        "gather, 19 double + 38 single blocks, scatter"}


def _three_stage_leg(avits, torch) -> dict:
    """One image through the whole three-stage sampler of Section 3.2 at the
    FLUX 1024^2 shape on the 57-block stack (random-init weights drawn on
    the GPU, 64 latent channels, 512 text tokens): 18 Euler steps split
    6 + 3 (Stage 1 at 32x32, the last 3 collecting snapshots and the text
    mass of every double block) + 4 (Stage 2, K = floor(0.3 * 1024) = 307
    tokens expanded: 2457 rows) + 5 (Stage 3 at 64x64: 4608 rows), with both
    transitions (scores, selection, re-layout, coordinate-bound noise)."""
    from paper_2608_17995_amd.step import ThreeStageSampler
    from synth import configs as C
    from synth import generator as G

    w = C.FLUX_STACK
    n1, nt, n2, n3, Cc = 6, 3, 4, 5, 64
    K = C.mixed_keep_count(w.rho, w.N_lr)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(w.seed + 100)
    doubles = [_gpu_block_weights(avits, torch, w, gen, avits.BLOCK_DOUBLE) for _ in range(w.n_double)]
    singles = [_gpu_block_weights(avits, torch, w, gen, avits.BLOCK_SINGLE) for _ in range(w.n_single)]

    def n(*shape, std=0.02, mean=0.0):
        return (torch.randn(*shape, generator=gen, device="cuda") * std + mean).to(torch.bfloat16)

    sw = {"embed_w": n(w.D, Cc), "embed_b": n(w.D), "final_mod": n(2, w.D), "final_w": n(Cc, w.D), "final_b": n(Cc)}
    text = n(w.L, w.D, std=1.0)
    samp = ThreeStageSampler(w.H_lr, w.W_lr, w.L, Cc, w.D, w.H, w.mlp_ratio * w.D, doubles, singles, sw,
                             torch.from_numpy(G.prefix_positions(w)).cuda(), K, n1, nt, n2, n3, torch.bfloat16,
                             seed=w.seed, alpha=w.alpha)
    samp.run(text)                        # warm-up
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    t0 = time.perf_counter()
    ev[0].record()
    samp.stage1(text)
    ev[1].record()
    samp.transition12()
    ev[2].record()
    samp.stage2(text)
    ev[3].record()
    samp.transition23()
    ev[4].record()
    samp.stage3(text)
    ev[5].record()
    torch.cuda.synchronize()
    total = (time.perf_counter() - t0) * 1e3
    parts = [ev[i].elapsed_time(ev[i + 1]) for i in range(5)]
    blocks = w.n_double + w.n_single
    fl = sum(k * blocks * block_flops(S, w.D)["total"] for k, S in ((n1 + nt, samp.S1), (n2, samp.S2), (n3, samp.S3)))
    return {"workload": w.name, "steps": [n1, nt, n2, n3], "K": K, "rows": [samp.S1, samp.S2, samp.S3],
            "ms_total": round(total, 2), "ms": {"stage1": round(parts[0], 2), "transition12": round(parts[1], 3),
                                                "stage2": round(parts[2], 2), "transition23": round(parts[3], 3),
                                                "stage3": round(parts[4], 2)},
            "tflops_blocks": round(fl / (total / 1e3) / 1e12, 1)}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--legs", default="all",
                    help="legs after the headline step: all, none, or a comma list of " + ", ".join(LEGS))
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain 512 MiB device-to-device copy (a kernel of known traffic, the "
                         "reference for scaling FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args(argv)
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2608_17995_amd as avits
    from paper_2608_17995_amd.step import SelectiveStep, StepShape
    from synth import configs as C
    from synth import generator as G

    torch.cuda.set_device(0)
    avits.load()
    copy_ms = None
    if args.copy_calibration:
        src = torch.empty(256 * 1024 * 1024, dtype=torch.int16, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        copy_ms = e0.elapsed_time(e1)
        del src, dst
    w = C.FLUX_1024
    dt = torch.bfloat16

    def cuda(a):
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dt).cuda()

    t_gen = time.perf_counter()
    si = G.score_inputs(w)
    lay = G.layout_inputs(w, si["feat_t"])
    wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
    t_gen = time.perf_counter() - t_gen

    q, kt, fp = cuda(si["latent_q"]), cuda(si["text_k"]), cuda(si["feat_prev"])
    k_all = cuda(np.concatenate([si["text_k"], si["ref_k"], si["latent_k"]]))
    high = cuda(lay["highres_prev"])       # = feat_t (hidden states); updated in place each step
    low, text = cuda(lay["lowres"]), cuda(np.concatenate([lay["text"], lay["ref"]]))
    bw = avits.BlockWeights(avits.BLOCK_DOUBLE, txt={k: cuda(v) for k, v in wt.items()},
                            img={k: cuda(v) for k, v in wi.items()})
    shape = StepShape(N=w.N, H_lr=w.H_lr, W_lr=w.W_lr, L=w.L, R=w.R, k=w.k, D=w.D, H=w.H, D_f=w.Df,
                      mlp_hidden=w.mlp_ratio * w.D)
    step = SelectiveStep(shape, bw, torch.from_numpy(G.prefix_positions(w)).cuda(), dt, alpha=w.alpha)
    lse = torch.empty(w.H, w.N, device="cuda")
    row_lse_host = None

    # Setup: the joint log-sum-exp over [text; image] keys (timed on its own).
    avits.avits_joint_lse(q, k_all, lse)
    torch.cuda.synchronize()
    row_lse_host = lse.double().cpu().numpy()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    for _ in range(5):
        avits.avits_joint_lse(q, k_all, lse)
    ev[1].record()
    torch.cuda.synchronize()
    joint_lse_ms = ev[0].elapsed_time(ev[1]) / 5

    stages = STEP_STAGES
    # Four copies of the step's inputs at different addresses; step i reads
    # set i % 4 (and updates that set's canvas in place).
    sets = _input_sets(torch, {"q": q, "kt": kt, "fp": fp, "high": high, "low": low, "text": text,
                               "k_all": k_all, "lse": lse}, max_sets=4)
    if len(sets) < 4:
        sets += [{k: v.clone() for k, v in sets[0].items()} for _ in range(4 - len(sets))]

    def run_step(i=0, events=None, with_lse=False):
        st = sets[i % len(sets)]

        def mark(j):
            if events is not None:
                events[j].record()
        if with_lse:
            avits.avits_joint_lse(st["q"], st["k_all"], st["lse"])
        mark(0)
        step.score(st["q"], st["kt"], st["lse"], st["high"], st["fp"])
        mark(1)
        step.select()
        mark(2)
        step.gather(st["low"], st["high"], st["text"])
        mark(3)
        step.block()
        mark(4)
        step.scatter(st["high"])
        mark(5)

    for i in range(args.warmup):
        run_step(i)
    torch.cuda.synchronize()

    # Timed region 1: K steps, nothing but the step's own launches -> value.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        run_step(i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps

    # Timed region 1b: the same steps with the joint log-sum-exp of each
    # step's queries over its [text; image] keys made inside the step.
    t0 = time.perf_counter()
    for i in range(args.steps):
        run_step(i, with_lse=True)
    torch.cuda.synchronize()
    ms_with_lse = (time.perf_counter() - t0) * 1e3 / args.steps

    # Timed region 1c: the distribution of single steps (>= 50, each between
    # two events on the stream, the input sets rotating) -> median, p10, p90.
    n_dist = max(50, args.steps)
    ev_d = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n_dist)]
    torch.cuda.synchronize()
    for i in range(n_dist):
        ev_d[i][0].record()
        run_step(i)
        ev_d[i][1].record()
    torch.cuda.synchronize()
    step_ms = sorted(a.elapsed_time(b) for a, b in ev_d)

    def pct(q):
        return round(step_ms[min(len(step_ms) - 1, int(round(q * (len(step_ms) - 1))))], 4)
    step_dist = {"steps": n_dist, "median_ms": pct(0.5), "p10_ms": pct(0.1), "p90_ms": pct(0.9),
                 "note": "each step between two HIP events on the launch stream"}

    # Timed region 2: the same K steps with stage events on the stream and the
    # library's own HIP events around every internal launch -> per-stage and
    # per-kernel times, the roofline of the dominant kernel.
    step_events = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(args.steps)]
    avits.avits_timing_reset()
    avits.avits_timing_enable(True)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for i in range(args.steps):
        run_step(i, step_events[i])
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    avits.avits_timing_enable(False)
    ms_instrumented = (t3 - t2) * 1e3 / args.steps

    stage_ms = {s: 0.0 for s in stages}
    for evs in step_events:
        for j, s in enumerate(stages):
            stage_ms[s] += evs[j].elapsed_time(evs[j + 1]) / args.steps
    fam = {}
    for f in ("score_spatial", "score_combine", "score_finalize", "select", "gather_upsample", "scatter",
              "ln_mod", "gemm", "splitk_reduce", "qk_rope", "attention"):
        tot, n = avits.avits_timing_read(f)
        fam[f] = {"ms_per_step": round(tot / args.steps, 4), "launches_per_step": n / args.steps,
                  "avg_launch_us": round(1e3 * tot / max(n, 1), 2)}

    S, D, F = w.S, w.D, w.mlp_ratio * w.D
    fl = block_flops(S, D, F)
    by = stage_bytes(w)
    gemm_bytes = gemm_min_bytes(S, D, F)
    gemm_tot_ms, gemm_n = avits.avits_timing_read("gemm")
    gemm_per_launch_flops = fl["gemm"] * args.steps / gemm_n
    gemm_avg_s = gemm_tot_ms / gemm_n / 1e3
    gemm_tflops = gemm_per_launch_flops / gemm_avg_s / 1e12
    red_ms, _ = avits.avits_timing_read("splitk_reduce")
    gemm_red_tflops = fl["gemm"] * args.steps / ((gemm_tot_ms + red_ms) / 1e3) / 1e12
    traffic = measured_traffic()
    attn_ms, attn_n = avits.avits_timing_read("attention")
    attn_tflops = fl["attention"] / (attn_ms / attn_n / 1e3) / 1e12   # one launch per step

    def gbs(nbytes, ms):
        return round(nbytes / (ms / 1e3) / 1e9, 1) if ms > 0 and nbytes > 0 else None

    result = {
        "metric": METRIC,
        "value": round(ms_per_step, 4),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "ms_per_step_instrumented": round(ms_instrumented, 4),
        "ms_per_step_with_joint_lse": round(ms_with_lse, 4),
        "input_sets": len(sets),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "hidden": D, "heads": w.H, "head_dim": w.d, "text_tokens": w.L,
                   "lowres_grid": [w.H_lr, w.W_lr], "highres_grid": [w.H_hr, w.W_hr], "keep_ratio": w.rho,
                   "k": w.k, "seq_len": S, "alpha": w.alpha, "upsample": "nearest"},
        "roofline": {
            "kernel": "gemm_bf16_pp_kernel",
            "bound": "mfma",
            "achieved": round(gemm_tflops, 1),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(gemm_tflops / PEAK_BF16_TFLOPS, 4),
            "traffic": None if traffic is None else traffic["bytes_per_launch"],
            "traffic_unit": "bytes per launch (HBM, counter-measured)",
            "algorithmic_bytes_per_launch": int(gemm_bytes * args.steps / gemm_n),
            "flops_per_launch": int(gemm_per_launch_flops),
            "avg_launch_us": round(gemm_avg_s * 1e6, 2),
            # The projections with their split-K / split-tail reduce kernels
            # (one of which also does the second modulated layer norm).
            "achieved_with_reduces": round(gemm_red_tflops, 1),
        },
        "stages_ms": {s: round(v, 4) for s, v in stage_ms.items()},
        "launch_families": fam,
        "attention": {"tflops": round(attn_tflops, 1), "mfma_frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
                      "flops": fl["attention"]},
        "block": {"ms": round(stage_ms["block"], 4), "flops": fl["total"],
                  "tflops": round(fl["total"] / (stage_ms["block"] / 1e3) / 1e12, 1),
                  "mfma_frac": round(fl["total"] / (stage_ms["block"] / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 4)},
        "hbm_gbs": {s: gbs(by[s], stage_ms[s]) for s in ("score", "select", "gather_upsample", "scatter")},
        "hbm_frac": {s: (round(gbs(by[s], stage_ms[s]) / PEAK_HBM_GBS, 4) if gbs(by[s], stage_ms[s]) else None)
                     for s in ("score", "select", "gather_upsample", "scatter")},
        # The same bytes over the stage's kernels alone: the sum of their
        # per-launch event times (no stage-boundary events or launch gaps).
        "hbm_gbs_kernels": {s: gbs(by[s], sum(fam[f]["avg_launch_us"] * fam[f]["launches_per_step"]
                                              for f in fs) / 1e3)
                            for s, fs in STAGE_FAMILIES.items()},
        "select_fused_into_score": w.N <= SelectiveStep.FUSED_MAX_N,
        "scatter_fused_into_block": True,
        "ln1_fused_into_gather": step.ln_vectors is not None,
        "stage_traffic": measured_stage_traffic(),
        "algorithmic_bytes": by,
        "step_ms_distribution": step_dist,
        "tokens_per_s": round(S / (ms_per_step / 1e3), 1),
        "tokens_per_s_block": round(S / (stage_ms["block"] / 1e3), 1),
        "canvas_tokens_per_s": round(w.N / (ms_per_step / 1e3), 1),
        "joint_lse_ms_untimed_setup": round(joint_lse_ms, 4),
        "input_generation_s": round(t_gen, 1),
        "copy_calibration_ms": None if copy_ms is None else round(copy_ms, 4),
    }
    legs = set(LEGS) if args.legs == "all" else set() if args.legs == "none" else set(args.legs.split(","))
    if "fused_scoring" in legs:
        result["fused_scoring"] = _fused_scoring(avits, torch, w, q, k_all, kt, high, fp, lse)
    if "block_mass" in legs:
        result["block_mass"] = _block_mass(avits, torch, w, bw, step.compact, step.pos)
    if "select_sweep" in legs:
        result["select_sweep"] = _select_sweep(avits, torch)
    if "mixed_stage2" in legs:
        result["mixed_stage2"] = _mixed_stage2(avits, torch, w, text, bw)
    if "batched" in legs:
        result["batched_block"] = _batched_block(avits, torch, w, bw, step.compact)
        result["batched_step"] = _batched_step(avits, torch, w, bw, shape,
                                               torch.from_numpy(G.prefix_positions(w)).cuda(), q, kt, lse, high, fp,
                                               low, cuda(lay["text"]), cuda(lay["ref"]), step)
    del sets
    if "workloads" in legs:
        result["workloads"] = _workload_legs(avits, torch, max(5, args.steps // 2), 2)
    if "stack" in legs:
        result["stack"] = _stack_leg(avits, torch)
    if "three_stage" in legs:
        result["three_stage"] = _three_stage_leg(avits, torch)
    if not args.no_cpu_baseline:
        host = dict(si)
        host.update(lay)
        result["cpu_baseline"] = _cpu_baseline(w, host, row_lse_host, wt, wi)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
