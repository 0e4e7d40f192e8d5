"""Full-size parity: the selective step at the tiny fp32, FLUX 1024^2, FLUX
2048^2 (keep ratios 0.1 / 0.3 / 0.5 / 1.0) and Qwen-Image-Edit shapes, run
stage by stage through the same launch sequence the benchmark times.

Every stage's oracle runs on exactly the GPU's inputs of that stage:
indices, gathered rows, positions and the scattered canvas bit-exact; scores
and block outputs within the parity bar.  The joint log-sum-exp and the text
attention mass are compared on every row at every shape (the oracle runs one
head per thread).  The block is compared on every row where the oracle
finishes in seconds (tiny, FLUX 1024^2, Qwen-Image-Edit); at the 2048^2
shapes on rows chosen so that every 128-row block of the sequence (every
attention unit and, two by two, every 256-row GEMM tile) holds one, plus the
text head and tail and the ragged last rows.  The oracle computes those rows
exactly, with keys and values over the whole sequence.

The end-to-end selection (the oracle's own LSE, scores and top-k against the
GPU's) runs at every shape, and every shape's step is re-run on the same
buffers to check that it is deterministic bit for bit.
"""
import concurrent.futures as cf

import numpy as np
import pytest
import torch

import oracle
from paper_2608_17995_amd.step import SelectiveStep, StepShape
from synth import configs as C
from synth import generator as G

from _gpu import assert_close, dev, double_weights_dev, host, rel_l2

pytestmark = [pytest.mark.gpu, pytest.mark.slow, pytest.mark.timeout(900)]

CASES = [C.TINY_F32, C.FLUX_1024] + [C.FLUX_2048.with_rho(r) for r in C.FLUX_2048_RHOS] + [C.QWEN_EDIT]
IDS = [w.name for w in CASES]

# Row count up to which the oracle evaluates the whole block (seconds on the host).
FULL_BLOCK_ROWS = 6000

# Per-head oracle results, shared by the four keep ratios of one shape (the
# scoring inputs do not depend on the keep ratio).
_HEAD_CACHE: dict = {}


def _per_head(fn, q, k_all, *extra):
    """[H, N] oracle result of fn(q_h, k_h, *extra) for every head, one head
    per thread (NumPy releases the interpreter lock in BLAS and ufuncs)."""
    from threadpoolctl import threadpool_limits
    H = q.shape[1]
    with threadpool_limits(1), cf.ThreadPoolExecutor(16) as ex:
        parts = list(ex.map(lambda h: fn(q[:, h:h + 1], k_all[:, h:h + 1], *extra), range(H)))
    return np.concatenate(parts, axis=0)


def _oracle_lse_mass(w, si, k_all):
    key = (w.seed, w.N, w.L, w.R)
    if key not in _HEAD_CACHE:
        print(f"[oracle] joint LSE and text mass over all {w.N} rows", flush=True)
        lse = _per_head(oracle.joint_lse, si["latent_q"], k_all)
        mass = _per_head(oracle.text_attention_mass, si["latent_q"], k_all, w.L)
        _HEAD_CACHE[key] = (lse, mass)
    return _HEAD_CACHE[key]


@pytest.fixture(scope="module", params=CASES, ids=IDS)
def run(gpu, request):
    w = request.param
    print(f"\n[workload] {w.name}: N={w.N} k={w.k} S={w.S} L={w.L} R={w.R}", flush=True)
    si = G.score_inputs(w)
    lay = G.layout_inputs(w, si["feat_t"])
    wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
    k_all = np.concatenate([si["text_k"], si["ref_k"], si["latent_k"]])
    t = {n: dev(si[n], w.dtype) for n in ("latent_q", "text_k", "feat_prev")}
    high = dev(lay["highres_prev"], w.dtype)
    low = dev(lay["lowres"], w.dtype)
    prefix_np = np.concatenate([lay["text"], lay["ref"]])
    prefix = dev(prefix_np, w.dtype)
    bw = gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(wt, w.dtype), img=double_weights_dev(wi, w.dtype))
    shape = StepShape(N=w.N, H_lr=w.H_lr, W_lr=w.W_lr, L=w.L, R=w.R, k=w.k, D=w.D, H=w.H, D_f=w.Df,
                      mlp_hidden=w.mlp_ratio * w.D)
    canvas = torch.empty_like(high)
    step = SelectiveStep(shape, bw, dev(G.prefix_positions(w)), high.dtype, alpha=w.alpha, canvas=canvas,
                         keep_lse=True)
    lse = torch.empty(w.H, w.N, device="cuda")
    gpu.avits_joint_lse(t["latent_q"], dev(k_all, w.dtype), lse)
    mass = torch.empty(w.H, w.N, device="cuda")
    gpu.avits_joint_attention_stats(t["latent_q"], dev(k_all, w.dtype), w.L, mass)
    step.score(t["latent_q"], t["text_k"], lse, high, t["feat_prev"])
    step.select()
    step.gather(low, high, prefix)
    torch.cuda.synchronize()
    out = {"w": w, "si": si, "lay": lay, "wt": wt, "wi": wi, "k_all": k_all, "prefix": prefix_np,
           "lse": host(lse), "mass": host(mass), "scores": step.scores.cpu().numpy(), "a": host(step.a_raw),
           "v": host(step.v_raw), "idx": step.idx.cpu().numpy(), "compact": host(step.compact),
           "pos": step.pos.cpu().numpy(), "canvas_gather": host(canvas)}
    step.block()
    torch.cuda.synchronize()
    out["x_out"] = host(step.x_out)
    out["lse_block"] = host(step.lse)
    step.scatter(high)
    torch.cuda.synchronize()
    out["canvas_scatter"] = host(canvas)
    # Kept for the determinism check (device tensors of this case).
    out["dev"] = {"step": step, "canvas": canvas, "lse": lse, "high": high, "low": low, "prefix": prefix, **t}
    yield out
    out.pop("dev")
    del step, canvas, lse, mass, high, low, prefix, t
    torch.cuda.empty_cache()


def test_joint_lse_all_rows(run):
    w = run["w"]
    ref, _ = _oracle_lse_mass(w, run["si"], run["k_all"])
    err = np.abs(run["lse"] - ref).max()
    assert err < (1e-4 if w.dtype == "f32" else 2e-3), err
    assert_close(run["lse"], ref, w.dtype, "joint_lse")


def test_text_mass_all_rows(run):
    w = run["w"]
    _, ref = _oracle_lse_mass(w, run["si"], run["k_all"])
    assert_close(run["mass"], ref, w.dtype, "text mass")
    assert np.abs(run["mass"] - ref).max() < (1e-4 if w.dtype == "f32" else 2e-3)


def test_score(run):
    w, si = run["w"], run["si"]
    s_ref, a_ref, v_ref = oracle.score(si["latent_q"], si["text_k"], run["lse"], si["feat_t"], si["feat_prev"],
                                       w.alpha, w.eps_minmax)
    assert_close(run["a"], a_ref, w.dtype, "A")
    assert_close(run["v"], v_ref, w.dtype, "V")
    assert_close(run["scores"], s_ref, w.dtype, "S")
    assert np.abs(run["scores"] - s_ref).max() < 1e-4


def test_select_bitexact(run):
    w = run["w"]
    idx = run["idx"]
    np.testing.assert_array_equal(idx, oracle.select_topk(run["scores"], w.k))
    assert idx.shape == (w.k,) and (w.k < 2 or np.all(np.diff(idx) > 0))


def test_gather_bitexact(run):
    w, lay = run["w"], run["lay"]
    compact, pos, canvas = oracle.gather_upsample(lay["lowres"], lay["highres_prev"], run["prefix"], run["idx"],
                                                  w.H_lr, w.W_lr)
    np.testing.assert_array_equal(run["compact"], compact)
    np.testing.assert_array_equal(run["pos"][w.LR:], pos)
    np.testing.assert_array_equal(run["pos"][:w.LR], G.prefix_positions(w))
    np.testing.assert_array_equal(run["canvas_gather"], canvas)


def _block_rows(w):
    """Every row where the oracle is quick; else one random row in every
    128-row block of the sequence plus the text head/tail and the last rows."""
    if w.S <= FULL_BLOCK_ROWS:
        return np.arange(w.S)
    g = np.random.default_rng(w.seed + 17)
    starts = np.arange(0, w.S, 128)
    per_block = starts + g.integers(0, 128, size=starts.size)
    per_block = per_block[per_block < w.S]
    rows = np.concatenate([np.arange(min(16, w.L)), np.arange(max(w.L - 8, 0), w.L), per_block,
                           np.arange(max(w.S - 8, 0), w.S)])
    return np.unique(rows)


def test_block_rows(run):
    w = run["w"]
    rows = _block_rows(w)
    if w.S > FULL_BLOCK_ROWS:
        # Every attention unit (128 query rows) holds a checked row.
        assert np.unique(rows // 128).size == -(-w.S // 128)
    ref, ref_lse = oracle.double_block(run["compact"], run["pos"], w.L, run["wt"], run["wi"], w.H, rows=rows)
    x = run["compact"][rows]
    got = run["x_out"][rows]
    assert_close(got, ref, w.dtype, "x_out rows")
    assert_close(got - x, ref - x, w.dtype, "block update rows")
    assert_close(run["lse_block"][:, rows], ref_lse, w.dtype, "block lse rows")


def test_scatter_bitexact(run):
    w = run["w"]
    ref = oracle.scatter(run["x_out"], run["idx"], w.LR, run["canvas_gather"])
    np.testing.assert_array_equal(run["canvas_scatter"], ref)


def test_end_to_end_selection_against_oracle_scores(run):
    # The oracle's own selection (its own joint LSE and scores) may differ from
    # the GPU's only at the selection boundary.
    w, si = run["w"], run["si"]
    lse, _ = _oracle_lse_mass(w, si, run["k_all"])
    s_ref, _, _ = oracle.score(si["latent_q"], si["text_k"], lse, si["feat_t"], si["feat_prev"], w.alpha,
                               w.eps_minmax)
    idx_ref = oracle.select_topk(s_ref, w.k)
    got = set(run["idx"].tolist())
    ref = set(idx_ref.tolist())
    assert len(got) == len(ref) == w.k
    if w.k in (0, w.N):
        assert got == ref
    else:
        kth = np.sort(s_ref.astype(np.float64))[::-1][w.k - 1]
        tol = 1e-4 if w.dtype == "f32" else 1e-2 * float(s_ref.max() - s_ref.min())
        for i in got ^ ref:
            assert abs(float(s_ref[i]) - kth) <= tol, (i, float(s_ref[i]), kth)
    if w.dtype == "f32":
        assert np.abs(run["scores"] - s_ref).max() <= 1e-4
    else:
        assert rel_l2(run["scores"], s_ref) < 1e-2


def test_step_is_deterministic(run):
    """The whole step again on the same inputs and buffers: indices, gathered
    rows, block output, LSE and canvas equal to the first run bit for bit."""
    d = run["dev"]
    step = d["step"]
    step.score(d["latent_q"], d["text_k"], d["lse"], d["high"], d["feat_prev"])
    step.select()
    step.gather(d["low"], d["high"], d["prefix"])
    step.block()
    step.scatter(d["high"])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(step.scores.cpu().numpy(), run["scores"])
    np.testing.assert_array_equal(step.idx.cpu().numpy(), run["idx"])
    np.testing.assert_array_equal(host(step.compact), run["compact"])
    np.testing.assert_array_equal(host(step.x_out), run["x_out"])
    np.testing.assert_array_equal(host(step.lse), run["lse_block"])
    np.testing.assert_array_equal(host(d["canvas"]), run["canvas_scatter"])


def test_step_graph_replay(run):
    """The whole step captured in a HIP graph (the library allocates, sets
    and synchronises nothing inside a call): every replay, with eager steps
    and synchronisations between the replays, equals the eager results bit
    for bit."""
    d = run["dev"]
    step = d["step"]

    def one():
        step.score(d["latent_q"], d["text_k"], d["lse"], d["high"], d["feat_prev"])
        step.select()
        step.gather(d["low"], d["high"], d["prefix"])
        step.block()
        step.scatter(d["high"])

    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        one()
    torch.cuda.synchronize()
    for rep in range(3):
        d["canvas"].fill_(0)
        step.x_out.fill_(0)
        graph.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(step.scores.cpu().numpy(), run["scores"], err_msg=f"replay {rep}")
        np.testing.assert_array_equal(step.idx.cpu().numpy(), run["idx"], err_msg=f"replay {rep}")
        np.testing.assert_array_equal(host(step.compact), run["compact"], err_msg=f"replay {rep}")
        np.testing.assert_array_equal(host(step.x_out), run["x_out"], err_msg=f"replay {rep}")
        np.testing.assert_array_equal(host(step.lse), run["lse_block"], err_msg=f"replay {rep}")
        np.testing.assert_array_equal(host(d["canvas"]), run["canvas_scatter"], err_msg=f"replay {rep}")
        one()  # eager work between replays
        torch.cuda.synchronize()
    del graph
