"""Every GEMM kernel instance on ragged shapes.  avits_linear (bias, plain
row-major store) with the plan forced to each unsplit tile form -- the
256-wide ping-pong kernel, the 192-wide kernel, the 128-wide kernel with one
and with two register stages -- and the fp32 kernel, on M, N and K that leave
partial row and column tiles, element by element against an fp64 product of
the same (bf16-rounded) operands.  The bound per element: the products are
summed in fp32 (at most K roundings of a partial sum no larger than
sum_k |x_k w_k|) and the result is rounded once to the output type (half an
ulp: 2^-8 relative for bf16).  Nothing is written past the M x N output."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

SHAPES = [(1, 8, 64), (255, 136, 128), (257, 264, 192), (600, 520, 448), (1030, 1288, 64)]
PLANS = ["256,1", "192,1", "128,1,8,1", "128,1,8,2"]


def _run(gpu, monkeypatch, M, N, K, dtype, plan=None):
    if plan is not None:
        monkeypatch.setenv("AVITS_GEMM_TILE_linear", plan)
    g = torch.Generator(device="cuda")
    g.manual_seed(M * 7919 + N * 31 + K)
    x = torch.randn(M, K, device="cuda", generator=g).to(dtype)
    w = (torch.randn(N, K, device="cuda", generator=g) * 0.05).to(dtype)
    b = (torch.randn(N, device="cuda", generator=g) * 0.05).to(dtype)
    pad = 4096
    buf = torch.full((M * N + pad,), 7.0, device="cuda", dtype=dtype)
    out = buf[:M * N].view(M, N)
    gpu.avits_linear(x, w, b, out)
    torch.cuda.synchronize()
    xs = x.float().cpu().numpy().astype(np.float64)
    ws = w.float().cpu().numpy().astype(np.float64)
    bs = b.float().cpu().numpy().astype(np.float64)
    ref = xs @ ws.T + bs
    mag = np.abs(xs) @ np.abs(ws).T + np.abs(bs)
    got = out.float().cpu().numpy().astype(np.float64)
    tail = buf[M * N:].float().cpu().numpy()
    return got, ref, mag, tail


def _check(got, ref, mag, tail, half_ulp, K):
    assert np.all(np.isfinite(got))
    acc = (K + 1) * 2.0 ** -24 * mag  # the fp32 sum's rounding (K products and the bias)
    bound = half_ulp * (np.abs(ref) + acc) + acc + 1e-30  # then one rounding of that sum
    excess = np.abs(got - ref) - bound
    assert np.all(excess <= 0), f"worst excess {excess.max():.3e} at {np.unravel_index(excess.argmax(), excess.shape)}"
    assert np.all(tail == 7.0), "written past the output"


@pytest.mark.parametrize("M,N,K", SHAPES, ids=[f"{m}x{n}x{k}" for m, n, k in SHAPES])
@pytest.mark.parametrize("plan", PLANS)
def test_linear_bf16_every_tile_form(gpu, monkeypatch, plan, M, N, K):
    got, ref, mag, tail = _run(gpu, monkeypatch, M, N, K, torch.bfloat16, plan)
    # The output is rounded to bf16 once: half an ulp is 2^-8 of the magnitude
    # (at most; 2^-9 of a value at the top of its binade).
    _check(got, ref, mag, tail, 2.0 ** -8, K)


@pytest.mark.parametrize("M,N,K", SHAPES, ids=[f"{m}x{n}x{k}" for m, n, k in SHAPES])
def test_linear_f32(gpu, monkeypatch, M, N, K):
    got, ref, mag, tail = _run(gpu, monkeypatch, M, N, K, torch.float32)
    _check(got, ref, mag, tail, 2.0 ** -24, K)
