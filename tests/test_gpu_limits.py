"""Operands beyond 4 GiB: the GEMM's buffer resources have 32-bit ranges, so
an activation matrix of 4 GiB or more must still be read in full (rows past
the 4 GiB mark neither zero-filled nor wrapped).  avits_linear on a
[M, 2048] bf16 input of 4.25 GiB, through the 256-wide (ping-pong) and the
128-wide tile kernels; rows around the 4 GiB mark and the last rows are
compared with an fp64 product of the same rows."""
import os

import numpy as np
import pytest
import torch

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

K = 2048
M = (1 << 32) // (2 * K) + 65536 + 77     # 4 GiB of rows, then 65613 more (a ragged last tile)


@pytest.mark.parametrize("tile,N", [("256,1", 256), ("128,1", 128)])
def test_linear_beyond_4gib(gpu, tile, N):
    print(f"\n[limits] linear M={M} K={K} N={N} tile={tile}", flush=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    x = torch.randn(M, K, device="cuda", generator=g).to(torch.bfloat16)
    w = (torch.randn(N, K, device="cuda", generator=g) * 0.02).to(torch.bfloat16)
    b = (torch.randn(N, device="cuda", generator=g) * 0.02).to(torch.bfloat16)
    out = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    old = os.environ.get("AVITS_GEMM_TILE_linear")
    os.environ["AVITS_GEMM_TILE_linear"] = tile
    try:
        gpu.avits_linear(x, w, b, out)
        torch.cuda.synchronize()
    finally:
        if old is None:
            os.environ.pop("AVITS_GEMM_TILE_linear", None)
        else:
            os.environ["AVITS_GEMM_TILE_linear"] = old
    edge = (1 << 32) // (2 * K)
    rows = np.unique(np.concatenate([np.arange(0, 8), np.arange(edge - 300, edge + 300), np.arange(M - 300, M)]))
    rt = torch.from_numpy(rows).cuda()
    xs = x.index_select(0, rt).float().cpu().numpy().astype(np.float64)
    got = out.index_select(0, rt).float().cpu().numpy().astype(np.float64)
    ref = xs @ w.float().cpu().numpy().astype(np.float64).T + b.float().cpu().numpy().astype(np.float64)
    err = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    assert err < 1e-2, err
    # No row past the 4 GiB mark came back as the bias alone (a zero-filled input row).
    tail = rows >= edge
    assert np.all(np.abs(got[tail] - ref[tail]).max(axis=1) < 0.05 * np.abs(ref[tail]).max(axis=1) + 1e-2)
    del x, out
    torch.cuda.empty_cache()
