"""The allocation-free selection (avits_select_noalloc) against avits_select.

The host-side checks run anywhere; the GPU test calls both entry points
through the C ABI on the same scores, twice in a row with the second input
smaller (the fixed device array keeps the first call's contents), and
requires the indices to match bit for bit.
"""
import numpy as np
import pytest

import paper_2608_17995_amd as avits

INVALID = -1
FAKE = 0x1000  # never dereferenced: the calls below fail validation first


def test_noalloc_validation():
    lib = avits.load()
    nmax = lib.avits_select_noalloc_max_n()
    assert nmax == 1 << 26
    assert lib.avits_select_noalloc(FAKE, nmax + 1, 5, FAKE, None) == INVALID      # beyond the fixed array
    assert b"N=" in lib.avits_last_error()
    assert lib.avits_select_noalloc(FAKE, 0, 0, FAKE, None) == INVALID             # N < 1
    assert lib.avits_select_noalloc(FAKE, 10, 11, FAKE, None) == INVALID           # k > N
    assert lib.avits_select_noalloc(FAKE, 10, -1, FAKE, None) == INVALID           # k < 0
    assert lib.avits_select_noalloc(None, 10, 3, None, None) == INVALID            # null pointers
    assert lib.avits_select_noalloc(None, 10, 0, None, None) == 0                  # k == 0: no-op


def _scores(torch, N, seed, ties):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    s = torch.rand(N, device="cuda", generator=g) ** 0.25
    if ties:
        s = torch.floor(s * 64) / 64     # heavy ties: the lowest index must win
    return s.contiguous()


@pytest.mark.gpu
@pytest.mark.parametrize("sizes", [((3_000_001, 900_000), (100_003, 30_001)),
                                   ((1 << 22, 1 << 20), (16_385, 7)),
                                   ((50_000, 49_999), (4096, 1229))])
def test_noalloc_matches_workspace_select(gpu, sizes):
    import torch
    for call, (N, k) in enumerate(sizes):
        for ties in (False, True):
            print(f"[noalloc] call {call}: N={N} k={k} ties={ties}", flush=True)
            s = _scores(torch, N, 1000 * call + N % 997, ties)
            want = torch.empty(k, dtype=torch.int32, device="cuda")
            got = torch.full((k,), -1, dtype=torch.int32, device="cuda")
            gpu.avits_select(s, k, want)
            gpu.avits_select_noalloc(s, k, got)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(got.cpu().numpy(), want.cpu().numpy())
            g = got.cpu().numpy()
            assert np.all(np.diff(g) > 0) and g[0] >= 0 and g[-1] < N
