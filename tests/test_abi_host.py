"""Host-side checks of the C ABI: the library loads, exports every declared
symbol, and rejects invalid arguments before touching any device memory."""
import os
import re
import subprocess

import pytest

import paper_2608_17995_amd as avits
from paper_2608_17995_amd import _binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "avits.h")

INVALID, UNSUPPORTED, WORKSPACE = -1, -2, -3
FAKE = 0x1000  # never dereferenced: every call below fails validation first


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]*?\b(avits_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(avits.lib_path()):
        pytest.fail("libavits.so is not built (python -m paper_2608_17995_amd.build)")
    return avits.load()


def test_header_declares_the_boundary():
    names = _declared()
    for want in ("avits_score", "avits_select", "avits_gather_upsample", "avits_block_forward",
                 "avits_scatter", "avits_joint_lse", "avits_last_error", "avits_version"):
        assert want in names


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", avits.lib_path()], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (avits_\w+)", out))
    missing = [n for n in _declared() if n not in exported]
    assert not missing, missing
    assert set(_binding.EXPORTS) <= exported


def test_version_and_error_text(lib):
    assert avits.version().count(".") == 2
    assert lib.avits_select(None, 10, 11, None, None, 0, None) == INVALID
    assert b"k=11" in lib.avits_last_error()


def test_select_validation(lib):
    assert lib.avits_select(None, 0, 0, None, None, 0, None) == INVALID       # N < 1
    assert lib.avits_select(None, 10, -1, None, None, 0, None) == INVALID     # k < 0
    assert lib.avits_select(None, 10, 0, None, None, 0, None) == 0            # k == 0: no-op
    assert lib.avits_select(None, 10, 3, None, None, 0, None) == INVALID      # null pointers
    assert lib.avits_select_workspace_bytes(4096) == 0
    need = lib.avits_select_workspace_bytes(20000)              # grid-wide path: state + chunk counts
    assert need > 0
    assert lib.avits_select(FAKE, 20000, 5, FAKE, None, need, None) == WORKSPACE
    assert lib.avits_select(FAKE, 20000, 5, FAKE, FAKE, need - 1, None) == WORKSPACE


def _score(lib, **kw):
    a = dict(q=FAKE, k=FAKE, lse=FAKE, ft=FAKE, fp=FAKE, N=16, L=4, H=2, d=64, Df=8, alpha=0.5, eps=1e-8,
             dtype=1, S=FAKE, ws=FAKE, wsb=1 << 30)
    a.update(kw)
    return lib.avits_score(a["q"], a["k"], a["lse"], a["ft"], a["fp"], a["N"], a["L"], a["H"], a["d"], a["Df"],
                           a["alpha"], a["eps"], a["dtype"], a["S"], None, None, a["ws"], a["wsb"], None)


def test_select_perturbed_and_batched_validation(lib):
    import ctypes
    f = lib.avits_select_perturbed
    assert f(FAKE, None, 10, 3, FAKE, None, 0, None) == INVALID          # delta required
    assert f(FAKE, FAKE, 10, 11, FAKE, None, 0, None) == INVALID         # k > N
    assert f(FAKE, FAKE, 20000, 5, FAKE, None, 0, None) == WORKSPACE     # grid path needs workspace
    assert f(None, None, 10, 0, None, None, 0, None) == 0                # k == 0: no-op
    b = lib.avits_select_batched
    I64 = ctypes.c_int64

    def arr(*v):
        return (I64 * len(v))(*v)

    assert b(FAKE, None, 0, arr(0), arr(), FAKE, None) == INVALID                    # B < 1
    assert b(FAKE, None, 65, arr(*range(66)), arr(*([1] * 65)), FAKE, None) == INVALID  # B > 64
    assert b(FAKE, None, 2, arr(1, 5, 9), arr(1, 1), FAKE, None) == INVALID           # offsets[0] != 0
    assert b(FAKE, None, 2, arr(0, 5, 5), arr(1, 0), FAKE, None) == INVALID           # empty element
    assert b(FAKE, None, 2, arr(0, 5, 9), arr(6, 1), FAKE, None) == INVALID           # k > N_b
    assert b(FAKE, None, 1, arr(0, 16385), arr(1), FAKE, None) == INVALID             # N_b > 16384
    assert b(None, None, 2, arr(0, 5, 9), arr(0, 0), None, None) == 0                 # nothing to select
    assert b(None, None, 2, arr(0, 5, 9), arr(1, 0), None, None) == INVALID           # null scores/idx


def test_score_validation(lib):
    assert _score(lib, N=0) == INVALID
    assert _score(lib, L=0) == INVALID
    assert _score(lib, alpha=1.5) == INVALID
    assert _score(lib, alpha=-0.1) == INVALID
    assert _score(lib, eps=-1.0) == INVALID
    assert _score(lib, d=96) == UNSUPPORTED
    assert _score(lib, dtype=7) == UNSUPPORTED
    assert _score(lib, q=None) == INVALID
    assert _score(lib, ws=None) == WORKSPACE
    need = lib.avits_score_workspace_bytes(16, 2)
    assert need >= 16 * 2 * 4
    assert _score(lib, wsb=need - 1) == WORKSPACE


def test_score_batched_validation(lib):
    def call(**kw):
        a = dict(q=FAKE, B=2, N=16, L=4, H=2, d=64, Df=8, alpha=0.5, dtype=1, ws=FAKE, wsb=1 << 30)
        a.update(kw)
        return lib.avits_score_batched(a["q"], FAKE, FAKE, FAKE, FAKE, a["B"], a["N"], a["L"], a["H"], a["d"],
                                       a["Df"], a["alpha"], 1e-8, a["dtype"], FAKE, None, None, a["ws"], a["wsb"],
                                       None)

    assert call(B=0) == INVALID
    assert call(B=4097) == INVALID
    assert call(N=0) == INVALID
    assert call(alpha=2.0) == INVALID
    assert call(d=32) == UNSUPPORTED
    assert call(q=None) == INVALID
    assert lib.avits_score_batched_workspace_bytes(0, 16, 2) == 0
    one = lib.avits_score_workspace_bytes(16, 2)
    assert lib.avits_score_batched_workspace_bytes(1, 16, 2) == one
    need = lib.avits_score_batched_workspace_bytes(3, 16, 2)
    assert need >= 3 * 16 * 2 * 4 * 2 and need > one      # per-image partials of A and V
    assert call(B=3, wsb=need - 1) == WORKSPACE
    assert call(B=3, ws=None) == WORKSPACE


def test_sampler_side_validation(lib):
    f = lib.avits_linear
    # (x, M, K, w, b, N, dtype, out, stream)
    assert f(FAKE, -1, 64, FAKE, None, 8, 1, FAKE, None) == INVALID
    assert f(FAKE, 4, 60, FAKE, None, 8, 1, FAKE, None) == INVALID        # K not a multiple of 64
    assert f(FAKE, 4, 64, FAKE, None, 12, 1, FAKE, None) == INVALID       # N not a multiple of 8
    assert f(FAKE, 4, 64, FAKE, None, 8, 5, FAKE, None) == UNSUPPORTED
    assert f(None, 0, 64, None, None, 8, 1, None, None) == 0              # M == 0: no-op
    assert f(None, 4, 64, FAKE, None, 8, 1, FAKE, None) == INVALID
    g = lib.avits_final_layer
    need = lib.avits_final_layer_workspace_bytes(16, 128, 1)
    assert need >= 16 * 128 * 2
    assert lib.avits_final_layer_workspace_bytes(16, 128, 7) == 0
    # (x, M, D, mod, w, b, C, dtype, out, ws, wsb, stream)
    assert g(FAKE, 16, 100, FAKE, FAKE, None, 64, 1, FAKE, FAKE, need, None) == INVALID
    assert g(FAKE, 16, 128, None, FAKE, None, 64, 1, FAKE, FAKE, need, None) == INVALID
    assert g(FAKE, 16, 128, FAKE, FAKE, None, 64, 1, FAKE, FAKE, need - 1, None) == WORKSPACE
    assert g(FAKE, 16, 128, FAKE, FAKE, None, 64, 1, FAKE, None, need, None) == WORKSPACE
    e = lib.avits_euler_update
    assert e(FAKE, FAKE, -1, 0.1, 1, None) == INVALID
    assert e(FAKE, FAKE, 8, float("nan"), 1, None) == INVALID
    assert e(FAKE, FAKE, 8, 0.1, 3, None) == UNSUPPORTED
    assert e(None, None, 0, 0.1, 1, None) == 0
    assert e(FAKE + 2, FAKE, 8, 0.1, 1, None) == INVALID                  # misaligned


def test_gather_and_scatter_validation(lib):
    g = lib.avits_gather_upsample
    # k > N (N = 4*2*2 = 16)
    assert g(FAKE, FAKE, None, FAKE, 17, 2, 2, 0, 64, 0, 1, FAKE, FAKE, FAKE, None) == INVALID
    assert g(FAKE, FAKE, None, FAKE, 3, 0, 2, 0, 64, 0, 1, FAKE, FAKE, FAKE, None) == INVALID   # H_lr
    assert g(FAKE, FAKE, None, FAKE, 3, 2, 2, 0, 64, 5, 1, FAKE, FAKE, FAKE, None) == INVALID   # mode
    assert g(FAKE, FAKE, None, FAKE, 3, 2, 2, 0, 60, 0, 1, FAKE, FAKE, FAKE, None) == INVALID   # 120-byte rows
    assert g(FAKE, FAKE, None, FAKE, 3, 2, 2, 4, 64, 0, 1, FAKE, FAKE, FAKE, None) == INVALID   # null prefix
    assert g(FAKE, FAKE, None, FAKE, 3, 2, 2, 0, 64, 0, 9, FAKE, FAKE, FAKE, None) == UNSUPPORTED
    s = lib.avits_scatter
    assert s(FAKE, FAKE, -1, 0, 64, 16, 1, FAKE, None) == INVALID
    assert s(FAKE, FAKE, 0, 0, 64, 16, 1, FAKE, None) == 0        # k == 0: no-op
    assert s(None, FAKE, 3, 0, 64, 16, 1, FAKE, None) == INVALID
    assert s(FAKE, FAKE, 3, 0, 64, 0, 1, FAKE, None) == INVALID     # n_canvas < 1
    assert s(FAKE, FAKE, 3, 0, 64, 16, 3, FAKE, None) == UNSUPPORTED


def test_batched_gather_and_scatter_validation(lib):
    import ctypes
    I64 = ctypes.c_int64

    def arr(*v):
        return (I64 * len(v))(*v)

    g = lib.avits_gather_upsample_batched
    # (lowres, highres, prefix, idx, idx_off, B, H_lr, W_lr, n_prefix, D, mode, dtype, compact, row_off, pos,
    #  canvas, stream); N = 16
    ok = dict(idx_off=arr(0, 3, 5), B=2, row_off=arr(0, 3))

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return g(FAKE, FAKE, None, FAKE, a["idx_off"], a["B"], 2, 2, 0, 64, 0, 1, FAKE, a["row_off"], FAKE, FAKE,
                 None)

    assert call(B=0) == INVALID
    assert call(B=65) == INVALID
    assert call(idx_off=None) == INVALID
    assert call(idx_off=arr(1, 3, 5)) == INVALID        # idx_off[0] != 0
    assert call(idx_off=arr(0, 3, 2)) == INVALID        # negative k_b
    assert call(idx_off=arr(0, 17, 18)) == INVALID      # k_b > N
    assert call(row_off=arr(0, -1)) == INVALID
    assert g(FAKE, FAKE, None, FAKE, arr(0, 1), 1, 2, 2, 0, 60, 0, 1, FAKE, arr(0), FAKE, FAKE, None) == INVALID
    assert g(FAKE, FAKE, None, FAKE, arr(0, 1), 1, 2, 2, 0, 64, 0, 9, FAKE, arr(0), FAKE, FAKE, None) == UNSUPPORTED
    s = lib.avits_scatter_batched
    # (out, idx, idx_off, B, row_off, N, D, dtype, canvas, stream)
    assert s(FAKE, FAKE, arr(0, 2), 0, arr(0), 16, 64, 1, FAKE, None) == INVALID      # B < 1
    assert s(FAKE, FAKE, arr(0, 17), 1, arr(0), 16, 64, 1, FAKE, None) == INVALID     # k_b > N
    assert s(FAKE, FAKE, arr(0, 2), 1, arr(-1), 16, 64, 1, FAKE, None) == INVALID     # row_off < 0
    assert s(None, None, arr(0, 0, 0), 2, arr(0, 0), 16, 64, 1, None, None) == 0      # nothing selected
    assert s(None, FAKE, arr(0, 2), 1, arr(0), 16, 64, 1, FAKE, None) == INVALID      # null out
    assert s(FAKE, FAKE, arr(0, 2), 1, arr(0), 16, 64, 3, FAKE, None) == UNSUPPORTED


def test_mixed_gather_and_scatter_validation(lib):
    g = lib.avits_gather_mixed
    # (lowres, prefix, idx, k, H_lr, W_lr, n_prefix, D, mode, dtype, compact, pos, children, stream)
    assert g(FAKE, None, FAKE, 5, 2, 2, 0, 64, 0, 1, FAKE, FAKE, None, None) == INVALID    # k > M' = 4
    assert g(FAKE, None, FAKE, 2, 0, 2, 0, 64, 0, 1, FAKE, FAKE, None, None) == INVALID    # H_lr
    assert g(FAKE, None, FAKE, 2, 2, 2, 0, 64, 7, 1, FAKE, FAKE, None, None) == INVALID    # mode
    assert g(FAKE, None, FAKE, 2, 2, 2, 0, 60, 0, 1, FAKE, FAKE, None, None) == INVALID    # 120-byte rows
    assert g(FAKE, None, FAKE, 2, 2, 2, 3, 64, 0, 1, FAKE, FAKE, None, None) == INVALID    # null prefix
    assert g(FAKE, None, None, 2, 2, 2, 0, 64, 0, 1, FAKE, FAKE, None, None) == INVALID    # null idx
    assert g(FAKE, None, FAKE, 2, 2, 2, 0, 64, 0, 1, FAKE, None, None, None) == INVALID    # null pos
    assert g(FAKE, None, FAKE, 2, 2, 2, 0, 64, 0, 4, FAKE, FAKE, None, None) == UNSUPPORTED
    s = lib.avits_scatter_mixed
    # (out, idx, k, H_lr, W_lr, row_offset, D, dtype, canvas_hr, state_lr, stream)
    assert s(FAKE, FAKE, 5, 2, 2, 0, 64, 1, FAKE, FAKE, None) == INVALID      # k > M'
    assert s(FAKE, FAKE, 2, 2, 2, -1, 64, 1, FAKE, FAKE, None) == INVALID     # row_offset
    assert s(FAKE, FAKE, 2, 2, 2, 0, 64, 1, None, FAKE, None) == INVALID      # canvas needed
    assert s(FAKE, FAKE, 2, 2, 2, 0, 64, 1, FAKE, None, None) == INVALID      # state needed
    assert s(None, FAKE, 2, 2, 2, 0, 64, 1, FAKE, FAKE, None) == INVALID
    assert s(FAKE, FAKE, 2, 2, 2, 0, 64, 2, FAKE, FAKE, None) == UNSUPPORTED


def test_joint_lse_validation(lib):
    f = lib.avits_joint_lse
    assert f(FAKE, FAKE, 0, 5, 2, 64, 1, FAKE, None) == INVALID
    assert f(FAKE, FAKE, 5, 0, 2, 64, 1, FAKE, None) == INVALID
    assert f(FAKE, FAKE, 5, 5, 2, 32, 1, FAKE, None) == UNSUPPORTED
    assert f(None, FAKE, 5, 5, 2, 64, 1, FAKE, None) == INVALID


def test_block_validation(lib):
    import ctypes
    w = _binding._BlockWeights()
    w.kind, w.mlp_hidden = 0, 256
    f = lib.avits_block_forward
    ws = lib.avits_block_workspace_bytes(0, 10, 1, 64, 256, 1)
    assert ws > 0
    assert f(FAKE, FAKE + 64, FAKE, 1.0, 5, 5, None, 1, 64, 1, None, FAKE, ws, None) == INVALID          # null weights
    assert f(FAKE, FAKE + 64, FAKE, 1.0, 5, 5, ctypes.byref(w), 1, 64, 1, None, FAKE, ws, None) == INVALID  # missing weights
    assert f(FAKE, FAKE + 64, FAKE, 0.0, 5, 5, ctypes.byref(w), 1, 64, 1, None, FAKE, ws, None) == INVALID  # pos_scale
    assert f(FAKE, FAKE + 64, FAKE, 1.0, 5, 5, ctypes.byref(w), 1, 80, 1, None, FAKE, ws, None) == UNSUPPORTED
    assert f(FAKE, FAKE + 64, FAKE, 1.0, -1, 5, ctypes.byref(w), 1, 64, 1, None, FAKE, ws, None) == INVALID
    assert f(FAKE, FAKE, FAKE, 1.0, 5, 5, ctypes.byref(w), 1, 64, 1, None, FAKE, ws, None) == INVALID  # alias
    assert f(FAKE, FAKE + 64, FAKE, 1.0, 0, 0, ctypes.byref(w), 1, 64, 1, None, None, 0, None) == 0    # S == 0
    for part in ("txt", "img"):
        for name, _ in _binding._DoubleStream._fields_:
            setattr(getattr(w, part), name, FAKE)
    assert f(FAKE, FAKE + 64, FAKE, 1.0, 5, 5, ctypes.byref(w), 1, 64, 1, None, FAKE, ws - 1, None) == WORKSPACE
    assert f(FAKE, FAKE + 64, FAKE, 1.0, 5, 5, ctypes.byref(w), 1, 64, 1, None, None, ws, None) == WORKSPACE
    w.kind = 5
    assert f(FAKE, FAKE + 64, FAKE, 1.0, 5, 5, ctypes.byref(w), 1, 64, 1, None, FAKE, ws, None) == INVALID
    w.kind, w.mlp_hidden = 0, 100
    assert f(FAKE, FAKE + 64, FAKE, 1.0, 5, 5, ctypes.byref(w), 1, 64, 1, None, FAKE, ws, None) == INVALID
    assert lib.avits_block_workspace_bytes(1, 10, 1, 64, 256, 1) > 0
    assert lib.avits_block_workspace_bytes(3, 10, 1, 64, 256, 1) == 0


def test_block_batched_validation(lib):
    import ctypes
    f = lib.avits_block_forward_batched
    w = _binding._BlockWeights()
    w.kind = 0
    w.mlp_hidden = 256
    ws = 1 << 30
    I64 = ctypes.c_int64

    def arr(*v):
        return (I64 * len(v))(*v)

    args = lambda B, to, io, dt=1: f(FAKE, FAKE + 64, FAKE, 1.0, B, to, io, ctypes.byref(w), 1, 64, dt, None, FAKE, ws, None)
    assert args(0, arr(0), arr(0)) == INVALID                      # B < 1
    assert args(17, arr(*range(18)), arr(*range(18))) == INVALID   # B > 16
    assert args(2, arr(1, 2, 3), arr(0, 1, 2)) == INVALID          # txt_off[0] != 0
    assert args(2, arr(0, 1, 1), arr(0, 1, 1)) == INVALID          # empty image
    assert args(2, arr(0, 2, 1), arr(0, 0, 3)) == INVALID          # decreasing offsets
    assert args(1, arr(0, 2), arr(0, 3)) == INVALID                # missing weights


def test_block_qk_validation(lib):
    import ctypes
    w = _binding._BlockWeights()
    w.kind, w.mlp_hidden = 0, 256
    f = lib.avits_block_qk
    ws = lib.avits_block_qk_workspace_bytes(10, 2, 64, 1)
    assert ws >= 10 * 128 * 2 and lib.avits_block_qk_workspace_bytes(10, 2, 64, 0) >= 10 * 128 * 4
    assert lib.avits_block_qk_workspace_bytes(10, 0, 64, 1) == 0
    q, k = FAKE + 4096, FAKE + 8192
    assert f(FAKE, FAKE, 1.0, 5, 5, None, 2, 64, 1, q, k, FAKE, ws, None) == INVALID                 # null weights
    assert f(FAKE, FAKE, 1.0, 5, 5, ctypes.byref(w), 2, 64, 1, q, k, FAKE, ws, None) == INVALID      # missing weights
    assert f(FAKE, FAKE, 1.0, 5, 5, ctypes.byref(w), 2, 96, 1, q, k, FAKE, ws, None) == UNSUPPORTED
    assert f(FAKE, FAKE, 1.0, 5, 5, ctypes.byref(w), 2, 64, 3, q, k, FAKE, ws, None) == UNSUPPORTED
    assert f(FAKE, FAKE, 1.0, 0, 0, ctypes.byref(w), 2, 64, 1, None, None, None, 0, None) == 0     # S == 0
    for part in ("txt", "img"):
        for name, _ in _binding._DoubleStream._fields_:
            setattr(getattr(w, part), name, FAKE)
    assert f(FAKE, FAKE, 1.0, 5, 5, ctypes.byref(w), 2, 64, 1, q, q, FAKE, ws, None) == INVALID      # q aliases k
    assert f(FAKE, FAKE, 1.0, 5, 5, ctypes.byref(w), 2, 64, 1, None, k, FAKE, ws, None) == INVALID
    assert f(FAKE, FAKE, 1.0, 5, 5, ctypes.byref(w), 2, 64, 1, q, k, FAKE, ws - 1, None) == WORKSPACE
    assert f(FAKE, FAKE, 1.0, 5, 5, ctypes.byref(w), 2, 64, 1, q, k, None, ws, None) == WORKSPACE
    assert b"block_qk" in lib.avits_last_error()


def test_stats_and_mass_score_validation(lib):
    f = lib.avits_joint_attention_stats
    assert f(FAKE, FAKE, 0, 5, 2, 2, 64, 1, None, FAKE, 0, None) == INVALID        # N < 1
    assert f(FAKE, FAKE, 5, 5, 6, 2, 64, 1, None, FAKE, 0, None) == INVALID        # L > Nk
    assert f(FAKE, FAKE, 5, 5, -1, 2, 64, 1, None, FAKE, 0, None) == INVALID       # L < 0
    assert f(FAKE, FAKE, 5, 5, 2, 2, 96, 1, None, FAKE, 0, None) == UNSUPPORTED    # head dim
    assert f(FAKE, FAKE, 5, 5, 2, 2, 64, 1, None, None, 0, None) == INVALID        # mass required
    import ctypes
    g = lib.avits_score_from_mass
    ws = lib.avits_score_workspace_bytes(16, 2)
    two = (ctypes.c_void_p * 2)(FAKE, FAKE)
    assert g(FAKE, 16, 2, 1, two, 1, 16, 8, 0.5, 1e-8, 1, FAKE, None, None, FAKE, ws, None) == INVALID  # n_t < 2
    assert g(FAKE, 16, 2, 1, two, 17, 16, 8, 0.5, 1e-8, 1, FAKE, None, None, FAKE, ws, None) == INVALID  # n_t > 16
    assert g(FAKE, 16, 2, 0, two, 2, 16, 8, 0.5, 1e-8, 1, FAKE, None, None, FAKE, ws, None) == INVALID  # count < 1
    assert g(FAKE, 16, 2, 1, two, 2, 16, 8, 1.5, 1e-8, 1, FAKE, None, None, FAKE, ws, None) == INVALID  # alpha
    assert g(FAKE, 16, 2, 1, two, 2, 16, 8, 0.5, 1e-8, 9, FAKE, None, None, FAKE, ws, None) == UNSUPPORTED
    assert g(FAKE, 16, 2, 1, two, 2, 16, 8, 0.5, 1e-8, 1, FAKE, None, None, FAKE, ws - 1, None) == WORKSPACE
    assert g(None, 16, 2, 1, two, 2, 16, 8, 0.5, 1e-8, 1, FAKE, None, None, FAKE, ws, None) == INVALID
    assert g(FAKE, 15, 2, 1, two, 2, 16, 8, 0.5, 1e-8, 1, FAKE, None, None, FAKE, ws, None) == INVALID  # mass_ld < N
    holes = (ctypes.c_void_p * 2)(FAKE, None)
    assert g(FAKE, 16, 2, 1, holes, 2, 16, 8, 0.5, 1e-8, 1, FAKE, None, None, FAKE, ws, None) == INVALID  # null snapshot


def test_position_and_noise_validation(lib):
    assert lib.avits_grid_positions(FAKE, -1, 4, 0, 1, 0, None) == INVALID
    assert lib.avits_grid_positions(FAKE, 5, 0, 0, 1, 0, None) == INVALID      # W < 1
    assert lib.avits_grid_positions(None, 0, 4, 0, 1, 0, None) == 0            # rows == 0: no-op
    assert lib.avits_scale_positions(None, 3, 2, FAKE, None) == INVALID
    f = lib.avits_noise_reinject
    assert f(FAKE, 4, 6, None, 0, 8, 8, 0.5, 1, 1, None) == INVALID           # C not a multiple of 4
    assert f(FAKE, 4, 8, None, 0, 7, 8, 0.5, 1, 1, None) == INVALID           # odd grid
    assert f(FAKE, 4, 8, None, 0, 8, 8, 1.5, 1, 1, None) == INVALID           # t > 1
    assert f(FAKE, 4, 8, None, 3, 8, 8, 0.5, 1, 1, None) == INVALID           # rows_kind
    assert f(FAKE, 65, 8, None, 0, 8, 8, 0.5, 1, 1, None) == INVALID          # more rows than pixels
    assert f(FAKE, 17, 8, None, 2, 8, 8, 0.5, 1, 1, None) == INVALID          # more rows than blocks
    assert f(FAKE, 4, 8, None, 1, 8, 8, 0.5, 1, 1, None) == INVALID           # half units need positions
    assert f(FAKE, 4, 8, None, 0, 8, 8, 0.5, 1, 7, None) == UNSUPPORTED
    assert f(None, 0, 8, None, 0, 8, 8, 0.5, 1, 1, None) == 0                 # rows == 0: no-op
    assert lib.avits_noise_bits(-1, 4, 8, 1, FAKE, None) == INVALID
    assert lib.avits_noise_bits(0, 4, 6, 1, FAKE, None) == INVALID
    assert lib.avits_noise_bits(0, 0, 8, 1, None, None) == 0
