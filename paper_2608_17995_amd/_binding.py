"""ctypes binding of libavits.so (argument marshalling only)."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

F32, BF16 = 0, 1
UP_NEAREST, UP_BILINEAR = 0, 1
BLOCK_DOUBLE, BLOCK_SINGLE = 0, 1

_c_void_p, _i64, _i32, _f32, _size = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t


class AvitsError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"avits error {code}: {msg}")
        self.code = code


class _DoubleStream(ctypes.Structure):
    _fields_ = [(n, _c_void_p) for n in ("mod", "w_qkv", "b_qkv", "g_q", "g_k", "w_o", "b_o",
                                          "w_mlp1", "b_mlp1", "w_mlp2", "b_mlp2")]


class _Single(ctypes.Structure):
    _fields_ = [(n, _c_void_p) for n in ("mod", "w_in", "b_in", "g_q", "g_k", "w_out", "b_out")]


class _BlockOutputs(ctypes.Structure):
    _fields_ = [("lse", ctypes.c_void_p), ("mass", ctypes.c_void_p), ("mass_accumulate", ctypes.c_int32),
                ("scatter_idx", ctypes.c_void_p), ("scatter_k", ctypes.c_int64), ("canvas", ctypes.c_void_p),
                ("n_canvas", ctypes.c_int64), ("h_in", ctypes.c_void_p), ("h_next", ctypes.c_void_p),
                ("next_w", ctypes.c_void_p)]


class _BlockWeights(ctypes.Structure):
    _fields_ = [("kind", _i32), ("mlp_hidden", _i32), ("txt", _DoubleStream), ("img", _DoubleStream),
                ("single", _Single)]


_SIGS = {
    "avits_version": (ctypes.c_char_p, []),
    "avits_last_error": (ctypes.c_char_p, []),
    "avits_score_workspace_bytes": (_size, [_i64, _i32]),
    "avits_score": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _i64, _i64, _i32, _i32,
                                   _i64, _f32, _f32, ctypes.c_int, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                                   _size, _c_void_p]),
    "avits_score_select": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _i64, _i64, _i32, _i32,
                                          _i64, _f32, _f32, ctypes.c_int, _c_void_p, _c_void_p, _c_void_p, _i64,
                                          _c_void_p, _c_void_p, _size, _c_void_p]),
    "avits_score_batched_workspace_bytes": (_size, [_i64, _i64, _i32]),
    "avits_score_batched": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _i64, _i64, _i64,
                                           _i32, _i32, _i64, _f32, _f32, ctypes.c_int, _c_void_p, _c_void_p,
                                           _c_void_p, _c_void_p, _size, _c_void_p]),
    "avits_select_workspace_bytes": (_size, [_i64]),
    "avits_select": (ctypes.c_int, [_c_void_p, _i64, _i64, _c_void_p, _c_void_p, _size, _c_void_p]),
    "avits_select_noalloc_max_n": (_size, []),
    "avits_select_noalloc": (ctypes.c_int, [_c_void_p, _i64, _i64, _c_void_p, _c_void_p]),
    "avits_select_perturbed": (ctypes.c_int, [_c_void_p, _c_void_p, _i64, _i64, _c_void_p, _c_void_p, _size,
                                              _c_void_p]),
    "avits_select_batched": (ctypes.c_int, [_c_void_p, _c_void_p, _i32, _c_void_p, _c_void_p, _c_void_p,
                                            _c_void_p]),
    "avits_gather_upsample": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _i64, _i32, _i32, _i64,
                                             _i64, ctypes.c_int, ctypes.c_int, _c_void_p, _c_void_p, _c_void_p,
                                             _c_void_p]),
    "avits_block_workspace_bytes": (_size, [_i32, _i64, _i32, _i32, _i32, ctypes.c_int]),
    "avits_block_forward": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _f32, _i64, _i64,
                                           ctypes.POINTER(_BlockWeights), _i32, _i32, ctypes.c_int, _c_void_p,
                                           _c_void_p, _size, _c_void_p]),
    "avits_block_forward_ex": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _f32, _i64, _i64,
                                              ctypes.POINTER(_BlockWeights), _i32, _i32, ctypes.c_int,
                                              ctypes.POINTER(_BlockOutputs), _c_void_p, _size, _c_void_p]),
    "avits_noise_reinject": (ctypes.c_int, [_c_void_p, _i64, _i64, _c_void_p, _i32, _i32, _i32, _f32,
                                            ctypes.c_uint64, ctypes.c_int, _c_void_p]),
    "avits_noise_bits": (ctypes.c_int, [_i64, _i64, _i64, ctypes.c_uint64, _c_void_p, _c_void_p]),
    "avits_grid_positions": (ctypes.c_int, [_c_void_p, _i64, _i32, _i32, _i32, _i32, _c_void_p]),
    "avits_scale_positions": (ctypes.c_int, [_c_void_p, _i64, _i32, _c_void_p, _c_void_p]),
    "avits_block_forward_batched": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _f32, _i32, _c_void_p, _c_void_p,
                                                   ctypes.POINTER(_BlockWeights), _i32, _i32, ctypes.c_int,
                                                   _c_void_p, _c_void_p, _size, _c_void_p]),
    "avits_block_forward_batched_ex": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _f32, _i32, _c_void_p,
                                                      _c_void_p, ctypes.POINTER(_BlockWeights), _i64, _i32, _i32,
                                                      ctypes.c_int, _c_void_p, _c_void_p, _size, _c_void_p]),
    "avits_block_qk_workspace_bytes": (_size, [_i64, _i32, _i32, ctypes.c_int]),
    "avits_block_qk": (ctypes.c_int, [_c_void_p, _c_void_p, _f32, _i64, _i64, ctypes.POINTER(_BlockWeights), _i32, _i32,
                                      ctypes.c_int, _c_void_p, _c_void_p, _c_void_p, _size, _c_void_p]),
    "avits_gather_upsample_ln": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _i64, _i32, _i32, _i64,
                                                 _i64, ctypes.c_int, ctypes.c_int, _c_void_p, _c_void_p, _c_void_p,
                                                 _i64, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                                                 _c_void_p]),
    "avits_scatter": (ctypes.c_int, [_c_void_p, _c_void_p, _i64, _i64, _i64, _i64, ctypes.c_int, _c_void_p,
                                     _c_void_p]),
    "avits_linear": (ctypes.c_int, [_c_void_p, _i64, _i64, _c_void_p, _c_void_p, _i64, ctypes.c_int, _c_void_p,
                                    _c_void_p]),
    "avits_final_layer_workspace_bytes": (_size, [_i64, _i64, ctypes.c_int]),
    "avits_final_layer": (ctypes.c_int, [_c_void_p, _i64, _i64, _c_void_p, _c_void_p, _c_void_p, _i64, ctypes.c_int,
                                         _c_void_p, _c_void_p, _size, _c_void_p]),
    "avits_euler_update": (ctypes.c_int, [_c_void_p, _c_void_p, _i64, _f32, ctypes.c_int, _c_void_p]),
    "avits_gather_upsample_batched": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _i32,
                                                     _i32, _i32, _i64, _i64, ctypes.c_int, ctypes.c_int, _c_void_p,
                                                     _c_void_p, _c_void_p, _c_void_p, _c_void_p]),
    "avits_scatter_batched": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _i32, _c_void_p, _i64, _i64,
                                             ctypes.c_int, _c_void_p, _c_void_p]),
    "avits_gather_mixed": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _i64, _i32, _i32, _i64, _i64,
                                          ctypes.c_int, ctypes.c_int, _c_void_p, _c_void_p, _c_void_p, _c_void_p]),
    "avits_scatter_mixed": (ctypes.c_int, [_c_void_p, _c_void_p, _i64, _i32, _i32, _i64, _i64, ctypes.c_int,
                                           _c_void_p, _c_void_p, _c_void_p]),
    "avits_joint_lse": (ctypes.c_int, [_c_void_p, _c_void_p, _i64, _i64, _i32, _i32, ctypes.c_int, _c_void_p,
                                       _c_void_p]),
    "avits_joint_attention_stats": (ctypes.c_int, [_c_void_p, _c_void_p, _i64, _i64, _i64, _i32, _i32, ctypes.c_int,
                                                   _c_void_p, _c_void_p, ctypes.c_int, _c_void_p]),
    "avits_score_from_mass": (ctypes.c_int, [_c_void_p, _i64, _i32, _i32, ctypes.POINTER(_c_void_p), _i32, _i64, _i64,
                                             _f32, _f32,
                                             ctypes.c_int, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _size,
                                             _c_void_p]),
    "avits_timing_enable": (ctypes.c_int, [ctypes.c_int]),
    "avits_timing_reset": (None, []),
    "avits_timing_read": (ctypes.c_int, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                         ctypes.POINTER(_i64)]),
}

EXPORTS = tuple(_SIGS)


def lib_path() -> str:
    return os.path.join(_HERE, "libavits.so")


def load():
    """Load libavits.so (after torch, so both use torch's HIP runtime)."""
    global _LIB
    if _LIB is None:
        import torch  # noqa: F401  (binds libamdhip64 before the library is loaded)
        path = lib_path()
        if not os.path.exists(path):
            raise AvitsError(-2, f"{path} is missing; build it with `python -m paper_2608_17995_amd.build`")
        lib = ctypes.CDLL(path)
        for name, (res, args) in _SIGS.items():
            fn = getattr(lib, name)
            fn.restype, fn.argtypes = res, args
        _LIB = lib
    return _LIB


def version() -> str:
    return load().avits_version().decode()


def _check(rc: int):
    if rc != 0:
        raise AvitsError(rc, load().avits_last_error().decode())


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise AvitsError(-2, f"unsupported dtype {t.dtype}")


def _dev(t, name, dtype=None):
    """Device pointer of a contiguous GPU tensor (None passes NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise AvitsError(-1, f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise AvitsError(-1, f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise AvitsError(-1, f"{name} must be {dtype}, got {t.dtype}")
    return t.data_ptr()


def _stream(stream):
    import torch
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _workspace(ws, nbytes, device):
    import torch
    if ws is None:
        ws = torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)
    return ws, _dev(ws, "workspace"), ws.numel() * ws.element_size()


# ---------------------------------------------------------------------------

def avits_score_workspace_bytes(N: int, H: int) -> int:
    return load().avits_score_workspace_bytes(N, H)


def avits_score(latent_q, text_k, row_lse, feat_t, feat_prev, alpha, eps, scores,
                a_raw=None, v_raw=None, workspace=None, stream=None):
    import torch
    N, H, d = latent_q.shape
    L = text_k.shape[0]
    D_f = feat_t.shape[1]
    dt = latent_q.dtype
    ws, wsp, wsb = _workspace(workspace, avits_score_workspace_bytes(N, H), latent_q.device)
    _check(load().avits_score(
        _dev(latent_q, "latent_q"), _dev(text_k, "text_k", dt), _dev(row_lse, "row_lse", torch.float32),
        _dev(feat_t, "feat_t", dt), _dev(feat_prev, "feat_prev", dt), N, L, H, d, D_f, alpha, eps,
        _dtype_code(latent_q), _dev(scores, "scores", torch.float32), _dev(a_raw, "a_raw", torch.float32),
        _dev(v_raw, "v_raw", torch.float32), wsp, wsb, _stream(stream)))
    return scores


def avits_score_select(latent_q, text_k, row_lse, feat_t, feat_prev, alpha, eps, scores, k, idx,
                       a_raw=None, v_raw=None, workspace=None, stream=None):
    """avits_score then avits_select(scores, k, idx) in one call (N <= 16384)."""
    import torch
    N, H, d = latent_q.shape
    L = text_k.shape[0]
    D_f = feat_t.shape[1]
    dt = latent_q.dtype
    ws, wsp, wsb = _workspace(workspace, avits_score_workspace_bytes(N, H), latent_q.device)
    _check(load().avits_score_select(
        _dev(latent_q, "latent_q"), _dev(text_k, "text_k", dt), _dev(row_lse, "row_lse", torch.float32),
        _dev(feat_t, "feat_t", dt), _dev(feat_prev, "feat_prev", dt), N, L, H, d, D_f, alpha, eps,
        _dtype_code(latent_q), _dev(scores, "scores", torch.float32), _dev(a_raw, "a_raw", torch.float32),
        _dev(v_raw, "v_raw", torch.float32), k, _dev(idx, "idx", torch.int32) if k else None, wsp, wsb,
        _stream(stream)))
    return scores, idx


def avits_score_batched_workspace_bytes(B: int, N: int, H: int) -> int:
    return load().avits_score_batched_workspace_bytes(B, N, H)


def avits_score_batched(latent_q, text_k, row_lse, feat_t, feat_prev, alpha, eps, scores,
                        a_raw=None, v_raw=None, workspace=None, stream=None):
    """Stacked images: latent_q [B, N, H, d], text_k [B, L, H, d], row_lse
    [B, H, N], feat_t / feat_prev [B, N, D_f]; scores (and a_raw, v_raw)
    [B, N]."""
    import torch
    Bn, N, H, d = latent_q.shape
    L = text_k.shape[1]
    D_f = feat_t.shape[2]
    dt = latent_q.dtype
    if (tuple(text_k.shape) != (Bn, L, H, d) or tuple(row_lse.shape) != (Bn, H, N)
            or tuple(feat_t.shape) != (Bn, N, D_f) or tuple(feat_prev.shape) != (Bn, N, D_f)
            or tuple(scores.shape) != (Bn, N) or any(t is not None and t.numel() != Bn * N for t in (a_raw, v_raw))):
        raise ValueError("avits_score_batched: inputs must be stacked over the same B images of one shape")
    ws, wsp, wsb = _workspace(workspace, avits_score_batched_workspace_bytes(Bn, N, H), latent_q.device)
    _check(load().avits_score_batched(
        _dev(latent_q, "latent_q"), _dev(text_k, "text_k", dt), _dev(row_lse, "row_lse", torch.float32),
        _dev(feat_t, "feat_t", dt), _dev(feat_prev, "feat_prev", dt), Bn, N, L, H, d, D_f, alpha, eps,
        _dtype_code(latent_q), _dev(scores, "scores", torch.float32), _dev(a_raw, "a_raw", torch.float32),
        _dev(v_raw, "v_raw", torch.float32), wsp, wsb, _stream(stream)))
    return scores


def avits_select_workspace_bytes(N: int) -> int:
    return load().avits_select_workspace_bytes(N)


def avits_select(scores, k, idx, workspace=None, stream=None):
    import torch
    N = scores.shape[0]
    ws, wsp, wsb = _workspace(workspace, avits_select_workspace_bytes(N), scores.device)
    _check(load().avits_select(_dev(scores, "scores", torch.float32), N, k, _dev(idx, "idx", torch.int32),
                               wsp, wsb, _stream(stream)))
    return idx


def avits_select_noalloc_max_n() -> int:
    return load().avits_select_noalloc_max_n()


def avits_select_noalloc(scores, k, idx, stream=None):
    """avits_select without a workspace (the library's fixed device array)."""
    import torch
    _check(load().avits_select_noalloc(_dev(scores, "scores", torch.float32), scores.shape[0], k,
                                       _dev(idx, "idx", torch.int32), _stream(stream)))
    return idx


def avits_select_perturbed(scores, delta, k, idx, workspace=None, stream=None):
    import torch
    N = scores.shape[0]
    ws, wsp, wsb = _workspace(workspace, avits_select_workspace_bytes(N), scores.device)
    _check(load().avits_select_perturbed(_dev(scores, "scores", torch.float32), _dev(delta, "delta", torch.float32),
                                         N, k, _dev(idx, "idx", torch.int32), wsp, wsb, _stream(stream)))
    return idx


def avits_select_batched(scores, offsets, k, idx, delta=None, stream=None):
    """offsets, k: host sequences of ints (B + 1 and B); idx holds sum(k) entries."""
    import torch
    B = len(k)
    off = (ctypes.c_int64 * (B + 1))(*[int(o) for o in offsets])
    kk = (ctypes.c_int64 * B)(*[int(x) for x in k])
    _check(load().avits_select_batched(_dev(scores, "scores", torch.float32), _dev(delta, "delta", torch.float32),
                                       B, off, kk, _dev(idx, "idx", torch.int32), _stream(stream)))
    return idx


def avits_gather_upsample(lowres, highres_prev, prefix, idx, H_lr, W_lr, compact, pos_sel, canvas,
                          mode=UP_NEAREST, stream=None):
    import torch
    dt = lowres.dtype
    n_prefix = 0 if prefix is None else prefix.shape[0]
    _check(load().avits_gather_upsample(
        _dev(lowres, "lowres"), _dev(highres_prev, "highres_prev", dt),
        _dev(prefix, "prefix", dt) if n_prefix else None, _dev(idx, "idx", torch.int32), idx.shape[0],
        H_lr, W_lr, n_prefix, lowres.shape[1], mode, _dtype_code(lowres), _dev(compact, "compact", dt),
        _dev(pos_sel, "pos_sel", torch.int32), _dev(canvas, "canvas", dt), _stream(stream)))
    return compact, pos_sel, canvas


def avits_gather_upsample_ln(lowres, highres_prev, prefix, idx, H_lr, W_lr, compact, pos_sel, canvas, n_txt,
                             shift_txt, scale_txt, shift_img, scale_img, h_out, mode=UP_NEAREST, stream=None):
    """avits_gather_upsample plus h_out = LN(compact)(1 + scale) + shift per
    row (text-stream vectors for the first n_txt rows, image-stream after)."""
    import torch
    dt = lowres.dtype
    n_prefix = 0 if prefix is None else prefix.shape[0]
    _check(load().avits_gather_upsample_ln(
        _dev(lowres, "lowres"), _dev(highres_prev, "highres_prev", dt),
        _dev(prefix, "prefix", dt) if n_prefix else None, _dev(idx, "idx", torch.int32), idx.shape[0],
        H_lr, W_lr, n_prefix, lowres.shape[1], mode, _dtype_code(lowres), _dev(compact, "compact", dt),
        _dev(pos_sel, "pos_sel", torch.int32), _dev(canvas, "canvas", dt), n_txt, _dev(shift_txt, "shift_txt", dt),
        _dev(scale_txt, "scale_txt", dt), _dev(shift_img, "shift_img", dt), _dev(scale_img, "scale_img", dt),
        _dev(h_out, "h_out", dt), _stream(stream)))
    return compact, pos_sel, canvas, h_out


def avits_linear(x, w, b, out, stream=None):
    """out [M, N] = x [M, K] w[N, K]^T + b [N] (b may be None)."""
    M, K = x.shape
    N = w.shape[0]
    dt = x.dtype
    if tuple(w.shape) != (N, K) or tuple(out.shape) != (M, N) or (b is not None and b.numel() != N):
        raise ValueError("avits_linear: x [M, K], w [N, K], b [N], out [M, N]")
    _check(load().avits_linear(_dev(x, "x"), M, K, _dev(w, "w", dt), _dev(b, "b", dt), N, _dtype_code(x),
                               _dev(out, "out", dt), _stream(stream)))
    return out


def avits_final_layer_workspace_bytes(M: int, D: int, dtype: int) -> int:
    return load().avits_final_layer_workspace_bytes(M, D, dtype)


def avits_final_layer(x, mod, w, b, out, workspace=None, stream=None):
    """out [M, C] = (LN(x) (1 + mod[1]) + mod[0]) w^T + b; x [M, D], mod [2, D]."""
    M, D = x.shape
    C = w.shape[0]
    dt = x.dtype
    if tuple(mod.shape) != (2, D) or tuple(w.shape) != (C, D) or tuple(out.shape) != (M, C):
        raise ValueError("avits_final_layer: x [M, D], mod [2, D], w [C, D], out [M, C]")
    ws, wsp, wsb = _workspace(workspace, avits_final_layer_workspace_bytes(M, D, _dtype_code(x)), x.device)
    _check(load().avits_final_layer(_dev(x, "x"), M, D, _dev(mod, "mod", dt), _dev(w, "w", dt), _dev(b, "b", dt), C,
                                    _dtype_code(x), _dev(out, "out", dt), wsp, wsb, _stream(stream)))
    return out


def avits_euler_update(z, v, dt, stream=None):
    """z += dt * v in place (fp32 arithmetic, one rounding)."""
    if z.shape != v.shape:
        raise ValueError("avits_euler_update: z and v must have one shape")
    _check(load().avits_euler_update(_dev(z, "z"), _dev(v, "v", z.dtype), z.numel(), dt, _dtype_code(z),
                                     _stream(stream)))
    return z


def _host_i64(values, n, name):
    values = [int(v) for v in values]
    if len(values) != n:
        raise ValueError(f"{name}: {len(values)} entries, expected {n}")
    return (ctypes.c_int64 * n)(*values)


def avits_gather_upsample_batched(lowres, highres_prev, prefix, idx, idx_off, H_lr, W_lr, compact, row_off, pos,
                                  canvas, mode=UP_NEAREST, stream=None):
    """Stacked images: lowres [B, H_lr*W_lr, D], highres_prev / canvas
    [B, N, D], prefix [B, n_prefix, D] or None; idx the concatenated
    selections, idx_off (B + 1) and row_off (B) host sequences; pos is
    indexed like compact's rows."""
    import torch
    dt = lowres.dtype
    Bn, _, D = lowres.shape
    n_prefix = 0 if prefix is None else prefix.shape[1]
    if prefix is not None and (prefix.shape[0] != Bn or prefix.shape[2] != D):
        raise ValueError("avits_gather_upsample_batched: prefix must be [B, n_prefix, D]")
    if highres_prev.shape[0] != Bn or canvas.shape[0] != Bn:
        raise ValueError("avits_gather_upsample_batched: highres_prev and canvas must be stacked over B images")
    _check(load().avits_gather_upsample_batched(
        _dev(lowres, "lowres"), _dev(highres_prev, "highres_prev", dt),
        _dev(prefix, "prefix", dt) if n_prefix else None, _dev(idx, "idx", torch.int32),
        _host_i64(idx_off, Bn + 1, "idx_off"), Bn, H_lr, W_lr, n_prefix, D, mode, _dtype_code(lowres),
        _dev(compact, "compact", dt), _host_i64(row_off, Bn, "row_off"), _dev(pos, "pos", torch.int32),
        _dev(canvas, "canvas", dt), _stream(stream)))
    return compact, pos, canvas


def avits_scatter_batched(out, idx, idx_off, row_off, canvas, stream=None):
    """canvas [B, N, D]; idx the concatenated selections; idx_off (B + 1),
    row_off (B) host sequences."""
    import torch
    Bn, N, D = canvas.shape
    _check(load().avits_scatter_batched(
        _dev(out, "out", canvas.dtype), _dev(idx, "idx", torch.int32), _host_i64(idx_off, Bn + 1, "idx_off"), Bn,
        _host_i64(row_off, Bn, "row_off"), N, D, _dtype_code(canvas), _dev(canvas, "canvas"), _stream(stream)))
    return canvas


def avits_scatter(out, idx, row_offset, canvas, stream=None):
    import torch
    _check(load().avits_scatter(_dev(out, "out"), _dev(idx, "idx", torch.int32), idx.shape[0], row_offset,
                                out.shape[1], canvas.shape[0], _dtype_code(out), _dev(canvas, "canvas", out.dtype),
                                _stream(stream)))
    return canvas


def avits_gather_mixed(lowres, prefix, idx, H_lr, W_lr, compact, pos, children=None, mode=UP_NEAREST,
                       stream=None):
    import torch
    dt = lowres.dtype
    n_prefix = 0 if prefix is None else prefix.shape[0]
    k = 0 if idx is None else idx.shape[0]
    _check(load().avits_gather_mixed(
        _dev(lowres, "lowres"), _dev(prefix, "prefix", dt) if n_prefix else None,
        _dev(idx, "idx", torch.int32) if k else None, k, H_lr, W_lr, n_prefix, lowres.shape[1], mode,
        _dtype_code(lowres), _dev(compact, "compact", dt), _dev(pos, "pos", torch.int32),
        _dev(children, "children", torch.int32), _stream(stream)))
    return compact, pos, children


def avits_scatter_mixed(out, idx, H_lr, W_lr, row_offset, canvas_hr, state_lr, stream=None):
    import torch
    dt = out.dtype
    k = 0 if idx is None else idx.shape[0]
    _check(load().avits_scatter_mixed(
        _dev(out, "out"), _dev(idx, "idx", torch.int32) if k else None, k, H_lr, W_lr, row_offset, out.shape[1],
        _dtype_code(out), _dev(canvas_hr, "canvas_hr", dt), _dev(state_lr, "state_lr", dt), _stream(stream)))
    return canvas_hr, state_lr


def avits_joint_lse(q, k_all, lse, stream=None):
    import torch
    N, H, d = q.shape
    _check(load().avits_joint_lse(_dev(q, "q"), _dev(k_all, "k_all", q.dtype), N, k_all.shape[0], H, d,
                                  _dtype_code(q), _dev(lse, "lse", torch.float32), _stream(stream)))
    return lse


class BlockWeights:
    """Device weights of one block, packed into the C struct (keeps the tensors alive)."""

    def __init__(self, kind: int, txt: dict | None = None, img: dict | None = None, single: dict | None = None):
        self.kind = kind
        self.tensors = {"txt": txt or {}, "img": img or {}, "single": single or {}}
        self.c = _BlockWeights()
        self.c.kind = kind
        if kind == BLOCK_DOUBLE:
            ref = (txt or img)
            self.c.mlp_hidden = ref["w_mlp1"].shape[0]
            for part, w in (("txt", txt), ("img", img)):
                if w:
                    cs = getattr(self.c, part)
                    for name, _ in _DoubleStream._fields_:
                        setattr(cs, name, _dev(w[name], f"{part}.{name}"))
        else:
            D = single["w_out"].shape[0]
            self.c.mlp_hidden = single["w_out"].shape[1] - D
            for name, _ in _Single._fields_:
                setattr(self.c.single, name, _dev(single[name], f"single.{name}"))


def avits_timing_enable(on: bool = True):
    _check(load().avits_timing_enable(1 if on else 0))


def avits_timing_reset():
    load().avits_timing_reset()


def avits_timing_read(family: str):
    """(total milliseconds, launches) recorded for one launch family."""
    ms, n = ctypes.c_double(), _i64()
    _check(load().avits_timing_read(family.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def avits_block_workspace_bytes(kind: int, S: int, H: int, d: int, mlp_hidden: int, dtype: int) -> int:
    return load().avits_block_workspace_bytes(kind, S, H, d, mlp_hidden, dtype)


def avits_block_forward(x_in, x_out, pos, n_txt, n_img, weights: BlockWeights, H, lse_out=None,
                        workspace=None, stream=None, pos_scale=1.0):
    import torch
    S, D = x_in.shape
    d = D // H
    code = _dtype_code(x_in)
    ws, wsp, wsb = _workspace(
        workspace, avits_block_workspace_bytes(weights.kind, S, H, d, weights.c.mlp_hidden, code), x_in.device)
    _check(load().avits_block_forward(
        _dev(x_in, "x_in"), _dev(x_out, "x_out", x_in.dtype), _dev(pos, "pos", torch.int32), pos_scale, n_txt, n_img,
        ctypes.byref(weights.c), H, d, code, _dev(lse_out, "lse_out", torch.float32), wsp, wsb, _stream(stream)))
    return x_out


def avits_block_forward_ex(x_in, x_out, pos, n_txt, n_img, weights: BlockWeights, H, lse_out=None, mass_out=None,
                           mass_accumulate=False, workspace=None, stream=None, pos_scale=1.0, scatter_idx=None,
                           canvas=None, h_in=None, h_next=None, next_weights=None):
    """avits_block_forward with the joint attention's statistics: lse_out and
    mass_out [H, S] fp32 (the softmax mass of each row on the text keys
    [0, n_txt), added to mass_out's contents when mass_accumulate); with
    scatter_idx [k] and canvas, the last k image rows' outputs also go to
    canvas[scatter_idx] (the fused Stage-3 scatter); with h_in [S, D], the
    first modulated layer norm comes precomputed (avits_gather_upsample_ln
    or the previous block's h_next); with h_next [S, D] and next_weights,
    the next block's first stage is written from this block's output."""
    import torch
    S, D = x_in.shape
    d = D // H
    code = _dtype_code(x_in)
    ws, wsp, wsb = _workspace(
        workspace, avits_block_workspace_bytes(weights.kind, S, H, d, weights.c.mlp_hidden, code), x_in.device)
    k = 0 if scatter_idx is None else scatter_idx.shape[0]
    outs = _BlockOutputs(_dev(lse_out, "lse_out", torch.float32), _dev(mass_out, "mass_out", torch.float32),
                         1 if mass_accumulate else 0, _dev(scatter_idx, "scatter_idx", torch.int32) if k else None, k,
                         _dev(canvas, "canvas", x_in.dtype) if canvas is not None else None,
                         canvas.shape[0] if canvas is not None else 0,
                         _dev(h_in, "h_in", x_in.dtype) if h_in is not None else None,
                         _dev(h_next, "h_next", x_in.dtype) if h_next is not None else None,
                         ctypes.addressof(next_weights.c) if next_weights is not None else None)
    _check(load().avits_block_forward_ex(
        _dev(x_in, "x_in"), _dev(x_out, "x_out", x_in.dtype), _dev(pos, "pos", torch.int32), pos_scale, n_txt, n_img,
        ctypes.byref(weights.c), H, d, code, ctypes.byref(outs), wsp, wsb, _stream(stream)))
    return x_out


def avits_grid_positions(pos, W, frame=0, scale=1, offset=0, stream=None):
    """pos [rows, 3] int32 <- (frame, (r / W) scale + offset, (r % W) scale + offset)."""
    import torch
    _check(load().avits_grid_positions(_dev(pos, "pos", torch.int32), pos.shape[0], W, frame, scale, offset,
                                       _stream(stream)))
    return pos


def avits_scale_positions(src, scale, dst, stream=None):
    """dst [rows, 3] int32 <- src * scale."""
    import torch
    _check(load().avits_scale_positions(_dev(src, "src", torch.int32), src.shape[0], scale,
                                        _dev(dst, "dst", torch.int32), _stream(stream)))
    return dst


NOISE_RASTER, NOISE_HALF_UNITS, NOISE_LOWRES = 0, 1, 2


def avits_noise_reinject(x, t, seed, H_hr, W_hr, pos=None, rows_kind=None, stream=None):
    """x [rows, C] <- (1 - t) x + t eps at the rows' coordinates: raster
    high-res rows (default), half-unit positions pos [rows, 3] (rows_kind
    NOISE_HALF_UNITS, the default when pos is given) or raster low-res rows
    (NOISE_LOWRES)."""
    import torch
    rows, C = x.shape
    if rows_kind is None:
        rows_kind = NOISE_RASTER if pos is None else NOISE_HALF_UNITS
    _check(load().avits_noise_reinject(_dev(x, "x"), rows, C, _dev(pos, "pos", torch.int32), rows_kind, H_hr, W_hr,
                                       float(t), int(seed), _dtype_code(x), _stream(stream)))
    return x


def avits_noise_bits(first_pixel, bits, seed, stream=None):
    """bits [n_pixels, C] uint32 (a torch int32 tensor): the generator's words."""
    import torch
    n, C = bits.shape
    _check(load().avits_noise_bits(first_pixel, n, C, int(seed), _dev(bits, "bits", torch.int32), _stream(stream)))
    return bits


def avits_block_qk_workspace_bytes(S: int, H: int, d: int, dtype: int) -> int:
    return load().avits_block_qk_workspace_bytes(S, H, d, dtype)


def avits_block_forward_batched(x_in, x_out, pos, txt_off, img_off, weights: BlockWeights, H, lse_out=None,
                                workspace=None, stream=None, pos_scale=1.0):
    """txt_off, img_off: host sequences of B + 1 ints (rows packed by stream)."""
    import torch
    S, D = x_in.shape
    d = D // H
    B = len(txt_off) - 1
    code = _dtype_code(x_in)
    ws, wsp, wsb = _workspace(workspace, avits_block_workspace_bytes(weights.kind, S, H, d, weights.c.mlp_hidden,
                                                                     code), x_in.device)
    to = (ctypes.c_int64 * (B + 1))(*[int(v) for v in txt_off])
    io = (ctypes.c_int64 * (B + 1))(*[int(v) for v in img_off])
    _check(load().avits_block_forward_batched(
        _dev(x_in, "x_in"), _dev(x_out, "x_out", x_in.dtype), _dev(pos, "pos", torch.int32), pos_scale, B, to, io,
        ctypes.byref(weights.c), H, d, code, _dev(lse_out, "lse_out", torch.float32), wsp, wsb, _stream(stream)))
    return x_out


def avits_block_forward_batched_ex(x_in, x_out, pos, txt_off, img_off, weights: BlockWeights, H, mod_stride: int,
                                   lse_out=None, workspace=None, stream=None, pos_scale=1.0):
    """avits_block_forward_batched with image b's modulation rows at the
    stream's mod + b * mod_stride elements (0: one set for all images)."""
    import torch
    S, D = x_in.shape
    d = D // H
    B = len(txt_off) - 1
    code = _dtype_code(x_in)
    ws, wsp, wsb = _workspace(workspace, avits_block_workspace_bytes(weights.kind, S, H, d, weights.c.mlp_hidden,
                                                                     code), x_in.device)
    to = (ctypes.c_int64 * (B + 1))(*[int(v) for v in txt_off])
    io = (ctypes.c_int64 * (B + 1))(*[int(v) for v in img_off])
    _check(load().avits_block_forward_batched_ex(
        _dev(x_in, "x_in"), _dev(x_out, "x_out", x_in.dtype), _dev(pos, "pos", torch.int32), pos_scale, B, to, io,
        ctypes.byref(weights.c), int(mod_stride), H, d, code, _dev(lse_out, "lse_out", torch.float32), wsp, wsb,
        _stream(stream)))
    return x_out


def avits_block_qk(x_in, pos, n_txt, n_img, weights: BlockWeights, H, q_out, k_out, workspace=None, stream=None,
                   pos_scale=1.0):
    """q_out, k_out [S, D] (or [S, H, d]): the block's normalised, rotated queries and keys."""
    import torch
    S, D = x_in.shape
    d = D // H
    code = _dtype_code(x_in)
    ws, wsp, wsb = _workspace(workspace, avits_block_qk_workspace_bytes(S, H, d, code), x_in.device)
    _check(load().avits_block_qk(
        _dev(x_in, "x_in"), _dev(pos, "pos", torch.int32), pos_scale, n_txt, n_img, ctypes.byref(weights.c), H, d, code,
        _dev(q_out, "q_out", x_in.dtype), _dev(k_out, "k_out", x_in.dtype), wsp, wsb, _stream(stream)))
    return q_out, k_out


def avits_joint_attention_stats(q, k_all, L, mass, lse=None, accumulate=False, stream=None):
    """q [N, H, d], k_all [Nk, H, d] (text keys first); mass [H, N] fp32 (added to when accumulate)."""
    import torch
    N, H, d = q.shape
    _check(load().avits_joint_attention_stats(
        _dev(q, "q"), _dev(k_all, "k_all", q.dtype), N, k_all.shape[0], L, H, d, _dtype_code(q),
        _dev(lse, "lse", torch.float32), _dev(mass, "mass", torch.float32), 1 if accumulate else 0, _stream(stream)))
    return mass


def avits_score_from_mass(mass, count, snapshots, alpha, eps, scores, a_raw=None, v_raw=None, workspace=None,
                          stream=None):
    """mass [H, N] fp32 (sum of `count` probes; rows may be strided, e.g.
    the image columns mass_all[:, L:] of a block's [H, S] mass); snapshots:
    N_T tensors [N, D_f], consecutive steps in order."""
    import torch
    H, N = mass.shape
    if mass.dtype != torch.float32 or not mass.is_cuda or mass.stride(1) != 1 or mass.stride(0) < N:
        raise AvitsError(-1, "mass must be a float32 GPU tensor [H, N] with unit column stride")
    snaps = list(snapshots)
    n_t = len(snaps)
    Df = snaps[0].shape[-1]
    for z in snaps:
        if tuple(z.shape) != (N, Df) or z.dtype != snaps[0].dtype:
            raise AvitsError(-1, "snapshots must all be [N, D_f] of one dtype")
    ptrs = (_c_void_p * n_t)(*[_dev(z, "snapshot") for z in snaps])
    ws, wsp, wsb = _workspace(workspace, avits_score_workspace_bytes(N, H), mass.device)
    _check(load().avits_score_from_mass(
        mass.data_ptr(), mass.stride(0), H, count, ptrs, n_t, N, Df, alpha, eps, _dtype_code(snaps[0]),
        _dev(scores, "scores", torch.float32), _dev(a_raw, "a_raw", torch.float32), _dev(v_raw, "v_raw", torch.float32),
        wsp, wsb, _stream(stream)))
    return scores
