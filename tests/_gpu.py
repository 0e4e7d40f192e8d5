"""Helpers shared by the GPU parity tests: host<->device conversion, tolerances."""
from __future__ import annotations

import numpy as np
import torch

TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def dev(a, dtype: str | None = None):
    """numpy -> cuda tensor; floats take the workload storage type (exact for generator data)."""
    a = np.ascontiguousarray(a)
    if a.dtype.kind in "iu":
        return torch.from_numpy(a.astype(np.int32)).cuda()
    t = torch.from_numpy(a.astype(np.float32))
    return t.to(TORCH_DT[dtype] if dtype else torch.float32).cuda()


def host(t):
    t = t.detach()
    if t.dtype in (torch.int32, torch.int64):
        return t.cpu().numpy()
    return t.float().cpu().numpy().astype(np.float64)


def rel_l2(x, ref):
    x, ref = np.asarray(x, np.float64), np.asarray(ref, np.float64)
    return float(np.linalg.norm(x - ref) / max(np.linalg.norm(ref), 1e-300))


def assert_close(x, ref, dtype: str, what: str, fp32_atol: float = 1e-4, bf16_rel: float = 1e-2):
    """The parity bar: max-abs <= 1e-4 for fp32 workloads, rel-L2 <= 1e-2 for bf16 ones."""
    x, ref = np.asarray(x, np.float64), np.asarray(ref, np.float64)
    assert x.shape == ref.shape, (what, x.shape, ref.shape)
    assert np.all(np.isfinite(x)), f"{what}: non-finite GPU values"
    if dtype == "f32":
        err = float(np.abs(x - ref).max()) if x.size else 0.0
        assert err <= fp32_atol, f"{what}: max-abs {err:.3e} > {fp32_atol}"
        return err
    err = rel_l2(x, ref)
    assert err <= bf16_rel, f"{what}: rel-L2 {err:.3e} > {bf16_rel}"
    return err


def double_weights_dev(w: dict, dtype: str) -> dict:
    return {k: dev(v, dtype) for k, v in w.items()}
