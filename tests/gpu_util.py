"""Helpers shared by the GPU tests: moving stored arrays to the device and back,
and the error measure used for parity."""
from __future__ import annotations

import numpy as np

import oracle

TOL = {"f32": 1e-5, "f16": 2e-2, "bf16": 2e-2}


def torch_dtype(dtype: str):
    import torch

    return {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[dtype]


def to_dev(a: np.ndarray, dtype: str | None = None, device="cuda"):
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype == "bf16":
        t = t.view(torch.bfloat16)
    return t.to(device)


def to_host64(t, dtype: str) -> np.ndarray:
    import torch

    if dtype == "bf16":
        return oracle.widen(t.view(torch.int16).cpu().numpy().view(np.uint16), "bf16")
    return t.cpu().numpy().astype(np.float64)


def rel_err_per_head(x: np.ndarray, ref: np.ndarray, floor: float, rows=None) -> float:
    """max over heads of max|x - ref| / max(max|ref|, floor), over the given rows."""
    if rows is not None:
        x, ref = x[rows], ref[rows]
    if x.size == 0:
        return 0.0
    worst = 0.0
    for h in range(x.shape[1]):
        dif = np.abs(x[:, h] - ref[:, h])
        if not np.all(np.isfinite(x[:, h])):
            return float("inf")
        scale = max(float(np.abs(ref[:, h]).max()), floor)
        worst = max(worst, float(dif.max()) / scale)
    return worst


def p999(x, ref):
    """99.9th percentile of |x - ref| / (|ref| + rms(ref))."""
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 1.0
    return float(np.percentile(np.abs(x - ref) / (np.abs(ref) + rms), 99.9)) if ref.size else 0.0
