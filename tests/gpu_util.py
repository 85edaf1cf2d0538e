"""Helpers shared by the GPU parity tests (no method arithmetic here)."""
import numpy as np

TOL = {"f32": 1e-4, "bf16": 2e-2}


def rel_err(got, ref) -> float:
    """Per-tensor max relative error: max|a - b| / max|b| (norm-wise, safe near 0)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    denom = np.abs(ref).max()
    if denom == 0:
        return float(np.abs(got).max())
    return float(np.abs(got - ref).max() / denom)


def torch_dtype(prec):
    import torch
    return torch.float32 if prec == "f32" else torch.bfloat16


def to_dev(a, prec=None):
    """numpy -> GPU tensor (activations in the path's dtype, RNE rounding)."""
    import torch
    t = torch.tensor(np.ascontiguousarray(a, dtype=np.float32), device="cuda")
    if prec == "bf16":
        t = t.to(torch.bfloat16)
    return t


def as_np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def rounded(a, prec):
    """The values the GPU actually sees for `a` (bf16 rounding when prec == 'bf16')."""
    import torch
    t = torch.tensor(np.ascontiguousarray(a, dtype=np.float32))
    if prec == "bf16":
        t = t.to(torch.bfloat16)
    return t.float().numpy().astype(np.float64)
