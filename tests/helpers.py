"""Shared test utilities: moving synthetic tensors to the GPU and error norms."""

from __future__ import annotations

import numpy as np

import synth

# Parity bars (relative Frobenius error against the fp64 oracle on the same
# inputs): fp32 operands, and bf16 operands with fp32 accumulation.
TOL_F32 = 1e-5
TOL_BF16 = 2e-3


def rel_fro(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    num = np.linalg.norm(got - ref)
    return float(num / den) if den > 0 else float(num)


def to_dev(t: synth.Tensor, device="cuda"):
    import torch
    if t.dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(t.raw)).to(device)
    return torch.from_numpy(np.ascontiguousarray(t.raw).view(np.int16)).view(torch.bfloat16).to(device)


def to_host(x) -> np.ndarray:
    import torch
    return x.detach().to(torch.float64).cpu().numpy()


def types_dev(t: np.ndarray, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(t, dtype=np.int32)).to(device)


def f32_dev(a: np.ndarray, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
