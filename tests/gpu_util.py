"""Helpers shared by the GPU parity tests: device transfer and error metrics."""

import numpy as np
import torch

import synth

DEV = "cuda"


def rel_inf(a, b) -> float:
    """max |a - b| / max |b| over a whole tensor (infinity-norm relative error)."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.max(np.abs(b)) if b.size else 0.0
    if den == 0.0:
        return float(np.max(np.abs(a - b))) if a.size else 0.0
    return float(np.max(np.abs(a - b)) / den)


def to_dev(a, dtype: str) -> torch.Tensor:
    if dtype == "bf16":
        return synth.bf16_tensor(np.asarray(a, np.float32)).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(DEV)


def i32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(DEV)


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def host_bits(t: torch.Tensor) -> np.ndarray:
    """Raw bit patterns, for bit-for-bit comparisons."""
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy()
    if t.dtype == torch.float32:
        return t.view(torch.int32).numpy()
    return t.numpy()


def torch_dtype(dtype: str):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


TOL = {"bf16": 2e-2, "f32": 1e-4}
