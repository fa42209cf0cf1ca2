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


GUARD_BYTES = 64 << 10  # red zone before and after a guarded tensor


class Guarded:
    """A device tensor between two red zones of GUARD_BYTES bytes that hold a
    seeded byte pattern. `t` is the tensor to pass to the library (256-byte
    aligned, contiguous); check() fails if any byte of either red zone changed,
    i.e. if a kernel wrote outside the buffer it was given."""

    def __init__(self, shape, dtype, seed=0):
        es = torch.empty((), dtype=dtype).element_size()
        n = int(np.prod(shape)) * es
        n_pad = (n + 255) // 256 * 256
        self.raw = torch.empty(2 * GUARD_BYTES + n_pad, dtype=torch.uint8, device=DEV)
        g = torch.Generator(device="cpu").manual_seed(seed)
        self.pattern = torch.randint(0, 256, (GUARD_BYTES,), dtype=torch.uint8, generator=g).to(DEV)
        self.raw[:GUARD_BYTES] = self.pattern
        self.raw[GUARD_BYTES + n_pad:] = self.pattern
        self.n_pad = n_pad
        self.t = self.raw[GUARD_BYTES:GUARD_BYTES + n].view(dtype).view(*shape)

    def check(self, name=""):
        before = self.raw[:GUARD_BYTES]
        after = self.raw[GUARD_BYTES + self.n_pad:]
        assert torch.equal(before, self.pattern), f"write before the start of {name}"
        assert torch.equal(after, self.pattern), f"write past the end of {name}"
