"""HSA active-token layer step for AMD MI355X (gfx950).

The computation lives in the HIP library libhsa_step.so (C ABI declared in
include/hsa_step.h); `hsa_step` is its ctypes binding and `layer` strings the
calls together into one HSA iteration on caller-owned device buffers.
"""

__all__ = ["hsa_step", "layer"]
