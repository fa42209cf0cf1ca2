"""The allocation-free attention entry point against hsa_active_attention.

hsa_active_attention_noalloc takes its workspace from the library's fixed
device array; with the same key-part split it must give exactly the output of
hsa_active_attention with a caller workspace. Two calls in a row on the same
GPU, the second with a smaller input (the array keeps the first call's
contents), then a call beyond the array's limit, which must be refused before
anything is enqueued.
"""

import numpy as np
import pytest
import torch

from gpu_util import DEV, host_bits, i32

H = pytest.importorskip("paper_2605_06892_amd.hsa_step")

pytestmark = pytest.mark.gpu


DT = {"bf16": torch.bfloat16, "f32": torch.float32}


def _case(N, heads, dh, n_active, seed, dtype="bf16"):
    def to_dev(a, _tag):
        return torch.from_numpy(a).to(DEV).to(DT[dtype])

    rng = np.random.default_rng(seed)
    d = heads * dh
    idx = np.sort(rng.choice(N, size=n_active, replace=False)).astype(np.int32)
    t = {
        "q": to_dev(rng.standard_normal((n_active, d), dtype=np.float32), "bf16"),
        "k": to_dev(rng.standard_normal((N, d), dtype=np.float32), "bf16"),
        "v": to_dev(rng.standard_normal((N, d), dtype=np.float32), "bf16"),
        "wo": to_dev(rng.standard_normal((d, d), dtype=np.float32) / np.float32(np.sqrt(d)), "bf16"),
        "out0": to_dev(rng.standard_normal((N, d), dtype=np.float32), "bf16"),
        "idx": i32(idx),
    }
    return t


def _both(t, heads, dh):
    n_active = t["q"].shape[0]
    scale = 1.0 / np.sqrt(dh)
    # the caller-workspace entry point, with room for every key-part split (as the fixed array has)
    nb = H.hsa_attention_parts_workspace_bytes(t["q"].dtype, n_active, heads, dh)
    ws = torch.empty(nb, dtype=torch.uint8, device=DEV)
    out_a = t["out0"].clone()
    H.hsa_active_attention(t["q"], t["k"], t["v"], t["idx"], n_active, heads, dh, scale, t["wo"], out_a, ws)
    out_b = t["out0"].clone()
    H.hsa_active_attention_noalloc(t["q"], t["k"], t["v"], t["idx"], n_active, heads, dh, scale, t["wo"], out_b)
    torch.cuda.synchronize()
    return out_a, out_b


@pytest.mark.parametrize("shape", [(4096, 8, 128, 1500, 300, "bf16"), (3000, 2, 64, 900, 77, "bf16"),
                                   (2000, 4, 64, 700, 50, "f32")], ids=str)
def test_noalloc_equals_workspace_entry_point(shape):
    N, heads, dh, n1, n2, dtype = shape
    for n_active, seed in ((n1, 1), (n2, 2)):  # two calls in a row, the second smaller
        print(f"noalloc attention {dtype} N={N} heads={heads} dh={dh} n_active={n_active}", flush=True)
        t = _case(N, heads, dh, n_active, seed + N, dtype)
        out_a, out_b = _both(t, heads, dh)
        np.testing.assert_array_equal(host_bits(out_b), host_bits(out_a))
        # rows outside the active set untouched
        skipped = np.setdiff1d(np.arange(N), t["idx"].cpu().numpy())
        np.testing.assert_array_equal(host_bits(out_b)[skipped], host_bits(t["out0"])[skipped])


def test_noalloc_rejects_beyond_its_array():
    heads, dh = 40, 128
    d = heads * dh
    limit = H.lib().hsa_attention_workspace_bytes(H.BF16, 1, d)
    n_max = (96 << 20) // limit
    assert n_max == 9830
    t = _case(64, 2, 64, 8, 3)  # small real buffers; the call must not read them
    out = t["out0"].clone()
    with pytest.raises(H.HsaStepError) as ei:
        st = H.lib().hsa_active_attention_noalloc(H.BF16, t["q"].data_ptr(), t["k"].data_ptr(), t["v"].data_ptr(),
                                                  t["idx"].data_ptr(), n_max + 1, n_max + 1, heads, dh, 0.088,
                                                  t["wo"].data_ptr(), out.data_ptr(), None)
        H._check("hsa_active_attention_noalloc", st)
    assert ei.value.name == "HSA_STEP_ERR_WORKSPACE"
    torch.cuda.synchronize()
    assert torch.equal(out, t["out0"])
