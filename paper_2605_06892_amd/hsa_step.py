"""Python binding of libhsa_step.so (include/hsa_step.h), via ctypes.

Argument marshalling only: every function takes torch tensors (device memory
from PyTorch-ROCm) and scalars, passes raw pointers and the current HIP stream
to the C entry point of the same name, and raises HsaStepError on a non-zero
status. No computation happens here; there is no fallback path. Importing this
module fails if the HIP library has not been built.
"""

from __future__ import annotations

import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhsa_step.so")

F32 = 0
BF16 = 1

_STATUS = {
    0: "HSA_STEP_OK",
    1: "HSA_STEP_ERR_NULL",
    2: "HSA_STEP_ERR_SHAPE",
    3: "HSA_STEP_ERR_BUDGET",
    4: "HSA_STEP_ERR_DTYPE",
    5: "HSA_STEP_ERR_ALIAS",
    6: "HSA_STEP_ERR_WORKSPACE",
    7: "HSA_STEP_ERR_LAUNCH",
}


class HsaStepError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        self.name = _STATUS.get(status, str(status))
        super().__init__(f"{fn}: {self.name} ({lib().hsa_step_status_string(status).decode()})")


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library. Raises ImportError if it was never built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise ImportError(f"{_LIB_PATH} is missing: build it with `python -m paper_2605_06892_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        P, I32, I64, F, S = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
        sig = {
            "hsa_step_status_string": (ctypes.c_char_p, [ctypes.c_int]),
            "hsa_build_active_set": (ctypes.c_int, [P, I64, I32, I32, I32, P, P, P, P]),
            "hsa_build_active_set_window": (ctypes.c_int, [P, I64, I32, I32, I32, I32, P, P, P, P]),
            "hsa_window_margin": (I32, [I32, I32]),
            "hsa_qkv_scatter": (ctypes.c_int, [ctypes.c_int, P, I32, P, I32, I64, I32, P, P, P, P, P, P, P]),
            "hsa_attention_core": (ctypes.c_int, [ctypes.c_int, P, P, P, I32, I64, I32, I32, F, P, P]),
            "hsa_attention_core_parts": (ctypes.c_int, [ctypes.c_int, P, P, P, I32, I64, I32, I32, F, P, P, S, P]),
            "hsa_out_scatter": (ctypes.c_int, [ctypes.c_int, P, P, I32, I64, I32, P, P, P]),
            "hsa_attention_workspace_bytes": (S, [ctypes.c_int, I32, I32]),
            "hsa_attention_parts_workspace_bytes": (S, [ctypes.c_int, I32, I32, I32]),
            "hsa_active_attention": (ctypes.c_int, [ctypes.c_int, P, P, P, P, I32, I64, I32, I32, F, P, P, P, S, P]),
            "hsa_active_attention_noalloc": (ctypes.c_int, [ctypes.c_int, P, P, P, P, I32, I64, I32, I32, F, P, P, P]),
            "hsa_cached_euler": (ctypes.c_int, [P, P, P, P, I32, I64, I32, F, F, P]),
            "hsa_gather_rows": (ctypes.c_int, [ctypes.c_int, P, P, I32, I64, I32, P, P]),
            "hsa_row_rms_scale": (ctypes.c_int, [ctypes.c_int, P, I32, I32, F, P, P]),
            "hsa_linear": (ctypes.c_int, [ctypes.c_int, P, I32, I32, P, I32, P, P, I32, ctypes.c_int, P, P]),
            "hsa_l1_rel_accumulate": (ctypes.c_int, [P, P, I64, I32, P, I32, P]),
            "hsa_rope_table_floats": (S, [I32, I32, I32, I32]),
            "hsa_reorder_plan": (ctypes.c_int, [P, I64, I32, P, P, P, P]),
            "hsa_permute_rows": (ctypes.c_int, [P, P, I64, I64, I32, P, P]),
            "hsa_rope_table": (ctypes.c_int, [F, I32, I32, I32, I32, P]),
            "hsa_assign_budgets_by_key": (ctypes.c_int, [P, I64, I32, P, P, I32, P, P]),
            "hsa_assign_budgets_workspace_bytes": (S, [I64]),
            "hsa_assign_budgets": (ctypes.c_int, [P, I64, I32, I32, P, P, I32, P, P, S, P]),
            "hsa_stack_iteration": (ctypes.c_int, [ctypes.POINTER(HsaStack), I32, I32, I32, I32, F, F, P, P,
                                                   I32, I32, P, P, P]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


EXPORTED = (
    "hsa_step_status_string",
    "hsa_build_active_set",
    "hsa_build_active_set_window",
    "hsa_window_margin",
    "hsa_qkv_scatter",
    "hsa_attention_core",
    "hsa_attention_core_parts",
    "hsa_out_scatter",
    "hsa_attention_workspace_bytes",
    "hsa_attention_parts_workspace_bytes",
    "hsa_active_attention",
    "hsa_active_attention_noalloc",
    "hsa_cached_euler",
    "hsa_gather_rows",
    "hsa_row_rms_scale",
    "hsa_linear",
    "hsa_assign_budgets_workspace_bytes",
    "hsa_assign_budgets",
    "hsa_l1_rel_accumulate",
    "hsa_assign_budgets_by_key",
    "hsa_rope_table_floats",
    "hsa_rope_table",
    "hsa_reorder_plan",
    "hsa_permute_rows",
    "hsa_stack_iteration",
)

SELECT_VELOCITY_NORM = 0
SELECT_L1_REL = 1


class HsaStack(ctypes.Structure):
    """struct hsa_stack of include/hsa_step.h."""

    _fields_ = [
        ("dtype", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("channels", ctypes.c_int32), ("reserved", ctypes.c_int32),
        ("n_tokens", ctypes.c_int64),
        ("w_embed", ctypes.c_void_p), ("w_head", ctypes.c_void_p),
        ("w_layers", ctypes.POINTER(ctypes.c_void_p)), ("caches", ctypes.POINTER(ctypes.c_void_p)),
        ("x", ctypes.c_void_p), ("v_hat", ctypes.c_void_p), ("budget", ctypes.c_void_p),
        ("idx", ctypes.c_void_p), ("n_active", ctypes.c_void_p), ("xa", ctypes.c_void_p),
        ("h", ctypes.c_void_p), ("q", ctypes.c_void_p), ("o", ctypes.c_void_p),
        ("v_fresh", ctypes.c_void_p), ("keys", ctypes.c_void_p), ("row_scale", ctypes.c_void_p),
        ("ffn_dim", ctypes.c_int32), ("ctx_len", ctypes.c_int32),
        ("w_cross", ctypes.POINTER(ctypes.c_void_p)), ("w_ffn", ctypes.POINTER(ctypes.c_void_p)),
        ("f", ctypes.c_void_p), ("v_prev", ctypes.c_void_p),
        ("rope_cs", ctypes.c_void_p), ("pos", ctypes.c_void_p),
        ("grid_f", ctypes.c_int32), ("grid_h", ctypes.c_int32), ("grid_w", ctypes.c_int32),
        ("reserved2", ctypes.c_int32),
        ("prefix_cache", ctypes.c_int32), ("reserved3", ctypes.c_int32), ("n_cached", ctypes.c_int64),
        ("k_tail", ctypes.c_void_p), ("v_tail", ctypes.c_void_p),
        ("attn_parts", ctypes.c_void_p), ("attn_parts_bytes", ctypes.c_int64),
    ]


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dtype(*ts) -> int:
    dts = {t.dtype for t in ts if t is not None}
    if len(dts) != 1:
        raise TypeError(f"tensors must share one dtype, got {dts}")
    dt = dts.pop()
    if dt == torch.bfloat16:
        return BF16
    if dt == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {dt}")


def _check(fn: str, st: int) -> None:
    if st != 0:
        raise HsaStepError(fn, st)


def _dev(*ts) -> None:
    for t in ts:
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise ValueError("tensors must be contiguous device tensors")


def hsa_window_margin(center_percent: int, T: int) -> int:
    """Margin of a caching window over the centre center_percent% of T steps."""
    m = lib().hsa_window_margin(int(center_percent), int(T))
    if m < 0:
        raise ValueError(f"hsa_window_margin: arguments out of range ({center_percent}, {T})")
    return m


def hsa_build_active_set(budget, T: int, iteration: int, margin: int, idx, n_active_dev,
                         read_back: bool = True, stream=None, outside_period: int = 1, host_buf=None):
    """Fill idx[:|A_i|] with the active set; returns |A_i| when read_back
    (one stream synchronization), else None. outside_period != 1 calls
    hsa_build_active_set_window. host_buf: optional pinned int32 CPU tensor
    of one element that receives the count (a direct DMA)."""
    _dev(budget, idx, n_active_dev)
    host = ctypes.c_int32(-2)
    if host_buf is not None:
        if host_buf.device.type != "cpu" or host_buf.dtype != torch.int32 or host_buf.numel() < 1:
            raise ValueError("host_buf must be a CPU int32 tensor with at least one element")
        hb = ctypes.c_void_p(host_buf.data_ptr()) if read_back else None
    else:
        hb = ctypes.byref(host) if read_back else None
    if outside_period == 1:
        fn = "hsa_build_active_set"
        st = lib().hsa_build_active_set(_ptr(budget), budget.numel(), T, iteration, margin, _ptr(idx),
                                        _ptr(n_active_dev), hb, _stream(stream))
    else:
        fn = "hsa_build_active_set_window"
        st = lib().hsa_build_active_set_window(_ptr(budget), budget.numel(), T, iteration, margin, outside_period,
                                               _ptr(idx), _ptr(n_active_dev), hb, _stream(stream))
    _check(fn, st)
    if not read_back:
        return None
    return int(host_buf[0]) if host_buf is not None else host.value


def hsa_qkv_scatter(x, idx, n_active: int, wq, wk, wv, q_out, k_cache, v_cache,
                    x_compact: bool = False, stream=None) -> None:
    _dev(x, idx, wq, wk, wv, q_out, k_cache, v_cache)
    dt = _dtype(x, wq, wk, wv, q_out, k_cache, v_cache)
    n_tokens, d = k_cache.shape
    st = lib().hsa_qkv_scatter(dt, _ptr(x), int(bool(x_compact)), _ptr(idx), n_active, n_tokens, d,
                               _ptr(wq), _ptr(wk), _ptr(wv), _ptr(q_out), _ptr(k_cache), _ptr(v_cache),
                               _stream(stream))
    _check("hsa_qkv_scatter", st)


def hsa_attention_core(q, k_cache, v_cache, n_active: int, heads: int, head_dim: int, scale: float,
                       o, stream=None, parts=None) -> None:
    """Attention of the active queries; with `parts` (a device scratch,
    uint8) the library may split the cached rows into key parts."""
    _dev(q, k_cache, v_cache, o)
    dt = _dtype(q, k_cache, v_cache, o)
    if parts is None:
        st = lib().hsa_attention_core(dt, _ptr(q), _ptr(k_cache), _ptr(v_cache), n_active, k_cache.shape[0],
                                      heads, head_dim, scale, _ptr(o), _stream(stream))
        _check("hsa_attention_core", st)
        return
    _dev(parts)
    st = lib().hsa_attention_core_parts(dt, _ptr(q), _ptr(k_cache), _ptr(v_cache), n_active, k_cache.shape[0],
                                        heads, head_dim, scale, _ptr(o), _ptr(parts),
                                        parts.numel() * parts.element_size(), _stream(stream))
    _check("hsa_attention_core_parts", st)


def hsa_out_scatter(o, idx, n_active: int, wo, out, stream=None) -> None:
    _dev(o, idx, wo, out)
    dt = _dtype(o, wo, out)
    n_tokens, d = out.shape
    st = lib().hsa_out_scatter(dt, _ptr(o), _ptr(idx), n_active, n_tokens, d, _ptr(wo), _ptr(out),
                               _stream(stream))
    _check("hsa_out_scatter", st)


def hsa_attention_workspace_bytes(dtype: torch.dtype, n_active: int, d: int) -> int:
    return int(lib().hsa_attention_workspace_bytes(_dtype(torch.empty(0, dtype=dtype)), n_active, d))


def hsa_attention_parts_workspace_bytes(dtype: torch.dtype, n_active: int, heads: int, head_dim: int) -> int:
    return int(lib().hsa_attention_parts_workspace_bytes(_dtype(torch.empty(0, dtype=dtype)), n_active, heads,
                                                          head_dim))


def hsa_active_attention(q, k_cache, v_cache, idx, n_active: int, heads: int, head_dim: int,
                         scale: float, wo, out, workspace, stream=None) -> None:
    _dev(q, k_cache, v_cache, idx, wo, out, workspace)
    dt = _dtype(q, k_cache, v_cache, wo, out)
    nbytes = workspace.numel() * workspace.element_size()
    st = lib().hsa_active_attention(dt, _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(idx), n_active,
                                    k_cache.shape[0], heads, head_dim, scale, _ptr(wo), _ptr(out),
                                    _ptr(workspace), nbytes, _stream(stream))
    _check("hsa_active_attention", st)


def hsa_active_attention_noalloc(q, k_cache, v_cache, idx, n_active: int, heads: int, head_dim: int,
                                 scale: float, wo, out, stream=None) -> None:
    _dev(q, k_cache, v_cache, idx, wo, out)
    dt = _dtype(q, k_cache, v_cache, wo, out)
    st = lib().hsa_active_attention_noalloc(dt, _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(idx), n_active,
                                            k_cache.shape[0], heads, head_dim, scale, _ptr(wo), _ptr(out),
                                            _stream(stream))
    _check("hsa_active_attention_noalloc", st)


def hsa_cached_euler(x, v_cache, v_fresh, idx, n_active: int, sigma_i: float, sigma_next: float,
                     stream=None) -> None:
    _dev(x, v_cache, v_fresh, idx)
    for t in (x, v_cache, v_fresh):
        if t is not None and t.dtype != torch.float32:
            raise TypeError("the cached Euler update is fp32")
    n_tokens, channels = x.shape
    st = lib().hsa_cached_euler(_ptr(x), _ptr(v_cache), _ptr(v_fresh), _ptr(idx), n_active, n_tokens,
                                channels, sigma_i, sigma_next, _stream(stream))
    _check("hsa_cached_euler", st)


def hsa_gather_rows(x, idx, n_active: int, xa, stream=None) -> None:
    """xa[:n_active] = x[idx[:n_active]] in xa's dtype (bf16 or fp32)."""
    _dev(x, idx, xa)
    if x.dtype != torch.float32:
        raise TypeError("the latent is fp32")
    n_tokens, channels = x.shape
    st = lib().hsa_gather_rows(_dtype(xa), _ptr(x), _ptr(idx), n_active, n_tokens, channels, _ptr(xa),
                               _stream(stream))
    _check("hsa_gather_rows", st)


RMS_EPS = 1e-6  # the eps of the stack's RMS normalization


def hsa_row_rms_scale(x, n_rows: int, scale, eps: float = RMS_EPS, stream=None) -> None:
    """scale[:n_rows] = 1 / sqrt(mean(x[m]^2) + eps) per row."""
    _dev(x, scale)
    if scale.dtype != torch.float32:
        raise TypeError("row scales are fp32")
    st = lib().hsa_row_rms_scale(_dtype(x), _ptr(x), n_rows, x.shape[1], eps, _ptr(scale), _stream(stream))
    _check("hsa_row_rms_scale", st)


def hsa_linear(x, n_rows: int, w, y, residual=None, row_scale=None, gelu: bool = False, stream=None) -> None:
    """y[:n_rows] = act(row_scale * (x[:n_rows] w^T)) (+ residual[:n_rows]);
    y's dtype is the output dtype (x's, or fp32 for bf16 x)."""
    _dev(x, w, y, residual, row_scale)
    dt = _dtype(x, w)
    d_out, d_in = w.shape
    st = lib().hsa_linear(dt, _ptr(x), n_rows, d_in, _ptr(w), d_out, _ptr(row_scale), _ptr(residual), int(gelu),
                          _dtype(y), _ptr(y), _stream(stream))
    _check("hsa_linear", st)


def hsa_assign_budgets_workspace_bytes(n_tokens: int) -> int:
    return int(lib().hsa_assign_budgets_workspace_bytes(n_tokens))


def _group_arrays(group_sizes):
    n = len(group_sizes)
    gb = (ctypes.c_int32 * max(n, 1))(*[int(s) for s, _ in group_sizes])
    gs = (ctypes.c_int64 * max(n, 1))(*[int(c) for _, c in group_sizes])
    return gb, gs, n


def hsa_assign_budgets(v, T: int, group_sizes, budget, workspace, stream=None) -> None:
    """budget = group of each token's velocity-norm rank; group_sizes is
    ((s_k, n_k), ...) in ascending budget order."""
    _dev(v, budget, workspace)
    n_tokens, channels = v.shape
    gb, gs, n = _group_arrays(group_sizes)
    nbytes = workspace.numel() * workspace.element_size()
    st = lib().hsa_assign_budgets(_ptr(v), n_tokens, channels, T, gb, gs, n, _ptr(budget), _ptr(workspace),
                                  nbytes, _stream(stream))
    _check("hsa_assign_budgets", st)


def hsa_l1_rel_accumulate(v, v_prev, acc, first: bool, stream=None) -> None:
    _dev(v, v_prev, acc)
    n_tokens, channels = v.shape
    st = lib().hsa_l1_rel_accumulate(_ptr(v), _ptr(v_prev), n_tokens, channels, _ptr(acc), int(first),
                                     _stream(stream))
    _check("hsa_l1_rel_accumulate", st)


def hsa_assign_budgets_by_key(keys, T: int, group_sizes, budget, stream=None) -> None:
    _dev(keys, budget)
    gb, gs, n = _group_arrays(group_sizes)
    st = lib().hsa_assign_budgets_by_key(_ptr(keys), keys.numel(), T, gb, gs, n, _ptr(budget), _stream(stream))
    _check("hsa_assign_budgets_by_key", st)


def hsa_reorder_plan(budget, T: int, perm, n_lead_dev, stream=None) -> int:
    """perm = non-baseline tokens then the budget-T group; returns their split
    (one stream synchronization)."""
    _dev(budget, perm, n_lead_dev)
    host = ctypes.c_int32(-2)
    st = lib().hsa_reorder_plan(_ptr(budget), budget.numel(), T, _ptr(perm), _ptr(n_lead_dev), ctypes.byref(host),
                                _stream(stream))
    _check("hsa_reorder_plan", st)
    return host.value


def hsa_permute_rows(src, perm, dst, inverse: bool = False, stream=None) -> None:
    """dst[i] = src[perm[i]] (inverse: dst[perm[i]] = src[i]) over the rows of
    src (first dimension)."""
    _dev(src, perm, dst)
    if src.dtype != dst.dtype or src.shape != dst.shape:
        raise TypeError("src and dst must match")
    n = src.shape[0]
    row_bytes = src.numel() // max(n, 1) * src.element_size()
    st = lib().hsa_permute_rows(_ptr(src), _ptr(perm), n, row_bytes, int(inverse), _ptr(dst), _stream(stream))
    _check("hsa_permute_rows", st)


def hsa_rope_table(theta: float, head_dim: int, grid) -> torch.Tensor:
    """The (cos, sin) table of the stack's rotary embedding, on the host
    (float32 [(F + H + W), head_dim])."""
    n = int(lib().hsa_rope_table_floats(head_dim, *grid))
    if n == 0:
        raise ValueError("invalid rotary table sizes")
    out = torch.empty(n, dtype=torch.float32)
    _check("hsa_rope_table", lib().hsa_rope_table(theta, head_dim, *grid, ctypes.c_void_p(out.data_ptr())))
    return out.view(-1, head_dim)


def make_stack(*, x, v_hat, budget, w_embed, w_head, layers, caches, idx, n_active, xa, h, q, o, v_fresh,
               keys, row_scale, heads: int, head_dim: int, cross=None, ffn=None, f=None,
               v_prev=None, rope_cs=None, pos=None, grid=(0, 0, 0), n_cached=None, k_tail=None,
               v_tail=None, attn_parts=None) -> HsaStack:
    """Fill a struct hsa_stack from device tensors. layers: per layer
    (wq, wk, wv, wo); caches: per layer (k_hat, v_hat); cross: per layer
    (wq_c, wo_c, k_c, v_c) or None; ffn: per layer (w1, w2) or None;
    attn_parts: scratch for key parts of the attention launches or None. The
    returned struct keeps its host pointer arrays alive; the tensors must
    outlive it."""
    ts = [x, v_hat, budget, w_embed, w_head, idx, n_active, xa, h, q, o, v_fresh, keys, row_scale, f, v_prev,
          rope_cs, pos, k_tail, v_tail, attn_parts]
    ts += [t for lw in layers for t in lw] + [t for c in caches for t in c]
    ts += [t for lw in (cross or ()) for t in lw] + [t for lw in (ffn or ()) for t in lw]
    _dev(*ts)
    n_tokens, channels = x.shape
    wl = (ctypes.c_void_p * max(1, 4 * len(layers)))(*[t.data_ptr() for lw in layers for t in lw])
    cl = (ctypes.c_void_p * max(1, 2 * len(caches)))(*[t.data_ptr() for c in caches for t in c])
    s = HsaStack(dtype=_dtype(w_embed, w_head, xa, h, q, o, *[t for lw in layers for t in lw],
                              *[t for c in caches for t in c]),
                 n_layers=len(layers), heads=heads, head_dim=head_dim, channels=channels, reserved=0,
                 n_tokens=n_tokens, w_embed=w_embed.data_ptr(), w_head=w_head.data_ptr(),
                 w_layers=ctypes.cast(wl, ctypes.POINTER(ctypes.c_void_p)),
                 caches=ctypes.cast(cl, ctypes.POINTER(ctypes.c_void_p)),
                 x=x.data_ptr(), v_hat=v_hat.data_ptr(), budget=budget.data_ptr(), idx=idx.data_ptr(),
                 n_active=n_active.data_ptr(), xa=xa.data_ptr(), h=h.data_ptr(), q=q.data_ptr(),
                 o=o.data_ptr(), v_fresh=v_fresh.data_ptr(), keys=keys.data_ptr(),
                 row_scale=row_scale.data_ptr(), ffn_dim=0 if not ffn else ffn[0][0].shape[0],
                 ctx_len=0 if not cross else cross[0][2].shape[0],
                 f=0 if f is None else f.data_ptr(), v_prev=0 if v_prev is None else v_prev.data_ptr(),
                 rope_cs=0 if rope_cs is None else rope_cs.data_ptr(), pos=0 if pos is None else pos.data_ptr(),
                 grid_f=grid[0], grid_h=grid[1], grid_w=grid[2], reserved2=0,
                 prefix_cache=0 if n_cached is None else 1, reserved3=0,
                 n_cached=0 if n_cached is None else int(n_cached),
                 k_tail=0 if k_tail is None else k_tail.data_ptr(), v_tail=0 if v_tail is None else v_tail.data_ptr(),
                 attn_parts=0 if attn_parts is None else attn_parts.data_ptr(),
                 attn_parts_bytes=0 if attn_parts is None else attn_parts.numel() * attn_parts.element_size())
    keep = [wl, cl]
    if cross:
        xl = (ctypes.c_void_p * (4 * len(cross)))(*[t.data_ptr() for lw in cross for t in lw])
        s.w_cross = ctypes.cast(xl, ctypes.POINTER(ctypes.c_void_p))
        keep.append(xl)
    if ffn:
        fl = (ctypes.c_void_p * (2 * len(ffn)))(*[t.data_ptr() for lw in ffn for t in lw])
        s.w_ffn = ctypes.cast(fl, ctypes.POINTER(ctypes.c_void_p))
        keep.append(fl)
    s._keep = tuple(keep)
    return s


def hsa_stack_iteration(stack: HsaStack, T: int, iteration: int, margin: int, sigma_i: float,
                        sigma_next: float, group_sizes=None, stream=None, outside_period: int = 1,
                        selection: int = SELECT_VELOCITY_NORM) -> tuple:
    """One multi-layer HSA iteration; returns (|A_i|, refreshed)."""
    gb, gs, n = _group_arrays(group_sizes or ())
    n_act = ctypes.c_int32(-1)
    ref = ctypes.c_int32(-1)
    st = lib().hsa_stack_iteration(ctypes.byref(stack), T, iteration, margin, outside_period, sigma_i, sigma_next,
                                   gb, gs, n, selection, ctypes.byref(n_act), ctypes.byref(ref), _stream(stream))
    _check("hsa_stack_iteration", st)
    return n_act.value, bool(ref.value)
