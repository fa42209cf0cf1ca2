"""Host-side tests of the C ABI (no GPU needed).

The library must load and export every entry point include/hsa_step.h
declares, and every argument error must be reported with its documented
status before anything is enqueued. Only error cases are called here (and the
pure-host helpers), so no kernel is ever launched.
"""

import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hsa_step.h")

H = pytest.importorskip("paper_2605_06892_amd.hsa_step")

OK, NULL, SHAPE, BUDGET, DTYPE, ALIAS, WORKSPACE, LAUNCH = range(8)
F32, BF16 = 0, 1
# fake device addresses: never dereferenced, every call below fails validation first
A = 0x7F0000000000
B = 0x7F1000000000
C = 0x7F2000000000
D = 0x7F3000000000
E = 0x7F4000000000
G = 0x7F5000000000
W = 0x7F6000000000


def declared_functions():
    text = open(HEADER).read()
    return re.findall(r"^(?:int|int32_t|size_t|const char\*)\s+(hsa_\w+)\s*\(", text, flags=re.M)


@pytest.fixture(scope="module")
def lib():
    try:
        return H.lib()
    except ImportError as e:  # pragma: no cover
        pytest.fail(f"HIP library not built: {e}")


def test_header_declares_the_four_hot_path_calls():
    names = declared_functions()
    for n in ("hsa_build_active_set", "hsa_qkv_scatter", "hsa_active_attention", "hsa_cached_euler"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 8
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(H.EXPORTED)
    out = subprocess.run(["nm", "-D", "--defined-only", H._LIB_PATH], capture_output=True, text=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    assert set(names) <= exported
    # nothing beyond the C ABI leaks out of the library
    assert {s for s in exported if not s.startswith("_")} == set(names)


def test_status_strings(lib):
    for s in range(8):
        assert lib.hsa_step_status_string(s)
    assert lib.hsa_step_status_string(99) == b"unknown status"


def test_noalloc_limit_checked_before_anything(lib):
    # beyond the fixed array: refused on the host, before any HIP call (fake pointers, no GPU)
    f = lib.hsa_active_attention_noalloc
    assert f(BF16, A, B, C, D, 9831, 32760, 40, 128, 0.088, E, G, None) == WORKSPACE
    assert f(7, A, B, C, D, 10, 100, 2, 64, 0.125, E, G, None) == DTYPE
    assert f(BF16, A, B, C, D, 10, 5, 2, 64, 0.125, E, G, None) == SHAPE
    assert f(BF16, A, B, C, D, 0, 5, 2, 64, 0.125, E, G, None) == OK  # nothing to do


def test_window_margin(lib):
    # Section 2.5, m = floor((1 - k) T / 2) in exact integers (HSA-50: k = 80%, T = 40 -> 4, not 3)
    assert lib.hsa_window_margin(80, 40) == 4
    assert lib.hsa_window_margin(50, 40) == 10
    assert lib.hsa_window_margin(100, 40) == 0
    assert lib.hsa_window_margin(0, 40) == 20
    assert lib.hsa_window_margin(0, 7) == 3
    for bad in ((-1, 40), (101, 40), (50, 0), (50, -3)):
        assert lib.hsa_window_margin(*bad) == -1
    # every margin it returns is one hsa_build_active_set accepts (0 <= m <= T/2)
    for T in range(1, 81):
        for k in range(101):
            m = lib.hsa_window_margin(k, T)
            assert 0 <= m <= T // 2 and m == ((100 - k) * T) // 200
    assert H.hsa_window_margin(80, 40) == 4
    with pytest.raises(ValueError):
        H.hsa_window_margin(120, 40)


def test_workspace_bytes(lib):
    assert lib.hsa_attention_workspace_bytes(BF16, 8190, 5120) == 8190 * 5120 * 2
    assert lib.hsa_attention_workspace_bytes(F32, 10, 256) == 10 * 256 * 4
    assert lib.hsa_attention_workspace_bytes(7, 10, 256) == 0
    assert lib.hsa_attention_workspace_bytes(BF16, -1, 256) == 0
    # the compact tensor from a 256-byte boundary, then 4 parts of fp32 (O, m, l)
    base = 8190 * 1536 * 2
    assert lib.hsa_attention_parts_workspace_bytes(BF16, 8190, 12, 128) == \
        (base + 255) // 256 * 256 + 4 * 8190 * 12 * (128 + 2) * 4
    assert lib.hsa_attention_parts_workspace_bytes(BF16, 10, 1, 64) == 1280 + 4 * 10 * 66 * 4
    assert lib.hsa_attention_parts_workspace_bytes(F32, 10, 4, 64) == 10 * 256 * 4
    assert lib.hsa_attention_parts_workspace_bytes(BF16, -1, 4, 64) == 0
    assert lib.hsa_attention_parts_workspace_bytes(BF16, 10, -4, 64) == 0


def test_build_active_set_errors(lib):
    f = lib.hsa_build_active_set
    assert f(A, 100, 0, 0, 0, B, C, None, None) == BUDGET        # T < 1
    assert f(A, 100, 40, 40, 0, B, C, None, None) == BUDGET      # iter >= T
    assert f(A, 100, 40, -1, 0, B, C, None, None) == BUDGET
    assert f(A, 100, 40, 0, 21, B, C, None, None) == BUDGET      # margin > T/2
    assert f(A, 100, 40, 0, -1, B, C, None, None) == BUDGET
    assert f(A, -1, 40, 0, 0, B, C, None, None) == SHAPE
    assert f(A, 1 << 31, 40, 0, 0, B, C, None, None) == SHAPE
    assert f(None, 100, 40, 0, 0, B, C, None, None) == NULL
    assert f(A, 100, 40, 0, 0, None, C, None, None) == NULL
    assert f(A, 100, 40, 0, 0, B, None, None, None) == NULL
    assert f(A, 100, 40, 0, 0, A + 8, C, None, None) == ALIAS    # idx overlaps budget
    assert f(A, 100, 40, 0, 0, B, B + 396, None, None) == ALIAS  # count inside idx
    g = lib.hsa_build_active_set_window
    assert g(A, 100, 40, 0, 4, 3, B, C, None, None) == BUDGET    # outside period does not divide T
    assert g(A, 100, 40, 0, 4, 0, B, C, None, None) == BUDGET
    assert g(A, 100, 40, 0, 4, 2, A + 8, C, None, None) == ALIAS


def test_qkv_scatter_errors(lib):
    f = lib.hsa_qkv_scatter
    args = lambda **k: dict(dict(dt=BF16, x=A, xc=0, idx=B, n=10, N=100, d=256, wq=C, wk=D, wv=E,  # noqa: E731
                                 q=G, kc=W, vc=W + 100 * 256 * 2), **k)
    call = lambda a: f(a["dt"], a["x"], a["xc"], a["idx"], a["n"], a["N"], a["d"], a["wq"], a["wk"],  # noqa: E731
                       a["wv"], a["q"], a["kc"], a["vc"], None)
    assert call(args(dt=5)) == DTYPE
    assert call(args(d=0)) == SHAPE
    assert call(args(d=200)) == SHAPE       # bf16 needs d % 64 == 0
    assert call(args(n=101)) == SHAPE       # more active rows than tokens
    assert call(args(n=-1)) == SHAPE
    assert call(args(x=None)) == NULL
    assert call(args(wv=None)) == NULL
    assert call(args(x=A + 2)) == SHAPE     # bf16 rows must be 16-byte aligned
    assert call(args(q=A)) == ALIAS         # q_out on top of x
    assert call(args(vc=W + 16)) == ALIAS   # the two caches overlap
    assert call(args(kc=C)) == ALIAS        # cache on top of a weight


def test_attention_errors(lib):
    f = lib.hsa_attention_core
    assert f(9, A, B, C, 10, 100, 4, 64, 0.125, D, None) == DTYPE
    assert f(BF16, A, B, C, 10, 100, 4, 96, 0.125, D, None) == SHAPE   # head_dim not 64/128
    assert f(BF16, A, B, C, 10, 100, 0, 64, 0.125, D, None) == SHAPE
    assert f(BF16, A, B, C, 10, 0, 4, 64, 0.125, D, None) == SHAPE     # no keys
    assert f(BF16, A, B, C, 10, 100, 4, 64, 0.0, D, None) == SHAPE     # scale must be > 0
    assert f(BF16, A, B, C, 10, 100, 4, 64, float("nan"), D, None) == SHAPE
    assert f(BF16, A, None, C, 10, 100, 4, 64, 0.125, D, None) == NULL
    assert f(BF16, A, B, C, 10, 100, 4, 64, 0.125, A, None) == ALIAS   # o on top of q
    assert f(BF16, A, B, C, 10, 100, 4, 64, 0.125, B + 512, None) == ALIAS
    s_ = lib.hsa_attention_core_parts
    assert s_(BF16, A, B, C, 10, 100, 4, 64, 0.125, D, A + 4096, 1 << 20, None) == ALIAS  # parts over q
    assert s_(BF16, A, B, C, 10, 100, 4, 64, 0.125, D, W + 4, 1 << 20, None) == SHAPE     # misaligned
    assert s_(BF16, A, B, C, 10, 100, 4, 96, 0.125, D, W, 1 << 20, None) == SHAPE
    g = lib.hsa_active_attention
    need = lib.hsa_attention_workspace_bytes(BF16, 10, 256)
    assert g(BF16, A, B, C, D, 10, 100, 4, 64, 0.125, E, G, None, need, None) == WORKSPACE
    assert g(BF16, A, B, C, D, 10, 100, 4, 64, 0.125, E, G, W, need - 1, None) == WORKSPACE
    assert g(BF16, A, B, C, D, 10, 100, 4, 64, 0.125, E, G, G, need, None) == ALIAS
    # out inside the key-part bytes past the compact tensor
    assert g(BF16, A, B, C, D, 10, 100, 4, 64, 0.125, E, W + 8192, W, 1 << 20, None) == ALIAS
    assert g(BF16, A, B, C, D, 10, 100, 4, 64, 0.125, W + 8192, G, W, 1 << 20, None) == ALIAS  # wo
    assert g(BF16, A, B, C, None, 10, 100, 4, 64, 0.125, E, G, W, need, None) == NULL
    assert g(BF16, A, B, C, D, 10, 100, 4, 64, 0.125, E, None, W, need, None) == NULL
    h = lib.hsa_out_scatter
    assert h(BF16, A, B, 10, 100, 256, C, A, None) == ALIAS           # out on top of o
    assert h(BF16, A, B, 10, 100, 100, C, D, None) == SHAPE
    assert h(BF16, A, None, 10, 100, 256, C, D, None) == NULL


def test_euler_errors(lib):
    f = lib.hsa_cached_euler
    assert f(A, B, None, None, 0, -1, 16, 1.0, 0.9, None) == SHAPE
    assert f(None, B, None, None, 0, 100, 16, 1.0, 0.9, None) == NULL
    assert f(A, B, C, None, 10, 100, 16, 1.0, 0.9, None) == NULL       # fresh rows need idx
    assert f(A, B, C, D, 101, 100, 16, 1.0, 0.9, None) == SHAPE
    assert f(A, A + 64, None, None, 0, 100, 16, 1.0, 0.9, None) == ALIAS
    assert f(A, B, B + 4, D, 10, 100, 16, 1.0, 0.9, None) == ALIAS     # fresh inside the cache
    # nothing to do is success without touching memory
    assert f(None, None, None, None, 0, 0, 16, 1.0, 0.9, None) == OK


def test_stack_struct_layout_matches_the_header(tmp_path):
    """The ctypes mirror of struct hsa_stack has the C compiler's layout."""
    fields = [f for f, _ in H.HsaStack._fields_]
    src = tmp_path / "layout.c"
    src.write_text("#include <stdio.h>\n#include <stddef.h>\n#include \"hsa_step.h\"\nint main(void) {\n"
                   "  printf(\"%zu\\n\", sizeof(hsa_stack));\n"
                   + "".join(f"  printf(\"%zu\\n\", offsetof(hsa_stack, {f}));\n" for f in fields)
                   + "  return 0;\n}\n")
    exe = tmp_path / "layout"
    r = subprocess.run(["gcc", "-std=c11", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                        "-I", "/opt/rocm/include", str(src), "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    got = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True).stdout.split()]
    assert got[0] == ctypes.sizeof(H.HsaStack)
    assert got[1:] == [getattr(H.HsaStack, f).offset for f in fields]


def test_gather_rows_errors(lib):
    f = lib.hsa_gather_rows
    assert f(3, A, B, 10, 100, 16, C, None) == DTYPE
    assert f(BF16, A, B, -1, 100, 16, C, None) == SHAPE
    assert f(BF16, A, B, 10, -1, 16, C, None) == SHAPE
    assert f(BF16, None, B, 10, 100, 16, C, None) == NULL
    assert f(BF16, A, B, 10, 100, 16, None, None) == NULL
    assert f(BF16, A, B, 10, 100, 16, A + 64, None) == ALIAS     # xa inside x
    assert f(BF16, A, B, 10, 100, 16, B, None) == ALIAS          # xa on top of idx
    assert f(F32, A + 2, B, 10, 100, 16, C, None) == SHAPE       # misaligned latent
    assert f(BF16, None, None, 0, 100, 16, None, None) == OK     # nothing to gather


def test_linear_errors(lib):
    f = lambda *a: lib.hsa_linear(*a[:6], None, a[6], 0, *a[-3:])  # noqa: E731
    assert f(F32, A, 10, 64, B, 64, None, BF16, C, None) == DTYPE   # fp32 in, bf16 out
    assert f(9, A, 10, 64, B, 64, None, BF16, C, None) == DTYPE
    assert f(BF16, A, 10, 100, B, 64, None, BF16, C, None) == SHAPE  # bf16 d_in % 64
    assert f(BF16, A, 10, 64, B, 62, None, BF16, C, None) == SHAPE   # bf16 d_out % 4
    assert f(BF16, A, 10, 64, B, 64, D, F32, C, None) == SHAPE       # fp32 output takes no residual
    assert f(BF16, A, -1, 64, B, 64, None, BF16, C, None) == SHAPE
    assert f(BF16, None, 10, 64, B, 64, None, BF16, C, None) == NULL
    assert f(BF16, A, 10, 64, B, 64, None, BF16, A + 64, None) == ALIAS   # y inside x
    assert f(BF16, A, 10, 64, B, 64, None, BF16, B, None) == ALIAS        # y on top of w
    assert f(BF16, A, 10, 64, B, 64, C + 16, BF16, C, None) == ALIAS      # residual partly over y
    assert f(BF16, A, 10, 64, B, 64, None, BF16, C + 8, None) == SHAPE    # misaligned
    assert f(BF16, None, 0, 64, None, 64, None, BF16, None, None) == OK
    g = lib.hsa_linear
    assert g(BF16, A, 10, 64, B, 64, C + 8, None, 0, BF16, C, None) == ALIAS  # row scales inside y
    assert g(BF16, A, 10, 64, B, 64, D + 2, None, 0, BF16, C, None) == SHAPE  # misaligned row scales
    assert g(BF16, A, 10, 64, B, 64, None, D, 1, BF16, C, None) == SHAPE     # GELU takes no residual
    assert g(BF16, A, 10, 64, B, 64, None, None, 1, F32, C, None) == SHAPE   # nor an fp32 output


def test_row_rms_scale_errors(lib):
    f = lib.hsa_row_rms_scale
    assert f(7, A, 10, 64, 1e-6, B, None) == DTYPE
    assert f(BF16, A, -1, 64, 1e-6, B, None) == SHAPE
    assert f(BF16, A, 10, 0, 1e-6, B, None) == SHAPE
    assert f(BF16, A, 10, 64, -1.0, B, None) == SHAPE
    assert f(BF16, A, 10, 64, float("inf"), B, None) == SHAPE
    assert f(BF16, None, 10, 64, 1e-6, B, None) == NULL
    assert f(BF16, A, 10, 64, 1e-6, None, None) == NULL
    assert f(BF16, A, 10, 64, 1e-6, A + 64, None) == ALIAS
    assert f(BF16, A + 1, 10, 64, 1e-6, B, None) == SHAPE
    assert f(BF16, None, 0, 64, 1e-6, None, None) == OK


def test_assign_budgets_errors(lib):
    f = lib.hsa_assign_budgets
    gb = lambda *v: (ctypes.c_int32 * len(v))(*v)  # noqa: E731
    gs = lambda *v: (ctypes.c_int64 * len(v))(*v)  # noqa: E731
    ws = lib.hsa_assign_budgets_workspace_bytes(100)
    assert ws == 800 and lib.hsa_assign_budgets_workspace_bytes(-3) == 0
    assert f(A, 100, 16, 40, gb(40, 10), gs(50, 50), 2, B, C, ws, None) == BUDGET   # not ascending
    assert f(A, 100, 16, 40, gb(10, 30), gs(50, 50), 2, B, C, ws, None) == BUDGET   # 30 does not divide 40
    assert f(A, 100, 16, 40, gb(10, 40), gs(50, 49), 2, B, C, ws, None) == BUDGET   # sizes do not sum to N
    assert f(A, 100, 16, 40, gb(10, 40), gs(-1, 101), 2, B, C, ws, None) == BUDGET
    assert f(A, 100, 16, 40, gb(10), gs(100), 0, B, C, ws, None) == BUDGET           # no groups
    assert f(A, 100, 16, 40, None, gs(100), 1, B, C, ws, None) == BUDGET
    assert f(A, 100, 16, 40, gb(40), gs(100), 1, B, None, ws, None) == WORKSPACE
    assert f(A, 100, 16, 40, gb(40), gs(100), 1, B, C, ws - 8, None) == WORKSPACE
    assert f(None, 100, 16, 40, gb(40), gs(100), 1, B, C, ws, None) == NULL
    assert f(A, 100, 16, 40, gb(40), gs(100), 1, A + 4, C, ws, None) == ALIAS       # budget inside v
    assert f(A, 100, 16, 40, gb(40), gs(100), 1, B, B + 8, ws, None) == ALIAS       # workspace over budget


def _stack(**over):
    base = 0x7E0000000000
    step = 1 << 32
    ptrs = {n: base + k * step for k, n in enumerate(
        ["w_embed", "w_head", "x", "v_hat", "budget", "idx", "n_active", "xa", "h", "q", "o", "v_fresh", "keys",
         "row_scale", "v_prev"])}
    L = over.pop("L", 2)
    wl = (ctypes.c_void_p * (4 * L))(*[0x7D0000000000 + k * step for k in range(4 * L)])
    cl = (ctypes.c_void_p * (2 * L))(*[0x7C0000000000 + k * step for k in range(2 * L)])
    fields = dict(dtype=BF16, n_layers=L, heads=12, head_dim=128, channels=64, reserved=0, n_tokens=1000,
                  w_layers=ctypes.cast(wl, ctypes.POINTER(ctypes.c_void_p)),
                  caches=ctypes.cast(cl, ctypes.POINTER(ctypes.c_void_p)), **ptrs)
    fields.update(over)
    s = H.HsaStack(**fields)
    s._keep = (wl, cl)
    return s, wl, cl


def test_stack_iteration_errors(lib):
    f = lib.hsa_stack_iteration
    gb = (ctypes.c_int32 * 2)(20, 40)
    gs = (ctypes.c_int64 * 2)(500, 500)
    call = lambda s, T=40, i=1, m=0, g=2, b=gb, p=1, sel=0: f(ctypes.byref(s), T, i, m, p, 1.0, 0.975, b,  # noqa: E731
                                                              gs, g, sel, None, None, None)
    assert f(None, 40, 0, 0, 1, 1.0, 0.975, None, None, 0, 0, None, None, None) == NULL
    assert call(_stack(dtype=4)[0]) == DTYPE
    assert call(_stack(head_dim=96)[0]) == SHAPE
    assert call(_stack(channels=16)[0]) == SHAPE           # bf16 stacks need C % 64 == 0
    assert call(_stack(n_tokens=0)[0]) == SHAPE
    assert call(_stack(reserved=1)[0]) == SHAPE
    assert call(_stack(n_layers=-1, L=1)[0]) == SHAPE
    assert call(_stack()[0], i=40) == BUDGET
    assert call(_stack()[0], m=21) == BUDGET
    assert call(_stack()[0], p=3) == BUDGET                           # outside period must divide T
    assert call(_stack()[0], p=0) == BUDGET
    assert call(_stack()[0], sel=2) == BUDGET                         # unknown selection
    assert call(_stack()[0], sel=1, m=1) == BUDGET                    # strategy D needs margin >= 2
    assert call(_stack()[0], sel=1, m=4, p=2) == BUDGET               # ... and every token active outside
    assert call(_stack(v_prev=None)[0], sel=1, m=4) == NULL
    assert call(_stack(ffn_dim=100)[0]) == SHAPE                      # bf16 FFN width % 64
    assert call(_stack(ffn_dim=128)[0]) == NULL                       # FFN weights and scratch missing
    assert call(_stack(ctx_len=-1)[0]) == SHAPE
    assert call(_stack(ctx_len=77)[0]) == NULL                        # cross-attention weights missing
    assert call(_stack()[0], b=(ctypes.c_int32 * 2)(20, 30)) == BUDGET   # 30 does not divide 40
    assert call(_stack()[0], g=-1) == BUDGET
    assert call(_stack(h=None)[0]) == NULL
    assert call(_stack(keys=None)[0]) == NULL                          # refresh needs the key scratch
    assert call(_stack(row_scale=None)[0]) == NULL
    s, wl, _ = _stack()
    wl[5] = None
    assert call(s) == NULL                                             # a missing layer weight
    s, _, cl = _stack()
    cl[3] = cl[2] + 64
    assert call(s) == ALIAS                                            # two caches overlap
    s, wl, cl = _stack()
    wl[0] = cl[1]
    assert call(s) == ALIAS                                            # a weight inside a cache
    assert call(_stack(q=0x7E0000000000 + 8 * (1 << 32) + 32)[0]) == ALIAS  # q inside h
    assert call(_stack(o=0x7E0000000000 + 3)[0]) == SHAPE              # misaligned
    assert call(_stack(attn_parts_bytes=-1)[0]) == SHAPE
    assert call(_stack(attn_parts_bytes=4096)[0]) == SHAPE             # bytes without a buffer
    assert call(_stack(attn_parts=0x7E0000000000 + 2 * (1 << 32) + 64, attn_parts_bytes=4096)[0]) == ALIAS  # inside x


def test_l1_rel_and_key_assignment_errors(lib):
    f = lib.hsa_l1_rel_accumulate
    assert f(A, B, -1, 16, C, 1, None) == SHAPE
    assert f(None, B, 100, 16, C, 1, None) == NULL
    assert f(A, A + 64, 100, 16, C, 0, None) == ALIAS      # v_prev inside v
    assert f(A, B, 100, 16, B + 8, 0, None) == ALIAS       # acc inside v_prev
    assert f(A, B, 100, 16, C + 4, 0, None) == SHAPE       # misaligned acc
    assert f(None, None, 0, 16, None, 0, None) == OK
    g = lib.hsa_assign_budgets_by_key
    gb = (ctypes.c_int32 * 2)(10, 40)
    gs = (ctypes.c_int64 * 2)(50, 50)
    assert g(A, 100, 40, (ctypes.c_int32 * 2)(40, 10), gs, 2, B, None) == BUDGET
    assert g(A, 100, 40, gb, (ctypes.c_int64 * 2)(50, 40), 2, B, None) == BUDGET
    assert g(None, 100, 40, gb, gs, 2, B, None) == NULL
    assert g(A, 100, 40, gb, gs, 2, A + 16, None) == ALIAS
    assert g(A + 4, 100, 40, gb, gs, 2, B, None) == SHAPE


def test_rope_table_matches_the_oracle_angles(lib):
    """The host-side rotary table holds cos/sin of the oracle's angles (within
    fp32 rounding) for every coordinate of its band, zeros elsewhere."""
    import numpy as np

    import oracle
    for dh, grid in ((128, (21, 30, 52)), (64, (3, 10, 10))):
        t = H.hsa_rope_table(10000.0, dh, grid).numpy().reshape(sum(grid), dh // 2, 2)
        F, Hh, W = grid
        nt, nh, nw = oracle.rope_bands(dh)
        for band, (lo, n, pairs) in enumerate(((0, F, range(0, nt)), (F, Hh, range(nt, nt + nh)),
                                                 (F + Hh, W, range(nt + nh, nt + nh + nw)))):
            coord = np.arange(n)
            p = [coord * Hh * W, coord * W, coord][band]  # a position with this coordinate, others 0
            ang = oracle.rope_angles(p, grid, dh)[:, list(pairs)]
            np.testing.assert_allclose(t[lo:lo + n, list(pairs), 0], np.cos(ang), rtol=0, atol=2e-7)
            np.testing.assert_allclose(t[lo:lo + n, list(pairs), 1], np.sin(ang), rtol=0, atol=2e-7)
            others = [k for k in range(dh // 2) if k not in pairs]
            assert np.all(t[lo:lo + n, others] == 0)
    assert lib.hsa_rope_table_floats(128, 0, 30, 52) == 0
    assert lib.hsa_rope_table(10000.0, 128, 2, 2, 2, None) == NULL
    assert lib.hsa_rope_table(0.5, 128, 2, 2, 2, A) == SHAPE


def test_reorder_and_permute_errors(lib):
    f = lib.hsa_reorder_plan
    assert f(A, -1, 40, B, C, None, None) == SHAPE
    assert f(A, 100, 0, B, C, None, None) == BUDGET
    assert f(None, 100, 40, B, C, None, None) == NULL
    assert f(A, 100, 40, B, None, None, None) == NULL
    assert f(A, 100, 40, A + 8, C, None, None) == ALIAS       # perm inside budget
    assert f(A, 100, 40, B, B + 16, None, None) == ALIAS      # count inside perm
    g = lib.hsa_permute_rows
    assert g(A, B, -1, 64, 0, C, None) == SHAPE
    assert g(None, B, 10, 64, 0, C, None) == NULL
    assert g(A, B, 10, 64, 0, A + 32, None) == ALIAS          # dst over src
    assert g(A, B, 10, 64, 0, B, None) == ALIAS               # dst over perm
    assert g(A, B + 2, 10, 64, 0, C, None) == SHAPE           # misaligned perm
    assert g(None, None, 0, 64, 0, None, None) == OK


def test_prefix_cache_stack_errors(lib):
    f = lib.hsa_stack_iteration
    gb = (ctypes.c_int32 * 2)(20, 40)
    gs = (ctypes.c_int64 * 2)(500, 500)
    call = lambda s, g=0: f(ctypes.byref(s), 40, 1, 0, 1, 1.0, 0.975, gb, gs, g, 0, None, None, None)  # noqa: E731
    assert call(_stack(prefix_cache=1, n_cached=512)[0], g=2) == BUDGET   # fixed groups only
    assert call(_stack(prefix_cache=1, n_cached=1001)[0]) == SHAPE
    assert call(_stack(prefix_cache=1, n_cached=-1)[0]) == SHAPE
    assert call(_stack(prefix_cache=1, n_cached=500)[0]) == SHAPE        # not a multiple of 64
    assert call(_stack(prefix_cache=2, n_cached=512)[0]) == SHAPE
    assert call(_stack(prefix_cache=1, n_cached=512)[0]) == NULL         # tails missing
    assert call(_stack(reserved3=1)[0]) == SHAPE
