"""The C ABI library loads, exports every declared symbol, and validates on the
host (no GPU needed: every rejected call returns before any HIP call)."""
import ctypes
import os
import re

import pytest

from paper_2609_36259_amd import cyfa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    txt = open(os.path.join(ROOT, "include", "cyfa.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(cyfa_[a-z_0-9]+)\s*\(", txt)))


def test_library_exports_every_declared_symbol():
    lib = cyfa.load()
    names = _declared_functions()
    assert set(names) == set(cyfa.EXPORTED), names
    for n in names:
        assert hasattr(lib, n), n
    assert lib.cyfa_version() >= 100
    for code in range(5):
        assert lib.cyfa_status_string(code)


def _ws(desc):
    return cyfa.forward_workspace_size(desc)


def test_workspace_sizes_and_kernel_selection():
    d = cyfa.forward_desc(4, 4096, 16, 128, 128, dtype=cyfa.BF16)
    assert _ws(d) >= 16 * 128 * 128 * 4
    d = cyfa.forward_desc(1, 256, 2, 64, 64, dtype=cyfa.F32, segments=1)
    assert _ws(d) == 2 * 128 * 128 * 4            # one chunk group: the readout matrices only
    d = cyfa.forward_desc(1, 256, 2, 64, 64, dtype=cyfa.F32)
    assert _ws(d) > 2 * 128 * 128 * 4             # automatic chunk groups: their entering states
    d = cyfa.forward_desc(1, 256, 2, 256, 64, dtype=cyfa.F32, segments=4)
    with pytest.raises(cyfa.CyfaError):
        _ws(d)                                    # groups need d <= 128
    dd = cyfa.decode_desc(256, 16, 128, 128)
    assert cyfa.decode_workspace_size(dd) == 16 * 128 * 128 * 4


@pytest.mark.parametrize("field,value,status", [
    ("m", 128, cyfa.CyfaError), ("m", 1, cyfa.CyfaError), ("m", 257, cyfa.CyfaError),
    ("d_k", 96, cyfa.CyfaError), ("d_v", 0, cyfa.CyfaError), ("B", 0, cyfa.CyfaError),
    ("H", 0, cyfa.CyfaError), ("T", -1, cyfa.CyfaError), ("dtype", 5, cyfa.CyfaError),
    ("kernel", 7, cyfa.CyfaError), ("segments", -1, cyfa.CyfaError), ("chunk", 48, cyfa.CyfaError),
])
def test_descriptor_validation(field, value, status):
    d = cyfa.forward_desc(2, 64, 2, 64, 64, dtype=cyfa.F32)
    setattr(d, field, value)
    with pytest.raises(status):
        _ws(d)


def test_status_codes():
    lib = cyfa.load()
    n = ctypes.c_size_t(0)
    d = cyfa.forward_desc(1, 16, 1, 64, 64, m=128)
    assert lib.cyfa_forward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 1
    d = cyfa.forward_desc(1, 16, 1, 64, 64, m=257)
    assert lib.cyfa_forward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 2
    assert b"255" in lib.cyfa_last_error()
    # 127 < m <= 255: 256 storage rows; fp32 or d = 64 on the vector-ALU kernel
    d = cyfa.forward_desc(1, 16, 1, 64, 64, m=255)
    assert lib.cyfa_forward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 0
    assert n.value == 256 * 256 * 4
    d = cyfa.forward_desc(1, 16, 1, 256, 64, m=255)
    assert lib.cyfa_forward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 2
    # bf16 with d = 128: the matrix-core kernel (the bf16 readout matrix and its
    # transpose, formed from R directly)
    d = cyfa.forward_desc(1, 16, 3, 128, 128, m=255, dtype=cyfa.BF16)
    assert cyfa.selected_kernel(d) == "mfma"
    assert lib.cyfa_forward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 0
    assert n.value == 2 * 3 * 256 * 256 * 2
    d = cyfa.forward_desc(1, 16, 1, 128, 128, m=129, dtype=cyfa.BF16, kernel=cyfa.KERNEL_MFMA)
    assert lib.cyfa_forward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 0
    # chunk groups (one workgroup each): their bf16 contributions, decays, clocks and a
    # copy of the initial states join the workspace
    d = cyfa.forward_desc(2, 4096, 4, 128, 128, m=255, dtype=cyfa.BF16)
    assert lib.cyfa_forward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 0
    G, BH = 32, 8
    assert n.value == (2 * 4 * 256 * 256 * 2 + BH * G * 2 * 256 * 128 * 2 + BH * G * 4
                       + BH * G * 8 + BH * 2 * 256 * 128 * 4)
    # m <= 63, bf16 with d = 128: the 64-row matrix-core kernel (its 64 x 64 bf16 readout
    # matrix; with chunk groups their bf16 contributions, decays, clocks and rows 0 .. 63
    # of the initial states)
    d = cyfa.forward_desc(1, 16, 3, 128, 128, m=63, dtype=cyfa.BF16)
    assert cyfa.selected_kernel(d) == "mfma"
    assert lib.cyfa_forward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 0
    assert n.value == 3 * 64 * 64 * 2
    d = cyfa.forward_desc(2, 4096, 4, 128, 128, m=63, dtype=cyfa.BF16)
    assert lib.cyfa_forward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 0
    G, BH = 96, 8                                 # ceil(768 / 8) groups of 32-token chunks
    assert n.value == (4 * 64 * 64 * 2 + BH * G * 2 * 64 * 128 * 2 + BH * G * 4 + BH * G * 8
                       + BH * 2 * 64 * 128 * 4)
    d = cyfa.forward_desc(1, 16, 1, 128, 128, m=255, dtype=cyfa.BF16, kernel=cyfa.KERNEL_MFMA, chunk=16)
    assert lib.cyfa_forward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 2
    d = cyfa.forward_desc(1, 16, 1, 96, 64)
    assert lib.cyfa_forward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 2
    assert lib.cyfa_forward_workspace_size(None, ctypes.byref(n)) == 1


def test_matrix_core_head_dims():
    """bf16 with d_k = d_v = 128 (m up to 255) or 256 (m <= 127) selects the
    matrix-core kernel; mixed head dims, d = 256 with m > 127 or fp32 inputs do not,
    and asking for it there fails with CYFA_ERR_UNSUPPORTED.  At 256 the workspace holds two 128 x 128 state
    pairs per head and segment."""
    lib = cyfa.load()
    n = ctypes.c_size_t(0)
    assert cyfa.selected_kernel(cyfa.forward_desc(2, 100, 2, 256, 256, dtype=cyfa.BF16)) == "mfma"
    assert cyfa.selected_kernel(cyfa.forward_desc(2, 100, 2, 128, 128, dtype=cyfa.BF16)) == "mfma"
    assert cyfa.selected_kernel(cyfa.forward_desc(2, 100, 2, 256, 128, dtype=cyfa.BF16)) == "valu"
    assert cyfa.selected_kernel(cyfa.forward_desc(2, 100, 2, 256, 256, dtype=cyfa.F32)) == "valu"
    assert cyfa.selected_kernel(cyfa.forward_desc(2, 100, 2, 256, 256, m=255, dtype=cyfa.BF16)) == "valu"
    for dk, dv, m, dt in ((256, 128, 127, cyfa.BF16), (128, 256, 127, cyfa.BF16),
                          (256, 256, 255, cyfa.BF16), (256, 256, 127, cyfa.F32), (64, 64, 127, cyfa.BF16)):
        d = cyfa.forward_desc(1, 64, 2, dk, dv, m=m, dtype=dt, kernel=cyfa.KERNEL_MFMA)
        assert lib.cyfa_forward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 2, (dk, dv, m, dt)
    w1 = _ws(cyfa.forward_desc(4, 4096, 4, 256, 256, segments=1, kernel=cyfa.KERNEL_MFMA))
    w8 = _ws(cyfa.forward_desc(4, 4096, 4, 256, 256, segments=8, kernel=cyfa.KERNEL_MFMA))
    # bf16 entering states: 2 pairs x 2 x 128 x 128 x 2 bytes per head and extra segment
    assert w8 - w1 >= 7 * 16 * 2 * 2 * 128 * 128 * 2
    h1 = _ws(cyfa.forward_desc(4, 4096, 4, 128, 128, segments=8, kernel=cyfa.KERNEL_MFMA))
    assert w8 > h1


def _call_forward(desc, ptrs, ws=0, ws_bytes=0):
    lib = cyfa.load()
    args = [ptrs.get(k) for k in ("q", "k", "v", "delta", "log_alpha", "beta", "R", "K0", "V0",
                                  "clock0", "o", "K_out", "V_out", "clock_out", "logits")]
    return lib.cyfa_forward(ctypes.byref(desc), *[ctypes.c_void_p(a) if a else None for a in args],
                            ctypes.c_void_p(ws) if ws else None, ctypes.c_size_t(ws_bytes), None)


def test_forward_rejects_before_launch():
    # fake, never dereferenced, suitably aligned addresses: every call below must
    # fail validation before touching the device
    base = 1 << 40
    good = dict(q=base, k=base + (1 << 20), v=base + (2 << 20), delta=base + (3 << 20),
                o=base + (4 << 20))
    d = cyfa.forward_desc(1, 16, 1, 64, 64, dtype=cyfa.F32)
    need = _ws(d)
    assert _call_forward(d, {k: v for k, v in good.items() if k != "q"}, base, need) == 1
    assert _call_forward(d, dict(good, q=base + 8), base, need) == 1          # misaligned
    assert _call_forward(d, good, 0, 0) == 3                                   # no workspace
    assert _call_forward(d, good, base, need - 1) == 3                         # too small
    assert _call_forward(d, good, base + 128, need) == 1                       # ws misaligned
    assert _call_forward(d, dict(good, K_out=base + (5 << 20), V_out=base + (5 << 20)), base, need) == 1
    d.kernel = cyfa.KERNEL_MFMA
    d.dtype = cyfa.F32
    assert _call_forward(d, good, base, need) == 2                             # unsupported


def test_decode_rejects_before_launch():
    lib = cyfa.load()
    d = cyfa.decode_desc(2, 2, 64, 64)
    args = [None] * 13
    st = lib.cyfa_decode_step(ctypes.byref(d), *args, ctypes.c_size_t(0), None)
    assert st == 1
    d = cyfa.decode_desc(2, 2, 64, 64, m=4)
    st = lib.cyfa_decode_step(ctypes.byref(d), *args, ctypes.c_size_t(0), None)
    assert st == 1


def test_decode_noalloc_rejects_before_launch():
    """The no-allocation decode step validates like cyfa_decode_step and refuses a
    readout scratch larger than its fixed array, all before any HIP call."""
    lib = cyfa.load()
    d = cyfa.decode_desc(2, 2, 64, 64)
    assert lib.cyfa_decode_step_noalloc(ctypes.byref(d), *([None] * 13)) == 1
    d = cyfa.decode_desc(2, 2, 64, 64, m=4)
    assert lib.cyfa_decode_step_noalloc(ctypes.byref(d), *([None] * 13)) == 1
    base = 1 << 30                                   # fake, aligned, never dereferenced
    ptr = lambda i: ctypes.c_void_p(base + (i << 24))  # noqa: E731
    args = [ptr(i) for i in range(4)] + [None, None, None] + [ptr(i) for i in range(4, 8)] + [None]
    for H, m in ((65, 127), (17, 255)):              # 4 MiB + 64 KiB, 4 MiB + 256 KiB of readout matrices
        d = cyfa.decode_desc(1, H, 128, 128, m=m)
        assert lib.cyfa_decode_step_noalloc(ctypes.byref(d), *args, None) == 2
        assert b"exceeds" in lib.cyfa_last_error()
    bad = list(args)
    bad[0] = ctypes.c_void_p(base + 8)               # misaligned q
    d = cyfa.decode_desc(1, 4, 128, 128)
    assert lib.cyfa_decode_step_noalloc(ctypes.byref(d), *bad, None) == 1


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(cyfa, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(cyfa, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        cyfa.load()


def _call_backward(desc, ptrs, ws=0, ws_bytes=0):
    lib = cyfa.load()
    names = ("q", "k", "v", "delta", "log_alpha", "beta", "R", "lens", "K0", "V0", "clock0", "d_o",
             "dK_T", "dV_T", "dq", "dk", "dv", "d_delta", "d_log_alpha", "d_beta", "d_R", "d_K0",
             "d_V0", "d_clock0")
    args = [ptrs.get(k) for k in names]
    return lib.cyfa_backward(ctypes.byref(desc), *[ctypes.c_void_p(a) if a else None for a in args],
                             ctypes.c_void_p(ws) if ws else None, ctypes.c_size_t(ws_bytes), None)


def test_backward_workspace_and_descriptor_checks():
    d = cyfa.forward_desc(4, 4096, 16, 128, 128, dtype=cyfa.BF16, kernel=cyfa.KERNEL_VALU)
    n = cyfa.backward_workspace_size(d)
    # vector-ALU: entering and adjoint states per 16-token chunk dominate, ~4.3 GB at this shape
    assert 4.0e9 < n < 5.0e9
    # matrix-core (the automatic choice here): u and dp per token in bf16 (2 x 67 MB), the
    # forward and adjoint states per chunk group (2 x 34 MB), the groups' dM (17 MB)
    d = cyfa.forward_desc(4, 4096, 16, 128, 128, dtype=cyfa.BF16)
    n = cyfa.backward_workspace_size(d)
    assert 2.0e8 < n < 2.6e8, n
    for field, value in (("d_k", 256), ("kernel", cyfa.KERNEL_MFMA), ("chunk", 32), ("m", 255)):
        d = cyfa.forward_desc(1, 64, 2, 64, 64, dtype=cyfa.F32)
        setattr(d, field, value)
        with pytest.raises(cyfa.CyfaError) as ei:
            cyfa.backward_workspace_size(d)
        assert ei.value.status == 2, (field, ei.value)


def test_backward_rejects_before_launch():
    base = 1 << 40
    slot = iter(range(1, 64))
    good = {k: base + (next(slot) << 20) for k in ("q", "k", "v", "delta", "d_o", "dq", "dk", "dv",
                                                   "d_delta")}
    d = cyfa.forward_desc(1, 16, 1, 64, 64, dtype=cyfa.F32)
    need = cyfa.backward_workspace_size(d)
    assert _call_backward(d, {k: v for k, v in good.items() if k != "d_o"}, base, need) == 1
    assert _call_backward(d, dict(good, d_beta=base + (40 << 20)), base, need) == 1   # no beta
    assert _call_backward(d, dict(good, d_R=base + (41 << 20)), base, need) == 1      # no R
    assert _call_backward(d, dict(good, dq=good["dk"]), base, need) == 1             # aliasing
    assert _call_backward(d, dict(good, dq=good["q"]), base, need) == 1
    assert _call_backward(d, dict(good, q=base + 8), base, need) == 1                # misaligned
    assert _call_backward(d, good, 0, 0) == 3
    assert _call_backward(d, good, base, need - 1) == 3


def _call_prologue(desc, ptrs):
    lib = cyfa.load()
    names = ("q_in", "k_in", "v_in", "conv_q", "conv_k", "conv_v", "norm_q", "norm_k", "z_delta",
             "b_delta", "z_alpha", "b_alpha", "A", "z_beta", "lens", "q", "k", "v", "delta",
             "log_alpha", "beta")
    args = [ptrs.get(k) for k in names]
    return lib.cyfa_mixer_prologue(ctypes.byref(desc), *[ctypes.c_void_p(a) if a else None for a in args], None)


def test_mixer_rejects_before_launch():
    base = 1 << 40
    slot = iter(range(1, 64))
    good = {k: base + (next(slot) << 20) for k in ("q_in", "k_in", "v_in", "q", "k", "v")}
    d = cyfa.MixDesc(1, 16, 2, 64, 64, 4, 0, 1e-6, cyfa.F32)
    assert _call_prologue(d, {k: v for k, v in good.items() if k != "q"}) == 1
    assert _call_prologue(d, dict(good, z_alpha=base + (40 << 20), log_alpha=base + (41 << 20))) == 1  # no A
    assert _call_prologue(d, dict(good, z_delta=base + (42 << 20))) == 1                            # no output
    assert _call_prologue(d, dict(good, q=good["q_in"])) == 1                                       # aliasing
    assert _call_prologue(d, dict(good, q_in=base + 8)) == 1                                        # misaligned
    for field, value, status in (("conv_size", 5, 2), ("conv_size", 0, 2), ("conv_act", 2, 1),
                                 ("eps", 0.0, 1), ("d_k", 96, 2), ("dtype", 7, 1)):
        bad = cyfa.MixDesc(1, 16, 2, 64, 64, 4, 0, 1e-6, cyfa.F32)
        setattr(bad, field, value)
        assert _call_prologue(bad, good) == status, field
    lib = cyfa.load()
    out = base + (50 << 20)
    assert lib.cyfa_mixer_epilogue(ctypes.byref(d), ctypes.c_void_p(out), None, None, None,
                                   ctypes.c_void_p(out), None) == 1                             # out aliases o
