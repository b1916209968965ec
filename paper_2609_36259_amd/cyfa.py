"""Thin Python binding of libcyfa.so (the C ABI in include/cyfa.h).

Argument marshalling only: tensors are torch CUDA (HIP) tensors, the work is
enqueued on torch's current stream, and every step of the operator runs in the
library's HIP kernels.  There is no fallback: if the library is missing the
calls raise.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcyfa.so")

F32, BF16 = 0, 1
KERNEL_AUTO, KERNEL_VALU, KERNEL_MFMA = 0, 1, 2
STATUS = {0: "CYFA_OK", 1: "CYFA_ERR_INVALID_ARGUMENT", 2: "CYFA_ERR_UNSUPPORTED",
          3: "CYFA_ERR_WORKSPACE", 4: "CYFA_ERR_LAUNCH"}
STORE_ROWS = 128


def store_rows(m: int) -> int:
    """Storage rows of the states: 128 for m <= 127, 256 for 127 < m <= 255."""
    return STORE_ROWS if m <= 127 else 2 * STORE_ROWS

# Every symbol include/cyfa.h declares.
EXPORTED = ("cyfa_forward_workspace_size", "cyfa_forward", "cyfa_forward_lens", "cyfa_forward_varlen",
            "cyfa_forward_mixer", "cyfa_forward_mixer_workspace_size",
            "cyfa_backward_workspace_size", "cyfa_backward", "cyfa_mixer_prologue",
            "cyfa_mixer_epilogue", "cyfa_decode_workspace_size", "cyfa_decode_step",
            "cyfa_decode_step_noalloc", "cyfa_set_timing_events",
            "cyfa_status_string", "cyfa_last_error", "cyfa_version")


class CyfaError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{STATUS.get(status, status)}: {detail}")
        self.status = status
        self.detail = detail


class FwdDesc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("T", ctypes.c_int32), ("H", ctypes.c_int32),
                ("d_k", ctypes.c_int32), ("d_v", ctypes.c_int32), ("m", ctypes.c_int32),
                ("chunk", ctypes.c_int32), ("segments", ctypes.c_int32),
                ("scale", ctypes.c_float), ("dtype", ctypes.c_int32), ("kernel", ctypes.c_int32)]


class MixDesc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("T", ctypes.c_int32), ("H", ctypes.c_int32),
                ("d_k", ctypes.c_int32), ("d_v", ctypes.c_int32), ("conv_size", ctypes.c_int32),
                ("conv_act", ctypes.c_int32), ("eps", ctypes.c_float), ("dtype", ctypes.c_int32)]


class MixWeights(ctypes.Structure):
    _fields_ = [("conv_size", ctypes.c_int32), ("conv_act", ctypes.c_int32), ("eps", ctypes.c_float),
                ("fuse_conv", ctypes.c_int32)] + \
        [(n, ctypes.c_void_p) for n in ("conv_q", "conv_k", "conv_v", "norm_q", "norm_k", "z_delta", "b_delta",
                                         "z_alpha", "b_alpha", "A", "z_beta", "gate", "norm_o")]


class DecDesc(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int32), ("H", ctypes.c_int32), ("d_k", ctypes.c_int32),
                ("d_v", ctypes.c_int32), ("m", ctypes.c_int32), ("scale", ctypes.c_float),
                ("dtype", ctypes.c_int32)]


_lib = None
_vp = ctypes.c_void_p


def load() -> ctypes.CDLL:
    """Load libcyfa.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "or python -m paper_2609_36259_amd.build")
        lib = ctypes.CDLL(LIB_PATH)
        lib.cyfa_forward_workspace_size.argtypes = [ctypes.POINTER(FwdDesc),
                                                    ctypes.POINTER(ctypes.c_size_t)]
        lib.cyfa_forward_workspace_size.restype = ctypes.c_int
        lib.cyfa_forward.argtypes = [ctypes.POINTER(FwdDesc)] + [_vp] * 16 + [ctypes.c_size_t, _vp]
        lib.cyfa_forward.restype = ctypes.c_int
        lib.cyfa_forward_lens.argtypes = [ctypes.POINTER(FwdDesc)] + [_vp] * 17 + [ctypes.c_size_t, _vp]
        lib.cyfa_forward_lens.restype = ctypes.c_int
        lib.cyfa_forward_varlen.argtypes = [ctypes.POINTER(FwdDesc)] + [_vp] * 17 + [ctypes.c_size_t, _vp]
        lib.cyfa_forward_varlen.restype = ctypes.c_int
        lib.cyfa_forward_mixer.argtypes = [ctypes.POINTER(FwdDesc), ctypes.POINTER(MixWeights)] + \
            [_vp] * 14 + [ctypes.c_size_t, _vp]
        lib.cyfa_forward_mixer.restype = ctypes.c_int
        lib.cyfa_forward_mixer_workspace_size.argtypes = [ctypes.POINTER(FwdDesc), ctypes.POINTER(MixWeights),
                                                          ctypes.POINTER(ctypes.c_size_t)]
        lib.cyfa_forward_mixer_workspace_size.restype = ctypes.c_int
        lib.cyfa_backward_workspace_size.argtypes = [ctypes.POINTER(FwdDesc),
                                                     ctypes.POINTER(ctypes.c_size_t)]
        lib.cyfa_backward_workspace_size.restype = ctypes.c_int
        lib.cyfa_backward.argtypes = [ctypes.POINTER(FwdDesc)] + [_vp] * 25 + [ctypes.c_size_t, _vp]
        lib.cyfa_backward.restype = ctypes.c_int
        lib.cyfa_mixer_prologue.argtypes = [ctypes.POINTER(MixDesc)] + [_vp] * 22
        lib.cyfa_mixer_prologue.restype = ctypes.c_int
        lib.cyfa_mixer_epilogue.argtypes = [ctypes.POINTER(MixDesc)] + [_vp] * 6
        lib.cyfa_mixer_epilogue.restype = ctypes.c_int
        lib.cyfa_decode_workspace_size.argtypes = [ctypes.POINTER(DecDesc),
                                                   ctypes.POINTER(ctypes.c_size_t)]
        lib.cyfa_decode_workspace_size.restype = ctypes.c_int
        lib.cyfa_decode_step.argtypes = [ctypes.POINTER(DecDesc)] + [_vp] * 13 + [ctypes.c_size_t, _vp]
        lib.cyfa_decode_step.restype = ctypes.c_int
        lib.cyfa_decode_step_noalloc.argtypes = [ctypes.POINTER(DecDesc)] + [_vp] * 13
        lib.cyfa_decode_step_noalloc.restype = ctypes.c_int
        lib.cyfa_status_string.argtypes = [ctypes.c_int]
        lib.cyfa_status_string.restype = ctypes.c_char_p
        lib.cyfa_last_error.argtypes = []
        lib.cyfa_last_error.restype = ctypes.c_char_p
        lib.cyfa_set_timing_events.argtypes = [_vp, _vp]
        lib.cyfa_set_timing_events.restype = ctypes.c_int
        lib.cyfa_version.argtypes = []
        lib.cyfa_version.restype = ctypes.c_int32
        _lib = lib
    return _lib


def _check(status: int):
    if status != 0:
        raise CyfaError(status, load().cyfa_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"q/k/v must be float32 or bfloat16, got {t.dtype}")


def _need(t, shape, dtype, name):
    if t is None:
        return None
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    return t


def _stream_handle(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def set_timing_events(start_event, stop_event):
    """Install (or clear with None, None) hipEvent_t handles recorded around the main kernel."""
    _check(load().cyfa_set_timing_events(start_event, stop_event))


def forward_desc(B, T, H, dk, dv, *, m=127, chunk=0, segments=0, scale=None, dtype=BF16,
                 kernel=KERNEL_AUTO) -> FwdDesc:
    return FwdDesc(B, T, H, dk, dv, m, chunk, segments,
                   float(dk ** -0.5 if scale is None else scale), dtype, kernel)


def forward_workspace_size(desc: FwdDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(load().cyfa_forward_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def selected_kernel(desc: FwdDesc) -> str:
    """Which kernel a forward with this descriptor runs: "mfma" or "valu"."""
    if desc.kernel == KERNEL_VALU:
        return "valu"
    if desc.kernel == KERNEL_MFMA:
        return "mfma"
    trial = FwdDesc.from_buffer_copy(desc)
    trial.kernel = KERNEL_MFMA
    n = ctypes.c_size_t(0)
    ok = load().cyfa_forward_workspace_size(ctypes.byref(trial), ctypes.byref(n)) == 0
    return "mfma" if ok and desc.chunk in (0, 32, 64) else "valu"


DEFAULT_CHUNK = {"mfma": 32, "valu": 16}


def forward(q, k, v, delta, log_alpha=None, beta=None, R=None, *, scale=None, m=127,
            chunk=0, segments=0, kernel=KERNEL_AUTO, K0=None, V0=None, clock0=None,
            lens=None, return_state=False, return_logits=False, out=None, workspace=None,
            K_out=None, V_out=None, clock_out=None, stream=None):
    """CyFA forward: q,k [B,T,H,dk], v [B,T,H,dv] (float32 or bfloat16), scalars [B,T,H] float32.

    ``lens`` (optional int32 [B] device tensor): sequence b has lens[b] tokens
    (cyfa_forward_lens); rows t >= lens[b] of the outputs are not written.
    Returns ``o`` [B,T,H,dv] (dtype of q) or a dict with ``o`` and, when requested,
    the final absolute-clock states ``K``/``V`` [B,H,S,d] (S = store_rows(m)), ``clock`` [B,H] (float64)
    and the slot ``logits`` [B,T,H,m].  ``K_out``/``V_out``/``clock_out``, when given, receive
    the final state (they may be ``K0``/``V0``/``clock0`` themselves: resume in place) and
    imply ``return_state``.
    """
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    dt = _dtype_code(q)
    _need(q, (B, T, H, dk), q.dtype, "q")
    _need(k, (B, T, H, dk), q.dtype, "k")
    _need(v, (B, T, H, dv), q.dtype, "v")
    for name, t in (("delta", delta), ("log_alpha", log_alpha), ("beta", beta)):
        _need(t, (B, T, H), torch.float32, name)
    _need(R, (H, m, m), torch.float32, "R")
    S = store_rows(m)
    _need(K0, (B, H, S, dk), torch.float32, "K0")
    _need(V0, (B, H, S, dv), torch.float32, "V0")
    _need(clock0, (B, H), torch.float64, "clock0")
    _need(lens, (B,), torch.int32, "lens")
    desc = forward_desc(B, T, H, dk, dv, m=m, chunk=chunk, segments=segments, scale=scale,
                        dtype=dt, kernel=kernel)
    nbytes = forward_workspace_size(desc)
    dev = q.device
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    o = out if out is not None else torch.empty((B, T, H, dv), dtype=q.dtype, device=dev)
    _need(o, (B, T, H, dv), q.dtype, "out")
    if K_out is not None or V_out is not None or clock_out is not None:
        return_state = True
    _need(K_out, (B, H, S, dk), torch.float32, "K_out")
    _need(V_out, (B, H, S, dv), torch.float32, "V_out")
    _need(clock_out, (B, H), torch.float64, "clock_out")
    if return_state:
        if K_out is None:
            K_out = torch.empty((B, H, S, dk), dtype=torch.float32, device=dev)
        if V_out is None:
            V_out = torch.empty((B, H, S, dv), dtype=torch.float32, device=dev)
    clk = clock_out
    if return_state and clk is None:
        clk = torch.empty((B, H), dtype=torch.float64, device=dev)
    logits = torch.empty((B, T, H, m), dtype=torch.float32, device=dev) if return_logits else None
    st = load().cyfa_forward_lens(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(delta),
                                  _ptr(log_alpha), _ptr(beta), _ptr(R), _ptr(lens), _ptr(K0),
                                  _ptr(V0), _ptr(clock0), _ptr(o), _ptr(K_out), _ptr(V_out),
                                  _ptr(clk), _ptr(logits), _ptr(workspace),
                                  ctypes.c_size_t(workspace.numel()), _stream_handle(stream))
    _check(st)
    if not (return_state or return_logits):
        return o
    res = {"o": o}
    if return_state:
        res.update(K=K_out, V=V_out, clock=clk)
    if return_logits:
        res["logits"] = logits
    return res


def forward_varlen(q, k, v, delta, cu_seqlens, log_alpha=None, beta=None, R=None, *, max_len,
                   scale=None, m=127, chunk=0, segments=0, kernel=KERNEL_AUTO, K0=None, V0=None,
                   clock0=None, return_state=False, return_logits=False, out=None, workspace=None,
                   stream=None):
    """CyFA forward over packed sequences (cyfa_forward_varlen): q,k [total,H,dk],
    v [total,H,dv], scalars [total,H]; ``cu_seqlens`` int32 [B+1] device offsets;
    ``max_len`` the longest sequence.  States are per sequence ([B,H,S,d], clock [B,H]).
    Returns ``o`` [total,H,dv] or a dict as ``forward``."""
    total, H, dk = q.shape
    dv = v.shape[-1]
    B = cu_seqlens.shape[0] - 1
    dt = _dtype_code(q)
    _need(q, (total, H, dk), q.dtype, "q")
    _need(k, (total, H, dk), q.dtype, "k")
    _need(v, (total, H, dv), q.dtype, "v")
    for name, t in (("delta", delta), ("log_alpha", log_alpha), ("beta", beta)):
        _need(t, (total, H), torch.float32, name)
    _need(R, (H, m, m), torch.float32, "R")
    _need(cu_seqlens, (B + 1,), torch.int32, "cu_seqlens")
    S = store_rows(m)
    _need(K0, (B, H, S, dk), torch.float32, "K0")
    _need(V0, (B, H, S, dv), torch.float32, "V0")
    _need(clock0, (B, H), torch.float64, "clock0")
    desc = forward_desc(B, int(max_len), H, dk, dv, m=m, chunk=chunk, segments=segments, scale=scale,
                        dtype=dt, kernel=kernel)
    nbytes = forward_workspace_size(desc)
    dev = q.device
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    o = out if out is not None else torch.empty((total, H, dv), dtype=q.dtype, device=dev)
    _need(o, (total, H, dv), q.dtype, "out")
    K_out = torch.empty((B, H, S, dk), dtype=torch.float32, device=dev) if return_state else None
    V_out = torch.empty((B, H, S, dv), dtype=torch.float32, device=dev) if return_state else None
    clk = torch.empty((B, H), dtype=torch.float64, device=dev) if return_state else None
    logits = torch.empty((total, H, m), dtype=torch.float32, device=dev) if return_logits else None
    st = load().cyfa_forward_varlen(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(delta),
                                    _ptr(log_alpha), _ptr(beta), _ptr(R), _ptr(cu_seqlens), _ptr(K0),
                                    _ptr(V0), _ptr(clock0), _ptr(o), _ptr(K_out), _ptr(V_out),
                                    _ptr(clk), _ptr(logits), _ptr(workspace),
                                    ctypes.c_size_t(workspace.numel()), _stream_handle(stream))
    _check(st)
    if not (return_state or return_logits):
        return o
    res = {"o": o}
    if return_state:
        res.update(K=K_out, V=V_out, clock=clk)
    if return_logits:
        res["logits"] = logits
    return res


def backward_workspace_size(desc: FwdDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(load().cyfa_backward_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def backward(q, k, v, delta, log_alpha=None, beta=None, R=None, *, d_o, scale=None, m=127,
             K0=None, V0=None, clock0=None, dK_T=None, dV_T=None, lens=None, groups=0,
             want_state_grads=True, kernel=KERNEL_AUTO, workspace=None, stream=None):
    """Gradients of sum <d_o, o> + <dK_T, K_out> + <dV_T, V_out> (cyfa_backward).

    Inputs as for ``forward``; ``d_o`` [B,T,H,dv] in q's dtype; ``dK_T``/``dV_T``
    [B,H,128,d] float32 or None.  Returns a dict with dq, dk, dv (q's dtype),
    d_delta, d_log_alpha / d_beta (None when the input is None), d_R (None without
    R) and, with ``want_state_grads``, d_K0, d_V0 [B,H,128,d] and d_clock0 [B,H].
    ``kernel``: KERNEL_AUTO (the matrix-core backward for bf16 with d = 128, else
    the vector-ALU one), KERNEL_VALU or KERNEL_MFMA.
    """
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    dt = _dtype_code(q)
    _need(q, (B, T, H, dk), q.dtype, "q")
    _need(k, (B, T, H, dk), q.dtype, "k")
    _need(v, (B, T, H, dv), q.dtype, "v")
    _need(d_o, (B, T, H, dv), q.dtype, "d_o")
    for name, t in (("delta", delta), ("log_alpha", log_alpha), ("beta", beta)):
        _need(t, (B, T, H), torch.float32, name)
    _need(R, (H, m, m), torch.float32, "R")
    _need(K0, (B, H, STORE_ROWS, dk), torch.float32, "K0")
    _need(V0, (B, H, STORE_ROWS, dv), torch.float32, "V0")
    _need(dK_T, (B, H, STORE_ROWS, dk), torch.float32, "dK_T")
    _need(dV_T, (B, H, STORE_ROWS, dv), torch.float32, "dV_T")
    _need(clock0, (B, H), torch.float64, "clock0")
    _need(lens, (B,), torch.int32, "lens")
    desc = forward_desc(B, T, H, dk, dv, m=m, chunk=0, segments=groups, scale=scale, dtype=dt,
                        kernel=kernel)
    nbytes = backward_workspace_size(desc)
    dev = q.device
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    e = lambda *shape, dtype=torch.float32: torch.empty(shape, dtype=dtype, device=dev)  # noqa: E731
    g = {"dq": e(B, T, H, dk, dtype=q.dtype), "dk": e(B, T, H, dk, dtype=q.dtype),
         "dv": e(B, T, H, dv, dtype=q.dtype), "d_delta": e(B, T, H),
         "d_log_alpha": e(B, T, H) if log_alpha is not None else None,
         "d_beta": e(B, T, H) if beta is not None else None,
         "d_R": e(H, m, m) if R is not None else None,
         "d_K0": e(B, H, STORE_ROWS, dk) if want_state_grads else None,
         "d_V0": e(B, H, STORE_ROWS, dv) if want_state_grads else None,
         "d_clock0": e(B, H, dtype=torch.float64) if want_state_grads else None}
    st = load().cyfa_backward(
        ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(delta), _ptr(log_alpha), _ptr(beta),
        _ptr(R), _ptr(lens), _ptr(K0), _ptr(V0), _ptr(clock0), _ptr(d_o), _ptr(dK_T), _ptr(dV_T),
        _ptr(g["dq"]), _ptr(g["dk"]), _ptr(g["dv"]), _ptr(g["d_delta"]), _ptr(g["d_log_alpha"]),
        _ptr(g["d_beta"]), _ptr(g["d_R"]), _ptr(g["d_K0"]), _ptr(g["d_V0"]), _ptr(g["d_clock0"]),
        _ptr(workspace), ctypes.c_size_t(workspace.numel()), _stream_handle(stream))
    _check(st)
    return g


def mixer_prologue(q_in, k_in, v_in, *, conv_q=None, conv_k=None, conv_v=None, norm_q=None,
                   norm_k=None, z_delta=None, b_delta=None, z_alpha=None, b_alpha=None, A=None,
                   z_beta=None, lens=None, conv_size=4, conv_act=0, eps=1e-6, stream=None):
    """ShortConv (+ SiLU) of q, k, v, RMSNorm of q and k, and the gate activations
    (cyfa_mixer_prologue).  Returns q, k, v and delta / log_alpha / beta (None where
    the projection is None)."""
    B, T, H, dk = q_in.shape
    dv = v_in.shape[-1]
    _need(k_in, (B, T, H, dk), q_in.dtype, "k_in")
    _need(v_in, (B, T, H, dv), q_in.dtype, "v_in")
    for name, t, d in (("conv_q", conv_q, dk), ("conv_k", conv_k, dk), ("conv_v", conv_v, dv)):
        _need(t, (H * d, conv_size), torch.float32, name)
    _need(norm_q, (dk,), torch.float32, "norm_q")
    _need(norm_k, (dk,), torch.float32, "norm_k")
    for name, t in (("z_delta", z_delta), ("z_alpha", z_alpha), ("z_beta", z_beta)):
        _need(t, (B, T, H), torch.float32, name)
    for name, t in (("b_delta", b_delta), ("b_alpha", b_alpha), ("A", A)):
        _need(t, (H,), torch.float32, name)
    _need(lens, (B,), torch.int32, "lens")
    desc = MixDesc(B, T, H, dk, dv, conv_size, conv_act, eps, _dtype_code(q_in))
    dev = q_in.device
    out = {"q": torch.empty_like(q_in), "k": torch.empty_like(k_in), "v": torch.empty_like(v_in)}
    for name, z in (("delta", z_delta), ("log_alpha", z_alpha), ("beta", z_beta)):
        out[name] = torch.empty((B, T, H), dtype=torch.float32, device=dev) if z is not None else None
    st = load().cyfa_mixer_prologue(
        ctypes.byref(desc), _ptr(q_in), _ptr(k_in), _ptr(v_in), _ptr(conv_q), _ptr(conv_k),
        _ptr(conv_v), _ptr(norm_q), _ptr(norm_k), _ptr(z_delta), _ptr(b_delta), _ptr(z_alpha),
        _ptr(b_alpha), _ptr(A), _ptr(z_beta), _ptr(lens), _ptr(out["q"]), _ptr(out["k"]),
        _ptr(out["v"]), _ptr(out["delta"]), _ptr(out["log_alpha"]), _ptr(out["beta"]),
        _stream_handle(stream))
    _check(st)
    return out


def mixer_epilogue(o, gate=None, norm_o=None, *, lens=None, eps=1e-6, out=None, stream=None):
    """RMSNorm(o) * norm_o * sigmoid(gate) per head vector (cyfa_mixer_epilogue)."""
    B, T, H, dv = o.shape
    _need(gate, (B, T, H, dv), o.dtype, "gate")
    _need(norm_o, (dv,), torch.float32, "norm_o")
    _need(lens, (B,), torch.int32, "lens")
    res = out if out is not None else torch.empty_like(o)
    _need(res, (B, T, H, dv), o.dtype, "out")
    desc = MixDesc(B, T, H, dv, dv, 1, 0, eps, _dtype_code(o))
    _check(load().cyfa_mixer_epilogue(ctypes.byref(desc), _ptr(o), _ptr(gate), _ptr(norm_o),
                                      _ptr(lens), _ptr(res), _stream_handle(stream)))
    return res


def forward_mixer(q_in, k_in, v_in, z_delta, *, conv_q=None, conv_k=None, conv_v=None, norm_q=None,
                  norm_k=None, b_delta=None, z_alpha=None, b_alpha=None, A=None, z_beta=None, gate=None,
                  norm_o=None, R=None, scale=None, m=127, segments=0, lens=None, conv_size=4, conv_act=0,
                  eps=1e-6, fuse_conv=0, K0=None, V0=None, clock0=None, return_state=False,
                  return_logits=False, out=None, workspace=None, stream=None):
    """Layer forward (cyfa_forward_mixer): mixer prologue, the operator and the mixer
    epilogue in one pass; bf16 q_in, k_in, v_in [B,T,H,128].  Returns ``out``
    [B,T,H,128] bf16, or a dict with ``out`` and the final state / logits as
    ``forward`` returns them."""
    B, T, H, d = q_in.shape
    if q_in.dtype != torch.bfloat16:
        raise CyfaError(2, "the layer forward takes bf16 projections")
    _need(k_in, (B, T, H, d), q_in.dtype, "k_in")
    _need(v_in, (B, T, H, d), q_in.dtype, "v_in")
    for name, t in (("conv_q", conv_q), ("conv_k", conv_k), ("conv_v", conv_v)):
        _need(t, (H * d, conv_size), torch.float32, name)
    for name, t in (("norm_q", norm_q), ("norm_k", norm_k), ("norm_o", norm_o)):
        _need(t, (d,), torch.float32, name)
    for name, t in (("z_delta", z_delta), ("z_alpha", z_alpha), ("z_beta", z_beta)):
        _need(t, (B, T, H), torch.float32, name)
    for name, t in (("b_delta", b_delta), ("b_alpha", b_alpha), ("A", A)):
        _need(t, (H,), torch.float32, name)
    _need(gate, (B, T, H, d), q_in.dtype, "gate")
    _need(R, (H, m, m), torch.float32, "R")
    _need(lens, (B,), torch.int32, "lens")
    S = store_rows(m)
    _need(K0, (B, H, S, d), torch.float32, "K0")
    _need(V0, (B, H, S, d), torch.float32, "V0")
    _need(clock0, (B, H), torch.float64, "clock0")
    desc = forward_desc(B, T, H, d, d, m=m, segments=segments, scale=scale, dtype=BF16, kernel=KERNEL_MFMA)
    mw = MixWeights(conv_size, conv_act, eps, int(fuse_conv),
                    *[_ptr(t) for t in (conv_q, conv_k, conv_v, norm_q, norm_k, z_delta, b_delta, z_alpha, b_alpha,
                                        A, z_beta, gate, norm_o)])
    n = ctypes.c_size_t(0)
    _check(load().cyfa_forward_mixer_workspace_size(ctypes.byref(desc), ctypes.byref(mw), ctypes.byref(n)))
    nbytes = n.value
    dev = q_in.device
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    res_out = out if out is not None else torch.empty_like(q_in)
    _need(res_out, (B, T, H, d), q_in.dtype, "out")
    K_out = V_out = clk = None
    if return_state:
        K_out = torch.empty((B, H, S, d), dtype=torch.float32, device=dev)
        V_out = torch.empty((B, H, S, d), dtype=torch.float32, device=dev)
        clk = torch.empty((B, H), dtype=torch.float64, device=dev)
    logits = torch.empty((B, T, H, m), dtype=torch.float32, device=dev) if return_logits else None
    _check(load().cyfa_forward_mixer(ctypes.byref(desc), ctypes.byref(mw), _ptr(q_in), _ptr(k_in), _ptr(v_in),
                                     _ptr(R), _ptr(lens), _ptr(K0), _ptr(V0), _ptr(clock0), _ptr(res_out),
                                     _ptr(K_out), _ptr(V_out), _ptr(clk), _ptr(logits), _ptr(workspace),
                                     ctypes.c_size_t(workspace.numel()), _stream_handle(stream)))
    if not (return_state or return_logits):
        return res_out
    res = {"out": res_out}
    if return_state:
        res.update(K=K_out, V=V_out, clock=clk)
    if return_logits:
        res["logits"] = logits
    return res


def decode_desc(N, H, dk, dv, *, m=127, scale=None, dtype=F32) -> DecDesc:
    return DecDesc(N, H, dk, dv, m, float(dk ** -0.5 if scale is None else scale), dtype)


def decode_workspace_size(desc: DecDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(load().cyfa_decode_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def decode_step(q, k, v, delta, K, V, clock, log_alpha=None, beta=None, R=None, *, scale=None,
                m=127, return_logits=False, out=None, workspace=None, stream=None):
    """One in-place decode step: q,k [N,H,dk], v [N,H,dv]; scalars [N,H] float32;
    states K [N,H,S,dk], V [N,H,S,dv] float32 (S = store_rows(m)) and clock [N,H] float64 (updated)."""
    N, H, dk = q.shape
    dv = v.shape[-1]
    dt = _dtype_code(q)
    _need(k, (N, H, dk), q.dtype, "k")
    _need(v, (N, H, dv), q.dtype, "v")
    for name, t in (("delta", delta), ("log_alpha", log_alpha), ("beta", beta)):
        _need(t, (N, H), torch.float32, name)
    _need(R, (H, m, m), torch.float32, "R")
    _need(K, (N, H, store_rows(m), dk), torch.float32, "K")
    _need(V, (N, H, store_rows(m), dv), torch.float32, "V")
    _need(clock, (N, H), torch.float64, "clock")
    desc = decode_desc(N, H, dk, dv, m=m, scale=scale, dtype=dt)
    nbytes = decode_workspace_size(desc)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    o = out if out is not None else torch.empty((N, H, dv), dtype=q.dtype, device=q.device)
    _need(o, (N, H, dv), q.dtype, "out")
    logits = torch.empty((N, H, m), dtype=torch.float32, device=q.device) if return_logits else None
    st = load().cyfa_decode_step(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(delta),
                                 _ptr(log_alpha), _ptr(beta), _ptr(R), _ptr(K), _ptr(V),
                                 _ptr(clock), _ptr(o), _ptr(logits), _ptr(workspace),
                                 ctypes.c_size_t(workspace.numel()), _stream_handle(stream))
    _check(st)
    return (o, logits) if return_logits else o


DECODE_NOALLOC_SCRATCH_BYTES = 4 << 20


def decode_step_noalloc(q, k, v, delta, K, V, clock, log_alpha=None, beta=None, R=None, *,
                        scale=None, m=127, out, logits_out=None, stream=None):
    """``decode_step`` through cyfa_decode_step_noalloc: no workspace, the library's
    fixed per-GPU scratch array instead.  The caller passes every output (``out``
    [N,H,dv] in q's dtype, optional ``logits_out`` [N,H,m] float32), so this call
    allocates nothing either.  Returns ``out``."""
    N, H, dk = q.shape
    dv = v.shape[-1]
    dt = _dtype_code(q)
    _need(k, (N, H, dk), q.dtype, "k")
    _need(v, (N, H, dv), q.dtype, "v")
    for name, t in (("delta", delta), ("log_alpha", log_alpha), ("beta", beta)):
        _need(t, (N, H), torch.float32, name)
    _need(R, (H, m, m), torch.float32, "R")
    _need(K, (N, H, store_rows(m), dk), torch.float32, "K")
    _need(V, (N, H, store_rows(m), dv), torch.float32, "V")
    _need(clock, (N, H), torch.float64, "clock")
    _need(out, (N, H, dv), q.dtype, "out")
    _need(logits_out, (N, H, m), torch.float32, "logits_out")
    desc = decode_desc(N, H, dk, dv, m=m, scale=scale, dtype=dt)
    st = load().cyfa_decode_step_noalloc(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(delta),
                                         _ptr(log_alpha), _ptr(beta), _ptr(R), _ptr(K), _ptr(V),
                                         _ptr(clock), _ptr(out), _ptr(logits_out),
                                         _stream_handle(stream))
    _check(st)
    return out
