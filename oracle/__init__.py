"""CyFA CPU oracle (ctypes wrapper around ``cyfa_oracle.c``).

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only ``tests/``, the package's
``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline`` leg may import
this package.  The GPU operator never calls it and shares no code with it.

The oracle evaluates the relative-time-slot recurrence and softmax readout of
Sec. 3.1 (Eqs. cyfa-physical-recurrence and cyfa-physical-readout) in double
precision, one token at a time, with the fractional cyclic shift
P(tau) = Phi U(tau) Phi^T of Eq. cyfa-fractional-shift rebuilt densely at every
token (real Fourier basis of App. A.1, Eq. app-real-fourier).

``oracle.backward`` gives the gradients of the same definition (reverse-mode
differentiation of a float64 token-by-token evaluation with torch on the CPU).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cyfa_oracle.c")
# CYFA_ORACLE_LIB points the wrapper at another build of the same source (the
# mutation check of tests/test_oracle_mutations.py loads deliberately broken copies)
_LIB = os.environ.get("CYFA_ORACLE_LIB") or os.path.join(_HERE, "libcyfa_oracle.so")
_lib = None

_dp = ctypes.POINTER(ctypes.c_double)
_fp = ctypes.POINTER(ctypes.c_float)
_ip = ctypes.POINTER(ctypes.c_int32)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (fp64, OpenMP).  Returns the library path."""
    global _lib
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O3", "-march=x86-64-v3", "-fopenmp", "-fPIC", "-shared",
               "-std=gnu11", "-Wall", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
        _lib = None
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        lib.cyfa_oracle_phi.argtypes = [ctypes.c_int, _dp]
        lib.cyfa_oracle_rotation.argtypes = [ctypes.c_int, ctypes.c_double, _dp]
        lib.cyfa_oracle_shift.argtypes = [ctypes.c_int, ctypes.c_double, _dp]
        lib.cyfa_oracle_to_absolute.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                                _dp, _dp]
        lib.cyfa_oracle_to_relative.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                                _dp, _dp]
        lib.cyfa_oracle_forward.restype = ctypes.c_int
        lib.cyfa_oracle_forward.argtypes = (
            [ctypes.c_int] * 6 + [ctypes.c_double] + [_fp] * 7 + [_dp] * 3 +
            [ctypes.c_int, _ip, ctypes.c_int] + [_dp] * 5 + [ctypes.c_int])
        _lib = lib
    return _lib


def _ptr(a, kind):
    if a is None:
        return None
    return a.ctypes.data_as(kind)


def _f32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def phi(m: int) -> np.ndarray:
    """Real Fourier basis Phi (App. A.1, Eq. app-real-fourier)."""
    out = np.empty((m, m))
    _load().cyfa_oracle_phi(m, _ptr(out, _dp))
    return out


def rotation(m: int, tau: float) -> np.ndarray:
    """U(tau) = 1 (+) Rot(2 pi j tau / m) (Sec. 3.1, Eq. cyfa-fractional-shift)."""
    out = np.empty((m, m))
    _load().cyfa_oracle_rotation(m, float(tau), _ptr(out, _dp))
    return out


def shift(m: int, tau: float) -> np.ndarray:
    """Fractional cyclic shift P(tau) = Phi U(tau) Phi^T (Sec. 3.1)."""
    out = np.empty((m, m))
    _load().cyfa_oracle_shift(m, float(tau), _ptr(out, _dp))
    return out


def to_absolute(m: int, lam: float, K: np.ndarray) -> np.ndarray:
    """Relative-time state -> absolute-clock state U(-lam) Phi^T K (App. A.4)."""
    K = _f64(K)
    out = np.empty_like(K)
    _load().cyfa_oracle_to_absolute(m, K.shape[1], float(lam), _ptr(K, _dp), _ptr(out, _dp))
    return out


def to_relative(m: int, lam: float, Kbar: np.ndarray) -> np.ndarray:
    """Absolute-clock state -> relative-time state Phi U(lam) Kbar (Eq. cyfa-relative-reconstruction)."""
    Kbar = _f64(Kbar)
    out = np.empty_like(Kbar)
    _load().cyfa_oracle_to_relative(m, Kbar.shape[1], float(lam), _ptr(Kbar, _dp),
                                    _ptr(out, _dp))
    return out


def forward(q, k, v, delta, log_alpha=None, beta=None, R=None, *, m: int = 127,
            scale: float = 1.0, pairs=None, T_run=None, K0=None, V0=None, lam0=None,
            want_z: bool = True, nthreads: int = 0) -> dict:
    """Run the relative-time recurrence on [B, T, H, ...] inputs.

    ``pairs`` selects flattened (b*H + h) sequences (default: all, in order);
    ``T_run`` limits the tokens processed.  K0/V0 are relative-time initial states
    [npairs, m, d]; ``lam0`` the initial clock per pair.  Returns a dict with
    ``o`` [npairs, T_run, dv], ``z`` [npairs, T_run, m] slot logits, relative-time
    final states ``K``/``V``, the final clock ``lam`` and ``threads`` used.
    """
    q, k, v, delta = _f32(q), _f32(k), _f32(v), _f32(delta)
    log_alpha, beta, R = _f32(log_alpha), _f32(beta), _f32(R)
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    if k.shape != q.shape or v.shape[:3] != (B, T, H) or delta.shape != (B, T, H):
        raise ValueError("shape mismatch")
    for s in (log_alpha, beta):
        if s is not None and s.shape != (B, T, H):
            raise ValueError("scalar shape mismatch")
    if R is not None and R.shape != (H, m, m):
        raise ValueError("R must be [H, m, m]")
    T_run = T if T_run is None else int(T_run)
    pr = None if pairs is None else np.ascontiguousarray(pairs, dtype=np.int32)
    npairs = B * H if pr is None else len(pr)
    K0, V0, lam0 = _f64(K0), _f64(V0), _f64(lam0)
    o = np.empty((npairs, T_run, dv))
    z = np.empty((npairs, T_run, m)) if want_z else None
    Ko = np.empty((npairs, m, dk))
    Vo = np.empty((npairs, m, dv))
    lo = np.empty((npairs,))
    used = _load().cyfa_oracle_forward(
        B, T, H, dk, dv, m, float(scale),
        _ptr(q, _fp), _ptr(k, _fp), _ptr(v, _fp), _ptr(delta, _fp),
        _ptr(log_alpha, _fp), _ptr(beta, _fp), _ptr(R, _fp),
        _ptr(K0, _dp), _ptr(V0, _dp), _ptr(lam0, _dp),
        npairs, _ptr(pr, _ip), T_run,
        _ptr(o, _dp), _ptr(z, _dp), _ptr(Ko, _dp), _ptr(Vo, _dp), _ptr(lo, _dp),
        int(nthreads))
    if used < 0:
        raise ValueError("oracle rejected its arguments")
    return dict(o=o, z=z, K=Ko, V=Vo, lam=lo, threads=used)


def absolute_storage(m: int, lam: float, K: np.ndarray, rows: int = 128) -> np.ndarray:
    """Relative-time state -> absolute-clock state in the padded storage layout.

    Rows 0..m-1 follow the basis order of App. A.1 (DC, then cos/sin pairs);
    rows m..rows-1 are the zero padding of App. A.7.
    """
    out = np.zeros((rows, K.shape[1]))
    out[:m] = to_absolute(m, lam, K)
    return out


def relative_from_storage(m: int, lam: float, Kst: np.ndarray) -> np.ndarray:
    """Inverse of ``absolute_storage`` (ignores the padding rows)."""
    return to_relative(m, lam, np.asarray(Kst, dtype=np.float64)[:m])
