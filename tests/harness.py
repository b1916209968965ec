"""Helpers shared by the GPU parity tests: upload seeded inputs, gather oracle
pairs, and the error metric.

Error metric (per tensor): max_i |x_i - y_i| / max_i |y_i|, with y the oracle.
Bars: 1e-4 for float32 inputs, 2e-2 for bfloat16 inputs with float32
accumulation.
"""
from __future__ import annotations

import numpy as np

import oracle

TOL_F32 = 1e-4
TOL_BF16 = 2e-2


def rel_err(x, y) -> float:
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    den = np.abs(y).max()
    return float(np.abs(x - y).max() / (den if den > 0 else 1.0))


def upload(x: dict, device="cuda", keys=("q", "k", "v", "delta", "log_alpha", "beta", "R")):
    import torch
    out = {}
    for key in keys:
        a = x.get(key)
        if a is None:
            out[key] = None
            continue
        t = torch.from_numpy(np.ascontiguousarray(a)).to(device)
        if key in ("q", "k", "v") and x.get("dtype") == "bf16":
            t = t.to(torch.bfloat16)
        out[key] = t
    return out


def pairs_view(t, pairs, H):
    """GPU [B, T, H, ...] tensor -> numpy [len(pairs), T, ...] for flattened b*H+h pairs."""
    a = t.float().cpu().numpy() if hasattr(t, "cpu") else np.asarray(t)
    return np.stack([a[p // H, :, p % H] for p in pairs])


def state_view(t, pairs, H):
    a = t.float().cpu().numpy() if hasattr(t, "cpu") else np.asarray(t)
    return np.stack([a[p // H, p % H] for p in pairs])


def store_rows(m: int) -> int:
    """Storage rows of the operator's states: 128 for m <= 127, 256 up to m = 255."""
    return 128 if m <= 127 else 256


def oracle_states_abs(ref: dict, m: int):
    """Oracle relative-time final states -> padded absolute-clock storage [n, rows, d]."""
    rows = store_rows(m)
    K = np.stack([oracle.absolute_storage(m, lam, Kr, rows) for lam, Kr in zip(ref["lam"], ref["K"])])
    V = np.stack([oracle.absolute_storage(m, lam, Vr, rows) for lam, Vr in zip(ref["lam"], ref["V"])])
    return K, V


def clock_err(gpu_clock, oracle_lam, m):
    """Distance on the circle of circumference m between reduced clocks."""
    d = np.mod(np.asarray(gpu_clock, np.float64) - np.asarray(oracle_lam, np.float64), m)
    return float(np.max(np.minimum(d, m - d)))


def run_oracle(x: dict, pairs=None, T_run=None, want_z=True, **kw):
    return oracle.forward(x["q"], x["k"], x["v"], x["delta"], x["log_alpha"], x["beta"], x["R"],
                          m=x["m"], scale=x["scale"], pairs=pairs, T_run=T_run, want_z=want_z, **kw)
