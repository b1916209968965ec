"""CyFA mixer prologue and epilogue oracle (numpy, float64).

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only ``tests/`` and the
benchmark's checks may import this module.  The GPU operator never calls it and
shares no code with it.

The mixer around the operator (Sec. 4, network design):

* ShortConv on q, k, v: a causal depthwise convolution over time of width K per
  channel, y_t = sum_{j<K} w[c, j] x_{t-K+1+j} (zero before the sequence start),
  optionally followed by SiLU;
* RMSNorm on the queries and keys, per head vector: x / sqrt(mean(x^2) + eps) * g;
* the scalar gates from their projections z (per token and head):
  delta = sigmoid(z_delta + b_delta) (Eq. clock_gradient_stabilization),
  alpha = exp(-A softplus(z_alpha + b_alpha)), so log alpha = -A softplus(.),
  beta = sigmoid(z_beta);
* after the operator, a head-wise RMSNorm of the outputs and a sigmoid output
  gate: out = RMSNorm(o) * sigmoid(g).

Rows t >= lens[b] of a ragged batch are padding: outputs there are zero.
"""
from __future__ import annotations

import numpy as np


def _f64(a):
    return None if a is None else np.asarray(a, dtype=np.float64)


def sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def softplus(x):
    return np.where(x > 30, x, np.log1p(np.exp(np.minimum(x, 30))))


def short_conv(x, w, act: str = "none", lens=None):
    """x [B, T, H, D]; w [H*D, K]: y[b, t, c] = sum_j w[c, j] x[b, t - K + 1 + j, c]."""
    x = _f64(x)
    B, T, H, D = x.shape
    K = np.asarray(w).shape[1]
    wc = _f64(w).reshape(H, D, K)
    y = np.zeros_like(x)
    for j in range(K):
        s = K - 1 - j                      # input lag of tap j
        if s >= T:
            continue
        y[:, s:] += wc[None, None, :, :, j] * x[:, : T - s]
    if act == "silu":
        y = y * sigmoid(y)
    return _mask(y, lens)


def rms_norm(x, g, eps: float):
    x = _f64(x)
    r = np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return x / r * (_f64(g) if g is not None else 1.0)


def _mask(y, lens):
    if lens is None:
        return y
    T = y.shape[1]
    keep = np.arange(T)[None, :] < np.clip(np.asarray(lens), 0, T)[:, None]
    return y * keep.reshape(keep.shape + (1,) * (y.ndim - 2))


def prologue(q, k, v, wq=None, wk=None, wv=None, gq=None, gk=None, z_delta=None, b_delta=None,
             z_alpha=None, b_alpha=None, A=None, z_beta=None, *, act: str = "none",
             eps: float = 1e-6, lens=None) -> dict:
    """Returns q, k, v (ShortConv, then RMSNorm on q and k when gq / gk are given)
    and the gates delta, log_alpha, beta (None where the projection is None)."""
    out = {}
    for name, x, w in (("q", q, wq), ("k", k, wk), ("v", v, wv)):
        y = short_conv(x, w, act, lens) if w is not None else _mask(_f64(x), lens)
        out[name] = y
    if gq is not None:
        out["q"] = _mask(rms_norm(out["q"], gq, eps), lens)
    if gk is not None:
        out["k"] = _mask(rms_norm(out["k"], gk, eps), lens)
    H = np.shape(q)[2]
    bias = lambda b: np.zeros(H) if b is None else _f64(b)  # noqa: E731
    out["delta"] = _mask(sigmoid(_f64(z_delta) + bias(b_delta)), lens) if z_delta is not None else None
    out["log_alpha"] = (_mask(-_f64(A) * softplus(_f64(z_alpha) + bias(b_alpha)), lens)
                        if z_alpha is not None else None)
    out["beta"] = _mask(sigmoid(_f64(z_beta)), lens) if z_beta is not None else None
    return out


def epilogue(o, g=None, go=None, *, eps: float = 1e-6, lens=None):
    """RMSNorm(o) * go, times sigmoid(g) when the gate projection g is given."""
    y = rms_norm(o, go, eps)
    if g is not None:
        y = y * sigmoid(_f64(g))
    return _mask(y, lens)
