"""Independent small numpy evaluations of CyFA used to pin the oracle.

Test-only code.  Each form below is written directly from a different passage
of the paper than the oracle's relative-time recurrence, so agreement between
them is evidence about both:

* ``absolute_clock_forward``: the absolute-clock recurrence and readout
  (Sec. 3.2, Eqs. cyfa-absolute-recurrence and cyfa-absolute-readout);
* ``chunkwise_forward``: the two-pass chunk form of App. B
  (Eqs. app-chunk-decay, app-temporal-writes, app-cyfa-key-chunk,
  app-cyfa-value-chunk);
* ``dirichlet_shift``: P(tau) from the closed form of App. A.2, Prop. 2.

The Fourier basis and the rotation are rebuilt here from their definitions
rather than taken from the oracle.
"""
from __future__ import annotations

import numpy as np


def fourier_basis(m: int) -> np.ndarray:
    r = np.arange(m)[:, None]
    j = np.arange(1, (m - 1) // 2 + 1)[None, :]
    ang = 2 * np.pi * j * r / m
    phi = np.empty((m, m))
    phi[:, 0] = 1 / np.sqrt(m)
    phi[:, 1::2] = np.sqrt(2 / m) * np.cos(ang)
    phi[:, 2::2] = np.sqrt(2 / m) * np.sin(ang)
    return phi


def rotate(m: int, tau: float, x: np.ndarray) -> np.ndarray:
    """U(tau) applied to x along axis 0 (pairs (2j-1, 2j) rotated by 2 pi j tau / m)."""
    j = np.arange(1, (m - 1) // 2 + 1)
    th = 2 * np.pi * j * tau / m
    c, s = np.cos(th), np.sin(th)
    shape = (-1,) + (1,) * (x.ndim - 1)
    c, s = c.reshape(shape), s.reshape(shape)
    out = np.array(x, dtype=np.float64, copy=True)
    a, b = x[1::2], x[2::2]
    out[1::2] = c * a - s * b
    out[2::2] = s * a + c * b
    return out


def dirichlet_shift(m: int, tau: float) -> np.ndarray:
    r = np.arange(m)[:, None]
    s = np.arange(m)[None, :]
    x = tau + s - r
    num = np.sin(np.pi * x)
    den = m * np.sin(np.pi * x / m)
    near = np.abs(den) < 1e-12
    val = np.where(near, 1.0, num / np.where(near, 1.0, den))
    # at x = k m the limit is cos(pi k m) / cos(pi k) = 1 for odd m
    return val


def _softmax(z):
    z = z - z.max()
    e = np.exp(z)
    return e / e.sum()


def absolute_clock_forward(q, k, v, delta, log_alpha, beta, R, scale, m,
                           Kbar0=None, Vbar0=None, lam0=0.0):
    """One (b, h) sequence; q,k: [T, dk], v: [T, dv], scalars [T].  Returns o, z, Kbar, Vbar, lam."""
    T, dk = q.shape
    dv = v.shape[1]
    phi = fourier_basis(m)
    b = phi.T[:, 0].copy()
    Rm = np.eye(m) if R is None else np.asarray(R, dtype=np.float64)
    Kb = np.zeros((m, dk)) if Kbar0 is None else np.array(Kbar0, dtype=np.float64)
    Vb = np.zeros((m, dv)) if Vbar0 is None else np.array(Vbar0, dtype=np.float64)
    lam = float(lam0)
    o = np.zeros((T, dv))
    zs = np.zeros((T, m))
    for t in range(T):
        lam += float(delta[t])
        al = 1.0 if log_alpha is None else np.exp(float(log_alpha[t]))
        be = 1.0 if beta is None else float(beta[t])
        a = be * rotate(m, -lam, b)
        Kb = al * Kb + np.outer(a, k[t].astype(np.float64))
        Vb = al * Vb + np.outer(a, v[t].astype(np.float64))
        op = Kb @ q[t].astype(np.float64)
        z = scale * (Rm @ (phi @ rotate(m, lam, op)))
        w = _softmax(z)
        opp = rotate(m, -lam, phi.T @ (Rm.T @ w))
        o[t] = Vb.T @ opp
        zs[t] = z
    return o, zs, Kb, Vb, lam


def chunkwise_forward(q, k, v, delta, log_alpha, beta, R, scale, m, C):
    """Two-pass chunk-wise evaluation (App. B) of one sequence from zero state."""
    T, dk = q.shape
    dv = v.shape[1]
    phi = fourier_basis(m)
    b = phi.T[:, 0].copy()
    Rm = np.eye(m) if R is None else np.asarray(R, dtype=np.float64)
    M = Rm @ phi
    g = np.zeros(T) if log_alpha is None else log_alpha.astype(np.float64)
    bt = np.ones(T) if beta is None else beta.astype(np.float64)
    lam = np.cumsum(delta.astype(np.float64))
    Kb = np.zeros((m, dk))
    Vb = np.zeros((m, dv))
    o = np.zeros((T, dv))
    zs = np.zeros((T, m))
    for c0 in range(0, T, C):
        sl = slice(c0, min(c0 + C, T))
        n = sl.stop - sl.start
        Q = q[sl].astype(np.float64)
        K = k[sl].astype(np.float64)
        V = v[sl].astype(np.float64)
        G = np.cumsum(g[sl])                       # log gamma^r, r = 1..n
        gam = np.exp(G)
        Gam = np.tril(np.exp(G[:, None] - G[None, :]))
        A = np.stack([bt[sl][r] * rotate(m, -lam[sl][r], b) for r in range(n)])
        right = np.exp(G[-1] - G)[:, None]         # gamma^C / gamma^r
        # key pass
        Op = gam[:, None] * (Q @ Kb.T) + ((Q @ K.T) * Gam) @ A
        Kb = gam[-1] * Kb + (right * A).T @ K
        # token-wise middle step
        Opp = np.zeros_like(Op)
        for r in range(n):
            x = rotate(m, lam[sl][r], Op[r])
            z = scale * (M @ x)
            zs[c0 + r] = z
            Opp[r] = rotate(m, -lam[sl][r], M.T @ _softmax(z))
        # value pass
        o[sl] = gam[:, None] * (Opp @ Vb) + ((Opp @ A.T) * Gam) @ V
        Vb = gam[-1] * Vb + A.T @ (right * V)
    return o, zs, Kb, Vb
