"""CyFA backward oracle.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only ``tests/`` may import this
module.  The GPU operator never calls it and shares no code with it.

Gradients of the operator by reverse-mode differentiation (torch.autograd on
the CPU, float64) of a token-by-token evaluation of its defining
relative-time-slot form (Sec. 3.1):

    K_t = alpha_t P(delta_t) K_{t-1} + beta_t e_0 k_t^T      Eq. cyfa-physical-recurrence
    V_t = alpha_t P(delta_t) V_{t-1} + beta_t e_0 v_t^T
    o_t = (R V_t)^T softmax(scale R K_t q_t)                  Eq. cyfa-physical-readout

with P(tau) = Phi U(tau) Phi^T (Eq. cyfa-fractional-shift) applied as its
three factors, and alpha_t = exp(log_alpha_t).  The arguments are taken in the
coordinates of the operator's interface: the initial state is given in
absolute-clock form (Kbar_0 with clock lambda_0) and mapped to relative time by
K_0 = Phi U(lambda_0) Kbar_0 (App. A.4, Eq. app-three-K); the final state is
returned in absolute-clock form, Kbar_T = U(-lambda_T) Phi^T K_T with
lambda_T = lambda_0 + sum_t delta_t, so that a loss may depend on it.

The loss is L = sum_t <do_t, o_t> + <dK_T, Kbar_T> + <dV_T, Vbar_T>; the result
is dL with respect to every input.  Rows t >= lens[b] of a ragged batch are not
part of sequence b (no write, no decay, no shift; zero gradient).
"""
from __future__ import annotations

import math

import numpy as np

from . import phi as _phi_np

STORE_ROWS = 128


def _torch():
    import torch
    return torch


def _rotate_pairs(torch, Y, tau, m, sign):
    """U(sign * tau) applied to the rows of Y [N, m, d]: identity on row 0, the
    rotation by sign * 2 pi j tau / m on rows (2j-1, 2j) (Sec. 3.1, U(tau))."""
    J = (m - 1) // 2
    j = torch.arange(1, J + 1, dtype=torch.float64)
    th = sign * 2.0 * math.pi * j[None, :] * tau[:, None] / m       # [N, J]
    c = torch.cos(th)[:, :, None]
    s = torch.sin(th)[:, :, None]
    a = Y[:, 1::2, :]                                                  # rows 2j-1
    b = Y[:, 2::2, :]                                                  # rows 2j
    ra = c * a - s * b
    rb = s * a + c * b
    out = torch.stack([ra, rb], dim=2).reshape(Y.shape[0], 2 * J, Y.shape[2])
    return torch.cat([Y[:, :1, :], out], dim=1)


def _run(torch, q, k, v, delta, la, be, R, Kb0, Vb0, lam0, lens_pairs, m, scale):
    """q, k: [N, T, dk]; v: [N, T, dv]; delta, la, be: [N, T]; R: [N, m, m];
    Kb0/Vb0: [N, m, d] absolute; lam0: [N].  Returns o [N, T, dv], z [N, T, m],
    Kbar_T [N, m, dk], Vbar_T [N, m, dv]."""
    N, T, dk = q.shape
    Phi = torch.from_numpy(_phi_np(m))                                # [m, m]
    K = Phi @ _rotate_pairs(torch, Kb0, lam0, m, +1.0)
    V = Phi @ _rotate_pairs(torch, Vb0, lam0, m, +1.0)
    lam = lam0
    e0 = torch.zeros(m, dtype=torch.float64)
    e0[0] = 1.0
    os_, zs = [], []
    for t in range(T):
        live = (t < lens_pairs).to(torch.float64)                     # [N]
        d_t = delta[:, t] * live
        a_t = torch.exp(la[:, t] * live)
        b_t = be[:, t] * live
        # P(delta_t) K = Phi U(delta_t) Phi^T K
        K = Phi @ _rotate_pairs(torch, Phi.T @ K, d_t, m, +1.0)
        V = Phi @ _rotate_pairs(torch, Phi.T @ V, d_t, m, +1.0)
        K = a_t[:, None, None] * K + b_t[:, None, None] * e0[None, :, None] * k[:, t][:, None, :]
        V = a_t[:, None, None] * V + b_t[:, None, None] * e0[None, :, None] * v[:, t][:, None, :]
        lam = lam + d_t
        z = scale * torch.einsum("nij,nj->ni", R, torch.einsum("njd,nd->nj", K, q[:, t]))
        w = torch.softmax(z, dim=-1)
        o = torch.einsum("nid,ni->nd", torch.einsum("nij,njd->nid", R, V), w)
        os_.append(o * live[:, None])
        zs.append(z)
    o = torch.stack(os_, dim=1)
    z = torch.stack(zs, dim=1)
    KbT = _rotate_pairs(torch, Phi.T @ K, lam, m, -1.0)
    VbT = _rotate_pairs(torch, Phi.T @ V, lam, m, -1.0)
    return o, z, KbT, VbT


def _pairs(a, B, H):
    """[B, T, H, ...] -> [B*H, T, ...] (pair n = b*H + h)."""
    a = np.asarray(a, dtype=np.float64)
    return np.ascontiguousarray(np.moveaxis(a, 2, 1).reshape((B * H,) + a.shape[1:2] + a.shape[3:]))


def _unpairs(a, B, H):
    a = np.asarray(a)
    return np.ascontiguousarray(np.moveaxis(a.reshape((B, H) + a.shape[1:]), 1, 2))


def backward(q, k, v, delta, log_alpha=None, beta=None, R=None, *, do, m: int = 127,
             scale: float = 1.0, K0=None, V0=None, clock0=None, dK_T=None, dV_T=None,
             lens=None, want_forward: bool = False) -> dict:
    """Gradients of L = <do, o> + <dK_T, Kbar_T> + <dV_T, Vbar_T>.

    Layouts follow the operator's interface: q, k [B, T, H, dk]; v, do
    [B, T, H, dv]; delta, log_alpha, beta [B, T, H]; R [H, m, m]; K0, dK_T
    [B, H, 128, dk] and V0, dV_T [B, H, 128, dv] absolute-clock states (rows
    >= m ignored); clock0 [B, H]; lens [B].  None means: alpha = 1, beta = 1,
    R = I, zero initial state and clock, no loss on the final state.
    Returns dq, dk, dv, ddelta, dlog_alpha, dbeta (None for absent gates),
    dR [H, m, m] (None without R), dK0 / dV0 [B, H, 128, d] and dclock0 [B, H];
    with ``want_forward`` also o, z [B, T, H, m] and the final states.
    """
    torch = _torch()
    q = np.asarray(q, np.float64)
    B, T, H, dk = q.shape
    dv = np.asarray(v).shape[-1]
    N = B * H
    tt = lambda a: torch.tensor(a, dtype=torch.float64, requires_grad=True)  # noqa: E731
    Q, Kx, Vx = tt(_pairs(q, B, H)), tt(_pairs(k, B, H)), tt(_pairs(v, B, H))
    D = tt(_pairs(delta, B, H))
    LA = tt(_pairs(log_alpha, B, H)) if log_alpha is not None else None
    BE = tt(_pairs(beta, B, H)) if beta is not None else None
    Rt = tt(np.asarray(R, np.float64)) if R is not None else None
    zeros = lambda *s: np.zeros(s)  # noqa: E731
    Kb0 = tt(np.asarray(K0, np.float64).reshape(N, STORE_ROWS, dk)[:, :m] if K0 is not None
             else zeros(N, m, dk))
    Vb0 = tt(np.asarray(V0, np.float64).reshape(N, STORE_ROWS, dv)[:, :m] if V0 is not None
             else zeros(N, m, dv))
    L0 = tt(np.asarray(clock0, np.float64).reshape(N) if clock0 is not None else zeros(N))
    lens_b = np.full(B, T) if lens is None else np.clip(np.asarray(lens, np.int64), 0, T)
    lens_pairs = torch.tensor(np.repeat(lens_b, H), dtype=torch.float64)
    la_use = LA if LA is not None else torch.zeros(N, T, dtype=torch.float64)
    be_use = BE if BE is not None else torch.ones(N, T, dtype=torch.float64)
    if Rt is not None:
        R_use = Rt.repeat(B, 1, 1)                   # pair n = b*H + h uses R[h]
    else:
        R_use = torch.eye(m, dtype=torch.float64).expand(N, m, m)
    o, z, KbT, VbT = _run(torch, Q, Kx, Vx, D, la_use, be_use, R_use, Kb0, Vb0, L0, lens_pairs,
                          m, scale)
    loss = (o * torch.tensor(_pairs(do, B, H))).sum()
    if dK_T is not None:
        loss = loss + (KbT * torch.tensor(np.asarray(dK_T, np.float64).reshape(N, STORE_ROWS, dk)[:, :m])).sum()
    if dV_T is not None:
        loss = loss + (VbT * torch.tensor(np.asarray(dV_T, np.float64).reshape(N, STORE_ROWS, dv)[:, :m])).sum()
    leaves = [Q, Kx, Vx, D, LA, BE, Rt, Kb0, Vb0, L0]
    live = [x for x in leaves if x is not None]
    grads = torch.autograd.grad(loss, live, allow_unused=True)
    g = {}
    it = iter(grads)
    for name, x in zip(["dq", "dk", "dv", "ddelta", "dlog_alpha", "dbeta", "dR", "dK0r", "dV0r",
                        "dclock0r"], leaves):
        if x is None:
            g[name] = None
        else:
            gr = next(it)
            g[name] = np.zeros(tuple(x.shape)) if gr is None else gr.detach().numpy()
    out = {}
    for name in ("dq", "dk", "dv"):
        out[name] = _unpairs(g[name], B, H)
    for name in ("ddelta", "dlog_alpha", "dbeta"):
        out[name] = None if g[name] is None else _unpairs(g[name], B, H)
    out["dR"] = g["dR"]
    dK0 = np.zeros((N, STORE_ROWS, dk))
    dK0[:, :m] = g["dK0r"]
    dV0 = np.zeros((N, STORE_ROWS, dv))
    dV0[:, :m] = g["dV0r"]
    out["dK0"] = dK0.reshape(B, H, STORE_ROWS, dk)
    out["dV0"] = dV0.reshape(B, H, STORE_ROWS, dv)
    out["dclock0"] = g["dclock0r"].reshape(B, H)
    if want_forward:
        out["o"] = _unpairs(o.detach().numpy(), B, H)
        out["z"] = _unpairs(z.detach().numpy(), B, H)
        KT = np.zeros((N, STORE_ROWS, dk))
        KT[:, :m] = KbT.detach().numpy()
        VT = np.zeros((N, STORE_ROWS, dv))
        VT[:, :m] = VbT.detach().numpy()
        out["K_T"] = KT.reshape(B, H, STORE_ROWS, dk)
        out["V_T"] = VT.reshape(B, H, STORE_ROWS, dv)
    return out
