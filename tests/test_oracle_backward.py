"""Pins of the backward oracle (CPU only).

The backward oracle differentiates its own token-by-token evaluation of the
relative-time form.  These tests tie it to things other than itself:

* its forward values equal the C oracle's (outputs, logits, final states);
* every gradient equals a central finite difference of the C oracle's forward
  (directional derivatives along random directions, for every input);
* the clock-gradient accumulation of Eq. app-clock-gradient-accumulation
  together with clock-origin invariance (Prop. 6): the gradient of the first
  clock increment equals that of the initial clock, and both vanish from a
  zero initial state;
* with a zero clock and R = I the operator reduces to scalar-decay linear
  attention, o_t = s_t e^{y_t} / (e^{y_t} + m - 1); the gradients of that closed
  form (differentiated separately) match;
* a ragged batch gives each sequence the gradients of its own prefix.
"""
import numpy as np
import pytest

import oracle
from oracle import backward as ob

torch = pytest.importorskip("torch")


def _inputs(seed, B=2, T=9, H=2, dk=4, dv=3, m=7, gates=True, with_R=True, init=True):
    rng = np.random.default_rng(seed)
    f32 = lambda a: np.asarray(a, np.float32)  # noqa: E731
    x = dict(
        q=f32(rng.standard_normal((B, T, H, dk))),
        k=f32(rng.standard_normal((B, T, H, dk))),
        v=f32(rng.standard_normal((B, T, H, dv))),
        delta=f32(np.log1p(np.exp(rng.standard_normal((B, T, H))))),
        log_alpha=f32(-np.log1p(np.exp(-(rng.standard_normal((B, T, H)) + 2)))) if gates else None,
        beta=f32(1 / (1 + np.exp(-rng.standard_normal((B, T, H))))) if gates else None,
        R=f32(np.eye(m) + 0.3 * rng.standard_normal((H, m, m))) if with_R else None,
        m=m, scale=0.7,
    )
    if init:
        K0 = np.zeros((B, H, 128, dk))
        V0 = np.zeros((B, H, 128, dv))
        K0[:, :, :m] = 0.5 * rng.standard_normal((B, H, m, dk))
        V0[:, :, :m] = 0.5 * rng.standard_normal((B, H, m, dv))
        x.update(K0=K0, V0=V0, clock0=rng.uniform(0, 3 * m, (B, H)))
    else:
        x.update(K0=None, V0=None, clock0=None)
    x["do"] = rng.standard_normal((B, T, H, dv))
    x["dK_T"] = np.zeros((B, H, 128, dk))
    x["dV_T"] = np.zeros((B, H, 128, dv))
    x["dK_T"][:, :, :m] = rng.standard_normal((B, H, m, dk))
    x["dV_T"][:, :, :m] = rng.standard_normal((B, H, m, dv))
    return x


def _c_forward(x, over=None):
    """The C oracle's forward with absolute-clock initial states; returns
    o [B,T,H,dv], z, and the final absolute states [B,H,128,d]."""
    y = dict(x)
    if over:
        y.update(over)
    B, T, H, dk = np.shape(y["q"])
    dv = np.shape(y["v"])[-1]
    m = y["m"]
    N = B * H
    K0r = V0r = lam0 = None
    if y.get("K0") is not None:
        lam0 = np.asarray(y["clock0"], np.float64).reshape(N)
        K0a = np.asarray(y["K0"], np.float64).reshape(N, 128, dk)
        V0a = np.asarray(y["V0"], np.float64).reshape(N, 128, dv)
        K0r = np.stack([oracle.relative_from_storage(m, lam0[n], K0a[n]) for n in range(N)])
        V0r = np.stack([oracle.relative_from_storage(m, lam0[n], V0a[n]) for n in range(N)])
    ref = oracle.forward(y["q"], y["k"], y["v"], y["delta"], y["log_alpha"], y["beta"], y["R"],
                         m=m, scale=y["scale"], K0=K0r, V0=V0r, lam0=lam0)
    o = np.moveaxis(ref["o"].reshape(B, H, T, dv), 1, 2)
    z = np.moveaxis(ref["z"].reshape(B, H, T, m), 1, 2)
    KT = np.stack([oracle.absolute_storage(m, lam, Kr) for lam, Kr in zip(ref["lam"], ref["K"])])
    VT = np.stack([oracle.absolute_storage(m, lam, Vr) for lam, Vr in zip(ref["lam"], ref["V"])])
    return o, z, KT.reshape(B, H, 128, dk), VT.reshape(B, H, 128, dv)


def _loss(x, over=None):
    o, _, KT, VT = _c_forward(x, over)
    return float((o * x["do"]).sum() + (KT * x["dK_T"]).sum() + (VT * x["dV_T"]).sum())


def _grads(x, **kw):
    return ob.backward(x["q"], x["k"], x["v"], x["delta"], x["log_alpha"], x["beta"], x["R"],
                       do=x["do"], m=x["m"], scale=x["scale"], K0=x["K0"], V0=x["V0"],
                       clock0=x["clock0"], dK_T=x["dK_T"], dV_T=x["dV_T"], **kw)


@pytest.mark.parametrize("m,gates,with_R", [(7, True, True), (5, False, False), (9, True, False)])
def test_forward_values_match_c_oracle(m, gates, with_R):
    x = _inputs(1, m=m, gates=gates, with_R=with_R)
    g = _grads(x, want_forward=True)
    o, z, KT, VT = _c_forward(x)
    np.testing.assert_allclose(g["o"], o, rtol=0, atol=1e-12)
    np.testing.assert_allclose(g["z"], z, rtol=0, atol=1e-11)
    np.testing.assert_allclose(g["K_T"], KT, rtol=0, atol=1e-12)
    np.testing.assert_allclose(g["V_T"], VT, rtol=0, atol=1e-12)


GRAD_OF = {"q": "dq", "k": "dk", "v": "dv", "delta": "ddelta", "log_alpha": "dlog_alpha",
           "beta": "dbeta", "R": "dR", "K0": "dK0", "V0": "dV0", "clock0": "dclock0"}


@pytest.mark.parametrize("m", [5, 7])
def test_gradients_match_finite_differences_of_c_oracle(m):
    x = _inputs(2, m=m)
    g = _grads(x)
    rng = np.random.default_rng(3)
    h = 2.0 ** -9
    for name, gname in GRAD_OF.items():
        base = np.asarray(x[name])
        for _ in range(2):
            d = rng.integers(-1, 2, base.shape).astype(np.float64)
            if name in ("K0", "V0"):
                d[:, :, m:] = 0
            if base.dtype == np.float32:
                xp = (base + h * d).astype(np.float32)
                xm = (base - h * d).astype(np.float32)
            else:
                xp, xm = base + h * d, base - h * d
            fd = _loss(x, {name: xp}) - _loss(x, {name: xm})
            an = float((g[gname] * (xp.astype(np.float64) - xm.astype(np.float64))).sum())
            scale = np.abs(g[gname]).sum() * 2 * h + 1e-12
            assert abs(fd - an) <= 2e-5 * scale, (name, fd, an)


def test_wrong_gradient_is_caught():
    """The finite-difference comparison rejects a gradient with a dropped term
    (here: dq with one token's row zeroed)."""
    x = _inputs(4, m=7)
    g = _grads(x)
    bad = g["dq"].copy()
    bad[0, 3] = 0
    h = 2.0 ** -9
    d = np.zeros_like(bad)
    d[0, 3] = 1
    xp = (x["q"] + h * d).astype(np.float32)
    xm = (x["q"] - h * d).astype(np.float32)
    fd = _loss(x, {"q": xp}) - _loss(x, {"q": xm})
    assert abs(fd - float((g["dq"] * (xp - xm)).sum())) < 1e-6 * max(1.0, abs(fd))
    assert abs(fd - float((bad * (xp - xm)).sum())) > 1e-3 * abs(fd)


def test_first_increment_and_initial_clock_share_their_gradient():
    """lambda_t = lambda_0 + sum_{u<=t} delta_u, so dL/ddelta_1 = sum_t dL/dlambda_t
    = dL/dlambda_0 (Eq. app-clock-gradient-accumulation); from a zero state the
    origin of the clock does not matter (Prop. 6), so both are zero."""
    x = _inputs(5, m=7)
    x["dK_T"][:] = 0
    x["dV_T"][:] = 0
    g = _grads(x)
    np.testing.assert_allclose(g["ddelta"][:, 0], g["dclock0"], rtol=1e-9, atol=1e-11)
    assert np.abs(g["dclock0"]).max() > 1e-3
    y = _inputs(5, m=7, init=False)
    y["dK_T"][:] = 0
    y["dV_T"][:] = 0
    gz = _grads(y)
    np.testing.assert_allclose(gz["ddelta"][:, 0], 0, atol=1e-11)
    np.testing.assert_allclose(gz["dclock0"], 0, atol=1e-11)


def test_zero_clock_reduces_to_scalar_decay_linear_attention():
    x = _inputs(6, B=1, T=8, H=1, m=7, with_R=False, init=False)
    x["delta"] = np.zeros_like(x["delta"])
    x["dK_T"][:] = 0
    x["dV_T"][:] = 0
    g = _grads(x)
    m, s = x["m"], x["scale"]
    tq = torch.tensor(x["q"][0, :, 0], dtype=torch.float64, requires_grad=True)
    tk = torch.tensor(x["k"][0, :, 0], dtype=torch.float64, requires_grad=True)
    tv = torch.tensor(x["v"][0, :, 0], dtype=torch.float64, requires_grad=True)
    tg = torch.tensor(x["log_alpha"][0, :, 0], dtype=torch.float64, requires_grad=True)
    tb = torch.tensor(x["beta"][0, :, 0], dtype=torch.float64, requires_grad=True)
    T = tq.shape[0]
    G = torch.cumsum(tg, 0)
    os_ = []
    for t in range(T):
        wts = torch.exp(G[t] - G[: t + 1]) * tb[: t + 1]            # prod alpha * beta_i
        y = s * (tq[t] * (wts[:, None] * tk[: t + 1]).sum(0)).sum()
        st = (wts[:, None] * tv[: t + 1]).sum(0)
        os_.append(st * torch.exp(y) / (torch.exp(y) + m - 1))
    o = torch.stack(os_)
    loss = (o * torch.tensor(x["do"][0, :, 0])).sum()
    dq, dk, dv, dg, db = torch.autograd.grad(loss, [tq, tk, tv, tg, tb])
    for a, b in ((g["dq"], dq), (g["dk"], dk), (g["dv"], dv), (g["dlog_alpha"], dg),
                 (g["dbeta"], db)):
        np.testing.assert_allclose(a[0, :, 0], b.numpy(), rtol=1e-10, atol=1e-12)


def test_ragged_batch_gives_each_sequence_its_prefix_gradients():
    x = _inputs(7, B=2, T=9, m=7)
    lens = [9, 5]
    g = _grads(x, lens=lens)
    for b, L in enumerate(lens):
        y = {key: (val[b:b + 1, :L] if key in ("q", "k", "v", "delta", "log_alpha", "beta", "do")
                   else val[b:b + 1] if key in ("K0", "V0", "clock0", "dK_T", "dV_T") else val)
             for key, val in x.items()}
        gb = _grads(y)
        for name in ("dq", "dk", "dv", "ddelta", "dlog_alpha", "dbeta"):
            np.testing.assert_allclose(g[name][b:b + 1, :L], gb[name], rtol=1e-10, atol=1e-12)
            assert np.all(g[name][b, L:] == 0)
        for name in ("dK0", "dV0", "dclock0"):
            np.testing.assert_allclose(g[name][b:b + 1], gb[name], rtol=1e-10, atol=1e-12)
