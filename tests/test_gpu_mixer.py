"""GPU parity of the mixer prologue / epilogue (cyfa_mixer_prologue,
cyfa_mixer_epilogue) against the mixer oracle, every element.  Bars: 1e-4 for
float32, 2e-2 for bfloat16 (max |x - y| / max |y| per tensor)."""
import numpy as np
import pytest

from oracle import mixer
from tests.harness import TOL_BF16, TOL_F32, rel_err

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _cyfa():
    from paper_2609_36259_amd import cyfa
    return cyfa


def _inputs(B, T, H, dk, dv, seed, dtype, K=4):
    rng = np.random.default_rng(seed)
    rnd = lambda *s: rng.standard_normal(s).astype(np.float32)  # noqa: E731
    x = dict(q=rnd(B, T, H, dk), k=rnd(B, T, H, dk), v=rnd(B, T, H, dv),
             wq=0.5 * rnd(H * dk, K), wk=0.5 * rnd(H * dk, K), wv=0.5 * rnd(H * dv, K),
             gq=1 + 0.1 * rnd(dk), gk=1 + 0.1 * rnd(dk),
             z_delta=rnd(B, T, H), b_delta=rnd(H), z_alpha=2 * rnd(B, T, H), b_alpha=rnd(H),
             A=np.exp(rnd(H)), z_beta=rnd(B, T, H),
             o=rnd(B, T, H, dv), g=2 * rnd(B, T, H, dv), go=1 + 0.1 * rnd(dv))
    if dtype == "bf16":
        for key in ("q", "k", "v", "o", "g"):
            x[key] = torch.tensor(x[key]).bfloat16().float().numpy()
    x["dtype"] = dtype
    return x


def _dev(a, dtype=torch.float32):
    return None if a is None else torch.tensor(a, dtype=dtype, device="cuda")


def _prologue(x, act=0, use=("conv", "norm", "gates"), lens=None, K=4):
    cyfa = _cyfa()
    dt = torch.bfloat16 if x["dtype"] == "bf16" else torch.float32
    conv = "conv" in use
    norm = "norm" in use
    gates = "gates" in use
    res = cyfa.mixer_prologue(
        _dev(x["q"], dt), _dev(x["k"], dt), _dev(x["v"], dt),
        conv_q=_dev(x["wq"]) if conv else None, conv_k=_dev(x["wk"]) if conv else None,
        conv_v=_dev(x["wv"]) if conv else None, norm_q=_dev(x["gq"]) if norm else None,
        norm_k=_dev(x["gk"]) if norm else None,
        z_delta=_dev(x["z_delta"]) if gates else None, b_delta=_dev(x["b_delta"]) if gates else None,
        z_alpha=_dev(x["z_alpha"]) if gates else None, b_alpha=_dev(x["b_alpha"]) if gates else None,
        A=_dev(x["A"]) if gates else None, z_beta=_dev(x["z_beta"]) if gates else None,
        lens=_dev(lens, torch.int32) if lens is not None else None, conv_size=K, conv_act=act)
    torch.cuda.synchronize()
    got = {k: (None if v is None else v.float().cpu().numpy()) for k, v in res.items()}
    ref = mixer.prologue(x["q"], x["k"], x["v"], x["wq"] if conv else None, x["wk"] if conv else None,
                         x["wv"] if conv else None, x["gq"] if norm else None, x["gk"] if norm else None,
                         x["z_delta"] if gates else None, x["b_delta"], x["z_alpha"] if gates else None,
                         x["b_alpha"], x["A"], x["z_beta"] if gates else None,
                         act="silu" if act else "none", lens=lens)
    return got, ref


def _check(got, ref, tol, bf16_keys=()):
    errs = {}
    for key, r in ref.items():
        if r is None:
            assert got[key] is None, key
            continue
        errs[key] = rel_err(got[key], r)
    print("errors", {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    for k, v in errs.items():
        assert v <= (tol if k in bf16_keys else TOL_F32), (k, v)


@pytest.mark.parametrize("act", [0, 1])
def test_prologue_f32(act):
    x = _inputs(2, 37, 3, 64, 128, seed=81, dtype="f32")
    got, ref = _prologue(x, act=act)
    _check(got, ref, TOL_F32)


def test_prologue_bf16_d128_ragged():
    x = _inputs(3, 50, 2, 128, 128, seed=82, dtype="bf16")
    lens = [50, 17, 0]
    got, ref = _prologue(x, lens=lens)
    _check(got, ref, TOL_BF16, bf16_keys=("q", "k", "v"))
    for key in ("q", "k", "v", "delta", "log_alpha", "beta"):
        assert np.all(got[key][1, 17:] == 0) and np.all(got[key][2] == 0), key


@pytest.mark.parametrize("use,K", [((), 4), (("conv",), 2), (("norm",), 4), (("conv", "norm"), 1)])
def test_prologue_optional_parts(use, K):
    x = _inputs(1, 21, 2, 256, 64, seed=83, dtype="f32", K=K)
    got, ref = _prologue(x, use=use, K=K)
    _check(got, ref, TOL_F32)


def _epilogue(x, with_gate=True, lens=None):
    cyfa = _cyfa()
    dt = torch.bfloat16 if x["dtype"] == "bf16" else torch.float32
    out = cyfa.mixer_epilogue(_dev(x["o"], dt), _dev(x["g"], dt) if with_gate else None, _dev(x["go"]),
                              lens=_dev(lens, torch.int32) if lens is not None else None)
    torch.cuda.synchronize()
    ref = mixer.epilogue(x["o"], x["g"] if with_gate else None, x["go"], lens=lens)
    return out.float().cpu().numpy(), ref


@pytest.mark.parametrize("dtype,d,gate", [("f32", 64, True), ("f32", 256, False), ("bf16", 128, True)])
def test_epilogue(dtype, d, gate):
    x = _inputs(2, 29, 3, d, d, seed=84, dtype=dtype)
    got, ref = _epilogue(x, with_gate=gate, lens=[29, 11])
    err = rel_err(got, ref)
    print("epilogue error", f"{err:.2e}", flush=True)
    assert err <= (TOL_BF16 if dtype == "bf16" else TOL_F32)
    assert np.all(got[1, 11:] == 0)


def test_full_size_layer_prologue_and_epilogue():
    """The 1.4B-scale layer (B=4, T=4096, H=16, d=128, bf16), every element."""
    x = _inputs(4, 4096, 16, 128, 128, seed=85, dtype="bf16")
    print("full-size prologue", flush=True)
    got, ref = _prologue(x)
    _check(got, ref, TOL_BF16, bf16_keys=("q", "k", "v"))
    print("full-size epilogue", flush=True)
    out, eref = _epilogue(x)
    assert rel_err(out, eref) <= TOL_BF16
