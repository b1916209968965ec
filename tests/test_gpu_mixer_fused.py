"""GPU parity of the layer forward (cyfa_forward_mixer: mixer prologue, operator and
mixer epilogue in one pass of the matrix-core kernel).

The fused call (ShortConv in the staging or in its own streaming kernel,
``fuse_conv`` 1 or 0) runs the standalone kernels' arithmetic in the same order, so its
output, final states, clocks and slot logits must be bit-identical to
cyfa_mixer_prologue -> cyfa_forward -> cyfa_mixer_epilogue on the same inputs and
segment plan; the layer output is also compared with the chain of the oracles
(bar 2e-2, bf16).  Cases: every optional mixer part present or absent, ShortConv
widths 1..4 with and without SiLU, ragged lengths (padding rows of the output
written as 0), initial states, several segments, a tail chunk.
"""
import numpy as np
import pytest

import oracle
from oracle import mixer
from tests.harness import TOL_BF16, rel_err

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

D = 128


def _cyfa():
    from paper_2609_36259_amd import cyfa
    return cyfa


def _bf16(a):
    return torch.tensor(np.asarray(a, np.float32)).bfloat16().float().numpy()


def _inputs(B, T, H, seed, K=4, m=127):
    rng = np.random.default_rng(seed)
    rnd = lambda *s: rng.standard_normal(s).astype(np.float32)  # noqa: E731
    return dict(q=_bf16(rnd(B, T, H, D)), k=_bf16(rnd(B, T, H, D)), v=_bf16(rnd(B, T, H, D)),
                wq=0.5 * rnd(H * D, K), wk=0.5 * rnd(H * D, K), wv=0.5 * rnd(H * D, K),
                gq=1 + 0.1 * rnd(D), gk=1 + 0.1 * rnd(D), z_delta=rnd(B, T, H), b_delta=rnd(H),
                z_alpha=rnd(B, T, H), b_alpha=rnd(H) + 2, A=np.exp(rnd(H) - 1), z_beta=rnd(B, T, H),
                R=(np.eye(m) + 0.1 * rnd(H, m, m)).astype(np.float32),
                gate=_bf16(2 * rnd(B, T, H, D)), go=1 + 0.1 * rnd(D), m=m, K=K)


def _dev(x, drop=()):
    bf = torch.bfloat16
    t = {}
    for key in ("q", "k", "v", "gate"):
        t[key] = None if key in drop else torch.tensor(x[key], dtype=bf, device="cuda")
    for key in ("wq", "wk", "wv", "gq", "gk", "z_delta", "b_delta", "z_alpha", "b_alpha", "A", "z_beta", "R",
                "go"):
        t[key] = None if key in drop else torch.tensor(x[key], dtype=torch.float32, device="cuda")
    return t


def _chain(t, x, segments, act=0, lens=None, K0=None, V0=None, clock0=None, logits=False):
    cyfa = _cyfa()
    pro = cyfa.mixer_prologue(t["q"], t["k"], t["v"], conv_q=t["wq"], conv_k=t["wk"], conv_v=t["wv"],
                              norm_q=t["gq"], norm_k=t["gk"], z_delta=t["z_delta"], b_delta=t["b_delta"],
                              z_alpha=t["z_alpha"], b_alpha=t["b_alpha"], A=t["A"], z_beta=t["z_beta"],
                              lens=lens, conv_size=x["K"], conv_act=act)
    res = cyfa.forward(pro["q"], pro["k"], pro["v"], pro["delta"], pro["log_alpha"], pro["beta"], t["R"],
                       scale=D ** -0.5, m=x["m"], kernel=cyfa.KERNEL_MFMA, segments=segments, lens=lens,
                       K0=K0, V0=V0, clock0=clock0, return_state=True, return_logits=logits)
    out = cyfa.mixer_epilogue(res["o"], t["gate"], t["go"], lens=lens)
    return out, res


def _fused(t, x, segments, act=0, lens=None, K0=None, V0=None, clock0=None, logits=False, fuse_conv=0):
    cyfa = _cyfa()
    return cyfa.forward_mixer(t["q"], t["k"], t["v"], t["z_delta"], conv_q=t["wq"], conv_k=t["wk"],
                              conv_v=t["wv"], norm_q=t["gq"], norm_k=t["gk"], b_delta=t["b_delta"],
                              z_alpha=t["z_alpha"], b_alpha=t["b_alpha"], A=t["A"], z_beta=t["z_beta"],
                              gate=t["gate"], norm_o=t["go"], R=t["R"], scale=D ** -0.5, m=x["m"],
                              segments=segments, lens=lens, conv_size=x["K"], conv_act=act, K0=K0, V0=V0,
                              clock0=clock0, return_state=True, return_logits=logits, fuse_conv=fuse_conv)


def _assert_same(f, out, res, logits=False):
    torch.cuda.synchronize()
    diff = (f["out"].float() - out.float()).abs().max().item()
    print(f"max |fused - chain| = {diff:.3e}", flush=True)
    assert torch.equal(f["out"], out)
    assert torch.equal(f["K"], res["K"]) and torch.equal(f["V"], res["V"])
    assert torch.equal(f["clock"], res["clock"])
    if logits:
        assert torch.equal(f["logits"], res["logits"])


@pytest.mark.parametrize("fuse_conv", [0, 1])
@pytest.mark.parametrize("segments", [1, 3])
def test_bit_identical_with_chain_and_oracle(segments, fuse_conv):
    B, T, H = 2, 32 * 5 + 11, 2
    x = _inputs(B, T, H, 201)
    t = _dev(x)
    out, res = _chain(t, x, segments, logits=True)
    f = _fused(t, x, segments, logits=True, fuse_conv=fuse_conv)
    _assert_same(f, out, res, logits=True)
    # the layer output against the chained oracles
    ref_pro = mixer.prologue(x["q"], x["k"], x["v"], x["wq"], x["wk"], x["wv"], x["gq"], x["gk"],
                             x["z_delta"], x["b_delta"], x["z_alpha"], x["b_alpha"], x["A"], x["z_beta"])
    qb, kb, vb = (_bf16(ref_pro[n]) for n in ("q", "k", "v"))
    f32 = lambda a: np.asarray(a, np.float32)  # noqa: E731
    ref = oracle.forward(qb, kb, vb, f32(ref_pro["delta"]), f32(ref_pro["log_alpha"]), f32(ref_pro["beta"]),
                         x["R"], m=x["m"], scale=D ** -0.5, want_z=False)
    o_ref = np.moveaxis(ref["o"].reshape(B, H, T, D), 1, 2)
    ref_out = mixer.epilogue(o_ref, x["gate"], x["go"])
    err = rel_err(f["out"].float().cpu().numpy(), ref_out)
    print(f"layer output vs oracles: {err:.2e}", flush=True)
    assert err <= TOL_BF16


@pytest.mark.parametrize("fuse_conv", [0, 1])
@pytest.mark.parametrize("variant", ["no_conv", "no_norm", "no_gates", "width1", "width2_silu", "width3",
                                     "no_out_gate"])
def test_optional_parts(variant, fuse_conv):
    B, T, H = 1, 32 * 3 + 7, 2
    K = {"width1": 1, "width2_silu": 2, "width3": 3}.get(variant, 4)
    x = _inputs(B, T, H, 202, K=K)
    drop = {"no_conv": ("wq", "wk", "wv"), "no_norm": ("gq", "gk"),
            "no_gates": ("z_alpha", "b_alpha", "A", "z_beta", "b_delta"),
            "no_out_gate": ("gate", "go")}.get(variant, ())
    t = _dev(x, drop)
    act = 1 if variant == "width2_silu" else 0
    out, res = _chain(t, x, 1, act=act)
    f = _fused(t, x, 1, act=act, fuse_conv=fuse_conv)
    _assert_same(f, out, res)


@pytest.mark.parametrize("fuse_conv", [0, 1])
@pytest.mark.parametrize("segments", [1, 2])
def test_ragged_and_initial_state(segments, fuse_conv):
    B, T, H, m = 4, 32 * 4 + 5, 2, 127
    x = _inputs(B, T, H, 203)
    t = _dev(x)
    lens = torch.tensor([T, 0, 37, 100], dtype=torch.int32, device="cuda")
    g = torch.Generator().manual_seed(204)
    K0 = (torch.randn(B, H, 128, D, generator=g) * 0.2)
    V0 = (torch.randn(B, H, 128, D, generator=g) * 0.2)
    K0[:, :, m:] = 0
    V0[:, :, m:] = 0
    K0, V0 = K0.cuda(), V0.cuda()
    c0 = (torch.rand(B, H, generator=g, dtype=torch.float64) * 2 * m).cuda()
    out, res = _chain(t, x, segments, lens=lens, K0=K0, V0=V0, clock0=c0)
    f = _fused(t, x, segments, lens=lens, K0=K0, V0=V0, clock0=c0, fuse_conv=fuse_conv)
    _assert_same(f, out, res)
    assert torch.count_nonzero(f["out"][1]) == 0 and torch.count_nonzero(f["out"][2, 37:]) == 0


def test_rejects_unsupported():
    cyfa = _cyfa()
    q = torch.zeros(1, 32, 1, 64, dtype=torch.bfloat16, device="cuda")
    z = torch.zeros(1, 32, 1, device="cuda")
    with pytest.raises(cyfa.CyfaError) as ei:
        cyfa.forward_mixer(q, q, q, z, m=127)
    assert ei.value.status == 2


@pytest.mark.parametrize("fuse_conv", [0, 1])
def test_full_size_bit_identical(fuse_conv):
    """The 1.4B-layer shape (B 4, T 4096, H 16) in the benchmark's launch
    configuration (automatic segment count): the layer forward against the three
    standalone calls, every output element and the final states."""
    B, T, H = 4, 4096, 16
    g = torch.Generator(device="cuda")
    g.manual_seed(205)
    rnd = lambda *s, dt=torch.float32: torch.randn(s, device="cuda", generator=g).to(dt)  # noqa: E731
    bf = torch.bfloat16
    t = dict(q=rnd(B, T, H, D, dt=bf), k=rnd(B, T, H, D, dt=bf), v=rnd(B, T, H, D, dt=bf),
             gate=rnd(B, T, H, D, dt=bf), wq=0.5 * rnd(H * D, 4), wk=0.5 * rnd(H * D, 4), wv=0.5 * rnd(H * D, 4),
             gq=1 + 0.1 * rnd(D), gk=1 + 0.1 * rnd(D), go=1 + 0.1 * rnd(D), z_delta=rnd(B, T, H), b_delta=rnd(H),
             z_alpha=rnd(B, T, H), b_alpha=rnd(H) + 2, A=(rnd(H) - 1).exp(), z_beta=rnd(B, T, H),
             R=torch.eye(127, device="cuda").expand(H, 127, 127).contiguous() + 0.1 * rnd(H, 127, 127))
    x = {"K": 4, "m": 127}
    out, res = _chain(t, x, 0)
    f = _fused(t, x, 0, fuse_conv=fuse_conv)
    _assert_same(f, out, res)
    assert torch.isfinite(f["out"].float()).all()


def test_deterministic():
    B, T, H = 2, 32 * 6 + 3, 2
    x = _inputs(B, T, H, 206)
    t = _dev(x)
    a = _fused(t, x, 3, fuse_conv=1)
    b = _fused(t, x, 3, fuse_conv=1)
    torch.cuda.synchronize()
    assert torch.equal(a["out"], b["out"]) and torch.equal(a["K"], b["K"])
