"""End-to-end parity of a CyFA layer's operator chain on the GPU: mixer prologue
(ShortConv, QK RMSNorm, gates) -> cyfa_forward -> mixer epilogue (head-wise
RMSNorm, sigmoid output gate), against the chain of the oracles on the same
inputs.  The GPU chain passes bf16 q, k, v between its kernels; the oracle chain
rounds its prologue's q, k, v to bf16 at the same point, so both see the same
operator inputs up to the prologue's own rounding.  Bar 2e-2 (bf16)."""
import numpy as np
import pytest

import oracle
from oracle import mixer
from tests.harness import TOL_BF16, rel_err

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _bf16(a):
    return torch.tensor(np.asarray(a, np.float32)).bfloat16().float().numpy()


@pytest.mark.parametrize("kernel", ["mfma", "valu"])
def test_layer_chain(kernel):
    from paper_2609_36259_amd import cyfa
    B, T, H, d, m = 2, 150, 2, 128, 127
    rng = np.random.default_rng(91)
    rnd = lambda *s: rng.standard_normal(s).astype(np.float32)  # noqa: E731
    x = dict(q=_bf16(rnd(B, T, H, d)), k=_bf16(rnd(B, T, H, d)), v=_bf16(rnd(B, T, H, d)),
             wq=0.5 * rnd(H * d, 4), wk=0.5 * rnd(H * d, 4), wv=0.5 * rnd(H * d, 4),
             gq=1 + 0.1 * rnd(d), gk=1 + 0.1 * rnd(d), z_delta=rnd(B, T, H), b_delta=rnd(H),
             z_alpha=rnd(B, T, H), b_alpha=rnd(H) + 2, A=np.exp(rnd(H) - 1), z_beta=rnd(B, T, H),
             R=(np.eye(m) + 0.1 * rnd(H, m, m)).astype(np.float32),
             gate=_bf16(2 * rnd(B, T, H, d)), go=1 + 0.1 * rnd(d))
    scale = d ** -0.5
    dev = lambda a, dt=torch.float32: torch.tensor(a, dtype=dt, device="cuda")  # noqa: E731
    bf = torch.bfloat16
    pro = cyfa.mixer_prologue(dev(x["q"], bf), dev(x["k"], bf), dev(x["v"], bf), conv_q=dev(x["wq"]),
                              conv_k=dev(x["wk"]), conv_v=dev(x["wv"]), norm_q=dev(x["gq"]),
                              norm_k=dev(x["gk"]), z_delta=dev(x["z_delta"]), b_delta=dev(x["b_delta"]),
                              z_alpha=dev(x["z_alpha"]), b_alpha=dev(x["b_alpha"]), A=dev(x["A"]),
                              z_beta=dev(x["z_beta"]))
    o = cyfa.forward(pro["q"], pro["k"], pro["v"], pro["delta"], pro["log_alpha"], pro["beta"],
                     dev(x["R"]), scale=scale, m=m,
                     kernel=cyfa.KERNEL_MFMA if kernel == "mfma" else cyfa.KERNEL_VALU)
    out = cyfa.mixer_epilogue(o, dev(x["gate"], bf), dev(x["go"]))
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()

    ref_pro = mixer.prologue(x["q"], x["k"], x["v"], x["wq"], x["wk"], x["wv"], x["gq"], x["gk"],
                             x["z_delta"], x["b_delta"], x["z_alpha"], x["b_alpha"], x["A"], x["z_beta"])
    # the operator consumes bf16 q, k, v and fp32 gates, as on the GPU
    qb, kb, vb = (_bf16(ref_pro[n]) for n in ("q", "k", "v"))
    f32 = lambda a: np.asarray(a, np.float32)  # noqa: E731
    ref = oracle.forward(qb, kb, vb, f32(ref_pro["delta"]), f32(ref_pro["log_alpha"]),
                         f32(ref_pro["beta"]), x["R"], m=m, scale=scale, want_z=False)
    o_ref = np.moveaxis(ref["o"].reshape(B, H, T, d), 1, 2)
    ref_out = mixer.epilogue(o_ref, x["gate"], x["go"])
    err = rel_err(got, ref_out)
    err_o = rel_err(o.float().cpu().numpy(), o_ref)
    print(f"layer chain ({kernel}): operator output {err_o:.2e}, layer output {err:.2e}", flush=True)
    assert err_o <= TOL_BF16 and err <= TOL_BF16
