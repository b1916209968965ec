"""Packed (concatenated) variable-length sequences: cyfa_forward_varlen.

Every sequence of the packed batch is compared with the oracle run on that
sequence alone (outputs, slot logits, final states and clocks), and the whole
call with cyfa_forward_lens on the same sequences padded to T rows, which runs
the same kernels: outputs, logits and states must be bit-identical.  Both the
matrix-core (bf16) and the vector-ALU (fp32) forward, with several segments /
chunk groups, empty and one-token sequences, and initial states.
"""
import numpy as np
import pytest

import oracle
from paper_2609_36259_amd.inputs import make_forward_inputs
from tests.harness import TOL_BF16, TOL_F32, clock_err, oracle_states_abs, rel_err, upload

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

LENS = [37, 0, 200, 129, 1, 64]


def _pack(t, lens):
    """padded [B, T, H, ...] device tensors -> packed [total, H, ...]"""
    out = {}
    for key, a in t.items():
        if a is None or key == "R":
            out[key] = a
            continue
        out[key] = torch.cat([a[b, :n] for b, n in enumerate(lens)], dim=0).contiguous()
    return out


def _states(B, H, d, m, seed):
    g = torch.Generator().manual_seed(seed)
    K0 = torch.randn(B, H, 128, d, generator=g) * 0.2
    V0 = torch.randn(B, H, 128, d, generator=g) * 0.2
    K0[:, :, m:] = 0
    V0[:, :, m:] = 0
    c0 = torch.rand(B, H, generator=g, dtype=torch.float64) * 2 * m
    return K0.cuda(), V0.cuda(), c0.cuda()


@pytest.mark.parametrize("kernel,dtype,segments", [("mfma", "bf16", 3), ("mfma", "bf16", 1),
                                                   ("valu", "f32", 4), ("valu", "f32", 1)])
@pytest.mark.parametrize("with_init", [False, True])
def test_varlen_matches_oracle_and_padded(kernel, dtype, segments, with_init):
    from paper_2609_36259_amd import cyfa
    kern = cyfa.KERNEL_MFMA if kernel == "mfma" else cyfa.KERNEL_VALU
    B, T, H, d, m = len(LENS), max(LENS), 2, 128, 127
    x = make_forward_inputs(B, T, H, d, d, seed=61, dtype=dtype)
    t = upload(x)
    tp = _pack(t, LENS)
    cu = torch.tensor(np.concatenate([[0], np.cumsum(LENS)]), dtype=torch.int32, device="cuda")
    lens = torch.tensor(LENS, dtype=torch.int32, device="cuda")
    init = _states(B, H, d, m, 62) if with_init else (None, None, None)
    res = cyfa.forward_varlen(tp["q"], tp["k"], tp["v"], tp["delta"], cu, tp["log_alpha"], tp["beta"],
                              t["R"], max_len=T, scale=x["scale"], kernel=kern, segments=segments,
                              K0=init[0], V0=init[1], clock0=init[2], return_state=True, return_logits=True)
    pad = cyfa.forward(t["q"], t["k"], t["v"], t["delta"], t["log_alpha"], t["beta"], t["R"],
                       scale=x["scale"], kernel=kern, segments=segments, lens=lens, K0=init[0], V0=init[1],
                       clock0=init[2], return_state=True, return_logits=True)
    torch.cuda.synchronize()
    # bit-identical with the padded entry point (same kernels, other addressing)
    assert torch.equal(res["o"], _pack({"o": pad["o"]}, LENS)["o"])
    assert torch.equal(res["logits"], _pack({"z": pad["logits"]}, LENS)["z"])
    assert torch.equal(res["K"], pad["K"]) and torch.equal(res["V"], pad["V"])
    assert torch.equal(res["clock"], pad["clock"])
    # every sequence against the oracle on its own tokens
    tol = TOL_BF16 if dtype == "bf16" else TOL_F32
    off = np.concatenate([[0], np.cumsum(LENS)])
    o_all = res["o"].float().cpu().numpy()
    z_all = res["logits"].cpu().numpy()
    worst = {}
    for b, n in enumerate(LENS):
        xs = {key: (a[b:b + 1, :max(n, 1)] if key not in ("R", "scale", "m", "dtype") and a is not None else a)
              for key, a in x.items()}
        kw = {}
        if with_init:
            Kr = np.stack([oracle.relative_from_storage(m, init[2][b, hh].item(), init[0][b, hh].cpu().numpy())
                           for hh in range(H)])
            Vr = np.stack([oracle.relative_from_storage(m, init[2][b, hh].item(), init[1][b, hh].cpu().numpy())
                           for hh in range(H)])
            kw = dict(K0=Kr, V0=Vr, lam0=init[2][b].cpu().numpy())
        ref = oracle.forward(xs["q"], xs["k"], xs["v"], xs["delta"], xs["log_alpha"], xs["beta"], x["R"],
                             m=m, scale=x["scale"], T_run=n, **kw)
        if n > 0:
            got = o_all[off[b]:off[b + 1]].transpose(1, 0, 2)            # [H, n, d]
            worst["o"] = max(worst.get("o", 0), rel_err(got, ref["o"]))
            gz = z_all[off[b]:off[b + 1]].transpose(1, 0, 2)
            worst["z"] = max(worst.get("z", 0), rel_err(gz, ref["z"]))
        Kref, Vref = oracle_states_abs(ref, m)
        if np.abs(Kref).max() > 0:
            worst["K"] = max(worst.get("K", 0), rel_err(res["K"][b].cpu().numpy(), Kref))
            worst["V"] = max(worst.get("V", 0), rel_err(res["V"][b].cpu().numpy(), Vref))
        else:
            assert torch.count_nonzero(res["K"][b]) == 0 and torch.count_nonzero(res["V"][b]) == 0
        worst["clock"] = max(worst.get("clock", 0), clock_err(res["clock"][b].cpu().numpy(), ref["lam"], m))
    print("errors", {k: f"{v:.2e}" for k, v in worst.items()}, flush=True)
    for key, v in worst.items():
        assert v <= (1e-9 if key == "clock" else tol), (key, v)


def test_varlen_rejects_missing_offsets():
    from paper_2609_36259_amd import cyfa
    q = torch.zeros(4, 2, 128, dtype=torch.bfloat16, device="cuda")
    d = torch.zeros(4, 2, device="cuda")
    with pytest.raises(cyfa.CyfaError):
        cyfa.load()
        desc = cyfa.forward_desc(2, 4, 2, 128, 128)
        ws = torch.empty(cyfa.forward_workspace_size(desc), dtype=torch.uint8, device="cuda")
        import ctypes
        cyfa._check(cyfa.load().cyfa_forward_varlen(ctypes.byref(desc), cyfa._ptr(q), cyfa._ptr(q), cyfa._ptr(q),
                                                     cyfa._ptr(d), None, None, None, None, None, None, None,
                                                     cyfa._ptr(q), None, None, None, None, cyfa._ptr(ws),
                                                     ctypes.c_size_t(ws.numel()), None))
