"""GPU parity of the vector-ALU forward kernel and of the decode step against the oracle."""
import numpy as np
import pytest
import oracle

from paper_2609_36259_amd.inputs import (DECODE, FWD_TINY, make_decode_inputs, make_forward_inputs,
                                         workload_inputs)
from tests.harness import (TOL_BF16, TOL_F32, clock_err, oracle_states_abs, pairs_view, rel_err,
                           run_oracle, state_view, upload)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _cyfa():
    from paper_2609_36259_amd import cyfa
    return cyfa


def _fwd(x, t, **kw):
    return _cyfa().forward(t["q"], t["k"], t["v"], t["delta"], t["log_alpha"], t["beta"], t["R"],
                           scale=x["scale"], m=x["m"], **kw)


def _check_full(x, res, tol, *, check_state=True):
    B, T, H = x["delta"].shape
    ref = run_oracle(x)
    pairs = list(range(B * H))
    e_o = rel_err(pairs_view(res["o"], pairs, H), ref["o"])
    out = {"o": e_o}
    if "logits" in res:
        out["z"] = rel_err(pairs_view(res["logits"], pairs, H), ref["z"])
    if check_state and "K" in res:
        Kref, Vref = oracle_states_abs(ref, x["m"])
        out["K"] = rel_err(state_view(res["K"], pairs, H), Kref)
        out["V"] = rel_err(state_view(res["V"], pairs, H), Vref)
        out["clock"] = clock_err(res["clock"].cpu().numpy().reshape(-1), ref["lam"], x["m"])
    print("errors", {k: f"{v:.2e}" for k, v in out.items()}, flush=True)
    for k, v in out.items():
        assert v <= (1e-9 if k == "clock" else tol), (k, v)
    return out


def test_tiny_f32_workload_full_parity():
    x = workload_inputs(FWD_TINY)
    t = upload(x)
    res = _fwd(x, t, return_state=True, return_logits=True)
    _check_full(x, res, TOL_F32)


@pytest.mark.parametrize("variant", ["no_beta_no_R", "peaky", "small_m", "ragged_chunk8",
                                     "d128_f32", "mixed_dims", "d256_f32", "mixed_256",
                                     "m255_d64", "m255_d128", "m255_mixed", "m129"])
def test_f32_variants(variant):
    kw = {}
    dk = dv = 64
    B, T, H, m = 1, 130, 2, 127
    if variant == "small_m":
        m = 7
    if variant == "ragged_chunk8":
        T, kw = 77, {"chunk": 8}
    if variant == "d128_f32":
        dk = dv = 128
    if variant == "d256_f32":          # the paper's head size (512-thread workgroups)
        dk = dv = 256
        T = 70
    if variant == "mixed_256":
        dk, dv, T = 256, 64, 70
    if variant.startswith("m255"):     # the largest slot count of the paper's ablation
        m, T = 255, 70
        dk, dv = {"m255_d64": (64, 64), "m255_d128": (128, 128), "m255_mixed": (128, 64)}[variant]
    if variant == "m129":              # smallest slot count with 256 storage rows
        m, T = 129, 53
    x = make_forward_inputs(B, T, H, dk, dv, seed=21, dtype="f32", m=m,
                            with_beta=variant != "no_beta_no_R", with_R=variant != "no_beta_no_R")
    if variant == "mixed_dims":
        y = make_forward_inputs(B, T, H, 128, 64, seed=22, dtype="f32")
        x = y
    if variant == "peaky":
        x["scale"] = 30.0
    t = upload(x)
    res = _fwd(x, t, return_state=True, return_logits=True, **kw)
    _check_full(x, res, TOL_F32)


def test_bf16_valu_kernel_d256():
    x = make_forward_inputs(1, 45, 2, 256, 256, seed=24, dtype="bf16")
    t = upload(x)
    res = _fwd(x, t, return_state=True, return_logits=True)
    _check_full(x, res, TOL_BF16)


def test_bf16_m255_and_resume():
    """m = 255 (256 storage rows) with bf16 inputs on the vector-ALU kernel (the
    matrix-core one has its own tests); split-and-resume through the 256-row states
    equals one pass."""
    cyfa = _cyfa()
    x = make_forward_inputs(2, 60, 2, 128, 128, seed=25, dtype="bf16", m=255)
    t = upload(x)
    full = _fwd(x, t, return_state=True, return_logits=True, kernel=cyfa.KERNEL_VALU)
    assert full["K"].shape == (2, 2, 256, 128)
    _check_full(x, full, TOL_BF16)
    t1 = 29
    a = {k: (v[:, :t1].contiguous() if v is not None and k != "R" else v) for k, v in t.items()}
    b = {k: (v[:, t1:].contiguous() if v is not None and k != "R" else v) for k, v in t.items()}
    first = _fwd(x, a, return_state=True, kernel=cyfa.KERNEL_VALU)
    second = cyfa.forward(b["q"], b["k"], b["v"], b["delta"], b["log_alpha"], b["beta"], b["R"],
                          scale=x["scale"], m=255, K0=first["K"], V0=first["V"], clock0=first["clock"],
                          return_state=True, kernel=cyfa.KERNEL_VALU)
    torch.cuda.synchronize()
    o_split = torch.cat([first["o"], second["o"]], dim=1).float().cpu().numpy()
    assert rel_err(o_split, full["o"].float().cpu().numpy()) <= 1e-2
    assert rel_err(second["K"].cpu().numpy(), full["K"].cpu().numpy()) <= 1e-5
    assert clock_err(second["clock"].cpu().numpy(), full["clock"].cpu().numpy(), 255) <= 1e-9


def test_bf16_valu_kernel():
    x = make_forward_inputs(2, 150, 3, 128, 128, seed=23, dtype="bf16")
    t = upload(x)
    res = _fwd(x, t, return_state=True, return_logits=True, kernel=_cyfa().KERNEL_VALU)
    _check_full(x, res, TOL_BF16)


def test_split_and_resume_equals_one_pass():
    cyfa = _cyfa()
    x = make_forward_inputs(2, 100, 2, 64, 64, seed=24, dtype="f32")
    t = upload(x)
    full = _fwd(x, t, return_state=True)
    t1 = 37
    a = {k: (v[:, :t1].contiguous() if v is not None and k != "R" else v) for k, v in t.items()}
    b = {k: (v[:, t1:].contiguous() if v is not None and k != "R" else v) for k, v in t.items()}
    first = _fwd(x, a, return_state=True)
    second = cyfa.forward(b["q"], b["k"], b["v"], b["delta"], b["log_alpha"], b["beta"], b["R"],
                          scale=x["scale"], K0=first["K"], V0=first["V"], clock0=first["clock"],
                          return_state=True)
    torch.cuda.synchronize()
    o_split = torch.cat([first["o"], second["o"]], dim=1)
    assert rel_err(o_split.cpu().numpy(), full["o"].cpu().numpy()) <= 1e-5
    assert rel_err(second["K"].cpu().numpy(), full["K"].cpu().numpy()) <= 1e-5
    assert clock_err(second["clock"].cpu().numpy(), full["clock"].cpu().numpy(), 127) <= 1e-9


def test_empty_sequence_returns_initial_state():
    cyfa = _cyfa()
    x = make_forward_inputs(1, 0, 2, 64, 64, seed=25, dtype="f32")
    t = upload(x)
    K0 = torch.randn(1, 2, 128, 64, device="cuda")
    K0[:, :, 127:] = 0
    V0 = torch.randn(1, 2, 128, 64, device="cuda")
    V0[:, :, 127:] = 0
    c0 = torch.tensor([[3.5, 200.25]], dtype=torch.float64, device="cuda")
    res = cyfa.forward(t["q"], t["k"], t["v"], t["delta"], t["log_alpha"], t["beta"], t["R"],
                       K0=K0, V0=V0, clock0=c0, return_state=True)
    torch.cuda.synchronize()
    assert torch.equal(res["K"], K0) and torch.equal(res["V"], V0)
    np.testing.assert_allclose(res["clock"].cpu().numpy(), [[3.5, 200.25 - 127]], atol=1e-12)


def test_deterministic():
    x = make_forward_inputs(1, 64, 2, 64, 64, seed=26, dtype="f32")
    t = upload(x)
    a = _fwd(x, t)
    b = _fwd(x, t)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_nan_input_propagates_without_fault():
    x = make_forward_inputs(1, 40, 1, 64, 64, seed=27, dtype="f32")
    x["q"][0, 10, 0, 3] = np.nan
    t = upload(x)
    o = _fwd(x, t)
    torch.cuda.synchronize()
    o = o.cpu().numpy()
    assert np.isnan(o[0, 10]).all()
    assert np.isfinite(o[0, :10]).all()


def _decode_case(N, H, d, prefix, steps, seed, dtype="f32", with_logits=True, m=127):
    cyfa = _cyfa()
    x = make_forward_inputs(N, prefix + steps, H, d, d, seed=seed, dtype=dtype, m=m)
    ref = run_oracle(x)
    t = upload(x)
    pre = {k: (v[:, :prefix].contiguous() if v is not None and k != "R" else v) for k, v in t.items()}
    st = cyfa.forward(pre["q"], pre["k"], pre["v"], pre["delta"], pre["log_alpha"], pre["beta"],
                      pre["R"], scale=x["scale"], m=m, return_state=True)
    K, V, clk = st["K"], st["V"], st["clock"]
    outs, logits = [], []
    for s in range(steps):
        tok = {k: (v[:, prefix + s].contiguous() if v is not None and k != "R" else v)
               for k, v in t.items()}
        o, z = cyfa.decode_step(tok["q"], tok["k"], tok["v"], tok["delta"], K, V, clk,
                                tok["log_alpha"], tok["beta"], t["R"], scale=x["scale"], m=m,
                                return_logits=True)
        outs.append(o.float().cpu().numpy())
        logits.append(z.cpu().numpy())
    torch.cuda.synchronize()
    pairs = list(range(N * H))
    got = np.stack(outs, axis=1)                       # [N, steps, H, d]
    got = np.stack([got[p // H, :, p % H] for p in pairs])
    zg = np.stack(logits, axis=1)
    zg = np.stack([zg[p // H, :, p % H] for p in pairs])
    e_o = rel_err(got, ref["o"][:, prefix:])
    e_z = rel_err(zg, ref["z"][:, prefix:])
    Kref, Vref = oracle_states_abs(ref, x["m"])
    e_K = rel_err(state_view(K, pairs, H), Kref)
    e_c = clock_err(clk.cpu().numpy().reshape(-1), ref["lam"], x["m"])
    print(f"decode errors o {e_o:.2e} z {e_z:.2e} K {e_K:.2e} clock {e_c:.1e}", flush=True)
    return e_o, e_z, e_K, e_c


@pytest.mark.parametrize("d", [64, 128, 256])
def test_decode_steps_match_oracle_f32(d):
    e_o, e_z, e_K, e_c = _decode_case(3, 2, d, prefix=33, steps=6, seed=30 + d)
    assert e_o <= TOL_F32 and e_z <= TOL_F32 and e_K <= TOL_F32 and e_c <= 1e-9


@pytest.mark.parametrize("d", [64, 128])
def test_decode_steps_match_oracle_m255(d):
    """256 storage rows (m = 255): forward prefix, then decode steps, against the oracle."""
    e_o, e_z, e_K, e_c = _decode_case(2, 2, d, prefix=21, steps=5, seed=40 + d, m=255)
    assert e_o <= TOL_F32 and e_z <= TOL_F32 and e_K <= TOL_F32 and e_c <= 1e-9


def test_decode_steps_match_oracle_bf16():
    e_o, e_z, e_K, e_c = _decode_case(2, 3, 128, prefix=20, steps=4, seed=33, dtype="bf16")
    assert e_o <= TOL_BF16 and e_z <= TOL_BF16 and e_K <= TOL_BF16 and e_c <= 1e-9


def test_decode_rejects_strided_output():
    cyfa = _cyfa()
    x = make_forward_inputs(2, 1, 2, 64, 64, seed=35, dtype="f32")
    t = upload(x)
    K = torch.zeros(2, 2, 128, 64, device="cuda")
    V = torch.zeros(2, 2, 128, 64, device="cuda")
    clk = torch.zeros(2, 2, dtype=torch.float64, device="cuda")
    big = torch.empty(2, 3, 2, 64, device="cuda")
    with pytest.raises(ValueError):
        cyfa.decode_step(t["q"][:, 0], t["k"][:, 0], t["v"][:, 0], t["delta"][:, 0], K, V, clk,
                         out=big[:, 1])


def test_decode_consistent_with_forward():
    """forward over T+1 tokens == forward over T tokens, then one decode step."""
    cyfa = _cyfa()
    x = make_forward_inputs(2, 41, 2, 128, 128, seed=34, dtype="f32")
    t = upload(x)
    full = _fwd(x, t, return_state=True)
    pre = {k: (v[:, :40].contiguous() if v is not None and k != "R" else v) for k, v in t.items()}
    st = cyfa.forward(pre["q"], pre["k"], pre["v"], pre["delta"], pre["log_alpha"], pre["beta"],
                      pre["R"], scale=x["scale"], return_state=True)
    tok = {k: (v[:, 40].contiguous() if v is not None and k != "R" else v) for k, v in t.items()}
    o = cyfa.decode_step(tok["q"], tok["k"], tok["v"], tok["delta"], st["K"], st["V"], st["clock"],
                         tok["log_alpha"], tok["beta"], t["R"], scale=x["scale"])
    torch.cuda.synchronize()
    assert rel_err(o.cpu().numpy(), full["o"][:, 40].cpu().numpy()) <= 1e-5
    assert rel_err(st["K"].cpu().numpy(), full["K"].cpu().numpy()) <= 1e-5


def test_decode_full_size_sampled():
    """256 streams x 16 heads, d = 128: 512-token prefix (GPU forward), then 64
    decode steps; every stream of one head (256 stream-heads, all sharing that
    head's readout matrix) plus stream-heads of the other heads compared with the
    oracle stepped token by token over all 576 tokens."""
    cyfa = _cyfa()
    N, H, d = DECODE.B, DECODE.H, DECODE.dk
    prefix, steps = DECODE.extra["prefix"], DECODE.extra["steps"]
    x = make_decode_inputs(N, H, d, prefix, steps, seed=DECODE.seed)
    x["dtype"] = "f32"
    t = upload(x)
    pre = {k: (v[:, :prefix].contiguous() if v is not None and k != "R" else v) for k, v in t.items()}
    st = cyfa.forward(pre["q"], pre["k"], pre["v"], pre["delta"], pre["log_alpha"], pre["beta"],
                      pre["R"], scale=x["scale"], return_state=True)
    del pre
    K, V, clk = st["K"], st["V"], st["clock"]
    outs = torch.empty((N, steps, H, d), device="cuda")
    ws = torch.empty(cyfa.decode_workspace_size(cyfa.decode_desc(N, H, d, d)), dtype=torch.uint8,
                     device="cuda")
    for s_ in range(steps):
        tok = {k: (v[:, prefix + s_].contiguous() if v is not None and k != "R" else v)
               for k, v in t.items()}
        o_step = cyfa.decode_step(tok["q"], tok["k"], tok["v"], tok["delta"], K, V, clk,
                                  tok["log_alpha"], tok["beta"], t["R"], scale=x["scale"],
                                  workspace=ws)
        outs[:, s_] = o_step
    torch.cuda.synchronize()
    head = 5
    pairs = [n * H + head for n in range(N)] + [0, N * H - 1, 1000, 2050, 3333, 17 * H + 11]
    ref = oracle_forward_decode(x, pairs)
    got = outs.cpu().numpy()
    got = np.stack([got[p // H, :, p % H] for p in pairs])
    e_o = rel_err(got, ref["o"][:, prefix:])
    Kref, _ = oracle_states_abs(ref, x["m"])
    e_K = rel_err(state_view(K, pairs, H), Kref)
    e_c = clock_err(clk.cpu().numpy().reshape(-1)[pairs], ref["lam"], x["m"])
    print(f"decode full-size errors o {e_o:.2e} K {e_K:.2e} clock {e_c:.1e}", flush=True)
    assert e_o <= TOL_F32 and e_K <= TOL_F32 and e_c <= 1e-9


def oracle_forward_decode(x, pairs):
    import oracle
    return oracle.forward(x["q"], x["k"], x["v"], x["delta"], x["log_alpha"], x["beta"], x["R"],
                          m=x["m"], scale=x["scale"], pairs=np.array(pairs, np.int32), want_z=False)


@pytest.mark.parametrize("segments,chunk", [(1, 16), (3, 16), (5, 8), (0, 16)])
def test_valu_chunk_groups(segments, chunk):
    """The vector-ALU forward over chunk groups (each group's entering state from a
    pre-pass over the earlier groups) against the oracle, with an initial state."""
    cyfa = _cyfa()
    x = make_forward_inputs(2, 16 * 9 + 5, 2, 64, 128, seed=26, dtype="f32")
    t = upload(x)
    g = torch.Generator().manual_seed(3)
    K0 = torch.randn(2, 2, 128, 64, generator=g) * 0.2
    V0 = torch.randn(2, 2, 128, 128, generator=g) * 0.2
    K0[:, :, 127:] = 0
    V0[:, :, 127:] = 0
    c0 = torch.rand(2, 2, generator=g, dtype=torch.float64) * 127
    res = _fwd(x, t, return_state=True, return_logits=True, kernel=cyfa.KERNEL_VALU, segments=segments,
               chunk=chunk, K0=K0.cuda(), V0=V0.cuda(), clock0=c0.cuda())
    torch.cuda.synchronize()
    B, T, H = x["delta"].shape
    pairs = list(range(B * H))
    Kr = np.stack([oracle.relative_from_storage(127, c0.reshape(-1)[p].item(), K0.reshape(4, 128, 64)[p].numpy())
                   for p in pairs])
    Vr = np.stack([oracle.relative_from_storage(127, c0.reshape(-1)[p].item(), V0.reshape(4, 128, 128)[p].numpy())
                   for p in pairs])
    ref = run_oracle(x, K0=Kr, V0=Vr, lam0=c0.reshape(-1).numpy())
    errs = {"o": rel_err(pairs_view(res["o"], pairs, H), ref["o"]),
            "z": rel_err(pairs_view(res["logits"], pairs, H), ref["z"])}
    Kref, Vref = oracle_states_abs(ref, 127)
    errs["K"] = rel_err(state_view(res["K"], pairs, H), Kref)
    errs["V"] = rel_err(state_view(res["V"], pairs, H), Vref)
    errs["clock"] = clock_err(res["clock"].cpu().numpy().reshape(-1), ref["lam"], 127)
    print("errors", {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    for k, v in errs.items():
        assert v <= (1e-9 if k == "clock" else TOL_F32), (k, v)


def test_valu_full_size_f32_chunk_groups():
    """The vector-ALU forward at the 1.4B layer shape (B4 T4096 H16 d128) with fp32
    inputs, in its automatic chunk-group split (the fp32 path of that shape);
    eight (b, h) sequences, first, last and interior, compared over all tokens."""
    from paper_2609_36259_amd.inputs import FWD_1P4B
    cyfa = _cyfa()
    w = FWD_1P4B
    x = make_forward_inputs(w.B, w.T, w.H, w.dk, w.dv, seed=w.seed, dtype="f32")
    t = upload(x)
    res = _fwd(x, t, kernel=cyfa.KERNEL_VALU, return_state=True, return_logits=True)
    torch.cuda.synchronize()
    B, T, H = x["delta"].shape
    pairs = [0, 1, 17, 31, 32, 46, 62, B * H - 1]
    ref = run_oracle(x, pairs=np.array(pairs, np.int32))
    errs = {"o": rel_err(pairs_view(res["o"], pairs, H), ref["o"]),
            "z": rel_err(pairs_view(res["logits"], pairs, H), ref["z"])}
    Kref, Vref = oracle_states_abs(ref, x["m"])
    errs["K"] = rel_err(state_view(res["K"], pairs, H), Kref)
    errs["V"] = rel_err(state_view(res["V"], pairs, H), Vref)
    errs["clock"] = clock_err(res["clock"].cpu().numpy().reshape(-1)[pairs], ref["lam"], x["m"])
    print("errors", {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    for k, v in errs.items():
        assert v <= (1e-9 if k == "clock" else TOL_F32), (k, v)
