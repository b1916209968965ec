"""GPU parity of the bf16 matrix-core forward at head dimension 256 (d_k = d_v =
256, the paper's head size) against the oracle.

Small cases compare every output element, slot logit, final state and clock
with the oracle over several 32-token chunks and a ragged tail, with sequences
cut into one or several segments; the paper's
operator shape (B 32, T 2048, H 4, d 256) runs in the benchmark's launch
configuration and is compared on sampled (b, h) sequences over all tokens.
Bar: max relative error 2e-2 (bf16 inputs, fp32 accumulation), clocks 1e-9.
"""
import numpy as np
import pytest

import oracle
from paper_2609_36259_amd.inputs import FWD_PAPER_OP, make_forward_inputs, workload_inputs
from tests.harness import (TOL_BF16, clock_err, oracle_states_abs, pairs_view, rel_err,
                           run_oracle, state_view, upload)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

D = 256


def _cyfa():
    from paper_2609_36259_amd import cyfa
    return cyfa


def _fwd(x, t, **kw):
    cyfa = _cyfa()
    kw.setdefault("kernel", cyfa.KERNEL_MFMA)
    return cyfa.forward(t["q"], t["k"], t["v"], t["delta"], t["log_alpha"], t["beta"], t["R"],
                        scale=x["scale"], m=x["m"], **kw)


def _errors(x, res, pairs=None, **okw):
    B, T, H = x["delta"].shape
    pairs = list(range(B * H)) if pairs is None else list(pairs)
    ref = run_oracle(x, pairs=np.array(pairs, np.int32), **okw)
    out = {"o": rel_err(pairs_view(res["o"], pairs, H), ref["o"])}
    if "logits" in res:
        out["z"] = rel_err(pairs_view(res["logits"], pairs, H), ref["z"])
    if "K" in res:
        Kref, Vref = oracle_states_abs(ref, x["m"])
        out["K"] = rel_err(state_view(res["K"], pairs, H), Kref)
        out["V"] = rel_err(state_view(res["V"], pairs, H), Vref)
        out["clock"] = clock_err(res["clock"].cpu().numpy().reshape(-1)[pairs], ref["lam"], x["m"])
    print("errors", {k: f"{v:.2e}" for k, v in out.items()}, flush=True)
    return out


def _assert_ok(err, tol=TOL_BF16):
    for k, v in err.items():
        assert v <= (1e-9 if k == "clock" else tol), (k, v)


def _init_states(B, H, m, seed):
    g = torch.Generator().manual_seed(seed)
    K0 = torch.randn(B, H, 128, D, generator=g) * 0.2
    V0 = torch.randn(B, H, 128, D, generator=g) * 0.2
    K0[:, :, m:] = 0
    V0[:, :, m:] = 0
    c0 = torch.rand(B, H, generator=g, dtype=torch.float64) * 3 * m
    return K0.cuda(), V0.cuda(), c0.cuda()


def _oracle_init(m, K0, V0, c0):
    """absolute-clock storage [B, H, 128, d] -> the oracle's relative-time states per pair"""
    B, H = c0.shape
    K, V, lam = [], [], []
    for b in range(B):
        for h in range(H):
            c = c0[b, h].item()
            K.append(oracle.relative_from_storage(m, c, K0[b, h].cpu().numpy()))
            V.append(oracle.relative_from_storage(m, c, V0[b, h].cpu().numpy()))
            lam.append(c)
    return dict(K0=np.stack(K), V0=np.stack(V), lam0=np.array(lam))


def test_selected_for_bf16_d256():
    cyfa = _cyfa()
    assert cyfa.selected_kernel(cyfa.forward_desc(2, 100, 2, D, D, dtype=cyfa.BF16)) == "mfma"


@pytest.mark.parametrize("chunk", [32, 64])
def test_small_full_parity(chunk):
    x = make_forward_inputs(2, 200, 3, D, D, seed=71, dtype="bf16")
    t = upload(x)
    res = _fwd(x, t, chunk=chunk, return_state=True, return_logits=True)
    _assert_ok(_errors(x, res))


def test_chunk_64_is_two_chunks_of_32():
    x = make_forward_inputs(1, 64 * 3 + 9, 2, D, D, seed=72, dtype="bf16")
    t = upload(x)
    for sgm in (1, 3):
        a = _fwd(x, t, chunk=32, segments=sgm, return_state=True)
        b = _fwd(x, t, chunk=64, segments=sgm, return_state=True)
        torch.cuda.synchronize()
        assert torch.equal(a["o"], b["o"]) and torch.equal(a["K"], b["K"]) and torch.equal(a["V"], b["V"])


@pytest.mark.parametrize("segments", [1, 2, 3, 7])
@pytest.mark.parametrize("with_init", [False, True])
def test_segments_against_oracle(segments, with_init):
    """Sequences cut into segments: the pre-pass and the scan of the entering
    states run on the two 128-channel blocks of each head; every output, logit,
    final state and clock against the oracle, with and without an initial state."""
    m = 127
    x = make_forward_inputs(2, 32 * 9 + 13, 2, D, D, seed=87, dtype="bf16", m=m)
    t = upload(x)
    if with_init:
        K0, V0, c0 = _init_states(2, 2, m, 88)
        res = _fwd(x, t, segments=segments, K0=K0, V0=V0, clock0=c0, return_state=True, return_logits=True)
        _assert_ok(_errors(x, res, **_oracle_init(m, K0, V0, c0)))
    else:
        res = _fwd(x, t, segments=segments, return_state=True, return_logits=True)
        _assert_ok(_errors(x, res))


def test_segment_count_changes_only_rounding():
    x = make_forward_inputs(1, 32 * 11 + 5, 2, D, D, seed=89, dtype="bf16")
    t = upload(x)
    outs = [_fwd(x, t, segments=sgm, return_state=True) for sgm in (1, 2, 5, 12)]
    torch.cuda.synchronize()
    base = outs[0]["o"].float().cpu().numpy()
    for r in outs[1:]:
        assert rel_err(r["o"].float().cpu().numpy(), base) <= 1e-2
        assert rel_err(r["K"].cpu().numpy(), outs[0]["K"].cpu().numpy()) <= 1e-2
        assert rel_err(r["V"].cpu().numpy(), outs[0]["V"].cpu().numpy()) <= 1e-2
        assert clock_err(r["clock"].cpu().numpy(), outs[0]["clock"].cpu().numpy(), 127) <= 1e-9


@pytest.mark.parametrize("variant", ["no_beta_no_R", "small_m", "m63", "short", "one_token"])
def test_variants(variant):
    B, T, H, m = 1, 150, 2, 127
    if variant == "small_m":
        m = 9
    if variant == "m63":
        m = 63
    if variant == "short":
        T = 37
    if variant == "one_token":
        T = 1
    x = make_forward_inputs(B, T, H, D, D, seed=73, dtype="bf16", m=m,
                            with_beta=variant != "no_beta_no_R", with_R=variant != "no_beta_no_R")
    t = upload(x)
    res = _fwd(x, t, return_state=True, return_logits=True)
    _assert_ok(_errors(x, res))


def test_extreme_and_mixed_gates():
    """Heavy forgetting (the state-rescaling path), no forgetting, near-total
    erasure, and a case with no gates at all."""
    x = make_forward_inputs(1, 517, 2, D, D, seed=74, dtype="bf16")
    g = x["log_alpha"]
    g[:, 40:140] = -6.0
    g[:, 200:330] = 0.0
    g[:, 400:410] = -40.0
    t = upload(x)
    for sgm in (1, 3):
        res = _fwd(x, t, segments=sgm, return_state=True, return_logits=True)
        _assert_ok(_errors(x, res))
    y = make_forward_inputs(1, 300, 2, D, D, seed=75, dtype="bf16")
    y["log_alpha"] = None
    y["beta"] = None
    res = _fwd(y, upload(y), segments=2, return_state=True)
    _assert_ok(_errors(y, res))


@pytest.mark.parametrize("gate", [-0.8, -1.5])
def test_eager_rescale_paths(gate):
    """Chunks whose decay leaves the lazy e^+-60 range: -0.8 rescales the states
    and factors the decay into a per-token scale, -1.5 keeps Gamma in the score
    tiles."""
    x = make_forward_inputs(1, 431, 2, D, D, seed=76, dtype="bf16")
    x["log_alpha"][:, 40:360] = gate
    res = _fwd(x, upload(x), segments=2, return_state=True, return_logits=True)
    _assert_ok(_errors(x, res))


def test_initial_state_against_oracle():
    m = 127
    x = make_forward_inputs(2, 161, 2, D, D, seed=77, dtype="bf16", m=m)
    K0, V0, c0 = _init_states(2, 2, m, 78)
    res = _fwd(x, upload(x), K0=K0, V0=V0, clock0=c0, return_state=True, return_logits=True)
    _assert_ok(_errors(x, res, **_oracle_init(m, K0, V0, c0)))


def test_resume_matches_one_call():
    cyfa = _cyfa()
    x = make_forward_inputs(2, 300, 2, D, D, seed=79, dtype="bf16")
    t = upload(x)
    full = _fwd(x, t, return_state=True)
    for t1 in (128, 157):
        a = {k: (v[:, :t1].contiguous() if v is not None and k != "R" else v) for k, v in t.items()}
        b = {k: (v[:, t1:].contiguous() if v is not None and k != "R" else v) for k, v in t.items()}
        first = _fwd(x, a, return_state=True)
        second = cyfa.forward(b["q"], b["k"], b["v"], b["delta"], b["log_alpha"], b["beta"], b["R"],
                              scale=x["scale"], K0=first["K"], V0=first["V"], clock0=first["clock"],
                              return_state=True, kernel=cyfa.KERNEL_MFMA)
        torch.cuda.synchronize()
        o_split = torch.cat([first["o"], second["o"]], dim=1).float().cpu().numpy()
        assert rel_err(o_split, full["o"].float().cpu().numpy()) <= 1e-2
        assert rel_err(second["K"].cpu().numpy(), full["K"].cpu().numpy()) <= 1e-2
        assert rel_err(second["V"].cpu().numpy(), full["V"].cpu().numpy()) <= 1e-2
        assert clock_err(second["clock"].cpu().numpy(), full["clock"].cpu().numpy(), 127) <= 1e-9
    _assert_ok(_errors(x, full))


@pytest.mark.parametrize("segments", [1, 3])
def test_resume_in_place(segments):
    """Final state and clock written over the initial ones; with several segments
    every workgroup must have read its entering clock and state before any writes
    them."""
    cyfa = _cyfa()
    x = make_forward_inputs(2, 300, 2, D, D, seed=80, dtype="bf16")
    t = upload(x)
    t1 = 137
    a = {k: (v[:, :t1].contiguous() if v is not None and k != "R" else v) for k, v in t.items()}
    b = {k: (v[:, t1:].contiguous() if v is not None and k != "R" else v) for k, v in t.items()}
    first = _fwd(x, a, return_state=True, segments=segments)
    K, V, clk = first["K"], first["V"], first["clock"]
    ref = cyfa.forward(b["q"], b["k"], b["v"], b["delta"], b["log_alpha"], b["beta"], b["R"],
                       scale=x["scale"], K0=K.clone(), V0=V.clone(), clock0=clk.clone(),
                       return_state=True, kernel=cyfa.KERNEL_MFMA, segments=segments)
    got = cyfa.forward(b["q"], b["k"], b["v"], b["delta"], b["log_alpha"], b["beta"], b["R"],
                       scale=x["scale"], K0=K, V0=V, clock0=clk, K_out=K, V_out=V, clock_out=clk,
                       kernel=cyfa.KERNEL_MFMA, segments=segments)
    torch.cuda.synchronize()
    assert torch.equal(got["o"], ref["o"])
    assert torch.equal(K, ref["K"]) and torch.equal(V, ref["V"])
    assert torch.equal(clk, ref["clock"])


def test_empty_sequence():
    cyfa = _cyfa()
    x = make_forward_inputs(1, 0, 2, D, D, seed=81, dtype="bf16")
    t = upload(x)
    K0 = torch.randn(1, 2, 128, D, device="cuda")
    K0[:, :, 127:] = 0
    c0 = torch.tensor([[5.25, 130.5]], dtype=torch.float64, device="cuda")
    res = cyfa.forward(t["q"], t["k"], t["v"], t["delta"], t["log_alpha"], t["beta"], t["R"],
                       K0=K0, clock0=c0, return_state=True, kernel=cyfa.KERNEL_MFMA)
    torch.cuda.synchronize()
    assert torch.allclose(res["K"], K0, atol=1e-5)
    assert torch.count_nonzero(res["V"]) == 0
    np.testing.assert_allclose(res["clock"].cpu().numpy(), [[5.25, 3.5]], atol=1e-9)


@pytest.mark.parametrize("segments", [1, 3])
@pytest.mark.parametrize("with_init", [False, True])
def test_ragged_lengths_and_packed(with_init, segments):
    """Per-sequence lengths (empty, one token, partial and whole chunks) through
    cyfa_forward_lens, each sequence against the oracle on its own tokens, and the
    same sequences packed (cyfa_forward_varlen), bit-identical."""
    cyfa = _cyfa()
    lens_l = [37, 0, 200, 129, 1, 64]
    B, T, H, m = len(lens_l), max(lens_l), 2, 127
    x = make_forward_inputs(B, T, H, D, D, seed=82, dtype="bf16")
    t = upload(x)
    lens = torch.tensor(lens_l, dtype=torch.int32, device="cuda")
    init = _init_states(B, H, m, 83) if with_init else (None, None, None)
    pad = _fwd(x, t, lens=lens, K0=init[0], V0=init[1], clock0=init[2], return_state=True,
               return_logits=True, segments=segments)
    tp = {k: (torch.cat([a[b, :n] for b, n in enumerate(lens_l)], 0).contiguous()
              if a is not None and k != "R" else a) for k, a in t.items()}
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens_l)]), dtype=torch.int32, device="cuda")
    pk = cyfa.forward_varlen(tp["q"], tp["k"], tp["v"], tp["delta"], cu, tp["log_alpha"], tp["beta"],
                             t["R"], max_len=T, scale=x["scale"], kernel=cyfa.KERNEL_MFMA, K0=init[0],
                             V0=init[1], clock0=init[2], return_state=True, return_logits=True,
                             segments=segments)
    torch.cuda.synchronize()
    assert torch.equal(pk["o"], torch.cat([pad["o"][b, :n] for b, n in enumerate(lens_l)], 0))
    assert torch.equal(pk["logits"], torch.cat([pad["logits"][b, :n] for b, n in enumerate(lens_l)], 0))
    assert torch.equal(pk["K"], pad["K"]) and torch.equal(pk["V"], pad["V"])
    assert torch.equal(pk["clock"], pad["clock"])
    worst = {}
    o_all = pad["o"].float().cpu().numpy()
    z_all = pad["logits"].cpu().numpy()
    for b, n in enumerate(lens_l):
        xs = {k: (a[b:b + 1, :max(n, 1)] if k not in ("R", "scale", "m", "dtype") and a is not None else a)
              for k, a in x.items()}
        kw = {}
        if with_init:
            kw = _oracle_init(m, init[0][b:b + 1], init[1][b:b + 1], init[2][b:b + 1])
        ref = oracle.forward(xs["q"], xs["k"], xs["v"], xs["delta"], xs["log_alpha"], xs["beta"], x["R"],
                             m=m, scale=x["scale"], T_run=n, **kw)
        if n > 0:
            print("sequence", b, "tokens", n, "o error", f"{rel_err(o_all[b, :n].transpose(1, 0, 2), ref['o']):.2e}")
            worst["o"] = max(worst.get("o", 0), rel_err(o_all[b, :n].transpose(1, 0, 2), ref["o"]))
            worst["z"] = max(worst.get("z", 0), rel_err(z_all[b, :n].transpose(1, 0, 2), ref["z"]))
        Kref, Vref = oracle_states_abs(ref, m)
        if np.abs(Kref).max() > 0:
            worst["K"] = max(worst.get("K", 0), rel_err(pad["K"][b].cpu().numpy(), Kref))
            worst["V"] = max(worst.get("V", 0), rel_err(pad["V"][b].cpu().numpy(), Vref))
        else:
            assert torch.count_nonzero(pad["K"][b]) == 0 and torch.count_nonzero(pad["V"][b]) == 0
        worst["clock"] = max(worst.get("clock", 0), clock_err(pad["clock"][b].cpu().numpy(), ref["lam"], m))
    print("errors", {k: f"{v:.2e}" for k, v in worst.items()}, flush=True)
    _assert_ok(worst)


def test_matches_vector_alu_kernel():
    cyfa = _cyfa()
    x = make_forward_inputs(1, 256, 2, D, D, seed=84, dtype="bf16")
    t = upload(x)
    a = _fwd(x, t, return_logits=True, return_state=True)
    b = _fwd(x, t, return_logits=True, return_state=True, kernel=cyfa.KERNEL_VALU)
    torch.cuda.synchronize()
    assert rel_err(a["o"].float().cpu().numpy(), b["o"].float().cpu().numpy()) <= TOL_BF16
    assert rel_err(a["logits"].cpu().numpy(), b["logits"].cpu().numpy()) <= TOL_BF16
    assert rel_err(a["K"].cpu().numpy(), b["K"].cpu().numpy()) <= TOL_BF16
    assert torch.equal(a["clock"], b["clock"])


def test_deterministic():
    x = make_forward_inputs(2, 257, 2, D, D, seed=85, dtype="bf16")
    t = upload(x)
    a = _fwd(x, t, return_state=True)
    b = _fwd(x, t, return_state=True)
    torch.cuda.synchronize()
    assert torch.equal(a["o"], b["o"]) and torch.equal(a["K"], b["K"])


def test_peaky_logits_diagnostic():
    """Large logit scale: a far-from-uniform softmax makes key-pass errors (both
    channel halves of the inter-chunk product) visible in the output."""
    x = make_forward_inputs(1, 192, 2, D, D, seed=86, dtype="bf16")
    x["scale"] = 30.0
    res = _fwd(x, upload(x), return_logits=True)
    _assert_ok(_errors(x, res))


def test_paper_op_shape_sampled():
    """B 32, T 2048, H 4, d 256 in the benchmark's configuration (automatic kernel
    choice and segment count); six sampled (b, h) sequences against the oracle over
    all tokens."""
    cyfa = _cyfa()
    x = workload_inputs(FWD_PAPER_OP)
    t = upload(x)
    B, T, H = x["delta"].shape
    assert cyfa.selected_kernel(cyfa.forward_desc(B, T, H, D, D, dtype=cyfa.BF16)) == "mfma"
    res = _fwd(x, t, kernel=cyfa.KERNEL_AUTO, return_state=True, return_logits=True)
    torch.cuda.synchronize()
    assert torch.isfinite(res["o"].float()).all()
    pairs = [0, 5, 42, 77, 100, B * H - 1]
    _assert_ok(_errors(x, res, pairs=pairs))
