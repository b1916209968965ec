"""Pins of the mixer oracle (CPU only): each definition against a library routine
or a property it must have."""
import numpy as np
import pytest

from oracle import mixer

torch = pytest.importorskip("torch")


def _rng(seed):
    return np.random.default_rng(seed)


def test_short_conv_is_numpy_convolution_per_channel():
    rng = _rng(1)
    x = rng.standard_normal((2, 11, 3, 5))
    w = rng.standard_normal((15, 4))
    y = mixer.short_conv(x, w)
    for b in range(2):
        for h in range(3):
            for d in range(5):
                c = h * 5 + d
                ref = np.convolve(x[b, :, h, d], w[c][::-1])[:11]
                np.testing.assert_allclose(y[b, :, h, d], ref, rtol=0, atol=1e-12)


def test_short_conv_identity_tap_causality_and_silu():
    rng = _rng(2)
    x = rng.standard_normal((1, 9, 2, 4))
    w = np.zeros((8, 4))
    w[:, 3] = 1.0                                    # the current token only
    np.testing.assert_allclose(mixer.short_conv(x, w), x, atol=0)
    w = rng.standard_normal((8, 4))
    y0 = mixer.short_conv(x, w)
    x2 = x.copy()
    x2[0, 5] += 1.0
    y1 = mixer.short_conv(x2, w)
    np.testing.assert_array_equal(y0[0, :5], y1[0, :5])          # nothing before t = 5 moves
    assert np.all(np.abs(y0[0, 5:] - y1[0, 5:]).max(axis=(1, 2)) > 0)   # t = 5 .. 8 see it
    x3 = x.copy()
    x3[0, 1] += 1.0
    np.testing.assert_array_equal(mixer.short_conv(x3, w)[0, 5:], y0[0, 5:])  # 4 taps: t = 1 is out of reach
    ys = mixer.short_conv(x, w, act="silu")
    np.testing.assert_allclose(ys, torch.nn.functional.silu(torch.tensor(y0)).numpy(), atol=1e-12)


def test_rms_norm_matches_torch():
    rng = _rng(3)
    x = rng.standard_normal((2, 7, 3, 16))
    g = rng.standard_normal(16)
    ref = torch.nn.functional.rms_norm(torch.tensor(x), (16,), torch.tensor(g), eps=1e-6).numpy()
    np.testing.assert_allclose(mixer.rms_norm(x, g, 1e-6), ref, rtol=1e-12, atol=1e-12)


def test_gates_match_library_forms():
    rng = _rng(4)
    z = 6 * rng.standard_normal((2, 5, 3))
    b = rng.standard_normal(3)
    A = np.exp(rng.standard_normal(3))
    out = mixer.prologue(rng.standard_normal((2, 5, 3, 4)), rng.standard_normal((2, 5, 3, 4)),
                         rng.standard_normal((2, 5, 3, 4)), z_delta=z, b_delta=b, z_alpha=z,
                         b_alpha=b, A=A, z_beta=z)
    np.testing.assert_allclose(out["delta"], torch.sigmoid(torch.tensor(z + b)).numpy(), atol=1e-14)
    np.testing.assert_allclose(out["log_alpha"], -A * np.logaddexp(0.0, z + b), rtol=1e-12)
    np.testing.assert_allclose(out["beta"], torch.sigmoid(torch.tensor(z)).numpy(), atol=1e-14)
    assert np.all(out["log_alpha"] <= 0)


def test_epilogue_and_ragged_padding():
    rng = _rng(5)
    o = rng.standard_normal((2, 6, 2, 8))
    g = rng.standard_normal((2, 6, 2, 8))
    go = rng.standard_normal(8)
    y = mixer.epilogue(o, g, go, eps=1e-6, lens=[6, 2])
    ref = torch.nn.functional.rms_norm(torch.tensor(o), (8,), torch.tensor(go), eps=1e-6) * \
        torch.sigmoid(torch.tensor(g))
    np.testing.assert_allclose(y[0], ref.numpy()[0], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(y[1, :2], ref.numpy()[1, :2], rtol=1e-12, atol=1e-12)
    assert np.all(y[1, 2:] == 0)
