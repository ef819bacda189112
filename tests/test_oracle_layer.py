"""Pins of the float64 layer oracle (no GPU): central finite differences of
<dout, out> on every input and parameter element, closed forms, packing
invariance, and GELU / RMSNorm against torch's CPU library routines."""

import math

import numpy as np
import pytest

from oracle import layer as LY


def _params(rng, h, scale=0.5):
    W = {"norm1": 1.0 + 0.2 * rng.standard_normal(h), "norm2": 1.0 + 0.2 * rng.standard_normal(h)}
    for n, shape in (("wq", (h, h)), ("wk", (h, h)), ("wv", (h, h)), ("wo", (h, h)), ("w_up", (h, 4 * h)),
                     ("w_down", (4 * h, h))):
        W[n] = scale * rng.standard_normal(shape) / math.sqrt(shape[0])
    return W


@pytest.mark.parametrize("causal", [False, True])
def test_finite_differences(causal):
    rng = np.random.default_rng(11 + causal)
    H, D = 2, 3
    h = H * D
    cu = np.array([0, 3, 7])
    T = 7
    x = rng.standard_normal((T, h))
    dout = rng.standard_normal((T, h))
    W = _params(rng, h)
    scale, eps = 0.7, 1e-5
    out, cache = LY.layer_forward(x, W, cu, H, D, scale, causal, eps)
    dx, g = LY.layer_backward(dout, W, cache, cu, H, D, scale, causal)

    def loss(xx, WW):
        return float(np.sum(dout * LY.layer_forward(xx, WW, cu, H, D, scale, causal, eps)[0]))

    step = 1e-6
    worst = 0.0
    for name in ("x",) + LY.PARAMS:
        arr = x if name == "x" else W[name]
        ana = dx if name == "x" else g[name]
        for idx in np.ndindex(arr.shape):
            keep = arr[idx]
            arr[idx] = keep + step
            lp = loss(x, W)
            arr[idx] = keep - step
            lm = loss(x, W)
            arr[idx] = keep
            num = (lp - lm) / (2 * step)
            worst = max(worst, abs(num - ana[idx]) / max(1.0, abs(num)))
    assert worst < 1e-6, worst


def test_zero_projections_are_the_identity():
    """With Wo = Wdown = 0 both residual branches vanish: out = x, dx = dout,
    and no gradient reaches the weights before those projections."""
    rng = np.random.default_rng(3)
    H, D = 2, 4
    h = H * D
    cu = np.array([0, 5, 9])
    x = rng.standard_normal((9, h))
    dout = rng.standard_normal((9, h))
    W = _params(rng, h)
    W["wo"][:] = 0
    W["w_down"][:] = 0
    out, cache = LY.layer_forward(x, W, cu, H, D, 0.5, False, 1e-6)
    dx, g = LY.layer_backward(dout, W, cache, cu, H, D, 0.5, False)
    assert np.array_equal(out, x) and np.array_equal(dx, dout)
    for n in ("norm1", "wq", "wk", "wv", "norm2", "w_up"):
        assert not np.any(g[n]), n


def test_packing_is_per_sequence():
    """Every step but attention is row-wise and attention stays inside a
    sequence: the packed layer equals the layer on each sequence alone."""
    rng = np.random.default_rng(4)
    H, D = 3, 2
    h = H * D
    lens = [4, 1, 6]
    cu = np.cumsum([0] + lens)
    x = rng.standard_normal((cu[-1], h))
    dout = rng.standard_normal((cu[-1], h))
    W = _params(rng, h)
    out, cache = LY.layer_forward(x, W, cu, H, D, 0.4, True, 1e-6)
    dx, g = LY.layer_backward(dout, W, cache, cu, H, D, 0.4, True)
    gsum = {n: 0 for n in LY.PARAMS}
    for b in range(len(lens)):
        sl = slice(cu[b], cu[b + 1])
        o1, c1 = LY.layer_forward(x[sl], W, np.array([0, lens[b]]), H, D, 0.4, True, 1e-6)
        d1, g1 = LY.layer_backward(dout[sl], W, c1, np.array([0, lens[b]]), H, D, 0.4, True)
        assert np.allclose(o1, out[sl], rtol=0, atol=1e-12) and np.allclose(d1, dx[sl], rtol=0, atol=1e-12)
        for n in LY.PARAMS:
            gsum[n] = gsum[n] + g1[n]
    for n in LY.PARAMS:
        assert np.allclose(gsum[n], g[n], rtol=0, atol=1e-11), n


def test_gelu_and_rmsnorm_against_torch():
    torch = pytest.importorskip("torch")
    u = np.linspace(-6, 6, 241)
    ref = torch.nn.functional.gelu(torch.from_numpy(u), approximate="tanh").numpy()
    assert np.max(np.abs(LY.gelu(u) - ref)) < 1e-14
    uu = torch.from_numpy(u).requires_grad_(True)
    torch.nn.functional.gelu(uu, approximate="tanh").sum().backward()
    assert np.max(np.abs(LY.gelu_grad(u) - uu.grad.numpy())) < 1e-13
    rng = np.random.default_rng(5)
    z = rng.standard_normal((6, 16))
    gain = rng.standard_normal(16)
    y, _ = LY.rmsnorm(z, gain, 1e-5)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(z), (16,), torch.from_numpy(gain), eps=1e-5).numpy()
    assert np.max(np.abs(y - ref)) < 1e-13
