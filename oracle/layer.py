"""Float64 oracle of the transformer layer that wraps the attention (the
per-layer unit the profiling of Sec. 3.5 times and Eqs. (4)-(6) count).

TEST INFRASTRUCTURE ONLY.  Imported by ``tests/``; the product layer is the
C ABI of libdcp (``dcp_layer_fwd`` / ``dcp_layer_bwd``, rocBLAS GEMMs and
HIP kernels) and shares no code with this file.  The attention block calls
``oracle.attention``.

The layer (the paper fixes no block internals; a pre-norm block is read):
    y1 = rms(x) * g1,   q, k, v = y1 Wq, y1 Wk, y1 Wv   (heads of width D)
    o  = softmax attention per sequence of q, k, v
    h  = x + o Wo,      y2 = rms(h) * g2,   u = y2 Wup,   a = gelu(u)
    out = h + a Wdown
with rms(z) = z / sqrt(mean(z^2) + eps) per row and the tanh form of GELU,
gelu(u) = u/2 (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3))).  The backward is
the chain rule of these steps, written out; it is pinned by finite
differences in the tests.
"""

from __future__ import annotations

import math

import numpy as np

from oracle import attention as A

PARAMS = ("norm1", "wq", "wk", "wv", "wo", "norm2", "w_up", "w_down")
_K0 = math.sqrt(2.0 / math.pi)
_K1 = 0.044715


def rmsnorm(z, g, eps):
    r = 1.0 / np.sqrt(np.mean(z * z, axis=-1, keepdims=True) + eps)
    return z * r * g, r


def rmsnorm_backward(dy, z, g, r):
    """d/dz and d/dg of y = z r g, r = (mean(z^2) + eps)^(-1/2)."""
    zh = z * r
    gdy = g * dy
    dz = r * (gdy - zh * np.mean(gdy * zh, axis=-1, keepdims=True))
    return dz, np.sum(dy * zh, axis=0)


def gelu(u):
    return 0.5 * u * (1.0 + np.tanh(_K0 * (u + _K1 * u ** 3)))


def gelu_grad(u):
    t = np.tanh(_K0 * (u + _K1 * u ** 3))
    return 0.5 * (1.0 + t) + 0.5 * u * (1.0 - t * t) * _K0 * (1.0 + 3.0 * _K1 * u * u)


def layer_forward(x, W, cu, H, D, scale, causal, eps):
    """Returns (out, cache) for the backward.  x [T, H*D], W by PARAMS."""
    T = x.shape[0]
    y1, r1 = rmsnorm(x, W["norm1"], eps)
    q, k, v = (y1 @ W[n] for n in ("wq", "wk", "wv"))
    o, lse = A.attention_forward(q.reshape(T, H, D), k.reshape(T, H, D), v.reshape(T, H, D), cu, scale, causal)
    o = o.reshape(T, H * D)
    h = x + o @ W["wo"]
    y2, r2 = rmsnorm(h, W["norm2"], eps)
    u = y2 @ W["w_up"]
    a = gelu(u)
    out = h + a @ W["w_down"]
    cache = dict(x=x, y1=y1, r1=r1, q=q, k=k, v=v, o=o, lse=lse, h=h, y2=y2, r2=r2, u=u, a=a)
    return out, cache


def layer_backward(dout, W, cache, cu, H, D, scale, causal):
    """Returns (dx, grads by PARAMS) of <dout, out>."""
    c = cache
    T = dout.shape[0]
    g = {}
    da = dout @ W["w_down"].T
    g["w_down"] = c["a"].T @ dout
    du = da * gelu_grad(c["u"])
    dy2 = du @ W["w_up"].T
    g["w_up"] = c["y2"].T @ du
    dh2, g["norm2"] = rmsnorm_backward(dy2, c["h"], W["norm2"], c["r2"])
    dh = dout + dh2
    do = dh @ W["wo"].T
    g["wo"] = c["o"].T @ dh
    dq, dk, dv = A.attention_backward(do.reshape(T, H, D), c["q"].reshape(T, H, D), c["k"].reshape(T, H, D),
                                      c["v"].reshape(T, H, D), cu, scale, causal)
    dq, dk, dv = (t.reshape(T, H * D) for t in (dq, dk, dv))
    dy1 = dq @ W["wq"].T + dk @ W["wk"].T + dv @ W["wv"].T
    g["wq"], g["wk"], g["wv"] = (c["y1"].T @ t for t in (dq, dk, dv))
    dx1, g["norm1"] = rmsnorm_backward(dy1, c["x"], W["norm1"], c["r1"])
    # x reaches the output through the residual (dh) and through norm1 (dx1)
    return dh + dx1, g
