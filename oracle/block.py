"""fp64 CPU oracle for the Gated DeltaNet block's prologue and epilogue.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU baseline leg of ``bench.py`` may import it; the product package never does
and shares no code with it.

The block design (Sec. 3.4 and the block-design figure and its caption)
generates the rule's inputs and post-processes its output:
  * q and k: linear projection -> short causal convolution -> SiLU -> L2
    normalisation per (token, head);  v: projection -> convolution -> SiLU;
  * the output: normalisation, then a gate (a projection through SiLU), then
    the output projection.
The projections are ordinary dense layers and are not part of this oracle.
Readings where the paper is silent (all arguments, nothing fixed here):
  * the convolution is depthwise over the time axis, causal, of width W, and
    restarts with zeros at every sequence start:
        u_t[c] = sum_{i < W} w[c, i] * x_{t - (W - 1) + i}[c];
  * L2 normalisation: y = z / sqrt(|z|^2 + eps);
  * the output normalisation is an RMS normalisation over the value channels
    of each (token, head) with a per-channel weight shared by the heads:
        y = o / sqrt(mean(o^2) + eps) * w * silu(g).
Every function works on float64 copies of its inputs and returns float64.
The vector-Jacobian products are derived by hand (chain rule on the
definitions above) and written out step by step.
"""
from __future__ import annotations

import numpy as np


def _f64(x):
    if x is None:
        return None
    if hasattr(x, "detach"):
        x = x.detach().to("cpu").double().numpy()
    return np.asarray(x, dtype=np.float64)


def _sequences(T_total, B, T, cu_seqlens):
    """(batch index, first token, length) of every sequence."""
    if cu_seqlens is None:
        return [(b, 0, T) for b in range(B)]
    cu = [int(c) for c in _f64(cu_seqlens)]
    return [(0, cu[n], cu[n + 1] - cu[n]) for n in range(len(cu) - 1)]


def sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def silu(x):
    return x * sigmoid(x)


def silu_grad(x):
    """d silu / dx = s + x s (1 - s), s = sigmoid(x)."""
    s = sigmoid(x)
    return s * (1.0 + x * (1.0 - s))


def _conv_one(x, w):
    """Causal depthwise convolution of one sequence x [L, H, d] with w [H*d, W]."""
    L, H, d = x.shape
    W = w.shape[1]
    wc = w.reshape(H, d, W)
    u = np.zeros_like(x)
    for t in range(L):
        for i in range(W):
            s = t - (W - 1) + i
            if s >= 0:
                u[t] += wc[:, :, i] * x[s]
    return u


def conv_silu(x, w, cu_seqlens=None, l2norm=True, eps=1e-6):
    """Prologue forward: x [B, T, H, d] -> y [B, T, H, d]."""
    x, w = _f64(x), _f64(w)
    B, T = x.shape[:2]
    y = np.zeros_like(x)
    for b, s0, L in _sequences(B * T, B, T, cu_seqlens):
        if L == 0:
            continue
        z = silu(_conv_one(x[b, s0:s0 + L], w))
        if l2norm:
            z = z / np.sqrt((z * z).sum(-1, keepdims=True) + eps)
        y[b, s0:s0 + L] = z
    return y


def conv_silu_vjp(x, w, dy, cu_seqlens=None, l2norm=True, eps=1e-6):
    """Gradients (dx, dw) of <dy, conv_silu(x, w)>."""
    x, w, dy = _f64(x), _f64(w), _f64(dy)
    B, T, H, d = x.shape
    W = w.shape[1]
    wc = w.reshape(H, d, W)
    dx = np.zeros_like(x)
    dwc = np.zeros((H, d, W))
    for b, s0, L in _sequences(B * T, B, T, cu_seqlens):
        if L == 0:
            continue
        xs = x[b, s0:s0 + L]
        u = _conv_one(xs, w)
        z = silu(u)
        g = dy[b, s0:s0 + L]
        if l2norm:
            n = np.sqrt((z * z).sum(-1, keepdims=True) + eps)
            y = z / n
            dz = (g - y * (y * g).sum(-1, keepdims=True)) / n
        else:
            dz = g
        du = dz * silu_grad(u)
        for t in range(L):
            for i in range(W):
                s = t - (W - 1) + i
                if s >= 0:
                    dx[b, s0 + s] += wc[:, :, i] * du[t]
                    dwc[:, :, i] += du[t] * xs[s]
    return dx, dwc.reshape(H * d, W)


def norm_gate(o, g, w, eps=1e-5):
    """Epilogue forward: o, g [B, T, H, dv], w [dv] -> y [B, T, H, dv]."""
    o, g, w = _f64(o), _f64(g), _f64(w)
    r = 1.0 / np.sqrt((o * o).mean(-1, keepdims=True) + eps)
    return o * r * w * silu(g)


def norm_gate_vjp(o, g, w, dy, eps=1e-5):
    """Gradients (do, dg, dw) of <dy, norm_gate(o, g, w)>."""
    o, g, w, dy = _f64(o), _f64(g), _f64(w), _f64(dy)
    dv = o.shape[-1]
    r = 1.0 / np.sqrt((o * o).mean(-1, keepdims=True) + eps)
    oh = o * r                      # normalised output
    a = oh * w                      # weighted
    sg = silu(g)
    dg = dy * a * silu_grad(g)
    da = dy * sg
    dw = (da * oh).reshape(-1, dv).sum(0)
    doh = da * w
    do = r * (doh - oh * (doh * oh).sum(-1, keepdims=True) / dv)
    return do, dg, dw
