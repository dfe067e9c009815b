"""Pins of the block prologue / epilogue oracle (oracle/block.py), CPU only.

Sec. 3.4 and the block-design figure fix what is computed (short causal
convolution, SiLU, L2 normalisation of q and k; output normalisation and
SiLU gate); the paper prints no numbers for them.  Each function is pinned by
facts that do not reuse its own code: finite differences of the forward for
every gradient, a banded-matrix (Toeplitz) form of the convolution, shift
and identity kernels, the SiLU identity silu(x) - silu(-x) = x, unit norms,
scale invariance of the RMS normalisation, and packed-equals-separate.
"""
import numpy as np
import pytest

from oracle import block

RNG = np.random.default_rng(1234)


def fd_grad(f, x, eps=1e-6):
    """Central finite differences of the scalar f at x (float64 array)."""
    g = np.zeros_like(x)
    it = np.nditer(x, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        old = x[i]
        x[i] = old + eps
        fp = f(x)
        x[i] = old - eps
        fm = f(x)
        x[i] = old
        g[i] = (fp - fm) / (2 * eps)
    return g


def packed_case(W=3, d=3, H=2):
    lens = [3, 0, 5, 1]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    T = int(cu[-1])
    x = RNG.standard_normal((1, T, H, d))
    w = RNG.standard_normal((H * d, W))
    return x, w, cu


@pytest.mark.parametrize("l2norm", [True, False])
@pytest.mark.parametrize("W", [1, 2, 4])
def test_conv_silu_vjp_matches_finite_differences(l2norm, W):
    x, w, cu = packed_case(W=W)
    dy = RNG.standard_normal(x.shape)
    dx, dw = block.conv_silu_vjp(x, w, dy, cu_seqlens=cu, l2norm=l2norm, eps=1e-3)
    f = lambda xx: float((block.conv_silu(xx, w, cu, l2norm, 1e-3) * dy).sum())
    fw = lambda ww: float((block.conv_silu(x, ww, cu, l2norm, 1e-3) * dy).sum())
    np.testing.assert_allclose(dx, fd_grad(f, x.copy()), rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(dw, fd_grad(fw, w.copy()), rtol=1e-6, atol=1e-8)


def test_conv_matches_banded_matrix_form():
    """u = sum_i diag(w_i) Shift^(W-1-i) x for one sequence, as a dense matmul."""
    L, H, d, W = 7, 1, 2, 4
    x = RNG.standard_normal((1, L, H, d))
    w = RNG.standard_normal((H * d, W))
    y = block.conv_silu(x, w, l2norm=False)
    u_ref = np.zeros((L, d))
    for c in range(d):
        M = np.zeros((L, L))  # lower-triangular band: tap i sits W-1-i below the diagonal
        for i in range(W):
            M += w[c, i] * np.eye(L, k=-(W - 1 - i))
        u_ref[:, c] = M @ x[0, :, 0, c]
    s = u_ref / (1.0 + np.exp(-u_ref))  # SiLU of the banded-matrix convolution
    np.testing.assert_allclose(y[0, :, 0, :], s, rtol=1e-12, atol=1e-14)


def test_shift_and_identity_kernels_restart_per_sequence():
    x, _, cu = packed_case(W=4, d=2, H=1)
    H, d, W = 1, 2, 4
    ident = np.zeros((H * d, W))
    ident[:, W - 1] = 1.0
    shift = np.zeros((H * d, W))
    shift[:, 0] = 1.0
    yi = block.conv_silu(x, ident, cu, l2norm=False)
    ys = block.conv_silu(x, shift, cu, l2norm=False)
    for n in range(len(cu) - 1):
        s0, s1 = int(cu[n]), int(cu[n + 1])
        seg = x[0, s0:s1]
        # identity kernel: u = x, and silu(x) - silu(-x) = x exactly
        yneg = block.conv_silu(-x, ident, cu, l2norm=False)
        np.testing.assert_allclose(yi[0, s0:s1] - yneg[0, s0:s1], seg, rtol=0, atol=1e-14)
        # shift kernel: u_t = x_{t-3} inside the sequence, zero before its start
        for t in range(s1 - s0):
            if t < W - 1:
                assert np.all(ys[0, s0 + t] == 0.0)
            else:
                np.testing.assert_array_equal(ys[0, s0 + t], yi[0, s0 + t - (W - 1)])


def test_l2_rows_have_unit_norm_and_packed_equals_separate():
    x, w, cu = packed_case(W=4, d=5, H=3)
    y = block.conv_silu(x, w, cu, l2norm=True, eps=0.0)
    nz = np.abs(y).sum(-1) > 0
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1)[nz], 1.0, rtol=1e-13)
    for n in range(len(cu) - 1):
        s0, s1 = int(cu[n]), int(cu[n + 1])
        if s1 > s0:
            alone = block.conv_silu(x[:, s0:s1], w, None, l2norm=True, eps=0.0)
            np.testing.assert_array_equal(alone[0], y[0, s0:s1])


def test_norm_gate_vjp_matches_finite_differences():
    o = RNG.standard_normal((2, 3, 2, 6))
    g = RNG.standard_normal(o.shape)
    w = RNG.standard_normal(6)
    dy = RNG.standard_normal(o.shape)
    do, dg, dw = block.norm_gate_vjp(o, g, w, dy, eps=1e-3)
    fo = lambda oo: float((block.norm_gate(oo, g, w, 1e-3) * dy).sum())
    fg = lambda gg: float((block.norm_gate(o, gg, w, 1e-3) * dy).sum())
    fw = lambda ww: float((block.norm_gate(o, g, ww, 1e-3) * dy).sum())
    np.testing.assert_allclose(do, fd_grad(fo, o.copy()), rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(dg, fd_grad(fg, g.copy()), rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(dw, fd_grad(fw, w.copy()), rtol=1e-6, atol=1e-8)


def test_norm_gate_scale_invariance_and_unit_rms():
    o = RNG.standard_normal((1, 4, 3, 8))
    g = np.full(o.shape, 40.0)  # silu(40) = 40 (1 - 4e-18)
    w = np.ones(8)
    y = block.norm_gate(o, g, w, eps=0.0)
    np.testing.assert_allclose(block.norm_gate(7.5 * o, g, w, eps=0.0), y, rtol=1e-13)
    # with w = 1 and silu(g) = 40, y / 40 has unit RMS over the channels
    np.testing.assert_allclose(np.sqrt(((y / 40.0) ** 2).mean(-1)), 1.0, rtol=1e-12)
    # a zero gate closes the output
    assert np.all(block.norm_gate(o, np.zeros_like(o), w) == 0.0)
