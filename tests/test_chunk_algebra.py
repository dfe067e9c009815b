"""The chunk algebra the kernels implement, checked against the oracle.

``chunk_ref`` (test-only numpy) restates the gated chunk equations of
Sec. 3.3 in the stored dk x dv orientation, with the output mask read as the
decay mask Gamma, and its exact reverse-mode derivative.  Here it must agree
with the oracle's token recurrence and VJP at every chunk size, including
ragged last chunks; the literal mask M must not.
"""
import numpy as np
import pytest

from tests import chunk_ref
from tests.test_oracle_pins import rand_problem


@pytest.mark.parametrize("C", [1, 2, 3, 4, 8, 16, 64])
def test_chunk_forward_matches_recurrence(oracle_mod, C):
    rng = np.random.default_rng(100 + C)
    q, k, v, beta, la, S0 = rand_problem(rng, B=1, T=37, H=1, dk=6, dv=5)
    o, ht = oracle_mod.fwd(q, k, v, beta, la, h0=S0)
    oc, Sc = chunk_ref.chunk_fwd(q[0, :, 0], k[0, :, 0], v[0, :, 0], beta[0, :, 0],
                                 la[0, :, 0], S0[0, 0], C=C)
    np.testing.assert_allclose(oc, o[0, :, 0], atol=1e-12, rtol=0)
    np.testing.assert_allclose(Sc, ht[0, 0], atol=1e-12, rtol=0)


def test_literal_causal_mask_disagrees(oracle_mod):
    rng = np.random.default_rng(7)
    q, k, v, beta, la, S0 = rand_problem(rng, B=1, T=32, H=1, dk=6, dv=5, decay=4.0)
    o, _ = oracle_mod.fwd(q, k, v, beta, la, h0=S0)
    om, _ = chunk_ref.chunk_fwd(q[0, :, 0], k[0, :, 0], v[0, :, 0], beta[0, :, 0],
                                la[0, :, 0], S0[0, 0], C=16, output_mask="M")
    assert np.abs(om - o[0, :, 0]).max() > 1e-2


@pytest.mark.parametrize("C", [1, 3, 4, 8, 64])
@pytest.mark.parametrize("beta_scale", [1.0, 2.0])
def test_chunk_backward_matches_vjp(oracle_mod, C, beta_scale):
    rng = np.random.default_rng(200 + C)
    q, k, v, beta, la, S0 = rand_problem(rng, B=1, T=29, H=1, dk=5, dv=4,
                                         beta_scale=beta_scale)
    dO = rng.standard_normal(v.shape)
    dSf = rng.standard_normal(S0.shape)
    r = oracle_mod.bwd(q, k, v, beta, la, dO, h0=S0, dht=dSf)
    c = chunk_ref.chunk_bwd(q[0, :, 0], k[0, :, 0], v[0, :, 0], beta[0, :, 0], la[0, :, 0],
                            dO[0, :, 0], S0[0, 0], dSf[0, 0], C=C)
    for name in ("dq", "dk", "dv", "dbeta", "dlog_alpha"):
        np.testing.assert_allclose(c[name], r[name][0, :, 0], atol=1e-11, rtol=0, err_msg=name)
    np.testing.assert_allclose(c["dh0"], r["dh0"][0, 0], atol=1e-11, rtol=0)


def test_chunk_backward_special_values(oracle_mod):
    """beta == 0 (no writes) and alpha == 1 (DeltaNet) through the chunk backward."""
    rng = np.random.default_rng(300)
    for beta_val, la_val in ((0.0, None), (None, 0.0)):
        q, k, v, beta, la, S0 = rand_problem(rng, B=1, T=21, H=1, dk=4, dv=3)
        if beta_val is not None:
            beta[:] = beta_val
        if la_val is not None:
            la[:] = la_val
        dO = rng.standard_normal(v.shape)
        r = oracle_mod.bwd(q, k, v, beta, la, dO, h0=S0)
        c = chunk_ref.chunk_bwd(q[0, :, 0], k[0, :, 0], v[0, :, 0], beta[0, :, 0],
                                la[0, :, 0], dO[0, :, 0], S0[0, 0], None, C=8)
        for name in ("dq", "dk", "dv", "dbeta", "dlog_alpha"):
            np.testing.assert_allclose(c[name], r[name][0, :, 0], atol=1e-11, err_msg=name)
