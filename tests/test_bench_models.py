"""The benchmark's algorithmic work model (CPU only).

bench.py credits each launch with the algorithmic FLOP of the method's steps
it performs (Sec. 3.3 chunk equations and their reverse-mode derivatives,
full 64 x 64 intra-chunk products counted) and with the bytes of the call's
own tensors.  Pinned here against per-workload totals worked out by hand
from the same per-token-head formulas:

    forward  FLOP 6 dk dv + 6 C dk + 4 C dv + C^2/3,
    backward FLOP 12 dk dv + 12 C dk + 8 C dv + 4 C^2,
    forward  bytes (2 dk + 2 dv) e + 8,  backward (4 dk + 3 dv) e + 16,
    plus dk dv fp32 per (sequence, head) for each state read or written,

and for consistency: the launches of one saved training step add up to the
path's totals, and the dominant kernel's figures in a bench line can be
recomputed from them."""
import importlib.util
import os
from types import SimpleNamespace

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_models", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def wl(dk, dv, dtype, backward, H):
    return SimpleNamespace(dk=dk, dv=dv, dtype=dtype, backward=backward, H=H)


# (workload, tokens, heads, states, has_h0, GFLOP, GB) by hand:
#  cfg 1: 131,072 token-heads x 181,589 FLOP = 23.80 GFLOP; x 1,032 B = 135.3 MB,
#         + 4 x 16 states of 64 KiB read (h0) and written (ht) = 8.4 MB
#  cfg 2: 196,608 x 1,017,173 = 199.98 GFLOP; x 3,080 B = 605.6 MB + 48 ht of 512 KiB
#  cfg 3: + backward 196,608 x 2,048,000 = 402.7 GFLOP, x 4,624 B = 909.1 MB,
#         + 48 x 2 states (dht in, dh0 out)
#  cfg 0: 512 x 66,901 = 34.25 MFLOP; x 1,032 B (fp32) = 528 KB + 2 ht of 16 KiB
CASES = [
    ("cfg1", 128, 128, "bf16", False, 16, 4 * 2048, 4, True, 23.801, 0.1437),
    ("cfg2", 256, 512, "bf16", False, 6, 8 * 4096, 8, False, 199.98, 0.6308),
    ("cfg3", 256, 512, "bf16", True, 6, 8 * 4096, 8, False, 602.64, 1.6908),
    ("cfg0", 64, 64, "f32", False, 2, 256, 1, False, 0.034253, 0.000561),
]


@pytest.mark.parametrize("name,dk,dv,dtype,bwd,H,tokens,nseq,h0,gflop,gbytes", CASES)
def test_path_totals_match_hand_counts(bench, name, dk, dv, dtype, bwd, H, tokens, nseq, h0,
                                       gflop, gbytes):
    w = wl(dk, dv, dtype, bwd, H)
    th = tokens * H
    assert bench.path_flops(w, th) / 1e9 == pytest.approx(gflop, rel=2e-4), name
    assert bench.path_bytes(w, th, nseq, h0) / 1e9 == pytest.approx(gbytes, rel=2e-3), name


def test_state_bytes_count_every_head(bench):
    """One more head adds its token-heads' bytes and its own fp32 states."""
    w1, w2 = wl(256, 512, "bf16", True, 1), wl(256, 512, "bf16", True, 2)
    d = bench.path_bytes(w2, 2000, 3, False) - bench.path_bytes(w1, 1000, 3, False)
    per_th = (2 * 256 + 2 * 512) * 2 + 8 + (4 * 256 + 3 * 512) * 2 + 16
    assert d == 1000 * per_th + 3 * 256 * 512 * 4 * 3  # ht, dht, dh0 of the new head


@pytest.mark.parametrize("dk,dv,dtype", [(64, 64, "f32"), (128, 128, "bf16"), (256, 512, "bf16")])
def test_saved_step_launches_add_up_to_the_path(bench, dk, dv, dtype):
    """prep + saving forward + reverse pass + gradient kernel = forward +
    backward FLOP.  Their bytes = the path's (each call's tensors once) plus
    dO once more: both backward launches need it (the reverse pass for dV'
    and dS, the gradient kernel for dP and Gq)."""
    w = wl(dk, dv, dtype, True, 3)
    th, nseq = 5000, 4
    e = 4 if dtype == "f32" else 2
    for h0 in (False, True):
        m = bench.kernel_models(w, th, nseq * w.H, h0)
        names = ("k_prep_save", "k_fwd_seq_save", "k_bwd_seq", "k_grad")
        assert sum(m[k][1] for k in names) == pytest.approx(bench.path_flops(w, th), rel=1e-12)
        got = sum(m[k][0] for k in names)
        assert got == bench.path_bytes(w, th, nseq, h0, saved=True) + th * dv * e, (h0, got)
        # the stateless backward reads h0 once more
        assert (bench.path_bytes(w, th, nseq, h0, saved=False)
                - bench.path_bytes(w, th, nseq, h0, saved=True)) == (
                    nseq * w.H * dk * dv * 4 if h0 else 0)


def test_dominant_kernel_figures_of_the_training_step(bench):
    """The reverse pass at the training workload: 6 dk dv + 4 C dv FLOP per
    token-head (dS and dV' products) = 180.4 GFLOP, and the bytes of dO and
    beta in, dv out, dht in and dh0 out = 0.4538 GB, as a bench line reports."""
    w = wl(256, 512, "bf16", True, 6)
    th = 8 * 4096 * 6
    b, f = bench.kernel_models(w, th, 8 * 6, False)["k_bwd_seq"]
    assert f / 1e9 == pytest.approx(180.39, rel=1e-4)
    assert b / 1e9 == pytest.approx(0.45377, rel=1e-4)


def test_decode_model(bench):
    """One token per sequence: the fp32 state read and written once per
    (sequence, head) dominates: 256 x 6 x 2 x 512 KiB = 1.61 GB."""
    w = SimpleNamespace(dk=256, dv=512, dtype="bf16", B=256, T=1, H=6)
    b, f = bench.recurrent_model(w, 256 * 6)["k_recurrent"]
    assert b == 256 * 6 * (2 * 256 * 512 * 4 + (2 * 256 + 2 * 512) * 2 + 8)
    assert f == 6 * 256 * 512 * 256 * 6
