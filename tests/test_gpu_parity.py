"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Error metric (per output tensor, computed in fp64):
    err(x, ref) = max_i |x_i - ref_i| / max_i |ref_i|
Bar: <= 1e-4 for float32 inputs, <= 2e-2 for bfloat16 inputs with fp32
accumulation.  The denominator has a floor of 1e-30: a reference tensor whose
magnitude lies below what fp32 represents (a state decayed by e^-170, say)
counts as zero, and then the result must be within 1e-30 * tol of it.  Both
sides see the same (already rounded) inputs, so input
quantisation is not counted as kernel error.
"""
import os

import numpy as np
import pytest
import torch

from paper_2412_06464_amd.inputs import WORKLOADS, make_inputs, workload_inputs

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}


def rel_err(x, ref):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = max(float(np.abs(ref).max()), 1e-30)
    return float(np.abs(x - ref).max() / den)


def f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def say(*a):
    print("[gpu-case]", *a, flush=True)


@pytest.fixture(scope="module")
def G():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2412_06464_amd import gdn
    gdn.load_library()
    return gdn


def to_dev(inp):
    return {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}


def gates(d):
    """log_alpha as the library takes it: None for ungated (alpha == 1) inputs."""
    return d["log_alpha"] if d.get("gated", True) else None


def run_fwd(G, d):
    o, ht = G.gdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], gates(d), h0=d.get("h0"),
                            cu_seqlens=d.get("cu_seqlens"))
    torch.cuda.synchronize()
    return o, ht


def run_bwd(G, d):
    r = G.gdn_chunk_bwd(d["q"], d["k"], d["v"], d["beta"], gates(d), d["dO"],
                        h0=d.get("h0"), dht=d.get("dht"), cu_seqlens=d.get("cu_seqlens"))
    torch.cuda.synchronize()
    return r


def check_fwd(G, oracle_mod, inp, tol, label):
    say(label, "fwd", tuple(inp["q"].shape), tuple(inp["v"].shape), inp["q"].dtype)
    d = to_dev(inp)
    o, ht = run_fwd(G, d)
    ro, rht = oracle_mod.fwd(inp["q"], inp["k"], inp["v"], inp["beta"], inp["log_alpha"],
                             h0=inp.get("h0"), cu_seqlens=inp.get("cu_seqlens"))
    eo = rel_err(f64(o).reshape(ro.shape), ro)
    eh = rel_err(f64(ht), rht)
    say(label, "err o=%.3g ht=%.3g" % (eo, eh))
    assert eo <= tol and eh <= tol, (eo, eh)
    return o, ht


def check_bwd(G, oracle_mod, inp, tol, label):
    say(label, "bwd", tuple(inp["q"].shape), tuple(inp["v"].shape), inp["q"].dtype)
    d = to_dev(inp)
    r = run_bwd(G, d)
    ref = oracle_mod.bwd(inp["q"], inp["k"], inp["v"], inp["beta"], inp["log_alpha"], inp["dO"],
                         h0=inp.get("h0"), dht=inp.get("dht"), cu_seqlens=inp.get("cu_seqlens"))
    errs = {}
    for name in ("dq", "dk", "dv", "dbeta", "dlog_alpha", "dh0"):
        errs[name] = rel_err(f64(r[name]).reshape(ref[name].shape), ref[name])
    say(label, "errs", {k: "%.3g" % v for k, v in errs.items()})
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, bad
    return r


# ------------------------------------------------------------------ forward, small


def test_fwd_f32_workload(G, oracle_mod):
    check_fwd(G, oracle_mod, workload_inputs("fwd_f32_b1_t256_h2_d64"), TOL["f32"],
              "fwd_f32_b1_t256_h2_d64")


@pytest.mark.parametrize("dtype,dk,dv,B,T,H", [
    ("f32", 64, 64, 2, 200, 3),
    ("f32", 128, 128, 2, 150, 2),
    ("f32", 256, 512, 1, 150, 2),
    ("bf16", 64, 64, 2, 200, 3),
    ("bf16", 128, 128, 2, 130, 2),
    ("bf16", 256, 512, 1, 150, 2),
])
def test_fwd_ragged_with_initial_state(G, oracle_mod, dtype, dk, dv, B, T, H):
    inp = make_inputs(B, T, H, dk, dv, dtype, seed=1, h0_std=0.05)
    check_fwd(G, oracle_mod, inp, TOL[dtype], "fwd_%s_%d_%d_T%d" % (dtype, dk, dv, T))


@pytest.mark.parametrize("label,kw", [
    ("weak_decay", dict(log_alpha_scale=0.01)),
    ("alpha_one", dict(log_alpha_value=0.0)),
    ("beta_0_2", dict(beta_scale=2.0, log_alpha_scale=0.1)),
    ("beta_zero", dict(beta_value=0.0, log_alpha_scale=0.05)),
    ("beta_zero_full_decay", dict(beta_value=0.0)),
    ("strong_decay", dict(log_alpha_scale=8.0)),
])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fwd_stress(G, oracle_mod, label, kw, dtype):
    inp = make_inputs(1, 333, 2, 64, 64, dtype, seed=3, h0_std=0.05, **kw)
    check_fwd(G, oracle_mod, inp, TOL[dtype], "fwd_stress_" + label)


@pytest.mark.parametrize("dtype,dk,dv", [("f32", 64, 64), ("f32", 128, 128), ("f32", 256, 512),
                                         ("bf16", 128, 128), ("bf16", 256, 512)])
def test_fwd_packed(G, oracle_mod, dtype, dk, dv):
    lens = [1, 0, 64, 65, 130, 7, 128]
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32)
    inp = make_inputs(1, int(cu[-1]), 2, dk, dv, dtype, seed=4, h0_std=0.05, cu_seqlens=cu)
    check_fwd(G, oracle_mod, inp, TOL[dtype], "fwd_packed_%s_%d" % (dtype, dk))


def test_packed_many_sequences(G, oracle_mod):
    """More than 256 sequences (the chunk table scans them 256 at a time),
    lengths 0 to 69, forward and stateless backward."""
    rng = np.random.default_rng(11)
    lens = rng.integers(0, 70, size=300)
    lens[5] = 0
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32)
    inp = make_inputs(1, int(cu[-1]), 1, 64, 64, "f32", seed=12, h0_std=0.05, backward=True,
                      cu_seqlens=cu)
    check_fwd(G, oracle_mod, inp, TOL["f32"], "packed_many")
    check_bwd(G, oracle_mod, inp, TOL["f32"], "packed_many")


def test_fwd_split_carry(G):
    inp = to_dev(make_inputs(2, 300, 2, 128, 128, "bf16", seed=5, h0_std=0.05))
    o, ht = run_fwd(G, inp)
    a = {k: (v[:, :100].contiguous() if k in ("q", "k", "v", "beta", "log_alpha") else v)
         for k, v in inp.items()}
    b = {k: (v[:, 100:].contiguous() if k in ("q", "k", "v", "beta", "log_alpha") else v)
         for k, v in inp.items()}
    oa, ha = run_fwd(G, a)
    b["h0"] = ha
    ob, hb = run_fwd(G, b)
    o2 = torch.cat([oa, ob], 1)
    assert rel_err(f64(o2), f64(o)) < 2e-2
    assert rel_err(f64(hb), f64(ht)) < 2e-2


def test_fwd_deterministic(G):
    inp = to_dev(make_inputs(2, 257, 3, 256, 512, "bf16", seed=6, h0_std=0.02))
    o1, h1 = run_fwd(G, inp)
    o2, h2 = run_fwd(G, inp)
    assert torch.equal(o1, o2) and torch.equal(h1, h2)


# ------------------------------------------------------------------ backward, small


@pytest.mark.parametrize("dtype,dk,dv,B,T,H", [
    ("f32", 64, 64, 1, 256, 2),
    ("f32", 64, 64, 2, 150, 2),
    ("f32", 128, 128, 1, 200, 2),
    ("f32", 256, 512, 1, 130, 2),
    ("bf16", 64, 64, 2, 150, 2),
    ("bf16", 128, 128, 1, 200, 2),
    ("bf16", 256, 512, 1, 130, 2),
])
def test_bwd_ragged(G, oracle_mod, dtype, dk, dv, B, T, H):
    inp = make_inputs(B, T, H, dk, dv, dtype, seed=7, h0_std=0.05, backward=True)
    check_bwd(G, oracle_mod, inp, TOL[dtype], "bwd_%s_%d_%d_T%d" % (dtype, dk, dv, T))


@pytest.mark.parametrize("label,kw", [
    ("weak_decay", dict(log_alpha_scale=0.01)),
    ("alpha_one", dict(log_alpha_value=0.0)),
    ("beta_0_2", dict(beta_scale=2.0, log_alpha_scale=0.1)),
    ("beta_zero", dict(beta_value=0.0, log_alpha_scale=0.05)),
    ("strong_decay", dict(log_alpha_scale=8.0)),  # in-chunk log gates to about -350
])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_bwd_stress(G, oracle_mod, label, kw, dtype):
    inp = make_inputs(1, 200, 2, 64, 64, dtype, seed=8, h0_std=0.05, backward=True, **kw)
    check_bwd(G, oracle_mod, inp, TOL[dtype], "bwd_stress_" + label)


@pytest.mark.parametrize("dtype,dk,dv", [("f32", 64, 64), ("f32", 128, 128), ("f32", 256, 512),
                                         ("bf16", 128, 128), ("bf16", 256, 512)])
def test_bwd_packed(G, oracle_mod, dtype, dk, dv):
    lens = [1, 0, 64, 65, 130, 7]
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32)
    inp = make_inputs(1, int(cu[-1]), 2, dk, dv, dtype, seed=9, h0_std=0.05, backward=True,
                      cu_seqlens=cu)
    check_bwd(G, oracle_mod, inp, TOL[dtype], "bwd_packed_%s_%d" % (dtype, dk))


def test_bwd_deterministic(G):
    inp = to_dev(make_inputs(1, 200, 2, 256, 512, "bf16", seed=10, backward=True))
    r1 = run_bwd(G, inp)
    r2 = run_bwd(G, inp)
    for k in r1:
        assert torch.equal(r1[k], r2[k]), k


# ------------------------------------------------------------------ saved-forward path


def run_saved(G, d):
    """Forward that saves, then the backward from its buffer; the buffer must
    come back unchanged."""
    o, ht, saved = G.gdn_chunk_fwd_save(d["q"], d["k"], d["v"], d["beta"], gates(d),
                                        h0=d.get("h0"), cu_seqlens=d.get("cu_seqlens"))
    torch.cuda.synchronize()
    snap = saved.clone()
    r = G.gdn_chunk_bwd_saved(d["q"], d["k"], d["v"], d["beta"], d["dO"], saved, dht=d.get("dht"),
                              cu_seqlens=d.get("cu_seqlens"))
    torch.cuda.synchronize()
    assert torch.equal(saved, snap), "the saved backward wrote to the saved buffer"
    return o, ht, r


def check_saved(G, oracle_mod, inp, tol, label):
    say(label, "saved", tuple(inp["q"].shape), tuple(inp["v"].shape), inp["q"].dtype)
    o, ht, r = run_saved(G, to_dev(inp))
    kw = dict(h0=inp.get("h0"), cu_seqlens=inp.get("cu_seqlens"))
    ro, rht = oracle_mod.fwd(inp["q"], inp["k"], inp["v"], inp["beta"], inp["log_alpha"], **kw)
    ref = oracle_mod.bwd(inp["q"], inp["k"], inp["v"], inp["beta"], inp["log_alpha"], inp["dO"],
                         dht=inp.get("dht"), **kw)
    errs = dict(o=rel_err(f64(o).reshape(ro.shape), ro), ht=rel_err(f64(ht), rht))
    for name in ("dq", "dk", "dv", "dbeta", "dlog_alpha", "dh0"):
        errs[name] = rel_err(f64(r[name]).reshape(ref[name].shape), ref[name])
    say(label, "errs", {k: "%.3g" % v for k, v in errs.items()})
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, bad


@pytest.mark.parametrize("dtype,dk,dv,B,T,H", [
    ("f32", 64, 64, 2, 150, 2),
    ("f32", 128, 128, 1, 200, 2),
    ("bf16", 64, 64, 1, 256, 2),
    ("bf16", 128, 128, 1, 200, 2),
    ("bf16", 256, 512, 1, 130, 2),
])
def test_saved_ragged(G, oracle_mod, dtype, dk, dv, B, T, H):
    inp = make_inputs(B, T, H, dk, dv, dtype, seed=11, h0_std=0.05, backward=True)
    check_saved(G, oracle_mod, inp, TOL[dtype], "saved_%s_%d_%d_T%d" % (dtype, dk, dv, T))


@pytest.mark.parametrize("label,kw", [
    ("alpha_one", dict(log_alpha_value=0.0)),
    ("beta_0_2", dict(beta_scale=2.0, log_alpha_scale=0.1)),
    ("strong_decay", dict(log_alpha_scale=8.0)),
])
@pytest.mark.parametrize("dk", [64, 128])
def test_saved_stress(G, oracle_mod, label, kw, dk):
    inp = make_inputs(1, 200, 2, dk, dk, "f32", seed=12, h0_std=0.05, backward=True, **kw)
    check_saved(G, oracle_mod, inp, TOL["f32"], "saved_stress_%s_%d" % (label, dk))


@pytest.mark.parametrize("label,kw", [
    ("weak_decay", dict(log_alpha_scale=0.01)),
    ("mid_decay", dict(log_alpha_scale=0.05)),
    ("beta_0_2", dict(beta_scale=2.0, log_alpha_scale=0.1)),
])
@pytest.mark.parametrize("dtype,dk,dv", [("bf16", 128, 128), ("bf16", 256, 512),
                                         ("f32", 256, 512)])
@pytest.mark.parametrize("path", ["fwd", "bwd", "saved"])
def test_stress_wide_heads(G, oracle_mod, path, dtype, dk, dv, label, kw):
    """Weak and intermediate decay and beta in (0, 2) at the wide head dims,
    whose kernels are separate instantiations: with e^{g_n} near 1 the
    carried state e^{g_n} S, its gradient and the <dS, S> gate term weigh as
    much as the in-chunk terms.  Four chunks, the last one ragged."""
    inp = make_inputs(1, 200, 2, dk, dv, dtype, seed=21, h0_std=0.05, backward=path != "fwd",
                      **kw)
    name = "stress_%s_%s_%d_%d_%s" % (path, dtype, dk, dv, label)
    if path == "fwd":
        check_fwd(G, oracle_mod, inp, TOL[dtype], name)
    elif path == "bwd":
        check_bwd(G, oracle_mod, inp, TOL[dtype], name)
    else:
        check_saved(G, oracle_mod, inp, TOL[dtype], name)


def test_saved_strong_decay_bf16_256_512(G, oracle_mod):
    """The bench shape's saved path when every decay factor past a few tokens
    underflows fp32 (per-token log gates of about -5.5)."""
    inp = make_inputs(1, 200, 2, 256, 512, "bf16", seed=8, h0_std=0.05, backward=True,
                      log_alpha_scale=8.0)
    check_saved(G, oracle_mod, inp, TOL["bf16"], "saved_strong_bf16_256")


@pytest.mark.parametrize("dtype,dk,dv", [("f32", 64, 64), ("f32", 128, 128), ("f32", 256, 512),
                                         ("bf16", 256, 512)])
def test_saved_packed(G, oracle_mod, dtype, dk, dv):
    lens = [1, 0, 64, 65, 130, 7]
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32)
    inp = make_inputs(1, int(cu[-1]), 2, dk, dv, dtype, seed=13, h0_std=0.05, backward=True,
                      cu_seqlens=cu)
    check_saved(G, oracle_mod, inp, TOL[dtype], "saved_packed_%s_%d" % (dtype, dk))


@pytest.mark.parametrize("dtype,dk,dv", [("f32", 64, 64), ("bf16", 256, 512)])
def test_dense_equals_packed(G, dtype, dk, dv):
    """Dense input locates its chunks arithmetically, packed input through the
    chunk table: the same two sequences given either way give the same bits,
    in both backward paths."""
    B, T, H = 2, 150, 2
    d = to_dev(make_inputs(B, T, H, dk, dv, dtype, seed=16, h0_std=0.05, backward=True))
    p = dict(d)
    for key in ("q", "k", "v", "beta", "log_alpha", "dO"):
        p[key] = d[key].reshape(1, B * T, *d[key].shape[2:]).contiguous()
    p["cu_seqlens"] = torch.tensor([0, T, 2 * T], dtype=torch.int32, device="cuda")
    say("dense_vs_packed", dtype, dk, dv)
    out = {}
    for name, x in (("dense", d), ("packed", p)):
        o, ht = run_fwd(G, x)
        r = run_bwd(G, x)
        o2, ht2, r2 = run_saved(G, x)
        out[name] = dict(o=o.reshape(B * T, -1), ht=ht, o2=o2.reshape(B * T, -1), ht2=ht2,
                         **{k: v.reshape(-1) for k, v in r.items()},
                         **{k + "_s": v.reshape(-1) for k, v in r2.items()})
    diff = {k: float((out["dense"][k].float() - out["packed"][k].float()).abs().max())
            for k in out["dense"]}
    say("dense_vs_packed max |diff|", diff)
    assert all(v == 0.0 for v in diff.values()), diff


@pytest.mark.parametrize("dtype,dk,dv", [("f32", 64, 64), ("bf16", 256, 512)])
def test_saved_equals_stateless(G, dtype, dk, dv):
    """Both backward paths evaluate the same expressions in the same order, so
    their results agree bit for bit, and so do the two forwards."""
    d = to_dev(make_inputs(1, 200, 2, dk, dv, dtype, seed=14, h0_std=0.05, backward=True))
    say("saved_vs_stateless", dtype, dk, dv)
    o, ht = run_fwd(G, d)
    r = run_bwd(G, d)
    o2, ht2, r2 = run_saved(G, d)
    diff = {k: float((r[k].float() - r2[k].float()).abs().max()) for k in r}
    diff.update(o=float((o.float() - o2.float()).abs().max()), ht=float((ht - ht2).abs().max()))
    say("saved_vs_stateless max |diff|", diff)
    assert all(v == 0.0 for v in diff.values()), diff


# ------------------------------------------------------------------ alpha == 1 (no gates)


@pytest.mark.parametrize("dtype,dk,dv,B,T,H", [
    ("f32", 64, 64, 2, 150, 2),
    ("f32", 256, 512, 1, 130, 2),
    ("bf16", 128, 128, 1, 200, 2),
    ("bf16", 256, 512, 1, 130, 2),
])
def test_ungated_matches_oracle(G, oracle_mod, dtype, dk, dv, B, T, H):
    """log_alpha = NULL is the ungated rule (DeltaNet, Sec. 2.2): against the
    oracle at log_alpha = 0, forward and backward, with and without the gate
    gradient."""
    inp = make_inputs(B, T, H, dk, dv, dtype, seed=15, h0_std=0.05, backward=True)
    zero = torch.zeros_like(inp["log_alpha"])
    label = "ungated_%s_%d_%d" % (dtype, dk, dv)
    say(label)
    d = to_dev(inp)
    o, ht = G.gdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], None, h0=d["h0"])
    r = G.gdn_chunk_bwd(d["q"], d["k"], d["v"], d["beta"], None, d["dO"], h0=d["h0"],
                        dht=d["dht"])
    r2 = G.gdn_chunk_bwd(d["q"], d["k"], d["v"], d["beta"], None, d["dO"], h0=d["h0"],
                         dht=d["dht"], need_dlog_alpha=False)
    torch.cuda.synchronize()
    ro, rht = oracle_mod.fwd(inp["q"], inp["k"], inp["v"], inp["beta"], zero, h0=inp["h0"])
    ref = oracle_mod.bwd(inp["q"], inp["k"], inp["v"], inp["beta"], zero, inp["dO"],
                         h0=inp["h0"], dht=inp["dht"])
    errs = dict(o=rel_err(f64(o).reshape(ro.shape), ro), ht=rel_err(f64(ht), rht))
    for name in ("dq", "dk", "dv", "dbeta", "dlog_alpha", "dh0"):
        errs[name] = rel_err(f64(r[name]).reshape(ref[name].shape), ref[name])
    say(label, "errs", {k: "%.3g" % v for k, v in errs.items()})
    bad = {k: v for k, v in errs.items() if not v <= TOL[dtype]}
    assert not bad, bad
    assert r2["dlog_alpha"] is None
    for name in ("dq", "dk", "dv", "dbeta", "dh0"):  # skipping dlog_alpha changes nothing else
        assert torch.equal(r[name], r2[name]), name


@pytest.mark.parametrize("dtype,dk,dv", [("f32", 64, 64), ("bf16", 256, 512)])
def test_ungated_equals_zero_gates(G, dtype, dk, dv):
    """Skipping the gate arithmetic gives exactly what log_alpha = 0 gives
    (every skipped factor is exp(0) = 1), on the stateless and saved paths."""
    d = to_dev(make_inputs(1, 200, 2, dk, dv, dtype, seed=16, h0_std=0.05, backward=True))
    d["log_alpha"] = torch.zeros_like(d["log_alpha"])
    say("ungated_vs_zero_gates", dtype, dk, dv)
    o, ht = run_fwd(G, d)
    r = run_bwd(G, d)
    o2, ht2 = G.gdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], None, h0=d["h0"])
    r2 = G.gdn_chunk_bwd(d["q"], d["k"], d["v"], d["beta"], None, d["dO"], h0=d["h0"],
                         dht=d["dht"])
    o3, ht3, saved = G.gdn_chunk_fwd_save(d["q"], d["k"], d["v"], d["beta"], None, h0=d["h0"])
    r3 = G.gdn_chunk_bwd_saved(d["q"], d["k"], d["v"], d["beta"], d["dO"], saved, dht=d["dht"])
    torch.cuda.synchronize()
    for x, y, z, name in ((o, o2, o3, "o"), (ht, ht2, ht3, "ht")):
        assert torch.equal(x, y) and torch.equal(x, z), name
    for name in r:
        assert torch.equal(r[name], r2[name]) and torch.equal(r[name], r3[name]), name


# ------------------------------------------------------------------ token-by-token form


def run_recurrent(G, d, **kw):
    o, ht = G.gdn_recurrent_fwd(d["q"], d["k"], d["v"], d["beta"], gates(d), h0=d.get("h0"),
                                cu_seqlens=d.get("cu_seqlens"), **kw)
    torch.cuda.synchronize()
    return o, ht


def check_recurrent(G, oracle_mod, inp, tol, label):
    say(label, "recurrent", tuple(inp["q"].shape), tuple(inp["v"].shape), inp["q"].dtype)
    o, ht = run_recurrent(G, to_dev(inp))
    ro, rht = oracle_mod.fwd(inp["q"], inp["k"], inp["v"], inp["beta"], inp["log_alpha"],
                             h0=inp.get("h0"), cu_seqlens=inp.get("cu_seqlens"))
    eo = rel_err(f64(o).reshape(ro.shape), ro)
    eh = rel_err(f64(ht), rht)
    say(label, "err o=%.3g ht=%.3g" % (eo, eh))
    assert eo <= tol and eh <= tol, (eo, eh)


@pytest.mark.parametrize("dtype,dk,dv,B,T,H", [
    ("f32", 64, 64, 2, 150, 2),
    ("f32", 128, 128, 2, 70, 2),
    ("f32", 256, 512, 1, 40, 2),
    ("bf16", 64, 64, 1, 1, 3),
    ("bf16", 128, 128, 2, 37, 2),
    ("bf16", 256, 512, 1, 70, 2),
])
def test_recurrent_matches_oracle(G, oracle_mod, dtype, dk, dv, B, T, H):
    inp = make_inputs(B, T, H, dk, dv, dtype, seed=17, h0_std=0.05)
    check_recurrent(G, oracle_mod, inp, TOL[dtype], "recurrent_%s_%d_%d_T%d" % (dtype, dk, dv, T))


@pytest.mark.parametrize("label,kw", [
    ("beta_0_2", dict(beta_scale=2.0)),
    ("alpha_one", dict(gated=False)),
    ("weak_decay", dict(log_alpha_scale=0.01)),
])
def test_recurrent_stress(G, oracle_mod, label, kw):
    inp = make_inputs(2, 40, 2, 64, 64, "f32", seed=18, h0_std=0.05, **kw)
    check_recurrent(G, oracle_mod, inp, TOL["f32"], "recurrent_stress_" + label)


def test_recurrent_packed(G, oracle_mod):
    lens = [1, 0, 64, 65, 7]
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32)
    inp = make_inputs(1, int(cu[-1]), 2, 128, 128, "bf16", seed=19, h0_std=0.05, cu_seqlens=cu)
    check_recurrent(G, oracle_mod, inp, TOL["bf16"], "recurrent_packed")


@pytest.mark.parametrize("dtype,dk,dv", [("f32", 64, 64), ("bf16", 256, 512)])
def test_decode_continues_prefill(G, oracle_mod, dtype, dk, dv):
    """Prefill with the chunked forward, then single-token decode steps that
    update the state in place: every step's output and the final state match
    the oracle run over the whole sequence."""
    T0, steps = 130, 3
    inp = make_inputs(2, T0 + steps, 2, dk, dv, dtype, seed=20, h0_std=0.05)
    say("decode_after_prefill", dtype, dk, dv)
    d = to_dev(inp)
    pre = {k: (v[:, :T0].contiguous() if isinstance(v, torch.Tensor) and k != "h0" else v)
           for k, v in d.items()}
    _, state = run_fwd(G, pre)
    outs = []
    for t in range(T0, T0 + steps):
        one = {k: v[:, t:t + 1].contiguous() for k, v in d.items()
               if k in ("q", "k", "v", "beta", "log_alpha")}
        o, st = G.gdn_recurrent_fwd(one["q"], one["k"], one["v"], one["beta"], one["log_alpha"],
                                    h0=state, ht=state)
        assert st is state
        outs.append(o)
    torch.cuda.synchronize()
    ro, rht = oracle_mod.fwd(inp["q"], inp["k"], inp["v"], inp["beta"], inp["log_alpha"],
                             h0=inp["h0"])
    eo = rel_err(f64(torch.cat(outs, dim=1)), ro[:, T0:])
    eh = rel_err(f64(state), rht)
    say("decode_after_prefill err o=%.3g ht=%.3g" % (eo, eh))
    assert eo <= TOL[dtype] and eh <= TOL[dtype], (eo, eh)


# ------------------------------------------------------------------ full-size workloads
# The HIP path runs the whole workload exactly as the benchmark launches it;
# the oracle recomputes a sample of independent (sequence, head) units.


def sample_units(inp, units):
    """The listed (sequence, head) units as independent one-head sequences of
    one packed problem: (inputs, [(unit, start, length)])."""
    cu = inp.get("cu_seqlens")
    parts = {k: [] for k in ("q", "k", "v", "beta", "log_alpha", "dO")}
    h0s, dhts, spans, at = [], [], [], 0
    for n, h in units:
        if cu is None:
            sl = lambda x: x[n, :, h:h + 1]
        else:
            s_, e_ = int(cu[n]), int(cu[n + 1])
            sl = lambda x, s_=s_, e_=e_: x[0, s_:e_, h:h + 1]
        for key in parts:
            if key in inp:
                parts[key].append(sl(inp[key]))
        if inp.get("h0") is not None:
            h0s.append(inp["h0"][n:n + 1, h:h + 1])
        if inp.get("dht") is not None:
            dhts.append(inp["dht"][n:n + 1, h:h + 1])
        L = parts["q"][-1].shape[0]
        spans.append(((n, h), at, L))
        at += L
    out = {k: torch.cat(v, 0).unsqueeze(0) for k, v in parts.items() if v}
    out["cu_seqlens"] = torch.tensor([0] + [a + L for _, a, L in spans], dtype=torch.int64)
    out["h0"] = torch.cat(h0s, 0) if h0s else None
    out["dht"] = torch.cat(dhts, 0) if dhts else None
    return out, spans


def full_size_units(w, cu):
    """Every head index at least once, and the first and the last sequence
    (and, packed, the longest) at least once each."""
    N = w.B if cu is None else cu.numel() - 1
    seqs = [0, N - 1]
    if cu is not None:
        seqs.append(int((cu[1:] - cu[:-1]).argmax()))
    rng = np.random.default_rng(0)
    seqs += [int(x) for x in rng.integers(0, N, size=max(0, w.H - len(seqs)))]
    units = {(seqs[h % len(seqs)], h) for h in range(w.H)}
    units |= {(n, int(rng.integers(w.H))) for n in seqs[:3]}
    return sorted(units)


FULL_CASES = [(name, "stateless") for name in WORKLOADS] + \
    [(name, "saved") for name, w in WORKLOADS.items() if w.backward]


@pytest.mark.parametrize("name,path", FULL_CASES)
def test_full_workload_sampled(G, oracle_mod, name, path):
    """The whole workload on the GPU as the benchmark launches it; the oracle
    recomputes a sample of (sequence, head) units that covers every head and
    the first, last and longest sequences.  Prints the per-tensor margin."""
    w = WORKLOADS[name]
    inp = workload_inputs(name)
    say(name, path, "full-size run")
    d = to_dev(inp)
    if path == "saved":
        o, ht, r = run_saved(G, d)
    elif w.recurrent:
        o, ht = run_recurrent(G, d)
        r = None
    else:
        o, ht = run_fwd(G, d)
        r = run_bwd(G, d) if w.backward else None
    del d
    tol = TOL[w.dtype]
    cu = inp.get("cu_seqlens")
    units = full_size_units(w, cu)
    s, spans = sample_units(inp, units)
    say(name, "oracle units", units)
    if w.backward:
        ref = oracle_mod.bwd(s["q"], s["k"], s["v"], s["beta"], s["log_alpha"], s["dO"],
                             h0=s["h0"], dht=s["dht"], cu_seqlens=s["cu_seqlens"])
    else:
        ro, rh = oracle_mod.fwd(s["q"], s["k"], s["v"], s["beta"], s["log_alpha"], h0=s["h0"],
                                cu_seqlens=s["cu_seqlens"])
        ref = dict(o=ro, ht=rh)
    worst = {}
    for i, ((n, h), at, L) in enumerate(spans):
        if cu is None:
            rows = lambda x: x[n, :, h]
        else:
            s_, e_ = int(cu[n]), int(cu[n + 1])
            rows = lambda x, s_=s_, e_=e_: x[0, s_:e_, h]
        got = dict(o=rows(o), ht=ht[n, h])
        want = dict(o=ref["o"][at:at + L, 0], ht=ref["ht"][i, 0])
        if r is not None:
            for key in ("dq", "dk", "dv", "dbeta", "dlog_alpha"):
                got[key] = rows(r[key])
                want[key] = ref[key][at:at + L, 0]
            got["dh0"] = r["dh0"][n, h]
            want["dh0"] = ref["dh0"][i, 0]
        errs = {k: rel_err(f64(v).reshape(want[k].shape), want[k]) for k, v in got.items()}
        for k, e in errs.items():
            worst[k] = max(worst.get(k, 0.0), e)
        say(name, path, (n, h), {k: "%.3g" % v for k, v in errs.items()})
        bad = {k: v for k, v in errs.items() if not v <= tol}
        assert not bad, ((n, h), bad)
    say("margin", name, path, "units=%d" % len(units), "tol=%g" % tol,
        {k: "%.3g (%.0f%% of tol)" % (v, 100 * v / tol) for k, v in worst.items()})


# ------------------------------------------------------------------ NaN isolation


@pytest.mark.parametrize("where", ["q", "k", "v", "beta", "log_alpha", "dO"])
@pytest.mark.parametrize("dtype,dk,dv", [("f32", 64, 64), ("bf16", 128, 128),
                                         ("bf16", 256, 512)])
def test_nan_stays_in_its_unit(G, dtype, dk, dv, where):
    """A NaN planted in one (sequence, head) unit's input leaves every other
    unit bit-identical on every path (forward, stateless backward, saving
    forward + saved backward); packed input, so chunks of several sequences
    share the launches.  No unit's work mixes with another's."""
    cu = torch.tensor([0, 70, 70, 200, 261], dtype=torch.int32)
    inp = make_inputs(1, 261, 3, dk, dv, dtype, seed=32, h0_std=0.05, backward=True,
                      cu_seqlens=cu)
    n0, h0, t0 = 2, 1, 150
    say("nan_isolation", dtype, dk, dv, where)
    clean = to_dev(inp)
    bad = {k: (v.clone() if isinstance(v, torch.Tensor) else v) for k, v in clean.items()}
    bad[where][0, t0, h0] = float("nan")

    def run_all(d):
        o, ht = run_fwd(G, d)
        r = run_bwd(G, d)
        o2, ht2, r2 = run_saved(G, d)
        out = dict(o=o, o2=o2, ht=ht, ht2=ht2)
        out.update({k: v for k, v in r.items()})
        out.update({k + "_s": v for k, v in r2.items()})
        return out

    a, b = run_all(clean), run_all(bad)
    s0, e0 = int(cu[n0]), int(cu[n0 + 1])
    hit = False
    for name in a:
        x, y = a[name].clone(), b[name].clone()
        if x.dim() == 4 and x.shape[0] == 1 and x.shape[1] == 261:  # token rows
            hit |= bool(torch.isnan(y[0, s0:e0, h0]).any())
            x[0, s0:e0, h0] = 0
            y[0, s0:e0, h0] = 0
        elif x.dim() == 3:  # [1, T, H] gates
            hit |= bool(torch.isnan(y[0, s0:e0, h0]).any())
            x[0, s0:e0, h0] = 0
            y[0, s0:e0, h0] = 0
        else:  # states [N, H, dk, dv]
            hit |= bool(torch.isnan(y[n0, h0]).any())
            x[n0, h0] = 0
            y[n0, h0] = 0
        assert torch.equal(x, y), name
    assert hit


# ------------------------------------------------------------------ seeded random cases

SPECIAL_LENGTHS = (0, 1, 2, 63, 64, 65, 127, 128, 129)
DIMS = (("f32", 64, 64), ("f32", 128, 128), ("f32", 256, 512),
        ("bf16", 64, 64), ("bf16", 128, 128), ("bf16", 256, 512))


def random_case(seed):
    """A seeded random problem: dims and dtype by turn; packed (0 to 6
    sequences, lengths drawn from chunk-boundary cases or uniformly) or dense
    (B up to 3, T up to 300); 1 to 3 heads; default, intermediate or weak
    decay; beta up to 1 or up to 2; with or without an initial state."""
    rng = np.random.default_rng(7000 + seed)
    dtype, dk, dv = DIMS[seed % len(DIMS)]
    cap = 300 if dk < 256 else 160
    H = int(rng.integers(1, 4))
    kw = dict(log_alpha_scale=float(rng.choice([1.0, 0.05, 0.01])),
              beta_scale=float(rng.choice([1.0, 2.0])),
              h0_std=0.05 if rng.random() < 0.5 else None)
    if seed % 2 == 0:
        n = int(rng.integers(1, 7))
        lens = [int(rng.choice(SPECIAL_LENGTHS)) if rng.random() < 0.5 else
                int(rng.integers(0, cap)) for _ in range(n)]
        if sum(lens) == 0:
            lens[-1] = 1
        if max(lens) <= 1:  # dlog_alpha would be zero by cancellation
            kw["h0_std"] = 0.05
        cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32)
        inp = make_inputs(1, int(cu[-1]), H, dk, dv, dtype, seed=seed, backward=True,
                          cu_seqlens=cu, **kw)
        shape = "packed %s" % lens
    else:
        B, T = int(rng.integers(1, 4)), int(rng.integers(1, cap))
        if T == 1:  # dlog_alpha would be zero by cancellation
            kw["h0_std"] = 0.05
        inp = make_inputs(B, T, H, dk, dv, dtype, seed=seed, backward=True, **kw)
        shape = "dense B%d T%d" % (B, T)
    label = "random%d %s %d/%d H%d %s %s" % (seed, dtype, dk, dv, H, shape,
                                            {k: v for k, v in kw.items() if v is not None})
    return inp, dtype, label


@pytest.mark.parametrize("seed", range(36))
def test_random_cases_all_paths(G, oracle_mod, seed):
    """Every path (forward, stateless and saved backward, token-by-token
    forward) on a seeded random problem against the oracle."""
    inp, dtype, label = random_case(seed)
    check_fwd(G, oracle_mod, inp, TOL[dtype], label)
    check_bwd(G, oracle_mod, inp, TOL[dtype], label)
    check_saved(G, oracle_mod, inp, TOL[dtype], label)
    check_recurrent(G, oracle_mod, inp, TOL[dtype], label)


@pytest.mark.parametrize("dtype,dk,dv,packed", [("f32", 64, 64, False), ("bf16", 256, 512, False),
                                                ("bf16", 128, 128, True)])
def test_one_token_sequences_without_state(G, oracle_mod, dtype, dk, dv, packed):
    """Sequences of at most one token and no initial state: the entry state is
    zero, so every term of dlog_alpha cancels and its exact value is zero
    (the oracle returns exact zeros).  The kernels form those terms in fp32
    and leave their rounding; the relative metric has no scale there, so the
    residue is bounded by the tolerance times the size of the terms that
    cancel (that of dbeta, whose terms are the same products of k, v and the
    state gradient).  Every other gradient is compared as usual."""
    if packed:
        cu = torch.tensor([0, 1, 1, 2, 3], dtype=torch.int32)
        inp = make_inputs(1, 3, 2, dk, dv, dtype, seed=91, backward=True, cu_seqlens=cu)
    else:
        inp = make_inputs(2, 1, 2, dk, dv, dtype, seed=91, backward=True)
    d = to_dev(inp)
    kw = dict(cu_seqlens=inp.get("cu_seqlens"))
    ref = oracle_mod.bwd(inp["q"], inp["k"], inp["v"], inp["beta"], inp["log_alpha"], inp["dO"],
                         dht=inp["dht"], **kw)
    assert not np.any(np.asarray(ref["dlog_alpha"])), "the oracle's dlog_alpha is not zero"
    scale = float(np.abs(np.asarray(ref["dbeta"])).max())
    assert scale > 0
    for label, r in (("stateless", run_bwd(G, d)), ("saved", run_saved(G, d)[2])):
        say("one_token", dtype, dk, dv, packed, label)
        for name in ("dq", "dk", "dv", "dbeta", "dh0"):
            e = rel_err(f64(r[name]).reshape(ref[name].shape), ref[name])
            assert e <= TOL[dtype], (label, name, e)
        resid = float(np.abs(f64(r["dlog_alpha"])).max())
        say("one_token", label, "dlog_alpha residue %.3g, scale %.3g" % (resid, scale))
        assert resid <= TOL[dtype] * scale, (label, resid, scale)
