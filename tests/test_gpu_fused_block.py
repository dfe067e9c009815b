"""GPU parity of the fused block (prologue inside the rule's kernels) against
the fp64 oracle composed the way the block is built (Sec. 3.4): the rule's
q, k, v = oracle block prologue of the projections, rounded to bf16 (the
dtype the fused kernels hand the rule), then the oracle rule; the backward
is the oracle rule's VJP followed by the prologue's VJP.

Same error metric and bar as tests/test_gpu_parity.py: per output tensor,
max|x - ref| / max|ref| <= 2e-2 (bf16 inputs, fp32 arithmetic).
"""
import numpy as np
import pytest
import torch

from paper_2412_06464_amd.inputs import make_block_inputs, make_inputs

pytestmark = pytest.mark.gpu

TOL = 2e-2
EPS = 1e-6


def rel_err(x, ref):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.abs(x - ref).max() / max(float(np.abs(ref).max()), 1e-30))


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


@pytest.fixture(scope="module")
def refs():
    from oracle import block, oracle
    return block, oracle


def fused_inputs(B, T, H, dk, dv, seed, width=4, cu=None, h0_std=0.02):
    """Projections and weights of the prologue, gates and gradients of the rule."""
    rule = make_inputs(B, T, H, dk, dv, "bf16", seed=seed, h0_std=h0_std, backward=True,
                       cu_seqlens=cu)
    blk = make_block_inputs(B, T, H, dk, dv, "bf16", seed=seed + 1000, width=width)
    out = {k: blk[k] for k in ("xq", "xk", "xv", "wq", "wk", "wv")}
    out.update({k: rule[k] for k in ("beta", "log_alpha", "h0", "dO", "dht") if k in rule})
    if cu is not None:
        out["cu_seqlens"] = rule["cu_seqlens"]
    return out


def bf16_round(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(torch.float32).to(torch.bfloat16)


def oracle_block(refs, inp, cu=None):
    """Forward and backward of prologue + rule in fp64."""
    block, oracle = refs
    q = bf16_round(block.conv_silu(inp["xq"], inp["wq"], cu, True, EPS))
    k = bf16_round(block.conv_silu(inp["xk"], inp["wk"], cu, True, EPS))
    v = bf16_round(block.conv_silu(inp["xv"], inp["wv"], cu, False, EPS))
    r = oracle.bwd(q, k, v, inp["beta"], inp["log_alpha"], inp["dO"], h0=inp.get("h0"),
                   dht=inp.get("dht"), cu_seqlens=cu)
    shape = lambda a, like: np.asarray(a).reshape(tuple(like.shape))
    dq, dk, dv = (torch.from_numpy(shape(r[n], t)) for n, t in (("dq", q), ("dk", k),
                                                                  ("dv", v)))
    r["dxq"], r["dwq"] = block.conv_silu_vjp(inp["xq"], inp["wq"], dq, cu, True, EPS)
    r["dxk"], r["dwk"] = block.conv_silu_vjp(inp["xk"], inp["wk"], dk, cu, True, EPS)
    r["dxv"], r["dwv"] = block.conv_silu_vjp(inp["xv"], inp["wv"], dv, cu, False, EPS)
    r["q"], r["k"], r["v"] = q, k, v
    return r


def run_fused(G, inp):
    d = {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}
    cu = d.get("cu_seqlens")
    cuh = inp.get("cu_seqlens")
    args = [d[n] for n in ("xq", "xk", "xv", "wq", "wk", "wv")]
    f = G.gdn_block_fwd(*args, d["beta"], d["log_alpha"], h0=d.get("h0"), eps=EPS,
                        cu_seqlens=cu, cu_seqlens_host=cuh, want_qkv=True, save=True)
    g = G.gdn_block_bwd_saved(*args, f["q"], f["k"], f["v"], d["beta"], d["dO"], f["saved"],
                              dht=d.get("dht"), eps=EPS, cu_seqlens=cu, cu_seqlens_host=cuh)
    plain = G.gdn_block_fwd(*args, d["beta"], d["log_alpha"], h0=d.get("h0"), eps=EPS,
                            cu_seqlens=cu, cu_seqlens_host=cuh)
    torch.cuda.synchronize()
    return f, g, plain


def compare(G, refs, inp, label):
    cu = inp.get("cu_seqlens")
    say(label, tuple(inp["xq"].shape), tuple(inp["xv"].shape), "W=%d" % inp["wq"].shape[1],
        "packed" if cu is not None else "dense")
    f, g, plain = run_fused(G, inp)
    r = oracle_block(refs, inp, cu)
    errs = {}
    for name in ("q", "k", "v"):
        errs[name] = rel_err(f64(f[name]), np.asarray(r[name].to(torch.float64)))
    errs["o"] = rel_err(f64(f["o"]).reshape(r["o"].shape), r["o"])
    errs["ht"] = rel_err(f64(f["ht"]), r["ht"])
    for name in ("dxq", "dxk", "dxv", "dwq", "dwk", "dwv"):
        errs[name] = rel_err(f64(g[name]).reshape(np.shape(r[name])), r[name])
    for name in ("dbeta", "dlog_alpha", "dh0"):
        errs[name] = rel_err(f64(g[name]).reshape(r[name].shape), r[name])
    say(label, {k: "%.3g" % v for k, v in errs.items()})
    bad = {k: v for k, v in errs.items() if not v <= TOL}
    assert not bad, "%s: %s" % (label, bad)
    # the forward without save writes the same o and ht
    assert torch.equal(plain["o"], f["o"]) and torch.equal(plain["ht"], f["ht"]), label


@pytest.mark.parametrize("dk,dv", [(64, 64), (128, 128), (256, 512)])
def test_fused_block_dense(G, refs, dk, dv):
    # 200 tokens: three full chunks and a ragged tail, two sequences
    inp = fused_inputs(2, 200, 2, dk, dv, seed=31)
    compare(G, refs, inp, "fused_dense_%d_%d" % (dk, dv))


@pytest.mark.parametrize("width", [1, 2, 3])
def test_fused_block_short_widths(G, refs, width):
    inp = fused_inputs(1, 150, 2, 64, 64, seed=32 + width, width=width)
    compare(G, refs, inp, "fused_width%d" % width)


@pytest.mark.parametrize("dk,dv", [(64, 64), (256, 512)])
def test_fused_block_packed(G, refs, dk, dv):
    # sequences of 1, 2, 65, 64 and 140 tokens: a sequence shorter than the
    # convolution, one chunk boundary a token into a sequence, exact chunks
    lens = [1, 2, 65, 64, 140]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    inp = fused_inputs(1, int(cu[-1]), 2, dk, dv, seed=37, cu=cu)
    compare(G, refs, inp, "fused_packed_%d_%d" % (dk, dv))


def test_fused_block_full_size_sampled(G, refs):
    """The training workload's shape (8 x 4096 tokens, 6 heads, dk 256, dv 512),
    in the launch configuration the benchmark times.  The oracle runs on head
    0 of every sequence (so dw of head 0 is complete) and on head 5 of the
    last sequence; the other rows of dw need every sequence of their head."""
    B, T, H, dk, dv = 8, 4096, 6, 256, 512
    inp = fused_inputs(B, T, H, dk, dv, seed=0, h0_std=None)
    say("fused full size")
    f, g, _ = run_fused(G, inp)
    units = [(b, 0) for b in range(B)] + [(B - 1, 5)]
    errs, dw0 = {}, {}

    def upd(name, e):
        errs[name] = max(errs.get(name, 0.0), e)

    for b, h in units:
        sub = {n: inp[n][b:b + 1, :, h:h + 1].contiguous() for n in ("xq", "xk", "xv", "beta",
                                                                     "log_alpha", "dO")}
        sub["dht"] = inp["dht"][b:b + 1, h:h + 1].contiguous()
        for n, d in (("wq", dk), ("wk", dk), ("wv", dv)):
            sub[n] = inp[n][h * d:(h + 1) * d].contiguous()
        r = oracle_block(refs, sub)
        upd("o", rel_err(f64(f["o"][b:b + 1, :, h:h + 1]).reshape(r["o"].shape), r["o"]))
        upd("ht", rel_err(f64(f["ht"][b:b + 1, h:h + 1]), r["ht"]))
        for n in ("dxq", "dxk", "dxv"):
            upd(n, rel_err(f64(g[n][b:b + 1, :, h:h + 1]).reshape(np.shape(r[n])), r[n]))
        for n in ("dbeta", "dlog_alpha"):
            upd(n, rel_err(f64(g[n][b:b + 1, :, h:h + 1]).reshape(r[n].shape), r[n]))
        upd("dh0", rel_err(f64(g["dh0"][b:b + 1, h:h + 1]), r["dh0"]))
        if h == 0:  # head 0's weight gradients: the sum over every sequence
            for n in ("dwq", "dwk", "dwv"):
                dw0[n] = dw0.get(n, 0.0) + np.asarray(r[n])
    for n, d in (("dwq", dk), ("dwk", dk), ("dwv", dv)):
        errs[n] = rel_err(f64(g[n][:d]), dw0[n])
    say("fused full size", {k: "%.3g" % v for k, v in errs.items()})
    bad = {k: v for k, v in errs.items() if not v <= TOL}
    assert not bad, bad


@pytest.mark.parametrize("seed", range(9))
def test_fused_block_random(G, refs, seed):
    """Seeded random fused-block problems: dims by turn, convolution width 1
    to 4, packed (lengths from chunk-boundary and convolution-halo cases, or
    uniform) or dense, 1 to 3 heads, with or without an initial state."""
    rng = np.random.default_rng(9000 + seed)
    dk, dv = ((64, 64), (128, 128), (256, 512))[seed % 3]
    width, H = int(rng.integers(1, 5)), int(rng.integers(1, 4))
    h0_std = 0.02 if rng.random() < 0.5 else None
    cap = 260 if dk < 256 else 150
    if rng.random() < 0.5:
        lens = [int(rng.choice((1, 2, 3, 4, 63, 64, 65, 67))) if rng.random() < 0.5 else
                int(rng.integers(1, cap)) for _ in range(int(rng.integers(1, 6)))]
        if max(lens) == 1:  # a zero entry state: dlog_alpha is zero by cancellation
            h0_std = 0.02
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        inp = fused_inputs(1, int(cu[-1]), H, dk, dv, seed=100 + seed, width=width, cu=cu,
                           h0_std=h0_std)
    else:
        B, T = int(rng.integers(1, 3)), int(rng.integers(1, cap))
        if T == 1:
            h0_std = 0.02
        inp = fused_inputs(B, T, H, dk, dv, seed=100 + seed, width=width, h0_std=h0_std)
    compare(G, refs, inp, "fused_random%d" % seed)


@pytest.mark.parametrize("mode", [1, 2])
@pytest.mark.parametrize("dk,dv,packed", [(64, 64, False), (64, 64, True), (128, 128, False),
                                          (128, 128, True), (256, 512, False), (256, 512, True)])
def test_fused_block_both_backward_forms(G, refs, mode, dk, dv, packed):
    """The saved backward's two forms at every size: the prologue's backward
    of q and k inside the gradient kernel (1) and the gradient kernel then
    the convolution backward (2); by default dk picks one."""
    lib = G.load_library()
    if packed:
        lens = [1, 2, 65, 64, 70]
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        inp = fused_inputs(1, int(cu[-1]), 2, dk, dv, seed=41, cu=cu)
    else:
        inp = fused_inputs(2, 150, 2, dk, dv, seed=41)
    prev = lib.gdn_debug_block_bwd(mode)
    try:
        compare(G, refs, inp, "fused_form%d_%d_%d%s" % (mode, dk, dv, "_packed" if packed else ""))
    finally:
        lib.gdn_debug_block_bwd(prev)
