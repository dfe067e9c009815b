"""The path under HIP graph capture (torch.cuda.CUDAGraph on the library's
stream argument): every entry point launches kernels only (no allocation,
no memset, no host synchronisation once outputs, workspaces and both copies
of the packed boundaries are passed in), so a captured call replays the same
kernels.  Each graph is replayed several times on new inputs written in
place, with eager work and synchronisations between the replays, and every
replay must equal, bit for bit, the eager call on the same inputs (the
kernels are deterministic)."""
import numpy as np
import pytest
import torch

from paper_2412_06464_amd.inputs import make_inputs

pytestmark = pytest.mark.gpu

REPLAYS = 3


@pytest.fixture(scope="module")
def G():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2412_06464_amd import gdn
    gdn.load_library()
    return gdn


def say(*a):
    print("[gpu-case]", *a, flush=True)


def dev_inputs(B, T, H, dk, dv, dtype, seed, cu=None, backward=False):
    inp = make_inputs(B, T, H, dk, dv, dtype, seed=seed, h0_std=0.05, backward=backward,
                      cu_seqlens=cu)
    return {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}


def refill(d, src):
    """Write src's tensors into d's (the captured addresses), in place."""
    for k, v in src.items():
        if isinstance(v, torch.Tensor) and k in d and k != "cu_seqlens":
            d[k].copy_(v)


def capture(fn):
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def assert_same(got, ref, label):
    for name, (a, b) in zip(ref.keys(), zip(got.values(), ref.values())):
        if a is None and b is None:
            continue
        assert torch.equal(a, b), (label, name)


@pytest.mark.parametrize("dtype,dk,dv,packed", [("bf16", 128, 128, False), ("f32", 64, 64, True),
                                                ("bf16", 256, 512, False)])
def test_forward_replays_match_eager(G, dtype, dk, dv, packed):
    say("graph_fwd", dtype, dk, dv, packed)
    cu = cu_host = None
    if packed:
        lens = [1, 0, 64, 65, 7]
        cu_host = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32)
        cu = cu_host.cuda()
    B, T = (1, int(cu_host[-1])) if packed else (2, 150)
    d = dev_inputs(B, T, 2, dk, dv, dtype, seed=31, cu=cu_host)
    kw = dict(h0=d["h0"], cu_seqlens=cu, cu_seqlens_host=cu_host)
    o, ht = G.gdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], **kw)
    p, keep = G.make_problem(d["q"], d["v"], cu, cu_host)
    ws = torch.empty(G.gdn_chunk_fwd_workspace_size(p), dtype=torch.uint8, device="cuda")

    def step():
        G.gdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], o=o, ht=ht,
                        workspace=ws, **kw)

    step()
    g = capture(step)
    for r in range(REPLAYS):
        refill(d, dev_inputs(B, T, 2, dk, dv, dtype, seed=40 + r, cu=cu_host))
        g.replay()
        torch.cuda.synchronize()
        ref = G.gdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], **kw)
        torch.cuda.synchronize()
        assert_same({"o": o, "ht": ht}, {"o": ref[0], "ht": ref[1]}, "replay %d" % r)
    del g


def test_noalloc_forward_replays_match_eager(G):
    say("graph_fwd_noalloc")
    d = dev_inputs(2, 130, 2, 64, 64, "bf16", seed=32)
    o = torch.empty_like(d["v"])
    ht = torch.empty((2, 2, 64, 64), dtype=torch.float32, device="cuda")

    def step():
        G.gdn_chunk_fwd_noalloc(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], h0=d["h0"],
                                o=o, ht=ht)

    step()  # the first call on a device looks up the static workspace
    g = capture(step)
    for r in range(REPLAYS):
        refill(d, dev_inputs(2, 130, 2, 64, 64, "bf16", seed=50 + r))
        g.replay()
        torch.cuda.synchronize()
        ref = G.gdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], h0=d["h0"])
        torch.cuda.synchronize()
        assert_same({"o": o, "ht": ht}, {"o": ref[0], "ht": ref[1]}, "replay %d" % r)
    del g


@pytest.mark.parametrize("dtype,dk,dv", [("bf16", 256, 512), ("f32", 128, 128)])
def test_saved_training_step_replays_match_eager(G, dtype, dk, dv):
    """The saving forward and the saved backward captured as one graph."""
    say("graph_saved", dtype, dk, dv)
    B, T, H = 1, 200, 2
    d = dev_inputs(B, T, H, dk, dv, dtype, seed=33, backward=True)
    la = d["log_alpha"]
    o, ht, saved = G.gdn_chunk_fwd_save(d["q"], d["k"], d["v"], d["beta"], la, h0=d["h0"])
    out = G.gdn_chunk_bwd_saved(d["q"], d["k"], d["v"], d["beta"], d["dO"], saved, dht=d["dht"])
    p, _ = G.make_problem(d["q"], d["v"], None, None)
    ws_f = torch.empty(G.gdn_chunk_fwd_save_workspace_size(p), dtype=torch.uint8, device="cuda")
    ws_b = torch.empty(G.gdn_chunk_bwd_saved_workspace_size(p), dtype=torch.uint8, device="cuda")

    def step():
        G.gdn_chunk_fwd_save(d["q"], d["k"], d["v"], d["beta"], la, h0=d["h0"], o=o, ht=ht,
                             saved=saved, workspace=ws_f)
        G.gdn_chunk_bwd_saved(d["q"], d["k"], d["v"], d["beta"], d["dO"], saved, dht=d["dht"],
                              workspace=ws_b, out=out)

    step()
    g = capture(step)
    for r in range(REPLAYS):
        refill(d, dev_inputs(B, T, H, dk, dv, dtype, seed=60 + r, backward=True))
        g.replay()
        torch.cuda.synchronize()
        o2, ht2, s2 = G.gdn_chunk_fwd_save(d["q"], d["k"], d["v"], d["beta"], la, h0=d["h0"])
        ref = G.gdn_chunk_bwd_saved(d["q"], d["k"], d["v"], d["beta"], d["dO"], s2, dht=d["dht"])
        torch.cuda.synchronize()
        assert_same({"o": o, "ht": ht}, {"o": o2, "ht": ht2}, "replay %d fwd" % r)
        assert_same({k: out[k] for k in ref}, ref, "replay %d bwd" % r)
    del g


def test_decode_steps_replay_match_eager(G):
    """A serving loop: one captured decode step (T = 1, state updated in place)
    replayed token after token against eager steps from the same state."""
    say("graph_decode")
    B, H, dk, dv = 4, 2, 256, 512
    d = dev_inputs(B, 1, H, dk, dv, "bf16", seed=34)
    state = d["h0"].clone()
    o = torch.empty_like(d["v"])

    def step():
        G.gdn_recurrent_fwd(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], h0=state, o=o,
                            ht=state)

    ref_state = state.clone()
    step()  # one eager step, then the same from the copied state below
    g = capture(step)
    state.copy_(ref_state)
    for r in range(REPLAYS):
        refill(d, {k: v for k, v in dev_inputs(B, 1, H, dk, dv, "bf16", seed=70 + r).items()
                   if k != "h0"})
        g.replay()
        torch.cuda.synchronize()
        o2, st2 = G.gdn_recurrent_fwd(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"],
                                      h0=ref_state)
        torch.cuda.synchronize()
        assert_same({"o": o, "ht": state}, {"o": o2, "ht": st2}, "token %d" % r)
        ref_state.copy_(st2)
    del g


def block_inputs(B, T, H, dk, dv, seed):
    from paper_2412_06464_amd.inputs import make_block_inputs
    rule = make_inputs(B, T, H, dk, dv, "bf16", seed=seed, h0_std=0.02, backward=True)
    blk = make_block_inputs(B, T, H, dk, dv, "bf16", seed=seed + 1000, width=4)
    out = {k: blk[k] for k in ("xq", "xk", "xv", "wq", "wk", "wv")}
    out.update({k: rule[k] for k in ("beta", "log_alpha", "h0", "dO", "dht")})
    return {k: v.cuda() for k, v in out.items()}


@pytest.mark.parametrize("dk,dv", [(64, 64), (256, 512)])
def test_fused_block_training_step_replays_match_eager(G, dk, dv):
    """The fused block's saving forward and saved backward (with the
    fix-up and the weight-gradient sums) captured as one graph."""
    say("graph_fused_block", dk, dv)
    B, T, H = 1, 200, 2
    d = block_inputs(B, T, H, dk, dv, seed=35)
    x = [d[n] for n in ("xq", "xk", "xv", "wq", "wk", "wv")]
    f = G.gdn_block_fwd(*x, d["beta"], d["log_alpha"], h0=d["h0"], save=True)
    out = G.gdn_block_bwd_saved(*x, f["q"], f["k"], f["v"], d["beta"], d["dO"], f["saved"],
                                dht=d["dht"])
    p, _ = G.make_problem(d["xq"], d["xv"], None, None)
    ws_f = torch.empty(G.gdn_chunk_fwd_save_workspace_size(p), dtype=torch.uint8, device="cuda")
    lib = G.load_library()
    import ctypes
    ws_b = torch.empty(lib.gdn_block_bwd_saved_workspace_size(ctypes.byref(p), 4),
                       dtype=torch.uint8, device="cuda")

    def step():
        G.gdn_block_fwd(*x, d["beta"], d["log_alpha"], h0=d["h0"], save=True, o=f["o"],
                        ht=f["ht"], q=f["q"], k=f["k"], v=f["v"], saved=f["saved"],
                        workspace=ws_f)
        G.gdn_block_bwd_saved(*x, f["q"], f["k"], f["v"], d["beta"], d["dO"], f["saved"],
                              dht=d["dht"], workspace=ws_b, out=out)

    step()
    g = capture(step)
    for r in range(REPLAYS):
        refill(d, block_inputs(B, T, H, dk, dv, seed=80 + r))
        g.replay()
        torch.cuda.synchronize()
        f2 = G.gdn_block_fwd(*x, d["beta"], d["log_alpha"], h0=d["h0"], save=True)
        ref = G.gdn_block_bwd_saved(*x, f2["q"], f2["k"], f2["v"], d["beta"], d["dO"],
                                    f2["saved"], dht=d["dht"])
        torch.cuda.synchronize()
        assert_same({k: f[k] for k in ("o", "ht", "q", "k", "v")},
                    {k: f2[k] for k in ("o", "ht", "q", "k", "v")}, "replay %d fwd" % r)
        assert_same({k: out[k] for k in ref}, ref, "replay %d bwd" % r)
    del g
