"""The no-allocation forward (gdn_chunk_fwd_noalloc) through the C ABI: the
same results, bit for bit, as gdn_chunk_fwd with a caller-owned workspace,
on two calls in a row (the second smaller, so it runs on what the first left
in the library's static array), and within the bf16 bar of the oracle."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2412_06464_amd.inputs import make_inputs

pytestmark = pytest.mark.gpu


def say(*a):
    print("[gpu-case]", *a, flush=True)


@pytest.fixture(scope="module")
def G():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2412_06464_amd import gdn
    gdn.load_library()
    return gdn


def dev(inp):
    return {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}


def test_noalloc_matches_workspace_forward(G, oracle_mod):
    cases = [
        ("dense", make_inputs(2, 300, 3, 256, 512, "bf16", seed=41, h0_std=0.05)),
        ("packed", make_inputs(1, 139, 2, 256, 512, "bf16", seed=42, h0_std=0.05,
                               cu_seqlens=torch.tensor([0, 1, 1, 75, 139], dtype=torch.int32))),
    ]
    refs = []
    for name, inp in cases:
        d = dev(inp)
        p, _ = G.make_problem(d["q"], d["v"], d.get("cu_seqlens"))
        need = G.gdn_chunk_fwd_workspace_size(p)
        say("noalloc", name, tuple(inp["q"].shape), "workspace", need)
        assert need <= G.NOALLOC_SCRATCH_BYTES
        o, ht = G.gdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], h0=d["h0"],
                                cu_seqlens=d.get("cu_seqlens"))
        torch.cuda.synchronize()
        refs.append((d, o.clone(), ht.clone()))
    # two no-allocation calls back to back, the second on a smaller problem
    outs = []
    for (name, inp), (d, _, _) in zip(cases, refs):
        o = torch.full_like(d["v"], float("nan"))
        ht = torch.full((d["h0"].shape), float("nan"), dtype=torch.float32, device="cuda")
        G.gdn_chunk_fwd_noalloc(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], h0=d["h0"],
                                cu_seqlens=d.get("cu_seqlens"), o=o, ht=ht)
        outs.append((o, ht))
    torch.cuda.synchronize()
    for (name, inp), (d, o_ref, ht_ref), (o, ht) in zip(cases, refs, outs):
        assert torch.equal(o, o_ref), name
        assert torch.equal(ht, ht_ref), name
        ro, rht = oracle_mod.fwd(inp["q"], inp["k"], inp["v"], inp["beta"], inp["log_alpha"],
                                 h0=inp["h0"], cu_seqlens=inp.get("cu_seqlens"))
        f = lambda t: t.detach().to("cpu", torch.float64).numpy()
        eo = np.abs(f(o).reshape(ro.shape) - ro).max() / np.abs(ro).max()
        eh = np.abs(f(ht) - rht).max() / np.abs(rht).max()
        say("noalloc", name, "err o=%.3g ht=%.3g" % (eo, eh))
        assert eo <= 2e-2 and eh <= 2e-2


def test_noalloc_rejects_too_large_problem(G):
    d = {"q": torch.zeros((8, 4096, 6, 256), dtype=torch.bfloat16, device="cuda"),
         "v": torch.zeros((8, 4096, 6, 512), dtype=torch.bfloat16, device="cuda")}
    beta = torch.zeros((8, 4096, 6), device="cuda")
    with pytest.raises(G.GdnError) as e:
        G.gdn_chunk_fwd_noalloc(d["q"], d["q"], d["v"], beta, beta)
    assert e.value.code == 5  # GDN_ERR_WORKSPACE
