#!/usr/bin/env python3
"""Throughput of the chunkwise gated delta rule on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

One step = one pass of the whole hot path over one batch of synthetic input.
For forward+backward workloads that is a training step: gdn_chunk_fwd_save
(the forward, keeping what the backward needs) followed by
gdn_chunk_bwd_saved; the stateless pair gdn_chunk_fwd + gdn_chunk_bwd (the
backward recomputes the chunk states) is timed the same way afterwards and
reported beside it.  Forward-only workloads run gdn_chunk_fwd.  Inputs,
outputs, the saved buffer and the workspaces are resident in HBM before the
timed region; the timed region is K steps between two device
synchronisations.  Per-kernel durations come from HIP events that the
library records around each of its launches on the same stream (the *_timed
entry points), one event set per step.

Prints one JSON line (rank 0; this build runs on one GPU only).
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

DEFAULT_WORKLOAD = "fwdbwd_bf16_b8_t4096_h6_dk256_dv512"
METRIC = "tokens/sec gated-delta chunk fwd+bwd (1 GPU); % bf16 MFMA peak"
METRIC_FWD = "tokens/sec gated-delta chunk fwd (1 GPU); % bf16 MFMA peak"
METRIC_RECURRENT = "tokens/sec gated-delta recurrent step (1 GPU); % HBM peak"
METRIC_BLOCK = "tokens/sec gated-delta block prologue+epilogue fwd+bwd (1 GPU); % HBM peak"
# block prologue / epilogue workloads: (B, T, H, dk, dv, conv width)
BLOCK_WORKLOADS = {"block_bf16_b8_t4096_h6_dk256_dv512": (8, 4096, 6, 256, 512, 4)}
PEAK_HBM = 8.0e12          # bytes/s, MI355X HBM3E
PEAK_MFMA_BF16 = 2.5e15    # dense bf16 MFMA FLOP/s
PEAK_MFMA_F32 = 157.3e12   # fp32 matrix FLOP/s
PEAK_VALU_F32 = 157.3e12   # fp32 vector FLOP/s (256 CUs x 2.4 GHz, packed FMA)
CH = 64


def path_flops(w, tokens_heads):
    """Algorithmic FLOP of the path per step (full C x C products counted).
    Forward 6 dk dv + 6 C dk + 4 C dv + C^2/3 per token-head; backward
    12 dk dv + 12 C dk + 8 C dv + 4 C^2 (the stateless recompute not credited)."""
    dk, dv, C = w.dk, w.dv, CH
    f = 6 * dk * dv + 6 * C * dk + 4 * C * dv + C * C / 3
    if w.backward:
        f += 12 * dk * dv + 12 * C * dk + 8 * C * dv + 4 * C * C
    return f * tokens_heads


def path_bytes(w, tokens_heads, n_states, has_h0):
    """Algorithmic HBM bytes per step: every call reads its inputs and writes
    its outputs once.  Forward (2 dk + 2 dv) e + 8 per token-head (q, k, v, o,
    beta, log_alpha); backward (4 dk + 3 dv) e + 16 (q, k, v, dO in; dq, dk, dv
    out; gates in, gate gradients out); plus the fp32 states (ht, h0 if
    given, and dht, dh0 for the backward)."""
    e = 4 if w.dtype == "f32" else 2
    dk, dv = w.dk, w.dv
    st = n_states * dk * dv * 4
    b = ((2 * dk + 2 * dv) * e + 8) * tokens_heads + st * (2 if has_h0 else 1)
    if w.backward:
        b += ((4 * dk + 3 * dv) * e + 16) * tokens_heads + st * (3 if has_h0 else 2)
    return b


def kernel_models(w, n_chunks_heads):
    """Algorithmic work of each kernel launch: {name: (bytes, flops)}.

    Bytes: the operands the kernel's step of the path must read and write
    once (inputs, outputs and the per-chunk intermediates it hands over), per
    chunk-head x number of chunk-heads.  Flops: its matrix products counted at
    full 64 x 64 chunk size (2 M N K each).  e = element bytes of q/k/v."""
    e = 4 if w.dtype == "f32" else 2
    dk, dv, C = w.dk, w.dv, CH
    f32 = 4
    kside, vside, st = C * dk * e, C * dv * e, dk * dv * e
    cc = C * C * e                     # one 64 x 64 operand in the element type
    gates = 2 * C * f32
    prod_dk = 2 * C * C * dk           # 64 x 64 times 64 x dk
    prod_dv = 2 * C * C * dv
    prod_s = 2 * C * dk * dv           # chunk rows times a dk x dv state
    per = {
        # q, k, v, gates in; g, W~, Kbar^T, U~, P out; Gram, inverse, W~, U~
        "fwd:k_prep": (2 * kside + vside + gates + C * f32 + 2 * kside + vside + cc,
                       3 * prod_dk + prod_dv + C ** 3 / 3),
        # as forward, plus P^T, T^T, -W~^T, (e^g Q)^T, and Ak^T
        "bwd:k_prep": (2 * kside + vside + gates + C * f32 + 4 * kside + vside + 3 * cc,
                       4 * prod_dk + prod_dv + C ** 3 / 3),
        # both of the above (P and P^T)
        "fwd:k_prep_save": (2 * kside + vside + gates + C * f32 + 4 * kside + vside + 4 * cc,
                            4 * prod_dk + prod_dv + C ** 3 / 3),
        # W~, q, Kbar^T, P, U~, g in; o out
        "k_fwd_seq": (3 * kside + cc + vside + C * f32 + vside, 3 * prod_s + prod_dv),
        # as k_fwd_seq, plus chunk states and V' out
        "k_fwd_seq_save": (3 * kside + cc + vside + C * f32 + vside + st + vside,
                           3 * prod_s + prod_dv),
        # W~, Kbar^T, U~ in; chunk states and V' out
        "k_fwd_seq_store": (2 * kside + vside + C * f32 + st + vside, 2 * prod_s),
        # k, (e^g Q)^T, -W~^T, P^T, T^T, dO, g, beta in; dS, dX, dv out
        "k_bwd_seq": (3 * kside + 2 * cc + vside + gates + st + 2 * vside,
                      3 * prod_s + 2 * prod_dv),
        # S, dS, q, k, v, dO, V', dX, P^T, Ak^T, gates in; dq, dk, dbeta, dlog_alpha out
        "k_grad": (2 * st + 2 * kside + 4 * vside + 2 * cc + 2 * gates
                   + 2 * kside + gates, 3 * prod_s + 2 * prod_dv + 3 * prod_dk),
        "k_chunk_table": (0, 0),
    }
    return {k: (b * n_chunks_heads, f * n_chunks_heads) for k, (b, f) in per.items()}


def recurrent_model(w, n_units):
    """Algorithmic work of one token-by-token launch: {name: (bytes, flops)}.
    Bytes: the fp32 state slice in and out once per (sequence, head), plus
    q, k, v, o and the two gates per token.  Flops: S^T k, S^T q and the
    rank-one update, 6 dk dv per token (vector ALU, not MFMA)."""
    e = 4 if w.dtype == "f32" else 2
    per_unit = 2 * w.dk * w.dv * 4
    per_tok = (2 * w.dk + 2 * w.dv) * e + 8
    tokens_heads = w.B * w.T * w.H
    return {"fwd:k_recurrent": (per_unit * n_units + per_tok * tokens_heads,
                                6 * w.dk * w.dv * tokens_heads)}


def model_for(models, name):
    """Model of a timed launch named 'fwd:k' / 'bwd:k'."""
    if name in models:
        return models[name]
    return models.get(name.split(":", 1)[-1], (0, 0))


def cpu_baseline(inp, w, budget_s=20.0):
    """Time the oracle (fp64, all host cores) on a bounded sample of the same
    workload: whole (sequence, head) units with their initial states, fwd
    (+bwd).  The sample is run again until about half the budget has passed
    (a decode step takes many passes), and the mean is taken."""
    import torch

    from oracle import oracle
    threads = oracle.default_threads()
    cu = inp.get("cu_seqlens")
    N = w.B if cu is None else cu.numel() - 1
    units = []
    for n in range(N):
        for h in range(w.H):
            units.append((n, h))
    # estimate: ~20 flop * dk * dv per token for fwd+bwd, ~6 for fwd, ~3 GFLOP/s a core
    per_tok = (20 if w.backward else 6) * w.dk * w.dv
    tok_per_unit = w.T if cu is None else w.T / N
    per_unit_s = per_tok * tok_per_unit / 3e9
    n_units = int(max(1, min(len(units), threads * max(1.0, budget_s / per_unit_s / 1.5))))
    if tok_per_unit >= 64:  # long units: a few per thread are enough
        n_units = min(n_units, max(threads, 1) * 4)
    sel = units[:n_units]
    sl = {}
    # pack the selected units as independent sequences of one head each
    qs, ks, vs, bs, las, dOs, dhts, h0s, cus = [], [], [], [], [], [], [], [], [0]
    for n, h in sel:
        if cu is None:
            s = (slice(n, n + 1), slice(None), slice(h, h + 1))
        else:
            s = (slice(0, 1), slice(int(cu[n]), int(cu[n + 1])), slice(h, h + 1))
        qs.append(inp["q"][s][0])
        ks.append(inp["k"][s][0])
        vs.append(inp["v"][s][0])
        bs.append(inp["beta"][s][0])
        las.append(inp["log_alpha"][s][0])
        if w.backward:
            dOs.append(inp["dO"][s][0])
            dhts.append(inp["dht"][n:n + 1, h:h + 1, :, :][0])
        if inp.get("h0") is not None:
            h0s.append(inp["h0"][n:n + 1, h:h + 1, :, :][0])
        cus.append(cus[-1] + qs[-1].shape[0])
    cat = lambda xs: torch.cat(xs, 0).unsqueeze(0)
    sl = dict(q=cat(qs), k=cat(ks), v=cat(vs), beta=cat(bs), log_alpha=cat(las))
    cu_s = torch.tensor(cus, dtype=torch.int64)
    tokens = int(cus[-1])
    h0 = torch.stack(h0s, 0) if h0s else None

    def one_pass():
        if w.backward:
            oracle.bwd(sl["q"], sl["k"], sl["v"], sl["beta"], sl["log_alpha"], cat(dOs), h0=h0,
                       dht=torch.stack(dhts, 0), cu_seqlens=cu_s, nthreads=threads)
        else:
            oracle.fwd(sl["q"], sl["k"], sl["v"], sl["beta"], sl["log_alpha"], h0=h0,
                       cu_seqlens=cu_s, nthreads=threads)

    passes, t0 = 0, time.perf_counter()
    while passes < 10000:
        one_pass()
        passes += 1
        if time.perf_counter() - t0 >= budget_s / 2:
            break
    dt = (time.perf_counter() - t0) / passes
    # each token of the workload carries H heads; the sample covers `tokens`
    # token-heads, i.e. tokens / H workload tokens
    value = (tokens / w.H) / dt
    return {"value": value, "unit": "tokens/s", "cores": min(threads, len(sel)),
            "kind": "oracle",
            "sample": "%d of %d (sequence, head) units, %d token-heads, %s, %.2f s per pass, "
                      "%d passes" % (len(sel), len(units), tokens,
                                     "fwd+bwd" if w.backward else "fwd", dt, passes)}


def kernel_source_digest():
    """sha256 over the HIP sources, to tell whether recorded counters are stale."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2412_06464_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".h")):
            h.update(name.encode())
            h.update(open(os.path.join(csrc, name), "rb").read())
    return h.hexdigest()


def traffic_from_profiles(kernel, workload):
    """HBM bytes per launch measured by rocprofv3 PMC (FETCH_SIZE + WRITE_SIZE,
    scaled by a copy-kernel calibration), if recorded for the current kernel
    source; otherwise None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except ValueError:
        return None
    digest = kernel_source_digest()
    ent = rec.get(workload, {}).get(kernel)
    if not ent or ent.get("kernel_source_sha256") != digest:
        return None
    return ent.get("bytes_per_launch")


def bench_block(args):
    """One step = the block's prologue and epilogue, forward and backward:
    conv+SiLU+L2 of q and k, conv+SiLU of v, RMS norm x gate of the output,
    then the backward of each.  Every call is timed with events on the
    stream the library launches on; the roofline is the slowest call's
    algorithmic bytes (its inputs and outputs once) over its mean time."""
    import torch

    from paper_2412_06464_amd import gdn
    from paper_2412_06464_amd.inputs import make_block_inputs

    B, T, H, dk, dv, W = BLOCK_WORKLOADS[args.workload]
    gdn.load_library()
    inp = make_block_inputs(B, T, H, dk, dv, "bf16", seed=0, width=W)
    d = {k: v.cuda() for k, v in inp.items()}
    out = {k: torch.empty_like(d[k]) for k in ("xq", "xk", "xv", "o")}
    grads = {k: torch.empty_like(d[k]) for k in ("xq", "xk", "xv", "o", "g")}
    dws = {k: torch.empty_like(d[k]) for k in ("wq", "wk", "wv", "wo")}
    pq, _ = gdn.block_problem(d["xq"])
    ws = torch.empty(max(gdn.load_library().gdn_conv_silu_workspace_size(pq, dv, W),
                         gdn.load_library().gdn_norm_gate_workspace_size(pq)), dtype=torch.uint8,
                     device="cuda")
    # C arguments prepared once: a step is eight library calls and nothing else
    import ctypes
    lib = gdn.load_library()
    P = lambda t: ctypes.c_void_p(t.data_ptr())
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    probs = {}
    for key in ("xq", "xv"):
        probs[key], _ = gdn.block_problem(d[key])
    pk, pv = ctypes.byref(probs["xq"]), ctypes.byref(probs["xv"])
    wsp, wsn = P(ws), ws.numel()
    eps_l2, eps_n = ctypes.c_float(1e-6), ctypes.c_float(1e-5)

    def conv_fwd(pp, dim, l2, x, w, y):
        args = (pp, dim, W, l2, eps_l2, P(d[x]), P(d[w]), P(out[y]), wsp, wsn, st)
        return lambda: lib.gdn_conv_silu_fwd(*args)

    def conv_bwd(pp, dim, l2, x, w, dy):
        args = (pp, dim, W, l2, eps_l2, P(d[x]), P(d[w]), P(d[dy]), P(grads[x]), P(dws[w]),
                wsp, wsn, st)
        return lambda: lib.gdn_conv_silu_bwd(*args)

    nf = (pv, eps_n, P(d["o"]), P(d["g"]), P(d["wo"]), P(out["o"]), st)
    nb = (pv, eps_n, P(d["o"]), P(d["g"]), P(d["wo"]), P(d["dy"]), P(grads["o"]), P(grads["g"]),
          P(dws["wo"]), wsp, wsn, st)
    calls = [
        ("conv_fwd_q", conv_fwd(pk, dk, 1, "xq", "wq", "xq"), 2 * dk),
        ("conv_fwd_k", conv_fwd(pk, dk, 1, "xk", "wk", "xk"), 2 * dk),
        ("conv_fwd_v", conv_fwd(pv, dv, 0, "xv", "wv", "xv"), 2 * dv),
        ("norm_gate_fwd", lambda: lib.gdn_norm_gate_fwd(*nf), 3 * dv),
        ("norm_gate_bwd", lambda: lib.gdn_norm_gate_bwd(*nb), 5 * dv),
        ("conv_bwd_q", conv_bwd(pk, dk, 1, "xq", "wq", "dq"), 3 * dk),
        ("conv_bwd_k", conv_bwd(pk, dk, 1, "xk", "wk", "dk"), 3 * dk),
        ("conv_bwd_v", conv_bwd(pv, dv, 0, "xv", "wv", "dv"), 3 * dv),
    ]
    for name, f, _ in calls:  # one checked call each before timing
        rc = f()
        if rc != 0:
            raise gdn.GdnError(rc)
    stream = torch.cuda.current_stream()

    def step(evs=None):
        for i, (_, f, _) in enumerate(calls):
            if evs:
                evs[i][0].record(stream)
            f()
            if evs:
                evs[i][1].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in calls] for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for k in range(args.steps):
        step(evs[k])
    end.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps
    call_ms = {name: sum(evs[k][i][0].elapsed_time(evs[k][i][1]) for k in range(args.steps))
               / args.steps for i, (name, _, _) in enumerate(calls)}
    th = B * T * H
    nbytes = {name: per * 2 * th for name, _, per in calls}  # bf16 elements per token-head
    dom = max(call_ms, key=lambda k: call_ms[k])
    ach = nbytes[dom] / (call_ms[dom] / 1e3)
    roof = {"bound": "hbm", "achieved": ach / 1e9, "peak": PEAK_HBM / 1e9, "unit": "GB/s",
            "frac": ach / PEAK_HBM, "traffic": traffic_from_profiles(dom, args.workload),
            "kernel": dom, "kernel_ms": call_ms[dom]}
    total_bytes = sum(nbytes.values())
    res = {
        "metric": METRIC_BLOCK, "value": B * T / (ms / 1e3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": args.workload, "B": B, "T": T, "H": H, "dk": dk, "dv": dv,
                   "conv_width": W},
        "hbm_frac": total_bytes / (ms / 1e3) / PEAK_HBM, "path_gbytes": total_bytes / 1e9,
        "calls_ms": call_ms, "roofline": roof,
    }
    if not args.no_cpu_baseline:
        from oracle import block
        t0 = time.perf_counter()
        n = 0
        while time.perf_counter() - t0 < 10.0 and n < B:
            sl = slice(n, n + 1)
            block.conv_silu(inp["xq"][sl], inp["wq"], None, True)
            block.conv_silu(inp["xk"][sl], inp["wk"], None, True)
            block.conv_silu(inp["xv"][sl], inp["wv"], None, False)
            block.norm_gate(inp["o"][sl], inp["g"][sl], inp["wo"])
            block.norm_gate_vjp(inp["o"][sl], inp["g"][sl], inp["wo"], inp["dy"][sl])
            block.conv_silu_vjp(inp["xq"][sl], inp["wq"], inp["dq"][sl], None, True)
            block.conv_silu_vjp(inp["xk"][sl], inp["wk"], inp["dk"][sl], None, True)
            block.conv_silu_vjp(inp["xv"][sl], inp["wv"], inp["dv"][sl], None, False)
            n += 1
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": n * T / dt, "unit": "tokens/s", "cores": 1,
                               "kind": "oracle",
                               "sample": "%d of %d sequences, all heads, fwd+bwd, %.1f s" % (
                                   n, B, dt)}
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--path", choices=("saved", "stateless"), default="saved",
                    help="backward path of the headline step (the other is timed beside it)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy 10 times (PMC calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build runs on one GPU only (no sharding, no collectives); "
              "use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2412_06464_amd import gdn
    from paper_2412_06464_amd.inputs import WORKLOADS, workload_inputs

    if args.workload in BLOCK_WORKLOADS:
        bench_block(args)
        return
    if args.copy_calibration:
        x = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        y = torch.empty_like(x)
        x.fill_(1)
        for _ in range(10):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": 1 << 30, "launches": 10}))
        return

    w = WORKLOADS[args.workload]
    gdn.load_library()
    inp = workload_inputs(args.workload, seed=0)
    dev = torch.device("cuda", 0)
    d = {k: (v.to(dev) if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}
    cu = d.get("cu_seqlens")
    cu_host = inp.get("cu_seqlens")
    n_states = w.B if cu is None else cu.numel() - 1

    # everything allocated before the timed region
    p, keep = gdn.make_problem(d["q"], d["v"], cu, cu_host)
    ws_f = torch.empty(gdn.gdn_chunk_fwd_workspace_size(p), dtype=torch.uint8, device=dev)
    o = torch.empty_like(d["v"])
    ht = torch.empty((n_states, w.H, w.dk, w.dv), dtype=torch.float32, device=dev)
    out_b = ws_b = saved = ws_fs = ws_bs = None
    if w.backward:
        ws_b = torch.empty(gdn.gdn_chunk_bwd_workspace_size(p), dtype=torch.uint8, device=dev)
        saved = torch.empty(gdn.gdn_chunk_saved_size(p), dtype=torch.uint8, device=dev)
        ws_fs = torch.empty(gdn.gdn_chunk_fwd_save_workspace_size(p), dtype=torch.uint8,
                            device=dev)
        ws_bs = torch.empty(gdn.gdn_chunk_bwd_saved_workspace_size(p), dtype=torch.uint8,
                            device=dev)
        out_b = dict(dq=torch.empty_like(d["q"]), dk=torch.empty_like(d["k"]),
                     dv=torch.empty_like(d["v"]), dbeta=torch.empty_like(d["beta"]),
                     dlog_alpha=torch.empty_like(d["log_alpha"]),
                     dh0=torch.empty_like(ht))
    fwd_kw = dict(h0=d.get("h0"), cu_seqlens=cu, cu_seqlens_host=cu_host, o=o, ht=ht)
    la = d["log_alpha"] if w.gated else None  # None: alpha == 1, no gate arithmetic

    state = torch.zeros((n_states, w.H, w.dk, w.dv), dtype=torch.float32, device=dev)
    if d.get("h0") is not None:
        state.copy_(d["h0"])

    def step_recurrent(timers=None):
        # one decode step per sequence, the state updated in place
        gdn.gdn_recurrent_fwd(d["q"], d["k"], d["v"], d["beta"], la, h0=state, ht=state,
                              cu_seqlens=cu, cu_seqlens_host=cu_host, o=o,
                              timer=timers[0] if timers else None)

    def step_stateless(timers=None):
        gdn.gdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], la, workspace=ws_f,
                          timer=timers[0] if timers else None, **fwd_kw)
        if w.backward:
            gdn.gdn_chunk_bwd(d["q"], d["k"], d["v"], d["beta"], la, d["dO"],
                              h0=d.get("h0"), dht=d["dht"], cu_seqlens=cu,
                              cu_seqlens_host=cu_host, workspace=ws_b, out=out_b,
                              timer=timers[1] if timers else None)

    def step_saved(timers=None):
        gdn.gdn_chunk_fwd_save(d["q"], d["k"], d["v"], d["beta"], la, saved=saved,
                               workspace=ws_fs, timer=timers[0] if timers else None, **fwd_kw)
        gdn.gdn_chunk_bwd_saved(d["q"], d["k"], d["v"], d["beta"], d["dO"], saved, dht=d["dht"],
                                cu_seqlens=cu, cu_seqlens_host=cu_host, workspace=ws_bs,
                                out=out_b, timer=timers[1] if timers else None)

    stream = torch.cuda.current_stream(dev)

    def timed_run(step):
        """Warm up, then time K steps; returns (ms per step, {kernel: mean ms})."""
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        timers = [(gdn.LaunchTimer(8), gdn.LaunchTimer(8) if w.backward else None)
                  for _ in range(args.steps)]
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(stream)
        for i in range(args.steps):
            step(timers[i])
        end.record(stream)
        torch.cuda.synchronize()
        per_kernel = {}
        for tf, tb in timers:
            for call, t in (("fwd", tf), ("bwd", tb)):
                if t is None:
                    continue
                for name, kms in t.durations_ms().items():
                    per_kernel.setdefault(call + ":" + name, []).append(kms)
            tf.close()
            if tb is not None:
                tb.close()
        return (start.elapsed_time(end) / args.steps,
                {k: sum(v) / len(v) for k, v in per_kernel.items()})

    path = args.path if w.backward else ("recurrent" if w.recurrent else "stateless")
    steps = {"saved": step_saved, "stateless": step_stateless, "recurrent": step_recurrent}
    ms, kern_ms = timed_run(steps[path])
    other = None
    if w.backward:
        oname = "stateless" if path == "saved" else "saved"
        oms, okern = timed_run(steps[oname])
        other = {"path": oname, "ms_per_step": oms, "value": w.B * w.T / (oms / 1e3),
                 "kernels_ms": okern}

    tokens = w.B * w.T
    tokens_heads = tokens * w.H
    n_chunks = (w.B * ((w.T + CH - 1) // CH) if cu_host is None else
                int(sum((int(cu_host[i + 1]) - int(cu_host[i]) + CH - 1) // CH
                        for i in range(n_states))))
    models = (recurrent_model(w, n_states * w.H) if w.recurrent else
              kernel_models(w, n_chunks * w.H))
    dom = max(kern_ms, key=lambda k: kern_ms[k])
    kb, kf = model_for(models, dom)
    peak_mfma = PEAK_MFMA_F32 if w.dtype == "f32" else PEAK_MFMA_BF16
    # the token-by-token kernel computes on the vector ALU, the others on MFMA
    peak_c, cbound = (PEAK_VALU_F32, "alu") if w.recurrent else (peak_mfma, "mfma")
    t_dom = kern_ms[dom] / 1e3
    if kb / PEAK_HBM >= kf / peak_c:
        roof = {"bound": "hbm", "achieved": kb / t_dom / 1e9, "peak": PEAK_HBM / 1e9,
                "unit": "GB/s"}
    else:
        roof = {"bound": cbound, "achieved": kf / t_dom / 1e12, "peak": peak_c / 1e12,
                "unit": "TFLOP/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = traffic_from_profiles(dom, args.workload)
    roof["kernel"] = dom
    roof["kernel_ms"] = kern_ms[dom]

    if w.recurrent:
        nbytes, flops = models["fwd:k_recurrent"]
    else:
        flops = path_flops(w, tokens_heads)
        nbytes = path_bytes(w, tokens_heads, n_states, d.get("h0") is not None)
    res = {
        "metric": METRIC if w.backward else (METRIC_RECURRENT if w.recurrent else METRIC_FWD),
        "value": tokens / (ms / 1e3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if w.dtype == "f32" else "bf16",
        "data": "synthetic",
        "config": {"workload": args.workload, "B": w.B, "T": w.T, "H": w.H, "dk": w.dk,
                   "dv": w.dv, "chunk": CH, "backward": w.backward,
                   "num_seqs": n_states, "path": path},
        "mfma_frac": None if w.recurrent else flops / (ms / 1e3) / peak_mfma,
        "hbm_frac": nbytes / (ms / 1e3) / PEAK_HBM,
        "path_gflop": flops / 1e9,
        "path_gbytes": nbytes / 1e9,
        "kernels_ms": kern_ms,
        "roofline": roof,
    }
    if other is not None:
        res["other_path"] = other
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(inp, w)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
