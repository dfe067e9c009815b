#!/usr/bin/env python3
"""Throughput of the chunkwise gated delta rule on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

One step = one pass of the whole hot path over one batch of synthetic input.
For forward+backward workloads that is a training step: gdn_chunk_fwd_save
(the forward, keeping what the backward needs) followed by
gdn_chunk_bwd_saved; the stateless pair gdn_chunk_fwd + gdn_chunk_bwd (the
backward recomputes the chunk states) is timed the same way afterwards and
reported beside it.  Forward-only workloads run gdn_chunk_fwd.

Timing.  Inputs, outputs, the saved buffer and the workspaces are resident in
HBM before anything is timed.  After W untimed warm-up steps, K steps are
timed one by one with HIP events on the launch stream, each after a 512 MiB
write to a scratch buffer that evicts the 256 MB last-level cache and the
L2s ("cold"); the headline is the median cold step, with p10 and p90.  K
more steps back to back without the write give the warm figures.  The
library records events around each of its own launches on the same stream
(the *_timed entry points), so every kernel's duration comes from the same
timed steps.  The headline step is then captured once as a HIP graph and
its replays timed the same way (`graph`; skipped with --no-graph): the
figure without the host work of the calls between the kernels.

Roofline.  Each kernel is credited only with the algorithmic work of its step
of the method: the FLOP of its products at full chunk size, and the bytes of
the call's own tensors (inputs, outputs, initial and final states) that it
reads or writes.  Intermediates the kernels hand each other (chunk states
and their gradients, the chunk-local operands, V', dX) are design overhead
and earn nothing; `traffic_ratio` = HBM bytes measured by counters / those
algorithmic bytes.

Prints one JSON line (this build runs on one GPU only).
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
METRIC_FUSED = "tokens/sec gated-delta block (prologue + chunk rule) fwd+bwd (1 GPU); % bf16 MFMA peak"
# block prologue / epilogue workloads: (B, T, H, dk, dv, conv width)
BLOCK_WORKLOADS = {"block_bf16_b8_t4096_h6_dk256_dv512": (8, 4096, 6, 256, 512, 4)}
# the fused block (prologue inside the rule's kernels), fwd+bwd: the rule's
# training workload of the same name without the prefix, plus its prologue
FUSED_WORKLOADS = {"fusedblock_fwdbwd_bf16_b8_t4096_h6_dk256_dv512":
                   ("fwdbwd_bf16_b8_t4096_h6_dk256_dv512", 4),
                   "fusedblock_fwdbwd_bf16_packed65536_h16_d128":
                   ("fwdbwd_bf16_packed65536_h16_d128", 4)}
PEAK_HBM = 8.0e12          # bytes/s, MI355X HBM3E
PEAK_MFMA_BF16 = 2.5e15    # dense bf16 MFMA FLOP/s
PEAK_MFMA_F32 = 157.3e12   # fp32 matrix FLOP/s
PEAK_VALU_F32 = 157.3e12   # fp32 vector FLOP/s (256 CUs x 2.4 GHz, packed FMA)
FLUSH_BYTES = 512 << 20    # scratch write before every cold step
CH = 64
TOL = {"f32": 1e-4, "bf16": 2e-2}


# ------------------------------------------------------------------ algorithmic work

def path_flops(w, tokens_heads):
    """Algorithmic FLOP of the path per step (full C x C products counted).
    Forward 6 dk dv + 6 C dk + 4 C dv + C^2/3 per token-head; backward
    12 dk dv + 12 C dk + 8 C dv + 4 C^2 (a stateless recompute not credited)."""
    dk, dv, C = w.dk, w.dv, CH
    f = 6 * dk * dv + 6 * C * dk + 4 * C * dv + C * C / 3
    if w.backward:
        f += 12 * dk * dv + 12 * C * dk + 8 * C * dv + 4 * C * C
    return f * tokens_heads


def path_bytes(w, tokens_heads, n_states, has_h0, saved=True):
    """Algorithmic HBM bytes per step: every call reads its inputs and writes
    its outputs once.  Forward (2 dk + 2 dv) e + 8 per token-head (q, k, v, o,
    beta, log_alpha); backward (4 dk + 3 dv) e + 16 (q, k, v, dO in; dq, dk, dv
    out; gates in, gate gradients out); plus the fp32 states of every
    (sequence, head): h0 if given and ht for the forward, dht and dh0 for the
    backward, and h0 again for the stateless backward (the saved backward
    takes its states from the saved buffer)."""
    e = 4 if w.dtype == "f32" else 2
    dk, dv = w.dk, w.dv
    st = n_states * w.H * dk * dv * 4
    b = ((2 * dk + 2 * dv) * e + 8) * tokens_heads + st * (2 if has_h0 else 1)
    if w.backward:
        b += ((4 * dk + 3 * dv) * e + 16) * tokens_heads + st * (3 if has_h0 and not saved else 2)
    return b


def kernel_models(w, tokens_heads, n_units, has_h0):
    """Algorithmic work of each launch: {name: (bytes, flops)}.

    FLOP per token-head of the method's step(s) the kernel performs (products
    at full 64-token chunks): a1 + a2 (gate cumsum, Gram matrices, inverse,
    W~, U~) 6 C dk + 2 C dv + C^2/3; a3 + a4 (state passing and output)
    6 dk dv + 2 C dv; a5 (reverse state pass) 6 dk dv + 4 C dv; a6 + a7
    (per-chunk gradients, gate scan) 6 dk dv + 12 C dk + 4 C dv + 4 C^2.  The
    sum is the path's forward + backward FLOP.  The stateless backward's
    recompute launches are credited with the recompute they perform.
    Bytes: only the call's own tensors the kernel reads or writes (e = element
    bytes; gates fp32; each state dk dv fp32 per (sequence, head))."""
    e = 4 if w.dtype == "f32" else 2
    dk, dv, C = w.dk, w.dv, CH
    st = w.dk * w.dv * 4 * n_units
    a12 = 6 * C * dk + 2 * C * dv + C * C / 3
    qkv_in = (2 * dk + dv) * e + 8                  # q, k, v, beta, log_alpha
    per = {
        "k_prep": (qkv_in, a12, 0),
        "k_prep_save": (qkv_in, a12, 0),
        "k_fwd_seq": (dv * e, 6 * dk * dv + 2 * C * dv, st * (2 if has_h0 else 1)),
        "k_fwd_seq_save": (dv * e, 6 * dk * dv + 2 * C * dv, st * (2 if has_h0 else 1)),
        "k_fwd_seq_store": (0, 4 * dk * dv, st if has_h0 else 0),
        # dO, beta in; dv out; dht in, dh0 out
        "k_bwd_seq": (2 * dv * e + 4, 6 * dk * dv + 4 * C * dv, 2 * st),
        # q, k, v, dO, beta in; dq, dk, dbeta, dlog_alpha out
        "k_grad": ((4 * dk + 2 * dv) * e + 12, 6 * dk * dv + 12 * C * dk + 4 * C * dv + 4 * C * C,
                   0),
        "k_chunk_table": (0, 0, 0),
    }
    return {k: (b * tokens_heads + s, f * tokens_heads) for k, (b, f, s) in per.items()}


def recurrent_model(w, n_units):
    """Algorithmic work of one token-by-token launch: {name: (bytes, flops)}.
    Bytes: the fp32 state in and out once per (sequence, head), plus q, k, v,
    o and the two gates per token.  Flops: S^T k, S^T q and the rank-one
    update, 6 dk dv per token (vector ALU, not MFMA)."""
    e = 4 if w.dtype == "f32" else 2
    per_unit = 2 * w.dk * w.dv * 4
    per_tok = (2 * w.dk + 2 * w.dv) * e + 8
    tokens_heads = w.B * w.T * w.H
    return {"k_recurrent": (per_unit * n_units + per_tok * tokens_heads,
                            6 * w.dk * w.dv * tokens_heads)}


def model_for(models, name):
    """Model of a timed launch named 'fwd:k' / 'bwd:k'."""
    return models.get(name.split(":", 1)[-1], (0, 0))


# ------------------------------------------------------------------ counters on record

def traffic_record(workload):
    """({kernel key: HBM bytes per launch}, HBM bytes per step) measured by
    rocprofv3 PMC (FETCH_SIZE + WRITE_SIZE, scaled by a copy-kernel
    calibration; paper_2412_06464_amd.profiling) on the current kernel
    sources, or ({}, None) if none is on record."""
    from paper_2412_06464_amd.profiling import TRAFFIC, kernel_source_digest
    if not os.path.exists(TRAFFIC):
        return {}, None
    try:
        rec = json.load(open(TRAFFIC)).get(workload)
    except ValueError:
        return {}, None
    if not rec or rec.get("kernel_source_sha256") != kernel_source_digest():
        return {}, None
    return ({k: e["bytes_per_launch"] for k, e in rec.get("kernels", {}).items()},
            rec.get("step_bytes"))


# ------------------------------------------------------------------ timing

def percentiles(xs):
    import numpy as np
    a = np.asarray(xs, dtype=np.float64)
    return {"median": float(np.median(a)), "p10": float(np.percentile(a, 10)),
            "p90": float(np.percentile(a, 90)), "mean": float(a.mean()), "n": int(a.size)}


class StepTimer:
    """Times steps one by one with events on `stream`, optionally after a
    cache-evicting write; collects the library's per-launch event timings."""

    def __init__(self, torch, stream, device):
        self.torch = torch
        self.stream = stream
        self.flush_buf = torch.empty(FLUSH_BYTES // 4, dtype=torch.int32, device=device)

    def run(self, step, k, cold, n_calls, gdn):
        torch = self.torch
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(k)]
        timers = [[gdn.LaunchTimer(8) for _ in range(n_calls)] for _ in range(k)]
        torch.cuda.synchronize()
        for i in range(k):
            if cold:
                self.flush_buf.fill_(i + 1)
            evs[i][0].record(self.stream)
            step(timers[i])
            evs[i][1].record(self.stream)
        torch.cuda.synchronize()
        step_ms = [a.elapsed_time(b) for a, b in evs]
        per_kernel = {}
        for tl in timers:
            for call, t in zip(("fwd", "bwd"), tl):
                for name, kms in t.durations_ms().items():
                    per_kernel.setdefault(call + ":" + name, []).append(kms)
                t.close()
        return step_ms, per_kernel

    def run_graph(self, graph, k, cold):
        """Times k replays of a captured step, one by one, like run()."""
        torch = self.torch
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(k)]
        torch.cuda.synchronize()
        for i in range(k):
            if cold:
                self.flush_buf.fill_(i + 1)
            evs[i][0].record(self.stream)
            graph.replay()
            evs[i][1].record(self.stream)
        torch.cuda.synchronize()
        return [a.elapsed_time(b) for a, b in evs]


# ------------------------------------------------------------------ CPU baseline and parity sample

def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo) and the threads this
    process may run on."""
    name = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                name = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        threads = len(os.sched_getaffinity(0))
    except AttributeError:
        threads = os.cpu_count() or 1
    return name, threads


def sample_units(inp, w, units):
    """Pack the listed (sequence, head) units of the workload as independent
    one-head sequences: (inputs, [(unit, first row, length)])."""
    import torch
    cu = inp.get("cu_seqlens")
    keys = ["q", "k", "v", "beta", "log_alpha"] + (["dO"] if w.backward else [])
    parts = {k: [] for k in keys}
    h0s, dhts, spans, at = [], [], [], 0
    for n, h in units:
        for key in keys:
            x = inp[key]
            parts[key].append(x[n, :, h:h + 1] if cu is None else
                              x[0, int(cu[n]):int(cu[n + 1]), h:h + 1])
        if inp.get("h0") is not None:
            h0s.append(inp["h0"][n:n + 1, h:h + 1])
        if w.backward:
            dhts.append(inp["dht"][n:n + 1, h:h + 1])
        L = parts["q"][-1].shape[0]
        spans.append(((n, h), at, L))
        at += L
    s = {k: torch.cat(v, 0).unsqueeze(0) for k, v in parts.items()}
    s["cu_seqlens"] = torch.tensor([0] + [a + L for _, a, L in spans], dtype=torch.int64)
    s["h0"] = torch.cat(h0s, 0) if h0s else None
    s["dht"] = torch.cat(dhts, 0) if dhts else None
    return s, spans


def oracle_pass(oracle, s, w, threads):
    if w.backward:
        return oracle.bwd(s["q"], s["k"], s["v"], s["beta"], s["log_alpha"], s["dO"], h0=s["h0"],
                          dht=s["dht"], cu_seqlens=s["cu_seqlens"], nthreads=threads)
    o, ht = oracle.fwd(s["q"], s["k"], s["v"], s["beta"], s["log_alpha"], h0=s["h0"],
                       cu_seqlens=s["cu_seqlens"], nthreads=threads)
    return {"o": o, "ht": ht}


def cpu_baseline(inp, w, budget_s=20.0):
    """Time the oracle (fp64) on a bounded sample of the same workload: whole
    (sequence, head) units with their initial states, fwd (+bwd), on every
    host thread, repeated until about half the budget has passed; then once
    more on one thread over a smaller sample.  Returns (record, sampled units,
    spans, oracle results of the multi-thread pass)."""
    from oracle import oracle
    model, threads = cpu_model()
    cu = inp.get("cu_seqlens")
    N = w.B if cu is None else cu.numel() - 1
    units = [(n, h) for n in range(N) for h in range(w.H)]
    # estimate: ~20 flop * dk * dv per token for fwd+bwd, ~6 for fwd, ~3 GFLOP/s a core
    per_tok = (20 if w.backward else 6) * w.dk * w.dv
    tok_per_unit = w.T if cu is None else w.T / N
    per_unit_s = per_tok * tok_per_unit / 3e9
    n_units = int(max(1, min(len(units), threads * max(1.0, budget_s / per_unit_s / 1.5))))
    if tok_per_unit >= 64:  # long units: a few per thread are enough
        n_units = min(n_units, max(threads, 1) * 4)
    # the first sequences with all their heads, and the last unit
    sel = sorted(set(units[:n_units]) | {(N - 1, w.H - 1)})
    s, spans = sample_units(inp, w, sel)
    tokens = int(spans[-1][1] + spans[-1][2])

    passes, t0, ref = 0, time.perf_counter(), None
    while passes < 10000:
        ref = oracle_pass(oracle, s, w, threads)
        passes += 1
        if time.perf_counter() - t0 >= budget_s / 2:
            break
    dt = (time.perf_counter() - t0) / passes
    # single thread: the first units of the sample, about budget / 4 of work
    n1 = max(1, min(len(sel), int(budget_s / 4 / max(per_unit_s, 1e-9))))
    s1, spans1 = sample_units(inp, w, sel[:n1])
    tok1 = int(spans1[-1][1] + spans1[-1][2])
    t1 = time.perf_counter()
    oracle_pass(oracle, s1, w, 1)
    dt1 = time.perf_counter() - t1
    # each token of the workload carries H heads; a sample of `tokens`
    # token-heads is tokens / H workload tokens
    rec = {"value": (tokens / w.H) / dt, "unit": "tokens/s", "cores": min(threads, len(sel)),
           "kind": "oracle", "cpu": model,
           "sample": "%d of %d (sequence, head) units, %d token-heads, %s, %.2f s per pass, "
                     "%d passes, %d threads" % (len(sel), len(units), tokens,
                                                "fwd+bwd" if w.backward else "fwd", dt, passes,
                                                threads),
           "single_thread": {"value": (tok1 / w.H) / dt1, "unit": "tokens/s",
                             "sample": "%d units, %d token-heads, %.2f s" % (n1, tok1, dt1)}}
    return rec, sel, spans, ref


def parity_sample(got, ref, spans, w, cu):
    """max |x - ref| / max |ref| per output tensor over the sampled units."""
    import numpy as np
    import torch
    errs = {}
    for i, ((n, h), at, L) in enumerate(spans):
        for key, x in got.items():
            if x is None:
                continue
            if key in ("ht", "dh0"):
                a, b = x[n, h], ref[key][i, 0]
            else:
                rows = x[n, :, h] if cu is None else x[0, int(cu[n]):int(cu[n + 1]), h]
                a, b = rows, ref[key][at:at + L, 0]
            a = a.detach().to("cpu", torch.float64).numpy().reshape(b.shape)
            num, den = float(np.abs(a - b).max(initial=0.0)), float(np.abs(b).max(initial=0.0))
            e = errs.setdefault(key, [0.0, 0.0])
            e[0], e[1] = max(e[0], num), max(e[1], den)
    out = {k: v[0] / max(v[1], 1e-30) for k, v in errs.items()}
    return {"units": len(spans), "tol": TOL[w.dtype], "err": out,
            "ok": all(v <= TOL[w.dtype] for v in out.values())}


# ------------------------------------------------------------------ block prologue / epilogue

def bench_block(args):
    """One step = the block's prologue and epilogue, forward and backward:
    conv+SiLU+L2 of q and k, conv+SiLU of v, RMS norm x gate of the output,
    then the backward of each.  Steps are timed as in the main path (cold
    median after a cache-evicting write); the roofline is the slowest call's
    algorithmic bytes (its inputs and outputs once) over its mean time."""
    import ctypes

    import torch

    from paper_2412_06464_amd import gdn
    from paper_2412_06464_amd.inputs import make_block_inputs

    B, T, H, dk, dv, W = BLOCK_WORKLOADS[args.workload]
    lib = gdn.load_library()
    inp = make_block_inputs(B, T, H, dk, dv, "bf16", seed=0, width=W)
    d = {k: v.cuda() for k, v in inp.items()}
    out = {k: torch.empty_like(d[k]) for k in ("xq", "xk", "xv", "o")}
    grads = {k: torch.empty_like(d[k]) for k in ("xq", "xk", "xv", "o", "g")}
    dws = {k: torch.empty_like(d[k]) for k in ("wq", "wk", "wv", "wo")}
    pq, _ = gdn.block_problem(d["xq"])
    ws = torch.empty(max(lib.gdn_conv_silu_workspace_size(pq, dv, W),
                         lib.gdn_norm_gate_workspace_size(pq)), dtype=torch.uint8,
                     device="cuda")
    # C arguments prepared once: a step is eight library calls and nothing else
    P = lambda t: ctypes.c_void_p(t.data_ptr())
    stream = torch.cuda.current_stream()
    st = ctypes.c_void_p(stream.cuda_stream)
    probs = {}
    for key in ("xq", "xv"):
        probs[key], _ = gdn.block_problem(d[key])
    pk, pv = ctypes.byref(probs["xq"]), ctypes.byref(probs["xv"])
    wsp, wsn = P(ws), ws.numel()
    eps_l2, eps_n = ctypes.c_float(1e-6), ctypes.c_float(1e-5)

    def conv_fwd(pp, dim, l2, x, w, y):
        a = (pp, dim, W, l2, eps_l2, P(d[x]), P(d[w]), P(out[y]), wsp, wsn, st)
        return lambda: lib.gdn_conv_silu_fwd(*a)

    def conv_bwd(pp, dim, l2, x, w, dy):
        a = (pp, dim, W, l2, eps_l2, P(d[x]), P(d[w]), P(d[dy]), P(grads[x]), P(dws[w]),
             wsp, wsn, st)
        return lambda: lib.gdn_conv_silu_bwd(*a)

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
    flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.int32, device="cuda")

    def run(k, cold):
        evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                for _ in calls] for _ in range(k)]
        se = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(k)]
        torch.cuda.synchronize()
        for i in range(k):
            if cold:
                flush.fill_(i + 1)
            se[i][0].record(stream)
            for j, (_, f, _) in enumerate(calls):
                evs[i][j][0].record(stream)
                f()
                evs[i][j][1].record(stream)
            se[i][1].record(stream)
        torch.cuda.synchronize()
        steps = [a.elapsed_time(b) for a, b in se]
        per = {name: [evs[i][j][0].elapsed_time(evs[i][j][1]) for i in range(k)]
               for j, (name, _, _) in enumerate(calls)}
        return steps, per

    for _ in range(args.warmup):
        for _, f, _ in calls:
            f()
    cold, per = run(args.steps, True)
    warm, _ = run(args.steps, False)
    tc, tw = percentiles(cold), percentiles(warm)
    ms = tc["median"]
    call_ms = {name: sum(v) / len(v) for name, v in per.items()}
    th = B * T * H
    nbytes = {name: n * 2 * th for name, _, n in calls}  # bf16 elements per token-head
    dom = max(call_ms, key=lambda k: call_ms[k])
    ach = nbytes[dom] / (call_ms[dom] / 1e3)
    from paper_2412_06464_amd.profiling import block_kernel_key
    traffic = traffic_record(args.workload)[0].get(block_kernel_key(dom, dk, dv))
    roof = {"bound": "hbm", "achieved": ach / 1e9, "peak": PEAK_HBM / 1e9, "unit": "GB/s",
            "frac": ach / PEAK_HBM, "traffic": traffic,
            "traffic_ratio": traffic / nbytes[dom] if traffic else None,
            "kernel": dom, "kernel_ms": call_ms[dom]}
    total_bytes = sum(nbytes.values())
    res = {
        "metric": METRIC_BLOCK, "value": B * T / (ms / 1e3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": args.workload, "B": B, "T": T, "H": H, "dk": dk, "dv": dv,
                   "conv_width": W},
        "timing": {"cold_ms": tc, "warm_ms": tw, "flush_bytes": FLUSH_BYTES},
        "hbm_frac": total_bytes / (ms / 1e3) / PEAK_HBM, "path_gbytes": total_bytes / 1e9,
        "calls_ms": call_ms, "roofline": roof,
    }
    if not args.no_cpu_baseline:
        from oracle import block
        model, _ = cpu_model()
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
                               "kind": "oracle", "cpu": model,
                               "sample": "%d of %d sequences, all heads, fwd+bwd, %.1f s" % (
                                   n, B, dt)}
    print(json.dumps(res), flush=True)


def fused_models(w, tokens_heads, n_units, has_h0):
    """kernel_models for the fused block's launches: the prologue's
    projections replace the rule's q, k, v as the prep's and the gradient
    kernel's inputs (same sizes), the gradient kernel writes dx instead of
    the rule's dq, dk, and the v prologue's backward reads xv and writes dxv
    (the rule's dv it reads is an intermediate).  The fix-up, which finishes
    three rows per chunk from partial sums, is credited with nothing."""
    m = kernel_models(w, tokens_heads, n_units, has_h0)
    m["k_prep_save_block"] = m["k_prep_save"]
    m["k_prep_block"] = m["k_prep"]
    m["k_grad_block"] = m["k_grad"]
    m["k_block_fixup"] = (0, 0)
    m["k_conv_bwd"] = (2 * w.dv * 2 * tokens_heads, 0)
    # at dk >= 128 the backward runs the plain gradient kernel (its dq, dk
    # are intermediates there) and then the convolution backward of q and k,
    # which reads xq, xk and writes dxq, dxk
    m["k_conv_bwd_qk"] = (4 * w.dk * 2 * tokens_heads, 0)
    return m


def fused_step_bytes(w, tokens_heads, n_states, has_h0):
    """(algorithmic bytes of the block step, bytes the fusion keeps off HBM).
    The block's own tensors: the projections xq, xk, xv read by the forward
    and again by the backward, beta, log_alpha, o, dO, the states, and the
    gradients dxq, dxk, dxv, dbeta, dlog_alpha (= the rule's path bytes, with
    the projections for q, k, v; the weights are a few kB).  Kept off HBM
    against the unfused composition, per token-head (e = 2): the read of the
    rule's q, k, v by the prep (the prologue wrote them; the fused prep writes
    them once, for the backward) (2 dk + dv) e, and at dk = 64, where the
    prologue's backward runs inside the gradient kernel, the rule's dq and dk
    written and read back 4 dk e."""
    e = 2
    kept = 2 * w.dk + w.dv + (4 * w.dk if w.dk < 128 else 0)
    return (path_bytes(w, tokens_heads, n_states, has_h0), kept * e * tokens_heads)


def bench_fused_block(args):
    """One step = the block's prologue and the chunked rule, forward and
    backward: gdn_block_fwd_save + gdn_block_bwd_saved.  The unfused
    composition on the same inputs (gdn_conv_silu_fwd for q, k, v, the
    rule's saving forward and saved backward, gdn_conv_silu_bwd for q, k, v)
    is timed the same way and reported beside it."""
    import ctypes

    import torch

    from paper_2412_06464_amd import gdn
    from paper_2412_06464_amd.inputs import WORKLOADS, make_block_inputs, workload_inputs

    rule_name, W = FUSED_WORKLOADS[args.workload]
    w = WORKLOADS[rule_name]
    lib = gdn.load_library()
    rule = workload_inputs(rule_name, seed=0)
    blk = make_block_inputs(w.B, w.T, w.H, w.dk, w.dv, "bf16", seed=1000, width=W)
    dev = torch.device("cuda", 0)
    d = {k: blk[k].to(dev) for k in ("xq", "xk", "xv", "wq", "wk", "wv")}
    d.update({k: rule[k].to(dev) for k in ("beta", "log_alpha", "dO", "dht")})
    B, T, H, dk, dv = w.B, w.T, w.H, w.dk, w.dv
    eps = 1e-6
    cuh = rule.get("cu_seqlens")  # packed workloads: the same boundaries for every call
    cu = dict(cu_seqlens=cuh.to(dev) if cuh is not None else None, cu_seqlens_host=cuh)
    # everything allocated before the timed region
    xs = (d["xq"], d["xk"], d["xv"], d["wq"], d["wk"], d["wv"])
    f0 = gdn.gdn_block_fwd(*xs, d["beta"], d["log_alpha"], eps=eps, save=True, **cu)
    g0 = gdn.gdn_block_bwd_saved(*xs, f0["q"], f0["k"], f0["v"], d["beta"], d["dO"],
                                 f0["saved"], dht=d["dht"], eps=eps, **cu)
    p, _ = gdn.make_problem(d["xq"], d["xv"], cu["cu_seqlens"], cuh)
    ws_f = torch.empty(gdn.gdn_chunk_fwd_save_workspace_size(p), dtype=torch.uint8, device=dev)
    ws_b = torch.empty(lib.gdn_block_bwd_saved_workspace_size(ctypes.byref(p), W),
                       dtype=torch.uint8, device=dev)
    y = {k: torch.empty_like(d["x" + k]) for k in ("q", "k", "v")}
    pk, _ = gdn.block_problem(d["xq"], cu["cu_seqlens"], cuh)
    ws_c = torch.empty(lib.gdn_conv_silu_workspace_size(ctypes.byref(pk), dv, W),
                       dtype=torch.uint8, device=dev)
    saved_u = torch.empty(gdn.gdn_chunk_saved_size(p), dtype=torch.uint8, device=dev)
    ws_bs = torch.empty(gdn.gdn_chunk_bwd_saved_workspace_size(p), dtype=torch.uint8,
                        device=dev)
    o_u = torch.empty_like(d["xv"])
    ht_u = torch.empty_like(f0["ht"])
    out_u = dict(dq=torch.empty_like(d["xq"]), dk=torch.empty_like(d["xk"]),
                 dv=torch.empty_like(d["xv"]), dbeta=torch.empty_like(d["beta"]),
                 dlog_alpha=torch.empty_like(d["beta"]), dh0=torch.empty_like(f0["ht"]))
    dx_u = {k: torch.empty_like(d["x" + k]) for k in ("q", "k", "v")}
    dw_u = {k: torch.empty_like(d["w" + k]) for k in ("q", "k", "v")}

    def step_fused(timers):
        gdn.gdn_block_fwd(*xs, d["beta"], d["log_alpha"], eps=eps, save=True, o=f0["o"],
                          ht=f0["ht"], q=f0["q"], k=f0["k"], v=f0["v"],
                          saved=f0["saved"], workspace=ws_f,
                          timer=timers[0], **cu)
        gdn.gdn_block_bwd_saved(*xs, f0["q"], f0["k"], f0["v"], d["beta"], d["dO"],
                                f0["saved"], dht=d["dht"], eps=eps, workspace=ws_b, out=g0,
                                timer=timers[1], **cu)

    def step_unfused(timers):
        for k in ("q", "k", "v"):
            gdn.gdn_conv_silu_fwd(d["x" + k], d["w" + k], l2norm=k != "v", eps=eps, y=y[k],
                                  workspace=ws_c, **cu)
        gdn.gdn_chunk_fwd_save(y["q"], y["k"], y["v"], d["beta"], d["log_alpha"], o=o_u,
                               ht=ht_u, saved=saved_u, workspace=ws_f, timer=timers[0], **cu)
        gdn.gdn_chunk_bwd_saved(y["q"], y["k"], y["v"], d["beta"], d["dO"], saved_u,
                                dht=d["dht"], workspace=ws_bs, out=out_u, timer=timers[1],
                                **cu)
        for k in ("q", "k", "v"):
            gdn.gdn_conv_silu_bwd(d["x" + k], d["w" + k], out_u["d" + k], l2norm=k != "v",
                                  eps=eps, dx=dx_u[k], dw=dw_u[k], workspace=ws_c, **cu)

    stream = torch.cuda.current_stream(dev)
    timer = StepTimer(torch, stream, dev)

    def measure(step):
        for _ in range(args.warmup):
            step([None, None])
        torch.cuda.synchronize()
        cold, kern = timer.run(step, args.steps, True, 2, gdn)
        warm, _ = timer.run(step, args.steps, False, 2, gdn)
        return percentiles(cold), percentiles(warm), {k: sum(v) / len(v) for k, v in kern.items()}

    tc, tw, kern_ms = measure(step_fused)
    unfused = agree = None
    if not args.no_other_path:
        uc, uw, ukern = measure(step_unfused)
        unfused = {"ms_per_step": uc["median"], "value": B * T / (uc["median"] / 1e3),
                   "warm_ms": uw["median"], "rule_kernels_ms": ukern}
        # the two compositions agree (same inputs; the fused backward's dx
        # against the unfused one's)
        step_fused([None, None])
        step_unfused([None, None])
        torch.cuda.synchronize()

        def rel(a, b):
            a, b = a.double(), b.double()
            return float((a - b).abs().max() / b.abs().max().clamp_min(1e-30))

        agree = {"o": rel(f0["o"], o_u), "dxq": rel(g0["dxq"], dx_u["q"]),
                 "dxk": rel(g0["dxk"], dx_u["k"]), "dxv": rel(g0["dxv"], dx_u["v"]),
                 "dwq": rel(g0["dwq"], dw_u["q"]),
                 "dbeta": rel(g0["dbeta"], out_u["dbeta"])}

    tokens = B * T
    tokens_heads = tokens * H
    n_states = B if cuh is None else cuh.numel() - 1
    models = fused_models(w, tokens_heads, n_states * H, False)
    dom = max(kern_ms, key=lambda k: kern_ms[k])
    kb, kf = model_for(models, dom)
    t_dom = kern_ms[dom] / 1e3
    if kb / PEAK_HBM >= kf / PEAK_MFMA_BF16:
        roof = {"bound": "hbm", "achieved": kb / t_dom / 1e9, "peak": PEAK_HBM / 1e9,
                "unit": "GB/s"}
    else:
        roof = {"bound": "mfma", "achieved": kf / t_dom / 1e12, "peak": PEAK_MFMA_BF16 / 1e12,
                "unit": "TFLOP/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    from paper_2412_06464_amd.profiling import block_kernel_key, kernel_key
    counters, step_counter = traffic_record(args.workload)
    tr = counters.get(kernel_key(dom, "bf16", dk, dv))
    roof["traffic"] = tr
    roof["traffic_ratio"] = tr / kb if tr and kb else None
    roof.update(kernel=dom, kernel_ms=kern_ms[dom], algorithmic_gbytes=kb / 1e9,
                algorithmic_gflop=kf / 1e9)
    nbytes, saved_model = fused_step_bytes(w, tokens_heads, n_states, False)
    flops = path_flops(w, tokens_heads)
    ms = tc["median"]
    # the unfused composition's counters: the rule's saving training step and
    # the standalone prologue kernels (q and k each one dk-wide call), as
    # measured on their own workloads (the slice sums of dw left out)
    _, rule_step = traffic_record(rule_name)
    bc, _ = traffic_record("block_bf16_b8_t4096_h6_dk256_dv512")
    conv = [(block_kernel_key(c, dk, dv), n) for c, n in (("conv_fwd_q", 2), ("conv_fwd_v", 1),
                                                          ("conv_bwd_q", 2), ("conv_bwd_v", 1))]
    unfused_counter = None
    if rule_step and all(k in bc for k, _ in conv):
        unfused_counter = rule_step + sum(bc[k] * n for k, n in conv)
    res = {
        "metric": METRIC_FUSED, "value": tokens / (ms / 1e3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": args.workload, "B": B, "T": T, "H": H, "dk": dk, "dv": dv,
                   "chunk": CH, "conv_width": W, "backward": True, "path": "fused"},
        "timing": {"cold_ms": tc, "warm_ms": tw, "flush_bytes": FLUSH_BYTES,
                   "warm_value": tokens / (tw["median"] / 1e3)},
        "mfma_frac": flops / (ms / 1e3) / PEAK_MFMA_BF16,
        "hbm_frac": nbytes / (ms / 1e3) / PEAK_HBM,
        "path_gflop": flops / 1e9, "path_gbytes": nbytes / 1e9,
        "fusion_saved_gbytes_model": saved_model / 1e9,
        "step_traffic_gbytes": step_counter / 1e9 if step_counter else None,
        "unfused_traffic_gbytes": unfused_counter / 1e9 if unfused_counter else None,
        "fusion_saved_gbytes_counters": ((unfused_counter - step_counter) / 1e9
                                         if unfused_counter and step_counter else None),
        "kernels_ms": kern_ms, "roofline": roof,
        "unfused": unfused, "fused_vs_unfused_rel": agree,
    }
    print(json.dumps(res), flush=True)


# ------------------------------------------------------------------ main path

def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-path", action="store_true",
                    help="time only the headline path of a fwd+bwd workload")
    ap.add_argument("--path", choices=("saved", "stateless"), default="saved",
                    help="backward path of the headline step (the other is timed beside it)")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip timing the headline step replayed as a captured HIP graph")
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
    if args.workload in FUSED_WORKLOADS:
        bench_fused_block(args)
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
    h0_dev = d.get("h0")

    if h0_dev is not None:
        state.copy_(h0_dev)

    def step_recurrent(timers=None):
        # one decode step per sequence, the state updated in place (every
        # step continues from the state the previous one left)
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
    timer = StepTimer(torch, stream, dev)
    n_calls = 2 if w.backward else 1

    def measure(step):
        """W warm-up steps, K cold steps, K warm steps."""
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        cold, kern = timer.run(step, args.steps, True, n_calls, gdn)
        warm, _ = timer.run(step, args.steps, False, n_calls, gdn)
        return percentiles(cold), percentiles(warm), {k: sum(v) / len(v) for k, v in kern.items()}

    path = args.path if w.backward else ("recurrent" if w.recurrent else "stateless")
    steps = {"saved": step_saved, "stateless": step_stateless, "recurrent": step_recurrent}
    tc, tw, kern_ms = measure(steps[path])
    ms = tc["median"]
    graph = None
    if not args.no_graph:
        # the same step captured once and replayed: the library launches
        # kernels only, so a graph removes the per-call host work between them
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            steps[path]()
        torch.cuda.synchronize()
        for _ in range(args.warmup):
            g.replay()
        gc = percentiles(timer.run_graph(g, args.steps, True))
        gw = percentiles(timer.run_graph(g, args.steps, False))
        graph = {"ms_per_step": gc["median"], "value": w.B * w.T / (gc["median"] / 1e3),
                 "cold_ms": gc, "warm_ms": gw}
        del g
    # outputs of the headline path, for the parity sample (a decode step
    # restarts from the prefill state)
    if w.recurrent and h0_dev is not None:
        state.copy_(h0_dev)
    steps[path]()
    torch.cuda.synchronize()
    got = {"o": o, "ht": state if w.recurrent else ht}
    if w.backward:
        got.update(out_b)
    got = {k: v.detach().to("cpu") for k, v in got.items()}
    other = None
    if w.backward and not args.no_other_path:
        oname = "stateless" if path == "saved" else "saved"
        oc, ow, okern = measure(steps[oname])
        other = {"path": oname, "ms_per_step": oc["median"],
                 "value": w.B * w.T / (oc["median"] / 1e3), "warm_ms": ow["median"],
                 "kernels_ms": okern}

    tokens = w.B * w.T
    tokens_heads = tokens * w.H
    has_h0 = d.get("h0") is not None
    models = (recurrent_model(w, n_states * w.H) if w.recurrent else
              kernel_models(w, tokens_heads, n_states * w.H, has_h0))
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
    from paper_2412_06464_amd.profiling import kernel_key
    counters, step_counter = traffic_record(args.workload)
    if path != ("saved" if w.backward else path):
        step_counter = None  # the counters are taken on the headline path
    tr = counters.get(kernel_key(dom, w.dtype, w.dk, w.dv))
    roof["traffic"] = tr
    roof["traffic_ratio"] = tr / kb if tr and kb else None
    roof.update(kernel=dom, kernel_ms=kern_ms[dom], algorithmic_gbytes=kb / 1e9,
                algorithmic_gflop=kf / 1e9)

    if w.recurrent:
        nbytes, flops = models["k_recurrent"]
    else:
        flops = path_flops(w, tokens_heads)
        nbytes = path_bytes(w, tokens_heads, n_states, has_h0, saved=path == "saved")
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
        "timing": {"cold_ms": tc, "warm_ms": tw, "flush_bytes": FLUSH_BYTES,
                   "warm_value": tokens / (tw["median"] / 1e3)},
        "mfma_frac": None if w.recurrent else flops / (ms / 1e3) / peak_mfma,
        "hbm_frac": nbytes / (ms / 1e3) / PEAK_HBM,
        "path_gflop": flops / 1e9,
        "path_gbytes": nbytes / 1e9,
        "step_traffic_gbytes": step_counter / 1e9 if step_counter else None,
        "step_traffic_ratio": step_counter / nbytes if step_counter else None,
        "kernels_ms": kern_ms,
        "roofline": roof,
    }
    if graph is not None:
        res["graph"] = graph
    if other is not None:
        res["other_path"] = other
    if not args.no_cpu_baseline:
        rec, sel, spans, ref = cpu_baseline(inp, w)
        res["cpu_baseline"] = rec
        res["parity"] = parity_sample(got, ref, spans, w, cu_host)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
