"""rocprofv3 output -> the text summaries kept under profiles/ and the
counter record bench.py reads (profiles/traffic.json).

    python -m paper_2412_06464_amd.profiling stats WORKLOAD TRACE_DIR OUT.md --cmd "..."
    python -m paper_2412_06464_amd.profiling traffic WORKLOAD FETCH_DIR WRITE_DIR \
        CAL_FETCH_DIR CAL_WRITE_DIR --step-kernel KEY --cmd "..." [--md OUT.md]
    python -m paper_2412_06464_amd.profiling summary WORKLOAD OUT.md --bench B.json \
        --trace TRACE_DIR --pmc FETCH WRITE CAL_FETCH CAL_WRITE --step-kernel KEY --cmd ...
    python -m paper_2412_06464_amd.profiling mfma WORKLOAD TRACE_DIR OUT.md SET1 SET2 SET3 \
        --cmd ...   (the counter runs of MFMA_SETS)

A kernel is identified by its key: base name and template arguments, e.g.
k_prep<bf16,256,512,2,1> (the saving prep with the block prologue),
k_fwd_seq<bf16,256,512,2>, k_grad<bf16,256,512,0>.  bench.py maps its timed
launches to keys with kernel_key().

Counters.  FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are taken in runs of
their own and scaled by what the same counter reads for a 1 GiB
device-to-device copy (bench.py --copy-calibration), so that a byte of the
record is a byte the copy moves.  A workload's record holds, per kernel key,
the mean bytes per dispatch and the number of dispatches, and the bytes of
one step: every gdn kernel's bytes over the run divided by the dispatches of
the step kernel (a kernel that runs once per step; the profiled run times
only the headline path).  The record is tied to the digest of the HIP
sources it was measured on; bench.py ignores it once they change.
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import hashlib
import json
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
TRAFFIC = os.path.join(ROOT, "profiles", "traffic.json")
COPY_BYTES = 1 << 30


def kernel_source_digest() -> str:
    """sha256 over the HIP sources and headers of libgdn (sorted by name)."""
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.h"))):
        h.update(os.path.basename(p).encode())
        h.update(open(p, "rb").read())
    return h.hexdigest()


def kernel_key_of(name: str) -> str:
    """Key of a kernel from its (mangled) name in a rocprofv3 CSV; names
    outside the library are returned cut at their argument list."""
    m = re.match(r"_ZN3gdn\d+(k_[a-z_0-9]+)(I(.*)E)?Ev", name)
    if not m:
        m2 = re.match(r"_ZN3gdn\d+(k_[a-z_0-9]+)Ev?", name)
        if m2:
            return m2.group(1)
        # already demangled: [void ]gdn::k_name<float, 64, 64, 0, false>(...)
        d = re.match(r"(?:void )?gdn::(k_[a-z_0-9]+)(?:<([^>]*)>)?", name)
        if d:
            if d.group(2) is None:
                return d.group(1)
            conv = {"float": "f32", "__bf16": "bf16", "false": "0", "true": "1"}
            args = [conv.get(x.strip(), x.strip()) for x in d.group(2).split(",")]
            return "%s<%s>" % (d.group(1), ",".join(args))
        return name.split("(")[0].replace("void ", "")
    base, tpl = m.group(1), m.group(3)
    if tpl is None:
        return base
    args = []
    i = 0
    while i < len(tpl):
        if tpl.startswith("DF16b", i):
            args.append("bf16")
            i += 5
        elif tpl[i] == "f" and not args:
            args.append("f32")
            i += 1
        elif tpl.startswith("Li", i) or tpl.startswith("Lb", i):
            j = tpl.index("E", i)
            args.append(tpl[i + 2:j])
            i = j + 1
        else:
            i += 1
    return "%s<%s>" % (base, ",".join(args))


def kernel_key(launch: str, dtype: str, dk: int, dv: int) -> str:
    """Key of the main kernel behind a timed launch of bench.py ('fwd:k_prep',
    'bwd:k_grad_block', ...); helper kernels (gate scan, slice sums) are not
    named by a launch."""
    call, _, name = launch.rpartition(":")
    t = "bf16" if dtype == "bf16" else "f32"
    blk = name.endswith("_block")
    base = name[:-len("_block")] if blk else name
    if base in ("k_prep", "k_prep_save"):
        mode = 2 if base == "k_prep_save" else (1 if call == "bwd" else 0)
        return "k_prep<%s,%d,%d,%d,%d>" % (t, dk, dv, mode, int(blk))
    modes = {"k_fwd_seq": 0, "k_fwd_seq_store": 1, "k_fwd_seq_save": 2}
    if base in modes:
        return "k_fwd_seq<%s,%d,%d,%d>" % (t, dk, dv, modes[base])
    if base == "k_grad":
        return "k_grad<%s,%d,%d,%d>" % (t, dk, dv, int(blk))
    if base in ("k_bwd_seq", "k_recurrent"):
        return "%s<%s,%d,%d>" % (base, t, dk, dv)
    if name == "k_block_fixup":
        return "k_block_fixup<%s,%d>" % (t, dk)
    if name == "k_conv_bwd":  # the v prologue (no row norm): slices of 256 channels
        return "k_conv_bwd<%s,%d,%d>" % (t, dv, min(dv, 256))
    return name


def block_kernel_key(call: str, dk: int, dv: int) -> str:
    """Key of a call of the standalone block bench (conv_fwd_q, norm_gate_bwd, ...)."""
    if call.startswith("conv_"):
        d = dv if call.endswith("_v") else dk
        l2 = not call.endswith("_v")
        dl = d if (l2 or d <= 256) else 256
        return "k_%s<bf16,%d,%d>" % (call.rsplit("_", 1)[0], d, dl)
    return "k_%s<bf16,%d>" % (call, dv)


def _csv_rows(d: str, suffix: str):
    paths = glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True)
    if not paths:
        raise FileNotFoundError("no *%s under %s" % (suffix, d))
    return list(csv.DictReader(open(paths[0])))


def _counter(d: str):
    """{kernel key: [bytes of each dispatch]} of one counter run (KiB -> bytes)."""
    acc = collections.defaultdict(list)
    for r in _csv_rows(d, "counter_collection.csv"):
        acc[kernel_key_of(r["Kernel_Name"])].append(float(r["Counter_Value"]) * 1024)
    return acc


def _calibration(d: str) -> float:
    """Bytes per counted byte: the copy kernel's largest dispatch against 1 GiB."""
    return COPY_BYTES / max(max(v) for v in _counter(d).values())


def traffic(workload, fetch_dir, write_dir, cal_fetch, cal_write, step_kernel, cmd, md=None):
    cf, cw = _calibration(cal_fetch), _calibration(cal_write)
    fe, wr = _counter(fetch_dir), _counter(write_dir)
    kernels = {}
    for key in sorted(set(fe) | set(wr)):
        f = fe.get(key, [0.0])
        w = wr.get(key, [0.0])
        rd, wb = sum(f) / len(f) * cf, sum(w) / len(w) * cw
        kernels[key] = {"bytes_per_launch": rd + wb, "read_bytes": rd, "write_bytes": wb,
                        "launches": max(len(fe.get(key, [])), len(wr.get(key, [])))}
    if step_kernel not in kernels:
        raise KeyError("step kernel %s not in the run (%s)" % (step_kernel, sorted(kernels)))
    steps = kernels[step_kernel]["launches"]
    gdn = {k: v for k, v in kernels.items() if k.startswith("k_")}
    step_bytes = sum(v["bytes_per_launch"] * v["launches"] for v in gdn.values()) / steps
    rec = json.load(open(TRAFFIC)) if os.path.exists(TRAFFIC) else {}
    rec[workload] = {"kernels": gdn, "step_bytes": step_bytes, "steps": steps,
                     "step_kernel": step_kernel,
                     "calibration": {"FETCH_SIZE": cf, "WRITE_SIZE": cw},
                     "kernel_source_sha256": kernel_source_digest(), "command": cmd}
    os.makedirs(os.path.dirname(TRAFFIC), exist_ok=True)
    json.dump(rec, open(TRAFFIC, "w"), indent=1, sort_keys=True)
    if md:
        lines = ["# HBM traffic per launch: %s" % workload, "",
                 "Commands (from the repository root, on one MI355X; rocprofv3 after "
                 "`cd /tmp && export TMPDIR=/tmp`):", "", "```", cmd, "```", "",
                 "FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each scaled by what it reads "
                 "for a 1 GiB device-to-device copy: x%.3f and x%.3f." % (cf, cw), "",
                 "| kernel | launches | read MB | write MB | total MB per launch |",
                 "|---|---|---|---|---|"]
        for k, v in sorted(gdn.items(), key=lambda kv: -kv[1]["bytes_per_launch"]):
            lines.append("| `%s` | %d | %.1f | %.1f | %.1f |" % (
                k, v["launches"], v["read_bytes"] / 1e6, v["write_bytes"] / 1e6,
                v["bytes_per_launch"] / 1e6))
        lines += ["", "One step (%d steps counted by `%s`): %.3f GB." % (
            steps, step_kernel, step_bytes / 1e9)]
        open(md, "w").write("\n".join(lines) + "\n")
    return rec[workload]


def stats(workload, trace_dir, out, cmd):
    rows = _csv_rows(trace_dir, "kernel_stats.csv")
    lines = ["# Kernel trace: %s" % workload, "",
             "Command (from the repository root, on one MI355X; rocprofv3 after "
             "`cd /tmp && export TMPDIR=/tmp`):", "", "```", cmd, "```", "",
             "| kernel | calls | avg µs | min µs | max µs | % of GPU time |",
             "|---|---|---|---|---|---|"]
    for r in rows:
        lines.append("| `%s` | %s | %.1f | %.1f | %.1f | %.1f |" % (
            kernel_key_of(r["Name"]), r["Calls"], float(r["AverageNs"]) / 1e3,
            float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3, float(r["Percentage"])))
    open(out, "w").write("\n".join(lines) + "\n")


def summary(workload, out, bench_json=None, trace_dir=None, pmc=None, step_kernel=None,
            commands=()):
    """One summary per workload: the bench line, the kernel trace and the
    counters (pmc = (fetch_dir, write_dir, cal_fetch_dir, cal_write_dir));
    commands are the ones that produced them, listed first."""
    lines = ["# %s" % workload, "",
             "Commands (from the repository root, on one MI355X; rocprofv3 after "
             "`cd /tmp && export TMPDIR=/tmp`; the last two build this file and "
             "profiles/traffic.json from their output):", "", "```"]
    lines += list(commands) + ["```", ""]
    if bench_json:
        j = json.loads(open(bench_json).read().strip().splitlines()[-1])
        lines += ["## bench.py line", "", "```json", json.dumps(j, indent=1), "```", ""]
    if trace_dir:
        rows = _csv_rows(trace_dir, "kernel_stats.csv")
        lines += ["## Kernel trace (rocprofv3 --kernel-trace --stats)", "",
                  "| kernel | calls | avg µs | min µs | max µs | % of GPU time |",
                  "|---|---|---|---|---|---|"]
        for r in rows:
            lines.append("| `%s` | %s | %.1f | %.1f | %.1f | %.1f |" % (
                kernel_key_of(r["Name"]), r["Calls"], float(r["AverageNs"]) / 1e3,
                float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3, float(r["Percentage"])))
        lines.append("")
    if pmc:
        rec = traffic(workload, *pmc, step_kernel, "\n".join(commands))
        cf, cw = rec["calibration"]["FETCH_SIZE"], rec["calibration"]["WRITE_SIZE"]
        lines += ["## HBM traffic per launch (rocprofv3 --pmc FETCH_SIZE, WRITE_SIZE)", "",
                  "Each counter scaled by what it reads for a 1 GiB device-to-device copy: "
                  "x%.3f and x%.3f." % (cf, cw), "",
                  "| kernel | launches | read MB | write MB | total MB per launch |",
                  "|---|---|---|---|---|"]
        for k, v in sorted(rec["kernels"].items(), key=lambda kv: -kv[1]["bytes_per_launch"]):
            lines.append("| `%s` | %d | %.1f | %.1f | %.1f |" % (
                k, v["launches"], v["read_bytes"] / 1e6, v["write_bytes"] / 1e6,
                v["bytes_per_launch"] / 1e6))
        lines += ["", "One step (%d steps counted by `%s`): %.3f GB." % (
            rec["steps"], step_kernel, rec["step_bytes"] / 1e9), ""]
    open(out, "w").write("\n".join(lines))


# Counter sets of the MFMA and stall profile, one rocprofv3 --pmc run each
# (within the per-run limits: at most 8 SQ, 4 TCP, 2 TA, 2 GRBM counters).
MFMA_SETS = (
    "SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CU_CYCLES SQ_INSTS_MFMA "
    "SQ_WAVE_CYCLES SQ_WAIT_INST_ANY SQ_ACTIVE_INST_VMEM GRBM_GUI_ACTIVE",
    "SQ_WAIT_ANY SQ_ACTIVE_INST_ANY SQ_WAIT_INST_LDS SQ_ACTIVE_INST_LDS SQ_INST_LEVEL_VMEM "
    "SQ_INSTS_VMEM_RD SQ_INSTS_VMEM_WR SQ_LEVEL_WAVES GRBM_GUI_ACTIVE",
    "TCP_TCC_READ_REQ_LATENCY_sum TCP_TCC_READ_REQ_sum TCP_TOTAL_CACHE_ACCESSES_sum TA_BUSY_avr "
    "GRBM_GUI_ACTIVE",
)


def mfma(workload, trace_dir, set_dirs, out, commands=()):
    """MFMA use and stalls per kernel from the counter runs of MFMA_SETS and
    the average durations of a kernel trace of the same build.  bf16 MFMA
    FLOP = 512 x SQ_INSTS_VALU_MFMA_MOPS_BF16; 'waiting' = SQ_WAIT_INST_ANY /
    SQ_WAVE_CYCLES (wave time in s_waitcnt), 'issuing' = SQ_ACTIVE_INST_ANY /
    SQ_WAVE_CYCLES; L2 read latency = TCP_TCC_READ_REQ_LATENCY_sum /
    TCP_TCC_READ_REQ_sum (cycles per L1-to-L2 read request); clock =
    GRBM_GUI_ACTIVE / XCDs / the same dispatch's duration (median over the
    dispatches of the three runs), and the MFMA fraction against the peak
    scaled to that clock (the 2.5 PFLOP/s peak is at 2.4 GHz)."""
    dur = {kernel_key_of(r["Name"]): float(r["AverageNs"]) * 1e-9
           for r in _csv_rows(trace_dir, "kernel_stats.csv")}
    acc = collections.defaultdict(lambda: collections.defaultdict(list))
    clk = collections.defaultdict(list)
    for d in set_dirs:
        xcc = 8
        for r in _csv_rows(d, "agent_info.csv"):
            if r.get("Agent_Type", "").upper().endswith("GPU") and int(r.get("Num_Xcc") or 0) > 0:
                xcc = int(r["Num_Xcc"])
        for r in _csv_rows(d, "counter_collection.csv"):
            key = kernel_key_of(r["Kernel_Name"])
            acc[key][r["Counter_Name"]].append(float(r["Counter_Value"]))
            ns = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
            if r["Counter_Name"] == "GRBM_GUI_ACTIVE" and ns > 0:
                clk[key].append(float(r["Counter_Value"]) / xcc / ns)
    m = {k: {c: sum(v) / len(v) for c, v in d.items()} for k, d in acc.items()}
    lines = ["# MFMA use and stalls: %s" % workload, "",
             "Commands (from the repository root, on one MI355X; rocprofv3 after "
             "`cd /tmp && export TMPDIR=/tmp`):", "", "```"] + list(commands) + ["```", "",
             mfma.__doc__.split("\n\n")[0].replace("\n    ", " ").strip() + "  Peak: 2.5 PFLOP/s "
             "dense bf16.", "",
             "| kernel | avg µs | bf16 MFMA GFLOP | achieved TFLOP/s | % of bf16 peak | "
             "clock GHz | % of peak at that clock | waiting | issuing | L2 read latency (cycles) |",
             "|---|---|---|---|---|---|---|---|---|---|"]
    for k in sorted(dur, key=lambda k: -dur[k]):
        d = m.get(k, {})
        fl = d.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) * 512
        if not fl:
            continue
        t, wave = dur[k], max(d.get("SQ_WAVE_CYCLES", 0.0), 1.0)
        lat = d.get("TCP_TCC_READ_REQ_LATENCY_sum", 0.0) / max(d.get("TCP_TCC_READ_REQ_sum", 1.0), 1.0)
        ghz = sorted(clk[k])[len(clk[k]) // 2] if clk.get(k) else float("nan")
        lines.append("| `%s` | %.0f | %.1f | %.0f | %.1f%% | %.2f | %.1f%% | %.0f%% | %.0f%% | %.0f |" % (
            k, t * 1e6, fl / 1e9, fl / t / 1e12, 100 * fl / t / 2.5e15, ghz,
            100 * fl / t / (2.5e15 * ghz / 2.4), 100 * d.get("SQ_WAIT_INST_ANY", 0.0) / wave,
            100 * d.get("SQ_ACTIVE_INST_ANY", 0.0) / wave, lat))
    open(out, "w").write("\n".join(lines) + "\n")


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="what", required=True)
    s = sub.add_parser("stats")
    s.add_argument("workload")
    s.add_argument("trace_dir")
    s.add_argument("out")
    s.add_argument("--cmd", required=True)
    t = sub.add_parser("traffic")
    t.add_argument("workload")
    for n in ("fetch_dir", "write_dir", "cal_fetch", "cal_write"):
        t.add_argument(n)
    t.add_argument("--step-kernel", required=True)
    t.add_argument("--cmd", required=True)
    t.add_argument("--md")
    u = sub.add_parser("summary")
    u.add_argument("workload")
    u.add_argument("out")
    u.add_argument("--bench")
    u.add_argument("--trace")
    u.add_argument("--pmc", nargs=4, metavar=("FETCH", "WRITE", "CAL_FETCH", "CAL_WRITE"))
    u.add_argument("--step-kernel")
    u.add_argument("--cmd", action="append", default=[])
    v = sub.add_parser("mfma")
    v.add_argument("workload")
    v.add_argument("trace_dir")
    v.add_argument("out")
    v.add_argument("set_dirs", nargs=len(MFMA_SETS))
    v.add_argument("--cmd", action="append", default=[])
    a = ap.parse_args()
    if a.what == "mfma":
        mfma(a.workload, a.trace_dir, a.set_dirs, a.out, a.cmd)
        return
    if a.what == "summary":
        summary(a.workload, a.out, a.bench, a.trace, a.pmc, a.step_kernel, a.cmd)
        return
    if a.what == "stats":
        stats(a.workload, a.trace_dir, a.out, a.cmd)
    else:
        r = traffic(a.workload, a.fetch_dir, a.write_dir, a.cal_fetch, a.cal_write,
                    a.step_kernel, a.cmd, a.md)
        print(json.dumps({"step_bytes": r["step_bytes"], "steps": r["steps"]}))


if __name__ == "__main__":
    main()
