"""Summaries of rocprofv3 output for the profiles/ folder.

Reads the CSV files rocprofv3 writes (``--kernel-trace --stats`` and ``--pmc``
runs of bench.py) and writes short Markdown summaries plus the per-launch HBM
traffic that bench.py reports as ``roofline.traffic`` (profiles/traffic.json,
keyed by workload, dtype and pass, stamped with the kernel source digest).

HBM bytes come from the L2-to-memory request counters, one pass for reads and
one for writes:
    read bytes  = 128 * (TCC_EA0_RDREQ - TCC_EA0_RDREQ_32B) + 32 * TCC_EA0_RDREQ_32B
    write bytes =  64 * TCC_EA0_WRREQ_64B + 32 * (TCC_EA0_WRREQ - TCC_EA0_WRREQ_64B)
On MI355X every non-32-byte read request moves one 128-byte line: a plain
device copy of S bytes reads exactly S / 128 requests (``bench.py
--calibrate-copy``), and TCC_BUBBLE, the documented 128-byte-request counter,
reads zero for these kernels, which is why rocprofv3's FETCH_SIZE (which
prices such a request at 64 bytes) reads half of the copy's bytes.  The
summary states the copy's reading next to the kernels'.

Usage (on the host, after copying the rocprofv3 output back):
    python -m paper_2607_21271_amd.profsum <dir> <workload> <dtype>
with <dir> holding kt/ (kernel trace), rd/ and wr/ (counter passes), copy_rd/
and copy_wr/ (the copy's counter passes) and pipe1/ pipe2/ (SQ counters).
"""
from __future__ import annotations

import collections
import csv
import glob
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROFILES = os.path.join(ROOT, "profiles")


def _csv(d, suffix):
    f = sorted(glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True))
    if not f:
        raise FileNotFoundError("no *%s under %s" % (suffix, d))
    return list(csv.DictReader(open(f[0])))


def kernel_stats(d):
    """[(name, calls, avg_us, min_us, max_us, total_ns)] from a kernel-trace run."""
    out = []
    for r in _csv(d, "kernel_stats.csv"):
        out.append((r["Name"], int(r["Calls"]), float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
                    float(r["MaxNs"]) / 1e3, float(r["TotalDurationNs"])))
    return out


def counters(d):
    """{kernel: {counter: median over dispatches}} from a --pmc run."""
    per = collections.defaultdict(float)
    names = {}
    for r in _csv(d, "counter_collection.csv"):
        di = int(r["Dispatch_Id"])
        per[(di, r["Counter_Name"])] += float(r["Counter_Value"])
        names[di] = r["Kernel_Name"]
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    for (di, c), v in per.items():
        vals[names[di]][c].append(v)
    return {k: {c: sorted(v)[len(v) // 2] for c, v in cs.items()} for k, cs in vals.items()}


def read_bytes(c):
    r32 = c.get("TCC_EA0_RDREQ_32B_sum", 0.0)
    return 128.0 * (c.get("TCC_EA0_RDREQ_sum", 0.0) - r32) + 32.0 * r32


def write_bytes(c):
    w64 = c.get("TCC_EA0_WRREQ_64B_sum", 0.0)
    return 64.0 * w64 + 32.0 * (c.get("TCC_EA0_WRREQ_sum", 0.0) - w64)


def short(name):
    return name.split("(")[0].replace("void ", "").replace("eqk::", "")


def passes_of(name, fused):
    """Entry points (bench.py pass names) whose launches include this kernel.
    With a single-pass plan the split reduction serves both the weight-gradient
    pass and the whole backward."""
    if "wspec" in name:
        return ["wspec"]
    if "bwd_fused" in name:
        return ["bwd"]
    if "wgrad_reduce" in name:
        return ["dw", "bwd"] if fused else ["dw"]
    if "wgrad" in name or "spec_rows" in name:
        return ["dw"]
    if "gemm_kernel" in name or "gemm_big_kernel" in name:
        targs = name.split("<")[1].split(">")[0].split(",")
        return ["dx"] if targs[2].strip() == "true" else ["fwd"]
    return []


def pass_of(name, fused=False):
    ps = passes_of(name, fused)
    return "/".join(ps) if ps else None


def summarize(d, workload, dt, digest, commands, layer=None):
    """Write the kernel-trace, traffic and pipe summaries of one workload
    (a layer of synth.LAYERS, or the one given)."""
    sys.path.insert(0, ROOT)
    import synth
    from paper_2607_21271_amd import roofline as rf
    L = layer if layer is not None else synth.LAYERS[workload]
    from paper_2607_21271_amd import _lib
    fused = bool(_lib.eqlinear_backward_is_fused(L.N, L.T, L.Cin, L.Cout,
                                                 _lib.EQL_F16 if dt == "f16" else _lib.EQL_F32))
    tag = "%s_%s" % (workload, dt)
    PASSES = ("wspec", "fwd", "dx", "dw") + (("bwd",) if fused else ())
    head = "Layer: T=%d, Cin=%d -> Cout=%d, N=%d, %s%s." % (L.T, L.Cin, L.Cout, L.N, dt,
                                                           ", with bias" if L.bias else "")
    # kernel trace
    st = kernel_stats(os.path.join(d, "kt"))
    tot = sum(r[5] for r in st)
    per = collections.defaultdict(float)
    lines = ["# Kernel trace: %s, %s" % (workload, dt), "", head, "", "Command (MI355X, rocprofv3 from ROCm 7.2):",
             "", "```", commands["kt"], "```", "", "Kernel source digest: `%s`" % digest, "",
             "| kernel | pass | calls | avg µs | min µs | max µs | share of GPU time |",
             "|---|---|---|---|---|---|---|"]
    for name, calls, avg, mn, mx, total in st:
        ps = passes_of(name, fused)
        lines.append("| `%s` | %s | %d | %.2f | %.2f | %.2f | %.1f%% |" % (
            short(name), "/".join(ps) or "(setup)", calls, avg, mn, mx, 100 * total / tot))
        for p in ps:
            per[p] += avg
    lines += ["", "Per pass (sum of its kernels' averages): " +
              ", ".join("%s %.2f µs" % (p, per[p]) for p in PASSES if p in per), ""]
    if fused:
        lines += ["The step runs the whole backward as one pass (`bwd`: the single-pass kernel and "
                  "the split reduction); the `dx` and `dw` passes are timed on their own entry "
                  "points for comparison.", ""]
    open(os.path.join(PROFILES, "%s_kernel_trace.md" % tag), "w").write("\n".join(lines))
    # traffic
    rd, wr = counters(os.path.join(d, "rd")), counters(os.path.join(d, "wr"))
    crd, cwr = counters(os.path.join(d, "copy_rd")), counters(os.path.join(d, "copy_wr"))
    ck = [k for k in crd if "copy" in k.lower()][0]
    copy_bytes = 256 << 20
    alg = {p: rf.pass_bytes(p, L.N, L.T, L.Cin, L.Cout, dt, L.bias) for p in PASSES}
    lines = ["# HBM traffic per launch: %s, %s" % (workload, dt), "", head, "",
             "Two counter passes per program (reads, then writes), and the same two on a plain "
             "256 MiB device copy:", "", "```", commands["rd"], commands["wr"], commands["copy_rd"],
             commands["copy_wr"], "```", "",
             "read bytes = 128 x (TCC_EA0_RDREQ - TCC_EA0_RDREQ_32B) + 32 x TCC_EA0_RDREQ_32B; "
             "write bytes = 64 x TCC_EA0_WRREQ_64B + 32 x (TCC_EA0_WRREQ - TCC_EA0_WRREQ_64B).  "
             "The copy (`%s`, %d bytes each way) reads %.0f requests (%.4f x its bytes / 128) and "
             "writes %.0f bytes by these formulas; TCC_BUBBLE reads %.0f." % (
                 short(ck), copy_bytes, crd[ck].get("TCC_EA0_RDREQ_sum", 0),
                 crd[ck].get("TCC_EA0_RDREQ_sum", 0) * 128 / copy_bytes, write_bytes(cwr[ck]),
                 crd[ck].get("TCC_BUBBLE_sum", 0)), "",
             "Kernel source digest: `%s`" % digest, "",
             "| kernel | pass | TCC_EA0_RDREQ | TCC_EA0_RDREQ_32B | TCC_BUBBLE | TCC_EA0_WRREQ | "
             "TCC_EA0_WRREQ_64B | read MB | write MB |", "|---|---|---|---|---|---|---|---|---|"]
    ppass = collections.defaultdict(lambda: [0.0, 0.0])
    for k in rd:
        ps = passes_of(k, fused)
        if not ps:
            continue
        a, b = rd[k], wr.get(k, {})
        rb, wb = read_bytes(a), write_bytes(b)
        for p in ps:
            ppass[p][0] += rb
            ppass[p][1] += wb
        lines.append("| `%s` | %s | %.0f | %.0f | %.0f | %.0f | %.0f | %.2f | %.2f |" % (
            short(k), "/".join(ps), a.get("TCC_EA0_RDREQ_sum", 0), a.get("TCC_EA0_RDREQ_32B_sum", 0),
            a.get("TCC_BUBBLE_sum", 0), b.get("TCC_EA0_WRREQ_sum", 0), b.get("TCC_EA0_WRREQ_64B_sum", 0),
            rb / 1e6, wb / 1e6))
    lines += ["", "| pass | HBM bytes per launch (read + write) | algorithmic bytes | ratio |",
              "|---|---|---|---|"]
    tpath = os.path.join(PROFILES, "traffic.json")
    traffic = json.load(open(tpath)) if os.path.exists(tpath) else {}
    for ps in PASSES:
        if ps not in ppass:
            continue
        rb, wb = ppass[ps]
        lines.append("| %s | %.2f MB (%.2f + %.2f) | %.2f MB | %.2f |" % (
            ps, (rb + wb) / 1e6, rb / 1e6, wb / 1e6, alg[ps] / 1e6, (rb + wb) / alg[ps]))
        traffic["%s/%s/%s" % (workload, dt, ps)] = {
            "hbm_bytes_per_launch": int(rb + wb), "read_bytes": int(rb), "write_bytes": int(wb),
            "source_digest": digest}
    lines.append("")
    open(os.path.join(PROFILES, "%s_hbm_traffic.md" % tag), "w").write("\n".join(lines))
    json.dump(traffic, open(tpath, "w"), indent=1, sort_keys=True)
    # pipe counters
    if os.path.isdir(os.path.join(d, "pipe1")):
        p1, p2 = counters(os.path.join(d, "pipe1")), counters(os.path.join(d, "pipe2"))
        lines = ["# Pipe utilisation per kernel: %s, %s" % (workload, dt), "", head, "",
                 "Two SQ counter passes:", "", "```", commands["pipe1"], commands["pipe2"], "```", "",
                 "Kernel source digest: `%s`" % digest, "",
                 "`GRBM_GUI_ACTIVE` is summed over the 8 XCDs, so a kernel lasts GRBM_GUI_ACTIVE / 8 "
                 "cycles at 2.4 GHz (counter runs are slower than the trace for small kernels).  MFMA "
                 "utilisation = `SQ_VALU_MFMA_BUSY_CYCLES` / (cycles x 1024 SIMDs); VALU issue = "
                 "`SQ_INSTS_VALU` x 4 / (cycles x 1024); LDS bytes per CU and clock assume 16 bytes per "
                 "lane per LDS instruction (an upper bound).", "",
                 "| kernel | pass | cycles µs | MFMA util | VALU issue | LDS B/CU/clk (max) | "
                 "LDS bank conflict / active | waves |", "|---|---|---|---|---|---|---|---|"]
        for k in p1:
            ps = pass_of(k, fused)
            if not ps:
                continue
            a, b = p1[k], p2.get(k, {})
            t = a["GRBM_GUI_ACTIVE"] / 8
            simd = t * 1024
            lines.append("| `%s` | %s | %.1f | %.1f%% | %.1f%% | %.0f | %.2f | %d |" % (
                short(k), ps, t / 2400, 100 * a.get("SQ_VALU_MFMA_BUSY_CYCLES", 0) / simd,
                100 * a.get("SQ_INSTS_VALU", 0) * 4 / simd, a.get("SQ_INSTS_LDS", 0) * 1024 / 256 / t,
                b.get("SQ_LDS_BANK_CONFLICT", 0) / max(1, b.get("SQ_LDS_IDX_ACTIVE", 1)),
                b.get("SQ_WAVES", 0)))
        lines.append("")
        open(os.path.join(PROFILES, "%s_pipe_counters.md" % tag), "w").write("\n".join(lines))


def commands_for(workload, dt):
    """The rocprofv3 commands whose output summarize() reads, with <out> for
    the output folder."""
    run = ("cd /tmp && export TMPDIR=/tmp && timeout -s KILL 120 rocprofv3 %s --output-format csv "
           "-d <out>/%s -o run -- python3 /root/repo/bench.py %s")
    wl = "--workload %s --dtype %s --no-cpu-baseline --steps 3 --warmup 1 --rotate 1" % (workload, dt)
    pipe1 = ("SQ_BUSY_CU_CYCLES SQ_VALU_MFMA_BUSY_CYCLES SQ_ACTIVE_INST_VALU SQ_ACTIVE_INST_LDS "
             "SQ_INSTS_MFMA SQ_INSTS_VALU SQ_INSTS_LDS GRBM_GUI_ACTIVE")
    pipe2 = "SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE SQ_WAVES GRBM_GUI_ACTIVE"
    return {
        "kt": "cd /tmp && export TMPDIR=/tmp && timeout -k 10 180 rocprofv3 --kernel-trace --stats "
              "--output-format csv -d <out>/kt -o run -- python3 /root/repo/bench.py --workload %s "
              "--dtype %s --no-cpu-baseline --steps 20 --warmup 5" % (workload, dt),
        "rd": run % ("--pmc TCC_EA0_RDREQ_sum TCC_EA0_RDREQ_32B_sum TCC_BUBBLE_sum", "rd", wl),
        "wr": run % ("--pmc TCC_EA0_WRREQ_sum TCC_EA0_WRREQ_64B_sum", "wr", wl),
        "copy_rd": run % ("--pmc TCC_EA0_RDREQ_sum TCC_EA0_RDREQ_32B_sum TCC_BUBBLE_sum", "copy_rd",
                          "--calibrate-copy 256"),
        "copy_wr": run % ("--pmc TCC_EA0_WRREQ_sum TCC_EA0_WRREQ_64B_sum", "copy_wr", "--calibrate-copy 256"),
        "pipe1": run % ("--pmc " + pipe1, "pipe1", wl),
        "pipe2": run % ("--pmc " + pipe2, "pipe2", wl),
    }


def main(argv):
    if argv[1] == "--commands":
        # shell lines for a GPU run: python -m ...profsum --commands <workload> <dtype> <out>
        for k, c in commands_for(argv[2], argv[3]).items():
            print(c.replace("<out>", argv[4]) + " > %s/%s.log 2>&1" % (argv[4], k))
        return None
    d, workload, dt = argv[1], argv[2], argv[3]
    sys.path.insert(0, ROOT)
    import importlib.util
    spec = importlib.util.spec_from_file_location("bench", os.path.join(ROOT, "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    digest = bench.source_digest()
    commands = {k: c.replace("<out>", d.rstrip("/")) + " > %s/%s.log 2>&1" % (d.rstrip("/"), k)
                for k, c in commands_for(workload, dt).items()}
    summarize(d, workload, dt, digest, commands, layer=bench.extra_layers().get(workload))
    return commands


if __name__ == "__main__":
    main(sys.argv)
