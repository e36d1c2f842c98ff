#!/usr/bin/env python3
"""Training-step throughput of the Flash EQ-Linear layer on one MI355X.

One step = the whole hot path for one batch: weight spectrum, forward (rDFT ->
per-bin MFMA GEMMs -> irDFT + bias), input gradient and weight gradient, all
through the C ABI of libeqlinear.so.  Default workload: the EQ-ViT-B MLP
up-projection, T = 8, Cin = 96 -> Cout = 384 per group element, N = 64*197 =
12608 tokens, fp16 storage; packed-fp16 forward transforms of x and dy, fp32
weight spectrum, accumulation, inverse transforms and bias.

Inputs are seeded synthetic tensors already resident in HBM.  ``--rotate``
input sets (default 4, about 0.8 GB for the default workload) are used in
turn so that no step finds its operands in the 256 MB MALL or in L2.

Prints one JSON line.  ``roofline`` is for the entry point with the largest
average duration, timed live with HIP events on the stream the kernels run
on; ``cpu_baseline`` times the fp64 oracle on the host cores on a sample of
rows of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "fwd+bwd tokens/s + MFMA util % at T=8, 96->384 ch, fp16 (EQ-ViT-B MLP shape)"
PROFILES = os.path.join(ROOT, "profiles")


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=None, help="layer name from synth.LAYERS or extra_layers()")
    ap.add_argument("--dtype", default=None, choices=["f32", "f16", "bf16"])
    ap.add_argument("--rotate", type=int, default=4, help="input sets used in turn")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-rows", type=int, default=0,
                    help="rows of the oracle sample (0: sized to about 20 s of host work)")
    ap.add_argument("--all", action="store_true",
                    help="also print the full record of every other workload and dtype (one JSON "
                         "line each on stderr)")
    ap.add_argument("--headline-only", action="store_true",
                    help="skip the other workloads (by default each is timed with up to 30 steps "
                         "and summarised under other_workloads in the JSON line)")
    ap.add_argument("--tables", action="store_true",
                    help="only rerun the paper's operator benchmark (Sec. 4.1, Tables 1-2): T=4, "
                         "32768 rows, c = 16..2048, fp32 and fp16; one JSON line per (dtype, c)")
    ap.add_argument("--tables-c", default="16,32,64,128,256,512,1024,2048",
                    help="per-group widths of --tables")
    ap.add_argument("--tables-runs", type=int, default=200, help="timed runs per measurement")
    ap.add_argument("--blocks", action="store_true",
                    help="only time drop-in equivariant ViT encoder blocks (Sec. 4.2; random "
                         "weights): this library's layer vs the naive unrolled layer vs a dense "
                         "ViT block; one JSON line per (model, dtype, linear)")
    ap.add_argument("--dihedral", action="store_true",
                    help="only time the layer over the dihedral group D_T (rotations and "
                         "reflections, Sec. 5) on the C_T kernels against the naive dense layer; "
                         "one JSON line per (shape, dtype)")
    ap.add_argument("--gconv", action="store_true",
                    help="only time the rotation-equivariant group convolution (Sec. 5) on the C_T "
                         "kernels against the naive dense convolution; one JSON line per (shape, dtype)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MiB",
                    help="only run a plain device copy of this many MiB, 5 times (reference "
                         "kernel for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE to bytes)")
    return ap.parse_args()


def calibrate_copy(mib):
    """A plain copy of known size: the counters it produces turn FETCH_SIZE and
    WRITE_SIZE readings of the layer's kernels into HBM bytes."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes": n * 4, "launches": 5}), flush=True)


def source_digest() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2607_21271_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def stored_traffic(workload, dtype, kernel_key, digest):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it was
    taken on the current kernel sources; else None."""
    path = os.path.join(PROFILES, "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        data = json.load(f)
    rec = data.get("%s/%s/%s" % (workload, dtype, kernel_key))
    if not rec or rec.get("source_digest") != digest:
        return None
    return rec.get("hbm_bytes_per_launch")


class Workload:
    def __init__(self, layer, dt, rotate):
        import numpy as np
        import torch

        import synth
        from paper_2607_21271_amd import ops
        self.layer, self.dt, self.ops = layer, dt, ops
        tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[dt]
        l = layer
        inp = synth.draw_layer(l).rounded(dt)
        self.inp = inp
        # bf16 values arrive held in float32 and convert exactly
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(tdt)
        self.w = dev(inp.w)
        self.b = dev(inp.b) if inp.b is not None else None
        x0, dy0 = dev(inp.x), dev(inp.dy)
        self.sets = []
        for r in range(rotate):
            # distinct buffers per set; contents of later sets are permuted copies
            x = x0 if r == 0 else torch.roll(x0, r, dims=0).contiguous()
            dy = dy0 if r == 0 else torch.roll(dy0, r, dims=0).contiguous()
            y = torch.empty(l.N, l.Cout, l.T, dtype=tdt, device="cuda")
            dx = torch.empty(l.N, l.Cin, l.T, dtype=tdt, device="cuda")
            self.sets.append((x, dy, y, dx))
        self.wspec = torch.empty(ops._lib.eqlinear_weight_spectrum_bytes(l.T, l.Cin, l.Cout,
                                                                         ops._DT[tdt]),
                                 dtype=torch.uint8, device="cuda")
        self.dw = torch.empty(l.T, l.Cout, l.Cin, dtype=tdt, device="cuda")
        self.db = torch.empty(l.Cout, dtype=tdt, device="cuda") if l.bias else None
        nws = max(ops.workspace_bytes(l.N, l.T, l.Cin, l.Cout, tdt),
                  ops.backward_workspace_bytes(l.N, l.T, l.Cin, l.Cout, tdt))
        self.fused = ops.backward_is_fused(l.N, l.T, l.Cin, l.Cout, tdt)
        self.ws = torch.empty(max(nws, 1), dtype=torch.uint8, device="cuda")
        self.stream = torch.cuda.current_stream()

    def step(self, i, stream=None):
        """One training step of the layer on input set i: weight spectrum,
        forward, then input, weight and bias gradients in one call of the
        whole-backward entry point (one fused pass where the library plans
        one, else the input- and weight-gradient kernels in turn)."""
        l, ops = self.layer, self.ops
        st = stream if stream is not None else self.stream
        x, dy, y, dx = self.sets[i % len(self.sets)]
        ops.weight_spectrum(self.w, out=self.wspec, stream=st)
        ops.forward(x, self.wspec, self.b, l.T, l.Cin, l.Cout, out=y, stream=st)
        ops.backward(x, dy, self.wspec, l.T, l.Cin, l.Cout, with_bias=l.bias, dx=dx, dw=self.dw,
                     db=self.db, workspace=self.ws, stream=st)

    def _graph(self, fn):
        import torch
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn(torch.cuda.current_stream())
        return g

    def run_graph(self, steps, warmup, block=10):
        """Whole-step time with each input set's step (the same launches as the
        eager path) captured once in a HIP graph and replayed.  Exactly
        ``steps`` steps are timed, bracketed by device synchronisation and by
        HIP events on the replay stream at their two ends only (an event
        recorded between replays costs the GPU about 11 us at the headline, so
        none sits inside the timed run); their mean is the reported step time.
        A second run of ``steps`` replays with an event after every ``block``
        replays gives the distribution of block means (the event cost spread
        over ``block`` steps)."""
        import torch
        graphs = [self._graph(lambda st, r=r: self.step(r, stream=st))
                  for r in range(len(self.sets))]
        for i in range(warmup):
            graphs[i % len(graphs)].replay()
        torch.cuda.synchronize()
        st = torch.cuda.current_stream()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(st)
        for i in range(steps):
            graphs[(warmup + i) % len(graphs)].replay()
        e1.record(st)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        ev_mean = e0.elapsed_time(e1) * 1e3 / steps  # us
        block = max(1, min(block, steps))
        nb = max(1, steps // block)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(nb + 1)]
        ev[0].record(st)
        for b in range(nb):
            for i in range(block):
                graphs[(b * block + i) % len(graphs)].replay()
            ev[b + 1].record(st)
        torch.cuda.synchronize()
        per = [ev[b].elapsed_time(ev[b + 1]) * 1e3 / block for b in range(nb)]  # us per step
        del graphs
        return (t1 - t0) / steps, ev_mean, per

    def run_passes(self, reps, settle_s=0.05):
        """Average duration of one launch of each entry point: per pass, one HIP
        graph holds one call per input set back to back (no host time between
        the launches) and is replayed until ``reps`` calls have run (after
        untimed replays for at least ``settle_s`` seconds); HIP events on the
        replay stream bracket all of them."""
        import torch
        l, ops = self.layer, self.ops
        R = len(self.sets)

        def launch(kind, r, st):
            x, dy, y, dx = self.sets[r]
            if kind == "wspec":
                ops.weight_spectrum(self.w, out=self.wspec, stream=st)
            elif kind == "fwd":
                ops.forward(x, self.wspec, self.b, l.T, l.Cin, l.Cout, out=y, stream=st)
            elif kind == "bwd":
                ops.backward(x, dy, self.wspec, l.T, l.Cin, l.Cout, with_bias=l.bias, dx=dx,
                             dw=self.dw, db=self.db, workspace=self.ws, stream=st)
            elif kind == "dx":
                ops.backward_input(dy, self.wspec, l.T, l.Cin, l.Cout, out=dx, stream=st)
            else:
                ops.backward_weight(x, dy, l.T, l.Cin, l.Cout, with_bias=l.bias, dw=self.dw,
                                    db=self.db, workspace=self.ws, stream=st)

        ops.weight_spectrum(self.w, out=self.wspec)
        out = {}
        for kind in ("wspec", "fwd", "bwd", "dx", "dw"):
            g = self._graph(lambda st: [launch(kind, r, st) for r in range(R)])
            n = max(1, reps // R)
            # untimed replays of the same launches for at least settle_s, so
            # the GPU clocks have left their idle state when timing starts
            t_end = time.perf_counter() + settle_s
            while True:
                for _ in range(n):
                    g.replay()
                torch.cuda.synchronize()
                if time.perf_counter() >= t_end:
                    break
            st = torch.cuda.current_stream()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(st)
            for _ in range(n):
                g.replay()
            e1.record(st)
            torch.cuda.synchronize()
            out[kind] = e0.elapsed_time(e1) * 1e3 / (n * R)
            del g
        return out


def _pct(v, q):
    import numpy as np
    return float(np.percentile(np.asarray(v), q))


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(layer, dt, inp, rows_req):
    """Time the fp64 oracle (fwd, dx, dw each timed) on the host cores: the first
    rows of the same draw when the whole workload would take longer than
    about 20 s, else the whole workload repeated until about 20 s have passed
    (sized from a calibration slice of about 2 G multiply-adds, large enough
    that thread start-up does not dominate it)."""
    threads = len(os.sched_getaffinity(0))
    os.environ.setdefault("OMP_NUM_THREADS", str(threads))
    import oracle
    orc = oracle.oracle()
    l = layer
    macs_per_row = 3 * l.T * l.T * l.Cin * l.Cout
    if rows_req <= 0:
        # calibrate on a slice, then size the sample to about 20 s
        n0 = max(8, min(l.N, int(2e9 // macs_per_row)))
        t0 = time.perf_counter()
        orc.forward(inp.x[:n0], inp.w, inp.b)
        orc.backward_input(inp.dy[:n0], inp.w)
        orc.backward_weight(inp.x[:n0], inp.dy[:n0], with_bias=inp.b is not None)
        rate = n0 / max(time.perf_counter() - t0, 1e-6)
        rows_req = int(rate * 20.0)
    n = max(1, min(l.N, rows_req))
    reps = max(1, rows_req // n) if n == l.N else 1
    xs, dys = inp.x[:n], inp.dy[:n]
    per = {"fwd": 0.0, "dx": 0.0, "dw": 0.0}
    for _ in range(reps):
        t0 = time.perf_counter()
        orc.forward(xs, inp.w, inp.b)
        t1 = time.perf_counter()
        orc.backward_input(dys, inp.w)
        t2 = time.perf_counter()
        orc.backward_weight(xs, dys, with_bias=inp.b is not None)
        t3 = time.perf_counter()
        per["fwd"] += t1 - t0
        per["dx"] += t2 - t1
        per["dw"] += t3 - t2
    t = sum(per.values())
    what = ("first %d of %d rows" % (n, l.N)) if n < l.N else ("all %d rows, %d times" % (n, reps))
    return {"value": n * reps / t, "unit": "tokens/s", "cores": int(os.environ["OMP_NUM_THREADS"]),
            "kind": "oracle",
            "sample": "%s of the same seeded %s draw, fwd + dx + dw in fp64 (direct circular-"
                      "convolution sums), %.1f s" % (what, dt, t),
            "seconds": t, "cpu_model": cpu_model(),
            "pass_tokens_per_s": {k: round(n * reps / v, 1) for k, v in per.items()}}


KERNELS = {"wspec": "eqlinear_weight_spectrum (eql_wspec_kernel)",
           "fwd": "eqlinear_forward (eql_gemm_kernel, forward)",
           "dx": "eqlinear_backward_input (eql_gemm_kernel, input gradient)",
           "dw": "eqlinear_backward_weight (eql_wgrad_kernel + eql_wgrad_reduce_kernel)",
           "bwd": "eqlinear_backward, single pass (eql_bwd_fused_kernel + eql_wgrad_reduce_kernel)"}


def kernel_name(kind, l, dt):
    """The kernels behind one pass, for the JSON line: the library's size rules
    for its large-tile kernels (T = 2 or 4; forward / input gradient from 256
    channels each way with the contraction channels a multiple of 32, weight
    gradient from 768 (fp16, fp32) / 512 (bf16) channels each way)."""
    big = l.T in (2, 4)
    lo = min(l.Cin, l.Cout)
    if kind == "fwd" and big and lo >= 256 and l.Cin % 32 == 0:
        return "eqlinear_forward (eql_gemm_big_kernel, forward)"
    if kind == "dx" and big and lo >= 256 and l.Cout % 32 == 0:
        return "eqlinear_backward_input (eql_gemm_big_kernel, input gradient)"
    if kind == "dw" and big and lo >= (512 if dt == "bf16" else 768):
        return "eqlinear_backward_weight (eql_spec_rows_kernel x 2 + eql_wgrad_big_kernel + eql_wgrad_reduce_kernel)"
    return KERNELS[kind]


def measure(layer, dt, args, digest, with_cpu):
    import torch

    from paper_2607_21271_amd import roofline as rf
    l = layer
    wl = Workload(l, dt, max(1, args.rotate))
    # the passes: back-to-back launches of each entry point (run first, which
    # also brings the GPU out of its idle clocks before the timed steps); the
    # step: HIP-graph replays of whole steps (reported step time and its
    # distribution)
    per = wl.run_passes(max(args.steps, 4 * max(1, args.rotate)))
    sec, ev_mean_us, per_step = wl.run_graph(args.steps, args.warmup)
    N = l.N
    flops = 3 * rf.pass_flops(N, l.T, l.Cin, l.Cout)
    dense = 3 * rf.dense_equiv_flops(N, l.T, l.Cin, l.Cout)
    nbytes = {k: rf.pass_bytes(k, N, l.T, l.Cin, l.Cout, dt, l.bias)
              for k in ("wspec", "fwd", "bwd", "dx", "dw")}
    # the entry points the step runs: with a fused plan the whole backward is
    # one pass (plus its reduction), else its input- and weight-gradient passes
    step_passes = ("wspec", "fwd", "bwd") if wl.fused else ("wspec", "fwd", "dx", "dw")
    dom = max(step_passes[1:], key=lambda k: per[k])
    dom_flops = rf.pass_flops(N, l.T, l.Cin, l.Cout) * (2 if dom == "bwd" else 1)
    bound = "hbm" if nbytes[dom] / (rf.PEAK_HBM_GBS * 1e9) >= dom_flops / (
        rf.PEAK_MFMA_TFLOPS[dt] * 1e12) else "mfma"
    t_dom = per[dom] * 1e-6
    if bound == "hbm":
        achieved = nbytes[dom] / t_dom / 1e9
        peak, unit = rf.PEAK_HBM_GBS, "GB/s"
    else:
        achieved = dom_flops / t_dom / 1e12
        peak, unit = rf.PEAK_MFMA_TFLOPS[dt], "TFLOP/s"
    traffic = stored_traffic(l.name, dt, dom, digest)
    roof = {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "traffic": traffic, "kernel": kernel_name(dom, l, dt),
            "algorithmic_bytes_per_launch": nbytes[dom], "avg_launch_us": round(per[dom], 2)}
    roof_all = sum(rf.roofline_time_s(k, N, l.T, l.Cin, l.Cout, dt, l.bias) for k in step_passes)
    rec = {
        "metric": METRIC, "value": round(N / sec, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(sec * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dt,
        "data": "synthetic: seeded N(0,1) activations and gradients, N(0,1/(T*Cin)) weights, "
                "resident in HBM, %d input sets in turn" % max(1, args.rotate),
        "config": {"workload": "%s: T=%d Cin=%d Cout=%d N=%d %s, weight spectrum + forward + "
                               "input gradient + weight gradient%s" % (
                                   l.name, l.T, l.Cin, l.Cout, N, dt, " (+bias)" if l.bias else ""),
                   "T": l.T, "Cin": l.Cin, "Cout": l.Cout, "tokens": N, "bias": l.bias},
        "mfma_util_pct": round(100 * flops / sec / (rf.PEAK_MFMA_TFLOPS[dt] * 1e12), 2),
        "tflops_actual": round(flops / sec / 1e12, 2),
        "tflops_dense_equiv": round(dense / sec / 1e12, 2),
        "step_us": {"mean": round(sec * 1e6, 2), "event_mean": round(ev_mean_us, 2),
                    "median": round(_pct(per_step, 50), 2),
                    "p10": round(_pct(per_step, 10), 2), "p90": round(_pct(per_step, 90), 2),
                    "distribution": "means of %d-step blocks" % max(1, min(10, args.steps))},
        "backward": "single pass (eqlinear_backward: eql_bwd_fused_kernel + reduction)" if wl.fused
                    else "two passes (eqlinear_backward: input-gradient kernel, then weight-gradient "
                         "kernel + reduction)",
        "timing": "step = one replay of a HIP graph holding one input set's launches (weight "
                  "spectrum, forward, whole backward); ms_per_step is the mean "
                  "over the timed replays (host clock around all of them, HIP events only at "
                  "their two ends: event_mean), step_us median/p10/p90 the distribution of "
                  "10-step block means from a second run; pass_us = average launch "
                  "of each entry point, timed with HIP events around graph replays of "
                  "back-to-back launches on the replay stream",
        "pass_us": {k: round(v, 2) for k, v in per.items()},
        "pass_hbm_gbs": {k: round(nbytes[k] / (per[k] * 1e-6) / 1e9, 1) for k in per},
        "roofline": roof,
        "roofline_step_us": round(roof_all * 1e6, 2),
        "roofline_step_frac": round(roof_all / sec, 4),
        "source_digest": digest,
        "device": torch.cuda.get_device_name(0),
    }
    if with_cpu:
        rec["cpu_baseline"] = cpu_baseline(l, dt, wl.inp, args.cpu_sample_rows)
    del wl
    torch.cuda.empty_cache()
    return rec


def _time_fn(fn, runs, warmup=10):
    """Mean and median of ``runs`` calls of fn, each bracketed by HIP events on
    the current stream (host launch time between calls is not counted)."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * runs)]
    for i in range(runs):
        ev[2 * i].record(st)
        fn()
        ev[2 * i + 1].record(st)
    torch.cuda.synchronize()
    t = sorted(ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(runs))
    return {"mean_ms": round(sum(t) / runs, 4), "median_ms": round(t[runs // 2], 4)}


def run_tables(args):
    """The paper's operator benchmark (Sec. 4.1, Tables 1-2) on this GPU: input
    [B*N = 32768 rows, c, T = 4], output width D = C = 4c.  Three layers:
    Standard Linear (torch F.linear, a dense C -> C weight), Naive EQ-Linear
    (the equivariant weight unrolled into the dense T*c x T*c matrix
    W[o*T+t, c*T+s] = w[(t-s) mod T, o, c], then F.linear; autograd folds the
    dense gradient back onto w) and this library.  Forward = one layer call
    (for this library with the weight spectrum precomputed, which a frozen
    weight allows; its time is reported apart); backward = input, weight and
    bias gradients.  Mean and median of ``--tables-runs`` event-timed runs.
    For c >= 512 sampled rows of y and dx and sampled dw entries are checked
    against the fp64 oracle."""
    import numpy as np
    import torch
    import torch.nn.functional as F

    import synth
    from paper_2607_21271_amd import ops
    from paper_2607_21271_amd import roofline as rf
    T, N = 4, 32768
    runs = args.tables_runs
    for dt in ((args.dtype,) if args.dtype else ("f32", "f16", "bf16")):
        tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[dt]
        for c in [int(v) for v in args.tables_c.split(",")]:
            torch.cuda.empty_cache()
            inp = synth.draw(T, c, c, N, True, 6000 + c).rounded(dt)
            dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda().to(tdt)
            x, w, b, dy = dev(inp.x), dev(inp.w), dev(inp.b), dev(inp.dy)
            rec = {"table": "operator", "dtype": dt, "c": c, "T": T, "rows": N, "runs": runs}
            print("tables: %s c=%d" % (dt, c), file=sys.stderr, flush=True)
            # this library
            wspec = ops.weight_spectrum(w)
            y = torch.empty(N, c, T, dtype=tdt, device="cuda")
            dx = torch.empty_like(x)
            dw = torch.empty_like(w)
            db = torch.empty_like(b)
            ws = torch.empty(max(1, ops.workspace_bytes(N, T, c, c, tdt)), dtype=torch.uint8,
                             device="cuda")
            rec["flash_wspec"] = _time_fn(lambda: ops.weight_spectrum(w, out=wspec), runs)
            rec["flash_fwd"] = _time_fn(lambda: ops.forward(x, wspec, b, T, c, c, out=y), runs)
            rec["flash_bwd"] = _time_fn(lambda: (ops.backward_input(dy, wspec, T, c, c, out=dx),
                                                 ops.backward_weight(x, dy, T, c, c, True, dw=dw, db=db,
                                                                     workspace=ws)), runs)
            if c >= 512:
                import oracle
                orc = oracle.oracle()
                rs = np.random.RandomState(c)
                rows = np.unique(np.concatenate([rs.randint(0, N, 14), [0, N - 1]]))
                torch.cuda.synchronize()
                ry = orc.forward(inp.x[rows], inp.w, inp.b)
                rdx = orc.backward_input(inp.dy[rows], inp.w)
                jj, oo, cc = rs.randint(0, T, 24), rs.randint(0, c, 24), rs.randint(0, c, 24)
                rdw = orc.backward_weight_entries(inp.x, inp.dy, jj, oo, cc)
                err = lambda g, r: float(np.max(np.abs(g - r)) / np.max(np.abs(r)))
                rec["parity_sampled"] = {
                    "y": err(y.double().cpu().numpy()[rows], ry),
                    "dx": err(dx.double().cpu().numpy()[rows], rdx),
                    "dw": err(dw.double().cpu().numpy()[jj, oo, cc], rdw)}
            del wspec, y, dx, ws
            # Standard Linear: dense C -> C
            C = c * T
            xs = x.view(N, C).detach().requires_grad_(True)
            W = (torch.randn(C, C, device="cuda") / C ** 0.5).to(tdt).requires_grad_(True)
            bs = torch.zeros(C, dtype=tdt, device="cuda", requires_grad=True)
            dys = dy.view(N, C)
            with torch.no_grad():
                rec["standard_fwd"] = _time_fn(lambda: F.linear(xs, W, bs), runs)
            ys = F.linear(xs, W, bs)
            rec["standard_bwd"] = _time_fn(
                lambda: torch.autograd.grad(ys, (xs, W, bs), dys, retain_graph=True), runs)
            del ys, W
            # Naive EQ-Linear: unrolled weight, autograd through the unrolling
            t_idx = torch.arange(T, device="cuda")
            lag = (t_idx[:, None] - t_idx[None, :]) % T            # [t, s]
            wn = w.detach().clone().requires_grad_(True)
            bn = b.detach().clone().requires_grad_(True)

            def naive():
                Wd = wn[lag].permute(2, 0, 3, 1).reshape(c * T, c * T)   # [o*T+t, c*T+s]
                return F.linear(xs, Wd, bn.repeat_interleave(T))
            with torch.no_grad():
                rec["naive_fwd"] = _time_fn(naive, runs)
            yn = naive()
            rec["naive_bwd"] = _time_fn(
                lambda: torch.autograd.grad(yn, (xs, wn, bn), dys, retain_graph=True), runs)
            del yn
            fl = rf.pass_flops(N, T, c, c)
            rec["flash_fwd_tflops"] = round(fl / (rec["flash_fwd"]["mean_ms"] * 1e-3) / 1e12, 2)
            rec["flash_bwd_tflops"] = round(2 * fl / (rec["flash_bwd"]["mean_ms"] * 1e-3) / 1e12, 2)
            rec["flash_fwd_hbm_gbs"] = round(rf.pass_bytes("fwd", N, T, c, c, dt, True) /
                                             (rec["flash_fwd"]["mean_ms"] * 1e-3) / 1e9, 1)
            rec["speedup_fwd_vs_standard"] = round(rec["standard_fwd"]["mean_ms"] /
                                                   rec["flash_fwd"]["mean_ms"], 2)
            rec["speedup_bwd_vs_standard"] = round(rec["standard_bwd"]["mean_ms"] /
                                                   rec["flash_bwd"]["mean_ms"], 2)
            print(json.dumps(rec), flush=True)


# ViT scales of the paper's Table 6 (embedding width, heads), run at T = 4 with
# the paper's inference batch of 128 images of 197 tokens (224 / 16 patches and
# a class token).
BLOCK_MODELS = {"vit_s": (480, 6), "vit_b": (768, 12), "vit_l": (1024, 16)}


def run_blocks(args):
    """Per-block latency of EQ-ViT encoder blocks whose four linear layers are
    this library's layer ("flash"), the naive unrolled layer ("naive"), or a
    dense non-equivariant layer of the same widths ("standard"): forward
    (inference, no autograd), the four linear layers' share of it, and forward
    + backward.  Mean of ``--tables-runs`` event-timed runs."""
    import torch

    from paper_2607_21271_amd.blocks import EQViTBlock
    T, B, L = 4, 128, 197
    runs = max(10, args.tables_runs // 4)
    for name, (width, heads) in BLOCK_MODELS.items():
        C = width // T
        for dt in ("f32", "f16"):
            tdt = {"f32": torch.float32, "f16": torch.float16}[dt]
            torch.manual_seed(0)
            x0 = torch.randn(B, L, C, T, device="cuda", dtype=tdt)
            gy = torch.randn_like(x0)
            res = {}
            for lin in ("standard", "naive", "flash"):
                print("blocks: %s %s %s" % (name, dt, lin), file=sys.stderr, flush=True)
                torch.manual_seed(1)
                blk = EQViTBlock(T, C, heads, linear=lin, device="cuda", dtype=tdt)
                with torch.no_grad():
                    fwd = _time_fn(lambda: blk(x0), runs)
                    h = blk.norm1(x0)
                    a = blk.attention(blk.qkv(h))
                    m = torch.nn.functional.gelu(blk.fc1(blk.norm2(x0)))
                    lin_t = _time_fn(lambda: (blk.qkv(h), blk.proj(a), blk.fc1(h), blk.fc2(m)), runs)
                res[lin] = {"fwd": fwd, "linear_fwd": lin_t}
                if dt == "f32":   # training step in fp32 only (torch's fp16 attention backward is not used)
                    x = x0.clone().requires_grad_(True)

                    def train():
                        y = blk(x)
                        y.backward(gy)
                    res[lin]["fwd_bwd"] = _time_fn(train, runs)
                    del x
                del blk
                torch.cuda.empty_cache()
            rec = {"table": "block", "model": name, "dtype": dt, "T": T, "C_per_group": C,
                   "heads": heads, "tokens": B * L, "runs": runs, "results": res,
                   "fwd_speedup_vs_naive": round(res["naive"]["fwd"]["mean_ms"] /
                                                 res["flash"]["fwd"]["mean_ms"], 2),
                   "fwd_speedup_vs_standard": round(res["standard"]["fwd"]["mean_ms"] /
                                                    res["flash"]["fwd"]["mean_ms"], 2),
                   "fwd_bwd_speedup_vs_naive": (round(res["naive"]["fwd_bwd"]["mean_ms"] /
                                                      res["flash"]["fwd_bwd"]["mean_ms"], 2)
                                                if dt == "f32" else None),
                   "linear_share_flash": round(res["flash"]["linear_fwd"]["mean_ms"] /
                                               res["flash"]["fwd"]["mean_ms"], 3),
                   "linear_share_naive": round(res["naive"]["linear_fwd"]["mean_ms"] /
                                               res["naive"]["fwd"]["mean_ms"], 3)}
            print(json.dumps(rec), flush=True)


DIHEDRAL_LAYERS = [("vit_b_mlp_up_d8", 8, 48, 192, 12608), ("swin_s1_d4", 4, 12, 48, 401408)]


def run_dihedral(args):
    """The layer over the dihedral group D_T (rotations and reflections) on the
    C_T kernels, against the naive layer: the dense [Cout*2T, Cin*2T] weight
    M[(o,g),(c,h)] = W[h^-1 g][o][c] applied with F.linear (autograd folds
    its gradient back onto W).  Two shapes whose C_T layer (2Cin -> 2Cout) is
    the EQ-ViT-B MLP up-projection and the Swin stage-1 MLP.  Forward = one
    layer call with the C_T weights and spectrum precomputed (a frozen weight);
    training step = weight expansion, spectrum, forward, whole backward and
    gradient fold (naive: dense weight gather, F.linear forward and backward).
    Mean and median of ``--tables-runs`` event-timed runs."""
    import numpy as np
    import torch
    import torch.nn.functional as F

    from paper_2607_21271_amd import dihedral, ops
    runs = args.tables_runs
    for name, T, Cin, Cout, N in DIHEDRAL_LAYERS:
        G = 2 * T
        # index of h^-1 g for the naive dense weight: (t, m) = r^t s^m at m*T + t
        inv = lambda a: (a // T) * T + ((a % T) if a // T else (T - a % T) % T)
        mul = lambda a, b: ((a // T) ^ (b // T)) * T + (((a % T) - (b % T)) if a // T else
                                                     ((a % T) + (b % T))) % T
        idx = torch.tensor([[mul(inv(h), g) for h in range(G)] for g in range(G)], device="cuda")
        for dt in ("f32", "f16"):
            tdt = {"f32": torch.float32, "f16": torch.float16}[dt]
            torch.cuda.empty_cache()
            print("dihedral: %s %s" % (name, dt), file=sys.stderr, flush=True)
            rs = np.random.RandomState(8100 + T)
            x = torch.from_numpy(rs.standard_normal((N, Cin, G))).to("cuda", tdt)
            W = torch.from_numpy(rs.standard_normal((G, Cout, Cin)) / (G * Cin) ** 0.5).to("cuda", tdt)
            b = torch.from_numpy(0.1 * rs.standard_normal(Cout)).to("cuda", tdt)
            gy = torch.from_numpy(rs.standard_normal((N, Cout, G))).to("cuda", tdt)
            rec = {"table": "dihedral", "layer": name, "group": "D%d" % T, "dtype": dt, "Cin": Cin,
                   "Cout": Cout, "rows": N, "runs": runs,
                   "ct_layer": "T=%d %d->%d" % (T, 2 * Cin, 2 * Cout)}
            w_ct, b_ct = dihedral.expand(W, b)
            wspec = ops.weight_spectrum(w_ct)
            x2 = x.view(N, 2 * Cin, T)
            y2 = torch.empty(N, 2 * Cout, T, dtype=tdt, device="cuda")
            rec["flash_fwd"] = _time_fn(lambda: ops.forward(x2, wspec, b_ct, T, 2 * Cin, 2 * Cout, out=y2), runs)
            xg = x.clone().requires_grad_(True)
            Wg = W.clone().requires_grad_(True)
            bg = b.clone().requires_grad_(True)

            def flash_train():
                dihedral._CACHE.clear()
                y = dihedral.DihedralEQLinearFunction.apply(xg, Wg, bg)
                y.backward(gy)
            rec["flash_train"] = _time_fn(flash_train, runs)

            def dense(Wt):
                return Wt[idx].permute(2, 0, 3, 1).reshape(Cout * G, Cin * G)
            M = dense(W)
            bd = b.repeat_interleave(G)
            xf = x.view(N, Cin * G)
            rec["naive_fwd"] = _time_fn(lambda: F.linear(xf, M, bd), runs)
            xn = x.clone().requires_grad_(True)
            Wn = W.clone().requires_grad_(True)
            bn = b.clone().requires_grad_(True)

            def naive_train():
                y = F.linear(xn.view(N, Cin * G), dense(Wn), bn.repeat_interleave(G))
                y.backward(gy.view(N, Cout * G))
            rec["naive_train"] = _time_fn(naive_train, runs)
            with torch.no_grad():
                yf = ops.forward(x2, wspec, b_ct, T, 2 * Cin, 2 * Cout).view(N, Cout, G).float()
                yn = F.linear(xf, M, bd).view(N, Cout, G).float()
                rec["flash_vs_naive_rel_err"] = float((yf - yn).abs().max() / yn.abs().max())
            rec["fwd_speedup"] = round(rec["naive_fwd"]["mean_ms"] / rec["flash_fwd"]["mean_ms"], 2)
            rec["train_speedup"] = round(rec["naive_train"]["mean_ms"] / rec["flash_train"]["mean_ms"], 2)
            print(json.dumps(rec), flush=True)
            del x, W, b, gy, xg, Wg, bg, xn, Wn, bn, M, w_ct, wspec, x2, y2


GCONV_LAYERS = [("p4_c24_56px", 4, 24, 24, 3, 32, 56), ("p4_c64_28px", 4, 64, 64, 3, 32, 28)]


def run_gconv(args):
    """The rotation-equivariant group convolution (Sec. 5) on the C_T kernels
    (patch gather, C_T layer with k*k*Cin input channels, and for training the
    gradient scatter and weight permutation) against the naive dense form: the
    [Cout*T, Cin*T, k, k] kernel Wd[(o,r),(c,s),a,b] = psi[R^-r (a,b)][(s-r) mod T][o][c]
    applied with torch's conv2d on NCHW features (its autograd folds the
    gradient back onto psi).  Forward = one layer call with the C_T weight and
    spectrum precomputed (a frozen weight), reading the patches straight from
    the features where the channel count allows, else gather + layer call;
    training step = weight permutations (forward and adjoint), spectra,
    forward, backward (input gradient as the adjoint convolution where Cout
    allows).  Mean and median of ``--tables-runs`` runs."""
    import numpy as np
    import torch
    import torch.nn.functional as F

    from paper_2607_21271_amd import gconv, ops
    runs = args.tables_runs
    for name, T, Cin, Cout, k, B, H in GCONV_LAYERS:
        h = k // 2
        # index of psi used by the dense kernel entry (r, s, a, b): offset R^-r (a, b), lag (s - r)
        def rot(n, a, b):
            for _ in range(((n % T) + T) % T * (4 // T if T > 1 else 0)):
                a, b = -b, a
            return a, b
        idx = np.zeros((T, T, k, k), np.int64)
        for r in range(T):
            for s_ in range(T):
                for a in range(-h, h + 1):
                    for b in range(-h, h + 1):
                        ra, rb = rot(-r, a, b)
                        idx[r, s_, a + h, b + h] = ((ra + h) * k + (rb + h)) * T + (s_ - r) % T
        idx_t = torch.from_numpy(idx).cuda()
        for dt in ("f32", "f16", "bf16"):
            tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[dt]
            torch.cuda.empty_cache()
            print("gconv: %s %s" % (name, dt), file=sys.stderr, flush=True)
            rs = np.random.RandomState(8300 + Cin)
            f = torch.from_numpy(rs.standard_normal((B, H, H, Cin, T))).to("cuda", tdt)
            psi = torch.from_numpy(rs.standard_normal((k, k, T, Cout, Cin)) /
                                   np.sqrt(k * k * T * Cin)).to("cuda", tdt)
            bias = torch.from_numpy(0.1 * rs.standard_normal(Cout)).to("cuda", tdt)
            gy = torch.from_numpy(rs.standard_normal((B, H, H, Cout, T))).to("cuda", tdt)
            rec = {"table": "gconv", "layer": name, "T": T, "Cin": Cin, "Cout": Cout, "k": k,
                   "image": [B, H, H], "dtype": dt, "runs": runs,
                   "ct_layer": "T=%d %d->%d over %d rows" % (T, k * k * Cin, Cout, B * H * H)}
            w_ct = gconv.pack_weight(psi)
            wspec = ops.weight_spectrum(w_ct)

            def explicit_fwd():
                xcol = gconv.gather(f, T, k)
                return ops.forward(xcol, wspec, bias, T, k * k * Cin, Cout)
            if gconv.implicit_ok(Cin):
                def flash_fwd():
                    return gconv.forward_implicit(f, wspec, bias, T, Cout, k)
                rec["forward_kind"] = "implicit gather"
                rec["explicit_fwd"] = _time_fn(explicit_fwd, runs)
            else:
                flash_fwd = explicit_fwd
                rec["forward_kind"] = "gather + C_T forward"
            rec["flash_fwd"] = _time_fn(flash_fwd, runs)
            xcol = gconv.gather(f, T, k)
            rec["gather"] = _time_fn(lambda: gconv.gather(f, T, k), runs)
            rec["ct_forward"] = _time_fn(lambda: ops.forward(xcol, wspec, bias, T, k * k * Cin, Cout), runs)
            rec["scatter"] = _time_fn(lambda: gconv.scatter(xcol, B, H, H, T, Cin, k), runs)
            del xcol
            fg = f.clone().requires_grad_(True)
            pg = psi.clone().requires_grad_(True)
            bg = bias.clone().requires_grad_(True)

            def flash_train():
                gconv._CACHE.clear()
                gconv._CACHE_ADJ.clear()
                y = gconv.GroupConv2dFunction.apply(fg, pg, bg)
                y.backward(gy)
            rec["flash_train"] = _time_fn(flash_train, runs)

            def dense(p):
                flat = p.reshape(k * k * T, Cout, Cin)           # [(a, b, lag), o, c]
                g = flat[idx_t]                                   # [r, s, a, b, o, c]
                return g.permute(4, 0, 5, 1, 2, 3).reshape(Cout * T, Cin * T, k, k)
            xn = f.permute(0, 3, 4, 1, 2).reshape(B, Cin * T, H, H).contiguous()
            gyn = gy.permute(0, 3, 4, 1, 2).reshape(B, Cout * T, H, H).contiguous()
            Wd = dense(psi)
            bd = bias.repeat_interleave(T)
            rec["naive_fwd"] = _time_fn(lambda: F.conv2d(xn, Wd, bd, padding=h), runs)
            xr = xn.clone().requires_grad_(True)
            pr = psi.clone().requires_grad_(True)
            br = bias.clone().requires_grad_(True)

            def naive_train():
                y = F.conv2d(xr, dense(pr), br.repeat_interleave(T), padding=h)
                y.backward(gyn)
            rec["naive_train"] = _time_fn(naive_train, runs)
            with torch.no_grad():
                yf = flash_fwd().view(B, H, H, Cout, T).permute(0, 3, 4, 1, 2).reshape(B, Cout * T, H, H).float()
                yn = F.conv2d(xn, Wd, bd, padding=h).float()
                rec["flash_vs_naive_rel_err"] = float((yf - yn).abs().max() / yn.abs().max())
            rec["fwd_speedup"] = round(rec["naive_fwd"]["mean_ms"] / rec["flash_fwd"]["mean_ms"], 2)
            rec["train_speedup"] = round(rec["naive_train"]["mean_ms"] / rec["flash_train"]["mean_ms"], 2)
            print(json.dumps(rec), flush=True)
            del f, psi, bias, gy, fg, pg, bg, xn, gyn, Wd, xr, pr, br, w_ct, wspec


# bf16 runs of the headline and Swin stage-1 shapes, reported beside the rest
EXTRA_DTYPES = {"vit_b_mlp_up": ("bf16",), "swin_s1": ("bf16",)}


def extra_layers():
    """Workloads measured beside the survey's layers (not parity-test shapes:
    the fp64 oracle could not check them whole): the paper's operator
    benchmark at c = 1024 (T = 4, 32,768 rows, Sec. 4.1 Tables 1-2), the
    MFMA-bound regime of the large-tile kernels."""
    import synth
    return {"table_T4_c1024": synth.Layer("table_T4_c1024", 4, 1024, 1024, 32768, True, 6000, ("f16", "bf16"),
                                          "operator benchmark row, c = 1024 per group element")}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the layer's hot path runs on a single MI355X "
              "and no multi-GPU path is built (requested --gpus %d, WORLD_SIZE %d)" %
              (args.gpus, world), file=sys.stderr)
        sys.exit(2)
    import torch

    import synth
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.calibrate_copy > 0:
        calibrate_copy(args.calibrate_copy)
        return
    if args.tables:
        run_tables(args)
        return
    if args.blocks:
        run_blocks(args)
        return
    if args.dihedral:
        run_dihedral(args)
        return
    if args.gconv:
        run_gconv(args)
        return
    digest = source_digest()
    layers = dict(synth.LAYERS)
    layers.update(extra_layers())
    name = args.workload or synth.HEADLINE
    layer = layers[name]
    dt = args.dtype or layer.dtypes[0]
    rec = measure(layer, dt, args, digest, with_cpu=not args.no_cpu_baseline)
    if args.all or not (args.headline_only or args.workload):
        # every other workload of the survey's configurations, at its own
        # shape, with the same protocol and fewer steps
        a2 = argparse.Namespace(**vars(args))
        a2.steps, a2.warmup = min(args.steps, 30), min(args.warmup, 5)
        others = {}
        for n2, l2 in layers.items():
            for d2 in l2.dtypes + EXTRA_DTYPES.get(n2, ()):
                if (n2, d2) == (name, dt):
                    continue
                print("bench: %s %s" % (n2, d2), file=sys.stderr, flush=True)
                r2 = measure(l2, d2, a2 if not args.all else args, digest, with_cpu=False)
                if args.all:
                    print(json.dumps(r2), file=sys.stderr, flush=True)
                others["%s/%s" % (n2, d2)] = {
                    "tokens_per_s": r2["value"], "steps": r2["steps"], "step_us": r2["step_us"],
                    "pass_us": r2["pass_us"], "backward": r2["backward"].split(" (")[0],
                    "roofline_kernel": r2["roofline"]["kernel"], "roofline_frac": r2["roofline"]["frac"],
                    "roofline_step_frac": r2["roofline_step_frac"],
                    "mfma_util_pct": r2["mfma_util_pct"]}
        rec["other_workloads"] = others
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
