"""Benchmark: forward + backward of the CP-factorised 3x3 conv layer of ResNet
stage-1 shape (X[128,64,56,56], C_in = C_out = 64, rank 32) on one MI355X.

One step = the whole hot path once: parse the conv_einsum string, bind sizes,
plan (tnn-cost sequencer, lowering, workspace), forward, backward (all five
gradients).  Inputs are resident in HBM before the timed region.

Prints one JSON line (see the keys below).  `value` is effective TFLOP/s:
6 x (forward multiplications of the planned path) per step / time.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
PEAK_MFMA_TFLOPS = {"f32": 157.3, "bf16": 2500.0}
# layer floors use the dense MFMA peak of the input type (157.3 / 2516.6 TFLOP/s)
PEAK_LAYER_TFLOPS = {"f32": 157.3, "bf16": 2516.6}
# the five layers of the metric; C2 in float32 is the headline line itself
CONFIGS = [("C2", "f32"), ("C2_bf16", "bf16"), ("C3", "bf16"), ("C4", "f32"), ("C5a", "bf16"),
           ("C5b", "bf16")]
# kernels whose arithmetic runs on the vector ALU (no MFMA tile fits their
# contractions): peak = 256 CUs x 64 lanes x 2.4 GHz x flops per lane-op,
# 4 for v_dot2_f32_bf16 (two products) and 2 for an fp32 FMA
ALU_BOUND = {"rcp_fwd": 157.3, "rcp_bwd": 157.3, "cred": 78.6, "credw": 78.6}


def parse_args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    # the chip's clocks rise over tens of milliseconds of load: 500 steps of
    # the default layer (about 90 ms) reach the steady state, 5 steps do not
    # (C2 fp32: 0.227 ms a step after 5, 0.183 ms after 200)
    ap.add_argument("--warmup", type=int, default=500)
    ap.add_argument("--workload", default="C2")
    ap.add_argument("--dtype", default=None, help="f32 or bf16 (default: the workload's)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--launch-table", action="store_true",
                    help="print per-launch averages of the timed steps to stderr")
    ap.add_argument("--cpu-batch", type=int, default=128, help="batch of the oracle CPU sample")
    ap.add_argument("--generic", action="store_true", help="generic kernel only")
    ap.add_argument("--path", choices=["optimal", "ltr"], default="optimal",
                    help="pairwise order: the planner's optimum or the left-to-right baseline")
    ap.add_argument("--max-elements", type=int, default=None,
                    help="cap on the elements of every intermediate (memory-limited order)")
    ap.add_argument("--save-budget", type=float, default=None, metavar="MiB",
                    help="checkpointing: MiB of forward intermediates the backward may read "
                         "instead of recomputing (default: recompute every one)")
    ap.add_argument("--graph", action="store_true",
                    help="also time forward + backward replayed from a HIP graph (no host work)")
    ap.add_argument("--compare-ltr", action="store_true",
                    help="also time the left-to-right order on the same kernels")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-layer lines of the other configurations")
    ap.add_argument("--sample-steps", type=int, default=100,
                    help="individually timed steps for the median / min")
    ap.add_argument("--sweep", action="store_true",
                    help="only the ResNet-34 CP-layer sweep: planned vs left-to-right order")
    ap.add_argument("--sweep-batch", type=int, default=16,
                    help="batch of the timed sweep steps (FLOPs are also given at 128)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MiB",
                    help="only run plain device copies of this size (counter calibration)")
    return ap.parse_args()


# device code of each kernel: its source file and the headers it includes
KERNEL_SOURCES = {
    "cp_": ("kernels_cp.hip", "desc.h", "hip_util.h"),
    "reduce_multi": ("kernels_fast.hip", "desc.h", "hip_util.h"),
}


def source_hashes(files):
    import hashlib
    csrc = os.path.join(ROOT, "paper_2401_03384_amd", "csrc")
    return {f: hashlib.sha256(open(os.path.join(csrc, f), "rb").read()).hexdigest() for f in files}


def measured_traffic(kname, dtype):
    """HBM bytes per dispatch of `kname` from the committed counter summary,
    or None when there is none or the kernel's sources changed since."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_c2_{dtype}.json")
    if not os.path.exists(path):
        return None
    info = json.load(open(path))
    entry = info.get("kernels", {}).get(kname)
    if entry is None or entry["sources"] != source_hashes(sorted(entry["sources"])):
        return None
    return entry["bytes_per_dispatch"]


def kernel_totals(records):
    by = {}
    for kname, step, ms, nbytes, flops in records:
        d = by.setdefault(kname, [0.0, 0, 0.0, 0.0])
        d[0] += ms
        d[1] += 1
        d[2] += nbytes
        d[3] += flops
    return by


def roofline(records, dtype, share):
    """Roofline of the dominant kernel from its live launch records (every
    record is a launch of that kernel, bracketed by HIP events on its own
    stream); `share` is its share of kernel time."""
    by = kernel_totals(records)
    assert len(by) == 1, by.keys()
    kname, (ms, n, nbytes, flops) = next(iter(by.items()))
    ai = flops / max(nbytes, 1.0)
    ridge = PEAK_MFMA_TFLOPS[dtype] * 1e12 / (PEAK_HBM_GBS * 1e9)
    avg_s = ms / n / 1e3
    alu = [v for k, v in ALU_BOUND.items() if kname.startswith(k)]
    if alu:
        achieved, peak, unit, bound = flops / n / avg_s / 1e12, alu[0], "TFLOP/s", "alu"
    elif ai < ridge:
        achieved, peak, unit, bound = nbytes / n / avg_s / 1e9, PEAK_HBM_GBS, "GB/s", "hbm"
    else:
        achieved, peak, unit, bound = flops / n / avg_s / 1e12, PEAK_MFMA_TFLOPS[dtype], "TFLOP/s", "mfma"
    traffic = measured_traffic(kname, dtype)
    extra = {}
    if alu:
        # the same work against the dense MFMA peak of its input type
        mf = flops / n / avg_s / 1e12
        extra = {"frac_vs_mfma_peak": round(mf / PEAK_LAYER_TFLOPS[dtype], 5)}
    return {"kernel": kname, "bound": bound, "achieved": round(achieved, 2), "peak": peak,
            "unit": unit, "frac": round(achieved / peak, 4), **extra,
            "traffic": None if traffic is None else round(traffic),
            "alg_bytes_per_launch": round(nbytes / n),
            "launches": n, "avg_us": round(ms / n * 1e3, 2),
            "avg_us_timing": "HIP events bracketing each launch on its stream",
            "share_of_kernel_time": round(share, 3)}


def prod(xs):
    out = 1
    for x in xs:
        out *= int(x)
    return out


def layer_floor_us(w, dtype, macs):
    """Forward + backward floor of a layer: max(F / MFMA peak, B / HBM peak)
    with F = 6 x planned forward MACs and B = the compulsory bytes (X and dY
    read, Y and dX written once in the input type; factors read once and
    their float32 gradients written once)."""
    e = 2 if dtype == "bf16" else 4
    nx, ny = prod(w.shapes[0]), prod(w.out_shape)
    nf = sum(prod(s) for s in w.shapes[1:])
    nbytes = e * (2 * nx + 2 * ny) + nf * (e + 4)
    return max(6 * macs / (PEAK_LAYER_TFLOPS[dtype] * 1e12), nbytes / (PEAK_HBM_GBS * 1e9)) * 1e6


def launch_table(records, steps):
    """Per-launch averages over the timed steps (launch order of one step)."""
    per = len(records) // max(steps, 1)
    rows = []
    for i in range(per):
        rs = records[i::per]
        ms = sum(r[2] for r in rs) / len(rs)
        kname, step, _, nbytes, flops = rs[0]
        rows.append((ms, kname, step, nbytes, flops))
    tot = sum(r[0] for r in rows)
    lines = [f"{'us':>9s} {'share':>6s} {'GB/s':>8s} {'TF/s':>7s}  kernel | step"]
    for ms, kname, step, nbytes, flops in rows:
        s = ms / 1e3
        lines.append(f"{ms * 1e3:9.1f} {ms / tot:6.1%} {nbytes / s / 1e9 if s else 0:8.0f} "
                     f"{flops / s / 1e12 if s else 0:7.2f}  {kname} | {step}")
    return "\n".join(lines)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(w, batch):
    """The float64 oracle's pairwise forward + backward on a batch sample."""
    import numpy as np
    import oracle as O
    import workloads as W
    from threadpoolctl import threadpool_info

    shapes = [list(s) for s in w.shapes]
    shapes[0][0] = batch
    ws = W.Workload(w.name + "_cpu", w.spec, tuple(tuple(s) for s in shapes), w.dtype, w.seed,
                    w.sigmas, (batch,) + tuple(w.out_shape[1:]), True)
    ins, dy = W.make_inputs(ws)
    e = O.bind(O.parse(ws.spec), ws.shapes)
    tree, macs = O.optimal_tree(e)
    # whole passes until about ten seconds of CPU work (at most 30 passes)
    passes, t0 = 0, time.perf_counter()
    while True:
        O.eval_pairwise(e, ins, tree)
        O.grads_pairwise(e, ins, tree, dy)
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= 10.0 or passes >= 30:
            break
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": round(6 * macs * passes / dt / 1e12, 6), "unit": "TFLOP/s", "cores": threads,
            "cpu": cpu_model(), "host_cpus": os.cpu_count(),
            "kind": "oracle", "seconds": round(dt, 2), "passes": passes,
            "sample": f"{ws.name}: batch {batch} of {w.shapes[0][0]}, other sizes full; "
                      f"float64 pairwise forward + backward along the planned tree, "
                      f"{passes} passes"}


def warm(step, min_steps, min_s=0.1):
    """Untimed steps until at least min_steps have run and min_s seconds have
    passed: the GPU clocks ramp up over tens of milliseconds of load, and
    every layer here is set up after host work that leaves the GPU idle."""
    import torch

    t0 = time.perf_counter()
    n = 0
    while n < min_steps or time.perf_counter() - t0 < min_s:
        step()
        n += 1
        if n % 8 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()


def compare_ltr(w, dtype, xs, d, ltr, flags, stream, cdt, args):
    """The paper's baseline order on the same kernels: forward + backward time,
    forward multiplications and workspace of the left-to-right plan."""
    import torch
    import paper_2401_03384_amd as P

    dev = xs[0].device
    pl = P.Plan(w.spec, w.shapes, dtype, flags=flags, path=ltr)
    ws = torch.empty(max(pl.ws_fwd, pl.ws_bwd, 1), dtype=torch.uint8, device=dev)
    out = torch.empty(pl.out_shape, dtype=xs[0].dtype, device=dev)
    grads = [torch.empty(s, dtype=pl.grad_dtype(i), device=dev) for i, s in enumerate(w.shapes)]
    in_ptrs = [x.data_ptr() for x in xs]
    g_ptrs = [g.data_ptr() for g in grads]

    def run():
        P.ce_forward(pl.handle, in_ptrs, out.data_ptr(), ws.data_ptr(), ws.numel(), stream)
        P.ce_backward(pl.handle, in_ptrs, d.data_ptr(), g_ptrs, ws.data_ptr(), ws.numel(), stream)

    warm(run, 2)
    n = max(3, args.steps // 5)
    t0 = time.perf_counter()
    for _ in range(n):
        run()
    torch.cuda.synchronize()
    t = (time.perf_counter() - t0) / n
    return {"ms_per_step": round(t * 1e3, 4), "fwd_macs": pl.fwd_macs,
            "workspace_bytes": {"fwd": pl.ws_fwd, "bwd": pl.ws_bwd},
            "steps": n}


class Runner:
    """One layer on the device: seeded inputs resident in HBM, output,
    gradient and workspace buffers, and step() = parse + plan + forward +
    backward through the C ABI on torch's current stream."""

    def __init__(self, w, dtype, flags=0, path=None, max_elements=None, strides=None, save_budget=None):
        import numpy as np
        import torch
        import paper_2401_03384_amd as P
        import workloads as W

        if dtype != w.dtype:
            w = W.Workload(w.name, w.spec, w.shapes, dtype, w.seed, w.sigmas, w.out_shape, w.backward)
        self.w, self.dtype, self.flags, self.path, self.max_elements = w, dtype, flags, path, max_elements
        self.save_budget = save_budget
        self.strides = dict(strides or {})
        dev = torch.device("cuda:0")
        tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
        ins, dy = W.make_inputs(w)
        self.xs = [torch.from_numpy(a.astype(np.float32)).to(tdt).to(dev) for a in ins]
        self.d = torch.from_numpy(dy.astype(np.float32)).to(tdt).to(dev)
        del ins, dy
        self.ref = P.Plan(w.spec, w.shapes, dtype, flags=flags, path=path, max_elements=max_elements,
                          strides=self.strides, save_budget=save_budget)
        ref = self.ref
        self.ws = torch.empty(max(ref.ws_fwd, ref.ws_bwd, 1), dtype=torch.uint8, device=dev)
        self.out = torch.empty(ref.out_shape, dtype=tdt, device=dev)
        self.grads = [torch.empty(s, dtype=ref.grad_dtype(i), device=dev) for i, s in enumerate(w.shapes)]
        self.in_ptrs = [x.data_ptr() for x in self.xs]
        self.g_ptrs = [g.data_ptr() for g in self.grads]
        self.stream = torch.cuda.current_stream(dev).cuda_stream
        self.shapes = [tuple(s) for s in w.shapes]
        self.cdt = P.CE_BF16 if dtype == "bf16" else P.CE_F32
        self.P, self.torch = P, torch

    def step(self, fwd=True, bwd=True):
        P, w = self.P, self.w
        e = P.ce_expr_parse(w.spec, self.shapes)
        for label, st in self.strides.items():
            P.ce_expr_set_stride(e, label, st)
        if self.path is None and self.save_budget is not None:
            p = P.ce_plan_create_ex(e, P.CE_COST_FWD, self.cdt, self.flags, 0, self.max_elements or 0,
                                    self.save_budget)
        elif self.path is None and self.max_elements is not None:
            p = P.ce_plan_create_limited(e, P.CE_COST_FWD, self.cdt, self.flags, self.max_elements)
        elif self.path is None:
            p = P.ce_plan_create(e, P.CE_COST_FWD, self.cdt, self.flags)
        else:
            p = P.ce_plan_create_with_path(e, self.path, self.cdt, self.flags)
        P.ce_expr_destroy(e)
        if fwd:
            P.ce_forward(p, self.in_ptrs, self.out.data_ptr(), self.ws.data_ptr(), self.ws.numel(),
                         self.stream)
        if bwd:
            P.ce_backward(p, self.in_ptrs, self.d.data_ptr(), self.g_ptrs, self.ws.data_ptr(),
                          self.ws.numel(), self.stream)
        P.ce_plan_destroy(p)

    def timed(self, n, **kw):
        torch = self.torch
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(n):
            self.step(**kw)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / n

    def sampled(self, n):
        """n steps each bracketed by events on the launch stream: median,
        min and mean in ms."""
        torch = self.torch
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(n)]
        torch.cuda.synchronize()
        for a, b in evs:
            a.record()
            self.step()
            b.record()
        torch.cuda.synchronize()
        ts = sorted(a.elapsed_time(b) for a, b in evs)
        return {"median_ms": round(ts[len(ts) // 2], 4), "min_ms": round(ts[0], 4),
                "mean_ms": round(sum(ts) / len(ts), 4), "samples": n}

    def dominant(self):
        """One step with every launch timed: the kernel with the largest
        total time and its share of the step's kernel time."""
        P = self.P
        P.ce_timing_begin()
        self.step()
        probe = [P.ce_timing_record(i) for i in range(P.ce_timing_end())]
        by = kernel_totals(probe)
        k = max(by, key=lambda x: by[x][0])
        return k, by[k][0] / sum(v[0] for v in by.values())

    def kernel_roofline(self, kname, share, n):
        """Roofline of kernel `kname` over n steps, only its launches bracketed."""
        P = self.P
        P.ce_timing_begin_kernel(kname)
        t = self.timed(n)
        records = [P.ce_timing_record(i) for i in range(P.ce_timing_end())]
        return t, roofline(records, self.dtype, share)


def checkpoint_line(plan):
    """The plan's checkpointing choice: steps whose results the forward keeps
    for the backward, their bytes, and the multiplications recomputed."""
    import paper_2401_03384_amd as P

    steps, nbytes, macs = P.ce_plan_checkpoint(plan.handle)
    return {"saved_steps": [s for s in range(64) if steps >> s & 1], "saved_bytes": nbytes,
            "recompute_macs": macs}


def max_batch_line(w):
    """Largest batch whose training step fits an HBM budget (planning only):
    the planned order vs left-to-right with recomputation and left-to-right
    keeping every intermediate (both unfused), as in the paper's
    maximum-batch comparison; budgets: 11 GiB and 288 GB."""
    import paper_2401_03384_amd as P
    out = {}
    for label, budget in (("11GiB", 11 << 30), ("288GB", 288 * 10 ** 9)):
        out[label] = {
            "optimal": P.max_batch(w.spec, w.shapes, budget, w.dtype),
            "ltr_recompute": P.max_batch(w.spec, w.shapes, budget, w.dtype, "ltr", fusion=False),
            "ltr_keep_all": P.max_batch(w.spec, w.shapes, budget, w.dtype, "ltr", save=True,
                                        fusion=False)}
    return out


def config_line(name, dtype, steps, samples):
    """fwd+bwd figures of one configuration (see CONFIGS)."""
    import workloads as W

    r = Runner(W.WORKLOADS[name], dtype)
    warm(r.step, 3)
    kname, share = r.dominant()
    t, roof = r.kernel_roofline(kname, share, max(5, steps // 2))
    t_mean = r.timed(steps)
    smp = r.sampled(samples)
    macs = r.ref.fwd_macs
    floor = layer_floor_us(r.w, dtype, macs)
    w = r.w
    out = {"workload": f"{w.name}: {w.spec} X{list(w.shapes[0])}", "dtype": dtype,
           "ms_per_step": round(t_mean * 1e3, 4), **smp,
           "tflops": round(6 * macs / t_mean / 1e12, 3),
           "floor_us": round(floor, 1), "floor_frac": round(floor / (t_mean * 1e6), 4),
           "floor_frac_median": round(floor / (smp["median_ms"] * 1e3), 4),
           "workspace_bytes": {"fwd": r.ref.ws_fwd, "bwd": r.ref.ws_bwd},
           "dominant": {k: roof[k] for k in ("kernel", "bound", "achieved", "unit", "peak", "frac",
                                             "avg_us", "share_of_kernel_time")
                        if k in roof}}
    if "frac_vs_mfma_peak" in roof:
        out["dominant"]["frac_vs_mfma_peak"] = roof["frac_vs_mfma_peak"]
    out["max_batch"] = max_batch_line(r.w)
    del r
    import torch
    torch.cuda.empty_cache()
    return out


def sweep(args):
    """ResNet-34's convolutions as CP layers at compression rate 100% (the
    paper's per-layer FLOPs comparison, Section 5, Table 2): for the planned
    and the left-to-right order on the same kernels, forward FLOPs at batch
    128, and forward + backward time, FLOP rate and workspace at
    --sweep-batch.  One JSON line."""
    import torch
    import paper_2401_03384_amd as P
    import workloads as W

    ltr = [(0, 1), (0, 3), (0, 2), (0, 1)]
    rows = []
    for name, *_ in W.RESNET34_CONVS:
        w128, st = W.resnet34_cp_layer(name, batch=128)
        rows.append({"layer": name, "stride": st.get("h", 1), "rank": w128.shapes[1][0],
                     "X": list(w128.shapes[0])})
    # every layer's planned order first, then every left-to-right run: a step
    # timed right after a left-to-right run (gigabytes of workspace allocated
    # and freed) ran several times slower than the same step alone
    for order, path in (("optimal", None), ("left_to_right", ltr)):
        for row in rows:
            name = row["layer"]
            w128, st = W.resnet34_cp_layer(name, batch=128)
            p128 = P.Plan(w128.spec, w128.shapes, "f32", strides=st, path=path)
            w, _ = W.resnet34_cp_layer(name, batch=args.sweep_batch)
            r = Runner(w, args.dtype or "f32", path=path, strides=st)
            warm(r.step, 2)
            n = 3 if order == "left_to_right" else 10
            t = r.timed(n)
            row[order] = {"fwd_gflop_b128": round(2 * p128.fwd_macs / 1e9, 3),
                          "ms_fwd_bwd": round(t * 1e3, 4),
                          "tflops": round(6 * r.ref.fwd_macs / t / 1e12, 2),
                          "workspace_gb": [round(r.ref.ws_fwd / 1e9, 3), round(r.ref.ws_bwd / 1e9, 3)],
                          "steps": [[a, b] for a, b, _ in r.ref.steps]}
            del r
            torch.cuda.empty_cache()
            print(f"sweep {name} {order}: {row[order]['ms_fwd_bwd']} ms", file=sys.stderr, flush=True)
    for row in rows:
        row["flop_ratio"] = round(row["left_to_right"]["fwd_gflop_b128"] /
                                  row["optimal"]["fwd_gflop_b128"], 2)
        row["time_ratio"] = round(row["left_to_right"]["ms_fwd_bwd"] / row["optimal"]["ms_fwd_bwd"], 2)
    print(json.dumps({"sweep": "ResNet-34 CP layers, compression rate 100%", "dtype": args.dtype or "f32",
                      "timed_batch": args.sweep_batch, "layers": rows}), flush=True)


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); multi-GPU is "
              "not part of this build", file=sys.stderr)
        sys.exit(2)
    import torch

    if args.calibrate_copy:
        # a plain copy kernel of known size: read n bytes, write n bytes
        n = args.calibrate_copy << 20
        a = torch.ones(n // 4, dtype=torch.float32, device="cuda:0")
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n, "launches": 5}), flush=True)
        return

    if args.sweep:
        sweep(args)
        return

    import paper_2401_03384_amd as P
    import workloads as W

    w = W.WORKLOADS[args.workload]
    dtype = args.dtype or w.dtype
    flags = P.CE_FLAG_GENERIC_ONLY if args.generic else 0
    n_in = len(w.shapes)
    # left-to-right in the list format of ce_plan_create_with_path
    ltr = [(0, 1)] + [(0, n_in - 1 - k) for k in range(1, n_in - 1)]
    path = ltr if args.path == "ltr" else None
    budget = None if args.save_budget is None else int(args.save_budget * 2**20)
    r = Runner(w, dtype, flags, path, args.max_elements, save_budget=budget)
    w, ref = r.w, r.ref

    for _ in range(args.warmup):
        r.step()
    torch.cuda.synchronize()
    dominant, share = r.dominant()
    # timed region: exactly --steps whole steps, nothing recorded in between
    t_step = r.timed(args.steps)
    # the same number of steps again with the dominant kernel's launches
    # bracketed by HIP events on their stream (the other launches run without
    # events in between): its average duration for the roofline
    t_events, roof = r.kernel_roofline(dominant, share, args.steps)
    roof["ms_per_step_with_events"] = round(t_events * 1e3, 4)
    if args.launch_table:
        P.ce_timing_begin()
        r.timed(args.steps)
        table = [P.ce_timing_record(i) for i in range(P.ce_timing_end())]
        print(launch_table(table, args.steps), file=sys.stderr, flush=True)
    smp = r.sampled(max(args.sample_steps, args.steps))
    # forward-only and backward-only steps (reported beside the main figure)
    t_fwd = r.timed(max(5, args.steps // 2), bwd=False)
    t_bwd = r.timed(max(5, args.steps // 2), fwd=False)
    t0 = time.perf_counter()
    for _ in range(200):
        e = P.ce_expr_parse(w.spec, r.shapes)
        p = P.ce_plan_create(e, P.CE_COST_FWD, r.cdt, flags)
        P.ce_expr_destroy(e)
        P.ce_plan_destroy(p)
    t_plan = (time.perf_counter() - t0) / 200

    macs = ref.fwd_macs
    value = 6 * macs / t_step / 1e12
    floor = layer_floor_us(w, dtype, macs)
    line = {
        "metric": "effective TFLOP/s (fwd+bwd) of a CP-factorised 3x3 conv layer, 1 MI355X",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(t_step * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic (seeded N(0,1) input, Kaiming-scaled factors)",
        "config": {"workload": f"{w.name}: {w.spec} X{list(w.shapes[0])} rank {w.shapes[1][0]}",
                   "global_batch": w.shapes[0][0], "fwd_macs": macs,
                   "flops_per_step": 6 * macs,
                   "path": ("left-to-right" if path else "optimal")
                   + (f", intermediates <= {args.max_elements} elements" if args.max_elements else "")
                   + (f", save budget {args.save_budget} MiB" if budget is not None else "")
                   + (", generic kernel" if args.generic else "")},
        "step_ms": smp,
        "floor_us": round(floor, 1),
        "floor_frac": round(floor / (t_step * 1e6), 4),
        "workspace_bytes": {"fwd": ref.ws_fwd, "bwd": ref.ws_bwd},
        "checkpoint": checkpoint_line(ref),
        "max_batch": max_batch_line(w),
        "fwd_ms": round(t_fwd * 1e3, 4),
        "bwd_ms": round(t_bwd * 1e3, 4),
        "plan_ms": round(t_plan * 1e3, 4),
        "roofline": roof,
    }
    if args.graph:
        g = P.GraphStep(ref, r.xs, r.d)
        for _ in range(3):
            g.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            g.replay()
        torch.cuda.synchronize()
        tg = (time.perf_counter() - t0) / args.steps
        line["graph"] = {"ms_per_step": round(tg * 1e3, 4), "tflops": round(6 * macs / tg / 1e12, 3),
                         "note": "forward + backward replayed from one HIP graph; no parse or plan"}
    if args.compare_ltr and path is None:
        lt = compare_ltr(w, dtype, r.xs, r.d, ltr, flags, r.stream, r.cdt, args)
        lt["time_ratio_vs_optimal"] = round(lt["ms_per_step"] / (t_step * 1e3), 3)
        line["left_to_right"] = lt
    default_run = (args.workload == "C2" and dtype == "f32" and path is None and
                   not args.max_elements and not args.generic and budget is None)
    if not args.no_configs and default_run:
        del r
        torch.cuda.empty_cache()
        cfgs = {}
        for name, dt in CONFIGS:
            if name == "C2" and dt == "f32":
                continue
            cfgs[name] = config_line(name, dt, max(20, args.steps), args.sample_steps)
            print(f"config {name}: {cfgs[name]['ms_per_step']} ms", file=sys.stderr, flush=True)
        line["configs"] = cfgs
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, min(args.cpu_batch, w.shapes[0][0]))
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
