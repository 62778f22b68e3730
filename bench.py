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


def parse_args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="C2")
    ap.add_argument("--dtype", default=None, help="f32 or bf16 (default: the workload's)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--launch-table", action="store_true",
                    help="print per-launch averages of the timed steps to stderr")
    ap.add_argument("--cpu-batch", type=int, default=128, help="batch of the oracle CPU sample")
    ap.add_argument("--generic", action="store_true", help="generic kernel only")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MiB",
                    help="only run plain device copies of this size (counter calibration)")
    return ap.parse_args()


def kernel_sources_sha256():
    """Hash of every kernel source: counter results stay valid only while it matches."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2401_03384_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(os.listdir(csrc)):
        if f.endswith(".hip"):
            h.update(f.encode())
            h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()


def measured_traffic(kname, dtype):
    """HBM bytes per dispatch of `kname` from the committed counter summary,
    or None when there is none or any kernel source changed since."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_c2_{dtype}.json")
    if not os.path.exists(path):
        return None
    info = json.load(open(path))
    if info.get("kernel_sources_sha256") != kernel_sources_sha256():
        return None
    return info["bytes_per_dispatch"].get(kname)


def roofline(records, dtype):
    """Dominant kernel (largest total time) from the live launch records."""
    by = {}
    for kname, step, ms, nbytes, flops in records:
        d = by.setdefault(kname, [0.0, 0, 0.0, 0.0])
        d[0] += ms
        d[1] += 1
        d[2] += nbytes
        d[3] += flops
    kname, (ms, n, nbytes, flops) = max(by.items(), key=lambda kv: kv[1][0])
    ai = flops / max(nbytes, 1.0)
    ridge = PEAK_MFMA_TFLOPS[dtype] * 1e12 / (PEAK_HBM_GBS * 1e9)
    avg_s = ms / n / 1e3
    if ai < ridge:
        achieved, peak, unit, bound = nbytes / n / avg_s / 1e9, PEAK_HBM_GBS, "GB/s", "hbm"
    else:
        achieved, peak, unit, bound = flops / n / avg_s / 1e12, PEAK_MFMA_TFLOPS[dtype], "TFLOP/s", "mfma"
    total = sum(v[0] for v in by.values())
    traffic = measured_traffic(kname, dtype)
    return {"kernel": kname, "bound": bound, "achieved": round(achieved, 2), "peak": peak,
            "unit": unit, "frac": round(achieved / peak, 4),
            "traffic": None if traffic is None else round(traffic),
            "alg_bytes_per_launch": round(nbytes / n),
            "launches": n, "avg_us": round(ms / n * 1e3, 2),
            "share_of_kernel_time": round(ms / total, 3)}


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
            "kind": "oracle", "seconds": round(dt, 2), "passes": passes,
            "sample": f"{ws.name}: batch {batch} of {w.shapes[0][0]}, other sizes full; "
                      f"float64 pairwise forward + backward along the planned tree, "
                      f"{passes} passes"}


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); multi-GPU is "
              "not part of this build", file=sys.stderr)
        sys.exit(2)
    import numpy as np
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

    import paper_2401_03384_amd as P
    import workloads as W

    w = W.WORKLOADS[args.workload]
    dtype = args.dtype or w.dtype
    if dtype != w.dtype:
        w = W.Workload(w.name, w.spec, w.shapes, dtype, w.seed, w.sigmas, w.out_shape, w.backward)
    dev = torch.device("cuda:0")
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    ins, dy = W.make_inputs(w)
    xs = [torch.from_numpy(a.astype(np.float32)).to(tdt).to(dev) for a in ins]
    d = torch.from_numpy(dy.astype(np.float32)).to(tdt).to(dev)
    flags = P.CE_FLAG_GENERIC_ONLY if args.generic else 0
    ref = P.Plan(w.spec, w.shapes, dtype, flags=flags)
    ws = torch.empty(max(ref.ws_fwd, ref.ws_bwd, 1), dtype=torch.uint8, device=dev)
    out = torch.empty(ref.out_shape, dtype=tdt, device=dev)
    grads = [torch.empty(s, dtype=ref.grad_dtype(i), device=dev) for i, s in enumerate(w.shapes)]
    in_ptrs = [x.data_ptr() for x in xs]
    g_ptrs = [g.data_ptr() for g in grads]
    stream = torch.cuda.current_stream(dev).cuda_stream
    shapes = [tuple(s) for s in w.shapes]
    cdt = P.CE_BF16 if dtype == "bf16" else P.CE_F32

    def step(fwd=True, bwd=True):
        e = P.ce_expr_parse(w.spec, shapes)
        p = P.ce_plan_create(e, P.CE_COST_FWD, cdt, flags)
        P.ce_expr_destroy(e)
        if fwd:
            P.ce_forward(p, in_ptrs, out.data_ptr(), ws.data_ptr(), ws.numel(), stream)
        if bwd:
            P.ce_backward(p, in_ptrs, d.data_ptr(), g_ptrs, ws.data_ptr(), ws.numel(), stream)
        P.ce_plan_destroy(p)

    def timed(n, **kw):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(n):
            step(**kw)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / n

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # timed region: whole steps, with per-launch HIP events recorded live
    P.ce_timing_begin()
    t_step = timed(args.steps)
    n_rec = P.ce_timing_end()
    records = [P.ce_timing_record(i) for i in range(n_rec)]
    if args.launch_table:
        print(launch_table(records, args.steps), file=sys.stderr, flush=True)
    # forward-only and backward-only steps (reported beside the main figure)
    t_fwd = timed(max(5, args.steps // 2), bwd=False)
    t_bwd = timed(max(5, args.steps // 2), fwd=False)
    t0 = time.perf_counter()
    for _ in range(200):
        e = P.ce_expr_parse(w.spec, shapes)
        p = P.ce_plan_create(e, P.CE_COST_FWD, cdt, flags)
        P.ce_expr_destroy(e)
        P.ce_plan_destroy(p)
    t_plan = (time.perf_counter() - t0) / 200

    macs = ref.fwd_macs
    value = 6 * macs / t_step / 1e12
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
                   "flops_per_step": 6 * macs, "path": "generic" if args.generic else "default"},
        "fwd_ms": round(t_fwd * 1e3, 4),
        "bwd_ms": round(t_bwd * 1e3, 4),
        "plan_ms": round(t_plan * 1e3, 4),
        "roofline": roofline(records, dtype),
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_batch)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
