"""Benchmark of the bf16x3 compensated GEMM (heal_gemm_f32) on one MI355X.

One step = one compensated product over the whole workload, inputs resident in
HBM.  Default workload: M = N = K = 8192, A and B ~ N(0, 1) FP32.
Prints ONE JSON line:
  value        FP32-equivalent TFLOP/s, 2*M*N*K per step / time
  roofline     the GEMM kernel against the bf16 dense MFMA peak: it executes
               6*M*N*K bf16 flops per launch (three products), so
               frac = (6MNK / t) / peak = (2MNK / t) / (peak / 3)
  cpu_baseline the CPU oracle on a bounded row sample of the same product
  comparison   MI355X native FP32 GEMM (torch.matmul, no TF32) on the same inputs
  bit_repro    every timed step's output bitwise equal to the first
Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu]
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

BF16_DENSE_PEAK_TFLOPS = 2516.6   # 256 CU x 2.4 GHz x 4096 bf16 flop/clk/CU (MI355X, dense)
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="square8192")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target duration of the CPU oracle sample")
    ap.add_argument("--traffic", default=None,
                    help="JSON file with measured HBM bytes per launch for this workload")
    return ap.parse_args()


def cpu_baseline(w, A, B, target_s):
    """Time the CPU oracle on the first R rows of the product, R sized to ~target_s."""
    from oracle import oracle
    orc = oracle.default()
    rows = 1
    t = 0.0
    while True:
        t0 = time.perf_counter()
        orc.gemm3(A[:rows], B)
        t = time.perf_counter() - t0
        if t >= target_s or rows >= A.shape[0]:
            break
        grow = max(2, int(target_s / max(t, 1e-3)))
        rows = min(A.shape[0], rows * grow)
    flops = 2.0 * rows * w.N * w.K * w.batch
    return {"value": flops / t / 1e12, "unit": "TFLOP/s", "cores": orc.num_threads(),
            "kind": "oracle", "seconds": round(t, 3),
            "sample": "first %d of %d rows of the %s product (%dx%dx%d), FP64 accumulation, "
                      "B split included" % (rows, w.M, w.name, rows, w.N, w.K)}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the compensated GEMM is a single-GPU kernel "
              "and this build has no multi-GPU path (--gpus %d requested)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2606_21023_amd as heal
    from paper_2606_21023_amd import workloads as wl

    w = wl.WORKLOADS[args.workload]
    A, B = wl.make_inputs(w)
    torch.cuda.init()
    dev = torch.device("cuda:0")
    Ad = torch.from_numpy(A).to(dev)
    Bd = torch.from_numpy(B).to(dev)
    batched = w.trans_b or w.batch > 1
    if batched:
        Cd = torch.empty((w.batch, w.M, w.N), dtype=torch.float32, device=dev)
        run = lambda out: heal.heal_gemm_f32_strided_batched(Ad, Bd, alpha=w.alpha,
                                                             trans_b=w.trans_b, out=out)
    else:
        Cd = torch.empty((w.M, w.N), dtype=torch.float32, device=dev)
        run = lambda out: heal.heal_gemm_f32(Ad, Bd, out=out)
    first = torch.empty_like(Cd)

    for _ in range(args.warmup):
        run(Cd)
    run(first)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    identical = True
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record(stream)
        run(Cd)
        ends[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    identical = bool(torch.equal(Cd.view(torch.int32), first.view(torch.int32)))
    launch_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    total_ms = starts[0].elapsed_time(ends[-1])
    ms_per_step = total_ms / args.steps
    avg_launch_ms = float(np.mean(launch_ms))

    flops = w.flops
    value = flops / (ms_per_step * 1e-3) / 1e12
    mfma_flops = 3.0 * flops
    achieved = mfma_flops / (avg_launch_ms * 1e-3) / 1e12
    traffic = None
    if args.traffic and os.path.exists(args.traffic):
        with open(args.traffic) as f:
            traffic = json.load(f).get(w.name)
    roofline = {"bound": "mfma", "achieved": round(achieved, 2),
                "peak": BF16_DENSE_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / BF16_DENSE_PEAK_TFLOPS, 4), "traffic": traffic,
                "kernel": "gemm_bf16x3_kernel (large instance)",
                "per_launch": "6*M*N*K bf16 MFMA flops = %.4g" % mfma_flops}

    # MI355X native FP32 GEMM on the same inputs, TF32 off
    torch.backends.cuda.matmul.allow_tf32 = False
    torch.set_float32_matmul_precision("highest")
    mm = (lambda: torch.matmul(Ad, Bd.transpose(-1, -2))) if batched else (lambda: Ad @ Bd)
    for _ in range(3):
        mm()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = max(3, min(20, args.steps))
    e0.record(stream)
    for _ in range(reps):
        mm()
    e1.record(stream)
    torch.cuda.synchronize()
    native_ms = e0.elapsed_time(e1) / reps
    comparison = {"torch_fp32_matmul_tflops": round(flops / (native_ms * 1e-3) / 1e12, 2),
                  "torch_fp32_matmul_ms": round(native_ms, 4)}

    cpu = None
    if not args.no_cpu:
        Ah = A[0] if batched else A
        Bh = np.ascontiguousarray(B[0].T) if batched else B
        wc = wl.Workload(w.name, w.M, w.N, w.K, w.seed)
        cpu = cpu_baseline(wc, Ah, Bh, args.cpu_seconds)

    line = {
        "metric": "FP32-equiv TFLOP/s of compensated GEMM; % of bf16 MFMA peak/3; bit-repro",
        "value": round(value, 2),
        "unit": "TFLOP/s (FP32-equivalent, 2MNK/t)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16x3-f32acc",
        "data": "synthetic",
        "config": {"workload": w.name, "M": w.M, "N": w.N, "K": w.K, "batch": w.batch,
                   "trans_b": w.trans_b, "alpha": w.alpha, "seed": w.seed,
                   "inputs": w.note},
        "pct_of_bf16_peak_div3": round(100.0 * value / (BF16_DENSE_PEAK_TFLOPS / 3), 2),
        "bit_repro": {"runs": args.steps + 1, "identical": identical},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "comparison": comparison,
        "wall_s": round(wall, 3),
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
