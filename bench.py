"""Benchmark of the bf16x3 compensated GEMM (heal_gemm_f32) on one MI355X.

One step = one compensated product over the whole workload (every step of the
method: split, three bf16 products, FP32 accumulation and output, all inside
one kernel launch), inputs resident in HBM when the timed region starts.
Default workload: M = N = K = 8192, A and B ~ N(0, 1) FP32, the square case the
throughput target is quoted on.  Other workloads (--workload) are the
LLM-layer shapes of the parity tests.

Prints ONE JSON line:
  value        FP32-equivalent TFLOP/s, 2*M*N*K*batch per step / time per step
  roofline     the GEMM kernel (the only kernel of a step) against its bound:
                 mfma: 6*M*N*K bf16 flops per launch (three products) over the
                       bf16 dense MFMA peak, so frac = value / (peak / 3);
                 hbm:  FP32 A, B read once and C written once per launch over
                       the 8 TB/s HBM peak;
               the launches of the timed region run back to back on one
               stream (pre-built C-ABI arguments, no per-call marshalling;
               --graph captures them into one HIP graph and times one replay
               of it, for microsecond kernels under a tracer, whose host
               cost per launch would leave gaps); the launch duration is the
               HIP-event time of the region on that stream divided by the
               number of launches.  traffic is
               the HBM bytes per launch measured by FETCH_SIZE / WRITE_SIZE
               counters (scaled by a plain copy of known size), taken from
               profiles/traffic.json only while the kernel sources are the
               ones it was measured on, else null.
  cpu_baseline the CPU oracle timed on a bounded row sample of the same product
  comparison   MI355X native FP32 GEMM (torch.matmul, TF32 off) on the same inputs;
               for MFMA-bound products also one plain bf16 GEMM of the same
               shape (hipBLASLt), timed after the timed region
  bit_repro    every timed launch writes its own output buffer (up to 64 GiB of
               them); all are compared bitwise with the first timed output
  build_id     the source hash libheal.so was built from (checked at start)
  step_stats   median, minimum and standard error of the per-launch times
               of a separate pass of the same launches with an event between
               each (the paper's timing convention), run before the warm-up
               launches; the FP32 comparison (below) runs before it.  Both
               take the GPU out of its idle clocks, which would otherwise
               slow the first tens of launches

--method selects the product (default bf16x3, the line above):
  presplit    heal_gemm_f32_presplit: B split once into packed bf16 (hi, lo)
              before the timed region; same MFMAs, bitwise equal results;
  f16_full    heal_gemm_f16w, HEAL-Full: W = B^T packed to FP16 (scaled by
              2^e) before the timed region, two FP16 products per chunk;
  f16_base    heal_gemm_f16w, HEAL-Base: one FP16 product per chunk;
  i16_scores  heal_scores_i16 on the attention workload: Q and K quantized to
              INT16 before the timed region (as stored in the KV cache), four
              FP16 products per chunk;
  split       heal_split_f32 over the workload's B operand: value is GB/s
              (8 bytes per element), HBM-bound.
For every GEMM method a step is one launch of its GEMM kernel over the
workload; value is FP32-equivalent TFLOP/s (2*M*N*K*batch per step); the
roofline uses the method's own MFMA flops and operand bytes.
Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                       [--method NAME] [--no-cpu] [--graph]
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

BF16_DENSE_PEAK_TFLOPS = 2516.6   # 256 CU x 2.4 GHz x 4096 bf16 flop/clk/CU (MI355X, dense)
HBM_PEAK_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
# the kernel each instance of heal_gemm_f32 launches (16-byte aligned
# operands), and the sources that define it
KERNEL_NAMES = {1: "gemm_large8_kernel (256x256 tiles, 8 waves of 64x128)",
                2: "gemm_bf16x3_kernel<128,128,64,32,64,512,2> (medium, 8 waves, register ring)",
                3: "gemm_skinny_kernel (column strips, M <= 64)"}
KERNEL_SOURCES = {1: ["heal_gemm_large.hip", "heal_device.h", "heal_internal.h"],
                  2: ["heal_gemm.hip", "heal_device.h", "heal_internal.h"],
                  3: ["heal_gemm_skinny.hip", "heal_device.h", "heal_internal.h"],
                  "op": ["heal_gemm_op.hip", "heal_device.h", "heal_internal.h"],
                  "panel": ["heal_gemm_panel.hip", "heal_device.h", "heal_internal.h"],
                  "split": ["heal_split.hip", "heal_device.h", "heal_internal.h"]}
OP_INSTANCE_NAMES = {1: "large 128x256, 8 waves", 2: "medium 128x128, 8 waves, two register sets",
                     3: "skinny M<=64, 256-column tiles"}


def skinny_strip_width(N, M):
    """Column-strip width of an M x N output with M <= 64, as the library
    picks it (skinny_strip_width in heal_gemm_skinny.hip): the widest of 256,
    128, 64 and 32 columns with at least 480 strips at up to 32 rows (240
    above), else 32 if that still gives 160 strips, else 16."""
    least = 480 if M <= 32 else 240
    for w in (256, 128, 64, 32):
        if -(-N // w) >= least:
            return w
    return 32 if -(-N // 32) >= 160 else 16


def skinny_row_groups(N, M, trans_b, batch):
    """Row groups of the bf16x3 skinny kernel (skinny_row_groups in
    heal_gemm_skinny.hip): where the width rule gives 16-column strips, a
    product with one batch entry runs on 32-column strips with the rows in
    G groups (1, 2 or 4, dividing M; at most 256 workgroups, at least 128;
    with B stored N x K more than one group only above 32 rows, and at
    least 160 workgroups); 0 where they do not apply."""
    if batch != 1 or M < 1 or skinny_strip_width(N, M) != 16:
        return 0
    strips = -(-N // 32)
    gmax = 1 if trans_b and M <= 32 else 4
    g = 1
    while g < gmax and strips * 2 * g <= 256 and M % (2 * g) == 0:
        g *= 2
    return g if strips * g >= (160 if trans_b else 128) else 0


# MFMA products per 32-deep chunk and output block, and bytes per operand element
METHODS = {
    "bf16x3": {"products": 3, "a_bytes": 4, "b_bytes": 4, "dtype": "bf16x3-f32acc"},
    "presplit": {"products": 3, "a_bytes": 4, "b_bytes": 4, "dtype": "bf16x3-f32acc"},
    "f16_full": {"products": 2, "a_bytes": 4, "b_bytes": 2, "dtype": "f16x2-f32acc"},
    "f16_base": {"products": 1, "a_bytes": 4, "b_bytes": 2, "dtype": "f16-f32acc"},
    "i16_scores": {"products": 4, "a_bytes": 2, "b_bytes": 2, "dtype": "i16-dual-f16-f32acc"},
    "split": {"products": 0, "a_bytes": 0, "b_bytes": 4, "dtype": "f32->bf16x2"},
}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    # about 0.2 s of warm-up at 8192^3: sub-millisecond launches reach their
    # steady rate only after ~0.1-0.2 s of back-to-back work
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="square8192")
    ap.add_argument("--method", default="bf16x3", choices=sorted(METHODS))
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--graph", action="store_true",
                    help="capture the K timed launches into one HIP graph and time one replay "
                         "of it, instead of issuing them one by one from Python (for "
                         "microsecond kernels under a tracer, whose per-launch host cost "
                         "would otherwise leave gaps between them)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target duration of the CPU oracle sample")
    ap.add_argument("--profile-summary", metavar="DIR",
                    help="print the markdown summary of a rocprofv3 run of this script "
                         "(no GPU work)")
    ap.add_argument("--out", metavar="PATH",
                    help="with --profile-summary: write the summary to PATH and record the "
                         "measured HBM bytes per launch in profiles/traffic.json")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed region, copy a 1 GiB buffer 3 times (a plain copy "
                         "kernel of known size, for scaling HBM byte counters)")
    return ap.parse_args()


# Rows of the panels of the short-K kernel (heal_gemm_panel.hip) per product.
PANEL_BM = {"bf16x3": 256, "i16_scores": 128}


def panel_applies(method, M, N, K, trans_b):
    """Whether the library runs the product on the short-K panel kernel: the
    conditions of panel_kernel_applies / scores_panel_applies for the dense,
    16-byte aligned operands bench.py allocates (the scores always take B
    as N x K rows)."""
    if method not in PANEL_BM or not (trans_b or method == "i16_scores"):
        return False
    es = 4 if method == "bf16x3" else 2
    return 0 < K <= 128 and (K * es) % 16 == 0 and N % 4 == 0 and M >= PANEL_BM[method]


def kernel_source_hash(instance):
    """Hash of the sources of the kernel an instance launches ("op": heal_gemm_op.hip)."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[instance]:
        with open(os.path.join(ROOT, "paper_2606_21023_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(key, instance):
    """HBM bytes per launch from counters, if measured on the current kernel sources.
    key: the workload name (bf16x3) or "method:workload"."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as f:
        t = json.load(f)
    e = t.get("workloads", {}).get(key)
    if not e or e.get("kernel_source_sha") != kernel_source_hash(instance):
        return None
    rf = e.get("read_factor", t.get("read_factor"))
    wf = e.get("write_factor", t.get("write_factor"))
    return e["fetch_kib"] * 1024.0 * rf + e["write_kib"] * 1024.0 * wf


def cpu_baseline(w, A, B, target_s, method="bf16x3", extra=None):
    """Time the CPU oracle of the method on the first R rows of the product, R
    grown to ~target_s.  A is M x K; B is K x N (bf16x3, presplit), the N x K
    weight (f16_*), or the N x K INT16 keys (i16_scores, A the INT16 queries)."""
    from oracle import oracle
    orc = oracle.default()
    if method in ("bf16x3", "presplit"):
        fn = lambda r: orc.gemm3(A[:r], B)
        N, K = B.shape[1], B.shape[0]
        what = "split of B included, FP64 accumulation"
    elif method in ("f16_full", "f16_base"):
        prods = METHODS[method]["products"]
        fn = lambda r: orc.gemm_f16w(A[:r], B, extra["e"], prods)
        N, K = B.shape
        what = "FP16 weight cast included, FP64 accumulation"
    else:
        fn = lambda r: orc.scores_i16(A[:r], B, extra["maxQ"], extra["maxK"], w.alpha)
        N, K = B.shape
        what = "dual-FP16 unpack included, FP64 accumulation"
    rows = 1
    while True:
        t0 = time.perf_counter()
        fn(rows)
        t = time.perf_counter() - t0
        if t >= target_s or rows >= A.shape[0]:
            break
        grow = max(2, int(target_s / max(t, 1e-3)))
        rows = min(A.shape[0], rows * grow)
    flops = 2.0 * rows * N * K
    return {"value": round(flops / t / 1e12, 5), "unit": "TFLOP/s", "cores": orc.num_threads(),
            "kind": "oracle", "seconds": round(t, 3),
            "sample": "%s oracle: first %d of %d rows of one %s product (%dx%dx%d of the "
                      "%d-entry batch), %s" % (method, rows, A.shape[0], w.name, rows, N, K,
                                                w.batch, what)}


def step_stats(run, steps, stream):
    """Per-launch durations from one HIP event before and after every launch,
    in a pass of its own before the warm-up launches (so that the timed
    region holds nothing but the launches).  Returns a function that, once
    the stream has drained, gives the median, minimum and standard error of
    the mean in ms: the pass does not wait for the GPU, so the warm-up
    launches follow it without an idle gap (a few ms idle put the clock
    back on its ramp)."""
    import torch
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record(stream)
    for i in range(steps):
        run(i)
        ev[i + 1].record(stream)

    def result():
        d = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(steps)], dtype=np.float64)
        sem = float(d.std(ddof=1) / math.sqrt(len(d))) if len(d) > 1 else 0.0
        return {"launches": steps, "median_ms": round(float(np.median(d)), 5),
                "min_ms": round(float(d.min()), 5), "sem_ms": round(sem, 6)}
    return result


def graph_of(steps, launch):
    """A HIP graph holding `steps` launches: launch(i, stream) issues launch
    i on the given stream (the capture stream while capturing)."""
    import ctypes
    import torch
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        cs = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        for i in range(steps):
            launch(i, cs)
    torch.cuda.synchronize()
    return g


def bench_split(args, w):
    """heal_split_f32 over the workload's B operand (K x N FP32 elements):
    4 bytes read and 2 + 2 bytes written per element, HBM-bound."""
    import ctypes
    import torch
    import paper_2606_21023_amd as heal
    from paper_2606_21023_amd import workloads as wl

    _, B = wl.make_inputs(w)
    X = np.ascontiguousarray(B[0] if B.ndim == 3 else B).reshape(-1)
    n = X.size
    alg_bytes = 8.0 * n
    dev = torch.device("cuda:0")
    n_rot = int(min(16, max(1, math.ceil(float(1 << 30) / alg_bytes))))
    xs = [torch.from_numpy(X).to(dev) for _ in range(n_rot)]
    # one (hi, lo) pair per timed launch, up to 64 GiB of outputs
    n_out = int(max(1, min(args.steps, (64 << 30) // (4 * n))))
    # written once before the timed region (no timed launch first-touches
    # its outputs)
    outs = [(torch.zeros(n, dtype=torch.uint16, device=dev),
             torch.zeros(n, dtype=torch.uint16, device=dev)) for _ in range(n_out)]
    torch.cuda.synchronize()
    L = heal.lib()
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    calls = [(xs[i % n_rot].data_ptr(), outs[i % n_out][0].data_ptr(),
              outs[i % n_out][1].data_ptr(), n)
             for i in range(max(args.steps, args.warmup, 1))]

    def run(i, s=sp):
        st = L.heal_split_f32(*calls[i % len(calls)], s)
        if st != 0:
            raise heal.HealError("launch failed with status %d" % st)

    # dispatch order: statistics pass, warmup launches, timed launches (the
    # statistics pass first also takes the GPU out of its idle clocks)
    stats = step_stats(run, args.steps, stream)
    for i in range(args.warmup):
        run(i)
    torch.cuda.synchronize()
    g = graph_of(args.steps, run) if args.graph else None
    e_start = torch.cuda.Event(enable_timing=True)
    e_end = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e_start.record(stream)
    if g is not None:
        g.replay()
    else:
        for i in range(args.steps):
            run(i)
    e_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    n_cmp = min(args.steps, n_out)
    identical = all(torch.equal(outs[j][0], outs[0][0]) and torch.equal(outs[j][1], outs[0][1])
                    for j in range(1, n_cmp))
    ms = e_start.elapsed_time(e_end) / args.steps
    gbs = alg_bytes / (ms * 1e-3) / 1e9
    traffic = measured_traffic("split:%s" % w.name, "split")
    roofline = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(gbs / HBM_PEAK_GBS, 4),
                "traffic": None if traffic is None else round(traffic),
                "kernel": "split_kernel<true> (8 elements per thread and step)",
                "per_launch": "8*n bytes (4 read, 2+2 written per element) = %.4g" % alg_bytes,
                "avg_launch_us": round(ms * 1e3, 2)}
    # Context for an MFMA-bound product: the vendor library's rate for ONE
    # plain bf16 GEMM of the same shape on this board (torch.matmul on bf16
    # copies of the inputs, hipBLASLt), timed after the timed region so that
    # it cannot change the measured launches.
    comparison = native()
    if roofline["bound"] == "mfma" and not batched:
        Ab = torch.from_numpy(A).to(dev).bfloat16()
        Bb = torch.from_numpy(B).to(dev).bfloat16()
        if w.trans_b:                       # B stored N x K
            Bb = Bb.t().contiguous()
        for _ in range(10):
            Ab @ Bb
        b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = max(20, min(100, args.steps))
        b0.record(torch.cuda.current_stream())
        for _ in range(reps):
            Ab @ Bb
        b1.record(torch.cuda.current_stream())
        torch.cuda.synchronize()
        ms_bf16 = b0.elapsed_time(b1) / reps
        tf_bf16 = w.flops / (ms_bf16 * 1e-3) / 1e12
        comparison.update({"torch_bf16_matmul_tflops": round(tf_bf16, 1),
                           "torch_bf16_matmul_frac_of_peak": round(tf_bf16 / BF16_DENSE_PEAK_TFLOPS, 4),
                           "torch_bf16_matmul_ms": round(ms_bf16, 4)})
        del Ab, Bb

    cpu = None
    if not args.no_cpu:
        from oracle import oracle
        orc = oracle.default()
        m = min(n, 1 << 20)
        while True:
            t1 = time.perf_counter()
            orc.split(X[:m])
            t = time.perf_counter() - t1
            if t >= args.cpu_seconds or m >= n:
                break
            m = min(n, m * max(2, int(args.cpu_seconds / max(t, 1e-3))))
        cpu = {"value": round(8.0 * m / t / 1e9, 3), "unit": "GB/s", "cores": orc.num_threads(),
               "kind": "oracle", "seconds": round(t, 3),
               "sample": "split oracle: first %d of the %d elements of the %s B operand"
                         % (m, n, w.name)}
    line = {
        "metric": "GB/s of heal_split_f32 (FP32 -> bf16 hi, lo planes); % of HBM peak; bit-repro",
        "value": round(gbs, 1),
        "unit": "GB/s (8 bytes per element)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": METHODS["split"]["dtype"],
        "data": "synthetic",
        "config": {"workload": w.name, "method": "split", "elements": n,
                   "inputs": "the B operand of: " + w.note, "operand_copies_rotated": n_rot},
        "timing": ("one replay of a HIP graph holding the K launches" if args.graph
                   else "K launches issued one by one"),
        "bit_repro": {"runs": n_cmp, "identical": identical,
                      "compared": ("both planes of every timed launch (one buffer pair each) "
                                   "against the first" if n_cmp == args.steps
                                   else "both planes of the last %d timed launches (one buffer "
                                   "pair each, reused in turn) against each other" % n_cmp)},
        "step_stats": stats(),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "build_id": heal.build_id(),
        "wall_s": round(wall, 3),
    }
    print(json.dumps(line))
    sys.stdout.flush()
    if args.copy_calibration:
        src = torch.ones(256 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()


def _kernel_base_name(full):
    """`void heal::(anonymous namespace)::gemm_large8_kernel<...>(...)` ->
    `gemm_large8_kernel`."""
    n = full.replace("(anonymous namespace)::", "").replace("void ", "", 1)
    for stop in ("<", "("):
        n = n.split(stop)[0]
    return n.split("::")[-1].strip()


def profile_summary(d, out=None):
    """Markdown summary of one rocprofv3 run of this script, from the
    directory DIR it wrote (printed on stdout):
      DIR/commands.txt  the rocprofv3 commands, one per line (they run
                        committed files only);
      DIR/trace/        --kernel-trace --stats CSV of the measured command,
                        DIR/trace.log its stdout (the bench.py JSON line);
      DIR/p1/, DIR/p2/  --pmc FETCH_SIZE / --pmc WRITE_SIZE CSV of a short
                        run with --copy-calibration (optional);
      DIR/p3/           --pmc of SQ and GRBM counters (optional).
    The measured kernel is the one the JSON line names; its dispatches come
    in the order of this script (statistics pass, warm-up, timed), so the
    average over the timed dispatches alone is reported next to the HIP-event
    time of the same launches.  With `out` (a path under profiles/) the
    summary is written there and the HBM bytes per launch go into
    profiles/traffic.json, tied to the kernel's current sources."""
    import csv
    import glob

    def rows(pattern):
        out = []
        for f in sorted(glob.glob(os.path.join(d, pattern))):
            with open(f) as fh:
                out += list(csv.DictReader(fh))
        return out

    with open(os.path.join(d, "commands.txt")) as f:
        commands = [c.strip() for c in f if c.strip()]
    with open(os.path.join(d, "trace.log")) as f:
        line_text = [l for l in f.read().splitlines() if l.startswith("{")][-1]
    line = json.loads(line_text)
    W, K = line["warmup"], line["steps"]
    kname = line["roofline"]["kernel"].split()[0].split("<")[0]
    cfg = line["config"]
    disp = sorted((r for r in rows("trace/*kernel_trace.csv")
                   if _kernel_base_name(r["Kernel_Name"]) == kname),
                  key=lambda r: int(r["Dispatch_Id"]))
    assert len(disp) == W + 2 * K, "%d dispatches of %s, expected %d" % (len(disp), kname,
                                                                         W + 2 * K)
    dur = np.array([int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in disp],
                   np.float64)
    second, timed = dur[:K], dur[K + W:]
    stats = rows("trace/*kernel_stats.csv")
    full = disp[0]["Kernel_Name"]
    L = ["# %s, %s, workload %s\n" % (kname, cfg["method"], cfg["workload"])]
    L.append("Commands, run from the repository root on an MI355X (rocprofv3 writes CSV under "
             "each -d directory); this summary is `python bench.py --profile-summary DIR` of "
             "their output directory:\n")
    L.append("```\n%s\n```\n" % "\n".join(commands))
    L.append("## Kernel statistics (`--kernel-trace --stats`)\n")
    L.append("| kernel | calls | average ns | min ns | max ns | % of GPU time |")
    L.append("|---|---|---|---|---|---|")
    for r in stats[:8]:
        n = r["Name"]
        if "Cijk" in n:
            t = n.split("_")[3] if n.count("_") > 3 else "?"
            n = ("hipBLASLt %s GEMM (torch.matmul comparison)"
                 % ("FP32" if t == "S" else "bf16" if t.startswith("B") else t))
        else:
            n = n[:100]
        L.append("| %s | %s | %.0f | %s | %s | %.2f |" % (n, r["Calls"], float(r["AverageNs"]),
                                                        r["MinNs"], r["MaxNs"],
                                                        float(r["Percentage"])))
    L.append("\nFull name of the measured kernel: `%s`\n" % full)
    L.append("## The timed launches\n")
    L.append("Dispatches of the measured kernel in the traced process, in order: %d of the "
             "per-launch statistics pass, %d warm-up, %d timed (%d in all).\n"
             % (K, W, K, len(disp)))
    L.append("| source | launches | mean us | min us | max us |")
    L.append("|---|---|---|---|---|")
    L.append("| bench.py HIP events, timed region / launches | %d | %.2f | | |"
             % (K, line["roofline"]["avg_launch_us"]))
    L.append("| rocprofv3, the timed dispatches | %d | %.2f | %.2f | %.2f |"
             % (K, timed.mean() / 1e3, timed.min() / 1e3, timed.max() / 1e3))
    L.append("| rocprofv3, the statistics pass | %d | %.2f | %.2f | %.2f |"
             % (K, second.mean() / 1e3, second.min() / 1e3, second.max() / 1e3))
    L.append("| rocprofv3, warm-up dispatches | %d | %s | | |"
             % (W, "%.2f" % (dur[K:K + W].mean() / 1e3) if W else "-"))
    rl = line["roofline"]
    per = rl["achieved"] * rl["avg_launch_us"]            # algorithmic units per launch x us
    frac_trace = per / (timed.mean() / 1e3) / rl["peak"]
    L.append("\nroofline.frac from the timed dispatches' trace average: %.4f (bench.py line: "
             "%.4f; %s bound, peak %s %s).\n" % (frac_trace, rl["frac"], rl["bound"], rl["peak"],
                                                rl["unit"]))
    fe = [r for r in rows("p1/*counter_collection.csv")
          if _kernel_base_name(r["Kernel_Name"]) == kname and r["Counter_Name"] == "FETCH_SIZE"]
    wr = [r for r in rows("p2/*counter_collection.csv")
          if _kernel_base_name(r["Kernel_Name"]) == kname and r["Counter_Name"] == "WRITE_SIZE"]
    traffic = None
    if fe and wr:
        cf = sorted((r for r in rows("p1/*counter_collection.csv")
                     if "copyBuffer" in r["Kernel_Name"] and r["Counter_Name"] == "FETCH_SIZE"),
                    key=lambda r: int(r["Dispatch_Id"]))[-3:]
        cw = sorted((r for r in rows("p2/*counter_collection.csv")
                     if "copyBuffer" in r["Kernel_Name"] and r["Counter_Name"] == "WRITE_SIZE"),
                    key=lambda r: int(r["Dispatch_Id"]))[-3:]
        assert len(cf) == 3 and len(cw) == 3, "the three 1 GiB calibration copies"
        fetch = np.mean([float(r["Counter_Value"]) for r in fe])
        write = np.mean([float(r["Counter_Value"]) for r in wr])
        cfv = np.mean([float(r["Counter_Value"]) for r in cf])
        cwv = np.mean([float(r["Counter_Value"]) for r in cw])
        rf, wf = 1048576.0 / cfv, 1048576.0 / cwv
        traffic = fetch * 1024 * rf + write * 1024 * wf
        L.append("## HBM traffic per dispatch\n")
        L.append("| counter | mean KiB per dispatch | dispatches | scale (1 GiB copy) | bytes |")
        L.append("|---|---|---|---|---|")
        L.append("| FETCH_SIZE | %.1f | %d | x%.4f | %.4g |" % (fetch, len(fe), rf,
                                                            fetch * 1024 * rf))
        L.append("| WRITE_SIZE | %.1f | %d | x%.4f | %.4g |" % (write, len(wr), wf,
                                                            write * 1024 * wf))
        L.append("\nCalibration: the same process copies a 1 GiB buffer three times after its "
                 "timed region; FETCH_SIZE reads %.0f KiB and WRITE_SIZE %.0f KiB per copy, so "
                 "reads are scaled by %.4f and writes by %.4f.  Traffic %.4g bytes per launch; "
                 "algorithmic: %s.\n" % (cfv, cwv, rf, wf, traffic, rl["per_launch"]))
    sq = [r for r in rows("p3/*counter_collection.csv")
          if _kernel_base_name(r["Kernel_Name"]) == kname]
    if sq:
        acc = {}
        for r in sq:
            acc.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
        L.append("## SQ and GRBM counters, mean per dispatch\n")
        L.append("| counter | mean | dispatches |")
        L.append("|---|---|---|")
        for c in sorted(acc):
            L.append("| %s | %.6g | %d |" % (c, np.mean(acc[c]), len(acc[c])))
        if "SQ_VALU_MFMA_BUSY_CYCLES" in acc and "GRBM_GUI_ACTIVE" in acc:
            busy = np.mean(acc["SQ_VALU_MFMA_BUSY_CYCLES"])
            act = np.mean(acc["GRBM_GUI_ACTIVE"])
            L.append("\nMFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 XCDs x 1024 "
                     "SIMDs) = %.3f; clock = GRBM_GUI_ACTIVE / 8 / trace mean = %.2f GHz.\n"
                     % (busy / (act / 8 * 1024), act / 8 / timed.mean()))
    # further counter passes (DIR/p4, DIR/p5, ...): cache, request-size,
    # latency and MFMA-operation counters of the measured kernel
    extra = {}
    for sub in sorted(glob.glob(os.path.join(d, "p[4-9]"))):
        for r in rows(os.path.join(os.path.basename(sub), "*counter_collection.csv")):
            if _kernel_base_name(r["Kernel_Name"]) == kname:
                extra.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    if extra:
        L.append("## Further counters (cache, request sizes, latency, MFMA operations), mean per "
                 "dispatch\n")
        L.append("| counter | mean | dispatches |")
        L.append("|---|---|---|")
        for c in sorted(extra):
            L.append("| %s | %.6g | %d |" % (c, np.mean(extra[c]), len(extra[c])))
        m = {c: np.mean(v) for c, v in extra.items()}
        notes = []
        if "TCC_HIT_sum" in m and "TCC_MISS_sum" in m:
            notes.append("L2 hit rate TCC_HIT / (TCC_HIT + TCC_MISS) = %.3f"
                         % (m["TCC_HIT_sum"] / max(1.0, m["TCC_HIT_sum"] + m["TCC_MISS_sum"])))
        if "TCC_EA0_RDREQ_sum" in m and "TCC_EA0_RDREQ_128B_sum" in m:
            notes.append("share of L2-to-memory read requests that are 128-byte: %.3f"
                         % (m["TCC_EA0_RDREQ_128B_sum"] / max(1.0, m["TCC_EA0_RDREQ_sum"])))
        if "TCP_TCC_READ_REQ_LATENCY_sum" in m and "TCP_TCC_READ_REQ_sum" in m:
            notes.append("mean L1-to-L2 read latency TCP_TCC_READ_REQ_LATENCY / TCP_TCC_READ_REQ "
                         "= %.0f cycles" % (m["TCP_TCC_READ_REQ_LATENCY_sum"]
                                            / max(1.0, m["TCP_TCC_READ_REQ_sum"])))
        # matrix-core work: the MOPS counters count multiply-add operations in
        # units of 512 flops; the product does P 16-bit products of 2MNK each
        products = {"bf16x3": (3, "BF16"), "presplit": (3, "BF16"), "f16_full": (2, "F16"),
                    "f16_base": (1, "F16"), "i16_scores": (4, "F16")}.get(cfg["method"])
        if products and "SQ_INSTS_VALU_MFMA_MOPS_" + products[1] in m:
            P, T = products
            flops = 512.0 * m["SQ_INSTS_VALU_MFMA_MOPS_" + T]
            want = P * 2.0 * cfg["M"] * cfg["N"] * cfg["K"] * cfg.get("batch", 1)
            r = flops / want
            notes.append("MFMA work: SQ_INSTS_VALU_MFMA_MOPS_%s x 512 = %.4g flops per dispatch "
                         "= %.4f x %d product%s of 2MNK (%.4g%s)"
                         % (T, flops, r, P, "s" if P > 1 else "", want,
                            "; the excess is the zero padding of partial tiles"
                            if r > 1.00005 else ", exactly"))
        if notes:
            L.append("\n" + "; ".join(notes) + ".\n")
    L.append("## bench.py line of the traced run\n")
    L.append("```\n%s\n```" % line_text)
    text = "\n".join(L) + "\n"
    if out is None:
        sys.stdout.write(text)
        return text
    with open(out, "w") as f:
        f.write(text)
    if traffic is not None:
        inst = {"bf16x3": None, "split": "split"}.get(cfg["method"], "op")
        if cfg["method"] != "split" and panel_applies(cfg["method"], cfg["M"], cfg["N"], cfg["K"],
                                                      cfg.get("trans_b", False)):
            inst = "panel"
        elif inst is None:
            import paper_2606_21023_amd as heal
            inst = heal.select_instance(cfg["M"], cfg["N"])
        key = cfg["workload"] if cfg["method"] == "bf16x3" else "%s:%s" % (cfg["method"],
                                                                           cfg["workload"])
        t = {"workloads": {}}
        if os.path.exists(TRAFFIC_FILE):
            with open(TRAFFIC_FILE) as f:
                t = json.load(f)
        t["workloads"][key] = {"fetch_kib": round(float(fetch), 1),
                               "write_kib": round(float(write), 1), "dispatches": len(fe),
                               "read_factor": round(rf, 4), "write_factor": round(wf, 4),
                               "profile": os.path.relpath(os.path.abspath(out), ROOT),
                               "kernel_source_sha": kernel_source_hash(inst)}
        with open(TRAFFIC_FILE, "w") as f:
            json.dump(t, f, indent=1)
    return text


def main():
    args = parse()
    if args.profile_summary:
        profile_summary(args.profile_summary, args.out)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the compensated GEMM is measured on one "
              "GPU's share and there is no multi-GPU path (--gpus %d requested)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2606_21023_amd as heal
    from paper_2606_21023_amd import workloads as wl

    heal.check_build()      # refuse a libheal.so built from other sources
    method = args.method
    w = wl.WORKLOADS[args.workload]
    if method == "split":
        return bench_split(args, w)
    if method == "i16_scores" and w.name != "attn_scores":
        print("--method i16_scores runs on the attn_scores workload", file=sys.stderr)
        sys.exit(2)
    if method in ("presplit", "f16_full", "f16_base") and (w.batch > 1 or w.trans_b):
        print("--method %s runs on the linear-layer workloads" % method, file=sys.stderr)
        sys.exit(2)
    A, B = wl.make_inputs(w)
    torch.cuda.init()
    dev = torch.device("cuda:0")
    batched = w.trans_b or w.batch > 1
    meta = METHODS[method]

    # Operand preparation outside the timed region (done once per weight or
    # cache entry in use): FP16 weight packing, B pre-split, INT16 codes.
    extra = {}
    if method in ("f16_full", "f16_base"):
        Wh = np.ascontiguousarray(B.T)            # the N x K weight of a linear layer
        extra["e"] = heal.heal_f16_weight_exponent(float(np.abs(Wh).max()))
    if method == "i16_scores":
        q, mq = heal.heal_quantize_i16(torch.from_numpy(A).to(dev))
        k, mk = heal.heal_quantize_i16(torch.from_numpy(B).to(dev))
        torch.cuda.synchronize()
        Aq, Bq = q.cpu().numpy(), k.cpu().numpy()
        extra["maxQ"], extra["maxK"] = float(mq.item()), float(mk.item())

    # algorithmic bytes per launch: A and B read once in the method's storage
    # format, C written once in FP32
    b_elems = w.K * w.N
    if method in ("presplit", "f16_full", "f16_base"):
        planes = 2 if method == "presplit" else 1
        b_elems = heal.heal_packed_size(w.K, w.N, planes) // planes   # padded to 16 x 32 blocks
    alg_bytes = float(w.batch) * (meta["a_bytes"] * w.M * w.K + meta["b_bytes"] * b_elems +
                                  4.0 * w.M * w.N)

    # Rotate through copies of the operands so that HBM-bound shapes are not
    # served from the 256 MB Infinity Cache: at least 1 GiB of inputs in turn.
    n_rot = int(min(16, max(1, math.ceil(float(1 << 30) / alg_bytes))))
    sets = []
    for _ in range(n_rot):
        if method == "i16_scores":
            Ad, Bd = torch.from_numpy(Aq).to(dev), torch.from_numpy(Bq).to(dev)
            sets.append((Ad, Bd, mq.clone(), mk.clone()))
            continue
        Ad = torch.from_numpy(A).to(dev)
        if method in ("f16_full", "f16_base"):
            Bd = heal.heal_pack_f16_weight(torch.from_numpy(Wh).to(dev), extra["e"])
        elif method == "presplit":
            Bd = heal.heal_presplit_b(torch.from_numpy(B).to(dev))
        else:
            Bd = torch.from_numpy(B).to(dev)
        sets.append((Ad, Bd))
    # One output buffer per timed launch (up to 64 GiB of outputs), so that
    # every timed launch's whole output can be compared afterwards.
    c_shape = (w.batch, w.M, w.N) if batched else (w.M, w.N)
    c_bytes = 4 * w.batch * w.M * w.N
    n_out = int(max(1, min(args.steps, (64 << 30) // c_bytes)))
    # written once before the timed region, so that no timed launch is the
    # first to touch its output's pages
    outs = [torch.zeros(c_shape, dtype=torch.float32, device=dev) for _ in range(n_out)]
    torch.cuda.synchronize()

    # MI355X native FP32 GEMM on the same (FP32) inputs, TF32 off; it runs
    # first, so that the GPU has left its idle clocks before the warm-up
    # launches of the product (a few warm-up launches of a 2 ms kernel are
    # otherwise still on the clock ramp)
    torch.backends.cuda.matmul.allow_tf32 = False
    torch.set_float32_matmul_precision("highest")
    Af, Bf = torch.from_numpy(A).to(dev), torch.from_numpy(B).to(dev)
    mm = (lambda: torch.matmul(Af, Bf.transpose(-1, -2))) if w.trans_b else (lambda: Af @ Bf)
    for _ in range(3):
        mm()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = max(3, min(20, args.steps))
    e0.record(torch.cuda.current_stream())
    for _ in range(reps):
        mm()
    e1.record(torch.cuda.current_stream())
    # no wait here: the product's launches queue behind these, so the GPU
    # does not idle in between; the time is read after the timed region
    def native():
        ms = e0.elapsed_time(e1) / reps
        return {"torch_fp32_matmul_tflops": round(w.flops / (ms * 1e-3) / 1e12, 2),
                "torch_fp32_matmul_ms": round(ms, 4)}
    del Af, Bf

    # Launch through the C ABI with pre-built arguments, so that the timed
    # loop measures the kernels rather than argument marshalling: every step
    # is one library call on the current stream.
    import ctypes
    L = heal.lib()
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)

    def make_call(i):
        st, Cd = sets[i % n_rot], outs[i % n_out]
        Ad, Bd = st[0], st[1]
        if method == "i16_scores":
            cargs = (w.M, w.N, w.K, Ad.data_ptr(), w.K, w.M * w.K, st[2].data_ptr(), Bd.data_ptr(),
                     w.K, w.N * w.K, st[3].data_ptr(), ctypes.c_float(w.alpha), Cd.data_ptr(),
                     w.N, w.M * w.N, w.batch)
            return L.heal_scores_i16, cargs
        if method in ("f16_full", "f16_base"):
            cargs = (meta["products"], w.M, w.N, w.K, Ad.data_ptr(), w.K, Bd.data_ptr(),
                     extra["e"], Cd.data_ptr(), w.N)
            return L.heal_gemm_f16w, cargs
        if method == "presplit":
            cargs = (w.M, w.N, w.K, Ad.data_ptr(), w.K, Bd.data_ptr(), Cd.data_ptr(), w.N)
            return L.heal_gemm_f32_presplit, cargs
        if batched:
            lda, ldb, ldc = w.K, (w.K if w.trans_b else w.N), w.N
            cargs = (w.M, w.N, w.K, ctypes.c_float(w.alpha), Ad.data_ptr(), lda, w.M * w.K,
                     Bd.data_ptr(), ldb, w.N * w.K, 1 if w.trans_b else 0, Cd.data_ptr(), ldc,
                     w.M * w.N, w.batch)
            return L.heal_gemm_f32_strided_batched, cargs
        cargs = (w.M, w.N, w.K, Ad.data_ptr(), Bd.data_ptr(), Cd.data_ptr(), w.K, w.N, w.N)
        return L.heal_gemm_f32, cargs

    calls = [make_call(i) for i in range(max(args.steps, args.warmup, 1))]

    def run(i, s=sp):
        fn, cargs = calls[i % len(calls)]
        st = fn(*cargs, s)
        if st != 0:
            raise heal.HealError("launch failed with status %d" % st)

    # dispatch order of the kernel: the launches of the per-launch statistics
    # pass, the warm-up launches, the timed launches.  The FP32 comparison
    # and the statistics pass before the warm-up take the GPU out of its
    # idle clocks, and nothing waits for the GPU between them and the
    # warm-up: after even 4 ms idle an 8192^3 launch takes 2.4-2.6 ms (2.5-3.2
    # after 40 ms) and settles near 2.2 ms only after some 50-100 ms of
    # back-to-back work.
    stats = step_stats(run, args.steps, stream)
    for i in range(args.warmup):
        run(i)
    torch.cuda.synchronize()
    # --graph: the timed launches captured once into a HIP graph (not timed),
    # so that the timed region is the kernels back to back rather than the
    # rate at which Python issues them (graph replays measured 1-3% slower
    # than eager launches for the millisecond kernels)
    g = graph_of(args.steps, run) if args.graph else None

    e_start = torch.cuda.Event(enable_timing=True)
    e_end = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e_start.record(stream)
    if g is not None:
        g.replay()
    else:
        for i in range(args.steps):
            run(i)
    e_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # every timed launch's whole output against the first timed launch's
    n_cmp = min(args.steps, n_out)
    ref = outs[0].view(torch.int32)
    identical = all(bool(torch.equal(outs[j].view(torch.int32), ref)) for j in range(1, n_cmp))
    total_ms = e_start.elapsed_time(e_end)
    ms_per_step = total_ms / args.steps
    # launches run back to back on one stream: the mean launch duration is
    # the timed region over the number of launches
    avg_launch_ms = ms_per_step

    flops = w.flops
    value = flops / (ms_per_step * 1e-3) / 1e12
    mfma_flops = meta["products"] * flops
    t_mfma = mfma_flops / (BF16_DENSE_PEAK_TFLOPS * 1e12)
    t_hbm = alg_bytes / (HBM_PEAK_GBS * 1e9)
    instance = heal.select_instance(w.M, w.N)
    if panel_applies(method, w.M, w.N, w.K, w.trans_b):
        key = w.name if method == "bf16x3" else "%s:%s" % (method, w.name)
        traffic = measured_traffic(key, "panel")
        kernel = ("gemm_panel_kernel<%s> (%d-row A panels in LDS, 4 waves of 32 columns, "
                  "B fragments straight to registers)" % (method, PANEL_BM[method]))
    elif method == "bf16x3":
        traffic = measured_traffic(w.name, instance)
        kernel = KERNEL_NAMES.get(instance, "?")
        if instance == 3:
            groups = skinny_row_groups(w.N, w.M, w.trans_b, w.batch)
            if groups:
                kernel = ("gemm_skinny_kernel (32-column strips, the rows in %d group%s, M <= 64)"
                          % (groups, "s" if groups > 1 else ""))
            else:
                kernel = ("gemm_skinny_kernel (%d-column strips, M <= 64)"
                          % skinny_strip_width(w.N, w.M))
    else:
        traffic = measured_traffic("%s:%s" % (method, w.name), "op")
        label = OP_INSTANCE_NAMES.get(instance, "?")
        kname = "gemm_op_kernel"
        sw = skinny_strip_width(w.N, w.M) if instance == 3 else 0
        if instance == 3 and sw in (32, 64, 128):
            label = "skinny M<=64, %d-column tiles, loader waves beside the MFMA waves" % sw
        elif instance == 3 and method != "i16_scores" and sw == 16:
            # M <= 64 with too few wider tiles: the streamed narrow tiles
            # (loader waves and one computing wave, 16 columns)
            kname = "gemm_op_stream_kernel"
            label = "narrow 16-column tiles, loader waves + one MFMA wave, LDS ring"
        elif instance == 1 and method != "i16_scores":
            # 16-byte aligned rows: the hand-scheduled kernel, 224 columns
            # where that takes fewer rounds of one workgroup per CU
            cus = torch.cuda.get_device_properties(0).multi_processor_count
            def cost(bn):
                wgs = -(-w.M // 256) * -(-w.N // bn) * w.batch
                return -(-wgs // cus) * bn
            bn = 224 if method != "f16_base" and cost(224) < cost(256) else 256
            kname = "gemm_op8_kernel"
            label = "large 256x%d, 8 waves of 64x%d, hand-scheduled" % (bn, bn // 2)
        kernel = "%s<%s> (%s)" % (kname, method, label)
    mfma_dtype = "bf16" if meta["products"] == 3 else "f16"
    if t_mfma >= t_hbm:
        achieved = mfma_flops / (avg_launch_ms * 1e-3) / 1e12
        roofline = {"bound": "mfma", "achieved": round(achieved, 2),
                    "peak": BF16_DENSE_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(achieved / BF16_DENSE_PEAK_TFLOPS, 4)}
        per_launch = "%d*2*M*N*K*batch %s MFMA flops = %.4g" % (meta["products"], mfma_dtype,
                                                               mfma_flops)
    else:
        achieved = alg_bytes / (avg_launch_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4)}
        per_launch = ("(%d*M*K + %d*K*N + 4*M*N)*batch bytes = %.4g"
                      % (meta["a_bytes"], meta["b_bytes"], alg_bytes))
    roofline.update({"traffic": None if traffic is None else round(traffic),
                     "kernel": kernel, "per_launch": per_launch,
                     "avg_launch_us": round(avg_launch_ms * 1e3, 2)})

    # Context for an MFMA-bound product: the vendor library's rate for ONE
    # plain bf16 GEMM of the same shape on this board (torch.matmul on bf16
    # copies of the inputs, hipBLASLt), timed after the timed region so that
    # it cannot change the measured launches.
    comparison = native()
    if roofline["bound"] == "mfma" and not batched:
        Ab = torch.from_numpy(A).to(dev).bfloat16()
        Bb = torch.from_numpy(B).to(dev).bfloat16()
        if w.trans_b:                       # B stored N x K
            Bb = Bb.t().contiguous()
        for _ in range(10):
            Ab @ Bb
        b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = max(20, min(100, args.steps))
        b0.record(torch.cuda.current_stream())
        for _ in range(reps):
            Ab @ Bb
        b1.record(torch.cuda.current_stream())
        torch.cuda.synchronize()
        ms_bf16 = b0.elapsed_time(b1) / reps
        tf_bf16 = w.flops / (ms_bf16 * 1e-3) / 1e12
        comparison.update({"torch_bf16_matmul_tflops": round(tf_bf16, 1),
                           "torch_bf16_matmul_frac_of_peak": round(tf_bf16 / BF16_DENSE_PEAK_TFLOPS, 4),
                           "torch_bf16_matmul_ms": round(ms_bf16, 4)})
        del Ab, Bb

    cpu = None
    if not args.no_cpu:
        if method == "i16_scores":
            cpu = cpu_baseline(w, Aq[0], Bq[0], args.cpu_seconds, method, extra)
        elif method in ("f16_full", "f16_base"):
            cpu = cpu_baseline(w, A, Wh, args.cpu_seconds, method, extra)
        else:
            Ah = A[0] if batched else A
            Bh = np.ascontiguousarray(B[0].T) if w.trans_b else (B[0] if batched else B)
            cpu = cpu_baseline(w, Ah, Bh, args.cpu_seconds, method, extra)

    names = {"bf16x3": "compensated GEMM", "presplit": "compensated GEMM, pre-split B",
             "f16_full": "HEAL-Full FP16 GEMM", "f16_base": "HEAL-Base FP16 GEMM",
             "i16_scores": "INT16 dual-FP16 attention scores"}
    line = {
        "metric": "FP32-equiv TFLOP/s of %s; %% of bf16 MFMA peak/3; bit-repro" % names[method],
        "value": round(value, 2),
        "unit": "TFLOP/s (FP32-equivalent, 2MNK/t)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": meta["dtype"],
        "data": "synthetic",
        "config": {"workload": w.name, "method": method, "M": w.M, "N": w.N, "K": w.K,
                   "batch": w.batch, "trans_b": w.trans_b, "alpha": w.alpha, "seed": w.seed,
                   "inputs": w.note, "operand_copies_rotated": n_rot},
        "pct_of_bf16_peak_div3": round(100.0 * value / (BF16_DENSE_PEAK_TFLOPS / 3), 2),
        "hbm_gbs": round(alg_bytes / (ms_per_step * 1e-3) / 1e9, 1),
        "timing": ("one replay of a HIP graph holding the K launches" if args.graph
                   else "K launches issued one by one"),
        "bit_repro": {"runs": n_cmp, "identical": identical,
                      "compared": ("whole output of every timed launch (one buffer each) "
                                   "against the first" if n_cmp == args.steps
                                   else "whole output of the last %d timed launches (one buffer "
                                   "each, reused in turn) against each other" % n_cmp)},
        "step_stats": stats(),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "comparison": comparison,
        "build_id": heal.build_id(),
        "wall_s": round(wall, 3),
    }
    if "e" in extra:
        line["config"]["weight_exponent"] = extra["e"]
    print(json.dumps(line))
    sys.stdout.flush()

    if args.copy_calibration:
        src = torch.ones(256 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()


if __name__ == "__main__":
    main()
