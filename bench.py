"""Benchmark: throughput of the structured-derivatives empirical NTK on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

A step is one full NTK evaluation Theta(X1, X2) (every stage of the path: forward
pass keeping layer inputs, batched cotangent backward, Grams, fused contraction)
on the synthetic workload, with all inputs already resident in HBM.  The default
workload is the ReLU MLP of depth 8 and width 2048 (input 3072, O = 10,
X1 and X2 of 512 samples each).  One JSON line is printed on stdout.

The timed steps are launched eagerly.  --graph times replays of the HIP graph the library
records of one ntk_compute instead (NTK_OPT_GRAPH: every kernel of the step runs again on
every replay, on the same device buffers; the graph is recorded by one untimed call before the
warm-up, like the handle's set-up).

The steps that give the throughput run without per-kernel events.  roofline: the dominant
kernel class (largest time share) is then timed live with HIP events recorded by the library
around each launch on its own stream, over as many further eager steps (ms_per_step_profiled
is their mean step time);
`achieved` = its algorithmic FLOPs per launch / average launch time.
cpu_baseline: the fp64 Jacobian-contraction oracle on a bounded sample of the same
workload (a few samples of X1 x X2, all outputs), timed on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "NTK entries/sec (N1·N2·O²) and fp32 MFMA TFLOP/s, FCN depth 8 width 2048"
FP32_MFMA_PEAK_TFLOPS = 157.3      # MI355X dense fp32 matrix peak
FP64_MFMA_PEAK_TFLOPS = 78.6       # MI355X dense fp64 matrix peak (the forward passes)
HBM_PEAK_GBS = 8000.0

# kernel class -> stage of the FLOP counter
STAGE_OF = {"dense_fwd": "forward", "dense_bwd": "backward", "gram": "gram",
            "ntk_fcn": "contraction", "conv_fwd": "forward", "conv_bwd": "backward",
            "conv_wgrad": "wgrad", "ntk_splitk": "contraction", "conv_pairsum": "pairsum",
            "ntk_diag": "contraction", "struct_fwd": "struct_forward",
            "struct_bwd": "struct_backward", "struct_wgrad": "struct_wgrad"}
# kernel class -> stage of the NTK-vector product's counter
VP_STAGE_OF = {"dense_fwd": "forward", "dense_bwd": "vjp_backward", "gram": "gram_products",
               "conv_fwd": "forward_and_jvp", "conv_bwd": "vjp_backward",
               "conv_wgrad": "weight_cotangent"}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="relu_mlp_d8_w2048")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--output", default="full", choices=["full", "trace", "logit"],
                    help="output-axis variant (the default is the full O x O block)")
    ap.add_argument("--batch", default="full", choices=["full", "diagonal"],
                    help="batch-axis variant (diagonal: Theta(x1_n, x2_n) only)")
    ap.add_argument("--logit", type=int, default=0, help="o* of --output logit")
    ap.add_argument("--method", default="structured", choices=["structured", "jacobian"],
                    help="structured derivatives (default) or the Jacobian-contraction baseline")
    ap.add_argument("--conv-order", default="auto", choices=["auto", "outside_in", "inside_out"],
                    help="contraction order of the 3x3 and pointwise convolutions (auto: the cost model)")
    ap.add_argument("--op", default="ntk", choices=["ntk", "vp"],
                    help="ntk: Theta(X1, X2); vp: the NTK-vector product Theta(X1, X2) v")
    ap.add_argument("--graph", action="store_true",
                    help="time the NTK steps (op ntk, structured method) replayed from a HIP graph "
                         "(NTK_OPT_GRAPH); the per-kernel timing then comes from as many further "
                         "eager steps")
    ap.add_argument("--samples", type=int, default=0,
                    help="use only the first N samples of X1 and of X2 (0: the whole workload)")
    ap.add_argument("--cpu-samples", type=int, default=6,
                    help="samples per side of the oracle's bounded sample")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain device copy of known size (for HBM counter scaling)")
    return ap.parse_args()


def sources_sha16(kernel_file="kernels_fcn.hip"):
    """Hash of the sources a kernel is compiled from: its .hip file and every shared header."""
    import glob
    import hashlib
    csrc = os.path.join(ROOT, "paper_2206_08720_amd", "csrc")
    files = [os.path.join(csrc, kernel_file)] + sorted(glob.glob(os.path.join(csrc, "*.hpp")))
    h = hashlib.sha256()
    for f in files:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(name, kernel):
    """HBM bytes per launch from the committed FETCH_SIZE/WRITE_SIZE record, or None when the
    record is for another kernel/workload or the kernel sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"{name}_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("kernel") != kernel or \
            rec.get("sources_sha256_16") != sources_sha16(rec.get("kernel_source", "kernels_fcn.hip")):
        return None
    return (rec["fetch_size_kib_per_launch"] * rec["fetch_scale"]
            + rec["write_size_kib_per_launch"] * rec["write_scale"]) * 1024.0


def measured_mfma_busy(name, kernel):
    """Fraction of the class's kernel time the matrix cores were busy, from the committed
    SQ_VALU_MFMA_BUSY_CYCLES / SQ_BUSY_CU_CYCLES record (a CU has 4 SIMDs: busy fraction =
    MFMA-busy cycles / (4 x CU-busy cycles)), or None when the record is for another
    kernel/workload or the kernel sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"{name}_mfma_busy.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    cls = rec.get("classes", {}).get(kernel)
    if cls is None or cls.get("sources_sha256_16") != sources_sha16(cls.get("kernel_source", "kernels_fcn.hip")):
        return None
    return cls["mfma_busy"]


def cpu_baseline(name, n, n1_full, n2_full):
    """Time the fp64 Jacobian-contraction oracle on Theta(X1[:n], X2[:n]) (after an untimed
    one-sample call), and extrapolate to the full Theta: the per-sample part (forward, O
    backward passes, Jacobian rows) linear in the samples, the contraction 2 N1 N2 O^2 P
    FLOPs at the host's fp64 GEMM rate measured here."""
    import numpy as np
    import oracle
    import workloads as wl
    from threadpoolctl import threadpool_info
    spec, params, X1, X2 = wl.make_workload(name)
    oracle.ntk_jc(spec, params, X1[:1], X2[:1])          # warm-up (page faults, BLAS threads)
    t0 = time.perf_counter()
    th = oracle.ntk_jc(spec, params, X1[:n], X2[:n])
    dt = time.perf_counter() - t0
    A = np.random.default_rng(0).standard_normal((2048, 2048))
    gemm_s = []
    for _ in range(3):
        t1 = time.perf_counter()
        A @ A
        gemm_s.append(time.perf_counter() - t1)
    rate = 2 * 2048 ** 3 / min(gemm_s)
    O, P = th.shape[2], oracle.param_count(spec)
    per_pair = 2.0 * O * O * P / rate                    # contraction seconds per sample pair
    per_sample = max(0.0, (dt - per_pair * n * n) / (2 * n))
    full_s = per_sample * (n1_full + n2_full) + per_pair * n1_full * n2_full
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": th.size / dt, "unit": "NTK entries/s", "cores": threads, "kind": "oracle",
            "extrapolated_full_theta_s": full_s,
            "sample": f"Theta(X1[:{n}], X2[:{n}]) of {name}, all {O} outputs ({th.size} entries) "
                      f"by fp64 Jacobian contraction in {dt:.1f} s; host "
                      f"{platform.processor() or platform.machine()}, {os.cpu_count()} logical "
                      f"CPUs. extrapolated_full_theta_s (extrapolated, not measured): per-sample "
                      f"part {per_sample:.3g} s x (N1 + N2) + contraction 2 N1 N2 O^2 P FLOPs "
                      f"(P = {P}) at the measured fp64 GEMM rate {rate / 1e9:.0f} GFLOP/s"}


def copy_calibration():
    import torch
    n = 256 << 20  # 1 GiB of float32
    a = torch.empty(n, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": n * 4, "copy_calibration_bytes_written": n * 4}))


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the NTK's output blocks "
              "are independent and would shard over a 2-D grid of GPUs, but the library runs on one GPU "
              "per process.", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import workloads as wl
    from paper_2206_08720_amd import _lib
    from paper_2206_08720_amd.flops import ntk_entries, ntk_flops, vp_flops
    from paper_2206_08720_amd.ntk import NTK

    if args.copy_calibration:
        copy_calibration()
        return
    torch.cuda.set_device(0)
    name = args.workload
    spec, params, X1, X2 = wl.make_workload(name)
    if args.samples:
        aliased = X2 is X1
        X1 = X1[:args.samples]
        X2 = X1 if aliased else X2[:args.samples]
    sym = X2 is X1
    dev = [torch.from_numpy(p).cuda() for p in params]
    x1 = torch.from_numpy(X1).cuda()
    x2 = x1 if sym else torch.from_numpy(X2).cuda()
    n1, n2 = X1.shape[0], X2.shape[0]
    O = spec["layers"][-1]["out"]
    h = NTK(spec, n1, n2)
    h.set_variant(args.output, args.batch, args.logit)
    h.set_method(args.method)
    h.set_option(_lib.NTK_OPT_CONV_ORDER, {"auto": _lib.NTK_CONV_ORDER_AUTO,
                                           "outside_in": _lib.NTK_CONV_ORDER_OUTSIDE_IN,
                                           "inside_out": _lib.NTK_CONV_ORDER_INSIDE_OUT}[args.conv_order])
    stream = torch.cuda.current_stream()
    if args.op == "vp":
        vvec = torch.from_numpy(np.random.default_rng(0).standard_normal((n2, O)).astype(np.float32)).cuda()
        out = torch.empty((n1, O), dtype=torch.float32, device="cuda")

        def step():
            h.vector_product(dev, x1, x2, vvec, out=out)
    else:
        out = torch.empty(h.out_shape(n1, n2), dtype=torch.float32, device="cuda")

        def step():
            h.compute(dev, x1, x2, out=out)

    def timed(k, profiled):
        """Run k steps between HIP events on the stream; (mean ms, sorted per-step ms, wall s,
        per-kernel profile or None)."""
        if profiled:
            h.profile_read()                       # drop anything recorded so far
            h.profile_enable(True)
        torch.cuda.synchronize()
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(k + 1)]
        t0 = time.perf_counter()
        evs[0].record(stream)
        for i in range(k):
            step()
            evs[i + 1].record(stream)
        torch.cuda.synchronize()
        wall_s = time.perf_counter() - t0
        per = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(k))
        prof_ = None
        if profiled:
            prof_ = h.profile_read()
            h.profile_enable(False)
        return evs[0].elapsed_time(evs[-1]) / k, per, wall_s, prof_

    use_graph = args.graph and args.op == "ntk" and args.method == "structured"
    if use_graph:
        h.set_option(_lib.NTK_OPT_GRAPH, 1)
        step()                                  # records the graph (set-up, not a warm-up)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # the throughput comes from steps without the per-kernel events (each event record costs a
    # few microseconds of host and GPU time, a third of a step on the smallest workloads); the
    # kernel classes are then timed over as many eager steps with the library's HIP events
    ms, step_ms, wall, _ = timed(args.steps, profiled=False)
    if use_graph:
        h.set_option(_lib.NTK_OPT_GRAPH, 0)
        step()
    ms_profiled, _, _, prof = timed(args.steps, profiled=True)
    ms_median = step_ms[len(step_ms) // 2] if len(step_ms) % 2 else \
        0.5 * (step_ms[len(step_ms) // 2 - 1] + step_ms[len(step_ms) // 2])

    entries = ntk_entries(spec, n1, n2, args.output, args.batch)
    fl = ntk_flops(spec, n1, n2, symmetric=sym, output=args.output, batch=args.batch,
                   method=args.method, order=args.conv_order)
    stage_of = STAGE_OF
    if args.op == "vp":
        entries = n1 * O                    # outputs of one NTK-vector product
        fl = vp_flops(spec, n1, n2, symmetric=sym)
        stage_of = VP_STAGE_OF
    value = entries / (ms * 1e-3)
    tflops = fl["total"] / (ms * 1e-3) / 1e12

    kernels = {}
    for k, (tot, cnt) in prof.items():
        per_step = cnt / args.steps
        kernels[k] = {"ms_per_step": tot / args.steps, "launches_per_step": per_step}
        st = stage_of.get(k)
        if st and st in fl and cnt:
            kernels[k]["tflops"] = fl[st] / (tot / args.steps * 1e-3) / 1e12
    # the dominant matrix-core kernel class (the memory-bound struct_* classes are not priced
    # against the MFMA peak)
    dom = max((k for k in prof if stage_of.get(k) in fl and not stage_of[k].startswith("struct")),
              key=lambda k: prof[k][0])
    tot, cnt = prof[dom]
    avg_ms = tot / cnt
    flop_per_launch = fl[stage_of[dom]] / (cnt / args.steps)
    achieved = flop_per_launch / (avg_ms * 1e-3) / 1e12
    # every priced class runs on the matrix cores: the forward in fp64, the rest in fp32
    peak = FP64_MFMA_PEAK_TFLOPS if stage_of[dom] == "forward" else FP32_MFMA_PEAK_TFLOPS
    roofline = {"kernel": dom, "bound": "mfma", "achieved": achieved,
                "peak": peak, "unit": "TFLOP/s",
                "frac": achieved / peak, "traffic": measured_traffic(name, dom),
                "mfma_busy": measured_mfma_busy(name, dom),
                "flop_per_launch": flop_per_launch, "avg_launch_ms": avg_ms}

    h.close()
    num_cu, clock_khz = _lib.device_info()
    ceiling = {"fp32_tflops": _lib.mfma_peak("fp32"), "fp64_tflops": _lib.mfma_peak("fp64"),
               "kernel": "independent MFMA chains, 4 waves per SIMD"}
    roofline["measured_ceiling"] = ceiling["fp32_tflops"]
    roofline["frac_of_measured_ceiling"] = achieved / ceiling["fp32_tflops"]

    res = {
        "metric": METRIC if args.op == "ntk" else "NTK-vector product outputs/sec (N1 O)",
        "value": value, "unit": "NTK entries/s" if args.op == "ntk" else "(Theta v) entries/s",
        "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "ms_per_step_median": ms_median, "ms_per_step_min": step_ms[0], "ms_per_step_profiled": ms_profiled,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded N(0,1) inputs, He-init weights)",
        "config": {"workload": name, "n1": n1, "n2": n2, "O": O,
                   "layers": [[L.get("in"), L.get("out"), L.get("act")] for L in spec["layers"]],
                   "symmetric_schedule": sym, "parallelism": "single GPU",
                   "method": args.method, "op": args.op, "hip_graph": use_graph,
                   "conv_order": args.conv_order,
                   "variant": {"output": args.output, "batch": args.batch,
                               **({"logit": args.logit} if args.output == "logit" else {})}},
        "tflops": tflops, "frac_of_fp32_mfma_peak": tflops / FP32_MFMA_PEAK_TFLOPS,
        "algorithmic_flops": fl, "kernels": kernels, "roofline": roofline,
        "mfma_ceiling_measured": ceiling,
        "device": {"name": torch.cuda.get_device_name(0), "compute_units": num_cu,
                   "peak_clock_mhz": clock_khz / 1000.0},
        "wall_s_timed_region": wall,
    }
    if not args.no_cpu_baseline and args.output == "full" and args.batch == "full" \
            and not args.samples and args.op == "ntk":
        res["cpu_baseline"] = cpu_baseline(name, min(args.cpu_samples, n1, n2), n1, n2)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
