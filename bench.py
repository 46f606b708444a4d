"""Benchmark of the libmalt MALT / MALTER step on one MI355X.

Default workload: the GPT-2 Large matrix set (36 blocks, width 1280: 144
matrices, 707,788,800 fp32 parameters), MALT, 10 consecutive steps timed end
to end with persistent state, fresh seeded gradients per step.  Inputs are
drawn on the GPU before the timed region (synthetic: no dataset).

Prints one JSON line:  step latency (value, ms per step), the Newton-Schulz
GEMM kernel against the bf16 matrix-core peak (roofline), per-kernel achieved
HBM bandwidth / throughput, and the fp64 CPU oracle timed on a bounded sample
of the same workload (cpu_baseline).

  python bench.py [--steps K] [--warmup W] [--workload gpt2_large|gpt2_small|gpt2_medium|single_256x512|stress_4096]
                  [--no-cpu-baseline] [--no-vendor-ref] [--no-ceiling] [--small-case] [--gpus 1]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0    # MI355X dense bf16 matrix-core peak
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ns_update_gpt2_large_traffic.md")
# Sources of the update kernel (its shared pipeline header, then the kernel).
NS_SOURCES = [os.path.join(ROOT, "paper_2608_05088_amd", "csrc", f) for f in ("ns_common.h", "ns_update.hip")]
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E
METRIC = "MALT step latency (ms) per GPT-2 param set; NS MFMA % bf16 peak; HBM GB/s"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="gpt2_large")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--small-case", action="store_true",
                    help="also report the step latency of the single 256 x 512 matrix workload "
                         "(off by default so kernel traces of the default run cover one workload)")
    ap.add_argument("--no-vendor-ref", action="store_true",
                    help="skip timing torch.bmm (hipBLASLt) on the update products")
    ap.add_argument("--cpu-sample-layers", type=int, default=12)
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the matrix-core ceiling calibration (MFMA-only kernel with random operands)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after timing, run one plain 1 GiB device-to-device copy (HBM counter calibration)")
    return ap.parse_args()


def recorded_traffic(workload: str):
    """HBM bytes per ns_update_kernel launch from the committed PMC summary, or
    None when the summary is for another workload or an older kernel source."""
    import hashlib
    if workload != "gpt2_large" or not os.path.exists(TRAFFIC_FILE):
        return None
    fields = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            fields[k.strip().lstrip("- ").strip("`")] = v.strip().strip("`")
    sha = hashlib.sha256(b"".join(open(f, "rb").read() for f in NS_SOURCES)).hexdigest()
    if fields.get("source_sha256") != sha or "traffic_bytes_per_launch" not in fields:
        return None
    return float(fields["traffic_bytes_per_launch"])


def small_case_latency(lm, wl, dev, reps: int = 50):
    """Latency of one step on the single 256 x 512 matrix workload (MALT),
    which is bound by kernel latency (one or two workgroups per launch), not by
    bandwidth or matrix-core rate:
    median over `reps` individually timed steps."""
    import statistics

    import torch
    w = wl.WORKLOADS[1]
    shapes = list(w.shapes)
    Wd = [wl.weight_device(w.cid, i, s, dev) for i, s in enumerate(shapes)]
    Gd = [wl.grad_device(w.cid, 1, i, s, w.dist, dev) for i, s in enumerate(shapes)]
    plan = lm.Plan(shapes, w.variant, device=dev)
    hp = lm.make_hparams(lr=w.lr, mu1=w.mu1, mu2=w.mu2, eps=w.eps)
    stream = torch.cuda.current_stream()
    for _ in range(5):
        plan.step(Wd, Gd, hp, stream=stream)
    times = []
    for _ in range(reps):
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record(stream)
        plan.step(Wd, Gd, hp, stream=stream)
        e.record(stream)
        e.synchronize()
        times.append(s.elapsed_time(e))
    plan.close()
    return {"workload": w.name, "median_ms": round(statistics.median(times), 4), "reps": reps,
            "launches_per_step": 4 + 3 * 5 + 2}


def vendor_gemm_reference(w, dev):
    """Time the vendor bf16 GEMM (hipBLASLt through torch.bmm) on the update
    product of the workload, B'X for every matrix, one batched call per
    distinct canonical shape: context for the update kernel's rate."""
    import torch
    groups = {}
    for (r, c) in w.shapes:
        mp, np_ = min(r, c), max(r, c)
        groups[(mp, np_)] = groups.get((mp, np_), 0) + 1
    total_ms, total_flops, per = 0.0, 0.0, {}
    for (mp, np_), cnt in sorted(groups.items()):
        B = torch.randn(cnt, mp, mp, device=dev, dtype=torch.bfloat16)
        X = torch.randn(cnt, mp, np_, device=dev, dtype=torch.bfloat16)
        for _ in range(3):
            torch.bmm(B, X)
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        s.record()
        for _ in range(10):
            torch.bmm(B, X)
        e.record()
        torch.cuda.synchronize()
        ms = s.elapsed_time(e) / 10
        flops = 2.0 * cnt * mp * mp * np_
        per[f"{cnt}x({mp}x{mp} @ {mp}x{np_})"] = round(flops / (ms * 1e-3) / 1e12, 1)
        total_ms += ms
        total_flops += flops
        del B, X
    return {"what": "torch.bmm bf16 (hipBLASLt) on the same B'X products, one batched call per shape",
            "TFLOP_per_s": round(total_flops / (total_ms * 1e-3) / 1e12, 1), "per_shape_TFLOP_per_s": per}


def cpu_baseline(w, layers: int):
    """Time the fp64 oracle (as it stands) on `layers` transformer blocks' worth
    of matrices (one matrix of every shape per block) and scale per shape to
    one full step of the workload."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import OracleHparams, oracle_init, oracle_step
    from paper_2608_05088_amd import workloads as wl

    shapes = list(w.shapes)
    uniq = []
    for s in shapes:
        if s not in uniq:
            uniq.append(s)
    per_shape = {}
    sample_desc = []
    for s in uniq:
        idx = shapes.index(s)
        times = []
        for rep in range(layers):
            i = idx + rep * len(uniq) if idx + rep * len(uniq) < len(shapes) else idx
            G = wl.grad(w.cid, 1, i, s, w.dist)
            W0 = wl.weight(w.cid, i, s).astype(np.float64)
            st = oracle_init([s], w.variant)
            hp = OracleHparams(variant=w.variant, lr=w.lr, mu1=w.mu1, mu2=w.mu2, eps=w.eps)
            t0 = time.perf_counter()
            oracle_step([W0], [G], st, hp)
            times.append(time.perf_counter() - t0)
        per_shape[s] = sum(times) / len(times)
        sample_desc.append(f"{s[0]}x{s[1]}")
    total_s = sum(per_shape[s] for s in shapes)
    sampled_s = sum(per_shape[s] * layers for s in uniq)
    blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
    threads = max([p.get("num_threads", 1) for p in blas] or [1])
    cpu_model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    # The single 256 x 512 matrix workload on one BLAS thread (its three steps).
    from threadpoolctl import threadpool_limits
    w1 = wl.WORKLOADS[1]
    with threadpool_limits(limits=1, user_api="blas"):
        st1 = oracle_init(list(w1.shapes), w1.variant)
        hp1 = OracleHparams(variant=w1.variant, lr=w1.lr, mu1=w1.mu1, mu2=w1.mu2, eps=w1.eps)
        W1 = [wl.weight(w1.cid, 0, w1.shapes[0]).astype(np.float64)]
        t0 = time.perf_counter()
        for step in range(1, w1.steps + 1):
            W1, _ = oracle_step(W1, [wl.grad(w1.cid, step, 0, w1.shapes[0], w1.dist)], st1, hp1)
        c1_ms = (time.perf_counter() - t0) * 1e3 / w1.steps
    return {"value": total_s * 1e3, "unit": "ms per step (extrapolated per shape)", "cores": int(threads),
            "kind": "oracle",
            "sample": f"one oracle step on {layers} matrices of each shape ({', '.join(sample_desc)}), "
                      f"{sampled_s:.1f} s of CPU time, scaled by shape counts to all {len(shapes)} matrices",
            "host_cpus": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0)), "cpu_model": cpu_model,
            "blas": ", ".join(f"{p.get('internal_api')} {p.get('version')}" for p in blas),
            "single_256x512_one_thread_ms_per_step": round(c1_ms, 3)}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: across GPUs the step would shard by whole matrices, which "
              f"libmalt does not implement; --gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2608_05088_amd import libmalt as lm
    from paper_2608_05088_amd import workloads as wl

    byname = {w.name: w for w in wl.WORKLOADS.values()}
    w = byname[args.workload]
    K = args.steps if args.steps is not None else max(w.steps, 10 if w.cid == 4 else 5)
    Wu = args.warmup
    dev = torch.device("cuda:0")
    lm.lib()
    shapes = list(w.shapes)
    print(f"[bench] workload {w.name}: {len(shapes)} matrices, {w.numel} params, {w.variant}, "
          f"steps {K} warmup {Wu}", file=sys.stderr, flush=True)

    # Inputs resident in HBM before timing: weights + one fresh gradient set per step.
    Wd = [wl.weight_device(w.cid, i, s, dev) for i, s in enumerate(shapes)]
    grad_sets = []
    for t in range(1, Wu + K + 1):
        grad_sets.append([wl.grad_device(w.cid, t, i, s, w.dist, dev) for i, s in enumerate(shapes)])
    torch.cuda.synchronize()
    print(f"[bench] inputs ready ({torch.cuda.memory_allocated() / 2**30:.1f} GiB)", file=sys.stderr, flush=True)

    plan = lm.Plan(shapes, w.variant, device=dev)
    hp = lm.make_hparams(lr=w.lr, mu1=w.mu1, mu2=w.mu2, eps=w.eps)
    stream = torch.cuda.current_stream()
    for t in range(Wu):
        plan.step(Wd, grad_sets[t], hp, stream=stream)
    torch.cuda.synchronize()
    print("[bench] warmup done", file=sys.stderr, flush=True)

    # Headline: K consecutive steps with the library's per-phase events off.
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start.record(stream)
    for t in range(K):
        plan.step(Wd, grad_sets[Wu + t], hp, stream=stream)
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / K
    print(f"[bench] {ms_per_step:.3f} ms/step (wall {wall * 1e3 / K:.3f})", file=sys.stderr, flush=True)

    # Per-kernel figures: a second pass of K steps (the same gradient sets,
    # persistent state continuing) with HIP events recorded by the library
    # around every phase, on the step's stream.
    plan.profile_read(reset=True)
    plan.profile_enable(True)
    start.record(stream)
    for t in range(K):
        plan.step(Wd, grad_sets[Wu + t], hp, stream=stream)
    end.record(stream)
    torch.cuda.synchronize()
    prof_ms_per_step = start.elapsed_time(end) / K
    prof = plan.profile_read(reset=True)
    plan.profile_enable(False)
    print(f"[bench] profiled pass {prof_ms_per_step:.3f} ms/step", file=sys.stderr, flush=True)

    # Per-kernel figures (ms per step, achieved rate, fraction of the bound).
    kernels = {}
    for name, v in prof.items():
        if v["launches"] == 0:
            continue
        ms = v["ms"] / K
        ent = {"ms_per_step": round(ms, 4), "launches_per_step": v["launches"] // K,
               "avg_launch_ms": round(v["ms"] / v["launches"], 5)}
        if v["bytes"] > 0 and ms > 0:
            gbs = v["bytes"] / (ms * 1e-3) / 1e9
            ent.update({"bound": "hbm", "GB_per_s": round(gbs, 1), "frac": round(gbs / PEAK_HBM_GBS, 4),
                        "bytes_per_step": v["bytes"]})
        if v["flops"] > 0 and ms > 0:
            tf = v["flops"] / (ms * 1e-3) / 1e12
            ent.update({"bound": "mfma", "TFLOP_per_s": round(tf, 1), "frac": round(tf / PEAK_BF16_TFLOPS, 4),
                        "flops_per_step": v["flops"]})
        kernels[name] = ent
    ns = [prof[k] for k in ("ns_gram", "ns_poly", "ns_update")]
    ns_ms = sum(v["ms"] for v in ns)
    ns_flops_step = sum(v["flops"] for v in ns)
    # Dominant kernel: the Newton-Schulz update product B'X (ns_update_kernel).
    upd = prof["ns_update"]
    flops_per_launch = upd["flops"] * K / upd["launches"]
    avg_launch_s = upd["ms"] * 1e-3 / upd["launches"]
    achieved = flops_per_launch / avg_launch_s / 1e12
    roofline = {"bound": "mfma", "kernel": "ns_update_kernel (Newton-Schulz X' = B'X, all matrices)",
                "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": recorded_traffic(w.name),
                "flops_per_launch": flops_per_launch, "avg_launch_ms": round(avg_launch_s * 1e3, 4),
                "flops_basis": "2 m'^2 n' per matrix per launch (B'X)"}
    # Dense-equivalent count (4 m'^2 n' + 2 m'^3 per iteration): the Gram and
    # polynomial products counted without their symmetry.
    dense_step = 2 * prof["ns_gram"]["flops"] + 2 * prof["ns_poly"]["flops"] + prof["ns_update"]["flops"]
    ns_all = {"kernels": "ns_gemm_sym_kernel + ns_update_kernel", "ms_per_step": round(ns_ms / K, 4),
              "TFLOP_per_s": round(ns_flops_step * K / (ns_ms * 1e-3) / 1e12, 1),
              "frac": round(ns_flops_step * K / (ns_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
              "flops_per_step": ns_flops_step,
              "flops_basis": "symmetric minimum 3 m'^2 n' + m'^3 per matrix per NS iteration",
              "dense_equiv_TFLOP_per_s": round(dense_step * K / (ns_ms * 1e-3) / 1e12, 1),
              "dense_equiv_basis": "4 m'^2 n' + 2 m'^3 per matrix per NS iteration"}
    ew_bytes = sum(prof[k]["bytes"] for k in ("momentum_rowcol", "scale_convert", "backmap_write"))
    ew_ms = sum(prof[k]["ms"] for k in ("momentum_rowcol", "scale_convert", "backmap_write")) / K
    hbm = {"elementwise_GB_per_s": round(ew_bytes / (ew_ms * 1e-3) / 1e9, 1),
           "elementwise_frac": round(ew_bytes / (ew_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}

    plan.close()
    del grad_sets, Wd
    torch.cuda.empty_cache()
    small = small_case_latency(lm, wl, dev) if args.small_case else None
    vendor = None if args.no_vendor_ref else vendor_gemm_reference(w, dev)
    if vendor is not None:
        roofline["vendor_gemm_reference"] = vendor
    if not args.no_ceiling:
        # The matrix cores' sustained rate under the power budget with random
        # bf16 operands and no memory traffic, for the instruction the
        # Newton-Schulz kernels issue: context for the datasheet peak.
        from paper_2608_05088_amd.calib import mfma_ceiling
        ceil = mfma_ceiling("random", "16x16x32")
        roofline["power_limited_ceiling"] = {
            "what": "MFMA-only kernel (v_mfma_f32_16x16x32_bf16), random N(0,1) bf16 operands in registers, "
                    "every CU, no memory traffic, fastest of three launches",
            "TFLOP_per_s": ceil["TFLOP_per_s"], "clock_MHz": ceil["clock_MHz"],
            "frac_of_peak": round(ceil["TFLOP_per_s"] / PEAK_BF16_TFLOPS, 4),
            "update_frac_of_ceiling": round(achieved / ceil["TFLOP_per_s"], 4),
            "newton_schulz_frac_of_ceiling": round(ns_all["TFLOP_per_s"] / ceil["TFLOP_per_s"], 4)}
    if args.copy_calibration:
        # A plain copy kernel of known size (an elementwise x*1 kernel, not the
        # SDMA engine): 2^30 bytes read, 2^30 bytes written.
        src = torch.ones(2 ** 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, args.cpu_sample_layers)

    line = {"metric": METRIC, "value": round(ms_per_step, 4), "unit": "ms", "n_gpus": 1, "steps": K,
            "warmup": Wu, "ms_per_step": round(ms_per_step, 4), "higher_is_better": False,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16+fp32", "data": "synthetic",
            "config": {"workload": w.name, "variant": w.variant, "matrices": len(shapes), "params": w.numel,
                       "lr": w.lr, "grad_dist": w.dist, "timed": f"{K} consecutive steps, persistent state"},
            "roofline": roofline, "newton_schulz": ns_all, "hbm": hbm, "kernels": kernels,
            "profiled_pass": {"ms_per_step": round(prof_ms_per_step, 4),
                              "what": "per-kernel figures come from a second pass of the same K steps "
                                      "with per-phase HIP events on; the headline pass records none"},
            "small_case_latency": small,
            "cpu_baseline": cpu}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
