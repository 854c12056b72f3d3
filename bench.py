#!/usr/bin/env python3
"""Throughput of MiCRO's per-worker sparsify step on one MI355X.

A step is one pass of the whole hot path over one synthetic gradient: for each
rank the workload sweeps, the error-feedback add, the threshold test, the
residual update, the order-preserving compaction of the selected (index,
value) pairs, the selected-count readback and the threshold update -- one
micro_sparsify_step call per rank.  Gradients are generated before the timed
region and stay resident in HBM (a pool of distinct seeded gradients, one per
step while the pool lasts).

Default workload: the 1,315,723,264-value GPT-1.3B-shaped gradient as one
partition (world 1) at density 0.01; density 0.001 is measured in the same run
and reported under "extra".

Prints one JSON line.  --gpus above 1 is refused: the step involves no
collective and this benchmark runs on one GPU.
"""
import argparse
import hashlib
import json
import math
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("sparsify-step throughput (G elem/s, HBM GB/s % of peak); "
          "density error |d_act−d|/d")
HBM_PEAK_GBS = 8000.0
KERNEL_SRC = os.path.join(ROOT, "paper_2310_00967_amd", "csrc", "sparsify_kernel.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "sparsify_kernel_gpt_1p3b_traffic.txt")


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="gpt_1p3b",
                    choices=["toy", "resnet18", "resnet50", "bert_large", "gpt_1p3b"])
    ap.add_argument("--density", type=float, default=None,
                    help="headline density (default: the workload's last listed density)")
    ap.add_argument("--no-extra", action="store_true", help="skip the workload's other densities")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="target CPU time of the oracle baseline sample (0 disables)")
    ap.add_argument("--pool-gb", type=float, default=100.0,
                    help="HBM budget for the pre-generated gradient pool")
    ap.add_argument("--variant", default="staged", choices=["staged", "ticket"],
                    help="kernel schedule (staged is the library default)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of known size (HBM counter scaling)")
    return ap.parse_args()


def kernel_sha256():
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def read_traffic():
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when absent or taken on a different kernel source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    fields = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line:
            key, val = line.split(":", 1)
            fields[key.strip()] = val.strip()
    if fields.get("kernel_source_sha256") != kernel_sha256():
        return None
    try:
        return float(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def copy_calibration():
    """A plain device-to-device copy of exactly 4 GiB, ten times, for scaling
    the FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    n = 1 << 30
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(10):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": 4 * n, "copy_calibration_bytes_written": 4 * n,
                      "launches": 10}), flush=True)


class Run:
    """One workload at one density: gradient pool, residual, thresholds."""

    def __init__(self, w, density, pool, sp, micro):
        import torch
        self.w, self.d, self.pool, self.sp = w, density, pool, sp
        self.N = w.n_total
        self.res = torch.zeros(self.N, dtype=torch.float32, device="cuda")
        self.bounds = {r: micro.micro_partition(self.N, r, w.world) for r in w.ranks}
        from paper_2310_00967_amd import synth
        self.theta = {r: synth.initial_theta(w, pool[0], s, s + ln, density)
                      for r, (s, ln) in self.bounds.items()}
        self.theta0 = dict(self.theta)
        cap = max(ln for _, ln in self.bounds.values())
        self.out_idx, self.out_val = sp.outputs(cap)
        self.t = 0
        self.log = []   # (rank, P, k, kernel_ms, tiles redone by the gather pass)

    def step(self, timed):
        g = self.pool[self.t % len(self.pool)]
        for r in self.w.ranks:
            _, ln = self.bounds[r]
            k, th, _, _ = self.sp.step(g, self.res, r, self.w.world, self.d, self.theta[r],
                                       self.out_idx, self.out_val)
            self.theta[r] = th
            kernel_ms, redone, _ = self.sp.last_stats()
            self.log.append((r, ln, k, kernel_ms if timed else None, redone))
        self.t += 1


def measure(w, density, pool, sp, micro, warmup, steps):
    import torch
    run = Run(w, density, pool, sp, micro)
    for _ in range(warmup):
        run.step(timed=False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        run.step(timed=True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    timed = [x for x in run.log if x[3] is not None]
    elems = sum(x[1] for x in timed)
    alg_bytes = sum(12 * x[1] + 8 * x[2] for x in timed)
    kernel_s = sum(x[3] for x in timed) / 1e3
    per_step = [x for x in run.log]
    errs = [abs(x[2] / x[1] - density) / density for x in per_step if x[1] > 0]
    half = errs[len(errs) // 2:]
    return {
        "elapsed_s": elapsed,
        "elems": elems,
        "g_elem_s": elems / elapsed / 1e9,
        "wall_gbs": alg_bytes / elapsed / 1e9,
        "kernel_gbs": alg_bytes / kernel_s / 1e9,
        "kernel_ms_avg": kernel_s * 1e3 / len(timed),
        "launches": len(timed),
        "alg_bytes_per_launch": alg_bytes / len(timed),
        "k_avg": sum(x[2] for x in timed) / len(timed),
        "redone_tiles": sum(x[4] for x in timed),
        "density_error_last_half": sum(half) / len(half),
        "theta0": run.theta0,
        "theta_final": run.theta,
        "ms_per_step": elapsed * 1e3 / steps,
    }


def cpu_baseline(w, density, pool, target_s):
    """The C oracle, as it stands, on the host: same workload and density,
    its own error-feedback trajectory from a zero residual, gradients copied
    from the pool (copies not timed).  Runs steps until target_s of oracle
    time has accumulated."""
    import numpy as np
    import torch

    import oracle
    from paper_2310_00967_amd import synth
    N = w.n_total
    res = np.zeros(N, np.float32)
    g_host = torch.empty(N, dtype=torch.float32, pin_memory=True)
    bounds = {r: oracle.partition(N, r, w.world) for r in w.ranks}
    theta = {r: synth.initial_theta(w, pool[0], s, s + ln, density) for r, (s, ln) in bounds.items()}
    cap = max(ln for _, ln in bounds.values())
    out = (np.empty(max(1, cap), np.int32), np.empty(max(1, cap), np.float32))
    # fault every host page in before timing, as the device buffers are
    # resident before the GPU's timed region
    res[:] = 0.0
    out[0][:] = 0
    out[1][:] = 0.0
    spent, elems, steps = 0.0, 0, 0
    while spent < target_s and steps < 10000:
        g = pool[steps % len(pool)]
        for r, (s, ln) in bounds.items():
            g_host[s:s + ln].copy_(g[s:s + ln])
        gn = g_host.numpy()
        for r, (s, ln) in bounds.items():
            t0 = time.perf_counter()
            _, _, _, theta[r] = oracle.step(gn, res, r, w.world, density, theta[r], out=out)
            spent += time.perf_counter() - t0
            elems += ln
        steps += 1
    return {
        "value": elems / spent / 1e9,
        "unit": "G elem/s",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"{steps} step(s) of {w.name} at d={density} ({elems} values, "
                   f"{spent:.1f} s of single-threaded oracle time); host {cpu_model()}, "
                   f"nproc {os.cpu_count()}"),
    }


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py: --gpus {args.gpus} is not supported: the sparsify step has no collective "
              "and this build measures one GPU (one worker's partition at its real size).",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return

    import torch
    import paper_2310_00967_amd as micro
    from paper_2310_00967_amd import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    w = synth.get(args.workload)
    densities = list(w.densities)
    head = args.density if args.density is not None else densities[-1]
    others = [] if args.no_extra else [d for d in densities if d != head]

    n_pool = max(1, min(args.warmup + args.steps, int(args.pool_gb * 1e9 // (4 * w.n_total))))
    pool = [synth.gradient(w, t, "cuda") for t in range(n_pool)]
    torch.cuda.synchronize()
    variant = micro.MICRO_VARIANT_STAGED if args.variant == "staged" else micro.MICRO_VARIANT_TICKET
    sp = micro.Sparsifier(w.n_total, device="cuda", time_kernel=True, variant=variant)

    main_res = measure(w, head, pool, sp, micro, args.warmup, args.steps)
    extra = {}
    for d in others:
        r = measure(w, d, pool, sp, micro, args.warmup, args.steps)
        extra[f"d={d}"] = {k: r[k] for k in ("g_elem_s", "wall_gbs", "kernel_gbs", "kernel_ms_avg",
                                             "density_error_last_half", "ms_per_step")}
        extra[f"d={d}"]["kernel_hbm_frac"] = r["kernel_gbs"] / HBM_PEAK_GBS

    cpu = cpu_baseline(w, head, pool, args.cpu_seconds) if args.cpu_seconds > 0 else None
    sp.close()

    traffic = read_traffic() if args.workload == "gpt_1p3b" and head == 0.01 else None
    parts = sorted({ln for (_, ln) in (micro.micro_partition(w.n_total, r, w.world) for r in w.ranks)})
    line = {
        "metric": METRIC,
        "value": main_res["g_elem_s"],
        "unit": "G elem/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "n_total": w.n_total,
            "world": w.world,
            "ranks": list(w.ranks),
            "partition_len": parts,
            "density": head,
            "distribution": w.dist,
            "gradient_pool": n_pool,
            "parallelism": "one worker's partition on one GPU",
            "variant": args.variant,
        },
        "hbm_gbs_wall": main_res["wall_gbs"],
        "hbm_frac_wall": main_res["wall_gbs"] / HBM_PEAK_GBS,
        "density_error": main_res["density_error_last_half"],
        "roofline": {
            "bound": "hbm",
            "achieved": main_res["kernel_gbs"],
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": main_res["kernel_gbs"] / HBM_PEAK_GBS,
            "traffic": traffic,
            "kernel": ("stream_kernel + scan_kernel + move_kernel (one step, event-timed together)"
                       if args.variant == "staged" else "ticket_kernel"),
            "kernel_ms_avg": main_res["kernel_ms_avg"],
            "alg_bytes_per_launch": main_res["alg_bytes_per_launch"],
            "redone_tiles_timed": main_res["redone_tiles"],
        },
        "cpu_baseline": cpu,
        "extra": extra,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
