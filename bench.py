#!/usr/bin/env python3
"""Throughput of MiCRO's per-worker sparsify step on one MI355X.

A step is one pass of the whole hot path over one synthetic gradient: for each
worker the workload sweeps, the error-feedback add, the threshold test, the
residual update, the order-preserving compaction of the selected (index,
value) pairs, the selected-count readback and the threshold update -- one
micro_sparsify_step call per listed rank, each rank with its own threshold.
With --cycle, worker i searches partition ((t mod world) + i) mod world at
step t instead, as in Algorithm 1, so its partition (and the residual it
touches) changes from one step to the next; each partition then keeps its
own threshold.  Gradients are generated before the timed
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
KERNEL_HDR = os.path.join(ROOT, "paper_2310_00967_amd", "csrc", "sparsify_kernel.h")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "sparsify_kernel_gpt_1p3b_traffic.txt")
TRAFFIC_FILE_BERT = os.path.join(ROOT, "profiles", "sparsify_kernel_bert_large_rank3_traffic.txt")
TRAFFIC_FILE_EF = os.path.join(ROOT, "profiles", "ef_pass_bert_large_worker3_traffic.txt")
TRAFFIC_FILE_SWEEP = os.path.join(ROOT, "profiles", "sweep_resnet18_16_partitions_traffic.txt")
TRAFFIC_FILE_UNION = os.path.join(ROOT, "profiles", "union_gather_update_bert_large_traffic.txt")
UNION_SRC = os.path.join(ROOT, "paper_2310_00967_amd", "csrc", "union_kernel.hip")
TRAFFIC_FILE_TOPK = os.path.join(ROOT, "profiles", "topk_comparator_bert_large_rank3_traffic.txt")
TOPK_SOURCES = (os.path.join(ROOT, "paper_2310_00967_amd", "csrc", "topk_kernel.hip"),
                os.path.join(ROOT, "paper_2310_00967_amd", "csrc", "topk_kernel.h"), KERNEL_SRC, KERNEL_HDR)


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10,
                    help="untimed steps first: the threshold settles from its calibrated start (default 10)")
    ap.add_argument("--workload", default="gpt_1p3b",
                    choices=["toy", "resnet18", "resnet50", "bert_large", "gpt_1p3b"])
    ap.add_argument("--density", type=float, default=None,
                    help="headline density (default: the workload's last listed density)")
    ap.add_argument("--no-extra", action="store_true", help="skip the workload's other densities")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="target CPU time of the oracle baseline sample (0 disables)")
    ap.add_argument("--pool-gb", type=float, default=100.0,
                    help="HBM budget for the pre-generated gradient pool")
    ap.add_argument("--steps-jsonl", default=None, metavar="PATH",
                    help="also write one JSON record per step call (warm-up and timed) to PATH")
    ap.add_argument("--cycle", action="store_true",
                    help="rotate each worker's partition every step (Algorithm 1) instead of fixed ranks")
    ap.add_argument("--variant", default="auto", choices=["auto", "staged", "ticket"],
                    help="kernel schedule (auto, the library default, runs the ticket schedule up to "
                         "2^20 values per partition and the staged one above)")
    ap.add_argument("--separate-scan", action="store_true",
                    help="staged schedule: launch the scan pass on its own instead of inside the "
                         "streaming launch (the library default for partitions of up to a few hundred "
                         "million values)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of known size (HBM counter scaling)")
    ap.add_argument("--path", default="step", choices=["step", "ef", "union", "sweep", "ceiling", "topk"],
                    help="step: the partition-only sparsify step (default); ef: the full error-feedback "
                         "pass with cyclic partitions; union: the gather/reset and model update around "
                         "the exchange; sweep: every partition in one set of launches, with the "
                         "local-error norms; ceiling: vendor streams (torch's in-place add, a device "
                         "copy) beside the step on the same vector; topk: the exact top-k comparator "
                         "beside the threshold step and the hard-threshold rule on the same gradients")
    ap.add_argument("--topk-hint", choices=["last", "none", "high"], default="last",
                    help="with --path topk: the theta each top-k call gets: the k-th magnitude the last call "
                         "returned (default), NaN (no hint: the passes over the partition first), or 8 times the "
                         "last one (too high: the step lists fewer than k and the pick runs over the residual)")
    ap.add_argument("--topk-only", action="store_true",
                    help="with --path topk: the top-k rule alone (its HBM counters then cover only its kernels)")
    ap.add_argument("--local-error", action="store_true",
                    help="with --path ef: also return the squared norm of the whole residual (Eq. 1)")
    args = ap.parse_args()
    if args.path not in ("step", "ceiling") and args.workload == "gpt_1p3b" and "--workload" not in sys.argv:
        # world 1 makes these paths degenerate
        args.workload = "resnet18" if args.path == "sweep" else "bert_large"
    return args


def kernel_sha256(text=None, sources=None):
    """sha256 of the kernels' code (by default the sparsify kernel source
    followed by its header, whose constants shape the launches; the union
    kernels' counters use their own source and that header): // comments,
    trailing blanks and blank lines removed, so the stored counters stay
    valid across comment edits and go stale with any change to the code."""
    if text is None:
        parts = []
        for path in sources or (KERNEL_SRC, KERNEL_HDR):
            with open(path, encoding="utf-8") as f:
                parts.append(f.read())
        text = "\n".join(parts)
    code = []
    for line in text.splitlines():
        line = line.split("//", 1)[0].rstrip()
        if line:
            code.append(line)
    return hashlib.sha256("\n".join(code).encode()).hexdigest()


def read_traffic(path=None, workload=None, sources=None):
    """HBM bytes per launch from a committed rocprofv3 counter summary (the
    GPT-1.3B one by default), or None when absent, taken on a different
    kernel source, or (with `workload`) on a different workload line."""
    path = path or TRAFFIC_FILE
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            key, val = line.split(":", 1)
            fields[key.strip()] = val.strip()
    if fields.get("kernel_source_sha256") != kernel_sha256(sources=sources):
        return None
    if workload is not None and fields.get("workload") != workload:
        return None
    try:
        return float(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model():
    """The host CPU as /proc/cpuinfo names it: the model name string with the
    vendor, family, model and stepping numbers."""
    fields = {}
    try:
        for line in open("/proc/cpuinfo"):
            if ":" in line:
                key, val = (x.strip() for x in line.split(":", 1))
                fields.setdefault(key, val)
            if not line.strip() and fields:
                break  # the first processor's block
    except OSError:
        pass
    name = fields.get("model name") or platform.processor() or "unknown"
    ids = ", ".join(f"{k} {fields[k]}" for k in ("vendor_id", "cpu family", "model", "stepping") if k in fields)
    return f"{name} ({ids})" if ids else name


class OneCore:
    """Pins the calling thread to one core (the highest it may run on) for the
    oracle's timing and restores its previous affinity on exit, in-process."""

    def __enter__(self):
        self.previous = os.sched_getaffinity(0)
        self.core = max(self.previous)
        os.sched_setaffinity(0, {self.core})
        return self

    def __exit__(self, *exc):
        os.sched_setaffinity(0, self.previous)
        return False

    def describe(self):
        return (f"pinned to core {self.core} of {len(self.previous)} allowed "
                f"(nproc {os.cpu_count()}); host {cpu_model()}")


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

    def __init__(self, w, density, pool, sp, micro, cycle=False, keep_records=False):
        import torch
        self.w, self.d, self.pool, self.sp, self.micro, self.cycle = w, density, pool, sp, micro, cycle
        self.N = w.n_total
        self.res = torch.zeros(self.N, dtype=torch.float32, device="cuda")
        # every partition the workers visit, each with its own threshold
        parts = range(w.world) if cycle else w.ranks
        self.bounds = {p: micro.micro_partition(self.N, p, w.world) for p in parts}
        from paper_2310_00967_amd import synth
        self.theta = {r: synth.initial_theta(w, pool[0], s, s + ln, density)
                      for r, (s, ln) in self.bounds.items()}
        self.theta0 = dict(self.theta)
        cap = max(ln for _, ln in self.bounds.values())
        self.out_idx, self.out_val = sp.outputs(cap)
        self.t = 0
        self.log = []   # (rank, P, k, kernel_ms, tiles redone by the move kernel)
        self.records = [] if keep_records else None  # one dict per call for --steps-jsonl
        self.variant = None  # schedule of the last step
        self.fused = 0       # whether its stream and scan passes ran as one launch

    def step(self, timed):
        g = self.pool[self.t % len(self.pool)]
        for worker in self.w.ranks:
            p = self.micro.micro_cycle(self.t, worker, self.w.world) if self.cycle else worker
            _, ln = self.bounds[p]
            theta_in = self.theta[p]
            t0 = time.perf_counter() if self.records is not None else 0.0
            k, th, _, _ = self.sp.step(g, self.res, p, self.w.world, self.d, theta_in,
                                       self.out_idx, self.out_val)
            self.theta[p] = th
            kernel_ms, redone, variant, fused = self.sp.last_stats()
            self.log.append((p, ln, k, kernel_ms if timed else None, redone))
            self.variant = variant
            self.fused = fused
            if self.records is None:
                continue
            wall_s = time.perf_counter() - t0
            alg = 12 * ln + 8 * k
            self.records.append({
                "workload": self.w.name, "t": self.t, "timed": timed, "rank": p, "P": ln, "k": k,
                "density": self.d, "d_act": k / ln if ln else 0.0,
                "density_error": abs(k / ln - self.d) / self.d if ln else 0.0,
                "theta": theta_in, "theta_next": th, "device_us": kernel_ms * 1e3 if kernel_ms >= 0 else None,
                "wall_us": wall_s * 1e6, "alg_bytes": alg,
                "kernel_gbs": alg / (kernel_ms * 1e-3) / 1e9 if kernel_ms > 0 else None,
                "hbm_frac": alg / (kernel_ms * 1e-3) / 1e9 / HBM_PEAK_GBS if kernel_ms > 0 else None,
                "redone_tiles": redone, "fused": bool(fused)})
        self.t += 1


def measure(w, density, pool, sp, micro, warmup, steps, cycle=False, jsonl=None):
    import torch
    run = Run(w, density, pool, sp, micro, cycle, keep_records=bool(jsonl))
    for _ in range(warmup):
        run.step(timed=False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        run.step(timed=True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    if jsonl:
        with open(jsonl, "a") as f:
            for rec in run.records:
                f.write(json.dumps(rec) + "\n")
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
        "variant": run.variant,
        "fused": run.fused,
    }


def cpu_baseline(w, density, pool, target_s, cycle=False):
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
    bounds = {p: oracle.partition(N, p, w.world) for p in (range(w.world) if cycle else w.ranks)}
    theta = {p: synth.initial_theta(w, pool[0], s, s + ln, density) for p, (s, ln) in bounds.items()}
    cap = max(ln for _, ln in bounds.values())
    out = (np.empty(max(1, cap), np.int32), np.empty(max(1, cap), np.float32))
    # fault every host page in before timing, as the device buffers are
    # resident before the GPU's timed region
    res[:] = 0.0
    out[0][:] = 0
    out[1][:] = 0.0
    spent, elems, steps = 0.0, 0, 0
    with OneCore() as pin:
        while spent < target_s and steps < 10000:
            g = pool[steps % len(pool)]
            parts = [oracle.cycle(steps, worker, w.world) if cycle else worker for worker in w.ranks]
            for p in parts:
                s, ln = bounds[p]
                g_host[s:s + ln].copy_(g[s:s + ln])
            gn = g_host.numpy()
            for p in parts:
                _, ln = bounds[p]
                t0 = time.perf_counter()
                _, _, _, theta[p] = oracle.step(gn, res, p, w.world, density, theta[p], out=out)
                spent += time.perf_counter() - t0
                elems += ln
            steps += 1
    return {
        "value": elems / spent / 1e9,
        "unit": "G elem/s",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"{steps} step(s) of {w.name} at d={density} ({elems} values, "
                   f"{spent:.1f} s of single-threaded oracle time), {pin.describe()}"),
    }


def _partition_lengths(w):
    import paper_2310_00967_amd as micro
    return [micro.micro_partition(w.n_total, c, w.world)[1] for c in range(w.world)]


def measure_ef(w, density, pool, sp, warmup, steps, local_error=False):
    """Full error-feedback passes of worker w.ranks[0] at iterations 0, 1, ...
    (its searched partition rotates): 12 B per value of the whole vector plus
    8 B per selected value."""
    import torch
    import paper_2310_00967_amd as micro
    from paper_2310_00967_amd import synth
    worker = w.ranks[0]
    N = w.n_total
    res = torch.zeros(N, dtype=torch.float32, device="cuda")
    out_idx, out_val = sp.outputs(max(_partition_lengths(w)))
    s, ln = micro.micro_partition(N, micro.micro_cycle(0, worker, w.world), w.world)
    theta = synth.initial_theta(w, pool[0], s, s + ln, density)
    log = []
    t0 = time.perf_counter()
    for t in range(warmup + steps):
        if t == warmup:
            torch.cuda.synchronize()
            t0 = time.perf_counter()
        g = pool[t % len(pool)]
        out = sp.ef_step(g, res, t, worker, w.world, density, theta, out_idx, out_val, local_error=local_error)
        k, theta = out[0], out[1]
        if t >= warmup:
            log.append((N, k, sp.last_stats()[0]))
    fused = bool(sp.last_stats()[3])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    alg = sum(12 * n + 8 * k for n, k, _ in log)
    kernel_s = sum(ms for _, _, ms in log) / 1e3
    return {"g_elem_s": sum(n for n, _, _ in log) / elapsed / 1e9, "wall_gbs": alg / elapsed / 1e9,
            "kernel_gbs": alg / kernel_s / 1e9, "kernel_ms_avg": kernel_s * 1e3 / len(log),
            "alg_bytes_per_launch": alg / len(log), "ms_per_step": elapsed * 1e3 / steps,
            "k_avg": sum(k for _, k, _ in log) / len(log), "worker": worker, "fused": fused}


def measure_topk(w, density, pool, warmup, steps, only_topk=False, hint="last"):
    """The exact top-k comparator (MICRO_RULE_TOPK) on partition w.ranks[0],
    beside the threshold step (the default rule) and the hard-threshold rule
    (Sec. 1's comparators) on the same gradients, each with its own residual
    under error feedback: device time per step from the library's events
    (for top-k they include the host's wait between the step and the passes
    over its list), and the density each rule selects at every step, warm-up
    included.  Each top-k call gets the k-th magnitude the last one returned
    as its hint, as a training loop passes theta on; the first gets the
    calibrated initial threshold.  Algorithmic bytes for every rule: what any
    selection of the partition has to move, 12 B per value (grad and residual
    read, residual written) plus 8 B per selected value; the top-k rule's
    extra passes show in a lower fraction."""
    import torch
    import paper_2310_00967_amd as micro
    from paper_2310_00967_amd import synth
    rank = w.ranks[0]
    N = w.n_total
    start, ln = micro.micro_partition(N, rank, w.world)
    theta0 = synth.initial_theta(w, pool[0], start, start + ln, density)
    rules = {"topk": micro.MICRO_RULE_TOPK, "threshold": micro.MICRO_RULE_PROPORTIONAL,
             "hard_threshold": micro.MICRO_RULE_HARD_THRESHOLD}
    if only_topk:
        rules = {"topk": micro.MICRO_RULE_TOPK}
    out = {}
    for name, rule in rules.items():
        sp = micro.Sparsifier(N, device="cuda", time_kernel=True, rule=rule)
        res = torch.zeros(N, dtype=torch.float32, device="cuda")
        out_idx, out_val = sp.outputs(ln)
        theta = theta0
        ks, ms, routes = [], [], []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for t in range(warmup + steps):
            if t == warmup:
                torch.cuda.synchronize()
                t0 = time.perf_counter()
            theta_in = theta
            if rule == micro.MICRO_RULE_TOPK and hint != "last":
                theta_in = float("nan") if hint == "none" else 8.0 * theta
            k, theta_out, _, _ = sp.step(pool[t % len(pool)], res, rank, w.world, density, theta_in, out_idx,
                                         out_val)
            # a top-k call with no hint hands back the theta it got when it
            # selects nothing; keep the last k-th magnitude for the next call
            theta = theta_out if not (rule == micro.MICRO_RULE_TOPK and theta_out != theta_out) else theta
            ks.append(k)
            if t >= warmup:
                ms.append(sp.last_stats()[0])
            if rule == micro.MICRO_RULE_TOPK:
                routes.append(sp.last_topk_route())
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        sp.close()
        del res
        kernel_ms = sum(ms) / len(ms)
        k_avg = sum(ks[warmup:]) / steps
        alg = 12 * ln + 8 * k_avg
        dens = [k / ln for k in ks]
        half = dens[len(dens) // 2:]
        out[name] = {"kernel_ms_avg": kernel_ms, "ms_per_step": elapsed * 1e3 / steps,
                     "g_elem_s": ln * steps / elapsed / 1e9, "alg_bytes_per_launch": alg,
                     "kernel_gbs": alg / (kernel_ms * 1e-3) / 1e9,
                     "frac": alg / (kernel_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, "k_avg": k_avg,
                     "density_series": dens,
                     "density_error_last_half": sum(abs(x - density) / density for x in half) / len(half)}
        if routes:
            out[name]["route_series"] = routes
    out["partition"] = (rank, start, ln)
    return out


def build_up(w, density, steps, rho=0.5):
    """Sec. 5.2's gradient build-up on synthetic data: `world` simulated
    workers, each with its own residual and its own gradient per step
    (sqrt(rho) * a draw shared by all workers + sqrt(1 - rho) * its own draw,
    so the per-tensor scale is kept), select under three rules; the density of
    the union of their selections is what the all-reduce would carry.  Top-k
    and the hard threshold search the whole vector on every worker (the
    paper's comparators); MiCRO's workers each search partition
    ((t mod n) + i) mod n of Algorithm 1 (micro_ef_step), so their selections
    never overlap.  Returns the per-step union densities and the mean of the
    workers' own densities."""
    import torch
    import paper_2310_00967_amd as micro
    from paper_2310_00967_amd import synth
    n, N = w.world, w.n_total
    a, b = rho ** 0.5, (1.0 - rho) ** 0.5

    def grad(t, i):
        g = synth.gradient(w, t, "cuda")
        g.mul_(a).add_(synth.gradient(w, 100_000 + t * n + i, "cuda"), alpha=b)
        return g

    g0 = grad(0, 0)
    theta_hard = synth.initial_theta(w, g0, 0, N, density)
    theta_part = {p: synth.initial_theta(w, g0, s, s + ln, density)
                  for p, (s, ln) in ((p, micro.micro_partition(N, p, n)) for p in range(n))}
    del g0
    rules = {"topk": micro.Sparsifier(N, device="cuda", rule=micro.MICRO_RULE_TOPK),
             "hard_threshold": micro.Sparsifier(N, device="cuda", rule=micro.MICRO_RULE_HARD_THRESHOLD),
             "micro": micro.Sparsifier(N, device="cuda")}
    res = {r: [torch.zeros(N, dtype=torch.float32, device="cuda") for _ in range(n)] for r in rules}
    out_idx = torch.empty(N, dtype=torch.int32, device="cuda")
    out_val = torch.empty(N, dtype=torch.float32, device="cuda")
    theta_topk = [1.0] * n
    union = {r: [] for r in rules}
    own = {r: [] for r in rules}
    for t in range(steps):
        picked = {r: [] for r in rules}
        dens = {r: 0.0 for r in rules}
        for i in range(n):
            g = grad(t, i)
            k, theta_topk[i], idx, _ = rules["topk"].step(g, res["topk"][i], 0, 1, density, theta_topk[i],
                                                          out_idx, out_val)
            picked["topk"].append(idx.clone())
            dens["topk"] += k / N / n
            k, _, idx, _ = rules["hard_threshold"].step(g, res["hard_threshold"][i], 0, 1, density, theta_hard,
                                                        out_idx, out_val)
            picked["hard_threshold"].append(idx.clone())
            dens["hard_threshold"] += k / N / n
            part = micro.micro_cycle(t, i, n)
            k, theta_part[part], _, idx, _ = rules["micro"].ef_step(g, res["micro"][i], t, i, n, density,
                                                                    theta_part[part], out_idx, out_val)
            picked["micro"].append(idx.clone())
            dens["micro"] += k / (N / n) / n
            del g
        for r in rules:
            union[r].append(int(torch.unique(torch.cat(picked[r])).numel()) / N)
            own[r].append(dens[r])
    for sp in rules.values():
        sp.close()
    half = steps // 2
    return {"workers": n, "rho": rho, "steps": steps,
            "union_density": union, "worker_density": own,
            "union_over_target_last_half": {r: sum(v[half:]) / len(v[half:]) / density for r, v in union.items()}}


def cpu_baseline_topk(w, density, pool, target_s):
    """The oracle's top-k selection, single-threaded on one pinned core, on
    the worker's partition (a prefix of 2^25 values where the partition is
    longer: its sort is O(P log P)), repeated for about target_s seconds."""
    import oracle
    import paper_2310_00967_amd as micro
    start, ln = micro.micro_partition(w.n_total, w.ranks[0], w.world)
    n = min(ln, 1 << 25)
    g = pool[0][start:start + n].cpu().numpy()
    res0 = pool[1 % len(pool)][start:start + n].cpu().numpy() * 0.5
    done, elapsed = 0, 0.0
    with OneCore() as core:
        while elapsed < target_s or done == 0:
            res = res0.copy()
            t0 = time.perf_counter()
            oracle.topk_select(g, res, 0, n, density)
            elapsed += time.perf_counter() - t0
            done += 1
    what = "the partition" if n == ln else f"the first {n} values of the partition"
    return {"value": done * n / elapsed / 1e9, "unit": "G elem/s", "cores": 1, "kind": "oracle",
            "sample": f"{done} top-k selection(s) of {what} of {w.name} rank {w.ranks[0]} ({n} values, "
                      f"d={density}, {elapsed:.1f} s of single-threaded oracle time), {core.describe()}"}


def measure_sweep(w, density, pool, sp, warmup, steps):
    """Every partition of the workload per step in one micro_sweep_step call
    (with the local-error norms): 12 B per value plus 8 B per selected value."""
    import torch
    from paper_2310_00967_amd import synth
    N = w.n_total
    res = torch.zeros(N, dtype=torch.float32, device="cuda")
    out_idx, out_val = sp.outputs(N)
    thetas = []
    for r in range(w.world):
        s, ln = sp.partition(r, w.world)
        thetas.append(synth.initial_theta(w, pool[0], s, s + ln, density))
    log, errs = [], []
    t0 = time.perf_counter()
    for t in range(warmup + steps):
        if t == warmup:
            torch.cuda.synchronize()
            t0 = time.perf_counter()
        g = pool[t % len(pool)]
        k, thetas, sq, _, _ = sp.sweep(g, res, w.world, density, thetas, out_idx, out_val)
        if t >= warmup:
            log.append((N, sum(k), sp.last_stats()[0]))
            errs.append(math.sqrt(sum(sq)))
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    alg = sum(12 * n + 8 * k for n, k, _ in log)
    kernel_s = sum(ms for _, _, ms in log) / 1e3
    return {"g_elem_s": sum(n for n, _, _ in log) / elapsed / 1e9, "wall_gbs": alg / elapsed / 1e9,
            "kernel_gbs": alg / kernel_s / 1e9, "kernel_ms_avg": kernel_s * 1e3 / len(log),
            "alg_bytes_per_launch": alg / len(log), "ms_per_step": elapsed * 1e3 / steps,
            "k_avg": sum(k for _, k, _ in log) / len(log), "local_error_last": errs[-1],
            "fused": bool(sp.last_stats()[3])}


def build_union(w, density, g, sp):
    """The union of all n workers' selections on gradient g (each partition at
    its calibrated threshold), in partition order, and worker w.ranks[0]'s own
    run in it at its first cycle."""
    import torch
    import paper_2310_00967_amd as micro
    from paper_2310_00967_amd import synth
    parts, own_first = [], 0
    worker = w.ranks[0]
    mine = micro.micro_cycle(0, worker, w.world)
    for c in range(w.world):
        s, ln = micro.micro_partition(w.n_total, c, w.world)
        th = synth.initial_theta(w, g, s, s + ln, density)
        res = torch.zeros(w.n_total, dtype=torch.float32, device="cuda")
        k, _, idx, val = sp.step(g, res, c, w.world, density, th)
        if c == mine:
            own_first = sum(p[0].numel() for p in parts)
            own_val = val.clone()
        parts.append((idx.clone(), val.clone()))
        del res
    union = torch.cat([p[0] for p in parts])
    return union, own_first, own_val


def measure_union(w, density, g, sp, warmup, steps):
    """Gather/reset (micro_union_gather) and model update (micro_sparse_update)
    over the union of all workers' selections.  Algorithmic bytes per union
    entry: gather 16 B outside the worker's own run (index, residual read,
    output, residual reset), 8 B inside it (own value, output); update 16 B
    (index, sum, parameter read and write)."""
    import torch
    union, own_first, own_val = build_union(w, density, g, sp)
    m, k_own = union.numel(), own_val.numel()
    res = (g * 0.5).contiguous()           # any accumulated values
    x = torch.ones(w.n_total, dtype=torch.float32, device="cuda")
    out = torch.empty(m, dtype=torch.float32, device="cuda")
    log = []
    t0 = time.perf_counter()
    for t in range(warmup + steps):
        if t == warmup:
            torch.cuda.synchronize()
            t0 = time.perf_counter()
        sp.union_gather(res, union, own_first, own_val, out)
        ms_g = sp.last_stats()[0]
        sp.sparse_update(x, union, out, w.world)
        ms_u = sp.last_stats()[0]
        if t >= warmup:
            log.append((ms_g, ms_u))
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    alg_g = 16 * (m - k_own) + 8 * k_own
    alg_u = 16 * m
    kg = sum(a for a, _ in log) / 1e3
    ku = sum(b for _, b in log) / 1e3
    vendor = vendor_union_ops(union, res, x, out, w.world, warmup, steps)
    return {"g_entries_s": m * steps / elapsed / 1e9, "union_len": m, "own_len": k_own, "vendor": vendor,
            "wall_gbs": (alg_g + alg_u) * steps / elapsed / 1e9,
            "kernel_gbs": (alg_g + alg_u) * steps / (kg + ku) / 1e9,
            "gather_ms_avg": kg * 1e3 / steps, "update_ms_avg": ku * 1e3 / steps,
            "gather_gbs": alg_g * steps / kg / 1e9, "update_gbs": alg_u * steps / ku / 1e9,
            "alg_bytes_per_launch": (alg_g + alg_u), "ms_per_step": elapsed * 1e3 / steps,
            "union": union, "own_first": own_first, "own_val": own_val}


def vendor_union_ops(union, res, x, out, world, warmup, steps):
    """torch's own random-access kernels on the same union, event-timed on
    torch's stream, for comparison with the union kernels: a gather
    (index_select), a scatter of zeros (index_fill_) and a scatter-add
    (index_add_) at the union's indices (torch takes int64 indices)."""
    import torch
    idx64 = union.long()
    stream = torch.cuda.current_stream()
    vals = out.clone()

    def timed(fn):
        ms = []
        for i in range(warmup + steps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            e1.synchronize()
            if i >= warmup:
                ms.append(e0.elapsed_time(e1))
        return sum(ms) / len(ms)

    return {"index_select_ms": timed(lambda: torch.index_select(res, 0, idx64)),
            "index_fill_ms": timed(lambda: res.index_fill_(0, idx64, 0.0)),
            "index_add_ms": timed(lambda: x.index_add_(0, idx64, vals, alpha=-1.0 / world)),
            "entries": union.numel()}


def cpu_baseline_ef(w, density, pool, target_s):
    """The oracle's full pass on the host, as cpu_baseline does for the step."""
    import numpy as np
    import torch
    import oracle
    from paper_2310_00967_amd import synth
    N = w.n_total
    worker = w.ranks[0]
    res = np.zeros(N, np.float32)
    g_host = torch.empty(N, dtype=torch.float32, pin_memory=True)
    cap = max(_partition_lengths(w))
    out = (np.empty(max(1, cap), np.int32), np.empty(max(1, cap), np.float32))
    res[:] = 0.0
    out[0][:] = 0
    out[1][:] = 0.0
    s, ln = oracle.partition(N, oracle.cycle(0, worker, w.world), w.world)
    theta = synth.initial_theta(w, pool[0], s, s + ln, density)
    spent, elems, steps = 0.0, 0, 0
    with OneCore() as pin:
        while spent < target_s and steps < 10000:
            g_host.copy_(pool[steps % len(pool)])
            gn = g_host.numpy()
            t0 = time.perf_counter()
            _, _, _, theta, _ = oracle.ef_step(gn, res, steps, worker, w.world, density, theta, out=out)
            spent += time.perf_counter() - t0
            elems += N
            steps += 1
    return {"value": elems / spent / 1e9, "unit": "G elem/s", "cores": 1, "kind": "oracle",
            "sample": (f"{steps} full pass(es) of {w.name} worker {worker} at d={density} ({elems} values, "
                       f"{spent:.1f} s of single-threaded oracle time), {pin.describe()}")}


def cpu_baseline_sweep(w, density, pool, target_s):
    """The oracle's sweep (every partition, with the squared norms) on the host."""
    import numpy as np
    import torch
    import oracle
    from paper_2310_00967_amd import synth
    N = w.n_total
    res = np.zeros(N, np.float32)
    res[:] = 0.0
    g_host = torch.empty(N, dtype=torch.float32, pin_memory=True)
    thetas = []
    for r in range(w.world):
        s, ln = oracle.partition(N, r, w.world)
        thetas.append(synth.initial_theta(w, pool[0], s, s + ln, density))
    spent, elems, steps = 0.0, 0, 0
    with OneCore() as pin:
        while spent < target_s and steps < 10000:
            g_host.copy_(pool[steps % len(pool)])
            gn = g_host.numpy()
            t0 = time.perf_counter()
            _, _, _, thetas, _ = oracle.sweep(gn, res, w.world, density, thetas)
            spent += time.perf_counter() - t0
            elems += N
            steps += 1
    return {"value": elems / spent / 1e9, "unit": "G elem/s", "cores": 1, "kind": "oracle",
            "sample": (f"{steps} sweep(s) of {w.name} over {w.world} partitions at d={density} ({elems} values, "
                       f"{spent:.1f} s of single-threaded oracle time), {pin.describe()}")}


def cpu_baseline_union(w, g, union_res, target_s):
    """The oracle's gather, reset and update over the same union on the host."""
    import numpy as np
    import oracle
    union = union_res["union"].cpu().numpy()
    acc = (g * 0.5).cpu().numpy()
    x = np.ones(w.n_total, np.float32)
    spent, entries, reps = 0.0, 0, 0
    with OneCore() as pin:
        while spent < target_s and reps < 10000:
            t0 = time.perf_counter()
            vals = oracle.gather(acc, union)
            oracle.zero(acc, union)
            oracle.update(x, union, vals, w.world)
            spent += time.perf_counter() - t0
            entries += union.size
            reps += 1
    return {"value": entries / spent / 1e9, "unit": "G entries/s", "cores": 1, "kind": "oracle",
            "sample": (f"{reps} gather+reset+update pass(es) over a {union.size}-entry union of {w.name} "
                       f"({spent:.1f} s of single-threaded oracle time), {pin.describe()}")}


def bert_block(args):
    """BERT-large rank 3 of 8 (41,892,736 values, d = 0.01), the other
    workload whose partition holds at least 25M values, measured in the same
    run as the headline: its own gradient pool and context, the fixed rank and
    then worker 3 under Algorithm 1's rotation (every partition in turn, one
    threshold each)."""
    import torch
    import paper_2310_00967_amd as micro
    from paper_2310_00967_amd import synth
    w = synth.get("bert_large")
    d = w.densities[0]
    warmup, steps = max(args.warmup, 10), max(args.steps, 20)
    n_pool = max(1, min(warmup + steps, int(args.pool_gb * 1e9 // (4 * w.n_total))))
    pool = [synth.gradient(w, t, "cuda") for t in range(n_pool)]
    torch.cuda.synchronize()
    sp = micro.Sparsifier(w.n_total, device="cuda", time_kernel=True)
    block = {}
    for cycle in (False, True):
        r = measure(w, d, pool, sp, micro, warmup, steps, cycle)
        traffic = None if cycle else read_traffic(TRAFFIC_FILE_BERT, f"bert_large world 8 rank 3 d={d}")
        key = "bert_large_worker3_cycle" if cycle else "bert_large_rank3"
        block[key] = {
            "partition_len": micro.micro_partition(w.n_total, 3, w.world)[1], "density": d,
            "partitions": ("cyclic: partition ((t mod 8) + 3) mod 8 at step t" if cycle else "fixed: rank 3"),
            "warmup": warmup, "steps": steps, "gradient_pool": n_pool,
            "g_elem_s": r["g_elem_s"], "ms_per_step": r["ms_per_step"], "wall_gbs": r["wall_gbs"],
            "kernel_ms_avg": r["kernel_ms_avg"], "kernel_gbs": r["kernel_gbs"],
            "frac": r["kernel_gbs"] / HBM_PEAK_GBS, "alg_bytes_per_launch": r["alg_bytes_per_launch"],
            "traffic": traffic, "density_error_last_half": r["density_error_last_half"],
            "kernel": ("stream_scan_kernel + move_kernel" if r["fused"] else "stream_kernel + scan_kernel + move_kernel")
            + " (one step, event-timed together)",
            "redone_tiles_timed": r["redone_tiles"]}
    block["bert_large_rank3"]["vendor_add_rotating_out"] = vendor_add_rotating(w, pool, 3, warmup, steps)
    sp.close()
    del pool
    torch.cuda.empty_cache()
    return block


def vendor_add_rotating(w, pool, rank, warmup, steps):
    """torch.add(g, e, out=e) on one partition, the step's two-read, one-write
    stream without the selection, with the gradient rotating over the pool and
    e over three buffers (so no call re-reads an operand that the previous call
    left in the Infinity Cache); HIP events around each call."""
    import torch
    import paper_2310_00967_amd as micro
    start, n = micro.micro_partition(w.n_total, rank, w.world)
    gs = [g[start:start + n] for g in pool]
    outs = [torch.zeros(n, dtype=torch.float32, device="cuda") for _ in range(3)]
    stream = torch.cuda.current_stream()
    ms = []
    for i in range(warmup + steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        torch.add(gs[i % len(gs)], outs[i % 3], out=outs[i % 3])
        e1.record(stream)
        e1.synchronize()
        if i >= warmup:
            ms.append(e0.elapsed_time(e1))
    avg = sum(ms) / len(ms)
    gbs = 12.0 * n / (avg * 1e-3) / 1e9
    return {"ms_avg": avg, "bytes": 12.0 * n, "gbs": gbs, "frac": gbs / HBM_PEAK_GBS}


MALL_BYTES = 256 * 1024 * 1024  # MI355X Infinity Cache


def stream_ceiling(args, w, head, pool, sp):
    """Streams of the vendor libraries beside the library's step, on the
    worker's partition (the whole vector at world 1), each `steps` times after
    `warmup` runs on torch's current stream: torch.add(g, res, out=res) (two
    reads and one write per value: the step's streaming pattern without the
    selection), res.copy_(g) (one read, one write: a device copy), torch.sum(g)
    (reads only) and res.fill_ (writes only), and the sparsify step.  The
    gradient rotates over the pool.  Where an operand fits the 256 MB Infinity
    Cache, back-to-back calls on one output re-read it from that cache, which a
    training step (forward and backward passes between two selections) does
    not leave in place: the in-place add and the step are then also timed with
    the output (the residual) rotating over three buffers.  Event-timed; GB/s
    from the bytes each must move (12, 8, 4, 4 and 12 + 8 d bytes per value)."""
    import torch
    import paper_2310_00967_amd as micro
    from paper_2310_00967_amd import synth
    rank = w.ranks[0]
    start, N = micro.micro_partition(w.n_total, rank, w.world)
    gs = [g[start:start + N] for g in pool]
    res = torch.zeros(N, dtype=torch.float32, device="cuda")
    res_step = torch.zeros(w.n_total, dtype=torch.float32, device="cuda")
    cache_sized = 4 * N <= MALL_BYTES
    rot = [torch.zeros(N, dtype=torch.float32, device="cuda") for _ in range(3)] if cache_sized else []
    rot_step = ([torch.zeros(w.n_total, dtype=torch.float32, device="cuda") for _ in range(2)] + [res_step]
                if cache_sized else [])
    out_idx, out_val = sp.outputs(N)
    theta0 = synth.initial_theta(w, pool[0], start, start + N, head)
    stream = torch.cuda.current_stream()

    def timed(fn):
        ms = []
        for i in range(args.warmup + args.steps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn(i)
            e1.record(stream)
            e1.synchronize()
            if i >= args.warmup:
                ms.append(e0.elapsed_time(e1))
        return sum(ms) / len(ms)

    def stepper(residuals):
        state = {"theta": theta0, "ks": [], "lib_ms": []}

        def step(i):
            k, state["theta"], _, _ = sp.step(pool[i % len(pool)], residuals[i % len(residuals)], rank, w.world,
                                              head, state["theta"], out_idx, out_val)
            if i >= args.warmup:
                state["ks"].append(k)
                state["lib_ms"].append(sp.last_stats()[0])
        return step, state

    rows = {}
    rows["torch_add_inplace"] = (timed(lambda i: torch.add(gs[i % len(gs)], res, out=res)), 12.0 * N)
    if rot:
        rows["torch_add_inplace_rotating_out"] = (
            timed(lambda i: torch.add(gs[i % len(gs)], rot[i % 3], out=rot[i % 3])), 12.0 * N)
    rows["device_copy"] = (timed(lambda i: res.copy_(gs[i % len(gs)])), 8.0 * N)
    rows["torch_sum_read_only"] = (timed(lambda i: torch.sum(gs[i % len(gs)])), 4.0 * N)
    rows["torch_fill_write_only"] = (timed(lambda i: res.fill_(1.0)), 4.0 * N)
    step, st = stepper([res_step])
    step_ms = timed(step)
    k_avg = sum(st["ks"]) / len(st["ks"])
    rows["sparsify_step"] = (step_ms, 12.0 * N + 8.0 * k_avg)
    lib = {"sparsify_step": sum(st["lib_ms"]) / len(st["lib_ms"])}
    if rot_step:
        step, st = stepper(rot_step)
        step_ms = timed(step)
        k_rot = sum(st["ks"]) / len(st["ks"])
        rows["sparsify_step_rotating_residual"] = (step_ms, 12.0 * N + 8.0 * k_rot)
        lib["sparsify_step_rotating_residual"] = sum(st["lib_ms"]) / len(st["lib_ms"])
    kernels = {name: {"ms_avg": ms, "bytes": b, "gbs": b / (ms * 1e-3) / 1e9,
                      "frac": b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS} for name, (ms, b) in rows.items()}
    for name, ms in lib.items():  # the library's own events around its two launches
        b = rows[name][1]
        kernels[name].update({"lib_ms_avg": ms, "lib_gbs": b / (ms * 1e-3) / 1e9,
                              "lib_frac": b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS})
    line = {"metric": "streaming ceiling: vendor streams beside the sparsify step (GB/s of the bytes each must move)",
            "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "dtype": "f32", "data": "synthetic",
            "config": {"workload": w.name, "n_total": w.n_total, "world": w.world, "rank": rank,
                       "partition_len": N, "density": head},
            "kernels": kernels, "step_k_avg": k_avg}
    print(json.dumps(line), flush=True)


def main_path(args, w, head, pool, n_pool, sp):
    """The JSON line of --path ef / --path union."""
    common = {"n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "higher_is_better": True,
              "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic"}
    cfg = {"workload": w.name, "n_total": w.n_total, "world": w.world, "worker": w.ranks[0],
           "density": head, "distribution": w.dist, "gradient_pool": n_pool,
           "parallelism": "one worker on one GPU", "path": args.path}
    if args.path == "topk":
        r = measure_topk(w, head, pool, args.warmup, args.steps, args.topk_only, args.topk_hint)
        cpu = cpu_baseline_topk(w, head, pool, args.cpu_seconds) if args.cpu_seconds > 0 else None
        rank, start, ln = r.pop("partition")
        cfg.update({"rank": rank, "partition_len": ln, "parallelism": "one worker's partition on one GPU",
                    "topk_hint": args.topk_hint})
        tk = r["topk"]
        line = {"metric": "exact top-k comparator throughput (G elem/s of the partition), beside the threshold step",
                "value": tk["g_elem_s"], "unit": "G elem/s", "ms_per_step": tk["ms_per_step"], **common,
                "config": cfg, "k_avg": tk["k_avg"],
                "roofline": {"bound": "hbm", "achieved": tk["kernel_gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                             "frac": tk["frac"],
                             "traffic": (read_traffic(TRAFFIC_FILE_TOPK,
                                                      f"{w.name} world {w.world} rank {rank} topk d={head}",
                                                      sources=TOPK_SOURCES)
                                         if args.topk_hint == "last" else None),
                             "kernel": "the threshold step at 7/8 of the incoming theta (the last step's k-th "
                                       "magnitude), the wait, three topk_hist_kernel + topk_select_kernel passes "
                                       "over its output list and the trim (route_series 3; 4: the list fell short "
                                       "and the passes and the pick ran over the residual; 1 and 2: no hint, the "
                                       "passes over the partition first); event-timed together",
                             "kernel_ms_avg": tk["kernel_ms_avg"], "alg_bytes_per_launch": tk["alg_bytes_per_launch"]},
                "topk_over_threshold_step_time": (tk["kernel_ms_avg"] / r["threshold"]["kernel_ms_avg"]
                                                  if "threshold" in r else None),
                "rules": r,
                "build_up": (build_up(w, head, 24) if not args.topk_only and w.world > 1 else None),
                "cpu_baseline": cpu}
        print(json.dumps(line), flush=True)
        return
    if args.path == "sweep":
        r = measure_sweep(w, head, pool, sp, args.warmup, args.steps)
        cpu = cpu_baseline_sweep(w, head, pool, args.cpu_seconds) if args.cpu_seconds > 0 else None
        cfg["parallelism"] = "every partition of one vector on one GPU"
        cfg["ranks"] = list(range(w.world))
        traffic = read_traffic(TRAFFIC_FILE_SWEEP, f"{w.name} world {w.world} sweep d={head}")
        line = {"metric": "partition-sweep throughput (G elem/s of the whole vector, HBM GB/s % of peak)",
                "value": r["g_elem_s"], "unit": "G elem/s", "ms_per_step": r["ms_per_step"], **common,
                "config": cfg, "k_avg": r["k_avg"], "local_error_last": r["local_error_last"],
                "roofline": {"bound": "hbm", "achieved": r["kernel_gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                             "frac": r["kernel_gbs"] / HBM_PEAK_GBS, "traffic": traffic,
                             "kernel": ("stream_scan_sweep_kernel + move_sweep_kernel" if r["fused"] else
                                        "stream_sweep_kernel + scan_sweep_kernel + move_sweep_kernel")
                                       + " (one sweep, event-timed together)",
                             "kernel_ms_avg": r["kernel_ms_avg"], "alg_bytes_per_launch": r["alg_bytes_per_launch"]},
                "cpu_baseline": cpu}
    elif args.path == "ef":
        r = measure_ef(w, head, pool, sp, args.warmup, args.steps, args.local_error)
        cfg["local_error"] = args.local_error
        cpu = cpu_baseline_ef(w, head, pool, args.cpu_seconds) if args.cpu_seconds > 0 else None
        traffic = read_traffic(TRAFFIC_FILE_EF, f"{w.name} world {w.world} worker {w.ranks[0]} ef d={head}"
                               + (" local-error" if args.local_error else ""))
        line = {"metric": "full error-feedback pass throughput (G elem/s of the whole vector, HBM GB/s % of peak)",
                "value": r["g_elem_s"], "unit": "G elem/s", "ms_per_step": r["ms_per_step"], **common,
                "config": cfg, "k_avg": r["k_avg"],
                "roofline": {"bound": "hbm", "achieved": r["kernel_gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                             "frac": r["kernel_gbs"] / HBM_PEAK_GBS, "traffic": traffic,
                             "kernel": (("stream_scan_sweep_kernel + move_sweep_kernel" if r["fused"] else
                                         "stream_sweep_kernel + scan_sweep_kernel + move_sweep_kernel")
                                        + " over three segments (one pass with the local error, event-timed together)"
                                        if args.local_error else
                                        "accumulate_kernel + stream_scan_kernel + move_kernel "
                                        "(one pass, event-timed together)" if r["fused"] else
                                        "accumulate_kernel + stream_kernel + scan_kernel + move_kernel "
                                        "(one pass, event-timed together)"),
                             "kernel_ms_avg": r["kernel_ms_avg"], "alg_bytes_per_launch": r["alg_bytes_per_launch"]},
                "cpu_baseline": cpu}
    else:
        r = measure_union(w, head, pool[0], sp, args.warmup, args.steps)
        cpu = cpu_baseline_union(w, pool[0], r, args.cpu_seconds) if args.cpu_seconds > 0 else None
        cfg.update({"union_len": r["union_len"], "own_len": r["own_len"]})
        traffic = read_traffic(TRAFFIC_FILE_UNION, f"{w.name} world {w.world} worker {w.ranks[0]} union d={head}",
                               sources=(UNION_SRC, KERNEL_HDR))
        line = {"metric": "union gather/reset + model update throughput (G union entries/s, HBM GB/s % of peak)",
                "value": r["g_entries_s"], "unit": "G entries/s", "ms_per_step": r["ms_per_step"], **common,
                "config": cfg,
                "roofline": {"bound": "hbm", "achieved": r["kernel_gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                             "frac": r["kernel_gbs"] / HBM_PEAK_GBS, "traffic": traffic,
                             "kernel": "union_gather_kernel + sparse_update_kernel (event-timed each)",
                             "gather_ms_avg": r["gather_ms_avg"], "update_ms_avg": r["update_ms_avg"],
                             "gather_gbs": r["gather_gbs"], "update_gbs": r["update_gbs"],
                             "alg_bytes_per_launch": r["alg_bytes_per_launch"]},
                "vendor_random_access": r["vendor"],
                "cpu_baseline": cpu}
    print(json.dumps(line), flush=True)


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py: --gpus {args.gpus} is not supported: the sparsify step has no collective "
              "and this benchmark measures one GPU (one worker's partition at its real size).",
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
    variant = {"auto": micro.MICRO_VARIANT_AUTO, "staged": micro.MICRO_VARIANT_STAGED,
               "ticket": micro.MICRO_VARIANT_TICKET}[args.variant]
    sp = micro.Sparsifier(w.n_total, device="cuda", time_kernel=True, variant=variant,
                          separate_scan=args.separate_scan)
    if args.path == "ceiling":
        stream_ceiling(args, w, head, pool, sp)
        sp.close()
        return
    if args.path != "step":
        main_path(args, w, head, pool, n_pool, sp)
        sp.close()
        return

    main_res = measure(w, head, pool, sp, micro, args.warmup, args.steps, args.cycle, args.steps_jsonl)
    extra = {}
    for d in others:
        r = measure(w, d, pool, sp, micro, args.warmup, args.steps, args.cycle, args.steps_jsonl)
        extra[f"d={d}"] = {k: r[k] for k in ("g_elem_s", "wall_gbs", "kernel_gbs", "kernel_ms_avg",
                                             "density_error_last_half", "ms_per_step")}
        extra[f"d={d}"]["kernel_hbm_frac"] = r["kernel_gbs"] / HBM_PEAK_GBS

    cpu = cpu_baseline(w, head, pool, args.cpu_seconds, args.cycle) if args.cpu_seconds > 0 else None
    sp.close()
    if w.name == "gpt_1p3b" and not args.no_extra and not args.cycle:
        del pool
        torch.cuda.empty_cache()
        extra.update(bert_block(args))

    traffic_file, traffic_workload = {
        "gpt_1p3b": (TRAFFIC_FILE, "gpt_1p3b world 1 rank 0 d=0.01"),
        "bert_large": (TRAFFIC_FILE_BERT, "bert_large world 8 rank 3 d=0.01")}.get(args.workload, (None, None))
    traffic = (read_traffic(traffic_file, traffic_workload) if traffic_file and head == 0.01 and not args.cycle
               and not args.separate_scan and args.variant == "auto" else None)
    parts = sorted({ln for (_, ln) in (micro.micro_partition(w.n_total, p, w.world)
                                       for p in (range(w.world) if args.cycle else w.ranks))})
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
            "partitions": ("cyclic: worker i searches partition ((t mod world) + i) mod world at step t"
                           if args.cycle else "fixed: each listed rank searches its own partition every step"),
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
            "kernel": ("ticket_kernel" if main_res["variant"] != micro.MICRO_VARIANT_STAGED else
                       "stream_scan_kernel + move_kernel (one step, event-timed together)" if main_res["fused"] else
                       "stream_kernel + scan_kernel + move_kernel (one step, event-timed together)"),
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
