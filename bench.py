#!/usr/bin/env python3
"""Benchmark of the GEM commit pipeline on one MI355X.

One step is one simulated run of the workload's T commits: gem_sim_run plans
the passes (validation, snapshot routing) and launches the fused
stale-gradient + GEM-commit pass kernel once per K commits.  The schedule of
the asynchronous system (which worker commits when, with what staleness) is
the synthetic input: it is drawn by the library's host schedule generator
before timing, for warmup + steps consecutive runs, so the system keeps
running across steps.  The problem (h, theta*) is resident in HBM before the
timed region.

Prints one JSON line: parameter-commits/s (P x commits/s) and the fused
pass's algorithmic HBM bandwidth against the 8 TB/s peak, with the CPU oracle
timed on a bounded sample as a reported baseline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# VALU issue ceiling of one MI355X: the fp32 vector peak, 157.3 TFLOP/s =
# 256 CUs x 2.4 GHz x 256 flop per CU and cycle, is two wave64 FMA
# instructions (128 flop each) per CU and cycle: 1228.8 G wave64 VALU
# instructions per second.  Instructions slower than a full-rate FMA (64-bit
# integer multiplies, transcendental approximations) only lower what a real
# instruction mix can reach.
VALU_PEAK_GINST = 256 * 2.4 * 2
# The same figure counts two lanes' FMAs per packed-FP32 instruction slot; the
# library builds without packed FP32, and its integer and unpacked instructions
# issue at one wave64 instruction per SIMD every four cycles: 4 SIMDs x 256 CUs
# x 2.4 GHz / 4 = 614.4 G/s (the fp64 vector rate, 78.6 TFLOP/s, in the same
# units).
VALU_ISSUE_GINST = 256 * 2.4
METRIC = "parameter-commits/s (P×commits/s) + achieved HBM GB/s vs peak, P=25M n=100"
KERNEL_SOURCES = ("gem_kernels.hip", "gem_device.hpp", "gem_internal.hpp", "gem_plan.hpp",
                  "gem_layout.hpp")
# Committed rocprofv3 counter summaries of the dominant kernel, per (workload,
# proxy, pi scope), each taken with the library's own cache rule.
COUNTERS_FILES = {
    ("headline", "local", "element"): "pass_kernel_headline_counters.md",
    ("headline", "global", "element"): "pass_kernel_headline_global_proxy_counters.md",
    ("small", "local", "element"): "pass_kernel_small_counters.md",
    ("resnet18", "local", "element"): "pass_kernel_resnet18_counters.md",
    ("large", "local", "element"): "pass_kernel_large_counters.md",
    ("headline", "local", "segment"): "seg_step_kernel_headline_counters.md",
}


def kernel_hash() -> str:
    """Hash of the kernel sources' code: comments and blank lines removed, so
    an edit of comments alone keeps counter summaries taken on the same code."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_1805_08469_amd", "csrc", f)) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)      # block comments
        text = re.sub(r"//[^\n]*", "", text)                    # line comments
        code = "\n".join(line.rstrip() for line in text.splitlines() if line.strip())
        h.update(code.encode())
    return h.hexdigest()[:16]


def measured_counters(workload: str, proxy: str, scope: str):
    """The machine-readable block of the committed rocprofv3 counter summary
    for this configuration (HBM bytes and VALU instructions per launch of the
    dominant kernel), if it was taken on the current kernel source; else None."""
    name = COUNTERS_FILES.get((workload, proxy, scope))
    path = os.path.join(ROOT, "profiles", name) if name else None
    if path is None or not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"```json\s*(\{.*?\})\s*```", text, flags=re.S)
    if not m:
        return None
    d = json.loads(m.group(1))
    if (d.get("kernel_hash") != kernel_hash() or d.get("workload") != workload
            or d.get("proxy", "local") != proxy or d.get("pi_scope", "element") != scope):
        return None
    return d


def host_description() -> dict:
    """The CPU the oracle baseline ran on."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = None
    return {"cpu_model": model, "logical_cores": os.cpu_count(), "usable_cores": usable}


def cpu_baseline(wl, h, ts, worker, tau, sample_elems: int, sample_commits: int, ghp):
    """The oracle (single-threaded C, as it stands) on the first sample_commits
    commits of the same schedule over the first sample_elems parameters."""
    import numpy as np
    import oracle as O

    idx = np.arange(sample_elems, dtype=np.int64)
    hp = O.Hyper(lr=wl.lr, sigma=wl.sigma, momentum=wl.momentum, bf16=wl.bf16, seed=wl.seed,
                 kappa=ghp.kappa, pi_mode=ghp.pi_mode, rule=ghp.rule, proxy=ghp.proxy_mode)
    st = O.State.initial(wl.n, sample_elems)
    t0 = time.perf_counter()
    O.run(hp, wl.P, st, idx, h[:sample_elems], ts[:sample_elems], worker[:sample_commits],
          tau[:sample_commits])
    dt = time.perf_counter() - t0
    return {
        "value": sample_elems * sample_commits / dt,
        "unit": "param-commits/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"first {sample_commits} commits of the {wl.name} schedule on parameters "
                  f"0..{sample_elems - 1} ({dt:.1f} s, single thread)",
        "host": host_description(),
    }


def copy_ceiling(G, torch, nbytes: int, reps: int = 10) -> float:
    """Device-to-device copy bandwidth (read + write bytes / time) of the
    library's plain copy kernel, the practical HBM ceiling."""
    n = nbytes // 4
    src = torch.empty(n, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    G.gem_copy_f32(src.data_ptr(), dst.data_ptr(), n)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        assert G.gem_copy_f32(src.data_ptr(), dst.data_ptr(), n) == G.GEM_OK
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    return 2 * nbytes / (ms * 1e-3) / 1e9


def compute_floor(G, torch, wl, hp, cache: int, pi_hist: bool, passes: int = 12) -> float:
    """Milliseconds of compute per commit of the workload's pass kernel: the
    same kernel over the same P with one worker, in passes of GEM_K_MAX
    commits.  That worker's snapshot and moment stay in the register slots for
    the whole pass, so a pass moves 32 bytes per parameter for 32 commits and
    its time is the noise generator's and the commit arithmetic's.  A real
    configuration of the method (GEM with a single worker), run through
    gem_sim_run."""
    import numpy as np
    stream = torch.cuda.current_stream()
    K = G.GEM_K_MAX
    T = passes * K
    worker = np.zeros(T, dtype=np.int32)
    with G.Gem(wl.P, 1, hp, stream=stream.cuda_stream) as g:
        g.set_cache_policy(cache)
        g.set_quadratic(*problem_arrays(wl), wl.lr, wl.sigma, wl.seed, bf16=wl.bf16)
        g.sim_run(worker[:2 * K], None, K)                  # warm-up
        if pi_hist:
            G.gem_pi_hist_start(g.h, T)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        g.sim_run(worker, None, K)
        e1.record(stream)
        torch.cuda.synchronize()
    return e0.elapsed_time(e1) / T


_PROBLEM = {}


def problem_arrays(wl):
    """h and theta* of the workload (drawn once per process)."""
    from paper_1805_08469_amd.workloads import problem
    if wl.name not in _PROBLEM:
        _PROBLEM[wl.name] = problem(wl)
    return _PROBLEM[wl.name]


def compare_rules(G, P: int = 1 << 20, T: int = 3000, every: int = 500, K: int = 16):
    """Loss per parameter, every `every` commits, of GEM (mu = 0.9), DOWNPOUR and
    the adaptive-staleness rule (both mu = 0) on a synthetic diagonal quadratic
    (h ~ LogUniform[1e-3, 1], theta* ~ N(0, 1), noise sigma = 0.1), for n = 1..30
    exponential-time workers and a normal (0.01), a larger (0.1) and a
    misspecified (0.5) learning rate: the experiments of Sec. 4 on stability and
    misspecification, run through the library."""
    from paper_1805_08469_amd.workloads import make_problem
    h, ts = make_problem(P, 1e-3, 1.0, 31)
    rules = {"gem": (G.GEM_RULE_GEM, 0.9), "downpour": (G.GEM_RULE_DOWNPOUR, 0.0),
             "adaptive": (G.GEM_RULE_ADAPTIVE, 0.0)}
    table = []
    for lr in (0.01, 0.1, 0.5):
        for n in (1, 5, 10, 20, 30):
            worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=n)
            for name, (rule, mu) in rules.items():
                hp = G.gem_hyperparams_default()
                hp.rule, hp.momentum = rule, mu
                curve = []
                with G.Gem(P, n, hp) as g:
                    g.set_quadratic(h, ts, lr, 0.1, 9)
                    for c in range(0, T, every):
                        g.sim_run(worker[c:c + every], tau[c:c + every], K)
                        curve.append(G.gem_diag(g.h).loss / P)
                table.append({"lr": lr, "n": n, "rule": name, "commits_per_point": every,
                              "loss_per_param": curve})
    # Appendix B: the high-energy proxy, kappa in both forms, 20 workers, eta = 0.01.
    kappa_table = []
    worker, tau = G.gem_schedule_make(20, T, G.GEM_LAW_EXP, seed=20)
    for mode, name in ((G.GEM_KAPPA_LINEAR, "linear"), (G.GEM_KAPPA_SQRT, "sqrt")):
        for kappa in (1.0, 2.0, 3.0, 4.0, 8.0):
            hp = G.gem_hyperparams_default()
            hp.kappa, hp.kappa_mode = kappa, mode
            curve = []
            with G.Gem(P, 20, hp) as g:
                g.set_quadratic(h, ts, 0.01, 0.1, 9)
                for c in range(0, T, every):
                    g.sim_run(worker[c:c + every], tau[c:c + every], K)
                    curve.append(G.gem_diag(g.h).loss / P)
            kappa_table.append({"kappa": kappa, "form": name, "n": 20, "lr": 0.01,
                                "commits_per_point": every, "loss_per_param": curve})
    return {"experiment": "rule comparison on a synthetic quadratic", "P": P, "T": T, "K": K,
            "sigma": 0.1, "data": "synthetic", "table": table, "kappa_table": kappa_table}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="headline",
                    choices=["tiny", "small", "resnet18", "headline", "large"])
    ap.add_argument("--rule", default="gem", choices=["gem", "downpour", "adaptive"],
                    help="commit rule (GEM, or the DOWNPOUR / adaptive-staleness baselines)")
    ap.add_argument("--pi", default="clamp0", choices=["clamp0", "literal"])
    ap.add_argument("--proxy", default="local", choices=["local", "global"])
    ap.add_argument("--kappa", type=float, default=1.0)
    ap.add_argument("--pi-scope", default="element", choices=["element", "segment"],
                    help="pi per parameter, or per segment from norms (one global segment)")
    ap.add_argument("--pi-hist", action="store_true",
                    help="record the per-commit histograms of the scale factor during the timed "
                         "steps (the diagnostic kernel variant)")
    ap.add_argument("--cache", default="auto", choices=["auto", "keep", "stream"],
                    help="cache policy of the passes: the library's rule (stream when the state "
                         "outgrows the Infinity Cache), the default policy, or streaming")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle timing (profiling runs)")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the copy-ceiling and compute-floor measurements after the timed "
                         "steps (profiling runs: they launch the same kernels on other shapes)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run the copy kernel (counter calibration) and exit")
    ap.add_argument("--compare", action="store_true",
                    help="only run the rule comparison (GEM, DOWNPOUR, adaptive staleness over "
                         "worker counts and learning rates) and print its loss table")
    ap.add_argument("--cpu-sample-elems", type=int, default=1 << 20)
    ap.add_argument("--cpu-sample-commits", type=int, default=256)
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is not supported "
              "(the path shards by parameter index with no exchange per commit, but only the "
              "one-GPU kernel is built and measured)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_1805_08469_amd import gem as G
    from paper_1805_08469_amd.workloads import WORKLOADS, problem

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    torch.cuda.set_device(0)

    if args.copy_probe:
        gbs = copy_ceiling(G, torch, 1 << 30)
        print(json.dumps({"copy_probe_bytes": 1 << 30, "copy_GBps": gbs}), flush=True)
        return 0

    if args.compare:
        print(json.dumps(compare_rules(G)), flush=True)
        return 0

    wl = WORKLOADS[args.workload]
    h, ts = problem_arrays(wl)
    total = (args.warmup + args.steps) * wl.T
    worker, tau = G.gem_schedule_make(wl.n, total, wl.law, wl.law_p0, wl.law_p1, seed=wl.seed)

    hp = G.gem_hyperparams_default()
    hp.rule = {"gem": G.GEM_RULE_GEM, "downpour": G.GEM_RULE_DOWNPOUR,
               "adaptive": G.GEM_RULE_ADAPTIVE}[args.rule]
    hp.pi_mode = G.GEM_PI_LITERAL if args.pi == "literal" else G.GEM_PI_CLAMP0
    hp.proxy_mode = G.GEM_PROXY_GLOBAL if args.proxy == "global" else G.GEM_PROXY_LOCAL
    hp.kappa = args.kappa
    hp.pi_scope = G.GEM_PI_SEGMENT if args.pi_scope == "segment" else G.GEM_PI_ELEMENT
    fast = (args.rule, args.pi, args.kappa, args.pi_scope) == ("gem", "clamp0", 1.0, "element")
    variant = "General" if not fast else "FastGlobal" if args.proxy == "global" else "Fast"
    # The library's ring depth for these passes (deep: the default rule with
    # per-worker moments in passes of at least 16 commits).
    depth = 4 if variant == "Fast" and wl.K >= 16 else 2
    # The library streams (non-temporal accesses) when theta, h, theta* and the
    # snapshot/moment table outgrow the 256 MiB Infinity Cache.
    tiles = -(-(-(-wl.P // 64) * 64) // 8192)
    state_bytes = 4 * (tiles * wl.n * 2 * 8192 + 3 * (-(-wl.P // 64) * 64))
    streaming = state_bytes > (256 << 20) if args.cache == "auto" else args.cache == "stream"

    stream = torch.cuda.current_stream()
    cache = {"auto": G.GEM_CACHE_AUTO, "keep": G.GEM_CACHE_KEEP,
             "stream": G.GEM_CACHE_STREAM}[args.cache]
    g = G.Gem(wl.P, wl.n, hp, stream=stream.cuda_stream)
    g.set_cache_policy(cache)
    g.set_quadratic(h, ts, wl.lr, wl.sigma, wl.seed, bf16=wl.bf16)
    torch.cuda.synchronize()

    def step(k):
        sl = slice(k * wl.T, (k + 1) * wl.T)
        g.sim_run(worker[sl], tau[sl], wl.K)

    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    G.gem_stats_reset(g.h)
    if args.pi_hist:
        G.gem_pi_hist_start(g.h, args.steps * wl.T)

    # One event at every step boundary, on the stream the passes run on: the
    # first and last bracket the timed region, the others give per-step times.
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev[0].record(stream)
    for k in range(args.steps):
        step(args.warmup + k)
        ev[k + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    gpu_s = ev[0].elapsed_time(ev[-1]) * 1e-3
    step_ms = sorted(ev[k].elapsed_time(ev[k + 1]) for k in range(args.steps))
    stats = G.gem_stats(g.h)
    assert stats.commits == args.steps * wl.T
    g.close()
    copy_gbs = None if args.no_ceilings else copy_ceiling(G, torch, 2 << 30)
    # The compute floor of a pass of K commits (not defined for the
    # per-segment scope, whose commits are not fused).
    floor_ms = (compute_floor(G, torch, wl, hp, cache, args.pi_hist) * wl.K
                if args.pi_scope == "element" and not args.no_ceilings else None)

    elapsed = max(gpu_s, 1e-12)
    value = wl.P * stats.commits / elapsed
    passes = stats.passes
    alg_per_pass = stats.alg_bytes / passes
    avg_pass_s = elapsed / passes
    achieved = alg_per_pass / avg_pass_s / 1e9
    # The counter summaries were taken with the library's own cache rule.
    counted = (args.rule, args.pi, args.kappa) == ("gem", "clamp0", 1.0)
    cnt = (measured_counters(wl.name, args.proxy, args.pi_scope)
           if counted and args.cache == "auto" and not args.pi_hist else None)
    traffic = cnt.get("hbm_bytes_per_pass") if cnt else None
    floor_share = floor_ms / (avg_pass_s * 1e3) if floor_ms else None
    # The pass is reported against the ceiling it is nearer to: the compute
    # floor of its arithmetic, or the library's copy rate on HBM.  A pass far
    # from both (a launch-bound one over a tiny vector) keeps the HBM roofline.
    if floor_share is not None and copy_gbs and floor_share > max(achieved / copy_gbs, 0.5):
        valu = cnt.get("valu_instrs_per_pass") if cnt else None
        ach = valu / avg_pass_s / 1e9 if valu else None
        roof = {"bound": "alu", "achieved": ach, "peak": VALU_PEAK_GINST,
                "unit": "G wave64 VALU instructions/s",
                "frac": ach / VALU_PEAK_GINST if ach else None, "traffic": traffic,
                "valu_instrs_per_launch": valu,
                "unpacked_issue_peak": VALU_ISSUE_GINST,
                "frac_of_unpacked_issue": ach / VALU_ISSUE_GINST if ach else None,
                "hbm_GBps": achieved, "hbm_frac": achieved / HBM_PEAK_GBS}
    else:
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS, "traffic": traffic}

    result = {
        "metric": METRIC,
        "value": value,
        "unit": "param-commits/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3,
        "step_ms": {"median": step_ms[len(step_ms) // 2], "min": step_ms[0],
                    "max": step_ms[-1]},
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16-updates/f32" if wl.bf16 else "f32",
        "data": "synthetic",
        "config": {
            "workload": wl.name, "P": wl.P, "n": wl.n, "commits_per_step": wl.T, "K": wl.K,
            "sigma": wl.sigma, "lr": wl.lr, "momentum": wl.momentum,
            "worker_law": {0: "exp", 1: "exp_uniform_mean", 2: "exp_lognormal_mean",
                           3: "pareto"}[wl.law],
            "passes_per_step": passes / args.steps,
            "rule": args.rule, "pi": args.pi, "proxy": args.proxy, "kappa": args.kappa,
            "pi_scope": args.pi_scope, "cache": args.cache, "pi_hist": args.pi_hist,
            "parallelism": "single-gpu",
        },
        "roofline": {
            **roof,
            "alg_bytes_per_launch": alg_per_pass,
            "avg_launch_ms": avg_pass_s * 1e3,
            "kernel": (("seg_step_kernel + seg_blocks_kernel" + (", streaming" if streaming else ""))
                       if args.pi_scope == "segment"
                       # the default rule records through its recording pass; the
                       # other variants through the diagnostic one (depth 2, default policy)
                       else "pass_kernel<Generated, Fast, recording, depth %d%s>"
                       % (depth, ", streaming" if streaming else "")
                       if args.pi_hist and variant == "Fast"
                       else "pass_kernel<Generated, %s, diagnostic, depth 2>" % variant
                       if args.pi_hist
                       # a pass of one commit runs the kernel compiled for one commit
                       else "pass_kernel<Generated, %s, depth %d%s>"
                       % (variant, 1 if wl.K == 1 else depth,
                          ", streaming" if streaming else "")),
            "copy_ceiling_GBps": copy_gbs,
            "frac_of_copy": achieved / copy_gbs if copy_gbs else None,
            "compute_floor_ms": floor_ms,
            "frac_of_compute_floor": floor_share,
        },
        "wall_s": wall,
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, h, ts, worker, tau, min(args.cpu_sample_elems, wl.P),
                                              min(args.cpu_sample_commits, total), hp)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
