#!/usr/bin/env python3
"""Benchmark of SMAT's fused per-step transform on one MI355X.

One step = one pass of the whole hot path over the tensor list with inputs resident in HBM:
    set per-tensor params -> simulate (theta~ into the buffers) -> switch to simulated storage
    -> backward-accumulate (grad_theta += lambda t m g~) -> restore the expert storage.
Default workload: the 7B-shaped decoder list (290 tensors, 7,504,924,672 parameters, fp32 master
weights, bf16 base / simulated weights / upstream gradient).  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--config c4] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "fused simulate+backward params/s and achieved HBM GB/s (% of peak), 7B-shaped"
PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E
# Peak Philox4x32-10 rate on MI355X, derived from the chip: the fp32 vector peak (157.3 TFLOP/s =
# 78.6e12 FMA/s over 256 CUs x 4 SIMDs at 2.4 GHz) is 32 lanes per cycle per SIMD for single-rate
# operations; v_mad_u64_u32 runs at a quarter of that (measured 1.9e13/s chip-wide).  One call as the
# kernels form it costs 17 such products and 19 single-rate xors: 17 x 8 + 19 x 2 = 174 SIMD cycles
# per 64 calls, i.e. 1024 x 2.4e9 x 64 / 174 calls/s.
PEAK_PHILOX_CALLS = 1024 * 2.4e9 * 64 / 174
KERNEL_SOURCES = ("paper_2609_33437_amd/csrc/smat_kernels.hip", "paper_2609_33437_amd/csrc/smat_device.h",
                  "paper_2609_33437_amd/csrc/smat_tile.h")
MERGE_SOURCES = ("paper_2609_33437_amd/csrc/smat_merge.hip", "paper_2609_33437_amd/csrc/smat_device.h",
                 "paper_2609_33437_amd/csrc/smat_tile.h", "paper_2609_33437_amd/csrc/smat_launch.h")


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_hash(sources=KERNEL_SOURCES) -> str:
    h = hashlib.sha256()
    for rel in sources:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(kernel: str, workload: str, sources=KERNEL_SOURCES):
    """HBM bytes per launch from committed rocprofv3 counter runs, if taken on the current kernels."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_sha") != kernel_hash(sources):
        return None
    return rec


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default 20 on the 7B-shaped list; smaller lists take proportionally more, "
                         "at most 2000, so that every list times about the same amount of work)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed steps first (default: 5, or steps / 4)")
    ap.add_argument("--config", default="c4", choices=["c1", "c2", "c3", "c4", "c5"])
    ap.add_argument("--cpu-sample", type=int, default=3 << 27, help="most elements the CPU oracle baseline visits")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="CPU work budget of the oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--adamw", action="store_true",
                    help="also time a simulated training step whose optimizer update is fused with the gradient "
                         "through the simulation, against backward-accumulate + torch's AdamW on the same list")
    ap.add_argument("--offload", action="store_true",
                    help="theta0 in pinned host memory, copied into the simulated buffers at each restore; "
                         "also reports the prefetch's host-link rate")
    ap.add_argument("--summarize", metavar="DIR",
                    help="turn rocprofv3 CSV output under DIR (trace/, fetch/, write/, and opt_*/, merge_*/ when present) into the "
                         "summaries under profiles/ and exit")
    ap.add_argument("--train", action="store_true",
                    help="time SMAT inside a bf16 training loop of a Llama-1B-shaped synthetic decoder against "
                         "plain fine-tuning (AdamW, clipping at 1), print that comparison as the JSON line and exit")
    ap.add_argument("--merge", action="store_true",
                    help="time the N-expert merge (Task Arithmetic and DARE + Task Arithmetic) of seven bf16 "
                         "experts shaped like the chosen list, print that as the JSON line and exit")
    ap.add_argument("--graph", action="store_true",
                    help="time one simulated step (simulate + backward-accumulate, a new sampled scale per step) "
                         "issued from the host against the same step replayed from one captured HIP graph of "
                         "the device-driven calls, on the chosen list; print that as the JSON line and exit")
    ap.add_argument("--experts", type=int, default=7)
    ap.add_argument("--train-batch", type=int, default=8)
    ap.add_argument("--train-seq", type=int, default=512)
    ap.add_argument("--train-reps", type=int, default=3)
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain elementwise copy of 2^28 fp32 values (1 GiB read, 1 GiB written) "
                         "three times, whose HBM counters scale the kernels' counter readings")
    return ap.parse_args()


# Worker threads of the CPU baseline: one per host core the process may run on, at most 16, the host
# share that goes with one GPU on the MI355X boxes this runs on.
CPU_WORKER_CAP = 16


def default_steps(args, cfg):
    """(steps, warmup): as given, else 20 and 5 on the 7B-shaped list and, on a smaller list, as many
    more as it takes to time about the same work (at most 2000 steps): a few hundred microseconds per
    step are too short to time after the clock has settled with only 20 steps."""
    ref = 7_504_924_672
    k = args.steps if args.steps is not None else int(min(2000, max(20, -(-20 * ref // cfg.numel))))
    w = args.warmup if args.warmup is not None else (5 if k <= 20 else max(5, k // 4))
    return k, w


def sample_windows(cfg, max_elems: int, seed: int = 1234):
    """Windows (tensor, first element, length) of every tensor, each a fraction of its tensor,
    together at most about max_elems elements, in random tensor order."""
    import numpy as np
    frac = min(1.0, max_elems / cfg.numel)
    rng = np.random.default_rng(seed)
    wins = []
    for i in rng.permutation(cfg.count):
        n = cfg.specs[i].numel
        m = max(1, int(round(n * frac)))
        wins.append((int(i), int(rng.integers(0, n - m + 1)), m))
    return frac, wins


def window_tasks(wins, inp, g_pre, torch, np, piece: int = 1 << 20):
    """Host copies of the windows' inputs, split into pieces of at most `piece` elements so that the
    threads share the big tensors: (tensor, global offset, theta, theta0, grad_sim, grad_theta before
    the step).  bf16 arrays as their uint16 bits, as the oracle takes them."""
    def bits(x):
        return x.view(torch.int16).numpy().view(np.uint16) if x.dtype == torch.bfloat16 else x.numpy()

    tasks = []
    for (i, a, m), gp in zip(wins, g_pre):
        th = inp.theta[i].view(-1)[a:a + m].cpu().numpy()
        t0 = bits(inp.theta0[i].view(-1)[a:a + m].cpu())
        gs = bits(inp.grad_sim[i].view(-1)[a:a + m].cpu())
        for b in range(0, m, piece):
            e = min(m, b + piece)
            tasks.append((i, a + b, th[b:e], t0[b:e], gs[b:e], gp[b:e]))
    return tasks


def cpu_baseline(cfg, tasks, params, step, budget_s):
    """The CPU oracle on a bounded sample of the same workload (the windows of `tasks`): simulate with
    its rounding, then backward-accumulate, in fp64 NumPy on a pool of threads (NumPy's array loops
    run without the GIL).  No new window starts after `budget_s` seconds.  Returns the baseline
    record and the oracle outputs of every window it finished, for the parity check."""
    import concurrent.futures as cf

    import oracle

    t0_dt, g_dt, out_dt = cfg.theta0_dtype, cfg.grad_dtype, cfg.out_dtype
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = os.cpu_count() or 1
    workers = max(1, min(affinity, CPU_WORKER_CAP))
    start = time.perf_counter()
    deadline = start + budget_s

    def run(k):
        if time.perf_counter() >= deadline:
            return None
        i, off, th, t0, gs, gp = tasks[k]
        y, kept, eps = oracle.simulate_f64(th, t0, t0_dt, params[i], cfg.smat_seed, step, i, off)
        oracle.round_to(y, out_dt)
        want = oracle.backward_accum(gs, g_dt, gp, params[i], cfg.lam, cfg.smat_seed, step, i, off)
        return k, y, kept, eps, want

    with cf.ThreadPoolExecutor(max_workers=workers) as pool:
        outs = [r for r in pool.map(run, range(len(tasks))) if r is not None]
    secs = time.perf_counter() - start
    done = sum(tasks[r[0]][2].size for r in outs)
    log(f"cpu oracle: {done} elements in {secs:.1f} s on {workers} threads")
    rec = {"value": done / secs, "unit": "params/s", "cores": workers, "kind": "oracle",
           "affinity_cores": affinity, "worker_cap": CPU_WORKER_CAP,
           "sample": f"{done} elements: windows of {100 * min(1.0, done / cfg.numel):.3f}% of the {cfg.count} "
                     f"tensors in random order (simulate + backward, fp64 NumPy, {workers} threads), {secs:.1f} s wall"}
    return rec, outs


def parity_stats(cfg, tasks, oracle_outs, gpu_tt, gpu_g, params, np):
    """The verification step's GPU outputs against the oracle's, window by window, under the test
    suite's bars (tests/tolerances.py): theta~ within half an output ulp plus the fp32 error bound of
    the kernel's arithmetic (within 1 bf16 ulp of the oracle's rounding wherever that bound is below
    half an ulp, the "strict" elements), grad_theta within 1e-6 relative, dropped coordinates of
    grad_theta bit-unchanged."""
    import concurrent.futures as cf

    import oracle
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import tolerances

    t0_dt, g_dt, out_dt = cfg.theta0_dtype, cfg.grad_dtype, cfg.out_dtype

    def one(r):
        k, y, kept, eps, want = r
        i, off, th, t0, gs, gp = tasks[k]
        p = params[i]
        got, gg = gpu_tt[k], gpu_g[k]
        coef = np.where(kept, oracle.coefficient(p["s"], p["keep"], p.get("rescale", 1)), 0.0)
        ok, strict = tolerances.check_theta_tilde(got, out_dt, y, th, oracle.as_f64(t0, t0_dt), coef, eps, p["sigma"])
        if out_dt == "bf16":
            ulp = np.abs(tolerances.ordered(got) - tolerances.ordered(oracle.round_to_bf16_bits(y)))
        else:
            ulp = np.abs(got.view(np.int32).astype(np.int64) - oracle.round_to(y, "f32").view(np.int32).astype(np.int64))
        incr = np.abs(cfg.lam * coef * oracle.as_f64(gs, g_dt))
        gok = tolerances.check_grad(gg, want, gp, incr)
        scale = np.maximum(np.abs(want.astype(np.float64)), np.abs(gp.astype(np.float64)) + incr)
        rel = np.abs(gg.astype(np.float64) - want.astype(np.float64)) / np.where(scale > 0, scale, 1.0)
        dropped_changed = int(np.count_nonzero(gg.view(np.uint32)[~kept] != gp.view(np.uint32)[~kept]))
        return (th.size, int(np.count_nonzero(~ok)), int(ulp.max(initial=0)), int(ulp[strict].max(initial=0)),
                int(np.count_nonzero(~strict)), int(ulp[~strict].max(initial=0)), int(np.count_nonzero(~gok)),
                float(rel.max(initial=0.0)), dropped_changed, int(np.count_nonzero(kept)))

    with cf.ThreadPoolExecutor(max_workers=CPU_WORKER_CAP) as pool:
        rows = list(pool.map(one, oracle_outs))
    col = list(zip(*rows)) if rows else [[0]] * 10
    n = sum(col[0])
    return {"elements": n, "windows": len(rows),
            "theta_tilde": {"mismatches": sum(col[1]), "max_ulp": max(col[2]), "max_ulp_strict": max(col[3]),
                            "nonstrict": sum(col[4]), "nonstrict_max_ulp": max(col[5])},
            "grad_theta": {"mismatches": sum(col[6]), "max_rel_err": max(col[7]),
                           "dropped_changed": sum(col[8]), "kept": sum(col[9])},
            "bars": "theta~ within 1/2 ulp + the fp32 error bound of the kernel's arithmetic (strict elements: "
                    "1 bf16 ulp); grad_theta 1e-6 relative; dropped grad_theta bit-unchanged"}


def timed_copy(nbytes_step: int, torch, smat, reps: int = 5) -> dict:
    """The library's plain streaming copy (smat_stream_copy) moving the same bytes as one step:
    nbytes_step / 2 read and nbytes_step / 2 written, timed with HIP events."""
    n = nbytes_step // 8 // 4 * 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    smat.smat_stream_copy(src, dst)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        smat.smat_stream_copy(src, dst)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    assert bool(dst[-1] == 1.0)
    del src, dst
    torch.cuda.empty_cache()
    return {"bytes": 8 * n, "ms": round(ms, 4), "gbps": round(8 * n / (ms * 1e6), 1)}


# rocprofv3 passes behind profiles/.  Run from /tmp with TMPDIR=/tmp; $REPO is the repository root and
# $REPO/rocprof the output root that `bench.py --summarize $REPO/rocprof` reads.
PROF_NOTE = "run from /tmp with TMPDIR=/tmp; $REPO is the repository root"
TRACE_CMD = ("rocprofv3 --kernel-trace --stats -f csv -d $REPO/rocprof/trace -o c4 -- "
             "python3 $REPO/bench.py")  # the default run: the kernel times behind its JSON line
PMC_CMD = ("rocprofv3 --pmc {ctr} -f csv -d $REPO/rocprof/{tag} -o c4 --kernel-include-regex "
           "'k_simulate_multi|k_backward_multi|elementwise' -- "
           "python3 $REPO/bench.py --steps 2 --warmup 1 --no-cpu-baseline --calibrate-copy")
OPT_TRACE_CMD = ("rocprofv3 --kernel-trace --stats -f csv -d $REPO/rocprof/opt_trace -o c4 -- "
                 "python3 $REPO/bench.py --adamw --steps 10 --warmup 2 --no-cpu-baseline")
OPT_PMC_CMD = ("rocprofv3 --pmc {ctr} -f csv -d $REPO/rocprof/opt_{tag} -o c4 --kernel-include-regex "
               "'k_adamw_multi|k_sqnorm_multi' -- "
               "python3 $REPO/bench.py --adamw --steps 2 --warmup 1 --no-cpu-baseline")
MERGE_TRACE_CMD = ("rocprofv3 --kernel-trace --stats -f csv -d $REPO/rocprof/merge_trace -o c4 -- "
                   "python3 $REPO/bench.py --merge --steps 10 --warmup 2")
MERGE_PMC_CMD = ("rocprofv3 --pmc {ctr} -f csv -d $REPO/rocprof/merge_{tag} -o c4 --kernel-include-regex "
                 "'k_merge_multi' -- python3 $REPO/bench.py --merge --steps 2 --warmup 1")
VALU_CTRS = "VALUBusy SQ_INSTS_VALU SQ_INSTS_SALU SQ_WAVES"
VALU_CMDS = {  # VALU activity and instructions per wave of every kernel of ours, one pass per benchmark mode
    "valu_main": f"rocprofv3 --pmc {VALU_CTRS} -f csv -d $REPO/rocprof/valu_main -o c4 "
                 "--kernel-include-regex 'k_simulate_multi|k_backward_multi' -- "
                 "python3 $REPO/bench.py --steps 2 --warmup 1 --no-cpu-baseline",
    "valu_opt": f"rocprofv3 --pmc {VALU_CTRS} -f csv -d $REPO/rocprof/valu_opt -o c4 "
                "--kernel-include-regex 'k_adamw_multi|k_sqnorm_multi' -- "
                "python3 $REPO/bench.py --adamw --steps 2 --warmup 1 --no-cpu-baseline",
    "valu_merge": f"rocprofv3 --pmc {VALU_CTRS} -f csv -d $REPO/rocprof/valu_merge -o c4 "
                  "--kernel-include-regex 'k_merge_multi' -- python3 $REPO/bench.py --merge --steps 2 --warmup 1",
}
# the other lists: the bench line of `bench.py --config NAME` and its kernel trace, per list
CONFIG_NAMES = {"c1": "c1_flat1m", "c2": "c2_125m", "c3": "c3_1p5b", "c5": "c5_vlm8b"}
CONFIG_TRACE_CMD = ("rocprofv3 --kernel-trace --stats -f csv -d $REPO/rocprof/trace_{cfg} -o {cfg} -- "
                    "python3 $REPO/bench.py --config {cfg}")
CONFIG_BENCH_CMD = "python3 $REPO/bench.py --config {cfg} > $REPO/rocprof/bench_{cfg}.json"
COPY_GRID = 1 << 26   # threads of the calibration copy (2^28 fp32 values, 4 per thread)
COPY_BYTES = 1 << 30  # read and written by one calibration dispatch


def summarize(root: str) -> int:
    """Write profiles/ summaries from rocprofv3 CSV output (kernel stats, FETCH_SIZE, WRITE_SIZE)."""
    import csv
    import statistics

    def kind(name: str, grid: int):
        if "k_simulate_multi" in name:
            return "simulate"
        if "k_backward_multi" in name:
            return "backward"
        if "MulFunctor" in name and grid == COPY_GRID:
            return "copy"
        return None

    out_dir = os.path.join(ROOT, "profiles")
    os.makedirs(out_dir, exist_ok=True)
    stats = list(csv.DictReader(open(os.path.join(root, "trace", "c4_kernel_stats.csv"))))
    lines = ["# Kernel time on the 7B-shaped list (c4), rocprofv3 kernel trace", "",
             f"Command (on one MI355X; {PROF_NOTE}): `{TRACE_CMD}`", "",
             "The default `bench.py` run, whose JSON line quotes the same kernels' HIP-event times.  Each step "
             "launches one simulate and one backward over the 290-tensor list (7,504,924,672 parameters); "
             "5 warmup + 20 timed steps + 20 steps of the kernel-timing pass + 1 verification step = 46 calls "
             "each.  It first runs `smat_stream_copy` over the step's "
             "bytes, the plain-copy reference of the JSON line; the other kernels are torch's input "
             "generation and the runtime's copies (`__amd_rocclr_copyBuffer`) of the CPU baseline's windows "
             "to the host.", "",
             "| kernel | calls | average ms | min ms | max ms | share of GPU time |", "|---|---|---|---|---|---|"]
    for r in stats[:12]:
        name = r["Name"].replace("(anonymous namespace)", "{anon}").split("(")[0].replace("void ", "")
        lines.append(f"| `{name[:80]}` | {r['Calls']} | {float(r['AverageNs']) / 1e6:.4f} | "
                     f"{float(r['MinNs']) / 1e6:.4f} | {float(r['MaxNs']) / 1e6:.4f} | {float(r['Percentage']):.2f}% |")
    avg = {kind(r["Name"], 0): float(r["AverageNs"]) / 1e6 for r in stats if kind(r["Name"], 0)}
    with open(os.path.join(out_dir, "kernels_c4_7b_trace.md"), "w") as f:
        f.write("\n".join(lines) + "\n")

    vals = {}
    for tag, ctr in (("fetch", "FETCH_SIZE"), ("write", "WRITE_SIZE")):
        rows = csv.DictReader(open(os.path.join(root, tag, "c4_counter_collection.csv")))
        for r in rows:
            k = kind(r["Kernel_Name"], int(r["Grid_Size"]))
            if k and r["Counter_Name"] == ctr:
                vals.setdefault((k, tag), []).append(float(r["Counter_Value"]))
    fetch_factor = statistics.median(vals[("copy", "fetch")]) * 1024 / COPY_BYTES
    write_factor = statistics.median(vals[("copy", "write")]) * 1024 / COPY_BYTES
    P = 7504924672
    algo = {"simulate": (P * 6, P * 2), "backward": (P * 6, P * 4)}
    md = ["# HBM traffic per launch on the 7B-shaped list (c4), rocprofv3 counters", "",
          f"Commands ({PROF_NOTE}): `{PMC_CMD.format(ctr='FETCH_SIZE', tag='fetch')}` and the same with "
          "`WRITE_SIZE` (output `rocprof/write`).", "",
          "Counters are KiB per dispatch.  Scale: a plain elementwise copy of 2^28 fp32 values (1 GiB read, "
          f"1 GiB written) reads FETCH_SIZE = {fetch_factor:.4f} x and WRITE_SIZE = {write_factor:.4f} x its "
          "true bytes; kernel readings are divided by these factors.", "",
          "| kernel | FETCH_SIZE KiB | WRITE_SIZE KiB | read GB (scaled) | written GB (scaled) | algorithmic read GB "
          "| algorithmic written GB | traffic / algorithmic |", "|---|---|---|---|---|---|---|---|"]
    for k in ("simulate", "backward"):
        fk = statistics.median(vals[(k, "fetch")])
        wk = statistics.median(vals[(k, "write")])
        rd = fk * 1024 / fetch_factor
        wr = wk * 1024 / write_factor
        ar, aw = algo[k]
        md.append(f"| {k} | {fk:.0f} | {wk:.0f} | {rd / 1e9:.3f} | {wr / 1e9:.3f} | {ar / 1e9:.3f} | {aw / 1e9:.3f} | "
                  f"{(rd + wr) / (ar + aw):.4f} |")
        rec = {"kernel": k, "workload": "c4", "kernel_sha": kernel_hash(),
               "fetch_kib_per_dispatch": fk, "write_kib_per_dispatch": wk,
               "fetch_factor": fetch_factor, "write_factor": write_factor,
               "bytes_per_launch": round(rd + wr), "algorithmic_bytes_per_launch": ar + aw,
               "avg_launch_ms_trace": avg.get(k),
               "commands": [PMC_CMD.format(ctr="FETCH_SIZE", tag="fetch"), PMC_CMD.format(ctr="WRITE_SIZE", tag="write")]}
        with open(os.path.join(out_dir, f"traffic_{k}_c4.json"), "w") as f:
            json.dump(rec, f, indent=1)
    with open(os.path.join(out_dir, "traffic_c4_7b.md"), "w") as f:
        f.write("\n".join(md) + "\n")
    print("\n".join(lines + [""] + md))
    if os.path.isdir(os.path.join(root, "opt_trace")):
        summarize_optimizer(root, out_dir, fetch_factor, write_factor)
    if os.path.isdir(os.path.join(root, "merge_trace")):
        summarize_merge(root, out_dir, fetch_factor, write_factor)
    if all(os.path.isdir(os.path.join(root, d)) for d in VALU_CMDS):
        summarize_valu(root, out_dir)
    summarize_configs(root, out_dir)
    summarize_train(root, out_dir)
    return 0


TRAIN_CMDS = {"resident": "python3 $REPO/bench.py --train > $REPO/rocprof/train_resident.json",
              "offload": "python3 $REPO/bench.py --train --offload > $REPO/rocprof/train_offload.json"}
TRAIN_TRACE_CMD = ("rocprofv3 --kernel-trace --stats -f csv -d $REPO/rocprof/train_trace -o train -- "
                   "python3 $REPO/bench.py --train --train-reps 1")


def summarize_train(root: str, out_dir: str) -> None:
    """profiles/train_llama1b_<mode>.json (the `bench.py --train` lines: SMAT in a training loop
    against plain fine-tuning) and profiles/kernels_train_llama1b_trace.md (the kernels of one
    such run)."""
    import csv

    for mode, cmd in TRAIN_CMDS.items():
        line = os.path.join(root, f"train_{mode}.json")
        if os.path.exists(line):
            with open(line) as f:
                rec = json.loads(f.read().strip().splitlines()[-1])
            with open(os.path.join(out_dir, f"train_llama1b_{mode}.json"), "w") as f:
                json.dump({"command": cmd, "run_from": PROF_NOTE, "kernel_sha": kernel_hash(), "result": rec}, f,
                          indent=1)
                f.write("\n")
    stats_path = os.path.join(root, "train_trace", "train_kernel_stats.csv")
    if not os.path.exists(stats_path):
        return
    stats = list(csv.DictReader(open(stats_path)))
    ours = [r for r in stats if "smat::" in r["Name"]]
    lines = ["# Kernels of the training-loop benchmark (Llama-1B-shaped synthetic decoder), rocprofv3 kernel trace",
             "", f"Command (on one MI355X; {PROF_NOTE}): `{TRAIN_TRACE_CMD}`", "",
             "One repetition of the FT / SMAT / SMAT-fused blocks (each warm-up plus timed steps of batch 8 x 512, "
             "t = 4).  The model's GEMMs (hipBLASLt `Cijk_*`), torch's fused AdamW and elementwise kernels take "
             f"the time; the library's kernels are listed after the top ones.  Kernel sources hash {kernel_hash()}.",
             "", "| kernel | calls | average ms | min ms | max ms | share of GPU time |", "|---|---|---|---|---|---|"]
    for r in stats[:10] + [r for r in ours if r not in stats[:10]]:
        name = r["Name"].replace("(anonymous namespace)", "{anon}").split("(")[0].replace("void ", "")
        lines.append(f"| `{name[:80]}` | {r['Calls']} | {float(r['AverageNs']) / 1e6:.4f} | "
                     f"{float(r['MinNs']) / 1e6:.4f} | {float(r['MaxNs']) / 1e6:.4f} | {float(r['Percentage']):.2f}% |")
    with open(os.path.join(out_dir, "kernels_train_llama1b_trace.md"), "w") as f:
        f.write("\n".join(lines) + "\n")


def summarize_configs(root: str, out_dir: str) -> None:
    """profiles/step_<list>.json (the bench line of `bench.py --config NAME`, with its command and the
    kernel sources' hash) and profiles/kernels_<list>_trace.md (its rocprofv3 kernel trace), for the
    lists other than the headline one."""
    import csv

    for cfg, label in CONFIG_NAMES.items():
        line = os.path.join(root, f"bench_{cfg}.json")
        if os.path.exists(line):
            with open(line) as f:
                rec = json.loads(f.read().strip().splitlines()[-1])
            rec = {"command": CONFIG_BENCH_CMD.format(cfg=cfg), "run_from": PROF_NOTE, "kernel_sha": kernel_hash(),
                   "result": rec}
            with open(os.path.join(out_dir, f"step_{label}.json"), "w") as f:
                json.dump(rec, f, indent=1)
                f.write("\n")
        stats_path = os.path.join(root, f"trace_{cfg}", f"{cfg}_kernel_stats.csv")
        if not os.path.exists(stats_path):
            continue
        stats = list(csv.DictReader(open(stats_path)))
        lines = [f"# Kernel time on the {label} list ({cfg}), rocprofv3 kernel trace", "",
                 f"Command (on one MI355X; {PROF_NOTE}): `{CONFIG_TRACE_CMD.format(cfg=cfg)}`", "",
                 f"`bench.py --config {cfg}` with the defaults: 5 warmup + 20 timed steps + 20 steps of the "
                 "kernel-timing pass + 1 verification step, one simulate and one backward each; first the "
                 "plain-copy reference (`smat_stream_copy`); the other kernels generate the inputs and copy the "
                 f"CPU baseline's windows to the host.  Kernel sources hash {kernel_hash()}.", "",
                 "| kernel | calls | average ms | min ms | max ms | share of GPU time |", "|---|---|---|---|---|---|"]
        for r in stats[:12]:
            name = r["Name"].replace("(anonymous namespace)", "{anon}").split("(")[0].replace("void ", "")
            lines.append(f"| `{name[:80]}` | {r['Calls']} | {float(r['AverageNs']) / 1e6:.4f} | "
                         f"{float(r['MinNs']) / 1e6:.4f} | {float(r['MaxNs']) / 1e6:.4f} | "
                         f"{float(r['Percentage']):.2f}% |")
        with open(os.path.join(out_dir, f"kernels_{label}_trace.md"), "w") as f:
            f.write("\n".join(lines) + "\n")


def summarize_valu(root: str, out_dir: str) -> None:
    """profiles/valu_c4_7b.md: VALU activity of each kernel (rocprofv3 VALUBusy and SQ_INSTS_VALU),
    which tells the HBM-bound streams from the ones whose random draws bound them."""
    import csv
    import statistics

    P = 7504924672
    rows = {}
    for d in VALU_CMDS:
        recs = list(csv.DictReader(open(os.path.join(root, d, "c4_counter_collection.csv"))))
        recs.sort(key=lambda r: int(r["Dispatch_Id"]))
        for r in recs:
            name = r["Kernel_Name"]
            if "k_merge_multi" in name:
                # launch order: 3 Task Arithmetic merges, then 3 DARE merges
                k = "merge"
            else:
                k = next(x for x in ("k_simulate_multi", "k_backward_multi", "k_adamw_multi", "k_sqnorm_multi")
                         if x in name)
            rows.setdefault((k, r["Counter_Name"]), []).append(float(r["Counter_Value"]))
    label = {"k_simulate_multi": "simulate (mask + Gaussian noise draws)", "k_backward_multi": "backward (mask draws)",
             "k_adamw_multi": "fused AdamW (mask draws)", "k_sqnorm_multi": "gradient norm (mask draws, 2 B/param)"}
    md = ["# VALU activity and instructions per wave of the kernels on the 7B-shaped list (c4), rocprofv3 counters",
          "", "Commands (run from /tmp with TMPDIR=/tmp; $REPO is the repository root):", ""]
    md += [f"* `{c}`" for c in VALU_CMDS.values()]
    md += ["", "VALUBusy = 100 * sum(SQ_ACTIVE_INST_VALU) / CU_NUM / GRBM_GUI_ACTIVE (rocprofv3's own expression); "
           "SQ_INSTS_VALU and SQ_INSTS_SALU count wave-level vector and scalar instructions, SQ_WAVES the waves "
           "a launch ran; instructions are given per wave and per parameter of the launch.  Medians over the "
           f"dispatches of each kernel.  Kernel sources hash {kernel_hash()} (merge: {kernel_hash(MERGE_SOURCES)}).",
           "", "| kernel | dispatches | VALUBusy | waves | VALU / wave | SALU / wave | VALU / parameter |",
           "|---|---|---|---|---|---|---|"]

    def row(name, sel):
        vb = rows.get((sel[0], "VALUBusy"), [])[sel[1]]
        if not vb:
            return
        med = {c: statistics.median(rows[(sel[0], c)][sel[1]]) for c in ("SQ_INSTS_VALU", "SQ_INSTS_SALU", "SQ_WAVES")}
        md.append(f"| {name} | {len(vb)} | {statistics.median(vb):.1f} | {med['SQ_WAVES']:.0f} | "
                  f"{med['SQ_INSTS_VALU'] / med['SQ_WAVES']:.1f} | {med['SQ_INSTS_SALU'] / med['SQ_WAVES']:.1f} | "
                  f"{med['SQ_INSTS_VALU'] / P:.4f} |")

    for k in ("k_simulate_multi", "k_backward_multi", "k_adamw_multi", "k_sqnorm_multi"):
        row(label[k], (k, slice(None)))
    if len(rows.get(("merge", "VALUBusy"), [])) >= 6:
        row("merge, Task Arithmetic (7 experts, no draws)", ("merge", slice(0, 3)))
        row("merge, DARE + Task Arithmetic (7 mask draws per quad)", ("merge", slice(3, 6)))
    with open(os.path.join(out_dir, "valu_c4_7b.md"), "w") as f:
        f.write("\n".join(md) + "\n")
    print("\n".join(md))


def summarize_merge(root: str, out_dir: str, fetch_factor: float, write_factor: float) -> None:
    """profiles/ summaries of the N-expert merge on c4 (seven bf16 experts), scaled by the copy
    calibration of the simulate/backward counter runs."""
    import csv
    import statistics

    stats = list(csv.DictReader(open(os.path.join(root, "merge_trace", "c4_kernel_stats.csv"))))
    lines = ["# N-expert merge on the 7B-shaped list (c4, seven bf16 experts), rocprofv3 kernel trace", "",
             f"Command (on one MI355X; {PROF_NOTE}): `{MERGE_TRACE_CMD}`", "",
             "bench.py --merge runs Task Arithmetic (no mask) and then DARE + Task Arithmetic (drop 0.3 on "
             "the linear weights), 2 warmup + 10 timed merges each, through one merge plan; the other kernels "
             "generate the inputs.", "",
             "| kernel | calls | average ms | min ms | max ms | share of GPU time |", "|---|---|---|---|---|---|"]
    for r in stats[:8]:
        name = r["Name"].replace("(anonymous namespace)", "{anon}").split("(")[0].replace("void ", "")
        lines.append(f"| `{name[:90]}` | {r['Calls']} | {float(r['AverageNs']) / 1e6:.4f} | "
                     f"{float(r['MinNs']) / 1e6:.4f} | {float(r['MaxNs']) / 1e6:.4f} | {float(r['Percentage']):.2f}% |")
    with open(os.path.join(out_dir, "kernels_c4_7b_merge_trace.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    # per-dispatch counters in launch order: the first 3 merges are Task Arithmetic, the next 3 DARE
    vals = {}
    for tag, ctr in (("fetch", "FETCH_SIZE"), ("write", "WRITE_SIZE")):
        rows = [r for r in csv.DictReader(open(os.path.join(root, f"merge_{tag}", "c4_counter_collection.csv")))
                if r["Counter_Name"] == ctr]
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        merges = [float(r["Counter_Value"]) for r in rows if "k_merge_multi" in r["Kernel_Name"]]
        vals[tag] = (merges, fetch_factor if tag == "fetch" else write_factor)
    P, N = 7504924672, 7
    algo_r, algo_w = P * 2 * (N + 1), P * 2
    md = ["# HBM traffic per launch of the N-expert merge on c4 (seven bf16 experts), rocprofv3 counters", "",
          f"Commands ({PROF_NOTE}): `{MERGE_PMC_CMD.format(ctr='FETCH_SIZE', tag='fetch')}` and the same with "
          "`WRITE_SIZE` (output `rocprof/merge_write`).", "",
          f"Scaled by the plain-copy calibration of the simulate/backward counter runs (FETCH_SIZE x "
          f"{vals['fetch'][1]:.4f}, WRITE_SIZE x {vals['write'][1]:.4f}).  Algorithmic bytes per parameter: seven experts and theta0 read (16 B), "
          "the merged weights written (2 B).", "",
          "| merge | FETCH_SIZE KiB | WRITE_SIZE KiB | read GB (scaled) | written GB (scaled) | algorithmic GB | "
          "traffic / algorithmic |", "|---|---|---|---|---|---|---|"]
    recs = {}
    for k, sl in (("task_arithmetic", slice(0, 3)), ("dare_task_arithmetic", slice(3, 6))):
        fk = statistics.median(vals["fetch"][0][sl])
        wk = statistics.median(vals["write"][0][sl])
        rd, wr = fk * 1024 / vals["fetch"][1], wk * 1024 / vals["write"][1]
        md.append(f"| {k} | {fk:.0f} | {wk:.0f} | {rd / 1e9:.3f} | {wr / 1e9:.3f} | {(algo_r + algo_w) / 1e9:.3f} | "
                  f"{(rd + wr) / (algo_r + algo_w):.4f} |")
        recs[k] = round(rd + wr)
    with open(os.path.join(out_dir, "traffic_c4_7b_merge.md"), "w") as f:
        f.write("\n".join(md) + "\n")
    rec = {"kernel": "merge", "workload": "c4", "kernel_sha": kernel_hash(MERGE_SOURCES),
           "bytes_per_launch": recs, "algorithmic_bytes_per_launch": algo_r + algo_w,
           "commands": [MERGE_PMC_CMD.format(ctr="FETCH_SIZE", tag="fetch"),
                        MERGE_PMC_CMD.format(ctr="WRITE_SIZE", tag="write")]}
    with open(os.path.join(out_dir, "traffic_merge_c4.json"), "w") as f:
        json.dump(rec, f, indent=1)
    print("\n".join(lines + [""] + md))


def summarize_optimizer(root: str, out_dir: str, fetch_factor: float, write_factor: float) -> None:
    """profiles/ summaries of the optimizer-side kernels (fused AdamW, gradient norm) on c4."""
    import csv
    import statistics

    def kind(name: str):
        if "k_adamw_multi" in name:
            return "adamw"
        if "k_sqnorm_multi" in name:
            return "grad_norm"
        return None

    stats = list(csv.DictReader(open(os.path.join(root, "opt_trace", "c4_kernel_stats.csv"))))
    lines = ["# Optimizer-side kernel time on the 7B-shaped list (c4), rocprofv3 kernel trace", "",
             f"Command (on one MI355X; {PROF_NOTE}): `{OPT_TRACE_CMD}`", "",
             "bench.py --adamw first runs the simulate + backward benchmark, then the fused AdamW step "
             "(unclipped, then clipped at 1 after the gradient-norm pass), then backward-accumulate + "
             "torch's fused AdamW (unclipped, then with torch.nn.utils.clip_grad_norm_).", "",
             "| kernel | calls | average ms | min ms | max ms | share of GPU time |", "|---|---|---|---|---|---|"]
    for r in stats[:16]:
        name = r["Name"].replace("(anonymous namespace)", "{anon}").split("(")[0].replace("void ", "")
        lines.append(f"| `{name[:90]}` | {r['Calls']} | {float(r['AverageNs']) / 1e6:.4f} | "
                     f"{float(r['MinNs']) / 1e6:.4f} | {float(r['MaxNs']) / 1e6:.4f} | {float(r['Percentage']):.2f}% |")
    avg = {kind(r["Name"]): float(r["AverageNs"]) / 1e6 for r in stats if kind(r["Name"])}
    with open(os.path.join(out_dir, "kernels_c4_7b_optimizer_trace.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    vals = {}
    for tag, ctr in (("fetch", "FETCH_SIZE"), ("write", "WRITE_SIZE")):
        for r in csv.DictReader(open(os.path.join(root, f"opt_{tag}", "c4_counter_collection.csv"))):
            k = kind(r["Kernel_Name"])
            if k and r["Counter_Name"] == ctr:
                vals.setdefault((k, tag), []).append(float(r["Counter_Value"]))
    P = 7504924672
    algo = {"adamw": (P * 14, P * 12), "grad_norm": (P * 2, 0)}
    md = ["# HBM traffic per launch of the optimizer-side kernels on c4, rocprofv3 counters", "",
          f"Commands ({PROF_NOTE}): `{OPT_PMC_CMD.format(ctr='FETCH_SIZE', tag='fetch')}` and the same with "
          "`WRITE_SIZE` (output `rocprof/opt_write`).", "",
          f"Scaled by the copy calibration of the simulate/backward counter runs (FETCH_SIZE x {fetch_factor:.4f}, "
          f"WRITE_SIZE x {write_factor:.4f}).  Algorithmic bytes per parameter: fused AdamW reads g~ (bf16, 2 B) and "
          "theta, m1, m2 (12 B) and writes theta, m1, m2 (12 B); the norm pass reads g~ only (2 B).", "",
          "| kernel | avg ms (trace) | FETCH_SIZE KiB | WRITE_SIZE KiB | read GB (scaled) | written GB (scaled) | "
          "algorithmic GB | traffic / algorithmic | achieved GB/s (algorithmic / avg) |", "|---|---|---|---|---|---|---|---|---|"]
    for k in ("adamw", "grad_norm"):
        fk = statistics.median(vals[(k, "fetch")])
        wk = statistics.median(vals[(k, "write")])
        rd, wr = fk * 1024 / fetch_factor, wk * 1024 / write_factor
        ar, aw = algo[k]
        ms = avg.get(k)
        md.append(f"| {k} | {ms:.4f} | {fk:.0f} | {wk:.0f} | {rd / 1e9:.3f} | {wr / 1e9:.3f} | {(ar + aw) / 1e9:.3f} | "
                  f"{(rd + wr) / (ar + aw):.4f} | {(ar + aw) / (ms * 1e6):.0f} |")
    with open(os.path.join(out_dir, "traffic_c4_7b_optimizer.md"), "w") as f:
        f.write("\n".join(md) + "\n")
    print("\n".join(lines + [""] + md))


def bench_adamw(cfg, inp, outs, params, step_ids, seed, K, W, torch, smat):
    """Simulated training step with the optimizer: (a) simulate, switch, fused AdamW on the expert
    storage; (b) simulate, switch, backward-accumulate, switch, torch.optim.AdamW over the same tensors."""
    hp = dict(lr=2e-5, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-3, grad_scale=1.0, step=1)
    P = cfg.numel
    res = {}
    m1 = [torch.zeros(t.numel(), device="cuda") for t in inp.theta]
    m2 = [torch.zeros(t.numel(), device="cuda") for t in inp.theta]
    plan = smat.Plan(inp.theta, outs, inp.theta0, inp.grad_sim, inp.grad_theta)
    plan.bind_adam_state(m1, m2)

    def fused(k, ev=None):
        plan.set_params(params[k])
        plan.simulate(seed, step_ids[k])
        plan.switch_storage(smat.SMAT_SIMULATED)
        plan.switch_storage(smat.SMAT_EXPERT)
        if ev:
            ev[0].record()
        plan.adamw_fused(seed, step_ids[k], cfg.lam, dict(hp, step=k + 1))
        if ev:
            ev[1].record()

    for k in range(W):
        fused(k)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(K)]
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for k in range(K):
        fused(W + k, evs[k])
    b.record()
    torch.cuda.synchronize()
    kern = sum(e[0].elapsed_time(e[1]) for e in evs) / K
    nb = {"bf16": 2, "f32": 4}
    fused_bytes = P * (nb[cfg.grad_dtype] + 24)
    res["fused"] = {"ms_per_step": round(a.elapsed_time(b) / K, 4), "optimizer_kernel_ms": round(kern, 4),
                    "optimizer_kernel_gbps": round(fused_bytes / (kern * 1e6), 1),
                    "optimizer_bytes_per_param": fused_bytes / P}

    # the same with norm clipping at 1: norm pass (reads g~ only), factor kept on the GPU
    coef = torch.ones(1, dtype=torch.float32, device="cuda")

    def clipped(k, ev=None):
        plan.set_params(params[k])
        plan.simulate(seed, step_ids[k])
        plan.switch_storage(smat.SMAT_SIMULATED)
        plan.switch_storage(smat.SMAT_EXPERT)
        if ev:
            ev[0].record()
        plan.grad_norm(seed, step_ids[k], cfg.lam, False, 1.0, None, coef)
        if ev:
            ev[1].record()
        plan.adamw_fused(seed, step_ids[k], cfg.lam, dict(hp, step=W + K + k + 1), grad_scale_dev=coef)
        if ev:
            ev[2].record()

    for k in range(W):
        clipped(k)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
    a.record()
    for k in range(K):
        clipped(W + k, evs[k])
    b.record()
    torch.cuda.synchronize()
    norm_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / K
    clip_kern = sum(e[0].elapsed_time(e[2]) for e in evs) / K
    norm_bytes = P * nb[cfg.grad_dtype]
    res["fused_clipped"] = {"ms_per_step": round(a.elapsed_time(b) / K, 4),
                            "norm_plus_optimizer_ms": round(clip_kern, 4), "grad_norm_ms": round(norm_ms, 4),
                            "grad_norm_gbps": round(norm_bytes / (norm_ms * 1e6), 1),
                            "grad_norm_bytes_per_param": norm_bytes / P}
    plan.close()
    del m1, m2
    torch.cuda.empty_cache()

    params_t = [torch.nn.Parameter(t) for t in inp.theta]   # share the expert storage
    for prm, g in zip(params_t, inp.grad_theta):
        prm.grad = g
    kind = "fused"
    try:
        opt = torch.optim.AdamW(params_t, lr=hp["lr"], betas=(hp["beta1"], hp["beta2"]), eps=hp["eps"],
                                weight_decay=hp["weight_decay"], fused=True)
    except (RuntimeError, ValueError):
        kind = "foreach"
        opt = torch.optim.AdamW(params_t, lr=hp["lr"], betas=(hp["beta1"], hp["beta2"]), eps=hp["eps"],
                                weight_decay=hp["weight_decay"], foreach=True)
    plan = smat.Plan(inp.theta, outs, inp.theta0, inp.grad_sim, inp.grad_theta)

    clip_now = [False]

    def unfused(k, ev=None):
        plan.set_params(params[k])
        plan.simulate(seed, step_ids[k])
        plan.switch_storage(smat.SMAT_SIMULATED)
        if ev:
            ev[0].record()
        plan.backward_accum(seed, step_ids[k], cfg.lam)
        plan.switch_storage(smat.SMAT_EXPERT)
        if clip_now[0]:
            torch.nn.utils.clip_grad_norm_(params_t, 1.0)
        opt.step()
        if ev:
            ev[1].record()

    for k in range(W):
        unfused(k)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(K)]
    a.record()
    for k in range(K):
        unfused(W + k, evs[k])
    b.record()
    torch.cuda.synchronize()
    kern = sum(e[0].elapsed_time(e[1]) for e in evs) / K
    res["unfused"] = {"ms_per_step": round(a.elapsed_time(b) / K, 4), "backward_plus_optimizer_ms": round(kern, 4),
                      "optimizer": f"torch.optim.AdamW({kind}=True)"}
    res["speedup_of_gradient_plus_optimizer"] = round(kern / res["fused"]["optimizer_kernel_ms"], 3)
    clip_now[0] = True
    for k in range(W):
        unfused(k)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(K)]
    a.record()
    for k in range(K):
        unfused(W + k, evs[k])
    b.record()
    torch.cuda.synchronize()
    kern_c = sum(e[0].elapsed_time(e[1]) for e in evs) / K
    res["unfused_clipped"] = {"ms_per_step": round(a.elapsed_time(b) / K, 4),
                              "backward_clip_optimizer_ms": round(kern_c, 4),
                              "clip": "torch.nn.utils.clip_grad_norm_(max_norm=1)"}
    res["speedup_with_clipping"] = round(kern_c / res["fused_clipped"]["norm_plus_optimizer_ms"], 3)
    plan.close()
    log(f"adamw: fused optimizer {res['fused']['optimizer_kernel_ms']:.3f} ms vs backward + torch AdamW "
        f"{kern:.3f} ms; with clipping {res['fused_clipped']['norm_plus_optimizer_ms']:.3f} ms "
        f"(norm {norm_ms:.3f} ms) vs {kern_c:.3f} ms")
    return res


def bench_merge(args, torch, smat, workloads) -> int:
    """N-expert merge (Eq. merged-state) over a list shaped like `--config`: N bf16 experts, bf16
    theta0 and merged output; Task Arithmetic (gamma 0.3, no mask) and DARE + Task Arithmetic (drop
    probability 0.3 on the linear weights), the paper's language-model merger settings."""
    cfg = workloads.config(args.config)
    N = args.experts
    log(f"generating {N} experts shaped like {cfg.name}: {cfg.count} tensors, {cfg.numel} params each")
    t0s, experts = workloads.make_experts(cfg, N, device="cuda")
    outs = [torch.empty_like(t) for t in t0s]
    torch.cuda.synchronize()
    masked = [spec.kind == "linear" for spec in cfg.specs]
    modes = {
        "task_arithmetic": [[dict(gamma=0.3, keep=1.0, seed=0, step=0)] * N for _ in masked],
        "dare_task_arithmetic": [[dict(gamma=0.3, keep=0.7 if m else 1.0, seed=0xDA4E + j, step=0) for j in range(N)]
                                 for m in masked],
    }
    K, W = args.steps, args.warmup
    P = cfg.numel
    nbytes = P * (2 * N + 2 + 2)
    res = {}
    with smat.MergePlan(t0s, outs, experts) as plan:
        for mode, terms in modes.items():
            for _ in range(W):
                plan.merge(terms)
            torch.cuda.synchronize()
            evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(K)]
            for k in range(K):
                evs[k][0].record()
                plan.merge(terms)
                evs[k][1].record()
            torch.cuda.synchronize()
            ms = sum(e[0].elapsed_time(e[1]) for e in evs) / K
            res[mode] = {"ms": round(ms, 4), "gbps": round(nbytes / (ms * 1e6), 1),
                         "frac": round(nbytes / (ms * 1e6) / PEAK_HBM_GBPS, 4)}
            log(f"{mode}: {ms:.3f} ms = {nbytes / (ms * 1e6):.0f} GB/s")
    dom = max(res, key=lambda m: res[m]["ms"])
    traffic = load_traffic("merge", cfg.name, MERGE_SOURCES) if N == 7 else None
    # DARE draws one Philox call per quad of a masked tensor per expert (all tensors here are whole
    # quads, aligned): its VALU work, not HBM, bounds it, so its roofline is the Philox rate
    calls = {mode: sum(t.numel() // 4 * sum(1 for term in row if 0.0 < term["keep"] < 1.0)
                       for t, row in zip(t0s, terms)) for mode, terms in modes.items()}
    hbm_view = {"bound": "hbm", "achieved": res[dom]["gbps"], "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                "frac": res[dom]["frac"], "traffic": traffic["bytes_per_launch"][dom] if traffic else None,
                "algorithmic_bytes_per_launch": nbytes}
    if calls[dom]:
        rate = calls[dom] / (res[dom]["ms"] * 1e-3)
        roofline = {"bound": "alu", "achieved": round(rate, 1), "peak": round(PEAK_PHILOX_CALLS, 1),
                    "unit": "Philox4x32-10 calls/s", "frac": round(rate / PEAK_PHILOX_CALLS, 4),
                    "traffic": None, "kernel": f"merge ({dom})", "calls_per_launch": calls[dom],
                    "avg_launch_ms": res[dom]["ms"], "hbm": hbm_view}
    else:
        roofline = dict(hbm_view, kernel=f"merge ({dom})", avg_launch_ms=res[dom]["ms"])
    if args.calibrate_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
        log("ran the copy calibration kernel (1 GiB read + 1 GiB written) 3 times")
    result = {
        "metric": f"N-expert merge params/s and achieved HBM GB/s, {cfg.name}-shaped",
        "value": P / (res[dom]["ms"] * 1e-3),
        "unit": "params/s",
        "n_gpus": 1, "steps": K, "warmup": W, "ms_per_step": res[dom]["ms"], "higher_is_better": True,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.description}; {N} bf16 experts, bf16 theta0 and output",
                   "params": P, "tensors": cfg.count, "experts": N, "bytes_per_param": 2 * N + 4},
        "modes": res,
        "roofline": roofline,
    }
    print(json.dumps(result))
    return 0


def bench_graph(args, torch, smat, workloads) -> int:
    """Per-step cost of a simulated step on the chosen list when each step samples one scale
    alpha ~ U[alpha_min, 1] shared by every tensor (Sec. 4.1, "Scale"): issued from the host (new
    per-tensor records uploaded, then smat_simulate_multi and smat_backward_multi) against one
    captured HIP graph of smat_step_state_advance and the device-driven calls, whose replays advance
    the step and draw its scale on the device.  Both time K back-to-back steps after W warmup
    steps."""
    import numpy as np
    cfg = workloads.config(args.config)
    inp = workloads.make_inputs(cfg, device="cuda")
    dt = {"bf16": torch.bfloat16, "f32": torch.float32}
    outs = [torch.empty(t.numel(), dtype=dt[cfg.out_dtype], device="cuda") for t in inp.theta]
    K, W = args.steps, args.warmup
    amin = cfg.s_range[0]
    base = workloads.step_params(cfg, inp.settings, 0)
    arr = smat.op_params_array(cfg.count, 1.0, [p["keep"] for p in base], [p["sigma"] for p in base],
                               [p["rescale"] for p in base], [p["noise_kind"] for p in base])
    rng = np.random.default_rng(cfg.index)
    seed, lam = cfg.smat_seed, cfg.lam

    def timed(fn, n):
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t = time.perf_counter()
        a.record()
        for k in range(n):
            fn(k)
        b.record()
        host_us = (time.perf_counter() - t) / n * 1e6
        torch.cuda.synchronize()
        return {"gpu_us": round(a.elapsed_time(b) / n * 1e3, 2), "host_issue_us": round(host_us, 2)}

    res = {}
    with smat.Plan(inp.theta, outs, inp.theta0, inp.grad_sim, inp.grad_theta) as plan:
        def host_step(k):
            arr["s"] = np.float32(rng.uniform(amin, 1.0))
            plan.set_params(arr)
            plan.simulate(seed, k)
            plan.backward(seed, k, lam, True)

        for k in range(W):
            host_step(k)
        res["host_driven"] = timed(host_step, K)

        arr["s"] = 1.0
        plan.set_params(arr)
        state = smat.StepState(seed, 0, 1.0)

        def dev_step():
            state.advance(amin)             # step + 1 and its scale, drawn from (seed, step) on the GPU
            plan.simulate_dev(state)
            plan.backward_dev(state, lam, True)

        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            dev_step()
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            dev_step()
        for _ in range(W):
            graph.replay()
        res["graph_replay"] = timed(lambda k: graph.replay(), K)
        torch.cuda.synchronize()
        del graph
    for mode, r in res.items():
        log(f"{mode}: GPU {r['gpu_us']:.1f} us/step, host issue {r['host_issue_us']:.1f} us/step")
    g = res["graph_replay"]["gpu_us"]
    result = {
        "metric": f"simulated-step time issued from the host vs replayed from a captured HIP graph, {cfg.name}",
        "value": cfg.numel / (g * 1e-6),
        "unit": "params/s",
        "n_gpus": 1, "steps": K, "warmup": W, "ms_per_step": round(g / 1e3, 5), "higher_is_better": True,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.description}; one sampled scale per step shared by all tensors",
                   "params": cfg.numel, "tensors": cfg.count},
        "modes": res,
    }
    print(json.dumps(result))
    return 0


def bench_train(args, torch, smat) -> int:
    """SMAT in a training loop against plain fine-tuning (FT), the measurement behind the method's
    training-time table (App. "Implementation and Measurement Details"): same model, data and AdamW
    (lr 2e-5, weight decay 1e-3, gradient clipping at 1, App. "Training and Scheduling Details"),
    bf16 autocast over fp32 master weights.  Variants, timed in interleaved blocks of whole cycles:
      ft          forward, backward, clip, AdamW (torch, fused)
      smat        SMAT with t = 4: on simulated steps theta~ in the buffers, then the expert gradient
                  lambda alpha m g~ (backward-accumulate), clip and torch AdamW on the expert storage
      smat_fused  as smat, but the simulated step's clip and AdamW update are the library's norm pass
                  and fused optimizer kernel, fed by g~ directly."""
    from paper_2609_33437_amd.training import SimulatedMergeTraining
    from workloads.model import LLAMA_1B, make_decoder, parameter_count, token_batches

    shape = LLAMA_1B
    B, S, t = args.train_batch, args.train_seq, 4
    K = max(t, (args.steps // t) * t)
    W = max(t, -(-args.warmup // t) * t)
    clip = 1.0
    log(f"building the decoder ({parameter_count(shape) / 1e9:.2f}B params), batch {B} x {S} tokens")
    model = make_decoder(shape, 0, "cuda")
    batches = token_batches(shape, B, S, 8, 1, "cuda")
    params = list(model.parameters())
    opt = torch.optim.AdamW(params, lr=2e-5, betas=(0.9, 0.999), eps=1e-8, weight_decay=1e-3, fused=True)
    w = SimulatedMergeTraining.from_module(model, keep=0.5, alpha_min=0.2, sigma=2e-3, period=t, seed=0x7A11,
                                           offload=args.offload)
    extra = sum(b.numel() * b.element_size() for b in w.buffers)   # resident state beyond FT's
    if not args.offload:
        extra += sum(x.numel() * x.element_size() for x in w.theta0)
    hooks = {"begin": [], "end": []}
    counter = [0]

    def step(mode, timed):
        k = counter[0]
        counter[0] += 1
        opt.zero_grad(set_to_none=True)
        sim = False
        if mode != "ft":
            if timed:
                e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
                e[0].record()
            sim = w.begin(k)
            if timed and sim:
                e[1].record()
                hooks["begin"].append(e)
        with torch.autocast("cuda", dtype=torch.bfloat16):
            loss = model.loss(batches[k % len(batches)])
        loss.backward()
        if sim:
            if timed:
                e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
                e[0].record()
            if mode == "smat_fused":
                w.end(opt, fused=True, max_norm=clip)
            else:
                w.end()
                torch.nn.utils.clip_grad_norm_(params, clip)
                opt.step()
            if timed:
                e[1].record()
                hooks["end"].append(e)
            return
        torch.nn.utils.clip_grad_norm_(params, clip)
        opt.step()

    modes = ("ft", "smat", "smat_fused")
    for mode in modes:
        log(f"warmup {W} steps: {mode}")
        for _ in range(W):
            step(mode, False)
    torch.cuda.synchronize()
    times = {m: [] for m in modes}
    for r in range(args.train_reps):
        for mode in modes:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record()
            for _ in range(K):
                step(mode, True)
            b.record()
            torch.cuda.synchronize()
            times[mode].append(a.elapsed_time(b) / K)
            log(f"rep {r} {mode}: {times[mode][-1]:.3f} ms/step")
    med = {m: sorted(v)[len(v) // 2] for m, v in times.items()}
    begin_ms = sum(x[0].elapsed_time(x[1]) for x in hooks["begin"]) / max(1, len(hooks["begin"]))
    w.close()
    tokens = B * S
    result = {
        "metric": "training step time, SMAT (t = 4) vs plain fine-tuning, Llama-1B-shaped synthetic decoder",
        "unit": "ms/step",
        "higher_is_better": False,
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "reps": args.train_reps,
        "dtype": "bf16 autocast, fp32 master weights",
        "data": "synthetic",
        "ms_per_step": {m: round(v, 3) for m, v in med.items()},
        "ms_per_step_all_reps": {m: [round(x, 3) for x in v] for m, v in times.items()},
        "overhead_vs_ft": {m: round(med[m] / med["ft"] - 1.0, 4) for m in modes[1:]},
        "tokens_per_s": {m: round(tokens / (med[m] * 1e-3), 1) for m in modes},
        "begin_ms_per_simulated_step": round(begin_ms, 3),
        "config": {"workload": f"decoder d={shape.d} L={shape.layers} heads={shape.heads} ffn={shape.ffn} "
                               f"vocab={shape.vocab} tied, {parameter_count(shape)} params",
                   "batch": B, "seq_len": S, "optimizer": "torch.optim.AdamW(fused=True) lr 2e-5 wd 1e-3",
                   "clip": clip, "period": t, "keep": 0.5, "alpha_min": 0.2, "sigma": 2e-3, "noise": "uniform",
                   "buffers": "bf16", "theta0": "pinned host (offload)" if args.offload else "resident bf16",
                   "smat_extra_bytes": extra},
        "paper_h800_llama_1b_s_per_step": {"ft": 0.0687, "smat": 0.0700},
    }
    print(json.dumps(result))
    return 0


def main() -> int:
    args = parse_args()
    if args.summarize:
        return summarize(args.summarize)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the transform is elementwise "
              "and shards by elem_offset without communication, so no multi-GPU figure is produced.",
              file=sys.stderr)
        return 2
    import numpy as np
    import torch

    import paper_2609_33437_amd as smat
    import workloads

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    smat.lib()  # fail loudly if the HIP library is missing
    if args.train or args.merge or args.graph:
        args.steps = 20 if args.steps is None else args.steps
        args.warmup = 5 if args.warmup is None else args.warmup
    if args.train:
        return bench_train(args, torch, smat)
    if args.merge:
        return bench_merge(args, torch, smat, workloads)
    if args.graph:
        return bench_graph(args, torch, smat, workloads)
    cfg = workloads.config(args.config)
    args.steps, args.warmup = default_steps(args, cfg)
    dt = {"bf16": torch.bfloat16, "f32": torch.float32}
    nbytes = {"bf16": 2, "f32": 4}
    step_bytes = cfg.numel * (4 + nbytes[cfg.theta0_dtype] + nbytes[cfg.out_dtype] + nbytes[cfg.grad_dtype] + 8)
    copy = timed_copy(step_bytes, torch, smat)   # before the inputs exist, so both fit in HBM
    log(f"plain copy of {copy['bytes'] / 1e9:.1f} GB: {copy['ms']:.3f} ms = {copy['gbps']:.0f} GB/s")
    log(f"generating {cfg.name}: {cfg.count} tensors, {cfg.numel} params")
    t_gen = time.perf_counter()
    inp = workloads.make_inputs(cfg, device="cuda")
    outs = [torch.empty(t.numel(), dtype=dt[cfg.out_dtype], device="cuda") for t in inp.theta]
    torch.cuda.synchronize()
    log(f"generated in {time.perf_counter() - t_gen:.1f} s")

    prefetch = None
    if args.offload:
        if cfg.theta0_dtype != cfg.out_dtype:
            print("offload mode needs theta0 and the buffers in one dtype", file=sys.stderr)
            return 1
        log("copying theta0 into pinned host memory")
        hosts = [t.to("cpu").pin_memory() for t in inp.theta0]
        inp.theta0 = hosts  # the device copies are released; the CPU baseline reads the host copies
        torch.cuda.empty_cache()
        plan = smat.Plan(inp.theta, outs, None, inp.grad_sim, inp.grad_theta, offload=True, theta0_hosts=hosts,
                         dtypes=(smat.SMAT_BF16 if cfg.theta0_dtype == "bf16" else smat.SMAT_F32,) * 2 +
                                (smat.SMAT_BF16 if cfg.grad_dtype == "bf16" else smat.SMAT_F32,))
        # one prefetch on its own: restore (starts the copy) then a simulate that has to wait for it
        plan.set_params(workloads.step_params(cfg, inp.settings, 0))
        plan.simulate(cfg.smat_seed, 0)
        plan.switch_storage(smat.SMAT_SIMULATED)
        torch.cuda.synchronize()
        t_pf = time.perf_counter()
        plan.switch_storage(smat.SMAT_EXPERT)
        plan.close()  # waits for the plan's copy stream
        pf_s = time.perf_counter() - t_pf
        nb = sum(h.numel() * h.element_size() for h in hosts)
        prefetch = {"bytes": nb, "seconds": round(pf_s, 4), "gbps": round(nb / pf_s / 1e9, 2)}
        log(f"theta0 prefetch: {nb / 1e9:.2f} GB in {pf_s * 1e3:.1f} ms = {nb / pf_s / 1e9:.1f} GB/s")
        plan = smat.Plan(inp.theta, outs, None, inp.grad_sim, inp.grad_theta, offload=True, theta0_hosts=hosts,
                         dtypes=(smat.SMAT_BF16 if cfg.theta0_dtype == "bf16" else smat.SMAT_F32,) * 2 +
                                (smat.SMAT_BF16 if cfg.grad_dtype == "bf16" else smat.SMAT_F32,))
    else:
        plan = smat.Plan(inp.theta, outs, inp.theta0, inp.grad_sim, inp.grad_theta)
    K, W = args.steps, args.warmup
    # the hot path runs on simulated steps only: every step, or steps = 3 mod 4 for the periodic list.
    # W warmup steps, K timed steps, K steps of the kernel-timing pass, one verification step.
    step_ids = [k * cfg.period + cfg.period - 1 for k in range(W + 2 * K + 1)]
    params = [workloads.step_params(cfg, inp.settings, s) for s in step_ids]
    # each step's per-tensor records as one array of smat_op_params, built before any timing (the
    # caller's own preparation); the timed step hands it to smat_plan_set_params
    param_arrays = [smat.op_params_array(cfg.count, *[[p[f] for p in ps] for f in ("s", "keep", "sigma", "rescale",
                                                                                  "noise_kind")])
                    for ps in params]
    seed = cfg.smat_seed

    def one(k, ev=None):
        plan.set_params(param_arrays[k])
        if ev:
            ev[0].record()
        plan.simulate(seed, step_ids[k])
        if ev:
            ev[1].record()
        plan.switch_storage(smat.SMAT_SIMULATED)
        if ev:
            ev[2].record()
        plan.backward_accum(seed, step_ids[k], cfg.lam)
        if ev:
            ev[3].record()
        plan.switch_storage(smat.SMAT_EXPERT)

    log(f"warmup {W} steps")
    for k in range(W):
        one(k)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # the timed region: K whole steps with nothing but the steps' own calls between the two events
    log(f"timing {K} steps")
    torch.cuda.synchronize()
    start.record()
    for k in range(K):
        one(W + k)
    end.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    ms_step = total_ms / K
    # kernel pass: K more steps with HIP events around each kernel on the launch stream (the events
    # cost host issue time, which shows on small lists, so they stay out of the timed region)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    start.record()
    for k in range(K):
        one(W + K + k, evs[k])
    end.record()
    torch.cuda.synchronize()
    ms_step_events = start.elapsed_time(end) / K
    sim_ms = [e[0].elapsed_time(e[1]) for e in evs]
    bwd_ms = [e[2].elapsed_time(e[3]) for e in evs]
    sim_avg, bwd_avg = sum(sim_ms) / K, sum(bwd_ms) / K
    med = lambda v: sorted(v)[len(v) // 2]
    log(f"step {ms_step:.3f} ms (kernel pass {ms_step_events:.3f} ms)  simulate {sim_avg:.3f} ms  "
        f"backward {bwd_avg:.3f} ms")

    # verification step (untimed, the launch configuration timed above): windows of grad_theta before
    # it, then the windows of its outputs, for the oracle to check in the CPU baseline leg
    verify = None
    if not args.no_cpu_baseline:
        kv = W + 2 * K
        frac, wins = sample_windows(cfg, args.cpu_sample)
        g_pre = [inp.grad_theta[i].view(-1)[a:a + m].cpu().numpy() for i, a, m in wins]
        one(kv)
        torch.cuda.synchronize()
        tasks = window_tasks(wins, inp, g_pre, torch, np)
        piece = 1 << 20
        gpu_tt, gpu_g = [], []
        for i, a, m in wins:
            o = outs[i].view(-1)[a:a + m].cpu()
            o = o.view(torch.int16).numpy().view(np.uint16) if o.dtype == torch.bfloat16 else o.numpy()
            g = inp.grad_theta[i].view(-1)[a:a + m].cpu().numpy()
            for b in range(0, m, piece):
                gpu_tt.append(o[b:b + piece])
                gpu_g.append(g[b:b + piece])
        verify = (kv, tasks, gpu_tt, gpu_g)
        del g_pre

    P = cfg.numel
    sim_bytes = P * (4 + nbytes[cfg.theta0_dtype] + nbytes[cfg.out_dtype])
    bwd_bytes = P * (nbytes[cfg.grad_dtype] + 4 + 4)
    step_gbps = (sim_bytes + bwd_bytes) / (ms_step * 1e6)
    sim_gbps = sim_bytes / (sim_avg * 1e6)
    bwd_gbps = bwd_bytes / (bwd_avg * 1e6)

    if args.calibrate_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
        log("ran the copy calibration kernel (1 GiB read + 1 GiB written) 3 times")

    dominant = "simulate" if sim_avg >= bwd_avg else "backward"
    dom_gbps, dom_bytes = (sim_gbps, sim_bytes) if dominant == "simulate" else (bwd_gbps, bwd_bytes)
    traffic = load_traffic(dominant, cfg.name)
    roofline = {"bound": "hbm", "achieved": round(dom_gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                "frac": round(dom_gbps / PEAK_HBM_GBPS, 4),
                "traffic": traffic["bytes_per_launch"] if traffic else None,
                "kernel": dominant, "algorithmic_bytes_per_launch": dom_bytes,
                "avg_launch_ms": round(sim_avg if dominant == "simulate" else bwd_avg, 4)}

    result = {
        "metric": METRIC,
        "value": P / (ms_step * 1e-3),
        "unit": "params/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.description}", "params": P, "tensors": cfg.count,
                   "theta": "f32", "theta0": cfg.theta0_dtype, "theta_tilde": cfg.out_dtype,
                   "grad_sim": cfg.grad_dtype, "grad_theta": "f32",
                   "bytes_per_param_per_step": (sim_bytes + bwd_bytes) / P, "period": cfg.period},
        "hbm_gbps": round(step_gbps, 1),
        "hbm_frac_of_peak": round(step_gbps / PEAK_HBM_GBPS, 4),
        "kernels": {"simulate": {"avg_ms": round(sim_avg, 4), "median_ms": round(med(sim_ms), 4),
                                 "min_ms": round(min(sim_ms), 4), "gbps": round(sim_gbps, 1),
                                 "frac_of_copy": round(sim_gbps / copy["gbps"], 4)},
                    "backward": {"avg_ms": round(bwd_avg, 4), "median_ms": round(med(bwd_ms), 4),
                                 "min_ms": round(min(bwd_ms), 4), "gbps": round(bwd_gbps, 1),
                                 "frac_of_copy": round(bwd_gbps / copy["gbps"], 4)},
                    "timing": f"HIP events around each kernel in a second pass of {K} steps "
                              f"({round(ms_step_events, 4)} ms per step with the events)"},
        "copy": dict(copy, kernel="smat_stream_copy (plain nontemporal copy), same bytes as one step",
                     frac_of_peak=round(copy["gbps"] / PEAK_HBM_GBPS, 4)),
        "hbm_frac_of_copy": round(step_gbps / copy["gbps"], 4),
        "roofline": roofline,
        "cpu_baseline": None,
        "parity": None,
    }
    if cfg.period > 1:
        result["config"]["ms_per_training_step_avg"] = round(ms_step / cfg.period, 4)
    if prefetch is not None:
        result["config"]["mode"] = "offload: theta0 in pinned host memory, copied into the buffers at each restore"
        result["offload_prefetch"] = prefetch
    if args.adamw:
        plan.close()
        result["adamw_step"] = bench_adamw(cfg, inp, outs, params, step_ids, seed, K, W, torch, smat)
    if verify is not None:
        kv, tasks, gpu_tt, gpu_g = verify
        result["cpu_baseline"], oracle_outs = cpu_baseline(cfg, tasks, params[kv], step_ids[kv], args.cpu_seconds)
        result["parity"] = dict(parity_stats(cfg, tasks, oracle_outs, gpu_tt, gpu_g, params[kv], np),
                                step=step_ids[kv])
        log(f"parity: {result['parity']['elements']} elements, theta~ mismatches "
            f"{result['parity']['theta_tilde']['mismatches']} (max {result['parity']['theta_tilde']['max_ulp']} ulp), "
            f"grad mismatches {result['parity']['grad_theta']['mismatches']}")
    plan.close()
    print(json.dumps(result))
    return 0


if __name__ == "__main__":
    sys.exit(main())
