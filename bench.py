"""Benchmark: batched DistIR strategy simulation on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

NAME is random_tables (default) or one of the strategy grids (tiny_mlp,
large_mlp, gpt2_small, gpt2_small_train, gpt3_175b, gpt3_175b_gpipe,
gpt3_175b_recompute, gpt3_175b_zero, gpt3_175b_mi355x); a grid's line times
dsim_simulate_parametric + top-k over the whole grid.

A step is one pass of the hot path over one batch of synthetic input, with the
input already resident in HBM:
  * random_tables (default, the HBM-bound workload): simulate 1,000,000
    random programs of 2,048 ops over 8 devices from their explicit op tables
    (dsim_simulate_tables), then select the best feasible one (dsim_argmin).
    The tables (about 41 GB) are generated on the GPU before timing.
  * "parametric" (extra key of the same line): each strategy grid (tiny MLP,
    large MLP, GPT-2-small inference and training, GPT-3-175B) simulated by
    dsim_simulate_parametric + top-k, timed with HIP events;
  * "grids_as_tables": the tiny MLP grid written as explicit op tables
    (dsim_materialize_tables) and simulated by dsim_simulate_tables + top-k.
Prints one JSON line (rank 0).  The CPU oracle is timed on a bounded sample
of the same workload as `cpu_baseline`.
"""
import argparse
import hashlib
import re
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "simulated candidates/sec + simulated ops/sec; achieved HBM GB/s vs peak"
HBM_PEAK_GBPS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")


def kernel_hash(path):
    """A hash of a kernel source's code: comments and blank lines removed and
    runs of white space collapsed, so that a change of wording in a comment
    keeps counters taken on the same code."""
    with open(path) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    lines = (" ".join(line.split()) for line in text.splitlines())
    return hashlib.sha256("\n".join(line for line in lines if line).encode()).hexdigest()[:16]


def stored_traffic(kernel, workload, src):
    """HBM traffic per launch measured by rocprofv3 --pmc (profiles/), if the
    kernel source is unchanged since the counters were taken."""
    p = os.path.join(PROFILES, "traffic.json")
    if not os.path.exists(p):
        return None
    with open(p) as f:
        rec = json.load(f).get("%s/%s" % (kernel, workload))
    if not rec or rec.get("source_sha256_16") != kernel_hash(src):
        return None
    return rec.get("bytes_per_launch")


def cpu_baseline_random(spec, dev, budget_s=12.0, threads=None):
    """The oracle, as it stands, on strided candidates of the same workload
    until ~budget_s seconds of wall time are spent (all host threads, up to
    16, unless `threads` is given)."""
    import numpy as np
    import oracle
    threads = threads or max(1, min(os.cpu_count() or 1, 16))
    chunk = max(64, 2048 * threads // 8)
    done, t0 = 0, time.perf_counter()
    stride = 997
    # 997 is prime and does not divide n_cand, so the sample holds distinct candidates
    while time.perf_counter() - t0 < budget_s and done < spec.n_cand:
        n = min(chunk, spec.n_cand - done)
        cands = (np.arange(done, done + n, dtype=np.int64) * stride) % spec.n_cand
        oracle.run_random_tables(spec.seed, spec.n_ops, spec.n_dev, cands, dev, threads=threads, want_rows=False)
        done += n
    dt = time.perf_counter() - t0
    return {"value": done / dt, "unit": "candidates/s", "cores": threads, "kind": "oracle",
            "sample": "%d distinct candidates (index i*997 mod %d) of the %d x %d ops x %d devices workload, "
                      "generated and simulated by the C oracle in %.1f s on %d threads"
                      % (done, spec.n_cand, spec.n_cand, spec.n_ops, spec.n_dev, dt, threads),
            "ops_per_s": done * spec.n_ops / dt}


def bench_random_tables(args, torch, dsim, W):
    spec = W.tables
    dev = W.device
    N, J, ND = spec.n_cand, spec.n_ops, spec.n_dev
    tab = dsim.alloc_tables(N, J)
    dsim.dsim_generate_random_tables(spec.seed, N, J, ND, tab)
    res = dsim.alloc_results(N, ND)
    res["walked_ops"] = None   # equal to n_ops for tables
    k = W.top_k
    ws = torch.empty(max(dsim.dsim_argmin_workspace(N, k), 16), dtype=torch.uint8, device="cuda")
    out_idx = torch.empty(k, dtype=torch.int64, device="cuda")
    out_mk = torch.empty(k, dtype=torch.float64, device="cuda")
    found = torch.empty(1, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()

    ev = []

    def step(record):
        if record:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
        dsim.dsim_simulate_tables(tab, N, ND, dev, res)
        if record:
            e1.record()
            ev.append((e0, e1))
        dsim.dsim_argmin(res["makespan"], res["cand_peak"], res["status"], dev.mem_cap_bytes, k, ws, out_idx,
                         out_mk, found)

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(True)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    kern_ms = sum(a.elapsed_time(b) for a, b in ev) / len(ev)
    # algorithmic bytes per launch: 20 B per op record + 4 B op count per
    # candidate read; makespan 8 + finish 8*nd + peak 8*nd + cand_peak 8 +
    # n_ops 8 + status 4 written per candidate
    per_cand = J * 20 + 4 + 8 + 16 * ND + 8 + 8 + 4
    algo_bytes = per_cand * N
    achieved = algo_bytes / (kern_ms * 1e-3) / 1e9
    src = os.path.join(ROOT, "paper_2111_05426_amd", "csrc", "sim_tables.hip")
    out = {
        "metric": METRIC,
        "value": N * args.steps / dt,
        "unit": "candidates/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": dt / args.steps * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64", "data": "synthetic",
        "config": {"workload": "random_tables: %d programs x %d ops x %d devices (seed %d), simulate + top-%d"
                               % (N, J, ND, spec.seed, k),
                   "n_cand": N, "n_ops": J, "n_dev": ND, "seed": spec.seed, "top_k": k},
        "ops_per_s": N * J * args.steps / dt,
        "kernel_ms": kern_ms,
        "hbm_GBps": achieved,
        "best": {"index": int(out_idx[0].item()), "makespan_s": float(out_mk[0].item())},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": stored_traffic("k_sim_tables", "random_tables", src),
                     "kernel": "k_sim_tables<8>", "algorithmic_bytes_per_launch": algo_bytes},
    }
    return out


PARAMETRIC = ("tiny_mlp", "large_mlp", "gpt2_small", "gpt2_small_train", "gpt3_175b", "gpt3_175b_gpipe",
              "gpt3_175b_recompute", "gpt3_175b_zero", "gpt3_175b_overlap", "gpt3_175b_mi355x",
              "gpt3_175b_mi355x_overlap")


_SIDE = []


def side_stream(torch):
    """The second stream of the split transform launch, created once (default
    priority) so that every grid runs on the same pair of streams."""
    if not _SIDE:
        _SIDE.append(torch.cuda.Stream())
    return _SIDE[0]


# Vector issue rate of the chip: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz lane
# instructions per second (a wave64 vector instruction occupies a 16-lane
# SIMD for 4 cycles).  The transform's kernels are bound by dependent fp64
# adds, Send-chain steps and wave-wide votes, i.e. by vector issue and its
# latency, so their roofline is this rate and their achieved figure is the
# vector instructions they execute (rocprofv3 SQ_INSTS_VALU, 64 lanes each)
# per second of the live launch time.
VALU_PEAK_T = 256 * 4 * 16 * 2.4e9 / 1e12
PARAMETRIC_SRC = [os.path.join(ROOT, "paper_2111_05426_amd", "csrc", f) for f in ("parametric.hip", "model.h")]


def stored_valu(workload):
    """Vector instructions per dsim_simulate_parametric call of a grid,
    counted by rocprofv3 --pmc (profiles/), if the transform's sources are
    unchanged since the counters were taken."""
    p = os.path.join(PROFILES, "valu.json")
    if not os.path.exists(p):
        return None
    with open(p) as f:
        rec = json.load(f).get("k_parametric/%s" % workload)
    if not rec or rec.get("source_sha256_16") != [kernel_hash(f) for f in PARAMETRIC_SRC]:
        return None
    return rec


def bench_parametric(torch, dsim, W, reps, warmup=1, cpu_budget_s=0.0):
    """One grid of the transform-driven path: dsim_simulate_parametric over
    every strategy of the grid plus the top-k selection, with the strategies
    resident on the device.  Projected ops count the ops of the per-stage
    projection the kernel's result stands for (one replica per stage; the
    kernel adds repeated layers in closed form, so these are not arithmetic
    steps); program ops count every op of the global program."""
    strat = dsim.dsim_create_grid(W.model, W.grid)
    n = len(strat)
    rw = int(strat[:, 2].max())
    cand = torch.from_numpy(strat).cuda()
    res = dsim.alloc_results(n, rw)
    k = W.top_k
    ws = torch.empty(max(dsim.dsim_argmin_workspace(n, k), 16), dtype=torch.uint8, device="cuda")
    out_idx = torch.empty(k, dtype=torch.int64, device="cuda")
    out_mk = torch.empty(k, dtype=torch.float64, device="cuda")
    found = torch.empty(1, dtype=torch.int32, device="cuda")
    pws = dsim.alloc_parametric_workspace(n)
    side = side_stream(torch)   # the split launch of large transformer grids runs on two streams
    dev = W.device
    ev = []

    def step(record):
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record()
        dsim.dsim_simulate_parametric(W.model, cand, dev, res, workspace=pws, side_stream=side)
        e1.record()
        dsim.dsim_argmin(res["makespan"], res["cand_peak"], res["status"], dev.mem_cap_bytes, k, ws, out_idx,
                         out_mk, found)
        e2.record()
        if record:
            ev.append((e0, e1, e2))

    for _ in range(max(1, warmup)):
        step(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        step(True)
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - t0
    # per-call times from HIP events on the launch stream; the median over the
    # calls is reported (a call's events also count any gap in which the GPU
    # waits for the host to enqueue it, which now and then adds tens of ms)
    kern_reps = sorted(a.elapsed_time(b) for a, b, _ in ev)
    step_reps = sorted(a.elapsed_time(c) for a, _, c in ev)
    kern_ms = kern_reps[len(kern_reps) // 2]
    step_ms = step_reps[len(step_reps) // 2]
    projected = int(res["walked_ops"].sum().item())
    prog = int(res["n_ops"].sum().item())
    ok = int((res["status"] == 0).sum().item())
    out = {"workload": W.name, "n_cand": n, "valid": ok, "top_k": k, "found": int(found.item()),
           "best": {"index": int(out_idx[0].item()), "strategy_DHPK": strat[int(out_idx[0].item())].tolist(),
                    "makespan_s": float(out_mk[0].item())} if int(found.item()) > 0 else None,
           "kernel_ms": kern_ms, "step_ms": step_ms, "candidates_per_s": n / (step_ms * 1e-3),
           "projected_ops": projected, "projected_ops_per_s": projected / (kern_ms * 1e-3),
           "program_ops": prog, "program_ops_per_s": prog / (kern_ms * 1e-3), "wall_s": wall_s, "reps": reps,
           "kernel_ms_reps": kern_reps, "kernel_ms_mean": sum(kern_reps) / len(kern_reps)}
    rec = stored_valu(W.name)
    achieved = rec["valu_insts_per_call"] * 64 / (kern_ms * 1e-3) / 1e12 if rec else None
    out["roofline"] = {"bound": "alu", "achieved": achieved, "peak": VALU_PEAK_T,
                       "unit": "T vector lane-instructions/s", "frac": achieved / VALU_PEAK_T if rec else None,
                       "traffic": None, "kernel": "k_parametric + k_parametric_wide",
                       "valu_insts_per_call": rec["valu_insts_per_call"] if rec else None,
                       "counters": rec["summary"] if rec else "not current for this source"}
    if cpu_budget_s > 0:
        out["cpu_baseline"] = cpu_baseline_parametric(W, strat, budget_s=cpu_budget_s)
    return out


def bench_grid_as_tables(torch, dsim, W, reps, n_dev=8):
    """A strategy grid as explicit op tables: dsim_materialize_tables writes
    every op of every device (untimed, once), then a step is
    dsim_simulate_tables + top-k over those tables."""
    strat = dsim.dsim_create_grid(W.model, W.grid)
    n = len(strat)
    cand = torch.from_numpy(strat).cuda()
    t, mst = dsim.dsim_materialize_tables(W.model, cand, n_dev, 4096)
    torch.cuda.synchronize()
    max_ops = int(t["n_ops"].max().item())
    res = dsim.alloc_results(n, n_dev)
    k = W.top_k
    ws = torch.empty(max(dsim.dsim_argmin_workspace(n, k), 16), dtype=torch.uint8, device="cuda")
    out_idx = torch.empty(k, dtype=torch.int64, device="cuda")
    out_mk = torch.empty(k, dtype=torch.float64, device="cuda")
    found = torch.empty(1, dtype=torch.int32, device="cuda")
    ev = []
    for i in range(reps + 1):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dsim.dsim_simulate_tables(t, n, n_dev, W.device, res, init_live=t["init_live"])
        dsim.dsim_argmin(res["makespan"], res["cand_peak"], res["status"], W.device.mem_cap_bytes, k, ws, out_idx,
                         out_mk, found)
        e1.record()
        if i:
            ev.append((e0, e1))
    torch.cuda.synchronize()
    step_ms = sum(a.elapsed_time(b) for a, b in ev) / len(ev)
    ops = int(t["n_ops"].sum().item())
    best = int(out_idx[0].item())
    return {"workload": W.name + " as explicit tables", "n_cand": n, "ops_per_table_max": max_ops,
            "program_ops": ops, "materialize_status_nonzero": int((mst != 0).sum().item()),
            "step_ms": step_ms, "candidates_per_s": n / (step_ms * 1e-3),
            "best": {"index": best, "strategy_DHPK": strat[best].tolist(), "makespan_s": float(out_mk[0].item())}}


def bench_lowered_programs(torch, dsim, reps):
    """Programs through the front end: GPT-2-shaped layers (4 layers, d 768,
    12 heads) placed over 1-8 devices by hand (tensor x pipeline parallelism
    1x1, 2x2, 4x2, 2x4, 1x4), batch 1-16 and sequence 64-1024.  The program
    texts are written first (untimed); then dsim_lower_programs interprets
    them over the mixed abstract/concrete domain and lowers them to one set
    of candidate tables on the host (timed on one thread and on up to 16,
    best of 3 each), and a step is dsim_simulate_tables over all of them on
    the GPU."""
    import numpy as np
    from paper_2111_05426_amd import frontend as fe, programs
    from paper_2111_05426_amd.workloads import DeviceSpec
    cases = [(B, S, tp, pp) for tp, pp in ((1, 1), (2, 2), (4, 2), (2, 4), (1, 4))
             for B in range(1, 17) for S in (64, 128, 256, 512, 1024)]
    texts = [programs.gpt2_layers(B, S, n_layers=4, tp=tp, pp=pp) for B, S, tp, pp in cases]
    inputs = [{"%flat": [-1]}] * len(texts)
    threads = max(1, min(os.cpu_count() or 1, 16))
    host = {}
    for th in (1, threads):
        best = None
        for _ in range(3):
            t0 = time.perf_counter()
            p = fe.lower_batch(texts, inputs, n_dev=8, threads=th)
            dt = time.perf_counter() - t0
            best = dt if best is None else min(best, dt)
        host[th] = best
    n = len(cases)
    g = {k: torch.from_numpy(np.ascontiguousarray(p[k]).view(np.int32 if p[k].dtype == np.uint32 else p[k].dtype)).cuda()
         for k in ("code", "flops", "bytes", "alloc", "free", "mm_k", "n_ops")}
    init = torch.from_numpy(p["init_live"].view(np.int64)).cuda()
    res = dsim.alloc_results(n, 8)
    dev = DeviceSpec()
    ev = []
    for i in range(reps + 1):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dsim.dsim_simulate_tables(g, n, 8, dev, res, init_live=init)
        e1.record()
        if i:
            ev.append((e0, e1))
    torch.cuda.synchronize()
    ms = sum(a.elapsed_time(b) for a, b in ev) / len(ev)
    return {"workload": "gpt2-shaped layer programs through the front end", "programs": n,
            "records_per_table_max": int(p["code"].shape[0]), "records": int(p["n_ops"].sum()),
            "host_interpret_and_lower_ms": host[1] * 1e3, "host_ms_per_program": host[1] * 1e3 / n,
            "host_threads": threads, "host_ms_threaded": host[threads] * 1e3,
            "kernel_ms": ms, "programs_per_s": n / (ms * 1e-3)}


def cpu_baseline_parametric(W, strat, budget_s=10.0, threads=None):
    """The oracle (projection mode), as it stands, on strided candidates of
    the grid until ~budget_s seconds of wall time are spent (all host
    threads, up to 16, unless `threads` is given)."""
    import numpy as np
    import oracle
    threads = threads or max(1, min(os.cpu_count() or 1, 16))
    order = np.arange(len(strat))[::7] if len(strat) > 7 * 4 * threads else np.arange(len(strat))
    done, t0 = 0, time.perf_counter()
    while time.perf_counter() - t0 < budget_s and done < len(order):
        pick = order[done:done + 4 * threads]
        oracle.run_strategies(W.model, strat[pick], W.device, slice=True, row_width=int(strat[:, 2].max()),
                              threads=threads)
        done += len(pick)
    dt = time.perf_counter() - t0
    return {"value": done / dt, "unit": "candidates/s", "cores": threads, "kind": "oracle",
            "sample": "%d of the %d strategies (grid order%s), simulated by the C oracle (one replica "
                      "per stage) in %.1f s on %d threads" % (done, len(strat), ", every 7th" if len(order) < len(strat)
                                                              else "", dt, threads)}


def bench_parametric_line(args, torch, dsim, W):
    """The benchmark line for a strategy grid: a step is one
    dsim_simulate_parametric over the whole grid plus the top-k selection."""
    r = bench_parametric(torch, dsim, W, args.steps, args.warmup)
    out = {
        "metric": METRIC, "value": r["n_cand"] * r["reps"] / r["wall_s"], "unit": "candidates/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": r["wall_s"] / r["reps"] * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": "%s: %d strategies, simulate + top-%d" % (W.name, r["n_cand"], W.top_k),
                   "n_cand": r["n_cand"], "top_k": W.top_k},
        "ops_per_s": r["projected_ops_per_s"], "program_ops_per_s": r["program_ops_per_s"],
        "kernel_ms": r["kernel_ms"], "best": r["best"], "roofline": r["roofline"],
    }
    if not args.no_cpu_baseline:
        strat = dsim.dsim_create_grid(W.model, W.grid)
        out["cpu_baseline"] = cpu_baseline_parametric(W, strat)
        out["cpu_baseline"]["single_thread"] = cpu_baseline_parametric(W, strat, budget_s=4.0, threads=1)
    return out


def copy_calibration(torch, nbytes=4 << 30, reps=5):
    """A plain device-to-device copy of known size: its time gives the
    achievable streaming bandwidth; under rocprofv3 --pmc its FETCH_SIZE and
    WRITE_SIZE calibrate the counters (it reads and writes nbytes)."""
    a = torch.empty(nbytes // 4, dtype=torch.int32, device="cuda").fill_(1)
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    return {"bytes_read": nbytes, "bytes_written": nbytes, "ms": ms, "GBps": 2 * nbytes / (ms * 1e-3) / 1e9}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="random_tables")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-parametric", action="store_true",
                    help="skip the per-grid timings of the transform-driven kernel")
    ap.add_argument("--param-reps", type=int, default=7)
    ap.add_argument("--no-copy", action="store_true",
                    help="skip the plain 4 GiB device-to-device copy timed beside the kernel")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="time the 4 GiB copy (the default; kept for the profiling commands)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the simulator would shard candidates across GPUs, but runs on "
              "several GPUs are not supported (use --gpus 1)", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2111_05426_amd import dsim
    from paper_2111_05426_amd.workloads import ALL
    if not torch.cuda.is_available():
        print("bench.py needs a HIP device", file=sys.stderr)
        sys.exit(1)
    dsim.lib()
    if args.workload not in ALL:
        raise SystemExit("unknown workload %s (one of %s)" % (args.workload, ", ".join(ALL)))
    W = ALL[args.workload]
    if W.tables is None:
        print(json.dumps(bench_parametric_line(args, torch, dsim, W)), flush=True)
        return
    out = bench_random_tables(args, torch, dsim, W)
    if not args.no_parametric:
        # the large MLP, GPT-2-small and GPT-3-175B-shaped grids also time the
        # oracle on a bounded sample
        graded = ("large_mlp", "gpt2_small", "gpt3_175b")
        out["parametric"] = [bench_parametric(torch, dsim, ALL[name], args.param_reps,
                                              cpu_budget_s=0.0 if args.no_cpu_baseline or name not in graded else 3.0)
                             for name in PARAMETRIC]
        out["grids_as_tables"] = [bench_grid_as_tables(torch, dsim, ALL["tiny_mlp"], args.param_reps)]
        out["lowered_programs"] = bench_lowered_programs(torch, dsim, args.param_reps)
    if args.copy_calibration or not args.no_copy:
        # the achievable streaming rate on this GPU, beside the spec peak
        out["copy_calibration"] = copy_calibration(torch)
        out["roofline"]["copy_GBps"] = out["copy_calibration"]["GBps"]
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_random(W.tables, W.device)
        out["cpu_baseline"]["single_thread"] = cpu_baseline_random(W.tables, W.device, budget_s=4.0, threads=1)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
