"""GPU parity of the parametric D/H/P/K expander against the oracle.

Small models: the oracle materialises the whole distributed program (every
device of every replica).  Full-size grids: the oracle's projection onto one
replica per stage (itself pinned to the full program in
test_oracle_pins.py), on every candidate where that is cheap and on a seeded
sample of the GPT-3-shaped grid.  Bar: status, op counts and peak bytes
bit-exact; times within 1e-12 relative and expected bit-identical.
"""
import math
import os
from dataclasses import replace

import numpy as np
import pytest

from paper_2111_05426_amd.workloads import (ALL, DeviceSpec, GPT2_SMALL, GPT2_SMALL_TRAIN, GPT3_175B, INFER, SCHED_GPIPE,
                                            LARGE_MLP, TINY_MLP, TRAIN_ADAM, TRAIN_ADAM_MIXED, TRAIN_SGD, mlp,
                                            transformer)

pytestmark = pytest.mark.gpu
REL = 1e-12


@pytest.fixture(scope="module")
def torch_gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    from paper_2111_05426_amd import dsim
    dsim.lib()
    return torch


_SIDE = []


def side_stream(torch):
    """One second stream (default priority) for the split launch."""
    if not _SIDE:
        _SIDE.append(torch.cuda.Stream())
    return _SIDE[0]


def run_gpu(torch, model, strat, dev, row_width=None, side=True):
    from paper_2111_05426_amd import dsim
    strat = np.ascontiguousarray(strat, np.int32).reshape(-1, 4)
    rw = int(row_width or max(1, strat[:, 2].max()))
    r = dsim.alloc_results(len(strat), rw)
    cand = torch.from_numpy(strat).cuda()
    ws = dsim.alloc_parametric_workspace(len(strat))
    dsim.dsim_simulate_parametric(model, cand, dev, r, workspace=ws, side_stream=side_stream(torch) if side else None)
    torch.cuda.synchronize()
    out = {k: v.cpu().numpy() for k, v in r.items() if k != "row_width"}
    out["cand"] = cand
    out["gpu"] = r
    return out


def compare(g, o, strat):
    bad = []
    for name in ("status", "n_ops", "cand_peak"):
        a = g[name].astype(np.int64) if name != "cand_peak" else g[name].view(np.uint64)
        b = o[name].astype(np.int64) if name != "cand_peak" else o[name]
        if not np.array_equal(a, b):
            i = int(np.nonzero(a != b)[0][0])
            bad.append("%s differs first at %s: gpu %s oracle %s" % (name, strat[i].tolist(), a[i], b[i]))
    np.testing.assert_allclose(g["makespan"], o["makespan"], rtol=REL, atol=0)
    rw = o["finish"].shape[1]
    np.testing.assert_allclose(g["finish"][:, :rw], o["finish"], rtol=REL, atol=0)
    if not np.array_equal(g["peak"][:, :rw].view(np.uint64), o["peak"]):
        i = int(np.nonzero(np.any(g["peak"][:, :rw].view(np.uint64) != o["peak"], axis=1))[0][0])
        bad.append("stage peak differs at %s: gpu %s oracle %s" % (strat[i].tolist(), g["peak"][i, :rw],
                                                                  o["peak"][i]))
    assert not bad, "\n".join(bad)
    assert np.array_equal(g["makespan"], o["makespan"]), "within 1e-12 but not bit-identical"
    assert np.array_equal(g["finish"][:, :rw], o["finish"])
    ok = g["status"] == 0
    assert np.all(g["walked_ops"][ok] > 0) and np.all(g["walked_ops"] <= g["n_ops"])


def all_strats(D, H, P, K):
    return np.array([(d, h, p, k) for d in D for h in H for p in P for k in K], np.int32)


SMALL = [
    ("mlp_sgd", mlp(4, 64, 48, 4, TRAIN_SGD), all_strats([1, 2, 3], [1, 2], [1, 2, 4], [1, 2, 3, 5])),
    ("mlp_adam_uneven", mlp(6, 64, 40, 2, TRAIN_ADAM), all_strats([1, 2, 4], [1, 2], [1, 2, 3, 4, 5], [1, 3, 7])),
    ("mlp_mixed", mlp(8, 32, 36, 2, TRAIN_ADAM_MIXED), all_strats([1, 2], [1, 2, 4], [1, 2, 4, 8], [1, 2, 6])),
    ("mlp_infer", mlp(5, 64, 30, 4, INFER), all_strats([1, 2, 3], [1, 2], [1, 2, 3, 5], [1, 2, 4])),
    ("tf_train", transformer(4, 32, 4, 8, 101, 12, 2, TRAIN_ADAM), all_strats([1, 2, 3], [1, 2, 4], [1, 2, 3, 4],
                                                                             [1, 2, 5])),
    ("tf_mixed", transformer(5, 32, 4, 8, 64, 8, 2, TRAIN_ADAM_MIXED), all_strats([1, 2], [1, 2], [1, 2, 5], [1, 4])),
    ("tf_infer", transformer(6, 48, 6, 16, 97, 9, 2, INFER), all_strats([1, 3], [1, 2, 3], [1, 2, 4], [1, 2, 3])),
    ("tf_sgd", transformer(3, 32, 2, 8, 50, 6, 4, TRAIN_SGD), all_strats([1, 2], [1, 2], [1, 3], [1, 2, 3])),
    ("mlp_adam_gpipe", mlp(6, 64, 40, 2, TRAIN_ADAM, schedule=SCHED_GPIPE),
     all_strats([1, 2, 4], [1, 2], [1, 2, 3, 4, 5], [1, 3, 7])),
    ("tf_train_gpipe", transformer(4, 32, 4, 8, 101, 12, 2, TRAIN_ADAM, schedule=SCHED_GPIPE),
     all_strats([1, 2, 3], [1, 2, 4], [1, 2, 3, 4], [1, 2, 5])),
    ("mlp_adam_rc", mlp(7, 64, 40, 2, TRAIN_ADAM, recompute=1), all_strats([1, 2, 4], [1], [1, 2, 3, 4, 7], [1, 3, 7])),
    ("mlp_mixed_rc", mlp(8, 32, 36, 2, TRAIN_ADAM_MIXED, recompute=1), all_strats([1, 2], [1, 2, 4], [1, 2, 4, 8],
                                                                                    [1, 2, 6])),
    ("mlp_sgd_gpipe_rc", mlp(12, 64, 48, 4, TRAIN_SGD, schedule=SCHED_GPIPE, recompute=1),
     all_strats([1, 3], [1, 2], [1, 2, 3, 5], [1, 2, 5])),
    ("tf_train_rc", transformer(5, 32, 4, 8, 101, 12, 2, TRAIN_ADAM, recompute=1), all_strats([1, 2, 3], [1, 2, 4],
                                                                                            [1, 2, 3, 5], [1, 2, 5])),
    ("tf_mixed_gpipe_rc", transformer(6, 32, 4, 8, 64, 8, 2, TRAIN_ADAM_MIXED, schedule=SCHED_GPIPE, recompute=1),
     all_strats([1, 2], [1, 2], [1, 2, 4, 5], [1, 4])),
    ("tf_infer_rc", transformer(6, 48, 6, 16, 97, 9, 2, INFER, recompute=1), all_strats([1, 3], [1, 2], [1, 4], [1, 3])),
    # ZeRO: replicas own different groups; D up to twice the groups of a stage
    ("mlp_adam_zero", mlp(6, 64, 48, 2, TRAIN_ADAM, zero=1), all_strats([1, 2, 3, 4, 8, 16], [1, 2], [1, 2, 3],
                                                                        [1, 3])),
    ("mlp_sgd_zero_rc", mlp(8, 32, 48, 4, TRAIN_SGD, recompute=1, zero=1), all_strats([2, 3, 4, 6], [1, 2], [1, 2, 4],
                                                                                     [1, 2, 5])),
    ("mlp_mixed_zero_gpipe", mlp(8, 32, 48, 2, TRAIN_ADAM_MIXED, schedule=SCHED_GPIPE, zero=1),
     all_strats([2, 4, 12], [1, 2], [1, 2, 4], [1, 4])),
    ("tf_train_zero", transformer(4, 32, 4, 8, 101, 24, 2, TRAIN_ADAM, zero=1), all_strats([1, 2, 3, 4, 8], [1, 2],
                                                                                        [1, 2, 4], [1, 2, 3])),
    ("tf_mixed_zero_rc", transformer(5, 32, 4, 8, 64, 12, 2, TRAIN_ADAM_MIXED, recompute=1, zero=1),
     all_strats([2, 3, 6], [1, 2], [1, 2, 5], [1, 2])),
    ("tf_sgd_zero_gpipe", transformer(6, 32, 2, 8, 50, 16, 4, TRAIN_SGD, schedule=SCHED_GPIPE, zero=1),
     all_strats([2, 4, 8, 16], [1, 2], [1, 3, 6], [1, 2])),
    ("tf_infer_zero", transformer(6, 48, 6, 16, 97, 9, 2, INFER, zero=1), all_strats([1, 3], [1, 2], [1, 4], [1, 3])),
]


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_small_models_vs_full_program(torch_gpu, orc, case):
    name, model, strat = SMALL[case]
    dev = DeviceSpec(mem_cap_bytes=10 ** 6)
    g = run_gpu(torch_gpu, model, strat, dev)
    o = orc.run_strategies(model, strat, dev, slice=False, row_width=g["finish"].shape[1], threads=8)
    assert np.any(o["status"] == 0)
    compare(g, o, strat)


# empirical MatMul costs: random regression coefficients (and ones that make
# matrix multiplications cheap or dominant) on models of every family/mode;
# the reduction-length term alone, and with a floor that binds on the
# smaller products
MM_DEVICES = [DeviceSpec(mem_cap_bytes=10 ** 6, matmul=(6.1e-6, 2.3e-14, 7.7e-13)),
              DeviceSpec(mem_cap_bytes=10 ** 6, matmul=(0.0, 3.3e-16, 0.0)),
              DeviceSpec(mem_cap_bytes=10 ** 6, matmul=(2.0e-4, 1.9e-12, 4.1e-10)),
              DeviceSpec(mem_cap_bytes=10 ** 6, matmul=(0.0, 0.0, 0.0, 1.3e-7, 0.0)),
              DeviceSpec(mem_cap_bytes=10 ** 6, matmul=(6.1e-6, 2.3e-14, 7.7e-13, 4.3e-9, 2.9e-5))]
MM_CASES = [SMALL[0], SMALL[1], SMALL[3], SMALL[4], SMALL[6], SMALL[10], SMALL[13], SMALL[16], SMALL[19]]


@pytest.mark.parametrize("dev", range(len(MM_DEVICES)))
@pytest.mark.parametrize("case", range(len(MM_CASES)), ids=[c[0] for c in MM_CASES])
def test_matmul_regression_vs_full_program(torch_gpu, orc, case, dev):
    name, model, strat = MM_CASES[case]
    d = MM_DEVICES[dev]
    g = run_gpu(torch_gpu, model, strat, d)
    o = orc.run_strategies(model, strat, d, slice=False, row_width=g["finish"].shape[1], threads=8)
    assert np.any(o["status"] == 0)
    compare(g, o, strat)


# two-tier interconnect: nodes of 1, 2, 4, 8 devices and a slower network;
# strategies whose placement the nodes cut unevenly are flagged on both sides
NET_CASES = [SMALL[0], SMALL[2], SMALL[4], SMALL[5], SMALL[8], SMALL[13], SMALL[16], SMALL[20]]


@pytest.mark.parametrize("node", [1, 2, 4, 8])
@pytest.mark.parametrize("case", range(len(NET_CASES)), ids=[c[0] for c in NET_CASES])
def test_network_vs_full_program(torch_gpu, orc, case, node):
    name, model, strat = NET_CASES[case]
    d = DeviceSpec(mem_cap_bytes=10 ** 6, network=(node, 4.7e9, 1.9e-5))
    g = run_gpu(torch_gpu, model, strat, d)
    o = orc.run_strategies(model, strat, d, slice=False, row_width=g["finish"].shape[1], threads=8)
    assert np.any(o["status"] == 0)
    compare(g, o, strat)


# overlap: two streams per GPU, the gradient all-reduce on the second; hand-
# overs with a cost, free, or slow beside nodes of two GPUs
OV_DEVICES = [DeviceSpec(mem_cap_bytes=10 ** 6, streams=(2, 5.3e11, 1.7e-6)),
              DeviceSpec(mem_cap_bytes=10 ** 6, streams=(2, math.inf, 0.0)),
              DeviceSpec(mem_cap_bytes=10 ** 6, streams=(2, 2.1e9, 4.3e-5), network=(2, 4.7e9, 1.9e-5)),
              # rates so slow that clocks overflow to +inf on some strategies
              DeviceSpec(3e-302, 3e-302, 1e-303, 1e-6, 0.0, 10 ** 6, streams=(2, 1e-303, 0.0)),
              DeviceSpec(1e-301, 1e-301, 2e-303, 1e-6, 0.0, 10 ** 6, streams=(2, 2e-303, 0.0))]
OV_CASES = [(name, replace(model, overlap=1), strat) for name, model, strat in SMALL if not model.zero]


@pytest.mark.parametrize("dev", range(len(OV_DEVICES)))
@pytest.mark.parametrize("case", range(len(OV_CASES)), ids=[c[0] for c in OV_CASES])
def test_overlap_vs_full_program(torch_gpu, orc, case, dev):
    name, model, strat = OV_CASES[case]
    d = OV_DEVICES[dev]
    g = run_gpu(torch_gpu, model, strat, d)
    o = orc.run_strategies(model, strat, d, slice=False, row_width=g["finish"].shape[1], threads=8)
    assert np.any(o["status"] == 0)
    compare(g, o, strat)


GRIDS = [TINY_MLP, LARGE_MLP, GPT2_SMALL, GPT2_SMALL_TRAIN,
         replace(LARGE_MLP, name="large_mlp_mixed", model=replace(LARGE_MLP.model, mode=TRAIN_ADAM_MIXED)),
         replace(LARGE_MLP, name="large_mlp_gpipe", model=replace(LARGE_MLP.model, schedule=SCHED_GPIPE)),
         replace(GPT2_SMALL_TRAIN, name="gpt2_small_train_gpipe",
                 model=replace(GPT2_SMALL_TRAIN.model, schedule=SCHED_GPIPE)),
         replace(LARGE_MLP, name="large_mlp_recompute", model=replace(LARGE_MLP.model, recompute=1)),
         replace(GPT2_SMALL_TRAIN, name="gpt2_small_train_recompute", model=replace(GPT2_SMALL_TRAIN.model, recompute=1)),
         replace(LARGE_MLP, name="large_mlp_zero", model=replace(LARGE_MLP.model, zero=1)),
         replace(GPT2_SMALL_TRAIN, name="gpt2_small_train_zero", model=replace(GPT2_SMALL_TRAIN.model, zero=1)),
         replace(GPT2_SMALL_TRAIN, name="gpt2_small_train_matmul",
                 device=replace(GPT2_SMALL_TRAIN.device, matmul=(8.0e-6, 1.1e-14, 2.9e-13, 2.3e-9, 1.7e-5))),
         replace(LARGE_MLP, name="large_mlp_matmul",
                 device=replace(LARGE_MLP.device, matmul=(8.0e-6, 1.1e-14, 2.9e-13, 2.3e-9, 1.7e-5))),
         replace(LARGE_MLP, name="large_mlp_overlap", model=replace(LARGE_MLP.model, overlap=1),
                 device=replace(LARGE_MLP.device, streams=(2, 2.2e11, 3.1e-6))),
         replace(GPT2_SMALL_TRAIN, name="gpt2_small_train_overlap_rc",
                 model=replace(GPT2_SMALL_TRAIN.model, overlap=1, recompute=1),
                 device=replace(GPT2_SMALL_TRAIN.device, streams=(2, math.inf, 0.0)))]


@pytest.mark.parametrize("w", GRIDS, ids=[w.name for w in GRIDS])
def test_workload_grid_vs_oracle(torch_gpu, orc, w):
    from paper_2111_05426_amd import dsim
    strat = dsim.dsim_create_grid(w.model, w.grid)
    rw = int(strat[:, 2].max())
    print("%s: %d candidates" % (w.name, len(strat)), flush=True)
    g = run_gpu(torch_gpu, w.model, strat, w.device, rw)
    o = orc.run_strategies(w.model, strat, w.device, slice=True, row_width=rw, threads=8)
    compare(g, o, strat)
    # full-program oracle on the candidates whose program is small
    small = np.nonzero(o["n_ops"] <= 20000)[0][:60]
    if len(small):
        of = orc.run_strategies(w.model, strat[small], w.device, slice=False, row_width=rw, threads=8)
        sub = {k: (v[small] if isinstance(v, np.ndarray) else v) for k, v in g.items()}
        compare(sub, of, strat[small])
    # selection over the grid
    k = w.top_k
    idx, mk, found = dsim.select_topk(g["gpu"]["makespan"], g["gpu"]["cand_peak"], g["gpu"]["status"],
                                      w.device.mem_cap_bytes, k)
    ri, rm, rf = orc.topk(o["makespan"], o["cand_peak"], o["status"], w.device.mem_cap_bytes, k)
    torch_gpu.cuda.synchronize()
    assert int(found.item()) == rf and np.array_equal(idx.cpu().numpy(), ri)


# The GPT-3-shaped grids at full size (39,965 strategies each, the launch
# configuration the benchmark times: results row 64, a second stream, the
# 288e9-byte cap, top-16).  The plain 1F1B grid is compared with the oracle's
# projection on every strategy; each variant on every STRIDE-th strategy of
# the grid plus its top-16 and the extreme microbatch counts (the ZeRO oracle
# walks every data replica, hence its longer stride).
GPT3_GRIDS = {"1f1b": (GPT3_175B, 1), "gpipe": (ALL["gpt3_175b_gpipe"], 8),
              "recompute": (ALL["gpt3_175b_recompute"], 8), "zero": (ALL["gpt3_175b_zero"], 32),
              "overlap": (ALL["gpt3_175b_overlap"], 8), "mi355x_calibrated": (ALL["gpt3_175b_mi355x"], 8),
              "mi355x_overlap": (ALL["gpt3_175b_mi355x_overlap"], 8)}
GPT3_CHUNKS = 8
THREADS = max(1, min(16, os.cpu_count() or 1))
# full-program oracle on every sampled strategy whose program has at most
# 10^7 ops
FULL_MAX_OPS = 10_000_000


@pytest.fixture(scope="module")
def gpt3_runs():
    return {}


def gpt3_run(torch, cache, key):
    if key not in cache:
        from paper_2111_05426_amd import dsim
        w = GPT3_GRIDS[key][0]
        strat = dsim.dsim_create_grid(w.model, w.grid)
        assert len(strat) == 39965
        print("%s: simulating %d candidates" % (w.name, len(strat)), flush=True)
        g = run_gpu(torch, w.model, strat, w.device, 64)
        idx, mk, found = dsim.select_topk(g["gpu"]["makespan"], g["gpu"]["cand_peak"], g["gpu"]["status"],
                                          w.device.mem_cap_bytes, w.top_k)
        torch.cuda.synchronize()
        g = {k: v for k, v in g.items() if isinstance(v, np.ndarray)}
        cache[key] = (w, strat, g, (idx.cpu().numpy(), mk.cpu().numpy(), int(found.item())))
    return cache[key]


def sub(g, pick):
    return {k: v[pick] for k, v in g.items()}


@pytest.mark.parametrize("chunk", range(GPT3_CHUNKS))
def test_gpt3_grid_every_strategy(torch_gpu, orc, gpt3_runs, chunk):
    """Every strategy of the GPT-3-shaped 1F1B grid against the oracle's
    projection (an eighth of the grid per test)."""
    w, strat, g, _ = gpt3_run(torch_gpu, gpt3_runs, "1f1b")
    lo, hi = chunk * len(strat) // GPT3_CHUNKS, (chunk + 1) * len(strat) // GPT3_CHUNKS
    print("oracle on strategies %d..%d (%d threads)" % (lo, hi, THREADS), flush=True)
    o = orc.run_strategies(w.model, strat[lo:hi], w.device, slice=True, row_width=64, threads=THREADS)
    compare(sub(g, slice(lo, hi)), o, strat[lo:hi])


def variant_pick(strat, top, stride):
    K = strat[:, 3]
    return np.unique(np.concatenate([np.arange(0, len(strat), stride), top[top >= 0],
                                     np.nonzero(K == K.max())[0][:5], np.nonzero(K == 1)[0][:5]]))


@pytest.mark.parametrize("key", [k for k in GPT3_GRIDS if k != "1f1b"])
def test_gpt3_variant_strided(torch_gpu, orc, gpt3_runs, key):
    w, strat, g, (top, _, _) = gpt3_run(torch_gpu, gpt3_runs, key)
    pick = variant_pick(strat, top, GPT3_GRIDS[key][1])
    print("%s: oracle on %d strategies (every %d-th, the top-16, extreme K)" % (w.name, len(pick),
                                                                              GPT3_GRIDS[key][1]), flush=True)
    o = orc.run_strategies(w.model, strat[pick], w.device, slice=True, row_width=64, threads=THREADS)
    compare(sub(g, pick), o, strat[pick])


@pytest.mark.parametrize("key", list(GPT3_GRIDS))
def test_gpt3_grid_full_program(torch_gpu, orc, gpt3_runs, key):
    """The projection itself against the oracle's whole program (every
    device of every replica) on a seeded sample of 250 strategies (100 for
    ZeRO) plus the top-16: every one whose program has at most 10^7 ops."""
    w, strat, g, (top, _, _) = gpt3_run(torch_gpu, gpt3_runs, key)
    rng = np.random.default_rng(175)
    pick = np.unique(np.concatenate([rng.choice(len(strat), 100 if w.model.zero else 250, replace=False),
                                     top[top >= 0]]))
    lim = FULL_MAX_OPS
    small = pick[g["n_ops"][pick] <= lim]
    print("%s: whole program on %d of %d sampled strategies (<= %d ops, %.3g ops in all)"
          % (w.name, len(small), len(pick), lim, g["n_ops"][small].sum()), flush=True)
    assert len(small) >= 20
    of = orc.run_strategies(w.model, strat[small], w.device, slice=False, row_width=64, threads=THREADS)
    compare(sub(g, small), of, strat[small])


@pytest.mark.parametrize("key", list(GPT3_GRIDS))
def test_gpt3_grid_selection(torch_gpu, gpt3_runs, key):
    """The top-16 is the ordered prefix of the feasible strategies (status 0,
    peak within 288e9 bytes), ties to the lower index."""
    w, strat, g, (top, mk, found) = gpt3_run(torch_gpu, gpt3_runs, key)
    mk_all, st, cp = g["makespan"], g["status"], g["cand_peak"].view(np.uint64)
    feas = np.nonzero((st == 0) & (cp <= w.device.mem_cap_bytes))[0]
    order = feas[np.lexsort((feas, mk_all[feas]))][:16]
    assert found == len(order) and np.array_equal(top[:found], order)
    assert np.array_equal(mk[:found], mk_all[order])
    assert np.all(top[found:] == -1)
    if key != "gpipe":   # no GPipe strategy fits 288e9 bytes
        assert found == 16


@pytest.mark.parametrize("w", [GPT3_175B, ALL["gpt3_175b_zero"], ALL["gpt3_175b_overlap"]],
                         ids=["1f1b", "zero", "overlap"])
def test_split_launch_on_one_stream(torch_gpu, w):
    """The two kernels of a large transformer grid side by side (a second
    stream) or one after the other on the caller's stream: the same results,
    bit for bit, and a workspace reused by a second, smaller call."""
    from paper_2111_05426_amd import dsim
    strat = dsim.dsim_create_grid(w.model, w.grid)
    a = run_gpu(torch_gpu, w.model, strat, w.device, 64, side=True)
    b = run_gpu(torch_gpu, w.model, strat, w.device, 64, side=False)
    for k in ("makespan", "finish", "peak", "cand_peak", "n_ops", "walked_ops", "status"):
        assert np.array_equal(a[k], b[k]), k
    # one workspace for two calls in a row, the second smaller
    ws = dsim.alloc_parametric_workspace(len(strat))
    sub = strat[::3]
    for part in (strat, sub):
        r = dsim.alloc_results(len(part), 64)
        dsim.dsim_simulate_parametric(w.model, torch_gpu.from_numpy(np.ascontiguousarray(part)).cuda(), w.device,
                                      r, workspace=ws, side_stream=side_stream(torch_gpu))
        torch_gpu.cuda.synchronize()
        ref = a if part is strat else {k: v[::3] for k, v in a.items() if isinstance(v, np.ndarray)}
        for k in ("makespan", "cand_peak", "status"):
            assert np.array_equal(r[k].cpu().numpy(), ref[k]), k


def test_invalid_strategies(torch_gpu, orc):
    m = transformer(4, 32, 4, 8, 64, 12, 2, TRAIN_ADAM)
    strat = np.array([(5, 1, 1, 1),     # D does not divide the batch
                      (2, 1, 1, 7),     # K > B/D
                      (1, 1, 5, 1),     # P > L
                      (1, 3, 1, 1),     # H does not divide the heads
                      (0, 1, 1, 1), (1, 1, 1, 0), (1, 1, 1, 1)], np.int32)
    dev = DeviceSpec()
    g = run_gpu(torch_gpu, m, strat, dev, 5)
    o = orc.run_strategies(m, strat, dev, slice=False, row_width=5, threads=1)
    assert list(g["status"][:-1]) == [16] * 6 and g["status"][-1] == 0
    compare(g, o, strat)
    mm = mlp(6, 64, 12, 2, TRAIN_SGD)
    strat = np.array([(1, 2, 2, 1), (1, 2, 3, 1), (1, 2, 4, 1)], np.int32)   # pairs split by stages
    g = run_gpu(torch_gpu, mm, strat, dev, 4)
    o = orc.run_strategies(mm, strat, dev, slice=False, row_width=4, threads=1)
    assert list(g["status"]) == [16, 0, 16]
    compare(g, o, strat)


@pytest.mark.parametrize("case", [
    ("one_layer", mlp(1, 64, 16, 4, TRAIN_ADAM), [(1, 1, 1, 1), (2, 1, 1, 8), (16, 1, 1, 1)]),
    ("layer_per_stage", transformer(6, 32, 4, 8, 64, 8, 2, TRAIN_ADAM_MIXED), [(1, 2, 6, 8), (2, 1, 6, 4), (8, 1, 6, 1)]),
    ("row_per_microbatch", mlp(4, 32, 24, 2, TRAIN_SGD, schedule=SCHED_GPIPE), [(1, 1, 4, 24), (3, 2, 2, 8), (24, 1, 2, 1)]),
    ("tf_one_layer_infer", transformer(1, 32, 2, 4, 50, 3, 4, INFER), [(1, 1, 1, 3), (3, 2, 1, 1)]),
    ("single_candidate", transformer(3, 32, 4, 8, 101, 12, 2, TRAIN_ADAM, recompute=1), [(2, 2, 3, 3)]),
])
def test_degenerate_strategies(torch_gpu, orc, case):
    """One layer, one layer per stage, one row per microbatch or per
    replica, a lone candidate: parity with the full program."""
    name, model, strat = case
    strat = np.array(strat, np.int32)
    g = run_gpu(torch_gpu, model, strat, DeviceSpec())
    o = orc.run_strategies(model, strat, DeviceSpec(), slice=False, row_width=g["finish"].shape[1], threads=4)
    assert np.all(o["status"] == 0)
    compare(g, o, strat)


def test_microbatch_limit(torch_gpu, orc):
    """K up to 16,383 microbatches per candidate (then flagged); an empty
    call is a no-op."""
    from paper_2111_05426_amd import dsim
    m = mlp(2, 16, 20000, 4, TRAIN_SGD)
    strat = np.array([(1, 1, 2, 16383), (1, 1, 1, 16383), (1, 1, 2, 16384)], np.int32)
    g = run_gpu(torch_gpu, m, strat, DeviceSpec(), 2)
    o = orc.run_strategies(m, strat[:2], DeviceSpec(), slice=False, row_width=2, threads=2)
    assert list(g["status"]) == [0, 0, 16]
    compare({k: (v[:2] if isinstance(v, np.ndarray) else v) for k, v in g.items()}, o, strat[:2])
    r = dsim.alloc_results(0, 2)
    dsim.dsim_simulate_parametric(m, torch_gpu.zeros((0, 4), dtype=torch_gpu.int32, device="cuda"), DeviceSpec(), r)
    torch_gpu.cuda.synchronize()


def test_device_count_limit(torch_gpu, orc):
    """More than 2^24 devices per strategy is invalid on both sides (the
    size rule keeps every op count below 2^62); 2^24 devices simulate."""
    m = mlp(4, 16, 2 ** 26, 2, TRAIN_SGD)
    strat = np.array([(2 ** 25, 1, 1, 1), (2 ** 23, 2, 2, 1), (2 ** 22, 4, 4, 1), (2 ** 24, 1, 1, 1),
                      (2 ** 22, 2, 2, 1)], np.int32)
    g = run_gpu(torch_gpu, m, strat, DeviceSpec(), 4)
    assert list(g["status"]) == [16, 16, 16, 0, 0]
    for i in range(3):
        o = orc.sim_strategy(m, *strat[i].tolist(), DeviceSpec(), slice=True, want_devices=False)
        assert o["status"] == 16
    # op count of 2^24 replicas: linear in D (every replica runs the same
    # ops, one all-reduce per layer over all of them), from the oracle's
    # whole programs at D = 2 and 4
    n2 = orc.sim_strategy(m, 2, 1, 1, 1, DeviceSpec(), want_devices=False)["n_ops"]
    n4 = orc.sim_strategy(m, 4, 1, 1, 1, DeviceSpec(), want_devices=False)["n_ops"]
    per = (n4 - n2) // 2
    assert g["n_ops"][3] == 2 ** 24 * per + (n2 - 2 * per) and g["makespan"][3] > 0


def test_stage_limit_and_row_width(torch_gpu):
    """More than 64 pipeline stages, or more than results.row_width, is
    refused per candidate (DSIM_ST_BAD_STRATEGY), never overrun."""
    m = mlp(80, 16, 8, 4, INFER)
    strat = np.array([(1, 1, 70, 1), (1, 1, 8, 1), (1, 1, 9, 1)], np.int32)
    g = run_gpu(torch_gpu, m, strat, DeviceSpec(), 8)
    assert list(g["status"]) == [16, 0, 16]


# Device constants that are powers of two make every cost a short dyadic
# fraction, so clock + cost often lands exactly half way between two doubles
# (ties-to-even then depends on the clock's last bit); a large LM head beside
# tiny layers with no launch cost makes whole layers round away against the
# clock.  Both stress the exact long-run summation of repeated layers.
# Rates near the smallest accepted ones put the clocks in the top binades of
# the double range (near_overflow) or past it, to +inf, on some strategies
# and not others (overflow).
EDGE_DEVICES = [
    ("pow2", DeviceSpec(2.0 ** 40, 2.0 ** 36, 2.0 ** 30, 2.0 ** -18, 2.0 ** -16, 0)),
    ("pow2_nolaunch", DeviceSpec(2.0 ** 44, 2.0 ** 40, 2.0 ** 32, 0.0, 0.0, 0)),
    ("near_overflow", DeviceSpec(1e-298, 1e-298, 1e-299, 0.0, 0.0, 0)),
    ("overflow", DeviceSpec(1e-299, 1e-299, 1e-300, 1e-6, 0.0, 0)),
    ("default", DeviceSpec()),
]
EDGE_MODELS = [
    ("tf_long", transformer(24, 64, 4, 16, 1000, 16, 2, TRAIN_ADAM), all_strats([1, 2], [1, 2, 4], [1, 2, 3], [1, 2, 5, 16])),
    ("tf_tiny_layers", transformer(16, 8, 2, 2, 4_000_000, 8, 2, TRAIN_SGD), all_strats([1, 2], [1, 2], [1, 2], [1, 4, 8])),
    ("mlp_long", mlp(32, 128, 64, 2, TRAIN_ADAM), all_strats([1, 2], [1, 2], [1, 2, 4], [1, 3, 8, 32])),
    ("tf_infer_long", transformer(40, 32, 2, 8, 512, 32, 4, INFER), all_strats([1, 2], [1, 2], [1, 5], [1, 4, 32])),
    ("tf_long_rc", transformer(24, 64, 4, 16, 1000, 16, 2, TRAIN_ADAM, recompute=1),
     all_strats([1, 2], [1, 2, 4], [1, 2, 3], [1, 2, 5, 16])),
    ("mlp_long_rc", mlp(32, 128, 64, 2, TRAIN_ADAM, recompute=1), all_strats([1, 2], [1, 2], [1, 2, 4], [1, 3, 8, 32])),
    ("tf_long_zero", transformer(24, 64, 4, 16, 1000, 16, 2, TRAIN_ADAM, zero=1),
     all_strats([2, 4], [1, 2, 4], [1, 2, 3], [1, 2, 4])),
    # deep pipelines: the Sends of pipeline fill and drain (and every
    # forward and backward phase of GPipe) form runs of 12 and more, which
    # the kernel sums as prefix scans while the clocks stay in one binade and
    # no cost is a half-way case, else step by step; uneven microbatches
    # (K = 7, 5, 3) give a run two costs
    ("tf_deep_1f1b", transformer(64, 32, 4, 8, 100, 64, 2, TRAIN_ADAM),
     all_strats([1, 2], [1, 2], [16, 32, 64], [1, 7, 32])),
    ("tf_deep_gpipe", transformer(64, 32, 4, 8, 100, 64, 2, TRAIN_ADAM, schedule=SCHED_GPIPE),
     all_strats([1], [1, 2], [16, 64], [5, 32])),
    ("mlp_deep_infer", mlp(64, 64, 64, 2, INFER), all_strats([1, 2], [1], [32, 64], [3, 32])),
]


@pytest.mark.parametrize("dev", EDGE_DEVICES, ids=[d[0] for d in EDGE_DEVICES])
@pytest.mark.parametrize("case", EDGE_MODELS, ids=[c[0] for c in EDGE_MODELS])
def test_exact_long_runs(torch_gpu, orc, case, dev):
    name, model, strat = case
    g = run_gpu(torch_gpu, model, strat, dev[1])
    o = orc.run_strategies(model, strat, dev[1], slice=True, row_width=g["finish"].shape[1], threads=8)
    assert np.any(o["status"] == 0)
    compare(g, o, strat)
