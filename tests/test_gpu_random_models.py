"""Randomised GPU parity of the transform-driven simulation and of the table
materialiser: seeded random
small models (family, training mode, schedule, recomputation, ZeRO or
overlap) on random device models (MatMul regression, two-tier network,
streams, power-of-two constants that make rounding ties frequent) and
random strategies, against the oracle's whole distributed program.  Bar:
status, op counts and peaks exact, times bit-identical."""
import math
from dataclasses import replace

import numpy as np
import pytest

from paper_2111_05426_amd.workloads import (DeviceSpec, INFER, SCHED_GPIPE, TRAIN_ADAM, TRAIN_ADAM_MIXED, TRAIN_SGD,
                                            mlp, transformer)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    from paper_2111_05426_amd import dsim
    dsim.lib()
    return torch


def random_case(seed):
    rng = np.random.default_rng(10_000 + seed)
    mode = int(rng.choice([INFER, TRAIN_SGD, TRAIN_ADAM, TRAIN_ADAM_MIXED]))
    sched = SCHED_GPIPE if rng.random() < 0.4 else 0
    rc = int(rng.random() < 0.3)
    extra = rng.choice(["none", "zero", "overlap"], p=[0.5, 0.25, 0.25])
    zero, overlap = int(extra == "zero"), int(extra == "overlap")
    L = int(rng.integers(1, 9))
    batch = int(rng.choice([6, 8, 12, 16, 24, 30]))
    e = int(rng.choice([2, 4]))
    if rng.random() < 0.5:
        d = int(rng.choice([16, 32, 48, 64]))
        model = mlp(L, d, batch, e, mode, schedule=sched, recompute=rc, zero=zero, overlap=overlap)
    else:
        heads = int(rng.choice([2, 4]))
        d = heads * int(rng.choice([4, 8]))
        model = transformer(L, d, heads, int(rng.choice([4, 8])), int(rng.integers(20, 120)), batch, e, mode,
                            schedule=sched, recompute=rc, zero=zero, overlap=overlap)
    if rng.random() < 0.3:   # powers of two: costs land on half-way cases often
        dev = DeviceSpec(2.0 ** int(rng.integers(36, 44)), 2.0 ** int(rng.integers(32, 40)),
                         2.0 ** int(rng.integers(28, 34)), 2.0 ** -int(rng.integers(14, 20)),
                         2.0 ** -int(rng.integers(14, 20)), 0)
    else:
        dev = DeviceSpec(float(rng.uniform(1e12, 2e15)), float(rng.uniform(5e11, 6e12)), float(rng.uniform(1e10, 2e11)),
                         float(rng.uniform(0, 1e-5)), float(rng.uniform(0, 2e-5)), 0)
    if rng.random() < 0.3:
        dev = replace(dev, matmul=(float(rng.uniform(0, 2e-5)), float(rng.uniform(1e-16, 1e-13)),
                                   float(rng.uniform(0, 1e-12))))
        # half of them with the reduction-length term and a floor (drawn
        # from a stream of their own, so the other draws stay as they were)
        r2 = np.random.default_rng(20_000 + seed)
        if r2.random() < 0.5:
            dev = replace(dev, matmul=dev.matmul + (float(r2.uniform(0, 5e-8)), float(r2.uniform(0, 3e-5))))
    if rng.random() < 0.3:
        dev = replace(dev, network=(int(rng.choice([1, 2, 4])), float(rng.uniform(1e9, 5e10)), float(rng.uniform(0, 2e-5))))
    if overlap:
        dev = replace(dev, streams=(2, [math.inf, float(rng.uniform(1e11, 1e12))][int(rng.integers(0, 2))],
                                    float(rng.uniform(0, 2e-6))))
    strat = np.array([(int(rng.choice([1, 2, 3, 4])), int(rng.choice([1, 2])), int(rng.integers(1, min(L, 6) + 1)),
                       int(rng.integers(1, 9))) for _ in range(24)], np.int32)
    return model, dev, np.unique(strat, axis=0)


@pytest.mark.parametrize("seed", range(200))
def test_random_model_vs_full_program(torch_gpu, orc, seed):
    from paper_2111_05426_amd import dsim
    model, dev, strat = random_case(seed)
    rw = int(strat[:, 2].max())
    r = dsim.alloc_results(len(strat), rw)
    dsim.dsim_simulate_parametric(model, torch_gpu.from_numpy(strat).cuda(), dev, r)
    torch_gpu.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in r.items() if k != "row_width"}
    o = orc.run_strategies(model, strat, dev, slice=False, row_width=rw, threads=8)
    assert np.array_equal(g["status"], o["status"]), (seed, strat[g["status"] != o["status"]])
    ok = o["status"] == 0
    assert np.array_equal(g["n_ops"][ok], o["n_ops"][ok].astype(np.int64))
    assert np.array_equal(g["cand_peak"][ok].view(np.uint64), o["cand_peak"][ok])
    assert np.array_equal(g["peak"][ok].view(np.uint64), o["peak"][ok])
    assert np.array_equal(g["makespan"][ok], o["makespan"][ok])
    assert np.array_equal(g["finish"][ok], o["finish"][ok])


@pytest.mark.parametrize("seed", range(0, 200, 2))
def test_random_model_as_tables(torch_gpu, orc, seed):
    """The same random cases through dsim_materialize_tables and
    dsim_simulate_tables (programs of at most 8 devices), device by device
    against the oracle's whole program."""
    from paper_2111_05426_amd import dsim
    model, dev, strat = random_case(seed)
    S = 2 if model.overlap else 1
    strat = strat[S * strat[:, 0] * strat[:, 1] * strat[:, 2] <= 8]
    if len(strat) == 0:
        pytest.skip("no strategy of this case fits 8 devices")
    o = orc.run_strategies(model, strat, dev, slice=False, row_width=int(strat[:, 2].max()), threads=8)
    ok = o["status"] & 16 == 0                     # over the cap still simulates
    if not ok.any():
        pytest.skip("every strategy of this case is invalid")
    strat, o_mk = strat[ok], o["makespan"][ok]
    cand = torch_gpu.from_numpy(np.ascontiguousarray(strat)).cuda()
    t, mst = dsim.dsim_materialize_tables(model, cand, 8, int(o["n_ops"][ok].max()))
    r = dsim.alloc_results(len(strat), 8)
    dsim.dsim_simulate_tables(t, len(strat), 8, dev, r, init_live=t["init_live"])
    torch_gpu.cuda.synchronize()
    assert not mst.cpu().numpy().any()
    fin, pk = r["finish"].cpu().numpy(), r["peak"].cpu().numpy().view(np.uint64)
    assert np.array_equal(r["makespan"].cpu().numpy(), o_mk)
    for i, (D, H, P, K) in enumerate(strat.tolist()):
        ref = orc.sim_strategy(model, D, H, P, K, dev)
        n = S * D * H * P
        assert np.array_equal(fin[i, :n], ref["dev_finish"]), (seed, strat[i].tolist())
        assert np.array_equal(pk[i, :n], ref["dev_peak"]), (seed, strat[i].tolist())
