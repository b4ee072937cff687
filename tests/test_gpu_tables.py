"""GPU parity: table simulator, random-table generator and top-k selection
against the CPU oracle, element by element on the same seeded inputs.

Bar: integer outputs (peaks, status, op counts, indices, generated tables)
bit-exact; fp64 times within 1e-12 relative (both sides evaluate the same
IEEE expressions in the same order with contraction off, so they are
expected to be equal bit for bit, and the tests also record that).
"""
import os
from dataclasses import replace

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

REL = 1e-12


@pytest.fixture(scope="module")
def torch_gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    from paper_2111_05426_amd import dsim
    dsim.lib()
    return torch


def assert_times(gpu, ref):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    np.testing.assert_allclose(gpu, ref, rtol=REL, atol=0)
    assert np.array_equal(gpu, ref), "times agree to 1e-12 but not bit for bit"


def random_tables(rng, n_cand, max_ops, n_dev, bad=False, rooted=False, classes=False):
    """Seeded synthetic tables with every op kind; bad=True also plants
    invalid ops and frees larger than the live bytes; rooted=True adds
    broadcast and reduce records (their masks hold the root)."""
    p = [0.6, 0.15, 0.1, 0.08, 0.07] if rooted else [0.7, 0.2, 0.1]
    kind = rng.choice(len(p), size=(max_ops, n_cand), p=p).astype(np.uint32)
    a = rng.integers(0, n_dev, (max_ops, n_cand)).astype(np.uint32)
    b = rng.integers(0, n_dev, (max_ops, n_cand)).astype(np.uint32)
    if n_dev > 1:
        b = np.where(b == a, (a + 1) % n_dev, b)
    mask = rng.integers(1, 1 << n_dev, (max_ops, n_cand)).astype(np.uint32)
    code = np.where(kind == 2, 2 | (mask << 16), kind | (a << 8) | (b << 16)).astype(np.uint32)
    code = np.where(kind >= 3, kind | (a << 8) | ((mask | (1 << a)) << 16), code).astype(np.uint32)
    if classes:   # matrix multiplication records (cost class 1) among the compute ops
        code = np.where((kind == 0) & (rng.random((max_ops, n_cand)) < 0.5), code | (1 << 24), code).astype(np.uint32)
    if n_dev == 1:
        code = np.where(kind == 1, 0, code).astype(np.uint32)
    alloc = rng.integers(0, 5000, (max_ops, n_cand)).astype(np.uint32)
    free = rng.integers(0, 3000, (max_ops, n_cand)).astype(np.uint32)
    if bad:
        sel = rng.random((max_ops, n_cand)) < 0.002
        code = np.where(sel, rng.integers(0, 1 << 32, (max_ops, n_cand), dtype=np.uint64).astype(np.uint32), code)
        # near-valid records: reserved byte 0, any of the five kinds or one
        # beyond, device fields up to two past the last device (a send to
        # itself, a compute op on a missing device, an empty or oversized
        # all-reduce mask)
        near = (rng.integers(0, 6, (max_ops, n_cand)) | (rng.integers(0, n_dev + 2, (max_ops, n_cand)) << 8) |
                (rng.integers(0, min(1 << (n_dev + 1), 256), (max_ops, n_cand)) << 16)).astype(np.uint32)
        code = np.where(rng.random((max_ops, n_cand)) < 0.003, near, code).astype(np.uint32)
        free = np.where(rng.random((max_ops, n_cand)) < 0.01, 10 ** 6, free).astype(np.uint32)
    else:
        free = np.minimum(free, alloc)
    fl = np.exp(rng.uniform(np.log(1e6), np.log(1e12), (max_ops, n_cand))).astype(np.float32)
    by = np.exp(rng.uniform(np.log(1e3), np.log(1e9), (max_ops, n_cand))).astype(np.float32)
    if bad:   # fields that are not finite and >= 0 make an op invalid
        for arr in (fl, by):
            for v in (np.inf, -np.inf, np.nan, -0.0, -5.0):
                arr[rng.random((max_ops, n_cand)) < 0.0005] = np.float32(v)
    n_ops = rng.integers(0, max_ops + 1, n_cand).astype(np.uint32)
    n_ops[:3] = [0, max_ops, 1][:min(3, n_cand)] if n_cand >= 3 else n_ops[:3]
    init = rng.integers(0, 10 ** 5, (n_cand, n_dev)).astype(np.uint64)
    out = dict(code=code, flops=fl, bytes=by, alloc=alloc, free=free, n_ops=n_ops, init=init)
    if classes:   # reduction lengths, log-uniform up to 2^32 - 1 (read on class-1 records only)
        out["mm_k"] = np.exp(rng.uniform(0.0, np.log(2.0 ** 32 - 1), (max_ops, n_cand))).astype(np.uint32)
    return out


def to_gpu(torch, t):
    g = {}
    for k in ("code", "alloc", "free", "n_ops", "mm_k"):
        if k in t:
            g[k] = torch.from_numpy(t[k].view(np.int32)).cuda()
    for k in ("flops", "bytes"):
        g[k] = torch.from_numpy(t[k]).cuda()
    return g


def results_np(r):
    out = {}
    for k, v in r.items():
        if k == "row_width":
            continue
        out[k] = v.cpu().numpy()
    return out


@pytest.mark.parametrize("kinds", ["plain", "bcast_reduce", "matmul", "network", "streams"])
@pytest.mark.parametrize("n_dev", [1, 2, 3, 5, 8])
@pytest.mark.parametrize("bad", [False, True])
def test_tables_vs_oracle(torch_gpu, orc, n_dev, bad, kinds):
    from paper_2111_05426_amd import dsim
    from paper_2111_05426_amd.workloads import DeviceSpec
    torch = torch_gpu
    rooted, classes, net = kinds in ("bcast_reduce", "network", "streams"), kinds == "matmul", kinds == "network"
    streams = kinds == "streams"
    rng = np.random.default_rng(1000 + n_dev + 17 * bad + 101 * rooted + 211 * classes + 307 * net + 401 * streams)
    n_cand, max_ops = 777, 301   # several 256-lane blocks and a ragged tail
    t = random_tables(rng, n_cand, max_ops, n_dev, bad, rooted, classes)
    # the MatMul regression with its reduction-length term and a floor that
    # binds on part of the records (the floor above c0 + the smallest terms)
    dev = DeviceSpec(mem_cap_bytes=2 * 10 ** 5, matmul=(4.5e-6, 9.1e-15, 1.3e-12, 3.7e-14, 4.0e-5) if classes else None,
                     network=(max(1, n_dev // 2 - (n_dev == 5)), 3.3e9, 2.1e-5) if net else None)
    if streams:
        # two or three streams per GPU; GPUs in nodes of one for some sizes;
        # no byte term between streams for others
        dev = replace(dev, streams=(2 + n_dev % 2, np.inf if n_dev % 3 == 0 else 4.4e11, 1.3e-6),
                      network=(1, 3.3e9, 2.1e-5) if n_dev in (3, 8) else None)
    g = to_gpu(torch, t)
    init = torch.from_numpy(t["init"].view(np.int64)).cuda()
    rw = n_dev + 2
    r = dsim.alloc_results(n_cand, rw)
    dsim.dsim_simulate_tables(g, n_cand, n_dev, dev, r, init_live=init)
    torch.cuda.synchronize()
    R = results_np(r)
    mk, fin, pk, cp, st = [], [], [], [], []
    for c in range(n_cand):
        n = int(t["n_ops"][c])
        tab = {k: t[k][:n, c] for k in ("code", "flops", "bytes", "alloc", "free", "mm_k") if k in t}
        o = orc.sim_table(tab, n_dev, dev, init_live=t["init"][c])
        mk.append(o["makespan"]); fin.append(o["finish"]); pk.append(o["peak"])
        cp.append(o["cand_peak"]); st.append(o["status"])
    assert_times(R["makespan"], mk)
    assert_times(R["finish"][:, :n_dev], np.array(fin))
    assert np.all(R["finish"][:, n_dev:] == 0)
    assert np.array_equal(R["peak"][:, :n_dev].view(np.uint64), np.array(pk, np.uint64))
    assert np.array_equal(R["cand_peak"].view(np.uint64), np.array(cp, np.uint64))
    assert np.array_equal(R["status"], np.array(st, np.int32))
    assert np.array_equal(R["n_ops"], t["n_ops"].astype(np.int64))
    if bad:
        assert np.any(R["status"] & dsim.ST_MEM_UNDERFLOW)


@pytest.mark.parametrize("n_dev", [3, 8])
def test_tables_long_op_counts_and_large_resident_bytes(torch_gpu, orc, n_dev):
    """Lanes whose op count exceeds max_ops are flagged (DSIM_ST_BAD_OP) and
    simulate max_ops ops, also when another op of theirs (a broadcast or
    reduce record, a free that would underflow) sends them to the exact
    path; lanes starting with 2^62 or more live bytes on a device keep exact
    integer peaks.  Against the oracle on the first max_ops ops."""
    from paper_2111_05426_amd import dsim
    from paper_2111_05426_amd.workloads import DeviceSpec
    torch = torch_gpu
    rng = np.random.default_rng(9090 + n_dev)
    n_cand, max_ops = 520, 67
    t = random_tables(rng, n_cand, max_ops, n_dev, bad=True, rooted=True)
    over = rng.random(n_cand) < 0.4
    t["n_ops"] = np.where(over, max_ops + rng.integers(1, 1000, n_cand), t["n_ops"]).astype(np.uint32)
    big = rng.random((n_cand, n_dev)) < 0.2
    t["init"] = np.where(big, (np.uint64(1) << np.uint64(62)) + rng.integers(0, 1 << 40, (n_cand, n_dev)).astype(
        np.uint64), t["init"]).astype(np.uint64)
    t["init"][0] = np.uint64((1 << 64) - (1 << 20))   # near the top of the u64 range
    g = to_gpu(torch, t)
    init = torch.from_numpy(t["init"].view(np.int64)).cuda()
    dev = DeviceSpec()
    r = dsim.alloc_results(n_cand, n_dev)
    dsim.dsim_simulate_tables(g, n_cand, n_dev, dev, r, init_live=init)
    torch.cuda.synchronize()
    R = results_np(r)
    for c in range(n_cand):
        n = min(int(t["n_ops"][c]), max_ops)
        o = orc.sim_table({k: t[k][:n, c] for k in ("code", "flops", "bytes", "alloc", "free")}, n_dev, dev,
                          init_live=t["init"][c])
        want = o["status"] | (dsim.ST_BAD_OP if t["n_ops"][c] > max_ops else 0)
        assert R["status"][c] == want, c
        assert_times(R["finish"][c], o["finish"])
        assert np.array_equal(R["peak"][c].view(np.uint64), np.asarray(o["peak"], np.uint64)), c
    assert np.all(R["n_ops"] == np.minimum(t["n_ops"], max_ops))
    assert np.any(over & ((R["status"] & (dsim.ST_MEM_UNDERFLOW | dsim.ST_BAD_DEVICE)) != 0))


@pytest.mark.parametrize("n_dev", [3, 8])
def test_tables_overflowing_costs(torch_gpu, orc, n_dev):
    """Valid rates so slow that op costs and clocks overflow to +inf: both
    sides reach the same infinite (and finite) times, and no NaN appears."""
    from paper_2111_05426_amd import dsim
    from paper_2111_05426_amd.workloads import DeviceSpec
    torch = torch_gpu
    rng = np.random.default_rng(4242 + n_dev)
    n_cand, max_ops = 300, 257
    t = random_tables(rng, n_cand, max_ops, n_dev)
    dev = DeviceSpec(flops_per_s=1e-290, link_bytes_per_s=1e-300, launch_s=0.0)
    g = to_gpu(torch, t)
    init = torch.from_numpy(t["init"].view(np.int64)).cuda()
    r = dsim.alloc_results(n_cand, n_dev)
    dsim.dsim_simulate_tables(g, n_cand, n_dev, dev, r, init_live=init)
    torch.cuda.synchronize()
    R = results_np(r)
    mk, fin = [], []
    for c in range(n_cand):
        n = int(t["n_ops"][c])
        o = orc.sim_table({k: t[k][:n, c] for k in ("code", "flops", "bytes", "alloc", "free")}, n_dev, dev,
                          init_live=t["init"][c])
        mk.append(o["makespan"]); fin.append(o["finish"])
    mk, fin = np.array(mk), np.array(fin)
    assert np.isinf(mk).sum() > n_cand // 2 and np.isfinite(mk).sum() > 0 and not np.isnan(fin).any()
    assert_times(R["makespan"], mk)
    assert_times(R["finish"], fin)


@pytest.mark.parametrize("n_cand", [(1 << 28) - 1, 1 << 28])
def test_tables_largest_fast_path_and_beyond(torch_gpu, orc, n_cand):
    """The largest table the fast path takes (its loads reach four op rows,
    16 * n_cand bytes, through 32-bit offsets) and one candidate more, which
    the op-by-op path takes: sampled candidates, first and last included,
    against the oracle.  About 40 GB of tables, built on the GPU."""
    from paper_2111_05426_amd import dsim
    from paper_2111_05426_amd.workloads import DeviceSpec
    torch = torch_gpu
    n_dev, max_ops = 8, 8
    g = torch.Generator(device="cuda").manual_seed(77)
    shape = (max_ops, n_cand)
    kind = torch.randint(0, 10, shape, device="cuda", generator=g, dtype=torch.int32)
    kind = torch.where(kind < 7, 0, torch.where(kind < 9, 1, 2))
    a = torch.randint(0, n_dev, shape, device="cuda", generator=g, dtype=torch.int32)
    b = (a + torch.randint(1, n_dev, shape, device="cuda", generator=g, dtype=torch.int32)) % n_dev
    mask = torch.randint(1, 1 << n_dev, shape, device="cuda", generator=g, dtype=torch.int32)
    code = torch.where(kind == 2, 2 | (mask << 16), kind | (a << 8) | (b << 16)).to(torch.int32)
    del a, b, mask, kind
    t = {"code": code,
         "flops": torch.rand(shape, device="cuda", generator=g) * 1e9,
         "bytes": torch.rand(shape, device="cuda", generator=g) * 1e7,
         "alloc": torch.randint(0, 5000, shape, device="cuda", generator=g, dtype=torch.int32)}
    t["free"] = torch.minimum(t["alloc"], torch.randint(0, 5000, shape, device="cuda", generator=g, dtype=torch.int32))
    t["n_ops"] = torch.randint(0, max_ops + 1, (n_cand,), device="cuda", generator=g, dtype=torch.int32)
    t["n_ops"][-300:] = max_ops
    r = {"makespan": torch.empty(n_cand, dtype=torch.float64, device="cuda"),
         "cand_peak": torch.empty(n_cand, dtype=torch.int64, device="cuda"),
         "n_ops": torch.empty(n_cand, dtype=torch.int64, device="cuda"),
         "status": torch.empty(n_cand, dtype=torch.int32, device="cuda"), "row_width": 0}
    dev = DeviceSpec()
    dsim.dsim_simulate_tables(t, n_cand, n_dev, dev, r)
    torch.cuda.synchronize()
    rng = np.random.default_rng(n_cand)
    idx = np.unique(np.concatenate([[0, 1, n_cand - 257, n_cand - 1], rng.integers(0, n_cand, 200)]))
    it = torch.from_numpy(idx).cuda()
    cols = {k: t[k][:, it].cpu().numpy() for k in ("code", "flops", "bytes", "alloc", "free")}
    nops = t["n_ops"][it].cpu().numpy()
    for k in ("code", "alloc", "free"):
        cols[k] = cols[k].view(np.uint32)
    got = {k: r[k][it].cpu().numpy() for k in ("makespan", "cand_peak", "n_ops", "status")}
    mk, cp, st = [], [], []
    for i in range(len(idx)):
        n = int(nops[i])
        o = orc.sim_table({k: cols[k][:n, i] for k in cols}, n_dev, dev)
        mk.append(o["makespan"]); cp.append(o["cand_peak"]); st.append(o["status"])
    assert_times(got["makespan"], mk)
    assert np.array_equal(got["cand_peak"].view(np.uint64), np.array(cp, np.uint64))
    assert np.array_equal(got["status"], np.array(st, np.int32))
    assert np.array_equal(got["n_ops"], nops.astype(np.int64))


def gen_gpu(torch, seed, n_cand, n_ops, n_dev):
    from paper_2111_05426_amd import dsim
    g = dsim.alloc_tables(n_cand, n_ops)
    dsim.dsim_generate_random_tables(seed, n_cand, n_ops, n_dev, g)
    return g


@pytest.mark.parametrize("n_dev", [2, 5, 8])
def test_generator_bit_exact(torch_gpu, orc, n_dev):
    torch = torch_gpu
    n_cand, n_ops = 700, 513
    g = gen_gpu(torch, 11 + n_dev, n_cand, n_ops, n_dev)
    torch.cuda.synchronize()
    G = {k: v.cpu().numpy() for k, v in g.items()}
    for c in range(n_cand):
        o = orc.gen_table(11 + n_dev, c, n_ops, n_dev)
        for k, gk in (("code", "code"), ("alloc", "alloc"), ("free", "free")):
            assert np.array_equal(G[gk][:, c].view(np.uint32), o[k]), (c, k)
        for k in ("flops", "bytes"):
            assert np.array_equal(G[k][:, c].view(np.uint32), o[k].view(np.uint32)), (c, k)
    assert np.all(G["n_ops"] == n_ops)


def test_generated_tables_simulate_vs_oracle(torch_gpu, orc):
    from paper_2111_05426_amd import dsim
    from paper_2111_05426_amd.workloads import DeviceSpec
    torch = torch_gpu
    n_cand, n_ops, n_dev = 3000, 2048, 8
    dev = DeviceSpec()
    g = gen_gpu(torch, 0, n_cand, n_ops, n_dev)
    r = dsim.alloc_results(n_cand, n_dev)
    dsim.dsim_simulate_tables(g, n_cand, n_dev, dev, r)
    torch.cuda.synchronize()
    R = results_np(r)
    o = orc.run_random_tables(0, n_ops, n_dev, np.arange(n_cand), dev, threads=8)
    assert_times(R["makespan"], o["makespan"])
    assert_times(R["finish"], o["finish"])
    assert np.array_equal(R["peak"].view(np.uint64), o["peak"])
    assert np.array_equal(R["cand_peak"].view(np.uint64), o["cand_peak"])
    assert np.array_equal(R["status"], o["status"])
    assert np.all(R["status"] == 0)


FULL_CHUNKS = 4
THREADS = max(1, min(16, os.cpu_count() or 1))


@pytest.fixture(scope="module")
def full_size_tables(torch_gpu):
    """The measured workload at its full size, in the launch configuration the
    benchmark times (1,000,000 candidates x 2,048 ops x 8 devices, generated
    on the GPU), simulated once; the results come back to the host."""
    from paper_2111_05426_amd import dsim
    from paper_2111_05426_amd.workloads import RANDOM_TABLES
    torch = torch_gpu
    spec = RANDOM_TABLES.tables
    print("full-size random tables: generating", flush=True)
    g = gen_gpu(torch, spec.seed, spec.n_cand, spec.n_ops, spec.n_dev)
    r = dsim.alloc_results(spec.n_cand, spec.n_dev)
    dsim.dsim_simulate_tables(g, spec.n_cand, spec.n_dev, RANDOM_TABLES.device, r)
    idx, mk, found = dsim.select_topk(r["makespan"], r["cand_peak"], r["status"], 0, 4)
    torch.cuda.synchronize()
    print("full-size random tables: simulated", flush=True)
    rng = np.random.default_rng(5)
    cols = np.unique(np.concatenate([rng.integers(0, spec.n_cand, 40), [0, spec.n_cand - 1]]))
    gen = {c: {k: g[k][:, int(c)].cpu().numpy() for k in ("code", "flops", "bytes", "alloc", "free")} for c in cols}
    out = dict(spec=spec, dev=RANDOM_TABLES.device, res=results_np(r), gen=gen,
               top=(idx.cpu().numpy(), mk.cpu().numpy(), int(found.item())))
    del g, r
    torch.cuda.empty_cache()
    return out


@pytest.mark.parametrize("chunk", range(FULL_CHUNKS))
def test_random_tables_full_size_every_candidate(orc, full_size_tables, chunk):
    """Every candidate of the full-size workload against the oracle, element
    by element (a quarter of the million per test)."""
    F = full_size_tables
    spec, R = F["spec"], F["res"]
    lo, hi = chunk * spec.n_cand // FULL_CHUNKS, (chunk + 1) * spec.n_cand // FULL_CHUNKS
    print("oracle on candidates %d..%d (%d threads)" % (lo, hi, THREADS), flush=True)
    o = orc.run_random_tables(spec.seed, spec.n_ops, spec.n_dev, np.arange(lo, hi), F["dev"], threads=THREADS)
    assert_times(R["makespan"][lo:hi], o["makespan"])
    assert_times(R["finish"][lo:hi], o["finish"])
    assert np.array_equal(R["peak"][lo:hi].view(np.uint64), o["peak"])
    assert np.array_equal(R["cand_peak"][lo:hi].view(np.uint64), o["cand_peak"])
    assert np.array_equal(R["status"][lo:hi], o["status"])
    assert np.array_equal(R["n_ops"][lo:hi].astype(np.uint64), o["n_ops"])


def test_random_tables_full_size_generator_and_selection(orc, full_size_tables):
    """Sampled generated columns bit for bit, and the top-4 over the million
    equal to the ordered prefix of the simulated values."""
    F = full_size_tables
    spec, R = F["spec"], F["res"]
    for c, cols in F["gen"].items():
        ref = orc.gen_table(spec.seed, int(c), spec.n_ops, spec.n_dev)
        for k in ("code", "alloc", "free"):
            assert np.array_equal(cols[k].view(np.uint32), ref[k]), (c, k)
        for k in ("flops", "bytes"):
            assert np.array_equal(cols[k].view(np.uint32), ref[k].view(np.uint32)), (c, k)
    idx, mk, found = F["top"]
    order = np.lexsort((np.arange(spec.n_cand), R["makespan"]))[:4]
    assert found == 4 and np.array_equal(idx, order)
    assert_times(mk, R["makespan"][order])
    ri, rm, rf = orc.topk(R["makespan"], R["cand_peak"].view(np.uint64), R["status"], 0, 4)
    assert rf == 4 and np.array_equal(ri, idx)


@pytest.mark.parametrize("n", [0, 1, 255, 4097, 100_003, 1_000_000])
@pytest.mark.parametrize("k", [1, 5, 16, 64])
def test_argmin_vs_oracle(torch_gpu, orc, n, k):
    from paper_2111_05426_amd import dsim
    torch = torch_gpu
    rng = np.random.default_rng(n * 7 + k)
    mk = np.round(rng.uniform(0, 5, n), 2 if n > 1000 else 1)   # many exact ties
    pk = rng.integers(0, 1000, n).astype(np.uint64)
    st = np.where(rng.random(n) < 0.2, 8, 0).astype(np.int32)
    for cap in (0, 500):
        idx, mo, found = dsim.select_topk(torch.from_numpy(mk).cuda(), torch.from_numpy(pk.view(np.int64)).cuda(),
                                          torch.from_numpy(st).cuda(), cap, k)
        torch.cuda.synchronize()
        ri, rm, rf = orc.topk(mk, pk, st, cap, k)
        assert int(found.item()) == rf
        assert np.array_equal(idx.cpu().numpy(), ri)
        assert np.array_equal(mo.cpu().numpy(), rm)


def test_empty_inputs(torch_gpu):
    from paper_2111_05426_amd import dsim
    from paper_2111_05426_amd.workloads import DeviceSpec
    torch = torch_gpu
    g = dsim.alloc_tables(0, 16)
    r = dsim.alloc_results(0, 8)
    dsim.dsim_simulate_tables(g, 0, 8, DeviceSpec(), r)
    g = dsim.alloc_tables(5, 0)
    r = dsim.alloc_results(5, 8)
    dsim.dsim_generate_random_tables(0, 5, 0, 8, g)
    dsim.dsim_simulate_tables(g, 5, 8, DeviceSpec(), r)
    torch.cuda.synchronize()
    assert np.all(r["makespan"].cpu().numpy() == 0) and np.all(r["status"].cpu().numpy() == 0)
