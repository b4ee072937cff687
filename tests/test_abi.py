"""The C ABI on the host: library loads, exports what include/dsim.h
declares, enumerates the grid like the oracle, and rejects bad arguments
before any launch (none of these calls touches a GPU)."""
import ctypes as C

import numpy as np
import pytest

from paper_2111_05426_amd import dsim
from paper_2111_05426_amd.workloads import (ALL, DeviceSpec, GridSpec, INFER, TRAIN_SGD, mlp, transformer)


def test_exports_every_declared_function():
    names = dsim.header_functions()
    assert set(names) == {"dsim_last_error", "dsim_create_grid", "dsim_simulate_tables",
                          "dsim_simulate_parametric", "dsim_parametric_workspace", "dsim_argmin_workspace",
                          "dsim_argmin", "dsim_generate_random_tables", "dsim_materialize_tables",
                          "dsim_simulate_parametric_static", "dsim_interpret_program", "dsim_lower_programs"}
    L = dsim.lib()
    for n in names:
        assert hasattr(L, n), n


GRIDS = [(w.model, w.grid) for w in ALL.values() if w.model is not None] + [
    (mlp(16, 8192, 65536, 2, TRAIN_SGD), GridSpec(16, 1, 2, 128)),
    (transformer(24, 2048, 16, 1024, 50257, 128, 2, INFER), GridSpec(16, 1, 2, 128)),
    (mlp(6, 96, 60, 4, TRAIN_SGD), GridSpec(32, 0, 1, 40, 1)),
    (transformer(10, 60, 6, 16, 77, 36, 2, INFER), GridSpec(64, 0, 0, 64)),
]


@pytest.mark.parametrize("i", range(len(GRIDS)))
def test_grid_matches_oracle(orc, i):
    model, grid = GRIDS[i]
    a = dsim.dsim_create_grid(model, grid)
    b = orc.create_grid(model, grid)
    assert np.array_equal(a, b)


def test_grid_enospc():
    m, g = GRIDS[0]
    L = dsim.lib()
    out = np.zeros((3, 4), np.int32)
    n = C.c_int64()
    mm, gg = dsim.model_struct(m), dsim.dsim_grid_spec(g.max_devices, g.exact_devices, g.k_mode, g.k_max, 0)
    rc = L.dsim_create_grid(C.byref(mm), C.byref(gg), out.ctypes.data, 3, C.byref(n))
    assert rc == dsim.DSIM_ENOSPC and n.value > 3
    assert "cap" in dsim.dsim_last_error()


def _err(fn):
    with pytest.raises(dsim.DsimError) as e:
        fn()
    return e.value.code


def test_argument_errors_before_launch():
    L = dsim.lib()
    dev = dsim.device_model(DeviceSpec())
    res = dsim.dsim_results()
    tab = dsim.dsim_tables()
    tab.n_dev, tab.max_ops = 9, 4
    assert L.dsim_simulate_tables(C.byref(tab), 10, C.byref(dev), C.byref(res), None) == dsim.DSIM_ERANGE
    tab.n_dev = 0
    assert L.dsim_simulate_tables(C.byref(tab), 10, C.byref(dev), C.byref(res), None) == dsim.DSIM_ERANGE
    tab.n_dev = 4
    assert L.dsim_simulate_tables(C.byref(tab), 10, C.byref(dev), C.byref(res), None) == dsim.DSIM_EINVAL
    assert L.dsim_simulate_tables(C.byref(tab), 10, None, C.byref(res), None) == dsim.DSIM_EINVAL
    bad = dsim.device_model(DeviceSpec(flops_per_s=0.0))
    assert L.dsim_simulate_tables(C.byref(tab), 10, C.byref(bad), C.byref(res), None) == dsim.DSIM_EINVAL
    bad = dsim.device_model(DeviceSpec(link_latency_s=float("nan")))
    assert L.dsim_simulate_tables(C.byref(tab), 10, C.byref(bad), C.byref(res), None) == dsim.DSIM_EINVAL
    # rates whose reciprocal overflows (a zero byte count times 1/rate = inf
    # would be NaN); a rate just above that limit is accepted
    for spec in (DeviceSpec(flops_per_s=1e-310), DeviceSpec(mem_bytes_per_s=5e-309),
                 DeviceSpec(link_bytes_per_s=1e-320)):
        bad = dsim.device_model(spec)
        assert L.dsim_simulate_tables(C.byref(tab), 10, C.byref(bad), C.byref(res), None) == dsim.DSIM_EINVAL
        assert "reciprocal" in dsim.dsim_last_error()
    slow = dsim.device_model(DeviceSpec(flops_per_s=1e-290, link_bytes_per_s=6e-309))
    assert L.dsim_simulate_tables(C.byref(tab), 0, C.byref(slow), C.byref(res), None) == dsim.DSIM_OK
    # n_cand == 0 is a no-op; one lane per candidate in one dispatch caps it
    assert L.dsim_simulate_tables(C.byref(tab), 0, C.byref(dev), C.byref(res), None) == dsim.DSIM_OK
    assert L.dsim_simulate_tables(C.byref(tab), (1 << 32) - 255, C.byref(dev), C.byref(res), None) == dsim.DSIM_ERANGE
    assert "2^32" in dsim.dsim_last_error()
    assert L.dsim_materialize_tables(C.byref(dsim.model_struct(ALL["tiny_mlp"].model)), None, 1 << 32, 10, 4,
                                     *([None] * 10)) == dsim.DSIM_ERANGE
    # argmin
    assert L.dsim_argmin(None, None, None, 0, 0, 0, None, 0, None, None, None, None) == dsim.DSIM_ERANGE
    assert L.dsim_argmin(None, None, None, 0, 0, 65, None, 0, None, None, None, None) == dsim.DSIM_ERANGE
    assert dsim.dsim_argmin_workspace(10, 0) == 0 and dsim.dsim_argmin_workspace(10 ** 6, 16) > 0
    # generator limits
    for nd in (1, 9):
        assert L.dsim_generate_random_tables(0, 10, 10, nd, *([None] * 7)) == dsim.DSIM_ERANGE
    assert L.dsim_generate_random_tables(0, 10, 1 << 27, 8, *([None] * 7)) == dsim.DSIM_ERANGE
    assert L.dsim_generate_random_tables(0, (1 << 32) - 255, 10, 8, *([None] * 7)) == dsim.DSIM_ERANGE
    assert L.dsim_generate_random_tables(0, 10, 10, 8, *([None] * 7)) == dsim.DSIM_EINVAL
    # parametric: bad model / NULL candidates
    m = dsim.model_struct(ALL["tiny_mlp"].model)
    m.family = 7
    assert L.dsim_simulate_parametric(C.byref(m), None, 1, C.byref(dev), C.byref(res), None, 0, None, None) == dsim.DSIM_EINVAL
    m = dsim.model_struct(ALL["gpt2_small"].model)
    m.d_model = 770
    assert L.dsim_simulate_parametric(C.byref(m), None, 1, C.byref(dev), C.byref(res), None, 0, None, None) == dsim.DSIM_EINVAL
    m = dsim.model_struct(ALL["gpt2_small"].model)
    assert L.dsim_simulate_parametric(C.byref(m), None, 1, C.byref(dev), C.byref(res), None, 0, None, None) == dsim.DSIM_EINVAL
    assert "NULL" in dsim.dsim_last_error()
    # device model: MatMul regression and network tier
    tab4 = dsim.dsim_tables()
    tab4.n_dev, tab4.max_ops = 4, 4
    for spec, word in ((DeviceSpec(matmul=(-1e-6, 0.0, 0.0)), "regression"),
                       (DeviceSpec(matmul=(0.0, float("inf"), 0.0)), "regression"),
                       (DeviceSpec(matmul=(0.0, 0.0, 0.0, -1e-9, 0.0)), "regression"),
                       (DeviceSpec(matmul=(0.0, 0.0, 0.0, 0.0, float("nan"))), "regression"),
                       (DeviceSpec(matmul=(0.0, 0.0, 0.0, float("inf"), 1e-5)), "regression"),
                       (DeviceSpec(network=(-1, 1e9, 0.0)), "node_size"),
                       (DeviceSpec(network=(8, 0.0, 1e-6)), "network"),
                       (DeviceSpec(network=(8, 1e9, float("nan"))), "network"),
                       (DeviceSpec(network=(8, 1e-310, 0.0)), "network"),
                       (DeviceSpec(streams=(2, 1e-310, 0.0)), "stream bandwidth"),
                       (DeviceSpec(streams=(-1, 1e9, 0.0)), "streams_per_gpu"),
                       (DeviceSpec(streams=(2, 0.0, 0.0)), "stream bandwidth"),
                       (DeviceSpec(streams=(2, float("nan"), 0.0)), "stream bandwidth"),
                       (DeviceSpec(streams=(3, 1e9, -1e-6)), "stream bandwidth"),
                       (DeviceSpec(streams=(2, float("inf"), float("inf"))), "stream bandwidth")):
        bad = dsim.device_model(spec)
        assert L.dsim_simulate_tables(C.byref(tab4), 10, C.byref(bad), C.byref(res), None) == dsim.DSIM_EINVAL
        assert word in dsim.dsim_last_error()
    bad = dsim.device_model(DeviceSpec())
    bad.mm_enabled = 2
    assert L.dsim_simulate_tables(C.byref(tab4), 10, C.byref(bad), C.byref(res), None) == dsim.DSIM_EINVAL
    for field, bad in (("schedule", 2), ("recompute", 2), ("recompute", -1), ("zero", 3), ("zero", -1),
                       ("overlap", 2), ("overlap", -1)):
        m = dsim.model_struct(ALL["gpt2_small_train"].model)
        setattr(m, field, bad)
        assert L.dsim_simulate_parametric(C.byref(m), None, 1, C.byref(dev), C.byref(res), None, 0, None, None) == dsim.DSIM_EINVAL
        assert field in dsim.dsim_last_error()
    m = dsim.model_struct(ALL["gpt2_small_train"].model)
    m.overlap, m.zero = 1, 1
    assert L.dsim_simulate_parametric(C.byref(m), None, 1, C.byref(dev), C.byref(res), None, 0, None, None) == dsim.DSIM_EINVAL
    assert "overlap and zero" in dsim.dsim_last_error()
    # the transform's devices per GPU must match the device model's streams
    two = dsim.device_model(DeviceSpec(streams=(2, 1e12, 1e-6)))
    three = dsim.device_model(DeviceSpec(streams=(3, 1e12, 1e-6)))
    m = dsim.model_struct(ALL["gpt2_small_train"].model)
    for mm, d in ((0, two), (1, dev), (1, three)):
        m.overlap = mm
        assert L.dsim_simulate_parametric(C.byref(m), None, 1, C.byref(d), C.byref(res), None, 0, None, None) == dsim.DSIM_EINVAL
        assert "streams_per_gpu" in dsim.dsim_last_error()
    m.overlap = 1
    assert L.dsim_simulate_parametric(C.byref(m), None, 1, C.byref(two), C.byref(res), None, 0, None, None) == dsim.DSIM_EINVAL
    assert "NULL" in dsim.dsim_last_error()
    # one dispatch of the transform covers n_cand * (widest segment) lanes
    m = dsim.model_struct(ALL["gpt3_175b"].model)
    res64 = dsim.dsim_results()
    res64.makespan = res64.cand_peak = res64.status = 8
    res64.row_width = 64
    fake = C.c_void_p(16)   # never dereferenced: the call fails before any launch
    assert L.dsim_simulate_parametric(C.byref(m), fake, 1 << 27, C.byref(dev), C.byref(res64), fake,
                                      dsim.dsim_parametric_workspace(1 << 27), None, None) == dsim.DSIM_ERANGE
    assert "dispatch" in dsim.dsim_last_error()
    # materialiser: device count, op capacity, NULL buffers, bad model
    m = dsim.model_struct(ALL["tiny_mlp"].model)
    for nd in (0, 9):
        assert L.dsim_materialize_tables(C.byref(m), None, 1, 10, nd, *([None] * 10)) == dsim.DSIM_ERANGE
    assert L.dsim_materialize_tables(C.byref(m), None, 1, -1, 4, *([None] * 10)) == dsim.DSIM_ERANGE
    assert L.dsim_materialize_tables(C.byref(m), None, 1, 10, 4, *([None] * 10)) == dsim.DSIM_EINVAL
    assert L.dsim_materialize_tables(C.byref(m), None, 0, 10, 4, *([None] * 10)) == dsim.DSIM_OK
    m.family = 7
    assert L.dsim_materialize_tables(C.byref(m), None, 1, 10, 4, *([None] * 10)) == dsim.DSIM_EINVAL


def _grid_rc(model):
    L = dsim.lib()
    m = dsim.model_struct(model)
    g = dsim.dsim_grid_spec(1, 0, 0, 1, 0)
    n = C.c_int64()
    return L.dsim_create_grid(C.byref(m), C.byref(g), None, 0, C.byref(n))


def test_size_rule_at_both_sides_of_the_bound(orc):
    """The size rule (dsim.h) on the host: the largest Gemm of a one-layer
    MLP at 2^61 flops is accepted, at 2^62 refused; a 65,537-layer model and
    a 2^20-token GPT-3-shaped sequence are refused; the oracle agrees."""
    d = 2 ** 20
    cases = [(mlp(1, d, 2 ** 20, 2, TRAIN_SGD), dsim.DSIM_OK), (mlp(1, d, 2 ** 21, 2, TRAIN_SGD), dsim.DSIM_ERANGE),
             (mlp(65536, 64, 64, 2, TRAIN_SGD), dsim.DSIM_OK), (mlp(65537, 64, 64, 2, TRAIN_SGD), dsim.DSIM_ERANGE),
             (transformer(96, 12288, 96, 2 ** 16, 50257, 1536, 2, INFER), dsim.DSIM_OK),
             (transformer(96, 12288, 96, 2 ** 20, 50257, 1536, 2, INFER), dsim.DSIM_ERANGE)]
    for model, want in cases:
        assert _grid_rc(model) == want, model
        assert orc.model_size_ok(model) == (want == dsim.DSIM_OK)
    assert "size rule" in (_grid_rc(cases[1][0]) and dsim.dsim_last_error())
    L = dsim.lib()
    dev = dsim.device_model(DeviceSpec())
    res = dsim.dsim_results()
    m = dsim.model_struct(cases[1][0])
    assert L.dsim_simulate_parametric(C.byref(m), None, 1, C.byref(dev), C.byref(res), None, 0, None, None) == dsim.DSIM_ERANGE
    assert L.dsim_materialize_tables(C.byref(m), None, 1, 10, 4, *([None] * 10)) == dsim.DSIM_ERANGE


def test_size_rule_matches_oracle_on_random_models(orc):
    rng = np.random.default_rng(7)
    for i in range(400):
        tf = i % 2 == 1
        mode = int(rng.integers(0, 4))
        e = int(rng.choice([1, 2, 4, 8]))
        L = int(2 ** rng.uniform(0, 16.5))
        B = int(2 ** rng.uniform(0, 40))
        if tf:
            a = int(2 ** rng.uniform(0, 10))
            d = a * int(2 ** rng.uniform(0, 14))
            model = transformer(L, d, a, int(2 ** rng.uniform(0, 22)), int(2 ** rng.uniform(1, 24)), B, e, mode,
                                d_ff=int(2 ** rng.uniform(0, 20)))
        else:
            model = mlp(L, int(2 ** rng.uniform(0, 26)), B, e, mode)
        ok = orc.model_size_ok(model)
        assert (_grid_rc(model) == dsim.DSIM_OK) == ok, model


def test_parametric_workspace_is_checked():
    """dsim_simulate_parametric takes its grouping buffer from the caller:
    about 12 bytes per candidate, DSIM_ENOSPC when it is missing or short
    (checked before any launch)."""
    L = dsim.lib()
    assert dsim.dsim_parametric_workspace(-1) == 0
    for n in (1, 255, 256, 257, 39965, 10 ** 6):
        nb = (n + 255) // 256
        assert dsim.dsim_parametric_workspace(n) == 4 * (8 * nb + 32 + 3 * n + 16)
    m = dsim.model_struct(ALL["gpt3_175b"].model)
    dev = dsim.device_model(DeviceSpec())
    res = dsim.dsim_results()
    res.makespan = res.cand_peak = res.status = 8
    res.row_width = 64
    fake = C.c_void_p(16)   # never dereferenced: the calls fail before any launch
    need = dsim.dsim_parametric_workspace(1000)
    for ws, nbytes in ((None, need), (fake, need - 1), (fake, 0)):
        assert L.dsim_simulate_parametric(C.byref(m), fake, 1000, C.byref(dev), C.byref(res), ws, nbytes, None,
                                          None) == dsim.DSIM_ENOSPC
        assert "workspace" in dsim.dsim_last_error()


def test_struct_layouts_match_header():
    """Every struct of include/dsim.h and its ctypes mirror in the binding:
    the same fields, in the same order, of the same C types."""
    import re
    with open(dsim.HEADER) as f:
        text = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
    ctypes_of = {"double": C.c_double, "float": C.c_float, "int32_t": C.c_int32, "int64_t": C.c_int64,
                 "uint32_t": C.c_uint32, "uint64_t": C.c_uint64}
    structs = re.findall(r"typedef struct\s*\{(.*?)\}\s*(dsim_\w+)\s*;", text, flags=re.S)
    assert {n for _, n in structs} >= {"dsim_device_model", "dsim_model", "dsim_strategy", "dsim_grid_spec"}
    for body, name in structs:
        fields = []
        for decl in body.split(";"):
            decl = decl.strip()
            if not decl:
                continue
            m = re.match(r"(const\s+)?(\w+)\s*(\*?)\s*(.*)$", decl)
            ctype, ptr, names = m.group(2), m.group(3), m.group(4)
            for nm in names.split(","):
                nm = nm.strip()
                star = ptr or nm.startswith("*")
                fields.append((nm.lstrip("*").strip(), "ptr" if star else ctype))
        mirror = getattr(dsim, name)
        got = [(f[0], f[1]) for f in mirror._fields_]
        assert [f[0] for f in got] == [f[0] for f in fields], name
        for (fname, ctype), (_, ct) in zip(fields, got):
            if ctype == "ptr":
                assert ct in (C.c_void_p,) or hasattr(ct, "_type_") and issubclass(ct, C._Pointer), (name, fname)
            else:
                assert ct is ctypes_of[ctype], (name, fname, ctype, ct)
