"""ctypes wrapper around the reference CPU simulator in dsim_oracle.c.

TEST INFRASTRUCTURE ONLY: tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg are the only callers.  The product path
(paper_2111_05426_amd) never imports this package.
"""
import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "dsim_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

# status bits
ST_BAD_OP, ST_BAD_DEVICE, ST_SELF_SEND, ST_MEM_UNDERFLOW, ST_BAD_STRATEGY, ST_OVER_CAP = 1, 2, 4, 8, 16, 32
COMPUTE, SEND, ALLREDUCE, BCAST, REDUCE = 0, 1, 2, 3, 4
TF_RESIDENT, TF_KEEP = 1, 2

# op type tags (same order as the enum in dsim_oracle.c)
TYPES = ["SPLIT", "GEMM", "RELU", "AR_TP", "LOSSGRAD", "RELUGRAD", "GEMMDW", "ADDGRAD",
         "GEMMDX", "SEND_F", "SEND_B", "AR_DP", "OPT",
         "LN", "QKV", "SCORES", "SOFTMAX", "AV", "OUTPROJ", "RESADD", "FC1", "GELU", "FC2",
         "EMBED", "LMHEAD", "XENT_STATS", "XENT_GRAD", "LN_B", "RESADD_B", "GELU_B", "AV_B",
         "SOFTMAX_B", "SCORES_B", "EMBED_DW", "BCAST", "REDUCE", "STREAM", "GENERIC"]
T = {name: i for i, name in enumerate(TYPES)}
N_TYPES = len(TYPES)


def build(force=True):
    """Compile the oracle with gcc (-O2, no FMA contraction, no fast-math)."""
    if not force and os.path.exists(LIB) and os.path.getmtime(LIB) >= os.path.getmtime(SRC):
        return LIB
    tmp = LIB + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c99",
                           "-Wall", "-shared", "-fPIC", "-o", tmp, SRC, "-lpthread", "-lm"])
    os.replace(tmp, LIB)
    return LIB


class _Dev(C.Structure):
    _fields_ = [("flops_per_s", C.c_double), ("mem_bytes_per_s", C.c_double),
                ("link_bytes_per_s", C.c_double), ("link_latency_s", C.c_double),
                ("launch_s", C.c_double), ("mem_cap_bytes", C.c_uint64),
                ("mm_enabled", C.c_int32), ("mm_c0", C.c_double), ("mm_c1", C.c_double), ("mm_c2", C.c_double),
                ("node_size", C.c_int32), ("net_bytes_per_s", C.c_double), ("net_latency_s", C.c_double),
                ("streams_per_gpu", C.c_int32), ("stream_bytes_per_s", C.c_double),
                ("stream_latency_s", C.c_double), ("mm_c3", C.c_double), ("mm_floor", C.c_double)]


class _Model(C.Structure):
    _fields_ = [("family", C.c_int32), ("mode", C.c_int32), ("n_layers", C.c_int32),
                ("n_heads", C.c_int32), ("d_model", C.c_int64), ("d_ff", C.c_int64),
                ("seq_len", C.c_int64), ("vocab", C.c_int64), ("global_batch", C.c_int64),
                ("elem_bytes", C.c_int32), ("schedule", C.c_int32), ("recompute", C.c_int32),
                ("zero", C.c_int32), ("overlap", C.c_int32)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        _lib = C.CDLL(LIB)
    return _lib


def _dev(d):
    """The device model: matmul is None, (c0, c1, c2) -- the linear form --
    or (c0, c1, c2, c3, floor)."""
    mm = getattr(d, "matmul", None)
    net = getattr(d, "network", None)
    st = getattr(d, "streams", None)
    mmv = tuple(float(v) for v in mm) if mm is not None else (0.0, 0.0, 0.0)
    if len(mmv) == 3:
        mmv = mmv + (0.0, 0.0)
    if len(mmv) != 5:
        raise ValueError("matmul must be (c0, c1, c2) or (c0, c1, c2, c3, floor)")
    return _Dev(d.flops_per_s, d.mem_bytes_per_s, d.link_bytes_per_s, d.link_latency_s,
                d.launch_s, int(d.mem_cap_bytes), 1 if mm is not None else 0, *mmv[:3],
                *((int(net[0]), float(net[1]), float(net[2])) if net is not None else (0, 0.0, 0.0)),
                *((int(st[0]), float(st[1]), float(st[2])) if st is not None else (0, 0.0, 0.0)),
                *mmv[3:])


def _model(m):
    return _Model(m.family, m.mode, m.n_layers, m.n_heads, m.d_model, m.d_ff, m.seq_len,
                  m.vocab, m.global_batch, m.elem_bytes, getattr(m, "schedule", 0),
                  getattr(m, "recompute", 0), getattr(m, "zero", 0), getattr(m, "overlap", 0))


def _p(a):
    return a.ctypes.data_as(C.c_void_p) if a is not None else None


def cost(dev, kind, flops, nbytes, n, type=None, k=0.0):
    """Cost of one op; with an op type name (TYPES), matrix multiplications
    (reduction length k) take the device's empirical MatMul regression when
    it has one."""
    d = _dev(dev)
    if type is None:
        f = lib().or_cost
        f.restype = C.c_double
        f.argtypes = [C.POINTER(_Dev), C.c_int, C.c_double, C.c_double, C.c_int]
        return f(C.byref(d), kind, float(flops), float(nbytes), int(n))
    f = lib().or_cost_typed
    f.restype = C.c_double
    f.argtypes = [C.POINTER(_Dev), C.c_int, C.c_int, C.c_double, C.c_double, C.c_double, C.c_int, C.c_int]
    return f(C.byref(d), kind, TYPES.index(type), float(flops), float(nbytes), float(k), int(n), 0)


def cost_between_nodes(dev, kind, nbytes, n):
    """Cost of a communication op whose devices lie in more than one node."""
    d = _dev(dev)
    f = lib().or_cost_spans
    f.restype = C.c_double
    f.argtypes = [C.POINTER(_Dev), C.c_int, C.c_double, C.c_double, C.c_int, C.c_int]
    return f(C.byref(d), kind, 0.0, float(nbytes), int(n), 1)


def cost_on_one_gpu(dev, kind, nbytes, n):
    """Cost of a communication op whose devices are streams of one GPU."""
    d = _dev(dev)
    f = lib().or_cost_spans
    f.restype = C.c_double
    f.argtypes = [C.POINTER(_Dev), C.c_int, C.c_double, C.c_double, C.c_int, C.c_int]
    return f(C.byref(d), kind, 0.0, float(nbytes), int(n), 2)


def gen_table(seed, cand, n_ops, n_dev):
    code = np.zeros(n_ops, np.uint32)
    fl = np.zeros(n_ops, np.float32)
    by = np.zeros(n_ops, np.float32)
    al = np.zeros(n_ops, np.uint32)
    fr = np.zeros(n_ops, np.uint32)
    f = lib().or_gen_table
    f.argtypes = [C.c_uint64, C.c_int64, C.c_int32, C.c_int32] + [C.c_void_p] * 5 + [C.c_int64]
    rc = f(seed, cand, n_ops, n_dev, _p(code), _p(fl), _p(by), _p(al), _p(fr), 1)
    if rc:
        raise ValueError("or_gen_table failed: %d" % rc)
    return dict(code=code, flops=fl, bytes=by, alloc=al, free=fr)


def sim_table(tab, n_dev, dev, init_live=None):
    """Simulate one candidate's explicit table (dict of equal-length arrays)."""
    n = len(tab["code"])
    arr = {k: np.ascontiguousarray(tab[k]) for k in ("code", "flops", "bytes", "alloc", "free")}
    mmk = None if tab.get("mm_k") is None else np.ascontiguousarray(tab["mm_k"], np.uint32)
    fin = np.zeros(n_dev, np.float64)
    pk = np.zeros(n_dev, np.uint64)
    mk = C.c_double()
    cp = C.c_uint64()
    st = C.c_int32()
    il = None if init_live is None else np.ascontiguousarray(init_live, np.uint64)
    f = lib().or_sim_table
    f.argtypes = [C.c_int64, C.c_int] + [C.c_void_p] * 6 + [C.c_int64, C.c_void_p, C.POINTER(_Dev),
                                                            C.POINTER(C.c_double), C.c_void_p, C.c_void_p,
                                                            C.POINTER(C.c_uint64), C.POINTER(C.c_int32)]
    d = _dev(dev)
    rc = f(n, n_dev, _p(arr["code"]), _p(arr["flops"]), _p(arr["bytes"]), _p(arr["alloc"]),
           _p(arr["free"]), _p(mmk), 1, _p(il), C.byref(d), C.byref(mk), _p(fin), _p(pk), C.byref(cp), C.byref(st))
    if rc:
        raise ValueError("or_sim_table failed: %d" % rc)
    return dict(makespan=mk.value, finish=fin, peak=pk, cand_peak=cp.value, status=st.value)


def sim_program(ops, tensors, n_dev, dev, with_trace=False):
    """Simulate an explicit program.

    ops: list of dicts {kind, devs, ins, outs, cost (optional), flops, bytes,
         matmul (optional: the empirical MatMul cost applies), k (optional:
         the product's reduction length)}
    tensors: list of (device, size, flags)
    dev: object with the device-model attributes (flops_per_s, ...)
    """
    n = len(ops)
    kind = np.array([o.get("kind", COMPUTE) for o in ops], np.int32)
    cost_ = np.array([o.get("cost", -1.0) for o in ops], np.float64)
    fl = np.array([o.get("flops", 0.0) for o in ops], np.float64)
    by = np.array([o.get("bytes", 0.0) for o in ops], np.float64)

    def csr(key):
        beg = np.zeros(n + 1, np.int64)
        flat = []
        for i, o in enumerate(ops):
            flat.extend(o.get(key, []))
            beg[i + 1] = len(flat)
        return beg, np.array(flat if flat else [0], np.int32)

    db, dv = csr("devs")
    ib, iv = csr("ins")
    ob, ov = csr("outs")
    t_dev = np.array([t[0] for t in tensors] or [0], np.int32)
    t_size = np.array([t[1] for t in tensors] or [0], np.uint64)
    t_flags = np.array([t[2] for t in tensors] or [0], np.int32)
    mm = np.array([1 if o.get("matmul") else 0 for o in ops] or [0], np.int32)
    mmk = np.array([float(o.get("k", 0.0)) for o in ops] or [0.0], np.float64)
    fin = np.zeros(n_dev, np.float64)
    pk = np.zeros(n_dev, np.uint64)
    ts = np.zeros(max(n, 1), np.float64)
    te = np.zeros(max(n, 1), np.float64)
    f = lib().or_sim_program
    f.argtypes = [C.c_int64] + [C.c_void_p] * 10 + [C.c_int64] + [C.c_void_p] * 3 + \
        [C.c_int, C.POINTER(_Dev)] + [C.c_void_p] * 6
    d = _dev(dev)
    rc = f(n, _p(kind), _p(cost_), _p(fl), _p(by), _p(db), _p(dv), _p(ib), _p(iv), _p(ob), _p(ov),
           len(tensors), _p(t_dev), _p(t_size), _p(t_flags), n_dev, C.byref(d), _p(fin), _p(pk),
           _p(ts), _p(te), _p(mm), _p(mmk))
    if rc:
        raise ValueError("or_sim_program failed: %d" % rc)
    out = dict(finish=fin, peak=pk, makespan=float(fin.max()) if n_dev else 0.0)
    if with_trace:
        out["start"] = ts[:n]
        out["end"] = te[:n]
    return out


def sim_strategy(model, D, H, P, K, dev, slice=False, type_cost=None, want_devices=True):
    """Materialise (D,H,P,K) on the model and simulate it.  Returns a dict.
    With overlap every GPU has two devices (streams): 2g computes, 2g + 1
    communicates."""
    n_dev = (2 if getattr(model, "overlap", 0) else 1) * D * H * P
    sf = np.zeros(P, np.float64)
    sp = np.zeros(P, np.uint64)
    df = np.zeros(n_dev, np.float64) if want_devices else None
    dp = np.zeros(n_dev, np.uint64) if want_devices else None
    dr = np.zeros(n_dev, np.uint64) if want_devices else None
    fbt = np.zeros(3 * N_TYPES, np.float64)
    tc = None
    if type_cost is not None:
        tc = np.full(N_TYPES, -1.0)
        for k, v in type_cost.items():
            tc[T[k]] = v
    mk = C.c_double()
    cp = C.c_uint64()
    no = C.c_uint64()
    st = C.c_int32()
    f = lib().or_sim_strategy
    f.argtypes = [C.POINTER(_Model), C.c_int, C.c_int, C.c_int, C.c_int, C.POINTER(_Dev), C.c_int,
                  C.c_void_p] + [C.c_void_p] * 6 + [C.POINTER(C.c_double), C.POINTER(C.c_uint64),
                                                    C.POINTER(C.c_uint64), C.POINTER(C.c_int32)]
    m = _model(model)
    d = _dev(dev)
    rc = f(C.byref(m), D, H, P, K, C.byref(d), int(bool(slice)), _p(tc), _p(sf), _p(sp), _p(df), _p(dp),
           _p(dr), _p(fbt), C.byref(mk), C.byref(cp), C.byref(no), C.byref(st))
    if rc:
        raise ValueError("or_sim_strategy failed: %d" % rc)
    return dict(makespan=mk.value, cand_peak=cp.value, n_ops=no.value, status=st.value,
                stage_finish=sf, stage_peak=sp, dev_finish=df, dev_peak=dp, dev_resident=dr,
                flops_by_type={TYPES[i]: fbt[i] for i in range(N_TYPES)},
                bytes_by_type={TYPES[i]: fbt[N_TYPES + i] for i in range(N_TYPES)},
                k_by_type={TYPES[i]: fbt[2 * N_TYPES + i] for i in range(N_TYPES)})


def model_size_ok(model):
    """Whether the model is within the size rule of the transform's integer
    arithmetic (or_model_size_ok)."""
    f = lib().or_model_size_ok
    f.restype = C.c_int
    f.argtypes = [C.POINTER(_Model)]
    m = _model(model)
    return bool(f(C.byref(m)))


def create_grid(model, grid):
    f = lib().or_create_grid
    f.argtypes = [C.POINTER(_Model), C.c_int, C.c_int, C.c_int, C.c_int, C.c_int, C.c_void_p,
                  C.c_int64, C.POINTER(C.c_int64)]
    m = _model(model)
    n = C.c_int64()
    rc = f(C.byref(m), grid.max_devices, grid.exact_devices, grid.k_mode, grid.k_max,
           grid.require_k_divides, None, 0, C.byref(n))
    if rc:
        raise ValueError("or_create_grid failed: %d" % rc)
    out = np.zeros((max(n.value, 1), 4), np.int32)
    rc = f(C.byref(m), grid.max_devices, grid.exact_devices, grid.k_mode, grid.k_max,
           grid.require_k_divides, _p(out), n.value, C.byref(n))
    if rc:
        raise ValueError("or_create_grid failed: %d" % rc)
    return out[:n.value]


def topk(makespan, cand_peak, status, cap, k):
    mk = np.ascontiguousarray(makespan, np.float64)
    pk = np.ascontiguousarray(cand_peak, np.uint64)
    st = np.ascontiguousarray(status, np.int32)
    idx = np.zeros(k, np.int64)
    mo = np.zeros(k, np.float64)
    found = C.c_int32()
    f = lib().or_topk
    f.argtypes = [C.c_void_p] * 3 + [C.c_int64, C.c_uint64, C.c_int, C.c_void_p, C.c_void_p,
                                     C.POINTER(C.c_int32)]
    rc = f(_p(mk), _p(pk), _p(st), len(mk), int(cap), int(k), _p(idx), _p(mo), C.byref(found))
    if rc:
        raise ValueError("or_topk failed: %d" % rc)
    return idx, mo, found.value


def run_random_tables(seed, n_ops, n_dev, cands, dev, threads=1, want_rows=True):
    cands = np.ascontiguousarray(cands, np.int64)
    n = len(cands)
    mk = np.zeros(n, np.float64)
    fin = np.zeros(n * n_dev, np.float64) if want_rows else None
    pk = np.zeros(n * n_dev, np.uint64) if want_rows else None
    cp = np.zeros(n, np.uint64)
    no = np.zeros(n, np.uint64)
    st = np.zeros(n, np.int32)
    f = lib().or_run_random_tables
    f.argtypes = [C.c_uint64, C.c_int32, C.c_int32, C.c_void_p, C.c_int64, C.POINTER(_Dev), C.c_int] + \
        [C.c_void_p] * 6
    d = _dev(dev)
    rc = f(seed, n_ops, n_dev, _p(cands), n, C.byref(d), threads, _p(mk), _p(fin), _p(pk), _p(cp),
           _p(no), _p(st))
    if rc:
        raise ValueError("or_run_random_tables failed: %d" % rc)
    out = dict(makespan=mk, cand_peak=cp, n_ops=no, status=st)
    if want_rows:
        out["finish"] = fin.reshape(n, n_dev)
        out["peak"] = pk.reshape(n, n_dev)
    return out


def run_strategies(model, strat, dev, slice=False, row_width=None, threads=1):
    strat = np.ascontiguousarray(strat, np.int32).reshape(-1, 4)
    n = len(strat)
    rw = int(row_width or (strat[:, 2].max() if n else 1))
    mk = np.zeros(n, np.float64)
    fin = np.zeros(n * rw, np.float64)
    pk = np.zeros(n * rw, np.uint64)
    cp = np.zeros(n, np.uint64)
    no = np.zeros(n, np.uint64)
    st = np.zeros(n, np.int32)
    f = lib().or_run_strategies
    f.argtypes = [C.POINTER(_Model), C.c_void_p, C.c_int64, C.POINTER(_Dev), C.c_int, C.c_int, C.c_int] + \
        [C.c_void_p] * 6
    m = _model(model)
    d = _dev(dev)
    rc = f(C.byref(m), _p(strat), n, C.byref(d), int(bool(slice)), rw, threads, _p(mk), _p(fin), _p(pk),
           _p(cp), _p(no), _p(st))
    if rc:
        raise ValueError("or_run_strategies failed: %d" % rc)
    return dict(makespan=mk, finish=fin.reshape(n, rw), peak=pk.reshape(n, rw), cand_peak=cp,
                n_ops=no, status=st)
