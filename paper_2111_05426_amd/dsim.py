"""Python binding of libdsim (include/dsim.h): argument marshalling only.

Every function carries the C entry point's name and forwards to it through
ctypes; all simulation work runs in the HIP kernels of libdsim.so.  PyTorch
supplies device memory and the HIP stream.  There is no fallback: if the
library is missing or a call fails, an exception is raised.
"""
import ctypes as C
import os
import re

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdsim.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "dsim.h")

DSIM_OK, DSIM_EINVAL, DSIM_ERANGE, DSIM_ENOSPC, DSIM_EHIP = 0, -1, -2, -3, -4
ST_BAD_OP, ST_BAD_DEVICE, ST_SELF_SEND, ST_MEM_UNDERFLOW, ST_BAD_STRATEGY, ST_OVER_CAP = 1, 2, 4, 8, 16, 32


class DsimError(RuntimeError):
    def __init__(self, fn, code, msg):
        super().__init__("%s failed (%d): %s" % (fn, code, msg))
        self.code = code


class dsim_device_model(C.Structure):
    _fields_ = [("flops_per_s", C.c_double), ("mem_bytes_per_s", C.c_double),
                ("link_bytes_per_s", C.c_double), ("link_latency_s", C.c_double),
                ("launch_s", C.c_double), ("mem_cap_bytes", C.c_uint64),
                ("mm_enabled", C.c_int32), ("mm_c0", C.c_double), ("mm_c1", C.c_double), ("mm_c2", C.c_double),
                ("node_size", C.c_int32), ("net_bytes_per_s", C.c_double), ("net_latency_s", C.c_double),
                ("streams_per_gpu", C.c_int32), ("stream_bytes_per_s", C.c_double),
                ("stream_latency_s", C.c_double), ("mm_c3", C.c_double), ("mm_floor", C.c_double)]


class dsim_model(C.Structure):
    _fields_ = [("family", C.c_int32), ("mode", C.c_int32), ("n_layers", C.c_int32),
                ("n_heads", C.c_int32), ("d_model", C.c_int64), ("d_ff", C.c_int64),
                ("seq_len", C.c_int64), ("vocab", C.c_int64), ("global_batch", C.c_int64),
                ("elem_bytes", C.c_int32), ("schedule", C.c_int32), ("recompute", C.c_int32),
                ("zero", C.c_int32), ("overlap", C.c_int32)]


class dsim_strategy(C.Structure):
    _fields_ = [("D", C.c_int32), ("H", C.c_int32), ("P", C.c_int32), ("K", C.c_int32)]


class dsim_grid_spec(C.Structure):
    _fields_ = [("max_devices", C.c_int32), ("exact_devices", C.c_int32), ("k_mode", C.c_int32),
                ("k_max", C.c_int32), ("require_k_divides", C.c_int32)]


class dsim_tables(C.Structure):
    _fields_ = [("code", C.c_void_p), ("flops", C.c_void_p), ("bytes", C.c_void_p),
                ("alloc_bytes", C.c_void_p), ("free_bytes", C.c_void_p), ("n_ops", C.c_void_p),
                ("init_live", C.c_void_p), ("max_ops", C.c_int32), ("n_dev", C.c_int32), ("mm_k", C.c_void_p)]


class dsim_results(C.Structure):
    _fields_ = [("makespan", C.c_void_p), ("finish", C.c_void_p), ("peak", C.c_void_p),
                ("cand_peak", C.c_void_p), ("n_ops", C.c_void_p), ("walked_ops", C.c_void_p),
                ("status", C.c_void_p), ("row_width", C.c_int32)]


_lib = None


def lib():
    """Load libdsim.so; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libdsim.so is not built (run python -m paper_2111_05426_amd.build)")
        L = C.CDLL(LIB_PATH)
        L.dsim_last_error.restype = C.c_char_p
        L.dsim_create_grid.argtypes = [C.POINTER(dsim_model), C.POINTER(dsim_grid_spec), C.c_void_p,
                                       C.c_int64, C.POINTER(C.c_int64)]
        L.dsim_simulate_tables.argtypes = [C.POINTER(dsim_tables), C.c_int64, C.POINTER(dsim_device_model),
                                           C.POINTER(dsim_results), C.c_void_p]
        L.dsim_parametric_workspace.restype = C.c_size_t
        L.dsim_parametric_workspace.argtypes = [C.c_int64]
        L.dsim_simulate_parametric.argtypes = [C.POINTER(dsim_model), C.c_void_p, C.c_int64,
                                               C.POINTER(dsim_device_model), C.POINTER(dsim_results),
                                               C.c_void_p, C.c_size_t, C.c_void_p, C.c_void_p]
        L.dsim_simulate_parametric_static.argtypes = [C.POINTER(dsim_model), C.c_void_p, C.c_int64,
                                                      C.POINTER(dsim_device_model), C.POINTER(dsim_results),
                                                      C.c_void_p]
        L.dsim_argmin_workspace.restype = C.c_size_t
        L.dsim_argmin_workspace.argtypes = [C.c_int64, C.c_int32]
        L.dsim_argmin.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.c_uint64, C.c_int32,
                                  C.c_void_p, C.c_size_t, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.dsim_generate_random_tables.argtypes = [C.c_uint64, C.c_int64, C.c_int32, C.c_int32] + \
            [C.c_void_p] * 7
        L.dsim_materialize_tables.argtypes = [C.POINTER(dsim_model), C.c_void_p, C.c_int64, C.c_int32,
                                              C.c_int32] + [C.c_void_p] * 10
        L.dsim_interpret_program.argtypes = [C.c_char_p, C.c_char_p, C.c_int32, C.c_void_p, C.c_size_t,
                                             C.POINTER(C.c_size_t)]
        L.dsim_lower_programs.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.c_int32, C.c_int32] + \
            [C.c_void_p] * 8 + [C.POINTER(C.c_int32), C.POINTER(C.c_int32), C.c_int32]
        for name in ("dsim_create_grid", "dsim_simulate_tables", "dsim_simulate_parametric",
                     "dsim_simulate_parametric_static", "dsim_argmin",
                     "dsim_generate_random_tables", "dsim_materialize_tables", "dsim_interpret_program",
                     "dsim_lower_programs"):
            getattr(L, name).restype = C.c_int
        _lib = L
    return _lib


def header_functions():
    """Names of the functions include/dsim.h declares."""
    with open(HEADER) as f:
        text = f.read()
    return re.findall(r"DSIM_API\s+[\w\s\*]*?\b(dsim_\w+)\s*\(", text)


def dsim_last_error():
    return lib().dsim_last_error().decode()


def _check(fn, rc):
    if rc != 0:
        raise DsimError(fn, rc, dsim_last_error())


def _ptr(t):
    """Device (or host) address of a tensor / ndarray, None for None."""
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


class _Args:
    """Checks the tensor arguments of one call before their addresses go to
    the library: each a contiguous torch tensor of one of the given dtypes
    with the given shape (None entries free) or element count; then, once
    all of them have passed, that every one lies on a GPU.  Raises
    ValueError: a mismatch would make a kernel read or write out of bounds."""

    def __init__(self):
        self.seen = []

    def tensor(self, name, t, dtypes, shape=None, numel=None, optional=False):
        if t is None:
            if optional:
                return
            raise ValueError("%s is required" % name)
        if not hasattr(t, "data_ptr") or not hasattr(t, "dtype"):
            raise ValueError("%s must be a torch tensor" % name)
        if t.dtype not in dtypes:
            raise ValueError("%s must be of dtype %s, not %s" % (name, " or ".join(str(d) for d in dtypes),
                                                                  t.dtype))
        if shape is not None:
            if t.dim() != len(shape) or any(w is not None and int(a) != int(w) for a, w in zip(t.shape, shape)):
                raise ValueError("%s must have shape %s, not %s" % (name, tuple(shape), tuple(t.shape)))
        if numel is not None and t.numel() < numel:
            raise ValueError("%s holds %d elements, needs %d" % (name, t.numel(), numel))
        if not t.is_contiguous():
            raise ValueError("%s must be contiguous" % name)
        self.seen.append((name, t))

    def results(self, results, n, row_width_min=1):
        for name in ("makespan", "cand_peak", "status"):
            if results.get(name) is None:
                raise ValueError("results[%r] is required" % name)
        self.tensor("results['makespan']", results["makespan"], _dt("float64"), shape=(n,))
        self.tensor("results['cand_peak']", results["cand_peak"], _dt("int64", "uint64"), shape=(n,))
        self.tensor("results['status']", results["status"], _dt("int32"), shape=(n,))
        for name in ("n_ops", "walked_ops"):
            self.tensor("results[%r]" % name, results.get(name), _dt("int64", "uint64"), shape=(n,), optional=True)
        if results.get("finish") is not None or results.get("peak") is not None:
            rw = int(results.get("row_width", 0))
            if rw < row_width_min:
                raise ValueError("results row_width %d must be >= %d" % (rw, row_width_min))
            self.tensor("results['finish']", results.get("finish"), _dt("float64"), shape=(n, rw), optional=True)
            self.tensor("results['peak']", results.get("peak"), _dt("int64", "uint64"), shape=(n, rw),
                        optional=True)

    def on_gpu(self):
        for name, t in self.seen:
            if t.device.type != "cuda":
                raise ValueError("%s must be a GPU tensor, not on %s" % (name, t.device))


def _dt(*names):
    import torch
    return tuple(getattr(torch, n) for n in names)


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def device_model(spec):
    """dsim_device_model of a DeviceSpec; its matmul is None, (c0, c1, c2) or
    (c0, c1, c2, c3, floor)."""
    mm = getattr(spec, "matmul", None)
    net = getattr(spec, "network", None)
    st = getattr(spec, "streams", None)
    mmv = tuple(float(v) for v in mm) if mm is not None else (0.0, 0.0, 0.0)
    if len(mmv) == 3:
        mmv = mmv + (0.0, 0.0)
    if len(mmv) != 5:
        raise ValueError("matmul must be (c0, c1, c2) or (c0, c1, c2, c3, floor)")
    return dsim_device_model(spec.flops_per_s, spec.mem_bytes_per_s, spec.link_bytes_per_s,
                             spec.link_latency_s, spec.launch_s, int(spec.mem_cap_bytes), 1 if mm is not None else 0,
                             *mmv[:3],
                             *((int(net[0]), float(net[1]), float(net[2])) if net is not None else (0, 0.0, 0.0)),
                             *((int(st[0]), float(st[1]), float(st[2])) if st is not None else (0, 0.0, 0.0)),
                             *mmv[3:])


def model_struct(spec):
    return dsim_model(spec.family, spec.mode, spec.n_layers, spec.n_heads, spec.d_model, spec.d_ff,
                      spec.seq_len, spec.vocab, spec.global_batch, spec.elem_bytes, spec.schedule,
                      spec.recompute, spec.zero, getattr(spec, "overlap", 0))


def dsim_create_grid(model, grid):
    """Host call: the valid strategies as an (n, 4) int32 array (D, H, P, K)."""
    m = model_struct(model)
    g = dsim_grid_spec(grid.max_devices, grid.exact_devices, grid.k_mode, grid.k_max, grid.require_k_divides)
    n = C.c_int64()
    _check("dsim_create_grid", lib().dsim_create_grid(C.byref(m), C.byref(g), None, 0, C.byref(n)))
    out = np.zeros((max(n.value, 1), 4), np.int32)
    _check("dsim_create_grid", lib().dsim_create_grid(C.byref(m), C.byref(g), out.ctypes.data, n.value,
                                                      C.byref(n)))
    return out[:n.value]


def alloc_results(n, row_width, device="cuda"):
    """Caller-owned output buffers (torch tensors)."""
    import torch
    return dict(makespan=torch.empty(n, dtype=torch.float64, device=device),
                finish=torch.empty((n, row_width), dtype=torch.float64, device=device),
                peak=torch.empty((n, row_width), dtype=torch.int64, device=device),
                cand_peak=torch.empty(n, dtype=torch.int64, device=device),
                n_ops=torch.empty(n, dtype=torch.int64, device=device),
                walked_ops=torch.empty(n, dtype=torch.int64, device=device),
                status=torch.empty(n, dtype=torch.int32, device=device),
                row_width=row_width)


def _results(r):
    return dsim_results(_ptr(r.get("makespan")), _ptr(r.get("finish")), _ptr(r.get("peak")),
                        _ptr(r.get("cand_peak")), _ptr(r.get("n_ops")), _ptr(r.get("walked_ops")),
                        _ptr(r.get("status")), int(r.get("row_width", 0)))


def alloc_tables(n_cand, max_ops, device="cuda", mm_k=False):
    import torch
    shape = (max_ops, n_cand)
    t = dict(code=torch.empty(shape, dtype=torch.int32, device=device),
             flops=torch.empty(shape, dtype=torch.float32, device=device),
             bytes=torch.empty(shape, dtype=torch.float32, device=device),
             alloc=torch.empty(shape, dtype=torch.int32, device=device),
             free=torch.empty(shape, dtype=torch.int32, device=device),
             n_ops=torch.empty(n_cand, dtype=torch.int32, device=device))
    if mm_k:
        t["mm_k"] = torch.empty(shape, dtype=torch.int32, device=device)
    return t


def dsim_simulate_tables(tables, n_cand, n_dev, device, results, init_live=None, stream=None):
    """tables: dict of device tensors shaped (max_ops, n_cand) (code/alloc/free
    as int32 bit patterns of the uint32 fields), optional n_ops (n_cand,) and
    mm_k (max_ops, n_cand); init_live: optional (n_cand, n_dev) int64."""
    n_cand = int(n_cand)
    a = _Args()
    a.tensor("tables['code']", tables.get("code"), _dt("int32", "uint32"), shape=(None, n_cand))
    max_ops = int(tables["code"].shape[0])
    for name, dts in (("flops", ("float32",)), ("bytes", ("float32",)), ("alloc", ("int32", "uint32")),
                      ("free", ("int32", "uint32"))):
        a.tensor("tables[%r]" % name, tables.get(name), _dt(*dts), shape=(max_ops, n_cand))
    a.tensor("tables['n_ops']", tables.get("n_ops"), _dt("int32", "uint32"), shape=(n_cand,), optional=True)
    a.tensor("tables['mm_k']", tables.get("mm_k"), _dt("int32", "uint32"), shape=(max_ops, n_cand), optional=True)
    a.tensor("init_live", init_live, _dt("int64", "uint64"), shape=(n_cand, int(n_dev)), optional=True)
    a.results(results, n_cand, int(n_dev))
    a.on_gpu()
    t = dsim_tables(_ptr(tables["code"]), _ptr(tables["flops"]), _ptr(tables["bytes"]), _ptr(tables["alloc"]),
                    _ptr(tables["free"]), _ptr(tables.get("n_ops")), _ptr(init_live), max_ops, n_dev,
                    _ptr(tables.get("mm_k")))
    d = device_model(device)
    r = _results(results)
    _check("dsim_simulate_tables",
           lib().dsim_simulate_tables(C.byref(t), n_cand, C.byref(d), C.byref(r), _stream(stream)))


def dsim_parametric_workspace(n_cand):
    return int(lib().dsim_parametric_workspace(int(n_cand)))


def alloc_parametric_workspace(n_cand, device="cuda"):
    """A caller-owned workspace for dsim_simulate_parametric (torch uint8)."""
    import torch
    return torch.empty(max(dsim_parametric_workspace(n_cand), 16), dtype=torch.uint8, device=device)


def dsim_simulate_parametric(model, cand, device, results, workspace=None, side_stream=None, stream=None):
    """cand: device int32 tensor (n, 4) of (D, H, P, K).  workspace: a device
    uint8 tensor of at least dsim_parametric_workspace(n) bytes (None: one
    is allocated with torch for this call).  side_stream: a second stream
    (torch.cuda.Stream or a raw handle) for the split launch of large
    transformer grids, or None."""
    a = _Args()
    a.tensor("cand", cand, _dt("int32"), shape=(None, 4))
    n = int(cand.shape[0])
    a.results(results, n)
    if workspace is None:
        workspace = alloc_parametric_workspace(n, device=cand.device)
    a.tensor("workspace", workspace, _dt("uint8"), numel=dsim_parametric_workspace(n))
    a.on_gpu()
    m = model_struct(model)
    d = device_model(device)
    r = _results(results)
    side = None if side_stream is None else getattr(side_stream, "cuda_stream", side_stream)
    _check("dsim_simulate_parametric",
           lib().dsim_simulate_parametric(C.byref(m), _ptr(cand), n, C.byref(d), C.byref(r), _ptr(workspace),
                                          workspace.numel(), side, _stream(stream)))


def dsim_simulate_parametric_static(model, cand, device, results, stream=None):
    """dsim_simulate_parametric with the library's fixed scratch (no
    allocation; at most 2^20 candidates; calls overlapping on one GPU race)."""
    a = _Args()
    a.tensor("cand", cand, _dt("int32"), shape=(None, 4))
    n = int(cand.shape[0])
    a.results(results, n)
    a.on_gpu()
    m = model_struct(model)
    d = device_model(device)
    r = _results(results)
    _check("dsim_simulate_parametric_static",
           lib().dsim_simulate_parametric_static(C.byref(m), _ptr(cand), n, C.byref(d), C.byref(r), _stream(stream)))


def dsim_argmin_workspace(n, k):
    return int(lib().dsim_argmin_workspace(n, k))


def dsim_argmin(makespan, cand_peak, status, mem_cap, k, workspace, out_idx, out_makespan, out_found,
                stream=None):
    a = _Args()
    a.tensor("makespan", makespan, _dt("float64"), shape=(None,))
    n = int(makespan.shape[0])
    a.tensor("cand_peak", cand_peak, _dt("int64", "uint64"), shape=(n,))
    a.tensor("status", status, _dt("int32"), shape=(n,))
    k = int(k)
    a.tensor("out_idx", out_idx, _dt("int64"), numel=k)
    a.tensor("out_makespan", out_makespan, _dt("float64"), numel=k)
    a.tensor("out_found", out_found, _dt("int32"), numel=1)
    a.tensor("workspace", workspace, _dt("uint8", "int8", "int32", "int64", "float32", "float64"))
    a.on_gpu()
    ws_bytes = workspace.numel() * workspace.element_size()
    _check("dsim_argmin",
           lib().dsim_argmin(_ptr(makespan), _ptr(cand_peak), _ptr(status), n, int(mem_cap), int(k),
                             _ptr(workspace), ws_bytes, _ptr(out_idx), _ptr(out_makespan), _ptr(out_found),
                             _stream(stream)))


def dsim_generate_random_tables(seed, n_cand, n_ops, n_dev, tables, stream=None):
    n_cand, n_ops = int(n_cand), int(n_ops)
    a = _Args()
    for name, dts in (("code", ("int32", "uint32")), ("flops", ("float32",)), ("bytes", ("float32",)),
                      ("alloc", ("int32", "uint32")), ("free", ("int32", "uint32"))):
        a.tensor("tables[%r]" % name, tables.get(name), _dt(*dts), shape=(n_ops, n_cand))
    a.tensor("tables['n_ops']", tables.get("n_ops"), _dt("int32", "uint32"), shape=(n_cand,), optional=True)
    a.on_gpu()
    _check("dsim_generate_random_tables",
           lib().dsim_generate_random_tables(seed, n_cand, n_ops, n_dev, _ptr(tables["code"]),
                                             _ptr(tables["flops"]), _ptr(tables["bytes"]),
                                             _ptr(tables["alloc"]), _ptr(tables["free"]),
                                             _ptr(tables.get("n_ops")), _stream(stream)))


def dsim_materialize_tables(model, cand, n_dev, max_ops, stream=None):
    """Explicit op tables of the whole distributed program of each strategy
    (device int32 tensor of shape (n, 4)); returns the tables dict (with
    init_live, shape (n, n_dev)) and the per-candidate status tensor."""
    import torch
    a = _Args()
    a.tensor("cand", cand, _dt("int32"), shape=(None, 4))
    a.on_gpu()
    n = int(cand.shape[0])
    t = alloc_tables(n, max_ops, device=cand.device, mm_k=True)
    t["init_live"] = torch.empty((n, n_dev), dtype=torch.int64, device=cand.device)
    status = torch.empty(n, dtype=torch.int32, device=cand.device)
    m = model_struct(model)
    _check("dsim_materialize_tables",
           lib().dsim_materialize_tables(C.byref(m), _ptr(cand), n, max_ops, n_dev, _ptr(t["code"]),
                                         _ptr(t["flops"]), _ptr(t["bytes"]), _ptr(t["alloc"]), _ptr(t["free"]),
                                         _ptr(t["mm_k"]), _ptr(t["n_ops"]), _ptr(t["init_live"]), _ptr(status),
                                         _stream(stream)))
    return t, status


def select_topk(makespan, cand_peak, status, mem_cap, k, stream=None):
    """Convenience: allocate workspace/outputs with torch, run dsim_argmin."""
    import torch
    dev = makespan.device
    n = int(makespan.shape[0])
    ws = torch.empty(max(dsim_argmin_workspace(n, k), 16), dtype=torch.uint8, device=dev)
    idx = torch.empty(k, dtype=torch.int64, device=dev)
    mk = torch.empty(k, dtype=torch.float64, device=dev)
    found = torch.empty(1, dtype=torch.int32, device=dev)
    dsim_argmin(makespan, cand_peak, status, mem_cap, k, ws, idx, mk, found, stream=stream)
    return idx, mk, found
