"""Python binding of the program front end of libdsim (include/dsim.h:
dsim_interpret_program, dsim_lower_programs): argument marshalling only.

The front end itself -- the parser, the mixed abstract/concrete interpreter
of Algorithm 1 (Sec. 3; Sec. 3.3 and the Reshape snippet of Fig. 4) and the
lowering to op tables -- is host C++ in the library (csrc/frontend.cpp).
Program text, one statement per line (`#` starts a comment):

    func NAME(%a: Tensor[Float32, (256, 8, 768), 0], %w: Tensor[Float32, (768, 64), 0] keep, %s: Int32)
    %t = OpType[attr = value, ...](%a, %b)
    %u, %v = Split[axis = 0, split = [2, 2]](%t)
    return %u

Types: `Tensor[DTYPE, (d0, ...), DEVICE]` (a shape of `??` is unknown) or a
scalar `DTYPE` / `DTYPE[DEVICE]`.  A parameter marked `keep` (weights) stays
resident for the whole program.  Inputs are a dict {parameter: value}: a
number, a (nested) list or an array gives the parameter a concrete value, a
type string (`"Tensor[Int32, (2,), 0]"`) an abstract one.

Every function raises ValueError (FrontEndError) where the library refuses
the program, with its message (line numbers included).
"""
import ctypes as C
import json

import numpy as np

from . import dsim

DSIM_ENOSPC = dsim.DSIM_ENOSPC


class FrontEndError(ValueError):
    def __init__(self, fn, code, msg):
        super().__init__("%s failed (%d): %s" % (fn, code, msg))
        self.code = code


def _fail(fn, rc):
    raise FrontEndError(fn, rc, dsim.dsim_last_error())


def inputs_text(inputs):
    """The library's inputs text for {name: value}: `%name = [..]` for a
    concrete value, `%name: TYPE` for a type string."""
    lines = []
    for name, v in (inputs or {}).items():
        if isinstance(v, str):
            lines.append("%s: %s" % (name, v))
        else:
            lines.append("%s = %s" % (name, json.dumps(np.asarray(v).tolist())))
    return "\n".join(lines)


def _value(text):
    """One VALUE of dsim_interpret_program's output: a concrete value as a
    Python number / nested list, an abstract one as its type string."""
    if text.startswith("Tensor[") or text[:1].isalpha() and text not in ("inf", "nan"):
        return text
    return json.loads(text.replace("nan", "NaN").replace("inf", "Infinity"))


def interpret(text, inputs=None, mixed=True):
    """The final state of the interpretation: {variable: value}, parameters
    first, then every op's results in program order (Algorithm 1); mixed=False
    is the abstract-only interpretation."""
    L = dsim.lib()
    prog, inp = text.encode(), inputs_text(inputs).encode()
    need = C.c_size_t(0)
    cap = 1 << 16
    while True:
        buf = C.create_string_buffer(cap)
        rc = L.dsim_interpret_program(prog, inp, 1 if mixed else 0, buf, cap, C.byref(need))
        if rc == DSIM_ENOSPC and need.value > cap:
            cap = need.value
            continue
        if rc != 0:
            _fail("dsim_interpret_program", rc)
        break
    state = {}
    for line in buf.value.decode().splitlines():
        name, val = line.split(" = ", 1)
        state[name] = _value(val)
    return state


def _lower(texts, inputs, n_dev, threads):
    """dsim_lower_programs over a list of program texts."""
    L = dsim.lib()
    n = len(texts)
    progs = (C.c_char_p * max(n, 1))(*[t.encode() for t in texts])
    if inputs is None:
        inp = None
    else:
        if len(inputs) != n:
            raise ValueError("%d inputs for %d programs" % (len(inputs), n))
        inp = (C.c_char_p * max(n, 1))(*[inputs_text(i).encode() for i in inputs])
    # statements bound the record count: one record at most per line
    max_ops = max([t.count("\n") + 1 for t in texts] + [1])
    out = dict(code=np.empty((max_ops, n), np.uint32), flops=np.empty((max_ops, n), np.float32),
               bytes=np.empty((max_ops, n), np.float32), alloc=np.empty((max_ops, n), np.uint32),
               free=np.empty((max_ops, n), np.uint32), mm_k=np.empty((max_ops, n), np.uint32),
               n_ops=np.empty(n, np.uint32), init_live=np.empty((n, n_dev), np.uint64))
    used, devs = C.c_int32(0), C.c_int32(0)
    rc = L.dsim_lower_programs(C.cast(progs, C.c_void_p), None if inp is None else C.cast(inp, C.c_void_p), n,
                               n_dev, max_ops, *(out[k].ctypes.data for k in
                                                 ("code", "flops", "bytes", "alloc", "free", "mm_k", "n_ops",
                                                  "init_live")),
                               C.byref(used), C.byref(devs), int(threads))
    if rc != 0:
        _fail("dsim_lower_programs", rc)
    m = used.value
    for k in ("code", "flops", "bytes", "alloc", "free", "mm_k"):
        out[k] = out[k][:m]
    return out, devs.value


def lower(text, inputs=None, n_dev=None):
    """One program interpreted (mixed) and lowered to its op table: dict(code,
    flops, bytes, alloc, free, mm_k, init_live, n_dev) of uint32 / float32 /
    uint64 arrays (mm_k: each record's reduction length, 0 but on matrix
    products).  n_dev None: the devices the program uses."""
    out, used = _lower([text], None if inputs is None else [inputs], 8 if n_dev is None else n_dev, 1)
    nd = used if n_dev is None else n_dev
    return dict(code=out["code"][:, 0].copy(), flops=out["flops"][:, 0].copy(), bytes=out["bytes"][:, 0].copy(),
                alloc=out["alloc"][:, 0].copy(), free=out["free"][:, 0].copy(), mm_k=out["mm_k"][:, 0].copy(),
                init_live=out["init_live"][0, :nd].copy(), n_dev=nd)


def lower_batch(texts, inputs=None, n_dev=8, threads=1):
    """Many programs lowered into one set of candidate-fastest tables, the
    dsim_tables layout: arrays (max_ops, n_prog) plus n_ops (n_prog,) and
    init_live (n_prog, n_dev).  inputs: None or one dict per program."""
    out, _ = _lower(list(texts), inputs, n_dev, threads)
    out["n_dev"] = n_dev
    return out


def pack(tables):
    """Candidate-fastest arrays (max_ops, n_cand) of several lowered tables
    (one n_dev for all), with n_ops and init_live (n_cand, n_dev)."""
    nd = max(t["n_dev"] for t in tables)
    n = len(tables)
    m = max([len(t["code"]) for t in tables] + [1])
    out = dict(code=np.zeros((m, n), np.uint32), flops=np.zeros((m, n), np.float32),
               bytes=np.zeros((m, n), np.float32), alloc=np.zeros((m, n), np.uint32),
               free=np.zeros((m, n), np.uint32), mm_k=np.zeros((m, n), np.uint32), n_ops=np.zeros(n, np.uint32),
               init_live=np.zeros((n, nd), np.uint64), n_dev=nd)
    for c, t in enumerate(tables):
        k = len(t["code"])
        for f in ("code", "flops", "bytes", "alloc", "free", "mm_k"):
            if t.get(f) is not None:
                out[f][:k, c] = t[f]
        out["n_ops"][c] = k
        out["init_live"][c, :t["n_dev"]] = t["init_live"]
    return out
