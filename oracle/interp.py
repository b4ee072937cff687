"""Plain reference interpreter for the program front end.

TEST INFRASTRUCTURE ONLY (tests/ are the only callers).  It shares no code
with paper_2111_05426_amd/frontend.py: it parses the same program text with
its own code, runs Algorithm 1 (Sec. 3) -- op by op over a state mapping
variables to values -- with one branch per op type written out, and turns
the result into an explicit program over tensors (ops with devices, inputs
and outputs; tensors with a device and a size) for the oracle's program
simulator (def/use liveness, Sec. 3.3), instead of table records.

Values: a concrete value is a numpy array; an abstract tensor is
('T', dtype, shape or None, device); an abstract scalar is ('S', dtype,
device).  In the mixed interpretation (Sec. 3.3) an op whose arguments are
all concrete is evaluated concretely, Shape of an abstract tensor of known
shape is concrete, Reshape of an abstract tensor by a concrete target has a
known shape; in the abstract-only interpretation every concrete value is
replaced by its type as soon as it appears.

Readings shared with the front end (the paper leaves them open): shape
arithmetic is typed Int32; an op yielding no abstract tensor runs on the
host and is not part of the simulated program; Reshape, Unsqueeze,
Squeeze, Flatten and Identity are views of their input's memory; AllReduce
works in place, and a tensor whose last reader is an AllReduce stays live
to the end; a parameter marked keep is never freed.  Costs: elementwise ops
1 flop per output element (Gelu 8, Softmax 5, LayerNormalization 8, Cast 0),
MatMul 2 * (output elements) * k, Gemm the same plus one per output element
with a bias (k, the reduction length, also enters the empirical MatMul
cost), Transpose / Concat / Split / Gather no flops; bytes = every abstract
input and output tensor's size; Send and AllReduce move one input's bytes.
"""
import re

import numpy as np

import oracle

SIZE = {"Float64": 8, "Float32": 4, "Float16": 2, "BFloat16": 2, "Int64": 8, "Int32": 4, "Int8": 1, "Bool": 1}
VIEW_OPS = ("Reshape", "Unsqueeze", "Squeeze", "Flatten", "Identity")


def is_t(v):
    return isinstance(v, tuple) and v[0] == "T"


def is_s(v):
    return isinstance(v, tuple) and v[0] == "S"


def is_c(v):
    return isinstance(v, np.ndarray)


def n_elems(shape):
    n = 1
    for d in shape:
        n *= int(d)
    return n


def tbytes(v):
    if v[2] is None:
        raise ValueError("unknown shape")
    return n_elems(v[2]) * SIZE[v[1]]


def as_type(v, dev=None):
    """The type of a concrete value."""
    if not is_c(v):
        return v
    dt = "Float64" if v.dtype.kind == "f" else "Int32"
    if v.ndim == 0:
        return ("S", dt, dev)
    return ("T", dt, tuple(int(d) for d in v.shape), dev)


# ---------------------------------------------------------------------------
# Parsing
# ---------------------------------------------------------------------------
def literal(text):
    text = text.strip()
    if text.startswith("["):
        inner = text[1:-1].strip()
        return [literal(x) for x in split_commas(inner)] if inner else []
    if text.startswith("'") or text.startswith('"'):
        return text[1:-1]
    try:
        return int(text)
    except ValueError:
        return float(text)


def split_commas(text):
    out, depth, start = [], 0, 0
    for i, ch in enumerate(text):
        if ch in "([":
            depth += 1
        elif ch in ")]":
            depth -= 1
        elif ch == "," and depth == 0:
            out.append(text[start:i].strip())
            start = i + 1
    rest = text[start:].strip()
    if rest:
        out.append(rest)
    return out


def read_type(text):
    text = text.strip()
    if text.startswith("Tensor["):
        body = split_commas(text[len("Tensor["):-1])
        dt, shp, dev = body[0], body[1], int(body[2])
        if shp == "??":
            shape = None
        else:
            dims = [d for d in split_commas(shp.strip()[1:-1]) if d]
            shape = tuple(int(d) for d in dims)
        return ("T", dt, shape, dev)
    m = re.fullmatch(r"(\w+)(\[(-?\d+)\])?", text)
    return ("S", m.group(1), int(m.group(3)) if m.group(3) else None)


def read_program(text):
    params, ops = [], []
    for line in text.splitlines():
        line = line.split("#")[0].strip()
        if not line or line.startswith("return"):
            continue
        if line.startswith("func"):
            inner = line[line.index("(") + 1:line.rindex(")")]
            for p in split_commas(inner):
                name, typ = p.split(":", 1)
                typ = typ.strip()
                keep = typ.endswith("keep")
                if keep:
                    typ = typ[:-4].strip()
                params.append((name.strip(), read_type(typ), keep))
            continue
        lhs, rhs = line.split("=", 1)
        outs = [o.strip() for o in lhs.split(",")]
        rhs = rhs.strip()
        name = re.match(r"\w+", rhs).group(0)
        rest = rhs[len(name):].strip()
        attrs = {}
        if rest.startswith("["):
            depth = 0
            for i, ch in enumerate(rest):
                depth += ch == "["
                depth -= ch == "]"
                if depth == 0:
                    break
            for item in split_commas(rest[1:i]):
                k, v = item.split("=", 1)
                attrs[k.strip()] = literal(v)
            rest = rest[i + 1:].strip()
        args = [a for a in split_commas(rest[1:-1])]
        ops.append((outs, name, attrs, args))
    return params, ops


# ---------------------------------------------------------------------------
# Algorithm 1
# ---------------------------------------------------------------------------
def one_device(vals):
    devs = set()
    for v in vals:
        if is_t(v) and v[3] is not None:
            devs.add(v[3])
        if is_s(v) and v[2] is not None:
            devs.add(v[2])
    if len(devs) > 1:
        raise ValueError("inputs on several devices")
    return devs.pop() if devs else None


def resolve(shape, target):
    out = []
    for i, t in enumerate(int(x) for x in target):
        out.append(shape[i] if t == 0 else t)
    if -1 in out:
        rest = n_elems([d for d in out if d != -1])
        out[out.index(-1)] = n_elems(shape) // rest
    return tuple(out)


def run_op(name, attrs, a):
    """Results of one op on argument values a (mixed domain)."""
    if name == "Constant":
        v = np.array(attrs["value"])
        return [v.astype(np.int64) if v.dtype.kind in "iub" else v.astype(np.float64)]
    if all(is_c(x) for x in a):
        # every argument concrete: evaluate
        if name == "Shape":
            return [np.array(a[0].shape, np.int64)]
        if name == "Gather":
            return [np.array(np.take(a[0], a[1], axis=attrs.get("axis", 0)))]
        if name == "Unsqueeze":
            r = a[0]
            for ax in sorted(attrs["axes"]):
                r = np.expand_dims(r, ax)
            return [r]
        if name == "Squeeze":
            return [np.squeeze(a[0], axis=tuple(attrs["axes"]))]
        if name == "Concat":
            return [np.concatenate([np.atleast_1d(x) for x in a], axis=attrs.get("axis", 0))]
        if name == "Reshape":
            return [a[0].reshape(resolve(a[0].shape, a[1]))]
        if name in ("Add", "Sub", "Mul", "Pow"):
            f = {"Add": np.add, "Sub": np.subtract, "Mul": np.multiply, "Pow": np.power}[name]
            return [np.array(f(a[0], a[1]))]
        if name == "Div":
            return [np.array(np.divide(a[0], a[1]))]
        if name == "Cast":
            return [a[0].astype(np.float64 if attrs["to"].startswith("Float") else np.int64)]
        if name == "Relu":
            return [np.maximum(a[0], 0)]
        if name in ("Neg", "Sqrt", "Exp", "Tanh", "Identity"):
            f = {"Neg": np.negative, "Sqrt": np.sqrt, "Exp": np.exp, "Tanh": np.tanh, "Identity": np.array}[name]
            return [np.array(f(a[0]))]
    if name == "Shape":
        x = a[0]
        return [np.array(x[2], np.int64)] if x[2] is not None else [("T", "Int32", None, x[3])]
    if name == "Reshape":
        x, tgt = a
        if is_c(tgt) and x[2] is not None:
            return [("T", x[1], resolve(x[2], tgt), x[3])]
        return [("T", x[1], None, x[3])]
    av = [as_type(x) for x in a]
    if name == "Send":
        x = av[0]
        return [("T", x[1], x[2], attrs["device"])]
    if name == "AllReduce":
        if len({x[3] for x in av}) != len(av):
            raise ValueError("AllReduce inputs must lie on distinct devices")
        return list(av)
    dev = one_device(av)
    if name == "Gather":
        data, idx = av
        if is_t(data) and data[2] is not None and len(data[2]) == 1 and (is_s(idx) or (is_c(a[1]) and a[1].ndim == 0)):
            return [("S", data[1], dev)]
        ishape = () if is_s(idx) else idx[2]
        ax = attrs.get("axis", 0)
        if data[2] is None or ishape is None:
            return [("T", data[1], None, dev)]
        return [("T", data[1], data[2][:ax] + tuple(ishape) + data[2][ax + 1:], dev)]
    if name == "Unsqueeze":
        x = av[0]
        shp = [] if is_s(x) else (None if x[2] is None else list(x[2]))
        if shp is not None:
            for ax in sorted(attrs["axes"]):
                shp.insert(ax if ax >= 0 else ax + len(shp) + 1, 1)
        return [("T", x[1], None if shp is None else tuple(shp), dev)]
    if name == "Squeeze":
        x = av[0]
        if x[2] is None:
            return [x]
        drop = [ax % len(x[2]) for ax in attrs["axes"]]
        return [("T", x[1], tuple(d for i, d in enumerate(x[2]) if i not in drop), x[3])]
    if name == "Concat":
        if any(is_s(x) or x[2] is None for x in av):
            return [("T", av[0][1], None, dev)]
        ax = attrs.get("axis", 0)
        shp = list(av[0][2])
        shp[ax] = sum(x[2][ax] for x in av)
        return [("T", av[0][1], tuple(shp), dev)]
    if name in ("Add", "Sub", "Mul", "Div", "Pow"):
        if is_s(av[0]) and is_s(av[1]):
            return [("S", av[0][1], dev)]
        shapes = [() if is_s(x) else x[2] for x in av]
        dt = av[0][1] if is_t(av[0]) else av[1][1]
        if None in shapes:
            return [("T", dt, None, dev)]
        return [("T", dt, tuple(int(d) for d in np.broadcast_shapes(*shapes)), dev)]
    if name in ("Relu", "Neg", "Sqrt", "Exp", "Tanh", "Erf", "Gelu", "Identity", "Softmax"):
        return [av[0]]
    if name == "LayerNormalization":
        return [av[0]]
    if name == "Cast":
        x = av[0]
        return [("S", attrs["to"], x[2])] if is_s(x) else [("T", attrs["to"], x[2], x[3])]
    if name == "Transpose":
        x = av[0]
        if x[2] is None:
            return [x]
        perm = attrs.get("perm", list(range(len(x[2])))[::-1])
        return [("T", x[1], tuple(x[2][p] for p in perm), x[3])]
    if name == "Flatten":
        x = av[0]
        if x[2] is None:
            return [x]
        ax = attrs.get("axis", 1)
        return [("T", x[1], (n_elems(x[2][:ax]), n_elems(x[2][ax:])), x[3])]
    if name == "Split":
        x = av[0]
        ax = attrs.get("axis", 0)
        out = []
        for p in attrs["split"]:
            shp = None if x[2] is None else x[2][:ax] + (p,) + x[2][ax + 1:]
            out.append(("T", x[1], shp, x[3]))
        return out
    if name == "MatMul":
        x, y = av
        if x[2] is None or y[2] is None:
            return [("T", x[1], None, dev)]
        if len(y[2]) == 1:
            return [("T", x[1], x[2][:-1], dev)]
        batch = tuple(int(d) for d in np.broadcast_shapes(x[2][:-2], y[2][:-2]))
        return [("T", x[1], batch + (x[2][-2], y[2][-1]), dev)]
    if name == "Gemm":
        x, y = av[0], av[1]
        if x[2] is None or y[2] is None:
            return [("T", x[1], None, dev)]
        m = x[2][1] if attrs.get("transA", 0) else x[2][0]
        n = y[2][0] if attrs.get("transB", 0) else y[2][1]
        return [("T", x[1], (m, n), dev)]
    raise ValueError("op %s not known" % name)


def interpret(text, inputs=None, mixed=True):
    """Per op (outputs, values) in program order."""
    params, ops = read_program(text)
    env = {}
    for name, typ, _ in params:
        v = (inputs or {}).get(name, typ)
        if not isinstance(v, tuple):
            v = np.array(v)
            v = v.astype(np.int64) if v.dtype.kind in "iub" else v.astype(np.float64)
        if not mixed:
            v = as_type(v, typ[3] if is_t(typ) else typ[2])
        env[name] = v
    steps = []
    for outs, name, attrs, args in ops:
        a = [env[x] for x in args]
        res = run_op(name, attrs, a)
        if not mixed and any(is_c(r) for r in res):
            dev = one_device([as_type(x) for x in a])
            res = [as_type(r, dev) for r in res]
        for o, r in zip(outs, res):
            env[o] = r
        steps.append((outs, res))
    return steps


def show(v):
    """The figure's notation: concrete values as lists or numbers, types as
    Tensor[dtype, (shape), device] / dtype."""
    if is_c(v):
        return v.tolist()
    if is_s(v):
        return v[1]
    shp = "??" if v[2] is None else "(" + ", ".join(str(d) for d in v[2]) + ("," if len(v[2]) == 1 else "") + ")"
    return "Tensor[%s, %s, %s]" % (v[1], shp, v[3])


# ---------------------------------------------------------------------------
# The simulated program
# ---------------------------------------------------------------------------
FLOPS_PER_ELEM = {"Add": 1, "Sub": 1, "Mul": 1, "Div": 1, "Pow": 1, "Relu": 1, "Neg": 1, "Sqrt": 1, "Exp": 1,
                  "Tanh": 1, "Erf": 1, "Cast": 0, "Gelu": 8, "Softmax": 5, "LayerNormalization": 8}


def program(text, inputs=None):
    """(ops, tensors, n_dev) for oracle.sim_program: the mixed
    interpretation of the program with its concrete parts left out."""
    params, ops = read_program(text)
    env, tid = {}, {}
    tensors, prog = [], []
    for name, typ, keep in params:
        v = (inputs or {}).get(name, typ)
        if not isinstance(v, tuple):
            v = np.array(v)
            v = v.astype(np.int64) if v.dtype.kind in "iub" else v.astype(np.float64)
        env[name] = v
        if is_t(v):
            tid[name] = len(tensors)
            tensors.append([v[3], tbytes(v), oracle.TF_RESIDENT | (oracle.TF_KEEP if keep else 0)])
    for outs, name, attrs, args in ops:
        a = [env[x] for x in args]
        res = run_op(name, attrs, a)
        for o, r in zip(outs, res):
            env[o] = r
        t_in = [tid[x] for x, v in zip(args, a) if is_t(v)]
        if name == "Send":
            tid[outs[0]] = len(tensors)
            tensors.append([res[0][3], tbytes(res[0]), 0])
            prog.append(dict(kind=oracle.SEND, devs=[a[0][3], res[0][3]], ins=t_in, outs=[tid[outs[0]]],
                             bytes=float(tbytes(a[0]))))
            continue
        if name == "AllReduce":
            for o, x in zip(outs, args):
                tid[o] = tid[x]
            prog.append(dict(kind=oracle.ALLREDUCE, devs=[v[3] for v in a], ins=t_in, outs=[],
                             bytes=float(tbytes(a[0]))))
            continue
        if not any(is_t(r) for r in res):
            continue
        if name in VIEW_OPS:
            src = [x for x, v in zip(args, a) if is_t(v)][0]
            for o in outs:
                tid[o] = tid[src]
            continue
        dev = [r for r in res if is_t(r)][0][3]
        moved = sum(tbytes(v) for v in a if is_t(v)) + sum(tbytes(r) for r in res if is_t(r))
        out0 = res[0]
        kred = 0
        if name == "MatMul":
            kred = a[0][2][-1]
            flops = 2 * n_elems(out0[2]) * kred
        elif name == "Gemm":
            kred = a[0][2][0] if attrs.get("transA", 0) else a[0][2][1]
            flops = 2 * n_elems(out0[2]) * kred + (n_elems(out0[2]) if len(a) == 3 else 0)
        elif name in FLOPS_PER_ELEM:
            flops = FLOPS_PER_ELEM[name] * n_elems(out0[2])
        else:
            flops = 0
        new = []
        for o, r in zip(outs, res):
            if is_t(r):
                tid[o] = len(tensors)
                tensors.append([r[3], tbytes(r), 0])
                new.append(tid[o])
        prog.append(dict(kind=oracle.COMPUTE, devs=[dev], ins=t_in, outs=new, flops=float(flops),
                         bytes=float(moved), matmul=name in ("MatMul", "Gemm"), k=float(kred)))
    # a tensor whose last reader is an all-reduce stays live (in place)
    last = {}
    for i, op in enumerate(prog):
        for t in op["ins"]:
            last[t] = i
    for t, i in last.items():
        if prog[i]["kind"] == oracle.ALLREDUCE:
            tensors[t][2] |= oracle.TF_KEEP
    n_dev = 1 + max([t[0] for t in tensors] + [0])
    return prog, [tuple(t) for t in tensors], n_dev


def simulate(text, dev, inputs=None, n_dev=None):
    ops, tensors, nd = program(text, inputs)
    return oracle.sim_program(ops, tensors, n_dev or nd, dev)
