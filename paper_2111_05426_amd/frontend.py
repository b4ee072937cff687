"""Shape-inference front end: programs written op by op, interpreted over a
mixed abstract/concrete domain, lowered to the explicit op tables that
dsim_simulate_tables simulates.

Sec. 3 builds every analysis on one abstract interpreter (Algorithm 1): it
steps through the program's ops in order, keeping for every variable an
abstract description instead of data, and evaluates each op type through an
implementation that works on such descriptions.  For the simulator
(Sec. 3.3) the values are abstract tensors -- element type, shape, device --
and the cost of an op follows from the shapes of its inputs.  Ops such as
Shape make a shape depend on the concrete value of a tensor, so the domain
mixes concrete values (numbers, small integer arrays) with abstract ones, op
types carry concrete, mixed and abstract implementations, and the
interpreter dispatches each op to the most precise one whose argument kinds
match (Sec. 3.3; the Reshape snippet of Fig. 4 is the worked example).

Program text, one statement per line (`#` starts a comment):

    func NAME(%a: Tensor[Float32, (256, 8, 768), 0], %w: Tensor[Float32, (768, 64), 0] keep, %s: Int32)
    %t = OpType[attr = value, ...](%a, %b)
    %u, %v = Split[axis = 0, split = [2, 2]](%t)
    return %u

Types: `Tensor[DTYPE, (d0, ...), DEVICE]` (a shape of `??` is unknown) or a
scalar `DTYPE` / `DTYPE[DEVICE]`.  A parameter marked `keep` (weights) stays
resident for the whole program; every other tensor lives from the op that
defines it until the last op that reads it (Sec. 3.3).  The caller may give
any parameter a concrete value instead of its declared abstract type.

Lowering (readings of Sec. 3.3 for the table format): an op whose inputs are
all concrete is evaluated on the host and emits nothing; a view (Reshape,
Unsqueeze, Squeeze, Flatten, Identity) shares its input's memory and emits
nothing; every other op on abstract tensors becomes one table record on the
device of its inputs: compute (matrix products as cost class 1), Send,
AllReduce (in place over the devices of its inputs).  Costs per op are in
`_cost`; memory per record: the bytes of the tensors the op creates are
allocated on the op's device (a Send's receiver), and the tensors whose
last reader it is are freed there.
"""
import ast
import math
import re
from dataclasses import dataclass, field

import numpy as np

ELEM_BYTES = {"Float64": 8, "Float32": 4, "Float16": 2, "BFloat16": 2, "Int64": 8, "Int32": 4, "Int8": 1,
              "Bool": 1}


# ---------------------------------------------------------------------------
# Abstract values
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class Tensor:
    """An abstract tensor: element type, shape (None = unknown), device."""
    dtype: str
    shape: tuple
    device: int

    def __repr__(self):
        if self.shape is None:
            shape = "??"
        else:
            shape = "(%s%s)" % (", ".join(str(d) for d in self.shape), "," if len(self.shape) == 1 else "")
        return "Tensor[%s, %s, %s]" % (self.dtype, shape, self.device)

    @property
    def nbytes(self):
        if self.shape is None:
            raise ValueError("cannot simulate: the shape of a %s tensor is unknown" % self.dtype)
        return math.prod(self.shape) * ELEM_BYTES[self.dtype]

    @property
    def numel(self):
        if self.shape is None:
            raise ValueError("cannot simulate: a shape is unknown")
        return math.prod(self.shape)


@dataclass(frozen=True)
class Scalar:
    """An abstract scalar of an element type (on a device, or none)."""
    dtype: str
    device: int = None

    def __repr__(self):
        return self.dtype


def is_concrete(v):
    return isinstance(v, np.ndarray)


def concrete(v):
    """A concrete value as an array (numbers and lists included)."""
    a = np.asarray(v)
    return a.astype(np.int64) if a.dtype.kind in "iub" else a.astype(np.float64)


def dtype_of_array(a):
    if a.dtype.kind == "f":
        return "Float64" if a.dtype.itemsize == 8 else "Float32"
    if a.dtype.kind == "b":
        return "Bool"
    return "Int32"   # shape arithmetic: the paper's listings type it Int32


def abstract_of(v, device=None):
    """The abstraction of a concrete value (abstract-only interpretation)."""
    if not is_concrete(v):
        return v
    if v.ndim == 0:
        return Scalar(dtype_of_array(v), device)
    return Tensor(dtype_of_array(v), tuple(int(d) for d in v.shape), device)


# ---------------------------------------------------------------------------
# Programs
# ---------------------------------------------------------------------------
@dataclass
class Op:
    outs: list
    type: str
    attrs: dict
    ins: list
    line: int = 0


@dataclass
class Program:
    name: str
    params: list                     # (name, abstract type, keep)
    ops: list
    returns: list = field(default_factory=list)


_TENSOR = re.compile(r"Tensor\[\s*(\w+)\s*,\s*(\(.*?\)|\?\?)\s*,\s*(-?\d+)\s*\]")
_SCALAR = re.compile(r"(\w+)(?:\[\s*(-?\d+)\s*\])?$")
_OP = re.compile(r"^(%[\w.]+(?:\s*,\s*%[\w.]+)*)\s*=\s*(\w+)\s*(?:\[(.*?)\])?\s*\((.*)\)\s*$")


def parse_type(text):
    text = text.strip()
    m = _TENSOR.fullmatch(text)
    if m:
        shape = None if m.group(2) == "??" else tuple(int(d) for d in ast.literal_eval(m.group(2)))
        if m.group(1) not in ELEM_BYTES:
            raise ValueError("unknown element type %s" % m.group(1))
        return Tensor(m.group(1), shape, int(m.group(3)))
    m = _SCALAR.fullmatch(text)
    if m and m.group(1) in ELEM_BYTES:
        return Scalar(m.group(1), None if m.group(2) is None else int(m.group(2)))
    raise ValueError("cannot parse type %r" % text)


def _split_top(text, sep=","):
    """Split at separators outside brackets and parentheses."""
    parts, depth, cur = [], 0, ""
    for ch in text:
        if ch in "([":
            depth += 1
        elif ch in ")]":
            depth -= 1
        if ch == sep and depth == 0:
            parts.append(cur)
            cur = ""
        else:
            cur += ch
    if cur.strip():
        parts.append(cur)
    return [p.strip() for p in parts]


def _attrs(text):
    out = {}
    for item in _split_top(text or ""):
        k, v = item.split("=", 1)
        out[k.strip()] = ast.literal_eval(v.strip())
    return out


def parse(text):
    """A Program from its text."""
    prog = None
    for n, raw in enumerate(text.splitlines(), 1):
        line = raw.split("#", 1)[0].strip()
        if not line:
            continue
        if line.startswith("func "):
            m = re.match(r"func\s+(\w+)\s*\((.*)\)\s*$", line)
            if not m:
                raise ValueError("line %d: bad function header" % n)
            params = []
            for p in _split_top(m.group(2)):
                name, rest = p.split(":", 1)
                rest = rest.strip()
                keep = rest.endswith(" keep")
                if keep:
                    rest = rest[:-5]
                params.append((name.strip(), parse_type(rest), keep))
            prog = Program(m.group(1), params, [])
            continue
        if prog is None:
            raise ValueError("line %d: statement before the function header" % n)
        if line.startswith("return"):
            prog.returns = [v.strip() for v in line[6:].split(",") if v.strip()]
            continue
        m = _OP.match(line)
        if not m:
            raise ValueError("line %d: cannot parse %r" % (n, line))
        outs = [v.strip() for v in m.group(1).split(",")]
        ins = [v.strip() for v in _split_top(m.group(4))]
        prog.ops.append(Op(outs, m.group(2), _attrs(m.group(3)), ins, n))
    if prog is None:
        raise ValueError("no function")
    return prog


# ---------------------------------------------------------------------------
# Semantics: per op type, implementations by argument kind
# ---------------------------------------------------------------------------
# kinds: 'c' concrete, 't' abstract tensor, 's' abstract scalar, 'a' any
# abstract value, '*' anything
_IMPLS = {}


def impl(op_type, kinds):
    def reg(fn):
        _IMPLS.setdefault(op_type, []).append((kinds, fn))
        # most precise first: more arguments required concrete, then fewer wildcards
        _IMPLS[op_type].sort(key=lambda e: (-sum(k == "c" for k in e[0]), sum(k == "*" for k in e[0])))
        return fn
    return reg


def _kind_ok(k, v):
    if k == "*":
        return True
    if k == "c":
        return is_concrete(v)
    if k == "t":
        return isinstance(v, Tensor)
    if k == "s":
        return isinstance(v, Scalar)
    return not is_concrete(v)


def dispatch(op_type, args):
    """The most precise implementation of op_type matching the arguments."""
    for kinds, fn in _IMPLS.get(op_type, []):
        variadic = kinds.endswith("...")
        ks = kinds[:-3] if variadic else kinds
        if variadic:
            if len(args) < len(ks) - 1:
                continue
            ks = ks[:-1] + ks[-1] * (len(args) - len(ks) + 1)
        elif len(ks) != len(args):
            continue
        if all(_kind_ok(k, v) for k, v in zip(ks, args)):
            return fn
    raise ValueError("no implementation of %s for arguments %s" % (op_type, [type(a).__name__ for a in args]))


def _device(args):
    devs = {a.device for a in args if isinstance(a, (Tensor, Scalar)) and a.device is not None}
    if len(devs) > 1:
        raise ValueError("inputs on different devices %s" % sorted(devs))
    return devs.pop() if devs else None


def _bcast(*shapes):
    if any(s is None for s in shapes):
        return None
    return tuple(int(d) for d in np.broadcast_shapes(*shapes))


def _np_int(v):
    return np.asarray(v, dtype=np.int64)


# -- constants, shapes, index arithmetic --------------------------------------
@impl("Constant", "")
def _constant(attrs):
    v = np.asarray(attrs["value"])
    return [v.astype(np.int64) if v.dtype.kind in "iub" else v.astype(np.float64)]


@impl("Shape", "c")
def _shape_c(attrs, x):
    return [_np_int(x.shape)]


@impl("Shape", "t")
def _shape_t(attrs, x):
    if x.shape is None:
        return [Tensor("Int32", None, x.device)]
    return [_np_int(x.shape)]      # mixed: an abstract tensor's shape is known


@impl("Gather", "cc")
def _gather_c(attrs, data, idx):
    return [np.take(data, idx, axis=attrs.get("axis", 0))]


@impl("Gather", "aa")
def _gather_a(attrs, data, idx):
    dev = _device([data, idx])
    if isinstance(data, Tensor) and data.shape is not None and len(data.shape) == 1 and \
            (isinstance(idx, Scalar) or (is_concrete(idx) and idx.ndim == 0)):
        return [Scalar(data.dtype, dev)]
    ishape = () if isinstance(idx, Scalar) else (idx.shape if isinstance(idx, Tensor) else tuple(idx.shape))
    ax = attrs.get("axis", 0)
    if data.shape is None or ishape is None:
        return [Tensor(data.dtype, None, dev)]
    return [Tensor(data.dtype, data.shape[:ax] + tuple(ishape) + data.shape[ax + 1:], dev)]


@impl("Gather", "tc")
def _gather_tc(attrs, data, idx):
    return _gather_a(attrs, data, idx)


def _unsq_shape(shape, axes):
    out = list(shape)
    for a in sorted(a if a >= 0 else a + len(shape) + len(axes) for a in axes):
        out.insert(a, 1)
    return tuple(out)


@impl("Unsqueeze", "c")
def _unsqueeze_c(attrs, x):
    return [x.reshape(_unsq_shape(x.shape, attrs["axes"]))]


@impl("Unsqueeze", "a")
def _unsqueeze_a(attrs, x):
    if isinstance(x, Scalar):
        return [Tensor(x.dtype, _unsq_shape((), attrs["axes"]), x.device)]
    return [Tensor(x.dtype, None if x.shape is None else _unsq_shape(x.shape, attrs["axes"]), x.device)]


@impl("Squeeze", "c")
def _squeeze_c(attrs, x):
    return [np.squeeze(x, axis=tuple(attrs["axes"]))]


@impl("Squeeze", "t")
def _squeeze_t(attrs, x):
    if x.shape is None:
        return [x]
    axes = {a % len(x.shape) for a in attrs["axes"]}
    return [Tensor(x.dtype, tuple(d for i, d in enumerate(x.shape) if i not in axes), x.device)]


@impl("Concat", "c...")
def _concat_c(attrs, *xs):
    return [np.concatenate([np.atleast_1d(x) for x in xs], axis=attrs.get("axis", 0))]


@impl("Concat", "*...")
def _concat_a(attrs, *xs):
    vals = [abstract_of(x) for x in xs]
    dev = _device(vals)
    ax = attrs.get("axis", 0)
    if any(v.shape is None for v in vals if isinstance(v, Tensor)) or any(isinstance(v, Scalar) for v in vals):
        return [Tensor(vals[0].dtype, None, dev)]
    s0 = list(vals[0].shape)
    s0[ax] = sum(v.shape[ax] for v in vals)
    return [Tensor(vals[0].dtype, tuple(s0), dev)]


def _reshape_target(shape, target):
    target = [int(t) for t in target]
    out = [shape[i] if t == 0 else t for i, t in enumerate(target)]
    if -1 in out:
        known = int(np.prod([d for d in out if d != -1], dtype=np.int64))
        out[out.index(-1)] = int(np.prod(shape, dtype=np.int64)) // known
    if int(np.prod(out, dtype=np.int64)) != int(np.prod(shape, dtype=np.int64)):
        raise ValueError("cannot reshape %s to %s" % (shape, target))
    return tuple(out)


@impl("Reshape", "cc")
def _reshape_c(attrs, x, s):
    return [x.reshape(_reshape_target(x.shape, s))]


@impl("Reshape", "tc")
def _reshape_tc(attrs, x, s):
    return [Tensor(x.dtype, None if x.shape is None else _reshape_target(x.shape, s), x.device)]


@impl("Reshape", "ta")
def _reshape_ta(attrs, x, s):
    return [Tensor(x.dtype, None, x.device)]   # the target is not known


# -- elementwise ----------------------------------------------------------------
_BINARY = {"Add": np.add, "Sub": np.subtract, "Mul": np.multiply, "Div": np.divide, "Pow": np.power}
_UNARY = {"Relu": lambda a: np.maximum(a, 0), "Neg": np.negative, "Sqrt": np.sqrt, "Exp": np.exp,
          "Tanh": np.tanh, "Erf": None, "Gelu": None, "Identity": lambda a: a}


def _make_binary(name, fn):
    @impl(name, "cc")
    def _c(attrs, a, b):
        r = fn(a, b)
        return [r.astype(np.int64) if name != "Div" and r.dtype.kind in "iub" else r]

    @impl(name, "**")
    def _a(attrs, a, b):
        va, vb = abstract_of(a), abstract_of(b)
        dev = _device([va, vb])
        sa = () if isinstance(va, Scalar) else va.shape
        sb = () if isinstance(vb, Scalar) else vb.shape
        dt = va.dtype if isinstance(va, Tensor) else vb.dtype
        if isinstance(va, Scalar) and isinstance(vb, Scalar):
            return [Scalar(va.dtype, dev)]
        return [Tensor(dt, _bcast(sa, sb), dev)]


for _n, _f in _BINARY.items():
    _make_binary(_n, _f)


def _make_unary(name, fn):
    if fn is not None:
        @impl(name, "c")
        def _c(attrs, a):
            return [fn(a)]

    @impl(name, "a")
    def _a(attrs, a):
        return [a]


for _n, _f in _UNARY.items():
    _make_unary(_n, _f)


@impl("Cast", "c")
def _cast_c(attrs, a):
    return [a.astype(np.float64 if attrs["to"].startswith("Float") else np.int64)]


@impl("Cast", "a")
def _cast_a(attrs, a):
    if isinstance(a, Scalar):
        return [Scalar(attrs["to"], a.device)]
    return [Tensor(attrs["to"], a.shape, a.device)]


for _n in ("Softmax", "LayerNormalization"):
    impl(_n, "t")(lambda attrs, a: [a])


@impl("LayerNormalization", "ttt")
def _ln3(attrs, a, g, b):
    _device([a, g, b])
    return [a]


@impl("Transpose", "t")
def _transpose(attrs, a):
    if a.shape is None:
        return [a]
    perm = attrs.get("perm", list(range(len(a.shape)))[::-1])
    return [Tensor(a.dtype, tuple(a.shape[p] for p in perm), a.device)]


@impl("Flatten", "t")
def _flatten(attrs, a):
    if a.shape is None:
        return [a]
    ax = attrs.get("axis", 1)
    return [Tensor(a.dtype, (int(np.prod(a.shape[:ax], dtype=np.int64)),
                             int(np.prod(a.shape[ax:], dtype=np.int64))), a.device)]


@impl("Split", "t")
def _split(attrs, a):
    ax, parts = attrs.get("axis", 0), attrs["split"]
    if a.shape is None:
        return [Tensor(a.dtype, None, a.device) for _ in parts]
    if sum(parts) != a.shape[ax]:
        raise ValueError("split %s does not cover dimension %d" % (parts, a.shape[ax]))
    out = []
    for p in parts:
        s = list(a.shape)
        s[ax] = p
        out.append(Tensor(a.dtype, tuple(s), a.device))
    return out


# -- matrix products -------------------------------------------------------------
def _matmul_shape(sa, sb):
    if sa is None or sb is None:
        return None
    if sa[-1] != sb[-2 if len(sb) > 1 else 0]:
        raise ValueError("MatMul of %s and %s" % (sa, sb))
    batch = _bcast(sa[:-2], sb[:-2]) if len(sb) > 1 else sa[:-2]
    return tuple(batch) + (sa[-2],) + ((sb[-1],) if len(sb) > 1 else ())


@impl("MatMul", "tt")
def _matmul(attrs, a, b):
    return [Tensor(a.dtype, _matmul_shape(a.shape, b.shape), _device([a, b]))]


def _gemm_shape(attrs, sa, sb):
    if sa is None or sb is None:
        return None
    m, k = (sa[1], sa[0]) if attrs.get("transA", 0) else sa
    k2, n = (sb[1], sb[0]) if attrs.get("transB", 0) else sb
    if k != k2:
        raise ValueError("Gemm of %s and %s" % (sa, sb))
    return (m, n)


@impl("Gemm", "tt")
def _gemm(attrs, a, b):
    return [Tensor(a.dtype, _gemm_shape(attrs, a.shape, b.shape), _device([a, b]))]


@impl("Gemm", "ttt")
def _gemm_bias(attrs, a, b, c):
    return [Tensor(a.dtype, _gemm_shape(attrs, a.shape, b.shape), _device([a, b, c]))]


# -- communication -----------------------------------------------------------------
@impl("Send", "t")
def _send(attrs, a):
    if attrs["device"] == a.device:
        raise ValueError("Send to its own device %d" % a.device)
    return [Tensor(a.dtype, a.shape, attrs["device"])]


@impl("AllReduce", "t...")
def _allreduce(attrs, *xs):
    devs = [x.device for x in xs]
    if len(set(devs)) != len(devs):
        raise ValueError("AllReduce inputs must lie on distinct devices, got %s" % devs)
    if len({x.shape for x in xs}) != 1:
        raise ValueError("AllReduce of tensors of different shapes")
    return list(xs)


# ---------------------------------------------------------------------------
# Algorithm 1
# ---------------------------------------------------------------------------
VIEWS = {"Reshape", "Unsqueeze", "Squeeze", "Flatten", "Identity"}


def interpret(prog, inputs=None, mixed=True):
    """Run the program op by op over the abstract state (Algorithm 1).

    inputs: optional {parameter name: value}; a value is a concrete array
    (or Python number / list) or an abstract Tensor / Scalar, replacing the
    declared type.  mixed=False abstracts every concrete value (the
    abstract-only interpretation).  Returns (state, trace): the final map of
    variables to values, and per op (op, argument values, result values).
    """
    state = {}
    for name, typ, _ in prog.params:
        v = (inputs or {}).get(name, typ)
        if not isinstance(v, (Tensor, Scalar)):
            v = concrete(v)
        state[name] = v if mixed else abstract_of(v, getattr(typ, "device", None))
    trace = []
    for op in prog.ops:
        for o in op.outs:
            if o in state:
                raise ValueError("line %d: %s is defined twice" % (op.line, o))
        try:
            args = [state[v] for v in op.ins]
        except KeyError as e:
            raise ValueError("line %d: %s is not defined" % (op.line, e.args[0])) from None
        try:
            res = dispatch(op.type, args)(op.attrs, *args)
        except ValueError as e:
            raise ValueError("line %d (%s): %s" % (op.line, op.type, e)) from None
        res = [r if isinstance(r, (Tensor, Scalar)) else concrete(r) for r in res]
        if len(res) != len(op.outs):
            raise ValueError("line %d: %s gives %d values, %d names" % (op.line, op.type, len(res), len(op.outs)))
        if not mixed:
            dev = _device([abstract_of(a) for a in args])
            res = [abstract_of(r, dev) for r in res]
        for name, val in zip(op.outs, res):
            state[name] = val
        trace.append((op, args, res))
    return state, trace


# ---------------------------------------------------------------------------
# Costs (flops, bytes, class) of an op on abstract tensors
# ---------------------------------------------------------------------------
_ELEMENTWISE_FLOPS = {"Add": 1, "Sub": 1, "Mul": 1, "Div": 1, "Pow": 1, "Relu": 1, "Neg": 1, "Sqrt": 1,
                      "Exp": 1, "Tanh": 1, "Erf": 1, "Cast": 0, "Gelu": 8, "Softmax": 5, "LayerNormalization": 8}


def _tensor_bytes(vals):
    return sum(v.nbytes for v in vals if isinstance(v, Tensor))


def _cost(op, args, res):
    """(flops, bytes, cost class) of a compute op."""
    t = op.type
    moved = _tensor_bytes(args) + _tensor_bytes(res)
    if t == "MatMul":
        a, b = args
        k = a.shape[-1]
        return 2 * res[0].numel * k, moved, 1
    if t == "Gemm":
        a = args[0]
        k = a.shape[0] if op.attrs.get("transA", 0) else a.shape[1]
        fl = 2 * res[0].numel * k + (res[0].numel if len(args) == 3 else 0)
        return fl, moved, 1
    if t in _ELEMENTWISE_FLOPS:
        return _ELEMENTWISE_FLOPS[t] * res[0].numel, moved, 0
    if t in ("Transpose", "Concat", "Split", "Gather"):
        return 0, moved, 0
    raise ValueError("no cost function for %s" % t)


# ---------------------------------------------------------------------------
# Lowering to one candidate's op table
# ---------------------------------------------------------------------------
def lower(prog, inputs=None, n_dev=None):
    """Interpret (mixed) and lower to records.  Returns dict(code, flops,
    bytes, alloc, free, init_live, n_dev) with uint32 / float32 / uint64
    numpy arrays; raises ValueError where the program cannot be simulated
    (an unknown shape, an op on inputs of several devices, a received tensor
    nothing reads, a value that does not fit the record format).

    An op emits a record when it yields an abstract tensor (views excepted)
    or is a Send or AllReduce; ops that yield only concrete values (or
    abstract scalars) run on the host and hold no memory.  Memory is per
    storage: an op's new tensors get one each (allocated by its record, on
    its device), a view shares its input's; a storage lives until the last
    record that reads it and is freed there (a storage nothing reads, by
    the record that creates it); parameters are resident from t = 0, `keep`
    ones for good; a storage last read by an AllReduce stays live (the
    collective works in place and frees nothing)."""
    state, trace = interpret(prog, inputs, mixed=True)
    st_of = {}                     # variable -> storage id
    st_dev, st_bytes, st_keep, st_res = [], [], [], []

    def new_storage(t, resident=False, keep=False):
        st_dev.append(t.device)
        st_bytes.append(t.nbytes)
        st_keep.append(keep)
        st_res.append(resident)
        return len(st_dev) - 1

    for name, _, keep in prog.params:
        if isinstance(state[name], Tensor):
            st_of[name] = new_storage(state[name], resident=True, keep=keep)
    recs = []                      # (kind, a, b or mask, class, flops, bytes, created, read)
    for op, args, res in trace:
        read = sorted({st_of[v] for v, a in zip(op.ins, args) if isinstance(a, Tensor)})
        if op.type == "Send":
            out = new_storage(res[0])
            st_of[op.outs[0]] = out
            recs.append((1, args[0].device, res[0].device, 0, 0.0, float(args[0].nbytes), [out], read))
            continue
        if op.type == "AllReduce":
            mask = 0
            for a in args:
                mask |= 1 << a.device
            for o, v in zip(op.outs, op.ins):
                st_of[o] = st_of[v]          # in place
            recs.append((2, 0, mask, 0, 0.0, float(args[0].nbytes), [], read))
            continue
        if not any(isinstance(r, Tensor) for r in res):
            continue                           # host-side value arithmetic
        if op.type in VIEWS:
            src = next(v for v, a in zip(op.ins, args) if isinstance(a, Tensor))
            for o, r in zip(op.outs, res):
                st_of[o] = st_of[src]
            continue
        devs = {a.device for a in args if isinstance(a, Tensor)} | {r.device for r in res if isinstance(r, Tensor)}
        if len(devs) != 1 or None in devs:
            raise ValueError("line %d: %s on devices %s" % (op.line, op.type, sorted(devs, key=str)))
        fl, by, cls = _cost(op, args, res)
        created = []
        for o, r in zip(op.outs, res):
            if isinstance(r, Tensor):
                st_of[o] = new_storage(r)
                created.append(st_of[o])
        recs.append((0, devs.pop(), 0, cls, float(fl), float(by), created, read))
    last = [-1] * len(st_dev)
    for i, r in enumerate(recs):
        for s in r[6] + r[7]:
            last[s] = i
    nd = n_dev if n_dev is not None else 1 + max(st_dev + [0])
    if max(st_dev + [0]) >= nd:
        raise ValueError("a device beyond n_dev = %d" % nd)
    init = np.zeros(nd, np.uint64)
    for s, d in enumerate(st_dev):
        if st_res[s]:
            init[d] += np.uint64(st_bytes[s])
    n = len(recs)
    code = np.zeros(n, np.uint32)
    flops = np.zeros(n, np.float32)
    nbytes = np.zeros(n, np.float32)
    alloc = np.zeros(n, np.uint32)
    free = np.zeros(n, np.uint32)
    for i, (kind, a, b, cls, fl, by, created, read) in enumerate(recs):
        dying = [s for s in set(created) | set(read) if last[s] == i and not st_keep[s]]
        if kind == 1 and any(s in created for s in dying):
            raise ValueError("a received tensor nothing reads")
        fr = 0 if kind == 2 else sum(st_bytes[s] for s in dying)   # all on device a
        al = sum(st_bytes[s] for s in created)
        code[i] = kind | (a << 8) | (b << 16) | (cls << 24)
        flops[i], nbytes[i] = fl, by
        if float(flops[i]) != fl or float(nbytes[i]) != by or al >= 2 ** 32 or fr >= 2 ** 32:
            raise ValueError("op %d does not fit the table format exactly" % i)
        alloc[i], free[i] = al, fr
    return dict(code=code, flops=flops, bytes=nbytes, alloc=alloc, free=free, init_live=init, n_dev=nd)


def pack(tables):
    """Candidate-fastest arrays (max_ops, n_cand) of several lowered tables
    (one n_dev for all), with n_ops and init_live (n_cand, n_dev)."""
    nd = max(t["n_dev"] for t in tables)
    n = len(tables)
    m = max([len(t["code"]) for t in tables] + [1])
    out = dict(code=np.zeros((m, n), np.uint32), flops=np.zeros((m, n), np.float32),
               bytes=np.zeros((m, n), np.float32), alloc=np.zeros((m, n), np.uint32),
               free=np.zeros((m, n), np.uint32), n_ops=np.zeros(n, np.uint32),
               init_live=np.zeros((n, nd), np.uint64), n_dev=nd)
    for c, t in enumerate(tables):
        k = len(t["code"])
        for f in ("code", "flops", "bytes", "alloc", "free"):
            out[f][:k, c] = t[f]
        out["n_ops"][c] = k
        out["init_live"][c, :t["n_dev"]] = t["init_live"]
    return out
