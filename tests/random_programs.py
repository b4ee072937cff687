"""Seeded random programs in the front end's text form, for differential
tests of the front end against the oracle's interpreter.

Input generation only: a program is built by construction -- each op is
emitted on operands whose shapes the generator chose itself, so it is valid
-- and no cost, memory or simulation arithmetic happens here.  Programs mix
the op types of the text form: elementwise ops, matrix products with fresh
weights (MatMul with batch dimensions, Gemm with transposes and a bias),
Transpose, Reshape (by a Constant target, or by a target computed from Shape
/ Gather / Unsqueeze / Concat as in Fig. 4), Flatten, Unsqueeze / Squeeze,
Split, Concat, Gather, LayerNormalization with and without weights, Cast,
Send (each received tensor is read), AllReduce over copies on distinct
devices; parameters sometimes kept resident.
"""
import numpy as np

DTYPES = ["Float32", "Float16", "BFloat16"]


class _Gen:
    def __init__(self, seed, n_ops, n_dev):
        self.r = np.random.default_rng(seed)
        self.n_dev = n_dev
        self.params, self.lines, self.pool = [], [], []   # pool: (name, shape, dtype, device)
        self.k = 0
        self.n_ops = n_ops

    def name(self, p="v"):
        self.k += 1
        return "%%%s%d" % (p, self.k)

    def param(self, shape, dtype, dev, keep=False, pool=True):
        n = self.name("p")
        shp = "(%s%s)" % (", ".join(str(d) for d in shape), "," if len(shape) == 1 else "")
        self.params.append("%s: Tensor[%s, %s, %d]%s" % (n, dtype, shp, dev, " keep" if keep else ""))
        if pool:
            self.pool.append((n, tuple(shape), dtype, dev))
        return n

    def emit(self, line, outs=()):
        self.lines.append(line)
        self.pool.extend(outs)

    def dim(self):
        return int(self.r.choice([1, 2, 3, 4, 5, 6, 8, 12, 16, 24, 32]))

    def pick(self, rank_min=1):
        cands = [t for t in self.pool if len(t[1]) >= rank_min]
        if not cands:
            return None
        return cands[int(self.r.integers(len(cands)))]

    def step(self):
        r = self.r
        kind = r.choice(["unary", "binary", "matmul", "gemm", "transpose", "reshape_const", "reshape_fig4",
                         "flatten", "unsqueeze", "split", "concat", "gather", "layernorm", "cast", "send",
                         "allreduce"])
        t = self.pick(2 if kind in ("matmul", "gemm", "transpose", "flatten", "split", "concat", "gather") else 1)
        if t is None:
            return
        x, shp, dt, dev = t
        if kind == "unary":
            op = r.choice(["Relu", "Gelu", "Tanh", "Exp", "Neg", "Sqrt", "Erf", "Identity", "Softmax"])
            o = self.name()
            attr = "[axis = -1]" if op == "Softmax" else ""
            self.emit("%s = %s%s(%s)" % (o, op, attr, x), [(o, shp, dt, dev)])
        elif kind == "binary":
            op = r.choice(["Add", "Sub", "Mul", "Div", "Pow"])
            same = [u for u in self.pool if u[1] == shp and u[3] == dev]
            if r.random() < 0.3:   # broadcast against a fresh trailing-dimension parameter
                y = self.param(shp[-1:], dt, dev, keep=bool(r.random() < 0.5), pool=False)
            else:
                y = same[int(r.integers(len(same)))][0]
            o = self.name()
            a, b = (x, y) if r.random() < 0.5 else (y, x)
            self.emit("%s = %s(%s, %s)" % (o, op, a, b), [(o, shp, dt, dev)])
        elif kind == "matmul":
            n = self.dim()
            if r.random() < 0.5:
                w = self.param((shp[-1], n), dt, dev, keep=True, pool=False)
                out = shp[:-1] + (n,)
            else:                      # a batched right operand of the same batch shape
                w = self.param(shp[:-2] + (shp[-1], n), dt, dev, pool=False)
                out = shp[:-1] + (n,)
            o = self.name()
            self.emit("%s = MatMul(%s, %s)" % (o, x, w), [(o, out, dt, dev)])
        elif kind == "gemm":
            if len(shp) != 2:
                return
            m, k = shp
            n = self.dim()
            ta, tb = int(r.integers(2)), int(r.integers(2))
            a = x
            if ta:
                a = self.name()
                self.emit("%s = Transpose[perm = [1, 0]](%s)" % (a, x), [(a, (k, m), dt, dev)])
            w = self.param((n, k) if tb else (k, n), dt, dev, keep=True, pool=False)
            args = "%s, %s" % (a, w)
            if r.random() < 0.5:
                args += ", " + self.param((n,), dt, dev, keep=True, pool=False)
            o = self.name()
            self.emit("%s = Gemm[transA = %d, transB = %d](%s)" % (o, ta, tb, args), [(o, (m, n), dt, dev)])
        elif kind == "transpose":
            perm = [int(p) for p in r.permutation(len(shp))]
            o = self.name()
            self.emit("%s = Transpose[perm = [%s]](%s)" % (o, ", ".join(map(str, perm)), x),
                      [(o, tuple(shp[p] for p in perm), dt, dev)])
        elif kind == "reshape_const":
            total = int(np.prod(shp))
            if len(shp) >= 2 and r.random() < 0.5:
                tgt, out = [0, -1], (shp[0], total // shp[0])
            else:
                tgt, out = [-1], (total,)
            c, o = self.name("c"), self.name()
            self.emit("%s = Constant[value = [%s]]()" % (c, ", ".join(map(str, tgt))))
            self.emit("%s = Reshape(%s, %s)" % (o, x, c), [(o, out, dt, dev)])
        elif kind == "reshape_fig4":
            if len(shp) < 2:
                return
            s, i, g, u, m1, c, o = (self.name(p) for p in "sigumco")
            last = len(shp) - 1
            self.emit("%s = Shape(%s)" % (s, x))
            self.emit("%s = Constant[value = %d]()" % (i, last))
            self.emit("%s = Gather[axis = 0](%s, %s)" % (g, s, i))
            self.emit("%s = Unsqueeze[axes = [0]](%s)" % (u, g))
            self.emit("%s = Constant[value = [-1]]()" % m1)
            self.emit("%s = Concat[axis = 0](%s, %s)" % (c, m1, u))
            self.emit("%s = Reshape(%s, %s)" % (o, x, c), [(o, (int(np.prod(shp[:-1])), shp[-1]), dt, dev)])
        elif kind == "flatten":
            ax = int(r.integers(len(shp) + 1))
            o = self.name()
            self.emit("%s = Flatten[axis = %d](%s)" % (o, ax, x),
                      [(o, (int(np.prod(shp[:ax])), int(np.prod(shp[ax:]))), dt, dev)])
        elif kind == "unsqueeze":
            if len(shp) > 3:
                return
            ax = int(r.integers(len(shp) + 1))
            o, q = self.name(), self.name()
            self.emit("%s = Unsqueeze[axes = [%d]](%s)" % (o, ax, x), [])
            self.emit("%s = Squeeze[axes = [%d]](%s)" % (q, ax, o), [(q, shp, dt, dev)])
        elif kind == "split":
            ax = int(r.integers(len(shp)))
            if shp[ax] < 2:
                return
            cut = int(r.integers(1, shp[ax]))
            o1, o2 = self.name(), self.name()
            s1, s2 = list(shp), list(shp)
            s1[ax], s2[ax] = cut, shp[ax] - cut
            self.emit("%s, %s = Split[axis = %d, split = [%d, %d]](%s)" % (o1, o2, ax, cut, shp[ax] - cut, x),
                      [(o1, tuple(s1), dt, dev), (o2, tuple(s2), dt, dev)])
        elif kind == "concat":
            if np.prod(shp) > 2 ** 14:
                return
            same = [u for u in self.pool if u[1] == shp and u[3] == dev and u[2] == dt]
            y = same[int(r.integers(len(same)))][0]
            ax = int(r.integers(len(shp)))
            s = list(shp)
            s[ax] *= 2
            o = self.name()
            self.emit("%s = Concat[axis = %d](%s, %s)" % (o, ax, x, y), [(o, tuple(s), dt, dev)])
        elif kind == "gather":
            ax = int(r.integers(len(shp)))
            idx = [int(v) for v in r.integers(0, shp[ax], size=int(r.integers(1, 4)))]
            c, o = self.name("c"), self.name()
            s = list(shp)
            s[ax] = len(idx)
            self.emit("%s = Constant[value = [%s]]()" % (c, ", ".join(map(str, idx))))
            self.emit("%s = Gather[axis = %d](%s, %s)" % (o, ax, x, c), [(o, tuple(s), dt, dev)])
        elif kind == "layernorm":
            o = self.name()
            if r.random() < 0.5:
                g = self.param(shp[-1:], dt, dev, keep=True, pool=False)
                b = self.param(shp[-1:], dt, dev, keep=True, pool=False)
                self.emit("%s = LayerNormalization(%s, %s, %s)" % (o, x, g, b), [(o, shp, dt, dev)])
            else:
                self.emit("%s = LayerNormalization(%s)" % (o, x), [(o, shp, dt, dev)])
        elif kind == "cast":
            to = DTYPES[int(r.integers(len(DTYPES)))]
            o = self.name()
            self.emit('%s = Cast[to = "%s"](%s)' % (o, to, x), [(o, shp, to, dev)])
        elif kind == "send":
            if self.n_dev < 2:
                return
            to = int((dev + 1 + r.integers(self.n_dev - 1)) % self.n_dev)
            o, u = self.name(), self.name()
            self.emit("%s = Send[device = %d](%s)" % (o, to, x))
            self.emit("%s = Relu(%s)" % (u, o), [(u, shp, dt, to)])
        elif kind == "allreduce":
            if self.n_dev < 2:
                return
            k = int(r.integers(2, self.n_dev + 1))
            others = [d for d in r.permutation(self.n_dev) if d != dev][:k - 1]
            copies = [x]
            for d in others:
                o = self.name()
                self.emit("%s = Send[device = %d](%s)" % (o, int(d), x))
                copies.append(o)
            outs = [self.name() for _ in copies]
            self.emit("%s = AllReduce(%s)" % (", ".join(outs), ", ".join(copies)),
                      [(o, shp, dt, d) for o, d in zip(outs, [dev] + [int(d) for d in others])])

    def build(self):
        for d in range(self.n_dev):
            rank = int(self.r.integers(1, 4))
            self.param(tuple(self.dim() for _ in range(rank)), DTYPES[int(self.r.integers(2))], d,
                       keep=bool(self.r.random() < 0.3))
        while len(self.lines) < self.n_ops:
            self.step()
        return "func rnd(%s)\n%s\nreturn %s\n" % (", ".join(self.params), "\n".join(self.lines), self.pool[-1][0])


def random_program(seed, n_ops=40, n_dev=None):
    """Program text of about n_ops statements over n_dev devices (1..4,
    drawn from the seed when None)."""
    if n_dev is None:
        n_dev = int(np.random.default_rng(seed + 7919).integers(1, 5))
    return _Gen(seed, n_ops, n_dev).build()
