"""Pins of the oracle's transformer program: bytes moved by every op type and
the peak memory of one pipeline stage, derived by hand.

The paper fixes no per-op byte count for its GPT-2 programs (it imports them
from ONNX, Sec. 4); the transform here defines each op's bytes as the bytes
of the tensors it reads plus those it writes (Sec. 3.3: data movement
bounds an op's time in the roofline form), and memory by def/use liveness
(Sec. 3.3: a tensor is live from its creation until its last use).  This
test writes one tensor-parallel rank's program of a GPT-shaped decoder down
by hand -- every op of the forward and backward pass with the tensors it
reads and writes, their shapes taken from the architecture (Megatron
column/row parallel layers, vocabulary-parallel embedding and head), the
weight update -- and derives from it, with a ten-line liveness walk of its
own, (a) the bytes of every op type and (b) the peak live bytes of the
device.  Neither reuses the oracle's formulas: a wrong factor, a tensor read
twice or freed too early or too late in the oracle fails here.
"""
import pytest

from paper_2111_05426_amd.workloads import DeviceSpec, INFER, TRAIN_SGD, transformer

DEV = DeviceSpec()


class Prog:
    """A hand-written program: ops reading and writing named tensors."""

    def __init__(self):
        self.size = {}        # tensor -> bytes
        self.keep = set()     # never freed (weights, optimizer state)
        self.initial = []     # live at t = 0
        self.ops = []         # (type, reads [(tensor, bytes read)], writes [(tensor, bytes written, new)])
        self.flops = {}       # matrix-product flops by type
        self.kred = {}        # reduction lengths of the products by type

    def tensor(self, name, nbytes, keep=False, initial=False):
        self.size[name] = nbytes
        if keep:
            self.keep.add(name)
        if initial:
            self.initial.append(name)

    def op(self, typ, reads, writes):
        """reads: tensor names (whole tensor) or (name, bytes) for a part;
        writes: new tensor names (allocated and written whole), (name,
        bytes) for an in-place update of part of a live tensor, or (name,
        bytes, True) for a new tensor allocated whole of which this op
        writes `bytes`."""
        r = [(t, self.size[t]) if isinstance(t, str) else t for t in reads]
        w = []
        for t in writes:
            if isinstance(t, str):
                w.append((t, self.size[t], True))
            else:
                w.append((t[0], t[1], len(t) > 2 and t[2]))
        self.ops.append((typ, r, w))

    def mm(self, typ, M, Kd, N, reads, writes, count=1, ks=None):
        """A matrix product (M x Kd) . (Kd x N), `count` of them: 2*M*Kd*N
        flops each.  ks: the reduction length of each distinct product the
        op performs (default: the one product's Kd); the op's k is their
        sum."""
        self.op(typ, reads, writes)
        self.flops[typ] = self.flops.get(typ, 0) + count * 2 * M * Kd * N
        self.kred[typ] = self.kred.get(typ, 0) + sum(ks if ks is not None else (Kd,))

    def bytes_by_type(self):
        out = {}
        for typ, r, w in self.ops:
            out[typ] = out.get(typ, 0) + sum(b for _, b in r) + sum(b for _, b, _ in w)
        return out

    def peak(self):
        """Live from creation until last use; the peak is sampled after an
        op's outputs are allocated and before its dead inputs are freed; a
        tensor nothing reads dies with the op that makes it."""
        last = {}
        for i, (_, r, w) in enumerate(self.ops):
            for t, *_ in r + w:
                last[t] = i
        live = sum(self.size[t] for t in self.initial)
        peak = live
        for i, (_, r, w) in enumerate(self.ops):
            live += sum(self.size[t] for t, _, new in w if new)
            peak = max(peak, live)
            dead = {t for t, *_ in r + w if last[t] == i and t not in self.keep}
            live -= sum(self.size[t] for t in dead)
        return peak


def gpt_rank_program(L, d, a, s, V, F, B, e, H, train):
    """One tensor-parallel rank of a one-stage GPT (D = P = K = 1)."""
    T = B * s
    dH, FH, aH, Vh = d // H, F // H, a // H, -(-V // H)
    act, qkv, oh, s2, ff = e * T * d, e * T * 3 * dH, e * T * dH, e * B * aH * s * s, e * T * FH
    logit = e * T * Vh
    p = Prog()
    # weights of this rank (no biases, no LayerNorm parameters)
    shapes = {"E": Vh * d, "Wh": d * Vh}
    for l in range(L):
        shapes.update({"Wqkv%d" % l: d * 3 * dH, "Wo%d" % l: dH * d, "W1%d" % l: d * FH, "W2%d" % l: FH * d})
    for w, n in shapes.items():
        p.tensor(w, e * n, keep=True, initial=True)
    p.tensor("ids", 4 * T, initial=True)              # token ids, int32
    if train:
        p.tensor("tgt", 4 * T, initial=True)          # target ids, int32

    def ar(name):
        # all-reduce over the H ranks, in place; a collective's bytes are
        # its message, the tensor once
        if H > 1:
            p.op("AR_TP", [name], [(name, 0)])

    # forward
    p.tensor("x0", act)
    p.op("EMBED", ["ids", ("E", act)], ["x0"])        # gathers T rows of the table
    ar("x0")
    for l in range(L):
        x, n = "x%d" % l, lambda t: "%s%d" % (t, l)
        for t, sz in (("y1", act), ("qkv", qkv), ("sc", s2), ("p", s2), ("o", oh), ("a", act), ("x2", act),
                      ("y2", act), ("u", ff), ("g", ff), ("f", act)):
            p.tensor(n(t), sz)
        p.tensor("x%d" % (l + 1), act)
        p.op("LN", [x], [n("y1")])
        p.mm("QKV", T, d, 3 * dH, [n("y1"), n("Wqkv")], [n("qkv")])
        p.mm("SCORES", s, d // a, s, [(n("qkv"), 2 * oh)], [n("sc")], count=B * aH)   # Q and K, per head
        p.op("SOFTMAX", [n("sc")], [n("p")])
        p.mm("AV", s, s, d // a, [n("p"), (n("qkv"), oh)], [n("o")], count=B * aH)    # P and V, per head
        p.mm("OUTPROJ", T, dH, d, [n("o"), n("Wo")], [n("a")])
        ar(n("a"))
        p.op("RESADD", [x, n("a")], [n("x2")])
        p.op("LN", [n("x2")], [n("y2")])
        p.mm("FC1", T, d, FH, [n("y2"), n("W1")], [n("u")])
        p.op("GELU", [n("u")], [n("g")])
        p.mm("FC2", T, FH, d, [n("g"), n("W2")], [n("f")])
        ar(n("f"))
        p.op("RESADD", [n("x2"), n("f")], ["x%d" % (l + 1)])
    xl = "x%d" % L
    p.tensor("yf", act)
    p.tensor("logits", logit)
    p.op("LN", [xl], ["yf"])
    p.mm("LMHEAD", T, d, Vh, ["yf", "Wh"], ["logits"])
    if not train:
        return p
    # backward of the loss and the head: cross entropy over the vocabulary
    # shards (3 fp32 statistics per token, all-reduced), then the gradients
    p.tensor("stats", 12 * T)
    p.tensor("dlogits", logit)
    p.tensor("dyf", act)
    p.tensor("dWh", e * d * Vh)
    p.tensor("dx%d" % L, act)
    p.op("XENT_STATS", ["logits"], ["stats"])
    ar("stats")
    p.op("XENT_GRAD", ["logits", "stats", "tgt"], ["dlogits"])
    p.mm("GEMMDX", T, Vh, d, ["dlogits", "Wh"], ["dyf"])
    ar("dyf")
    p.mm("GEMMDW", d, T, Vh, ["yf", "dlogits"], ["dWh"])
    p.op("LN_B", ["dyf", xl], ["dx%d" % L])
    for l in range(L - 1, -1, -1):
        n = lambda t: "%s%d" % (t, l)
        dout = "dx%d" % (l + 1)
        for t, sz in (("dg", ff), ("dW2", e * FH * d), ("du", ff), ("dy2", act), ("dW1", e * d * FH), ("t2", act),
                      ("dx2", act), ("do", oh), ("dWo", e * dH * d), ("dp", s2), ("dqkv", qkv), ("ds", s2),
                      ("dy1", act), ("dWqkv", e * d * 3 * dH), ("t1", act)):
            p.tensor(n(t), sz)
        p.tensor("dx%d" % l, act)
        p.mm("GEMMDX", T, d, FH, [dout, n("W2")], [n("dg")])
        p.mm("GEMMDW", FH, T, d, [n("g"), dout], [n("dW2")])
        p.op("GELU_B", [n("dg"), n("u")], [n("du")])
        p.mm("GEMMDX", T, FH, d, [n("du"), n("W1")], [n("dy2")])
        ar(n("dy2"))
        p.mm("GEMMDW", d, T, FH, [n("y2"), n("du")], [n("dW1")])
        p.op("LN_B", [n("dy2"), n("x2")], [n("t2")])
        p.op("RESADD_B", [n("t2"), dout], [n("dx2")])
        p.mm("GEMMDX", T, d, dH, [n("dx2"), n("Wo")], [n("do")])
        p.mm("GEMMDW", dH, T, d, [n("o"), n("dx2")], [n("dWo")])
        # dP, and dV into a gradient buffer of Q, K and V allocated here
        p.mm("AV_B", s, d // a, s, [n("do"), n("p"), (n("qkv"), oh)], [n("dp"), (n("dqkv"), oh, True)],
             count=2 * B * aH, ks=(d // a, s))   # dP = dO V^T (over a head's width), dV = P^T dO (over s)
        p.op("SOFTMAX_B", [n("dp"), n("p")], [n("ds")])
        p.mm("SCORES_B", s, s, d // a, [n("ds"), (n("qkv"), 2 * oh)], [(n("dqkv"), 2 * oh)],
             count=2 * B * aH, ks=(s, s))   # dQ = dS K and dK = dS^T Q in place, per head, both over s
        p.mm("GEMMDX", T, 3 * dH, d, [n("dqkv"), n("Wqkv")], [n("dy1")])
        ar(n("dy1"))
        p.mm("GEMMDW", d, T, 3 * dH, [n("y1"), n("dqkv")], [n("dWqkv")])
        p.op("LN_B", [n("dy1"), "x%d" % l], [n("t1")])
        p.op("RESADD_B", [n("t1"), n("dx2")], ["dx%d" % l])
    p.tensor("dE", e * Vh * d)
    p.op("EMBED_DW", ["dx0", "ids"], ["dE"])
    # SGD update in place (reads the weight and its gradient, writes the
    # weight): the embedding, each layer's four weights, the head
    order = [("E", "dE")] + [(w + str(l), "d" + w + str(l)) for l in range(L) for w in ("Wqkv", "Wo", "W1", "W2")]
    for w, g in order + [("Wh", "dWh")]:
        p.op("OPT", [w, g], [(w, p.size[w])])
    return p


CASES = [(2, 32, 4, 8, 101, 128, 3, 2, 1), (2, 32, 4, 8, 101, 128, 3, 2, 2), (3, 48, 6, 16, 97, 96, 2, 4, 1),
         (1, 64, 8, 4, 1000, 256, 5, 2, 4), (2, 32, 4, 32, 50, 64, 2, 2, 2)]


@pytest.mark.parametrize("train", [False, True], ids=["infer", "train"])
@pytest.mark.parametrize("case", CASES, ids=["L%d_d%d_a%d_s%d_V%d_F%d_B%d_e%d_H%d" % c for c in CASES])
def test_bytes_of_every_op_type(orc, case, train):
    L, d, a, s, V, F, B, e, H = case
    hand = gpt_rank_program(L, d, a, s, V, F, B, e, H, train).bytes_by_type()
    m = transformer(L, d, a, s, V, B, e, TRAIN_SGD if train else INFER, d_ff=F)
    r = orc.sim_strategy(m, 1, H, 1, 1, DEV)
    got = {k: v for k, v in r["bytes_by_type"].items() if v}
    # the oracle materialises every rank; the hand program is one of H equal
    # ones, and a collective is one op for all H ranks
    want = {k: (v if k == "AR_TP" else H * v) for k, v in hand.items()}
    assert got == want


@pytest.mark.parametrize("train", [False, True], ids=["infer", "train"])
@pytest.mark.parametrize("case", CASES, ids=["L%d_d%d_a%d_s%d_V%d_F%d_B%d_e%d_H%d" % c for c in CASES])
def test_matmul_flops_of_every_type(orc, case, train):
    """2*M*K*N per product, from the shapes: the forward products, the two
    products of each one's backward, and the attention products per head."""
    L, d, a, s, V, F, B, e, H = case
    hand = gpt_rank_program(L, d, a, s, V, F, B, e, H, train).flops
    m = transformer(L, d, a, s, V, B, e, TRAIN_SGD if train else INFER, d_ff=F)
    r = orc.sim_strategy(m, 1, H, 1, 1, DEV)
    for typ, v in hand.items():
        assert r["flops_by_type"][typ] == H * v, typ


@pytest.mark.parametrize("train", [False, True], ids=["infer", "train"])
@pytest.mark.parametrize("case", CASES, ids=["L%d_d%d_a%d_s%d_V%d_F%d_B%d_e%d_H%d" % c for c in CASES])
def test_matmul_reduction_lengths_of_every_type(orc, case, train):
    """The reduction length k of every product (the inner dimension of its
    operands' shapes), summed per op type: the oracle's products carry the
    k the empirical MatMul cost reads.  An op that stands for two products
    (the attention gradients) carries the sum of theirs."""
    L, d, a, s, V, F, B, e, H = case
    hand = gpt_rank_program(L, d, a, s, V, F, B, e, H, train).kred
    m = transformer(L, d, a, s, V, B, e, TRAIN_SGD if train else INFER, d_ff=F)
    r = orc.sim_strategy(m, 1, H, 1, 1, DEV)
    got = {k: v for k, v in r["k_by_type"].items() if v}
    assert got == {k: H * v for k, v in hand.items()}


@pytest.mark.parametrize("train", [False, True], ids=["infer", "train"])
@pytest.mark.parametrize("case", CASES, ids=["L%d_d%d_a%d_s%d_V%d_F%d_B%d_e%d_H%d" % c for c in CASES])
def test_single_stage_peak(orc, case, train):
    L, d, a, s, V, F, B, e, H = case
    hand = gpt_rank_program(L, d, a, s, V, F, B, e, H, train).peak()
    m = transformer(L, d, a, s, V, B, e, TRAIN_SGD if train else INFER, d_ff=F)
    r = orc.sim_strategy(m, 1, H, 1, 1, DEV)
    assert r["cand_peak"] == hand
    assert all(int(p) == hand for p in r["dev_peak"])   # every rank alike
