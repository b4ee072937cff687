"""The program front end (mixed abstract/concrete interpretation, Sec. 3.3)
and its oracle, on the CPU: the front end is host C++ in libdsim
(dsim_interpret_program, dsim_lower_programs), called through its binding.

Pins: Fig. 4's two printed interpretations of the GPT-2 Reshape snippet
(tests/golden/fig4_reshape.json) for both interpreters, and table records
derived by hand.  Parity: the front end's tables, simulated by the oracle's
table simulator, against the oracle's own interpretation simulated as a
program over tensors (def/use liveness) -- the two share no code -- on the
GPT-2-shaped programs and on random programs (tests/random_programs.py).
"""
import ctypes as C
import json
import math
import os
from dataclasses import replace

import numpy as np
import pytest

from oracle import interp
from paper_2111_05426_amd import dsim
from paper_2111_05426_amd import frontend as fe
from paper_2111_05426_amd import programs
from paper_2111_05426_amd.workloads import DeviceSpec

GOLD = os.path.join(os.path.dirname(__file__), "golden", "fig4_reshape.json")


def fig4():
    with open(GOLD) as f:
        return json.load(f)


@pytest.mark.parametrize("mixed", [False, True])
def test_fig4_front_end(mixed):
    g = fig4()
    state = fe.interpret(g["program"], g["concrete_inputs"], mixed=mixed)
    got = [state[v] for v in g["variables"]]
    assert got == g["mixed" if mixed else "abstract_only"]


@pytest.mark.parametrize("mixed", [False, True])
def test_fig4_oracle(mixed):
    g = fig4()
    steps = interp.interpret(g["program"], g["concrete_inputs"], mixed=mixed)
    env = {o: v for outs, res in steps for o, v in zip(outs, res)}
    first = g["mixed"][0] if mixed else g["abstract_only"][0]   # the input itself
    got = [first] + [interp.show(env[v]) for v in g["variables"][1:]]
    assert got == g["mixed" if mixed else "abstract_only"]


def test_fig4_gemm_needs_the_mixed_domain():
    """Only the mixed interpretation knows the Gemm's input shape, so only
    it can cost the Gemm (Sec. 3.3)."""
    g = fig4()
    p = g["program"]
    with pytest.raises(ValueError, match="unknown"):
        fe.lower(p, {})                                  # %3114 left abstract
    t = fe.lower(p, g["concrete_inputs"])
    m, k, n = 2048, 768, 3072
    assert list(t["flops"]) == [256 * 8 * 768, 2 * m * k * n]
    assert list(t["code"] >> 24) == [0, 1]               # the Gemm is a matrix product


def test_records_by_hand():
    """A two-device program: its records, written out by hand.  Float32
    (4 bytes); x (8 x 16) on device 0, w (16 x 4) kept."""
    src = """
func f(%x: Tensor[Float32, (8, 16), 0], %w: Tensor[Float32, (16, 4), 0] keep, %v: Tensor[Float32, (8, 4), 1])
%s = Shape(%x)                          # host
%y = Gemm(%x, %w)                       # 2*8*16*4 flops; x dies here
%r = Relu(%y)                           # y dies
%r1 = Send[device = 1](%r)              # r dies on 0, r1 lives on 1
%t = Add(%r1, %v)                       # r1, v die; t is never read
%a0, %a1 = AllReduce(%t, %t)
return %a0
"""
    with pytest.raises(ValueError, match="distinct devices"):
        fe.lower(src)
    src = src.replace("%a0, %a1 = AllReduce(%t, %t)", "%z = Send[device = 0](%t)\n%u = Relu(%z)")
    t = fe.lower(src)
    x, w, y, v = 8 * 16 * 4, 16 * 4 * 4, 8 * 4 * 4, 8 * 4 * 4
    assert list(t["init_live"]) == [x + w, v]
    assert list(t["code"]) == [0 | 1 << 24, 0, 1 | 0 << 8 | 1 << 16, 1 << 8, 1 | 1 << 8 | 0 << 16, 0]
    assert list(t["flops"]) == [2 * 8 * 16 * 4, 8 * 4, 0, 8 * 4, 0, 8 * 4]
    assert list(t["bytes"]) == [x + w + y, 2 * y, y, 3 * y, y, 2 * y]
    assert list(t["alloc"]) == [y, y, y, y, y, y]
    assert list(t["free"]) == [x, y, y, y + v, y, y + y]


def test_views_share_memory_and_collectives_work_in_place():
    src = """
func f(%a: Tensor[Float16, (4, 6), 0], %b: Tensor[Float16, (4, 6), 1])
%c = Constant[value = [24]]()
%av = Reshape(%a, %c)
%bv = Reshape(%b, %c)
%a1, %b1 = AllReduce(%av, %bv)
%x = Relu(%a1)
return %x
"""
    t = fe.lower(src)
    assert list(t["code"]) == [2 | 0b11 << 16, 0]
    # a is read after the all-reduce and freed by the Relu; b's last reader
    # is the all-reduce, so b stays live
    assert list(t["alloc"]) == [0, 48] and list(t["free"]) == [0, 48 + 48]


@pytest.mark.parametrize("bad, msg", [
    ("%y = Add(%x, %v)", "different devices"),
    ("%y = Send[device = 0](%x)", "own device"),
    ("%y = Send[device = 1](%x)", "nothing reads"),
    ("%y = Gemm(%x, %x)", "Gemm"),
])
def test_errors(bad, msg):
    src = "func f(%x: Tensor[Float32, (8, 16), 0], %v: Tensor[Float32, (8, 16), 1])\n" + bad + "\n"
    with pytest.raises(ValueError, match=msg):
        fe.lower(src)


def test_dispatch_prefers_the_most_precise_implementation():
    """Reshape has a concrete, a mixed and an abstract implementation: a
    concrete input and target give a concrete array, a tensor and a concrete
    target a tensor of known shape, a tensor and an abstract target a tensor
    of unknown shape."""
    src = """
func f(%t: Tensor[Float32, (4, 6), 0], %c: Tensor[Int64, (24,), 0], %s: Tensor[Int32, (2,), 0])
%a = Reshape(%t, %s)
%z = Constant[value = [4, -1]]()
%b = Reshape(%c, %z)
"""
    st = fe.interpret(src, {"%s": [2, 12]})
    assert st["%a"] == "Tensor[Float32, (2, 12), 0]"
    assert st["%b"] == "Tensor[Int64, (4, 6), 0]"
    st = fe.interpret(src)
    assert st["%a"] == "Tensor[Float32, ??, 0]"
    st = fe.interpret(src, {"%s": [2, 12], "%c": list(range(24))})
    assert st["%b"] == np.arange(24).reshape(4, 6).tolist()


DEVICES = [DeviceSpec(), DeviceSpec(matmul=(5.2e-6, 1.1e-15, 2.3e-13)),
           DeviceSpec(network=(2, 4.9e10, 1.1e-5)),
           DeviceSpec(streams=(2, math.inf, 0.0), network=(1, 4.9e10, 1.1e-5)),
           # the reduction-length term and a floor that binds on small products
           DeviceSpec(matmul=(1.3e-6, 6.7e-16, 1.7e-13, 2.6e-9, 1.5e-5))]


@pytest.mark.parametrize("dev", range(len(DEVICES)))
@pytest.mark.parametrize("shape", [(1, 64, 1, 1), (3, 128, 2, 2), (8, 256, 4, 2), (5, 96, 2, 1), (2, 512, 1, 4)])
def test_front_end_matches_oracle(orc, shape, dev):
    B, S, tp, pp = shape
    d = DEVICES[dev]
    src = programs.gpt2_layers(B, S, n_layers=4, tp=tp, pp=pp)
    t = fe.lower(src, {"%flat": [-1]})
    assert t["n_dev"] == tp * pp
    a = orc.sim_table(t, t["n_dev"], d, init_live=t["init_live"])
    b = interp.simulate(src, d, {"%flat": [-1]})
    assert a["status"] == 0
    assert list(a["finish"]) == list(b["finish"])
    assert [int(v) for v in a["peak"]] == [int(v) for v in b["peak"]]


def test_pack():
    ts = [fe.lower(programs.gpt2_layers(B, 64), {"%flat": [-1]}) for B in (1, 2, 3)]
    p = fe.pack(ts)
    assert p["code"].shape == (max(len(t["code"]) for t in ts), 3)
    for c, t in enumerate(ts):
        n = len(t["code"])
        assert p["n_ops"][c] == n and np.array_equal(p["code"][:n, c], t["code"])
        assert np.array_equal(p["init_live"][c], t["init_live"])


# ---------------------------------------------------------------------------
# random programs: the front end against the oracle's interpreter
# ---------------------------------------------------------------------------
from random_programs import random_program  # noqa: E402

RAND = [(seed, 40) for seed in range(120)] + [(1000 + seed, 150) for seed in range(24)]


def _oracle_state(src, mixed):
    return {o: interp.show(v) for outs, res in interp.interpret(src, mixed=mixed) for o, v in zip(outs, res)}


@pytest.mark.parametrize("chunk", range(8))
def test_random_programs_interpret_like_the_oracle(chunk):
    for seed, n in RAND[chunk::8]:
        src = random_program(seed, n_ops=n)
        for mixed in (True, False):
            got = fe.interpret(src, mixed=mixed)
            for name, v in _oracle_state(src, mixed).items():
                assert got[name] == v, (seed, mixed, name)


@pytest.mark.parametrize("chunk", range(8))
def test_random_programs_simulate_like_the_oracle(orc, chunk):
    for seed, n in RAND[chunk::8]:
        src = random_program(seed, n_ops=n)
        t = fe.lower(src)
        for d in (DEVICES[0], DEVICES[1], DEVICES[3], DEVICES[4]):
            a = orc.sim_table(t, t["n_dev"], d, init_live=t["init_live"])
            b = interp.simulate(src, d)
            assert a["status"] == 0, seed
            assert list(a["finish"]) == list(b["finish"]), seed
            assert [int(v) for v in a["peak"]] == [int(v) for v in b["peak"]], seed


# ---------------------------------------------------------------------------
# batches, threads, the sizing pass and the format's limits
# ---------------------------------------------------------------------------
def _batch_texts():
    return [programs.gpt2_layers(B, S, n_layers=2, tp=tp, pp=pp) for B, S, tp, pp in
            ((1, 64, 1, 1), (3, 128, 2, 2), (2, 96, 4, 2), (5, 64, 2, 1))] + \
           [random_program(s, n_ops=30, n_dev=3) for s in range(6)]


def test_batch_equals_single_programs_and_threads_agree():
    texts = _batch_texts()
    inputs = [{"%flat": [-1]} if "%flat" in t else {} for t in texts]
    ref = fe.pack([fe.lower(t, i, n_dev=8) for t, i in zip(texts, inputs)])
    for threads in (1, 3, 8, 64):
        got = fe.lower_batch(texts, inputs, n_dev=8, threads=threads)
        for k in ("code", "flops", "bytes", "alloc", "free", "n_ops", "init_live"):
            assert np.array_equal(got[k], ref[k]), (threads, k)


def _raw(texts, n_dev=8, max_ops=512, arrays=True, threads=1):
    L = dsim.lib()
    n = len(texts)
    progs = (C.c_char_p * n)(*[t.encode() for t in texts])
    arr = dict(code=np.full((max_ops, n), 7, np.uint32), flops=np.zeros((max_ops, n), np.float32),
               bytes=np.zeros((max_ops, n), np.float32), alloc=np.zeros((max_ops, n), np.uint32),
               free=np.zeros((max_ops, n), np.uint32), mm_k=np.zeros((max_ops, n), np.uint32),
               n_ops=np.full(n, 99, np.uint32), init_live=np.zeros((n, n_dev), np.uint64))
    ptrs = [arr[k].ctypes.data if arrays else None for k in ("code", "flops", "bytes", "alloc", "free", "mm_k",
                                                              "n_ops", "init_live")]
    used, devs = C.c_int32(-1), C.c_int32(-1)
    rc = L.dsim_lower_programs(C.cast(progs, C.c_void_p), None, n, n_dev, max_ops, *ptrs, C.byref(used),
                               C.byref(devs), threads)
    return rc, used.value, devs.value, arr


def test_sizing_pass_and_enospc():
    texts = [random_program(s, n_ops=30, n_dev=2) for s in range(5)]
    ref = fe.lower_batch(texts, n_dev=8)
    need = int(ref["n_ops"].max())
    rc, used, devs, _ = _raw(texts, arrays=False)
    assert rc == 0 and used == need and devs == 2
    for threads in (1, 4):
        rc, used, devs, arr = _raw(texts, max_ops=need - 1, threads=threads)
        assert rc == dsim.DSIM_ENOSPC and used == need
        assert "max_ops" in dsim.dsim_last_error()
        fits = ref["n_ops"] <= need - 1
        assert np.array_equal(arr["n_ops"][fits], ref["n_ops"][fits]) and not arr["n_ops"][~fits].any()
    rc, used, devs, arr = _raw(texts, max_ops=need + 3)
    assert rc == 0
    assert np.array_equal(arr["code"][:need], ref["code"]) and not arr["code"][need:].any()


@pytest.mark.parametrize("src, code, msg", [
    ("func f(%x: Tensor[Float32, (4,), 8])\n%y = Relu(%x)\n", dsim.DSIM_ERANGE, "n_dev"),
    # 2^24 + 1 elements of Float32 bytes are exact, their flops (2^24 + 1) are not
    ("func f(%x: Tensor[Float32, (16777217,), 0])\n%y = Relu(%x)\n", dsim.DSIM_ERANGE, "exactly"),
    ("func f(%x: Tensor[Float32, (65536, 65536), 0])\n%y = Relu(%x)\n", dsim.DSIM_ERANGE, "exactly"),
    ("func f(%x: Tensor[Float32, (4,), 0])\n%y = Relu(%z)\n", dsim.DSIM_EINVAL, "line 2: %z is not defined"),
    ("func f(%x: Tensor[Float32, (4,), 0])\n%x = Relu(%x)\n", dsim.DSIM_EINVAL, "defined twice"),
    ("func f(%x: Tensor[Float32, (4,), 0])\n%y = Frobnicate(%x)\n", dsim.DSIM_EINVAL, "no implementation"),
    ("%y = Relu(%x)\n", dsim.DSIM_EINVAL, "before the function header"),
    ("func f(%x: Tensor[Float33, (4,), 0])\n", dsim.DSIM_EINVAL, "element type"),
    ("func f(%x: Tensor[Float32, (4,), 0])\n%y = Reshape(%x, %x)\n%z = Relu(%y)\n", dsim.DSIM_EINVAL, "unknown"),
    ("func f(%x: Tensor[Float32, (4, 6), 0])\n%c = Constant[value = [5, -1]]()\n%y = Reshape(%x, %c)\n",
     dsim.DSIM_EINVAL, "cannot reshape"),
    ("func f(%x: Tensor[Float32, (4, 6), 0])\n%a, %b = Split[axis = 1, split = [2, 2]](%x)\n", dsim.DSIM_EINVAL,
     "does not cover"),
])
def test_refusals(src, code, msg):
    rc, _, _, _ = _raw([src])
    assert rc == code
    assert msg in dsim.dsim_last_error()
    with pytest.raises(ValueError, match="program 0"):
        fe.lower_batch([src])


def test_error_names_the_first_failing_program_whatever_the_threads():
    good = random_program(5, n_ops=20, n_dev=2)
    bad = "func f(%x: Tensor[Float32, (4,), 0])\n%y = Relu(%q)\n"
    texts = [good] * 5 + [bad] + [good] * 3 + [bad] + [good] * 6
    for threads in (1, 2, 5, 16):
        rc, _, _, _ = _raw(texts, threads=threads)
        assert rc == dsim.DSIM_EINVAL and dsim.dsim_last_error().startswith("program 5: line 2")


def test_matmul_records_carry_their_reduction_length():
    """MatMul: the left operand's last dimension (batched too); Gemm: the
    shared dimension, transposed or not; every other record 0."""
    src = """
func f(%x: Tensor[Float32, (8, 16), 0], %w: Tensor[Float32, (16, 4), 0] keep, %b: Tensor[Float32, (3, 5, 7), 0], %c: Tensor[Float32, (3, 7, 2), 0], %v: Tensor[Float32, (4, 16), 0] keep)
%y = Gemm(%x, %w)
%r = Relu(%y)
%z = MatMul(%b, %c)
%t = Transpose[perm = [1, 0]](%x)
%u = Gemm[transA = 1, transB = 1](%t, %v)
"""
    t = fe.lower(src)
    assert list(t["code"] >> 24) == [1, 0, 1, 0, 1]
    assert list(t["mm_k"]) == [16, 0, 7, 0, 16]
