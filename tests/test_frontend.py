"""The program front end (mixed abstract/concrete interpretation, Sec. 3.3)
and its oracle, on the CPU.

Pins: Fig. 4's two printed interpretations of the GPT-2 Reshape snippet
(tests/golden/fig4_reshape.json) for both interpreters, and table records
derived by hand.  Parity: the front end's tables, simulated by the oracle's
table simulator, against the oracle's own interpretation simulated as a
program over tensors (def/use liveness) -- the two share no code.
"""
import json
import math
import os
from dataclasses import replace

import numpy as np
import pytest

from oracle import interp
from paper_2111_05426_amd import frontend as fe
from paper_2111_05426_amd import programs
from paper_2111_05426_amd.workloads import DeviceSpec

GOLD = os.path.join(os.path.dirname(__file__), "golden", "fig4_reshape.json")


def fig4():
    with open(GOLD) as f:
        return json.load(f)


def _fe_show(v):
    return v.tolist() if fe.is_concrete(v) else repr(v)


@pytest.mark.parametrize("mixed", [False, True])
def test_fig4_front_end(mixed):
    g = fig4()
    state, _ = fe.interpret(fe.parse(g["program"]), g["concrete_inputs"], mixed=mixed)
    got = [_fe_show(state[v]) for v in g["variables"]]
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
    p = fe.parse(g["program"])
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
        fe.lower(fe.parse(src))
    src = src.replace("%a0, %a1 = AllReduce(%t, %t)", "%z = Send[device = 0](%t)\n%u = Relu(%z)")
    t = fe.lower(fe.parse(src))
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
    t = fe.lower(fe.parse(src))
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
        fe.lower(fe.parse(src))


def test_dispatch_prefers_the_most_precise_implementation():
    """Reshape has a concrete, a mixed and an abstract implementation."""
    t = fe.Tensor("Float32", (4, 6), 0)
    assert fe.dispatch("Reshape", [t, np.array([2, 12])])({}, t, np.array([2, 12]))[0].shape == (2, 12)
    assert fe.dispatch("Reshape", [t, fe.Tensor("Int32", (2,), 0)])({}, t, None)[0].shape is None
    c = np.arange(24)
    assert fe.dispatch("Reshape", [c, np.array([4, -1])])({}, c, np.array([4, -1]))[0].shape == (4, 6)


DEVICES = [DeviceSpec(), DeviceSpec(matmul=(5.2e-6, 1.1e-15, 2.3e-13)),
           DeviceSpec(network=(2, 4.9e10, 1.1e-5)),
           DeviceSpec(streams=(2, math.inf, 0.0), network=(1, 4.9e10, 1.1e-5))]


@pytest.mark.parametrize("dev", range(len(DEVICES)))
@pytest.mark.parametrize("shape", [(1, 64, 1, 1), (3, 128, 2, 2), (8, 256, 4, 2), (5, 96, 2, 1), (2, 512, 1, 4)])
def test_front_end_matches_oracle(orc, shape, dev):
    B, S, tp, pp = shape
    d = DEVICES[dev]
    src = programs.gpt2_layers(B, S, n_layers=4, tp=tp, pp=pp)
    t = fe.lower(fe.parse(src), {"%flat": [-1]})
    assert t["n_dev"] == tp * pp
    a = orc.sim_table(t, t["n_dev"], d, init_live=t["init_live"])
    b = interp.simulate(src, d, {"%flat": [-1]})
    assert a["status"] == 0
    assert list(a["finish"]) == list(b["finish"])
    assert [int(v) for v in a["peak"]] == [int(v) for v in b["peak"]]


def test_pack():
    ts = [fe.lower(fe.parse(programs.gpt2_layers(B, 64)), {"%flat": [-1]}) for B in (1, 2, 3)]
    p = fe.pack(ts)
    assert p["code"].shape == (max(len(t["code"]) for t in ts), 3)
    for c, t in enumerate(ts):
        n = len(t["code"])
        assert p["n_ops"][c] == n and np.array_equal(p["code"][:n, c], t["code"])
        assert np.array_equal(p["init_live"][c], t["init_live"])
