"""Readings of Algorithm 1 (Sec. 3) in the oracle's interpreter, pinned on
small programs whose interpretation follows from the definition by hand.

Abstract-only interpretation: a concrete value is replaced by its type as
soon as it appears, typed on the device of the op's abstract arguments; an
op whose results are all abstract keeps them as they are, so a collective
over tensors of several devices interprets in both modes, each result on its
own input's device.  The type of a concrete value is Int32 for integer
(shape) arithmetic, as Fig. 4 prints it, and Float64 for a floating-point
value, the precision it is computed in."""
from oracle import interp

SRC = """
func f(%a: Tensor[Float16, (4, 6), 0], %b: Tensor[Float16, (4, 6), 1])
%s = Shape(%a)
%a1, %b1 = AllReduce(%a, %b)
%r = Relu(%b1)
"""


def _env(mixed):
    return {o: interp.show(v) for outs, res in interp.interpret(SRC, mixed=mixed) for o, v in zip(outs, res)}


def test_collective_results_keep_their_devices():
    for mixed in (True, False):
        env = _env(mixed)
        assert env["%a1"] == "Tensor[Float16, (4, 6), 0]"
        assert env["%b1"] == "Tensor[Float16, (4, 6), 1]"
        assert env["%r"] == "Tensor[Float16, (4, 6), 1]"


def test_concrete_results_take_their_type_on_the_argument_device():
    assert _env(True)["%s"] == [4, 6]
    assert _env(False)["%s"] == "Tensor[Int32, (2,), 0]"


def test_concrete_float_values_are_typed_float64():
    src = """
func g(%a: Tensor[Float16, (4, 6), 0])
%c = Constant[value = 0.5]()
%v = Constant[value = [0.5, 2.0]]()
%s = Shape(%a)
%h = Cast[to = "Float32"](%s)
"""
    env = {o: interp.show(v) for outs, res in interp.interpret(src, mixed=False) for o, v in zip(outs, res)}
    assert env["%c"] == "Float64" and env["%v"] == "Tensor[Float64, (2,), None]"
    assert env["%h"] == "Tensor[Float32, (2,), 0]"
    env = {o: interp.show(v) for outs, res in interp.interpret(src, mixed=True) for o, v in zip(outs, res)}
    assert env["%c"] == 0.5 and env["%h"] == [4.0, 6.0]
