"""The size rule of the transform's integer arithmetic, in the oracle.

Every size product the transform forms (an op's flops, bytes, allocation or
free) and every live-byte count must fit 64-bit integers; the rule (Q and Z
below 2^62, at most 65,536 layers, at most 2^24 devices per strategy) is a
precondition that both implementations check before simulating.  Pins:

* it admits every model the paper simulates (Table 1: the MLPs of Sec. 4 in
  training, the GPT-2 shapes in inference at every batch size of the grid,
  Sec. 5.1) and every workload of this project;
* it rejects models for which one of the transform's exact products -- the
  dense layer's Gemm flops 2·B·d², the attention P·V gradient flops
  4·B·s²·d (Sec. 4 shapes) -- reaches 2^63, computed here with Python's
  unbounded integers, and admits the same models one power of two below;
* growing any dimension never brings a rejected model back.
"""
from dataclasses import replace

import pytest

from paper_2111_05426_amd.workloads import (ALL, DeviceSpec, INFER, TRAIN_ADAM, TRAIN_ADAM_MIXED, TRAIN_SGD, mlp,
                                            transformer)

DEV = DeviceSpec()
I63 = 2 ** 63


def test_admits_the_papers_models(orc):
    # Table 1: MLP 1B / 17B / 103B training (16 x 8192, 64 x 16384,
    # 96 x 32768, fp16) and the GPT-2 1.6B / 13B / 175B shapes in inference
    # at every batch of the 1035-configuration grid (2^7 .. 2^20 sequences)
    for L, d in ((16, 8192), (64, 16384), (96, 32768)):
        assert orc.model_size_ok(mlp(L, d, 65536, 2, TRAIN_ADAM))
    for L, d, a in ((48, 1600, 25), (40, 5120, 40), (96, 12288, 96)):
        for e in range(7, 21):
            assert orc.model_size_ok(transformer(L, d, a, 1024, 50257, 2 ** e, 2, INFER))


@pytest.mark.parametrize("name", sorted(k for k, w in ALL.items() if w.model is not None))
def test_admits_every_workload(orc, name):
    assert orc.model_size_ok(ALL[name].model)


@pytest.mark.parametrize("mode", [INFER, TRAIN_SGD, TRAIN_ADAM_MIXED])
def test_mlp_gemm_flops_bound(orc, mode):
    d = 2 ** 20
    for B, fits in ((2 ** 20, True), (2 ** 22, False)):
        m = mlp(1, d, B, 2, mode)
        assert (2 * B * d * d < I63) == fits       # the Gemm's exact flop count
        assert orc.model_size_ok(m) == fits
    # between the two: 2^62 flops is still an int64, but the rule keeps a
    # factor of two of room
    assert 2 * 2 ** 21 * d * d < I63 and not orc.model_size_ok(mlp(1, d, 2 ** 21, 2, mode))


def test_attention_gradient_flops_bound(orc):
    base = transformer(96, 12288, 96, 2048, 50257, 1536, 2, TRAIN_ADAM_MIXED)
    assert orc.model_size_ok(base)
    long = replace(base, seq_len=2 ** 20)
    B, s, d = long.global_batch, long.seq_len, long.d_model
    assert 4 * B * s * s * d >= I63                  # P.V gradient flops of one layer, exact
    assert not orc.model_size_ok(long)
    shorter = replace(base, seq_len=2 ** 16)
    assert 4 * B * 2 ** 16 * 2 ** 16 * d < I63
    assert orc.model_size_ok(shorter)


def test_layer_count_bound(orc):
    assert orc.model_size_ok(mlp(65536, 64, 64, 2, TRAIN_SGD))
    assert not orc.model_size_ok(mlp(65537, 64, 64, 2, TRAIN_SGD))


def test_monotone_in_every_dimension(orc):
    base = transformer(24, 1024, 16, 1024, 50257, 512, 2, TRAIN_ADAM)
    for field in ("d_model", "d_ff", "seq_len", "vocab", "global_batch"):
        ok = [orc.model_size_ok(replace(base, **{field: getattr(base, field) * 2 ** k})) for k in range(0, 48, 2)]
        assert ok[0]
        first_bad = ok.index(False) if False in ok else len(ok)
        assert not any(ok[first_bad:]), field


def test_grid_and_strategy_calls_refuse_models_beyond_the_rule(orc):
    big = mlp(1, 2 ** 20, 2 ** 22, 2, TRAIN_SGD)
    with pytest.raises(ValueError):
        orc.sim_strategy(big, 1, 1, 1, 1, DEV, slice=True)
    from paper_2111_05426_amd.workloads import GridSpec
    with pytest.raises(ValueError):
        orc.create_grid(big, GridSpec(4, 0, 0, 4))


def test_device_count_bound(orc):
    # more than 2^24 devices is not a valid strategy, however they are split
    m = mlp(4, 16, 2 ** 26, 2, TRAIN_SGD)
    for D, H, P in ((2 ** 25, 1, 1), (2 ** 23, 2, 2), (2 ** 22, 4, 4)):
        bad = orc.sim_strategy(m, D, H, P, 1, DEV, slice=True, want_devices=False)
        assert bad["status"] == orc.ST_BAD_STRATEGY
    ok = orc.sim_strategy(m, 2 ** 8, 2, 2, 1, DEV, slice=True, want_devices=False)
    assert ok["status"] == 0
