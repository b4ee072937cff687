"""The allocation-free entry point dsim_simulate_parametric_static, through
the C ABI, against dsim_simulate_parametric (caller workspace, second
stream) on the same inputs: every output bit for bit, on two calls in a row
whose second is smaller (the fixed scratch keeps the first call's
contents), and the size limit refused on the host."""
import ctypes as C

import numpy as np
import pytest

from paper_2111_05426_amd.workloads import ALL, DeviceSpec

pytestmark = pytest.mark.gpu

KEYS = ("makespan", "finish", "peak", "cand_peak", "n_ops", "walked_ops", "status")


@pytest.fixture(scope="module")
def torch_gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    from paper_2111_05426_amd import dsim
    dsim.lib()
    return torch


def static_call(torch, w, strat, rw):
    """The new entry point through the raw C ABI."""
    from paper_2111_05426_amd import dsim
    cand = torch.from_numpy(np.ascontiguousarray(strat, np.int32)).cuda()
    r = dsim.alloc_results(len(strat), rw)
    for k in KEYS:
        r[k].fill_(-7)            # stale values must be overwritten
    m, d, res = dsim.model_struct(w.model), dsim.device_model(w.device), dsim._results(r)
    rc = dsim.lib().dsim_simulate_parametric_static(C.byref(m), C.c_void_p(cand.data_ptr()), len(strat), C.byref(d),
                                                    C.byref(res), C.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == dsim.DSIM_OK, dsim.dsim_last_error()
    torch.cuda.synchronize()
    return {k: r[k].cpu().numpy() for k in KEYS}


def regular_call(torch, w, strat, rw):
    from paper_2111_05426_amd import dsim
    cand = torch.from_numpy(np.ascontiguousarray(strat, np.int32)).cuda()
    r = dsim.alloc_results(len(strat), rw)
    dsim.dsim_simulate_parametric(w.model, cand, w.device, r, workspace=dsim.alloc_parametric_workspace(len(strat)),
                                  side_stream=torch.cuda.Stream())
    torch.cuda.synchronize()
    return {k: r[k].cpu().numpy() for k in KEYS}


@pytest.mark.parametrize("first,second", [("gpt3_175b", "gpt2_small_train"), ("gpt3_175b_zero", "large_mlp")])
def test_static_matches_workspace_entry_two_calls(torch_gpu, first, second):
    from paper_2111_05426_amd import dsim
    for name in (first, second):
        w = ALL[name]
        strat = dsim.dsim_create_grid(w.model, w.grid)
        rw = int(strat[:, 2].max())
        print("%s: %d strategies" % (name, len(strat)), flush=True)
        a = static_call(torch_gpu, w, strat, rw)
        b = regular_call(torch_gpu, w, strat, rw)
        for k in KEYS:
            assert np.array_equal(a[k], b[k]), (name, k)
        assert np.any(a["status"] == 0)


def test_static_smaller_subset_after_full_grid(torch_gpu):
    """A grid, then every fifth strategy of it in reverse order."""
    from paper_2111_05426_amd import dsim
    w = ALL["gpt3_175b_recompute"]
    strat = dsim.dsim_create_grid(w.model, w.grid)
    full = static_call(torch_gpu, w, strat, 64)
    sub = strat[::-5]
    part = static_call(torch_gpu, w, sub, 64)
    ref = regular_call(torch_gpu, w, sub, 64)
    for k in KEYS:
        assert np.array_equal(part[k], ref[k]), k
        assert np.array_equal(part[k], full[k][::-5]), k


def test_static_limits(torch_gpu):
    from paper_2111_05426_amd import dsim
    w = ALL["gpt3_175b"]
    m, d = dsim.model_struct(w.model), dsim.device_model(w.device)
    res = dsim.dsim_results()
    res.makespan = res.cand_peak = res.status = 8
    res.row_width = 64
    fake = C.c_void_p(16)   # never dereferenced: refused before any launch
    L = dsim.lib()
    assert L.dsim_simulate_parametric_static(C.byref(m), fake, (1 << 20) + 1, C.byref(d), C.byref(res),
                                             None) == dsim.DSIM_ERANGE
    assert "2^20" in dsim.dsim_last_error() or "1048576" in dsim.dsim_last_error()
    assert L.dsim_simulate_parametric_static(C.byref(m), None, 0, C.byref(d), C.byref(res), None) == dsim.DSIM_OK
    # the largest call: 2^20 strategies (the GPT-3 grid repeated)
    strat = dsim.dsim_create_grid(w.model, w.grid)
    big = np.resize(strat, (1 << 20, 4))
    a = static_call(torch_gpu, w, big, 64)
    assert np.array_equal(a["makespan"][:len(strat)], a["makespan"][len(strat):2 * len(strat)])
    b = regular_call(torch_gpu, w, big, 64)
    for k in KEYS:
        assert np.array_equal(a[k], b[k]), k
