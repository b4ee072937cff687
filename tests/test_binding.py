"""The Python binding refuses tensors that do not match what the library
reads or writes (dtype, shape, layout, device) before any call reaches it:
a mismatch would make a kernel read or write out of bounds.  CPU only: the
tensors here are CPU or meta tensors and no call reaches the GPU."""
import pytest
import torch

from paper_2111_05426_amd import dsim
from paper_2111_05426_amd.workloads import ALL, DeviceSpec

DEV = DeviceSpec()
N, J, ND = 10, 6, 4


def tables(n=N, j=J, device="cpu", **over):
    t = dict(code=torch.zeros((j, n), dtype=torch.int32, device=device),
             flops=torch.zeros((j, n), dtype=torch.float32, device=device),
             bytes=torch.zeros((j, n), dtype=torch.float32, device=device),
             alloc=torch.zeros((j, n), dtype=torch.int32, device=device),
             free=torch.zeros((j, n), dtype=torch.int32, device=device),
             n_ops=torch.zeros(n, dtype=torch.int32, device=device))
    t.update(over)
    return t


def results(n=N, rw=ND, device="cpu", **over):
    r = dict(makespan=torch.zeros(n, dtype=torch.float64, device=device),
             finish=torch.zeros((n, rw), dtype=torch.float64, device=device),
             peak=torch.zeros((n, rw), dtype=torch.int64, device=device),
             cand_peak=torch.zeros(n, dtype=torch.int64, device=device),
             n_ops=torch.zeros(n, dtype=torch.int64, device=device),
             walked_ops=torch.zeros(n, dtype=torch.int64, device=device),
             status=torch.zeros(n, dtype=torch.int32, device=device), row_width=rw)
    r.update(over)
    return r


def refused(fn, word):
    with pytest.raises(ValueError) as e:
        fn()
    assert word in str(e.value), str(e.value)


@pytest.mark.parametrize("device", ["cpu", "meta"])
def test_tables_call_checks_every_tensor(device):
    sim = lambda t=None, r=None, init=None, n=N, nd=ND: dsim.dsim_simulate_tables(
        t if t is not None else tables(device=device), n, nd, DEV, r if r is not None else results(device=device),
        init_live=init)
    refused(lambda: sim(n=N + 1), "shape")                                       # n_cand against the tables
    refused(lambda: sim(t=tables(device=device, flops=torch.zeros((J, N), dtype=torch.float64, device=device))),
            "dtype")
    refused(lambda: sim(t=tables(device=device, bytes=torch.zeros((J + 1, N), dtype=torch.float32, device=device))),
            "shape")
    refused(lambda: sim(t=tables(device=device, n_ops=torch.zeros(N - 1, dtype=torch.int32, device=device))),
            "shape")
    refused(lambda: sim(t=tables(device=device, alloc=torch.zeros((N, J), dtype=torch.int32, device=device).t())),
            "contiguous")
    refused(lambda: sim(init=torch.zeros((N, ND + 1), dtype=torch.int64, device=device)), "shape")
    refused(lambda: sim(r=results(device=device, makespan=torch.zeros(N - 1, dtype=torch.float64, device=device))),
            "shape")
    refused(lambda: sim(r=results(rw=ND - 1, device=device)), "row_width")
    refused(lambda: sim(r=results(device=device, status=torch.zeros(N, dtype=torch.int64, device=device))), "dtype")
    refused(lambda: sim(), "GPU")                                                # everything right but the device


@pytest.mark.parametrize("device", ["cpu", "meta"])
def test_parametric_call_checks_every_tensor(device):
    w = ALL["gpt2_small"]
    cand = torch.ones((N, 4), dtype=torch.int32, device=device)
    ws = torch.zeros(dsim.dsim_parametric_workspace(N), dtype=torch.uint8, device=device)
    sim = lambda c=cand, r=None, wsp=ws: dsim.dsim_simulate_parametric(
        w.model, c, w.device, r if r is not None else results(device=device), workspace=wsp)
    refused(lambda: sim(c=torch.ones((N, 3), dtype=torch.int32, device=device)), "shape")
    refused(lambda: sim(c=torch.ones((N, 4), dtype=torch.int64, device=device)), "dtype")
    refused(lambda: sim(r=results(n=N + 1, device=device)), "shape")
    refused(lambda: sim(wsp=ws[:-1]), "elements")
    refused(lambda: sim(), "GPU")


@pytest.mark.parametrize("device", ["cpu", "meta"])
def test_argmin_and_generator_check_every_tensor(device):
    mk = torch.zeros(N, dtype=torch.float64, device=device)
    pk = torch.zeros(N, dtype=torch.int64, device=device)
    st = torch.zeros(N, dtype=torch.int32, device=device)
    ws = torch.zeros(max(dsim.dsim_argmin_workspace(N, 4), 16), dtype=torch.uint8, device=device)
    idx = torch.zeros(4, dtype=torch.int64, device=device)
    om = torch.zeros(4, dtype=torch.float64, device=device)
    f = torch.zeros(1, dtype=torch.int32, device=device)
    refused(lambda: dsim.dsim_argmin(mk, pk[:-1], st, 0, 4, ws, idx, om, f), "shape")
    refused(lambda: dsim.dsim_argmin(mk, pk, st, 0, 5, ws, idx, om, f), "elements")
    refused(lambda: dsim.dsim_argmin(mk, pk, st.to(torch.int64), 0, 4, ws, idx, om, f), "dtype")
    refused(lambda: dsim.dsim_argmin(mk, pk, st, 0, 4, ws, idx, om, f), "GPU")
    t = tables(device=device)
    refused(lambda: dsim.dsim_generate_random_tables(0, N, J + 1, ND, t), "shape")
    refused(lambda: dsim.dsim_generate_random_tables(0, N, J, ND, t), "GPU")
