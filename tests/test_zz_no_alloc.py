"""muon_step_static (the entry point that allocates nothing) against
muon_step, through the C ABI: two calls in a row, the second on a smaller
plan, each bitwise equal to muon_step's W and M on the same inputs; plans
too large for the static workspace are refused before anything runs."""
import ctypes

import pytest
import torch

from paper_2606_27153_amd import _lib as L
from paper_2606_27153_amd.optim import MuonPlan
from paper_2606_27153_amd.workloads import custom_workload, make_grads, make_state

pytestmark = pytest.mark.gpu

KW = dict(lr=0.02, momentum=0.95, weight_decay=0.01, ns_steps=5)


def _static_step(lib, plan, params, grads, moms, stream):
    return lib.muon_step_static(plan.handle, L.ptr_array([t.data_ptr() for t in params]),
                                L.ptr_array([t.data_ptr() for t in grads]),
                                L.ptr_array([t.data_ptr() for t in moms]), KW["lr"], KW["momentum"],
                                KW["weight_decay"], KW["ns_steps"], 1, ctypes.c_void_p(stream))


def _compare(shapes, seed, steps=2):
    lib = L.load()
    dev = "cuda:0"
    wl = custom_workload(shapes, seed=seed)
    descs = [(m.rows, m.cols, m.param, m.grad) for m in wl.matrices]
    ref, stat = MuonPlan(descs), MuonPlan(descs)
    assert stat.workspace_bytes <= L.MUON_STATIC_WORKSPACE_BYTES
    pa, ma = make_state(torch, wl, dev)
    pb, mb = make_state(torch, wl, dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    for step in range(steps):
        g = make_grads(torch, wl, step, dev)
        ref.step(pa, g, ma, **KW)
        st = _static_step(lib, stat, pb, g, mb, stream)
        assert st == L.MUON_OK, L.last_error()
        torch.cuda.synchronize()
        for x, y in zip(pa + ma, pb + mb):
            assert torch.equal(x, y), f"step {step}"
    ref.close()
    stat.close()


def test_static_workspace_step_matches_muon_step_twice():
    # first call: Eq. 2 and Gram-space matrices, several kernel classes;
    # second call: a smaller plan that reuses the same array
    _compare([(256, 1024), (1024, 256), (384, 384), (64, 300), (512, 1100)], seed=61)
    _compare([(96, 160), (300, 700)], seed=62)


def test_static_workspace_refuses_a_plan_that_does_not_fit():
    lib = L.load()
    dev = "cuda:0"
    plan = MuonPlan([(4096, 4096, "bf16", "bf16")])
    assert plan.workspace_bytes > L.MUON_STATIC_WORKSPACE_BYTES
    wl = custom_workload([(4096, 4096)], seed=63)
    p, m = make_state(torch, wl, dev)
    g = make_grads(torch, wl, 0, dev)
    before = p[0].clone()
    st = _static_step(lib, plan, p, g, m, torch.cuda.current_stream(dev).cuda_stream)
    assert st == L.MUON_ERR_WORKSPACE_TOO_SMALL and "static workspace" in L.last_error()
    torch.cuda.synchronize()
    assert torch.equal(p[0], before)
    plan.close()
