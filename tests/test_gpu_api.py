"""GPU checks of the Python front end and the ABI extras: the torch.optim
wrapper, checkpoint/resume equivalence, launch timing, the pointer-table
refresh when buffers move, and the binding's refusal of buffers that do not
match the plan."""
import pytest
import torch

from paper_2606_27153_amd.optim import Muon, MuonPlan
from paper_2606_27153_amd.workloads import custom_workload, make_grads, make_state

pytestmark = pytest.mark.gpu

SHAPES = [(256, 768), (768, 256), (512, 512), (64, 300)]


SCHEDULE = [(3.4445, -4.7750, 2.0315)] * 3 + [(15 / 8, -10 / 8, 3 / 8)] * 2


@pytest.mark.parametrize("precision,abc", [("bf16", None), ("fp16", SCHEDULE)], ids=["bf16", "fp16-schedule"])
def test_optimizer_wrapper_matches_plan_step(precision, abc):
    wl = custom_workload(SHAPES, seed=21)
    pa, ma = make_state(torch, wl, "cuda:0")
    pb, _ = make_state(torch, wl, "cuda:0")
    params = [torch.nn.Parameter(p) for p in pb]
    opt = Muon(params, lr=0.02, momentum=0.95, weight_decay=0.01, ns_steps=5, precision=precision,
               ns_coefficients=abc)
    plan = MuonPlan([(m.rows, m.cols, m.param, m.grad) for m in wl.matrices], precision=precision, abc=abc)
    for step in range(3):
        g = make_grads(torch, wl, step, "cuda:0")
        plan.step(pa, g, ma, lr=0.02, momentum=0.95, weight_decay=0.01, ns_steps=5)
        for p, gi in zip(params, g):
            p.grad = gi.clone()
        opt.step()
    torch.cuda.synchronize()
    for x, y in zip(pa, params):
        assert torch.equal(x, y.data)
    for x, p in zip(ma, params):
        assert torch.equal(x, opt.state[p]["momentum_buffer"])
    plan.close()


def test_checkpoint_resume_is_bitwise_identical():
    wl = custom_workload(SHAPES, seed=22)
    descs = [(m.rows, m.cols, m.param, m.grad) for m in wl.matrices]
    kw = dict(lr=0.02, momentum=0.95, weight_decay=0.01, ns_steps=5)
    # uninterrupted run of 3 steps
    plan = MuonPlan(descs)
    p, m = make_state(torch, wl, "cuda:0")
    for step in range(3):
        plan.step(p, make_grads(torch, wl, step, "cuda:0"), m, **kw)
    torch.cuda.synchronize()
    # 2 steps, save W and M to host, new plan and new buffers, 3rd step
    plan2 = MuonPlan(descs)
    q, n = make_state(torch, wl, "cuda:0")
    for step in range(2):
        plan2.step(q, make_grads(torch, wl, step, "cuda:0"), n, **kw)
    torch.cuda.synchronize()
    saved = [(x.cpu(), y.cpu()) for x, y in zip(q, n)]
    plan2.close()
    del q, n
    plan3 = MuonPlan(descs)
    q = [x.cuda() for x, _ in saved]
    n = [y.cuda() for _, y in saved]
    plan3.step(q, make_grads(torch, wl, 2, "cuda:0"), n, **kw)
    torch.cuda.synchronize()
    for a, b in zip(p + m, q + n):
        assert torch.equal(a, b)
    plan.close()
    plan3.close()


def test_moved_buffers_refresh_the_pointer_table():
    wl = custom_workload(SHAPES, seed=23)
    plan = MuonPlan([(mm.rows, mm.cols, mm.param, mm.grad) for mm in wl.matrices])
    kw = dict(lr=0.02, momentum=0.95, weight_decay=0.01, ns_steps=5)
    p, m = make_state(torch, wl, "cuda:0")
    p2 = [x.clone() for x in p]
    m2 = [x.clone() for x in m]
    g = make_grads(torch, wl, 0, "cuda:0")
    plan.step(p, g, m, **kw)       # table holds p, m
    plan.step(p2, g, m2, **kw)     # different buffers: must be refreshed
    torch.cuda.synchronize()
    for a, b in zip(p + m, p2 + m2):
        assert torch.equal(a, b)
    plan.close()


@pytest.mark.parametrize("aspect", [0.0, 2.0])
def test_launch_timing_reports_every_kind(aspect):
    shapes = ((1024, 4096), (96, 300))
    wl = custom_workload(list(shapes) * 2, seed=24)
    plan = MuonPlan([(mm.rows, mm.cols, mm.param, mm.grad) for mm in wl.matrices], gram_min_aspect=aspect)
    p, m = make_state(torch, wl, "cuda:0")
    g = make_grads(torch, wl, 0, "cuda:0")
    plan.set_timing(True)
    plan.step(p, g, m, lr=0.02, momentum=0.95, weight_decay=0.01, ns_steps=5)
    plan.set_timing(False)
    stats = plan.timing_read()
    kinds = {s["kind"] for s in stats}
    gram = aspect > 0  # both shapes are at least 3x wider than tall
    # the last B*X applies the update: no apply launch when NS steps run
    assert kinds == {"momentum", "finalize", "gram", "poly", "bx"} | ({"symm"} if gram else set())
    info = plan.info()
    for s in stats:
        assert s["total_ms"] > 0
        if s["kind"] in ("gram", "poly", "bx", "symm"):
            assert s["algo_flops"] > 0
    k = 5
    if gram:   # Eq. 4: 3 m^2 n once, 4k - 3 symmetric m^3 products
        want = sum(3 * min(r, c) ** 2 * max(r, c) + (4 * k - 3) * min(r, c) ** 3 for r, c in shapes) * 2
    else:      # Eq. 2: 3 m^2 n + m^3 per step
        want = sum(3 * min(r, c) ** 2 * max(r, c) + min(r, c) ** 3 for r, c in shapes) * 2 * k
    got = sum(s["algo_flops"] for s in stats)
    assert abs(got - want) <= 1e-9 * want
    assert abs(info["ns_flops_fixed"] + k * info["ns_flops_step"] - want) <= 1e-9 * want
    # per kernel class: Eq. 2 launches Gram, A*A and B*X each step; Eq. 4 the
    # Gram product and B*X once, P_i each step and 3 (k - 1) other m^3
    # products in 2k - 1 launches (G P and P Q share one when both are due)
    per_class = {"gram": 1, "poly": k, "symm": 2 * k - 1, "bx": 1} if gram else {"gram": k, "poly": k, "bx": k}
    for s in stats:
        if s["kernel_class"] is not None:
            assert s["launches"] == per_class[s["kind"]], s
    assert plan.timing_read() == []     # records were dropped by the first read
    plan.close()


def test_step_captured_in_a_graph_matches_eager():
    # After one eager step with the same buffers (which uploads the plan's
    # pointer table), muon_step only enqueues kernels on the stream, so it
    # can be captured in a HIP graph.  Each replay, with new gradients copied
    # in eagerly between replays, must match an eager step bit for bit.
    wl = custom_workload([(256, 768), (768, 256), (300, 300), (64, 200), (512, 2048)], seed=41)
    descs = [(m.rows, m.cols, m.param, m.grad) for m in wl.matrices]
    dev = "cuda:0"
    pe, me = make_state(torch, wl, dev)
    pg, mg = make_state(torch, wl, dev)
    eager, graphed = MuonPlan(descs), MuonPlan(descs)
    we, wg = eager.workspace(dev), graphed.workspace(dev)
    ge = make_grads(torch, wl, 0, dev)
    gg = [g.clone() for g in ge]
    kw = dict(lr=0.02, momentum=0.95, weight_decay=0.01, ns_steps=5)
    eager.step(pe, ge, me, workspace=we, **kw)
    graphed.step(pg, gg, mg, workspace=wg, **kw)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        graphed.step(pg, gg, mg, workspace=wg, **kw)
    for step in range(1, 5):
        new = make_grads(torch, wl, step, dev)
        for a, b, g in zip(ge, gg, new):
            a.copy_(g)
            b.copy_(g)
        eager.step(pe, ge, me, workspace=we, **kw)
        graph.replay()
        torch.cuda.synchronize()
        for x, y in zip(pe, pg):
            assert torch.equal(x, y), f"replay {step}: params differ"
        for x, y in zip(me, mg):
            assert torch.equal(x, y), f"replay {step}: momentum differs"
    eager.close()
    graphed.close()


@pytest.mark.gpu
def test_bad_buffers_are_refused_before_launch(monkeypatch):
    import paper_2606_27153_amd.optim as O
    dev = "cuda:0"
    descs = [(96, 160, "bf16", "bf16"), (200, 64, "f32", "f32")]
    plan = MuonPlan(descs)
    params = [torch.randn(96, 160, device=dev).to(torch.bfloat16), torch.randn(200, 64, device=dev)]
    grads = [torch.randn(96, 160, device=dev).to(torch.bfloat16), torch.randn(200, 64, device=dev)]
    moms = [torch.zeros(96, 160, device=dev), torch.zeros(200, 64, device=dev)]
    kw = dict(lr=0.02, momentum=0.95, weight_decay=0.01)
    before = [p.clone() for p in params]
    bad = [params[0], torch.randn(64, 200, device=dev).t()]          # right shape, column-major
    with pytest.raises(ValueError, match="matrix 1 param is not contiguous"):
        plan.step(bad, grads, moms, **kw)
    with pytest.raises(ValueError, match="matrix 0 grad is not on a GPU"):
        plan.step(params, [grads[0].cpu(), grads[1]], moms, **kw)
    with pytest.raises(ValueError, match="matrix 1 momentum has dtype"):
        plan.step(params, grads, [moms[0], moms[1].to(torch.bfloat16)], **kw)
    torch.cuda.synchronize()
    assert all(torch.equal(a, b) for a, b in zip(params, before)), "a refused step changed a parameter"
    calls = []
    real = O.check_step_tensors
    monkeypatch.setattr(O, "check_step_tensors", lambda *a, **k: (calls.append(1), real(*a, **k)))
    plan.step(params, grads, moms, **kw)
    plan.step(params, grads, moms, **kw)            # same buffers: not checked again
    g2 = [g.clone() for g in grads]
    plan.step(params, g2, moms, **kw)               # new addresses: checked
    torch.cuda.synchronize()
    assert len(calls) == 2
    assert not any(torch.equal(a, b) for a, b in zip(params, before))
    plan.close()


@pytest.mark.gpu
def test_abi_vets_where_buffers_live():
    # the C ABI's own checks, for callers that bypass the binding: host
    # memory, pinned host memory and allocations shorter than the matrix are
    # refused by muon_check_buffers and by muon_step (before anything is
    # enqueued); a view into a larger allocation is fine
    import ctypes

    import numpy as np

    import paper_2606_27153_amd._lib as L
    lib = L.load()
    hip = ctypes.CDLL("libamdhip64.so.7")
    dev = "cuda:0"
    plan = MuonPlan([(96, 160, "f32", "f32")])
    p, g, m = (torch.randn(96, 160, device=dev) for _ in range(3))
    ws = plan.workspace(dev)

    def check(pp, gp, mp, wsp=None):
        st = lib.muon_check_buffers(plan.handle, L.ptr_array([pp]), L.ptr_array([gp]), L.ptr_array([mp]),
                                    ctypes.c_void_p(ws.data_ptr() if wsp is None else wsp), ws.numel(), None)
        return st, (L.last_error() if st else "")

    assert check(p.data_ptr(), g.data_ptr(), m.data_ptr()) == (L.MUON_OK, "")
    host = np.zeros(96 * 160 + 16, dtype=np.float32)
    hp = (host.ctypes.data + 15) // 16 * 16
    assert check(p.data_ptr(), hp, m.data_ptr()) == (L.MUON_ERR_INVALID_ARG, "matrix 0 grad is not device memory")
    pinned = torch.zeros(96 * 160, pin_memory=True)
    assert check(p.data_ptr(), g.data_ptr(), pinned.data_ptr())[1] == "matrix 0 momentum is not device memory"
    raw = ctypes.c_void_p()
    assert hip.hipMalloc(ctypes.byref(raw), ctypes.c_size_t(4096)) == 0
    try:
        st, msg = check(raw.value, g.data_ptr(), m.data_ptr())
        assert st == L.MUON_ERR_INVALID_ARG and msg.startswith("matrix 0 param needs 61440 bytes"), msg
        st, msg = check(p.data_ptr(), g.data_ptr(), m.data_ptr(), raw.value)
        assert st == L.MUON_ERR_INVALID_ARG and msg.startswith("the workspace needs"), msg
    finally:
        assert hip.hipFree(raw) == 0
    big = torch.zeros(4, 96, 160, device=dev)
    assert check(big[2].data_ptr(), g.data_ptr(), m.data_ptr())[0] == L.MUON_OK

    # muon_step makes the same checks when its buffer addresses change
    before = p.clone()
    stream = torch.cuda.current_stream(dev).cuda_stream

    def step(gp):
        return lib.muon_step(plan.handle, L.ptr_array([p.data_ptr()]), L.ptr_array([gp]),
                             L.ptr_array([m.data_ptr()]), 0.02, 0.95, 0.01, 5, 1,
                             ctypes.c_void_p(ws.data_ptr()), ws.numel(), ctypes.c_void_p(stream))

    assert step(hp) == L.MUON_ERR_INVALID_ARG and L.last_error() == "matrix 0 grad is not device memory"
    torch.cuda.synchronize()
    assert torch.equal(p, before)
    assert step(g.data_ptr()) == L.MUON_OK
    torch.cuda.synchronize()
    assert not torch.equal(p, before)
    plan.close()
