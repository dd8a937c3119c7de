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
    from paper_2606_27153_amd import _lib as L
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
    segs = [2, 2, 1]   # Eq. 4 restarts every 2 steps (the default)
    big, small = shapes       # only the 1024-row matrices reach the Gram-space minimum m of 256
    def eq2(r, c):
        return k * (3 * min(r, c) ** 2 * max(r, c) + min(r, c) ** 3)
    if gram:   # Eq. 4, per segment of L steps: 3 m^2 n and (4L - 3) m^3
        m, n = min(big), max(big)
        want = 2 * (sum(3 * m * m * n + (4 * L - 3) * m ** 3 for L in segs) + eq2(*small))
    else:      # Eq. 2: 3 m^2 n + m^3 per step
        want = 2 * (eq2(*big) + eq2(*small))
    got = sum(s["algo_flops"] for s in stats)
    assert abs(got - want) <= 1e-9 * want
    assert abs(plan.ns_flops(k) - want) <= 1e-9 * want
    # per Gram-space kernel class: per segment of L steps the Gram product and
    # B*X once, P_i each step and 3 (L - 1) other m^3 products in 2L - 1
    # launches (G P and P Q share one when both are due); Eq. 2 launches Gram,
    # A*A and B*X each step
    gram_cls = {"gram": len(segs), "poly": k, "symm": sum(2 * L - 1 for L in segs if L > 1), "bx": len(segs)}
    eq2_cls = {"gram": k, "poly": k, "bx": k}
    # the two shapes run in different kernel classes; with Eq. 4 on, the
    # big one's class runs the Gram-space schedule
    by_class = {}
    for s in stats:
        if s["kernel_class"] is not None:
            by_class.setdefault(s["kernel_class"], {})[s["kind"]] = s["launches"]
    big_cls = L.KERNEL_CLASSES[plan.matrix_info(0)["kernel_class"]]
    small_cls = L.KERNEL_CLASSES[plan.matrix_info(1)["kernel_class"]]
    assert big_cls != small_cls
    assert by_class[big_cls] == (gram_cls if gram else eq2_cls), by_class
    assert by_class[small_cls] == eq2_cls, by_class
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
    plan = MuonPlan([(96, 160, "f32", "f32")], check_buffers=True)
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

    # muon_step makes the same checks when its buffer addresses change (on a
    # plan created with MUON_PLAN_CHECK_BUFFERS)
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


def _alternating_grads(wl, dev, k):
    # k sets of gradient buffers with equal values, at k different addresses
    base = make_grads(torch, wl, 0, dev)
    return [[g.clone() for g in base] for _ in range(k)]


def test_moving_grad_buffers_match_fixed_ones_bitwise():
    # a step whose grads sit at new addresses every time (as under
    # zero_grad(set_to_none=True)) refreshes the pointer table on the stream,
    # without a host sync, and computes bitwise what fixed buffers give
    wl = custom_workload(SHAPES + [(1024, 3000), (2048, 700)], seed=25)
    descs = [(m.rows, m.cols, m.param, m.grad) for m in wl.matrices]
    kw = dict(lr=0.02, momentum=0.95, weight_decay=0.01, ns_steps=5)
    dev = "cuda:0"
    fixed, moving = MuonPlan(descs), MuonPlan(descs)
    pa, ma = make_state(torch, wl, dev)
    pb, mb = make_state(torch, wl, dev)
    ga = make_grads(torch, wl, 0, dev)
    for step in range(12):
        new = make_grads(torch, wl, step, dev)
        for a, g in zip(ga, new):
            a.copy_(g)
        fixed.step(pa, ga, ma, **kw)
        gb = [g.clone() for g in new]          # fresh addresses, enqueued without waiting
        moving.step(pb, gb, mb, **kw)
        del gb
    torch.cuda.synchronize()
    for x, y in zip(pa + ma, pb + mb):
        assert torch.equal(x, y)
    fixed.close()
    moving.close()


def test_moving_grad_buffers_cost_no_host_sync():
    # tiny set: steps alternating between two grad buffer sets (a pointer
    # refresh every step) take about as long as steps on one set
    from paper_2606_27153_amd.workloads import get_workload
    wl = get_workload("tiny")
    dev = "cuda:0"
    plan = MuonPlan([(m.rows, m.cols, m.param, m.grad) for m in wl.matrices])
    p, m = make_state(torch, wl, dev)
    sets = _alternating_grads(wl, dev, 2)
    kw = dict(lr=0.02, momentum=0.95, weight_decay=0.01, ns_steps=5)
    n = 60

    def timed(move):
        for i in range(5):
            plan.step(p, sets[i % 2 if move else 0], m, **kw)
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record()
        for i in range(n):
            plan.step(p, sets[i % 2 if move else 0], m, **kw)
        t1.record()
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / n

    fixed_ms, moving_ms = [], []
    for _ in range(4):
        fixed_ms.append(timed(False))
        moving_ms.append(timed(True))
    f, mv = min(fixed_ms), min(moving_ms)
    print(f"[gpu-test] tiny set: fixed buffers {f:.4f} ms per step, moving grads {mv:.4f} ms per step", flush=True)
    assert mv <= 1.10 * f, (fixed_ms, moving_ms)
    plan.close()


def test_null_grads_skip_their_matrices():
    # grads[i] = None: param and momentum untouched (no decay, no momentum
    # update), debug output untouched; the others bitwise as a plan over them
    # alone.  An all-zero gradient, by contrast, still decays its parameter.
    shapes = [(256, 768), (768, 256), (300, 300), (64, 200), (512, 2048), (1024, 1024)]
    wl = custom_workload(shapes, seed=26)
    dev = "cuda:0"
    kw = dict(lr=0.02, momentum=0.95, weight_decay=0.01, ns_steps=5)
    full = MuonPlan([(m.rows, m.cols, m.param, m.grad) for m in wl.matrices])
    live = [0, 2, 3, 5]
    sub = MuonPlan([(wl.matrices[i].rows, wl.matrices[i].cols, "bf16", "bf16") for i in live])
    pa, ma = make_state(torch, wl, dev)
    pb, mb = make_state(torch, wl, dev, live)
    for step in range(3):
        g = make_grads(torch, wl, step, dev)
        if step == 1:
            g[3] = torch.zeros_like(g[3])       # a zero gradient on a live matrix
        before = [(x.clone(), y.clone()) for x, y in zip(pa, ma)]
        outs = [torch.full((m.rows, m.cols), float("nan"), device=dev) for m in wl.matrices]
        full.step(pa, [g[i] if i in live else None for i in range(wl.n)], ma, update_out=outs, **kw)
        sub.step(pb, [g[i] for i in live], mb, **kw)
        torch.cuda.synchronize()
        for i in range(wl.n):
            if i in live:
                k = live.index(i)
                assert torch.equal(pa[i], pb[k]) and torch.equal(ma[i], mb[k]), (step, i)
                assert torch.isfinite(outs[i]).all()
            else:
                assert torch.equal(pa[i], before[i][0]) and torch.equal(ma[i], before[i][1]), (step, i)
                assert torch.isnan(outs[i]).all(), (step, i)
    full.close()
    sub.close()


def test_non_finite_gradients_poison_only_their_matrix():
    # NaN or Inf in a gradient is not sanitised: the matrix's momentum holds
    # it at that element, the norm of its NS input is not finite, and its
    # whole update -- hence every element of W -- turns NaN.  Every other
    # matrix is bitwise as in a clean step (Gram-space, Eq. 2 and the small
    # fp32 class each take one bad value).
    shapes = [(256, 768), (768, 256), (300, 300), (64, 200), (512, 2048), (1024, 1024)]
    wl = custom_workload(shapes, seed=28)
    dev = "cuda:0"
    kw = dict(lr=0.02, momentum=0.95, weight_decay=0.01, ns_steps=5)
    plan = MuonPlan([(m.rows, m.cols, m.param, m.grad) for m in wl.matrices])
    pa, ma = make_state(torch, wl, dev)
    pb, mb = make_state(torch, wl, dev)
    g = make_grads(torch, wl, 0, dev)
    gb = [x.clone() for x in g]
    bad = {1: float("nan"), 2: float("inf"), 3: float("-inf"), 4: float("nan")}
    for i, v in bad.items():
        gb[i][5, 7] = v
    plan.step(pa, g, ma, **kw)
    plan.step(pb, gb, mb, **kw)
    torch.cuda.synchronize()
    for i in range(wl.n):
        if i not in bad:
            assert torch.equal(pa[i], pb[i]) and torch.equal(ma[i], mb[i]), i
            continue
        assert torch.isnan(pb[i].float()).all(), i
        assert not torch.isfinite(mb[i][5, 7]), i
        same = torch.eq(ma[i], mb[i])
        same[5, 7] = True
        assert same.all(), i
    plan.close()


def test_optimizer_reuses_one_plan_while_experts_come_and_go():
    # MoE-like: each step a different subset of parameters has no gradient.
    # One plan per group, built once; GPU memory stays flat; every step is
    # bitwise a plan over that step's parameters alone.
    import random
    shapes = [(512, 1408), (1408, 512)] * 4 + [(512, 512), (128, 512)]
    wl = custom_workload(shapes, seed=27)
    dev = "cuda:0"
    kw = dict(lr=0.02, momentum=0.95, weight_decay=0.01, ns_steps=5)
    p_opt, _ = make_state(torch, wl, dev)
    params = [torch.nn.Parameter(t) for t in p_opt]
    opt = Muon(params, **kw)
    p_ref, m_ref = make_state(torch, wl, dev)
    rng = random.Random(5)
    mem = []
    for step in range(6):
        g = make_grads(torch, wl, step, dev)
        routed = sorted(rng.sample(range(wl.n), 6))
        for i, p in enumerate(params):
            p.grad = g[i].clone() if i in routed else None
        opt.step()
        ref = MuonPlan([(wl.matrices[i].rows, wl.matrices[i].cols, "bf16", "bf16") for i in routed])
        ref.step([p_ref[i] for i in routed], [g[i] for i in routed], [m_ref[i] for i in routed], **kw)
        torch.cuda.synchronize()
        ref.close()
        del ref
        for i in range(wl.n):
            assert torch.equal(params[i].data, p_ref[i]), (step, i)
            assert torch.equal(opt.state[params[i]]["momentum_buffer"], m_ref[i]), (step, i)
        for p in params:
            p.grad = None
        del g
        mem.append(torch.cuda.memory_allocated(dev))   # params, momenta, workspace, reference state
    assert len(opt._plans) == 1
    assert max(mem[1:]) <= mem[1], mem


def test_capture_with_moved_buffers_is_refused():
    from paper_2606_27153_amd import _lib as L
    wl = custom_workload([(256, 768), (300, 300)], seed=28)
    dev = "cuda:0"
    plan = MuonPlan([(m.rows, m.cols, m.param, m.grad) for m in wl.matrices])
    p, m = make_state(torch, wl, dev)
    g = make_grads(torch, wl, 0, dev)
    ws = plan.workspace(dev)
    kw = dict(lr=0.02, momentum=0.95, weight_decay=0.01, ns_steps=5, workspace=ws)
    plan.step(p, g, m, **kw)
    torch.cuda.synchronize()
    g2 = [x.clone() for x in g]
    before = [x.clone() for x in p]
    x = torch.zeros(4, device=dev)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        x.add_(1.0)
        with pytest.raises(L.MuonError) as e:
            plan.step(p, g2, m, **kw)
    assert e.value.status == L.MUON_ERR_INVALID_ARG and "captured" in str(e.value)
    graph.replay()
    torch.cuda.synchronize()
    assert all(torch.equal(a, b) for a, b in zip(p, before))
    plan.step(p, g2, m, **kw)      # eagerly, the same call goes through
    torch.cuda.synchronize()
    assert not torch.equal(p[0], before[0])
    plan.close()
