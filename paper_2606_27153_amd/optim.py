"""Python front end of the HIP Muon step: ``MuonPlan`` and ``Muon``.

``MuonPlan`` wraps muon_plan_create / muon_step / muon_step_debug for a fixed
list of matrix shapes; PyTorch supplies device memory (the tensors and the
workspace) and the stream.  ``Muon`` is a torch.optim.Optimizer over 2-D
parameters (DMuon's user surface, Sec. 4: the optimizer keeps the usual
optimizer protocol; its state is the per-matrix momentum buffer).
"""
from __future__ import annotations

import ctypes
from typing import List, Optional, Sequence

from . import _lib as L

_DT = {"f32": L.MUON_F32, "bf16": L.MUON_BF16}
# NS arithmetic: bf16 (the default), fp16 (the paper's implementation
# choice, Sec. 4) or fp32 (validation)
PRECISIONS = {"bf16": L.MUON_NS_BF16, "fp32": L.MUON_NS_FP32, "fp16": L.MUON_NS_FP16}


def default_gram_min_aspect(precision: str) -> float:
    """Aspect n/m from which a 16-bit matrix takes the Gram-space form by
    default (Eq. 4, restarted every 2 steps; also m >= 256).

    The restarted form costs 9m^2 n + 11m^3 against Eq. 2's 15m^2 n + 5m^3 at
    k = 5, fewer flops for n > m, but moves work to the m x m products, which
    run slower per flop than B*X.  From aspect 1.4 it is faster on the
    1408 x 2048 MoE experts (MoE set 344.5 -> 334.5 ms), and on planted
    spectra at aspect 1.45-1.5 it is as accurate as Eq. 2 in bf16 (mild
    7.2e-3 against 8.3e-3, 1/i 2.9e-2 against 3.3e-2).  The fp32 path keeps
    Eq. 2 whatever this says.
    """
    return 1.4


def check_step_tensors(descs: Sequence, params: List, grads: List, moms: List, workspace=None,
                       update_out: Optional[List] = None, only: Optional[Sequence[int]] = None) -> None:
    """Raises ValueError unless every buffer matches what the C ABI assumes of
    it: matrix i's param, grad and momentum are contiguous (row-major,
    leading dimension cols) tensors of descs[i]'s shape and dtypes (momentum
    fp32), all on one GPU, like the workspace and any update_out buffer (fp32).
    A grad may be None (the matrix is skipped for the step).  ``only``
    restricts the per-matrix checks to those indices.  The library itself
    only sees pointers and cannot tell."""
    n = len(descs)
    if not (len(params) == len(grads) == len(moms) == n):
        raise ValueError(f"expected {n} params, grads and momentum buffers")
    if update_out is not None and len(update_out) != n:
        raise ValueError(f"expected {n} update_out entries (None for no output)")
    checked = []
    for i in (range(n) if only is None else only):
        d = descs[i]
        rows, cols, pd, gd = d[:4]
        shape = (int(rows), int(cols))
        pc = _DT[pd] if isinstance(pd, str) else int(pd)
        gc = _DT[gd] if isinstance(gd, str) else int(gd)
        todo = [(params[i], "param", pc), (moms[i], "momentum", L.MUON_F32)]
        if grads[i] is not None:
            todo.insert(1, (grads[i], "grad", gc))
        if update_out is not None and update_out[i] is not None:
            todo.append((update_out[i], "update_out", L.MUON_F32))
        for t, name, code in todo:
            what = f"matrix {i} {name}"
            if tuple(t.shape) != shape:
                raise ValueError(f"{what} has shape {tuple(t.shape)}, the plan expects {shape}")
            if _dtype_code(t) != code:
                raise ValueError(f"{what} has dtype {t.dtype}, the plan expects "
                                 f"{'float32' if code == L.MUON_F32 else 'bfloat16'}")
            if not t.is_contiguous():
                raise ValueError(f"{what} is not contiguous (the library reads row-major rows of cols elements)")
            checked.append((t, what))
    device = params[0].device if n else None
    for t, what in checked:
        if not t.is_cuda:
            raise ValueError(f"{what} is not on a GPU")
        if device is None:
            device = t.device
        elif t.device != device:
            raise ValueError(f"{what} is on {t.device}, other buffers on {device}")
    if workspace is not None:
        if not workspace.is_contiguous() or not workspace.is_cuda or workspace.device != device:
            raise ValueError(f"the workspace must be a contiguous tensor on {device}")


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return L.MUON_F32
    if t.dtype == torch.bfloat16:
        return L.MUON_BF16
    raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16")


class MuonPlan:
    """A plan over matrix descriptors ``(rows, cols, param_dtype, grad_dtype)``
    or ``(rows, cols, param_dtype, grad_dtype, tile_hint)`` (0, 64, 128, 256).

    dtypes are 'f32' or 'bf16'; momentum is always fp32.  16-bit-path
    matrices with max(rows, cols) >= gram_min_aspect * min(rows, cols) run the
    Gram-space recurrence (Eq. 4); 0 keeps every matrix on Eq. 2; None takes
    ``default_gram_min_aspect(precision)`` (1.4 in both 16-bit precisions).  ``abc`` is
    one (a, b, c) for every NS step or a list with one triple per step (the
    per-step coefficient sets of Sec. 4); a list sets max_ns_steps to its
    length.  ``autotune`` picks each shape's GEMM tile by measurement on
    the GPU (see autotune.py), reading and filling the on-disk cache.
    ``check_buffers`` makes the library vet where the buffers of a step live
    whenever their addresses change (MUON_PLAN_CHECK_BUFFERS).
    ``gram_restart`` is the number of NS steps per Gram-space segment (0:
    the library's default of 2).
    """

    def __init__(self, descs: Sequence, *, precision: str = "bf16", max_ns_steps: int = 16,
                 abc: Optional[Sequence[float]] = None, eps: float = 1e-7,
                 small_m_threshold: int = 64, wave_bytes: int = 0, gram_min_aspect: Optional[float] = None,
                 host_only: bool = False, check_buffers: bool = False, autotune: bool = False,
                 tune_cache: Optional[str] = None, gram_restart: int = 0,
                 tune_ns_steps: int = 5):
        lib = L.load()
        n = len(descs)
        if gram_min_aspect is None:
            gram_min_aspect = default_gram_min_aspect(precision)
        if autotune:
            # measured tile per shape (cached on disk) for descriptors without a hint
            from .autotune import tune
            todo = [i for i, d in enumerate(descs) if len(d) < 5 or not d[4]]
            if todo:
                hints = tune([descs[i] for i in todo], precision=precision, gram_min_aspect=gram_min_aspect,
                             ns_steps=tune_ns_steps, cache_path=tune_cache)
                descs = list(descs)
                for i, h in zip(todo, hints):
                    descs[i] = tuple(descs[i][:4]) + (h,)
        arr = (L.muon_matrix_desc * max(n, 1))()
        for i, d in enumerate(descs):
            rows, cols, pd, gd = d[:4]
            arr[i].tile_hint = int(d[4]) if len(d) > 4 else 0
            arr[i].rows, arr[i].cols = int(rows), int(cols)
            arr[i].param_dtype = _DT[pd] if isinstance(pd, str) else int(pd)
            arr[i].grad_dtype = _DT[gd] if isinstance(gd, str) else int(gd)
            arr[i].momentum_dtype = L.MUON_F32
        opts = L.muon_plan_opts()
        L.check(lib.muon_plan_opts_default(ctypes.byref(opts)))
        opts.precision = PRECISIONS[precision]
        opts.max_ns_steps = int(max_ns_steps)
        schedule = None
        if abc is not None:
            abc = list(abc)
            if len(abc) == 3 and all(isinstance(v, (int, float)) for v in abc):
                opts.a, opts.b, opts.c = (float(v) for v in abc)
            else:
                # one (a, b, c) per NS step; the schedule sets max_ns_steps
                triples = [tuple(float(v) for v in t) for t in abc]
                if any(len(t) != 3 for t in triples) or not triples:
                    raise ValueError("abc must be a triple or a non-empty list of triples")
                opts.max_ns_steps = len(triples)
                schedule = (ctypes.c_float * (3 * len(triples)))(*[v for t in triples for v in t])
                opts.abc_per_step = schedule
        opts.eps = float(eps)
        opts.small_m_threshold = int(small_m_threshold)
        opts.wave_bytes = int(wave_bytes)
        opts.gram_min_aspect = float(gram_min_aspect)
        opts.gram_restart = int(gram_restart)
        opts.flags = (L.MUON_PLAN_HOST_ONLY if host_only else 0) | (L.MUON_PLAN_CHECK_BUFFERS if check_buffers else 0)
        h = ctypes.c_void_p()
        L.check(lib.muon_plan_create(arr, n, ctypes.byref(opts), ctypes.byref(h)))
        self._h = h
        self.n = n
        self.descs = list(descs)
        self.precision = precision
        self._workspace = None
        self._checked = None     # buffer addresses of the last checked call

    # ------------------------------------------------------------ inspection
    @property
    def handle(self):
        return self._h

    @property
    def workspace_bytes(self) -> int:
        v = ctypes.c_size_t()
        L.check(L.load().muon_plan_workspace_bytes(self._h, ctypes.byref(v)))
        return int(v.value)

    def info(self) -> dict:
        v = L.muon_plan_info()
        L.check(L.load().muon_plan_get_info(self._h, ctypes.byref(v)))
        return {f: getattr(v, f) for f, _ in v._fields_}

    def ns_flops(self, ns_steps: int) -> float:
        """The plan's own algorithmic NS flops for ``ns_steps`` steps."""
        v = ctypes.c_double()
        L.check(L.load().muon_plan_ns_flops(self._h, int(ns_steps), ctypes.byref(v)))
        return float(v.value)

    def matrix_info(self, i: int) -> dict:
        v = L.muon_matrix_info()
        L.check(L.load().muon_plan_matrix_info(self._h, int(i), ctypes.byref(v)))
        return {f: getattr(v, f) for f, _ in v._fields_}

    def set_timing(self, enable: bool) -> None:
        L.check(L.load().muon_plan_set_timing(self._h, 1 if enable else 0))

    def timing_read(self, reset: bool = True) -> list:
        """Event-timed launches aggregated by (kind, kernel class)."""
        lib = L.load()
        cap = 64
        arr = (L.muon_kernel_stat * cap)()
        cnt = ctypes.c_int32()
        L.check(lib.muon_plan_timing_read(self._h, arr, cap, ctypes.byref(cnt), 1 if reset else 0))
        out = []
        for i in range(min(cnt.value, cap)):
            s = arr[i]
            out.append({"kind": L.KERNEL_KINDS[s.kind],
                        "kernel_class": None if s.kernel_class < 0 else L.KERNEL_CLASSES[s.kernel_class],
                        "launches": s.launches, "total_ms": s.total_ms,
                        "algo_flops": s.algo_flops, "algo_bytes": s.algo_bytes})
        return out

    # ------------------------------------------------------------ stepping
    def workspace(self, device=None):
        """A cached torch uint8 workspace of the plan's size on ``device``."""
        import torch
        need = self.workspace_bytes
        ws = self._workspace
        if ws is None or ws.numel() < need or (device is not None and ws.device != torch.device(device)):
            self._workspace = torch.empty(max(need, 256), dtype=torch.uint8,
                                          device=device if device is not None else "cuda")
        return self._workspace

    def step(self, params: List, grads: List, moms: List, *, lr: float, momentum: float,
             weight_decay: float, ns_steps: int = 5, nesterov: bool = True, workspace=None,
             stream=None, update_out: Optional[List] = None) -> None:
        """Enqueues one Muon step on ``stream`` (default: torch's current stream).

        A grad may be None: that matrix is skipped (its param and momentum
        stay as they are).  The buffers whose addresses differ from the
        previous call's are checked against the plan (``check_step_tensors``:
        shape, dtype, row-major layout, one GPU); a failed check raises
        ValueError and nothing is launched."""
        import torch
        n = self.n
        if not (len(params) == len(grads) == len(moms) == n):
            raise ValueError(f"expected {n} params, grads and momentum buffers")
        if workspace is None:
            workspace = self.workspace(params[0].device)
        if stream is None:
            stream = torch.cuda.current_stream(params[0].device)
        sp = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
        pp = [t.data_ptr() for t in params]
        gp = [0 if t is None else t.data_ptr() for t in grads]
        mp = [t.data_ptr() for t in moms]
        op = None if update_out is None else [0 if t is None else t.data_ptr() for t in update_out]
        wsp = workspace.data_ptr()
        last = self._checked
        if last is None or last[4] != wsp or (last[3] is None) != (op is None):
            todo = None   # everything
        else:
            todo = [i for i in range(n) if pp[i] != last[0][i] or gp[i] != last[1][i] or mp[i] != last[2][i]
                    or (op is not None and op[i] != last[3][i])]
        if todo is None or todo:
            check_step_tensors(self.descs, params, grads, moms, workspace, update_out, only=todo)
        self._checked = (pp, gp, mp, op, wsp)
        args = (self._h, L.ptr_array(pp), L.ptr_array(gp), L.ptr_array(mp), float(lr), float(momentum),
                float(weight_decay), int(ns_steps), 1 if nesterov else 0, ctypes.c_void_p(wsp),
                workspace.numel() * workspace.element_size(), ctypes.c_void_p(sp))
        lib = L.load()
        if update_out is None:
            L.check(lib.muon_step(*args))
        else:
            L.check(lib.muon_step_debug(*args, L.ptr_array(op)))

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            L.check(L.load().muon_plan_destroy(self._h))
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _optimizer_base():
    import torch
    return torch.optim.Optimizer


class Muon(_optimizer_base()):
    """torch.optim-style Muon over 2-D parameters (fp32 or bf16).

    Per-parameter state: ``momentum_buffer`` (fp32).  Each param group has
    one plan over all of its parameters, built at the first step and kept
    while the group's shapes and dtypes stay the same; a parameter without a
    gradient is passed to the library as a skipped matrix (its param and
    momentum stay as they are), so a changing set of routed MoE experts
    reuses the same plan.  The plans of all groups share one workspace per
    device, sized to the largest.  ``ns_coefficients`` is None (the quintic
    (3.4445, -4.7750, 2.0315) at every step), one (a, b, c), or one triple
    per NS step.
    """

    def __init__(self, params, lr: float = 0.02, momentum: float = 0.95, weight_decay: float = 0.01,
                 ns_steps: int = 5, nesterov: bool = True, precision: str = "bf16",
                 gram_min_aspect: Optional[float] = None,
                 ns_coefficients=None, autotune: bool = False, tune_cache: Optional[str] = None):
        defaults = dict(lr=lr, momentum=momentum, weight_decay=weight_decay, ns_steps=ns_steps,
                        nesterov=nesterov, precision=precision, gram_min_aspect=gram_min_aspect,
                        ns_coefficients=ns_coefficients, autotune=autotune)
        super().__init__(params, defaults)
        self._plans = {}       # id(group) -> (key, MuonPlan)
        self._workspaces = {}  # device -> shared uint8 workspace
        self._tune_cache = tune_cache

    @staticmethod
    def _coef_key(abc):
        if abc is None:
            return None
        abc = list(abc)
        if len(abc) == 3 and all(isinstance(v, (int, float)) for v in abc):
            return tuple(float(v) for v in abc)
        return tuple(tuple(float(v) for v in t) for t in abc)

    def _plan_for(self, group, descs):
        key = (tuple(descs), group["precision"], group["gram_min_aspect"],
               self._coef_key(group.get("ns_coefficients")), group.get("autotune", False))
        held = self._plans.get(id(group))
        if held is not None and held[0] == key:
            return held[1]
        if held is not None:
            held[1].close()
        aspect = group["gram_min_aspect"]
        if aspect is None:
            aspect = default_gram_min_aspect(group["precision"])
        plan = MuonPlan(descs, precision=group["precision"], gram_min_aspect=aspect,
                        abc=group.get("ns_coefficients"), autotune=group.get("autotune", False),
                        tune_cache=self._tune_cache, tune_ns_steps=group["ns_steps"])
        self._plans[id(group)] = (key, plan)
        return plan

    def _workspace(self, device, need: int):
        import torch
        ws = self._workspaces.get(device)
        if ws is None or ws.numel() < need:
            self._workspaces[device] = None
            del ws
            ws = torch.empty(max(need, 256), dtype=torch.uint8, device=device)
            self._workspaces[device] = ws
        return ws

    def step(self, closure=None):
        import torch
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        for group in self.param_groups:
            ps = list(group["params"])
            if not any(p.grad is not None for p in ps):
                continue
            for p in ps:
                if p.ndim != 2:
                    raise ValueError("Muon steps 2-D parameters only")
            descs = []
            for p in ps:
                st = self.state[p]
                # a parameter's grad dtype is remembered from the last step
                # that had one (the param dtype until then)
                if p.grad is not None:
                    st["grad_dtype"] = _dtype_code(p.grad)
                gd = st.get("grad_dtype", _dtype_code(p))
                descs.append((p.shape[0], p.shape[1], _dtype_code(p), gd))
            plan = self._plan_for(group, descs)
            moms = []
            for p in ps:
                st = self.state[p]
                if "momentum_buffer" not in st:
                    st["momentum_buffer"] = torch.zeros_like(p, dtype=torch.float32,
                                                             memory_format=torch.contiguous_format)
                moms.append(st["momentum_buffer"])
            params = [p.data for p in ps]
            grads = [None if p.grad is None else p.grad.contiguous() for p in ps]
            ws = self._workspace(ps[0].device, plan.workspace_bytes)
            plan.step(params, grads, moms, lr=group["lr"], momentum=group["momentum"],
                      weight_decay=group["weight_decay"], ns_steps=group["ns_steps"],
                      nesterov=group["nesterov"], workspace=ws)
        return loss
