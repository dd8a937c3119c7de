"""Measured choice of the GEMM tile per shape, with a persistent cache.

Sec. 3.3 treats the kernel schedule as a per-shape problem: the first time a
shape is met, candidate schedules are timed on the GPU, the fastest is kept,
and the choice is recorded in a persistent cache keyed by problem shape and
execution mode, so later runs dispatch it without searching.

Here the candidates are the output tiles the operand type offers (256, 128,
64 for 16-bit operands; 128, 64 for fp32).  A shape is not timed alone:
matrices of one kernel class share grouped launches, so a tile that wins for
a shape in isolation (more blocks for a small batch) can lose inside the
whole set, where the batch is already full.  The tuner therefore times whole
steps of a reduced copy of the set (each shape at most ``max_per_shape``
times, keeping the mix) and runs one pass of coordinate descent from the
planner's own cost-model choice: for each shape, heaviest first, each other
tile is tried with the rest fixed and kept if the step gets faster by more
than ``min_gain``.  The result can only match or beat the cost model on the
reduced set.

The cache is a JSON file (``$MUON_TUNE_CACHE``, else
``~/.cache/mi355x_muon/tiles.json``); its key names the device, the library
ABI, the NS precision, the Gram-space threshold, the NS step count and the
multiset of (stored shape, dtypes, count).  A cached choice is a measurement,
not a correctness input: every tile computes the same step.
"""
from __future__ import annotations

import hashlib
import json
import os
import statistics
from typing import Callable, Dict, List, Optional, Sequence

CACHE_ENV = "MUON_TUNE_CACHE"
TUNER_VERSION = 2


def default_cache_path() -> str:
    return os.environ.get(CACHE_ENV) or os.path.join(os.path.expanduser("~"), ".cache", "mi355x_muon", "tiles.json")


def candidate_tiles(rows: int, cols: int, precision: str, small_m_threshold: int = 64) -> tuple:
    """Output tiles of the kernel classes that can run this matrix."""
    m = min(rows, cols)
    fp32 = precision == "fp32" or (precision == "bf16" and m <= small_m_threshold)
    return (128, 64) if fp32 else (256, 128, 64)


def _groups(descs: Sequence) -> Dict[tuple, List[int]]:
    g: Dict[tuple, List[int]] = {}
    for i, d in enumerate(descs):
        g.setdefault((int(d[0]), int(d[1]), d[2], d[3]), []).append(i)
    return g


def set_key(groups: Dict[tuple, List[int]], *, precision: str, gram_min_aspect: float, ns_steps: int,
            max_per_shape: int, device: str, abi: int) -> str:
    sig = ";".join(f"{r}x{c}:{pd}/{gd}:{len(ix)}" for (r, c, pd, gd), ix in sorted(groups.items()))
    digest = hashlib.sha256(sig.encode()).hexdigest()[:16]
    return (f"v{TUNER_VERSION}|{device}|abi{abi}|{precision}|aspect{gram_min_aspect:g}|k{ns_steps}|"
            f"cap{max_per_shape}|{digest}")


class TileCache:
    """The on-disk cache: {key: {"tiles": {"RxC:pd/gd": tile}, "ms": t, "base_ms": t0}}."""

    def __init__(self, path: Optional[str] = None):
        self.path = path or default_cache_path()
        self.data: Dict[str, dict] = {}
        if os.path.exists(self.path):
            with open(self.path) as f:
                self.data = json.load(f)

    def get(self, key: str) -> Optional[dict]:
        return self.data.get(key)

    def put(self, key: str, entry: dict) -> None:
        self.data[key] = entry

    def save(self) -> None:
        d = os.path.dirname(self.path)
        if d:
            os.makedirs(d, exist_ok=True)
        tmp = f"{self.path}.{os.getpid()}.tmp"
        with open(tmp, "w") as f:
            json.dump(self.data, f, indent=1, sort_keys=True)
        os.replace(tmp, self.path)


def _gkey(g: tuple) -> str:
    return f"{g[0]}x{g[1]}:{g[2]}/{g[3]}"


def measure_set_ms(descs: Sequence, *, precision: str, gram_min_aspect: float, ns_steps: int, steps: int = 3,
                   device: str = "cuda:0") -> float:
    """Median ms of one muon_step over seeded synthetic matrices with these
    descriptors (tile hints included)."""
    import dataclasses

    import torch

    from .optim import MuonPlan
    from .workloads import custom_workload, make_grads, make_state

    wl = custom_workload([(d[0], d[1]) for d in descs], seed=101)
    wl = dataclasses.replace(wl, ns_steps=ns_steps, matrices=[
        dataclasses.replace(m, param=d[2], grad=d[3]) for m, d in zip(wl.matrices, descs)])
    plan = MuonPlan(list(descs), precision=precision, gram_min_aspect=gram_min_aspect,
                    max_ns_steps=max(1, ns_steps))
    try:
        params, moms = make_state(torch, wl, device)
        grads = make_grads(torch, wl, 0, device)
        stream = torch.cuda.current_stream(device)
        kw = dict(lr=wl.lr, momentum=wl.momentum, weight_decay=wl.weight_decay, ns_steps=ns_steps,
                  nesterov=wl.nesterov, workspace=plan.workspace(device), stream=stream)
        plan.step(params, grads, moms, **kw)   # warm-up
        times = []
        for _ in range(steps):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            plan.step(params, grads, moms, **kw)
            b.record(stream)
            b.synchronize()
            times.append(a.elapsed_time(b))
        del params, moms, grads
        return statistics.median(times)
    finally:
        plan.close()


def planner_tiles(descs: Sequence, *, precision: str, gram_min_aspect: float) -> List[int]:
    """The tiles the planner's cost model gives these descriptors."""
    from .optim import MuonPlan
    plan = MuonPlan([tuple(d[:4]) for d in descs], precision=precision, gram_min_aspect=gram_min_aspect,
                    host_only=True)
    try:
        return [int(plan.matrix_info(i)["tile"]) for i in range(len(descs))]
    finally:
        plan.close()


def tune(descs: Sequence, *, precision: str = "bf16", gram_min_aspect: float = 1.4, ns_steps: int = 5,
         cache_path: Optional[str] = None, max_per_shape: int = 16, steps: int = 3, min_gain: float = 0.01,
         timer: Optional[Callable[[list], float]] = None, device_name: Optional[str] = None,
         abi: Optional[int] = None) -> List[int]:
    """A tile hint per descriptor ``(rows, cols, param_dtype, grad_dtype)``.

    ``timer(descs_with_hints)`` returns ms per step of the reduced set
    (default: ``measure_set_ms`` on the current GPU).
    """
    if device_name is None or abi is None:
        from . import _lib as L
        if abi is None:
            abi = int(L.load().muon_abi_version())
        if device_name is None:
            import torch
            device_name = torch.cuda.get_device_name(0)
    if timer is None:
        def timer(ds):
            return measure_set_ms(ds, precision=precision, gram_min_aspect=gram_min_aspect, ns_steps=ns_steps,
                                  steps=steps)
    groups = _groups(descs)
    key = set_key(groups, precision=precision, gram_min_aspect=gram_min_aspect, ns_steps=ns_steps,
                  max_per_shape=max_per_shape, device=device_name, abi=abi)
    cache = TileCache(cache_path)
    entry = cache.get(key)
    if entry is None:
        order = list(groups)
        base = planner_tiles([tuple(g) for g in order], precision=precision, gram_min_aspect=gram_min_aspect)
        choice = dict(zip(order, base))

        def reduced(ch):
            out = []
            for g in order:
                out += [tuple(g) + (ch[g],)] * min(len(groups[g]), max_per_shape)
            return out
        base_ms = best = float(timer(reduced(choice)))
        # heaviest shapes first (m^2 n per matrix times the count)
        for g in sorted(order, key=lambda g: -min(g[0], g[1]) ** 2 * max(g[0], g[1]) * len(groups[g])):
            for t in candidate_tiles(g[0], g[1], precision):
                if t == choice[g]:
                    continue
                trial = dict(choice)
                trial[g] = t
                ms = float(timer(reduced(trial)))
                if ms < best * (1.0 - min_gain):
                    best, choice = ms, trial
        entry = {"tiles": {_gkey(g): int(choice[g]) for g in order}, "ms": round(best, 4),
                 "base_ms": round(base_ms, 4)}
        cache.put(key, entry)
        cache.save()
    tiles = entry["tiles"]
    hints = [0] * len(descs)
    for g, idx in groups.items():
        for i in idx:
            hints[i] = int(tiles[_gkey(g)])
    return hints
