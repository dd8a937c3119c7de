"""Seeded synthetic matrix sets for the Muon step (inputs only).

This module holds the five matrix-shape sets the step is measured and
tested on and the seeded generators of their parameters and gradients.  It
contains none of the step's arithmetic, so both the HIP path and the oracle
may take their inputs from it.

The paper measures on production models (Wall-OSS, Pi0, Wall-WM,
Qwen2.5-7B; Sec. 5, Table 1) whose matrix shapes it does not list; these
sets stand in for them: a tiny transformer, Llama-style 1B and 8B sets, a
heterogeneous vision-language-action set and an MoE expert bank.  Step cost
depends only on shapes and dtypes, so synthetic N(0, sigma^2) values suffice.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclass(frozen=True)
class MatrixSpec:
    name: str
    rows: int
    cols: int
    param: str = BF16          # stored parameter dtype
    grad: str = BF16           # stored gradient dtype
    grad_std: float = 1e-3     # std of the synthetic gradient
    zero_grad: bool = False    # gradient identically zero (unrouted expert)


@dataclass(frozen=True)
class Workload:
    key: str
    description: str
    matrices: List[MatrixSpec]
    seed: int
    lr: float = 0.02
    momentum: float = 0.95
    weight_decay: float = 0.01
    ns_steps: int = 5
    nesterov: bool = True
    steps: int = 3
    param_std: float = 0.02
    extra: dict = field(default_factory=dict)

    @property
    def n(self) -> int:
        return len(self.matrices)

    def elements(self) -> int:
        return sum(m.rows * m.cols for m in self.matrices)


def _tiny() -> Workload:
    mats = []
    for layer in range(2):
        for nm, r, c in (("w_qkv", 256, 768), ("w_o", 256, 256), ("w_up", 256, 1024), ("w_down", 1024, 256)):
            mats.append(MatrixSpec(f"l{layer}.{nm}", r, c, F32, F32))
    return Workload("tiny", "tiny 2-layer transformer, fp32 params/grads (8 matrices)", mats, seed=0)


def _llama(key, layers, d, kv, ffn, seed, log_uniform_scale):
    rng = np.random.default_rng(seed)
    mats = []
    for layer in range(layers):
        for nm, r, c in (("wq", d, d), ("wk", d, kv), ("wv", d, kv), ("wo", d, d),
                         ("gate", d, ffn), ("up", d, ffn), ("down", ffn, d)):
            std = 1e-3
            if log_uniform_scale:
                std *= float(np.exp(rng.uniform(np.log(0.1), np.log(10.0))))
            mats.append(MatrixSpec(f"l{layer}.{nm}", r, c, BF16, BF16, std))
    return mats


def _llama_1b() -> Workload:
    mats = _llama("1b", 16, 2048, 512, 5632, 1, True)
    return Workload("1b", "Llama-style 1B set: 16 layers, d=2048, GQA kv 512, ffn 5632 (112 matrices)", mats, seed=1)


def _llama_8b() -> Workload:
    mats = _llama("8b", 32, 4096, 1024, 14336, 2, False)
    return Workload("8b", "Llama-style 8B set: 32 layers, d=4096, GQA kv 1024, ffn 14336 (224 matrices)", mats, seed=2)


def _vla() -> Workload:
    rng = np.random.default_rng(3)
    mats = []
    for layer in range(27):
        for nm, r, c in (("qkv", 1152, 3456), ("o", 1152, 1152), ("fc1", 1152, 4304), ("fc2", 4304, 1152)):
            mats.append(MatrixSpec(f"vision{layer}.{nm}", r, c))
    for layer in range(18):
        for nm, r, c in (("wq", 1024, 1024), ("wk", 1024, 256), ("wv", 1024, 256), ("wo", 1024, 1024),
                         ("gate", 1024, 4096), ("up", 1024, 4096), ("down", 4096, 1024)):
            mats.append(MatrixSpec(f"action{layer}.{nm}", r, c))
    rows = rng.choice([32, 64, 128, 256], size=200)
    cols = rng.choice([512, 1024], size=200)
    for i in range(200):
        mats.append(MatrixSpec(f"proj{i}", int(rows[i]), int(cols[i])))
    return Workload("vla", "VLA-style heterogeneous set: 27-layer vision tower, 18-layer action expert, "
                           "200 small projections (434 matrices)", mats, seed=3)


def _moe() -> Workload:
    rng = np.random.default_rng(4)
    mats = []
    for layer in range(24):
        zero = set(rng.permutation(64)[:16].tolist())
        for nm, r, c in (("wq", 2048, 2048), ("wk", 2048, 512), ("wv", 2048, 512), ("wo", 2048, 2048)):
            mats.append(MatrixSpec(f"l{layer}.{nm}", r, c))
        for e in range(64):
            for nm, r, c in (("gate", 2048, 1408), ("up", 2048, 1408), ("down", 1408, 2048)):
                mats.append(MatrixSpec(f"l{layer}.e{e}.{nm}", r, c, zero_grad=e in zero))
    return Workload("moe", "MoE expert bank: 24 layers x 64 experts (gate/up 2048x1408, down 1408x2048) "
                           "+ attention, 25% unrouted experts (4704 matrices)", mats, seed=4)


_BUILDERS = {"tiny": _tiny, "1b": _llama_1b, "8b": _llama_8b, "vla": _vla, "moe": _moe}
WORKLOAD_KEYS = tuple(_BUILDERS)


def get_workload(key: str) -> Workload:
    if key not in _BUILDERS:
        raise KeyError(f"unknown workload {key!r}; choose from {WORKLOAD_KEYS}")
    return _BUILDERS[key]()


def custom_workload(shapes: Sequence, param=BF16, grad=BF16, seed=0, **kw) -> Workload:
    mats = [MatrixSpec(f"m{i}", int(r), int(c), param, grad) for i, (r, c) in enumerate(shapes)]
    return Workload("custom", f"{len(mats)} custom matrices", mats, seed=seed, **kw)


# ---------------------------------------------------------------- generators

def tensor_seed(seed: int, step: int, index: int, kind: str) -> int:
    """64-bit seed of one tensor, keyed by (workload seed, step, matrix, kind)."""
    h = hashlib.blake2b(f"{seed}/{step}/{index}/{kind}".encode(), digest_size=8).digest()
    return int.from_bytes(h, "little") & ((1 << 63) - 1)


def _torch_dtype(torch, name):
    return {F32: torch.float32, BF16: torch.bfloat16}[name]


def make_param(torch, wl: Workload, i: int, device):
    spec = wl.matrices[i]
    g = torch.Generator(device=device)
    g.manual_seed(tensor_seed(wl.seed, 0, i, "param"))
    t = torch.randn(spec.rows, spec.cols, generator=g, device=device, dtype=torch.float32)
    t.mul_(wl.param_std)
    return t.to(_torch_dtype(torch, spec.param))


def make_grad(torch, wl: Workload, i: int, step: int, device):
    spec = wl.matrices[i]
    if spec.zero_grad:
        return torch.zeros(spec.rows, spec.cols, device=device, dtype=_torch_dtype(torch, spec.grad))
    g = torch.Generator(device=device)
    g.manual_seed(tensor_seed(wl.seed, step, i, "grad"))
    t = torch.randn(spec.rows, spec.cols, generator=g, device=device, dtype=torch.float32)
    t.mul_(spec.grad_std)
    return t.to(_torch_dtype(torch, spec.grad))


def make_state(torch, wl: Workload, device, indices: Optional[Sequence[int]] = None):
    """Params (seeded) and zero fp32 momentum buffers for the chosen matrices."""
    idx = range(wl.n) if indices is None else indices
    params = [make_param(torch, wl, i, device) for i in idx]
    moms = [torch.zeros(wl.matrices[i].rows, wl.matrices[i].cols, device=device, dtype=torch.float32)
            for i in idx]
    return params, moms


def make_grads(torch, wl: Workload, step: int, device, indices: Optional[Sequence[int]] = None):
    idx = range(wl.n) if indices is None else indices
    return [make_grad(torch, wl, i, step, device) for i in idx]


def planted_matrix(rows: int, cols: int, spectrum: Sequence[float], seed: int):
    """A rows x cols matrix with a chosen spectrum: U diag(spectrum) V^T with
    seeded random orthonormal U (rows x r) and V (cols x r), r = len(spectrum)
    <= min(rows, cols).  Returns (matrix, U, spectrum, V), all fp64 numpy.
    Input generation only (a QR of a Gaussian draw for each factor)."""
    s = np.asarray(spectrum, dtype=np.float64)
    r = len(s)
    if r > min(rows, cols):
        raise ValueError("spectrum longer than min(rows, cols)")
    rng = np.random.default_rng(seed)

    def orthonormal(n):
        q, t = np.linalg.qr(rng.standard_normal((n, r)))
        return q * np.sign(np.diag(t))

    u = orthonormal(rows)
    v = orthonormal(cols)
    return (u * s) @ v.T, u, s, v
