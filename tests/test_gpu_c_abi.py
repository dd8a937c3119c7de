"""A plain C caller of the library (tests/c_abi_step.c, built by
__graft_entry__.build()): seeded inputs written here, one muon_step_debug in a
separate process that links only the library and the HIP runtime, and its W,
M and O compared with the fp64 oracle."""
import dataclasses
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, os.path.join(ROOT, "tests"))

from oracle import muon_ref as R  # noqa: E402
from parity_utils import TOL_M, TOL_O, bf16_ulp, rel  # noqa: E402
from paper_2606_27153_amd import _lib as L  # noqa: E402
from paper_2606_27153_amd.workloads import custom_workload, make_grads, make_state  # noqa: E402

pytestmark = pytest.mark.gpu

EXE = os.path.join(ROOT, "tests", "c_abi_step")


def _raw(t: torch.Tensor) -> bytes:
    t = t.contiguous()
    return (t.view(torch.int16) if t.dtype == torch.bfloat16 else t).numpy().tobytes()


def _read(buf: bytes, off: int, shape, bf16: bool):
    n = shape[0] * shape[1]
    if bf16:
        a = np.frombuffer(buf, dtype=np.int16, count=n, offset=off).copy()
        v = torch.from_numpy(a).view(torch.bfloat16).double().numpy()
        return v.reshape(shape), off + 2 * n
    return np.frombuffer(buf, dtype=np.float32, count=n, offset=off).astype(np.float64).reshape(shape), off + 4 * n


def test_plain_c_caller_matches_oracle(tmp_path):
    assert os.path.exists(EXE), "tests/c_abi_step is missing: run __graft_entry__.build()"
    # wide, tall, Gram-space (n >= 1.4m), fp32 parameters with fp32 gradients,
    # and a small-m matrix on the fp32 NS classes
    wl = custom_workload([(200, 300), (300, 200), (512, 1100), (96, 160), (48, 700)], seed=33)
    mats = list(wl.matrices)
    mats[1] = dataclasses.replace(mats[1], grad="f32")
    mats[3] = dataclasses.replace(mats[3], param="f32", grad="f32")
    wl = dataclasses.replace(wl, matrices=mats)
    params, moms = make_state(torch, wl, "cpu")
    grads = make_grads(torch, wl, 0, "cpu")
    lr, mu, wd = (float(np.float32(v)) for v in (wl.lr, wl.momentum, wl.weight_decay))
    code = {"bf16": L.MUON_BF16, "f32": L.MUON_F32}
    blob = [np.array([wl.n], np.int32).tobytes(), np.array([lr, mu, wd], np.float32).tobytes(),
            np.array([wl.ns_steps, int(wl.nesterov)], np.int32).tobytes()]
    for i, m in enumerate(wl.matrices):
        blob += [np.array([m.rows, m.cols], np.int64).tobytes(), np.array([code[m.param], code[m.grad]], np.int32).tobytes(),
                 _raw(params[i]), _raw(grads[i]), _raw(moms[i])]
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    src.write_bytes(b"".join(blob))
    print(f"running {EXE} on {wl.n} matrices", flush=True)
    r = subprocess.run([EXE, str(src), str(dst)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    out = dst.read_bytes()
    off = 0
    for i, m in enumerate(wl.matrices):
        shape = (m.rows, m.cols)
        w, off = _read(out, off, shape, m.param == "bf16")
        mom, off = _read(out, off, shape, False)
        o, off = _read(out, off, shape, False)
        ref = R.muon_step_matrix(params[i].double().numpy(), grads[i].double().numpy(), np.zeros(shape), lr=lr,
                                 momentum=mu, weight_decay=wd, ns_steps=wl.ns_steps, nesterov=wl.nesterov,
                                 param_dtype=m.param)
        assert rel(o, ref["o"]) <= TOL_O["bf16"], (i, rel(o, ref["o"]))
        assert rel(mom, ref["m"]) <= TOL_M, (i, rel(mom, ref["m"]))
        rnd = float(np.linalg.norm(bf16_ulp(ref["w"]) if m.param == "bf16" else np.abs(ref["w"]) * 2.0 ** -23))
        bound = lr * R.shape_scale(m.rows, m.cols) * TOL_O["bf16"] * float(np.linalg.norm(ref["o"])) + rnd
        assert float(np.linalg.norm(w - ref["w"])) <= bound, i
    assert off == len(out)
