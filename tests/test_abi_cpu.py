"""C-ABI checks that need no GPU: exports, struct layout, host-only plans,
argument validation and error statuses."""
import ctypes
import os
import re
import subprocess

import pytest

from oracle import muon_ref as R
from paper_2606_27153_amd import _lib as L
from paper_2606_27153_amd.optim import MuonPlan
from paper_2606_27153_amd.workloads import WORKLOAD_KEYS, get_workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "muon.h")


def _declared_functions():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"^MUON_API\s+[\w\s\*]+?\b(muon_\w+)\(", txt, flags=re.M)))


def test_every_declared_symbol_is_exported(lib):
    names = _declared_functions()
    assert len(names) >= 11
    for name in names:
        assert hasattr(lib, name), name
        assert name in L.SIGNATURES, name
    assert lib.muon_abi_version() == 4


def test_struct_layout_matches_c_compiler(tmp_path):
    src = tmp_path / "layout.c"
    structs = {
        "muon_matrix_desc": L.muon_matrix_desc,
        "muon_plan_opts": L.muon_plan_opts,
        "muon_plan_info": L.muon_plan_info,
        "muon_matrix_info": L.muon_matrix_info,
        "muon_kernel_stat": L.muon_kernel_stat,
    }
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "muon.h"', "int main(void){"]
    for sname, cls in structs.items():
        lines.append(f'printf("{sname} size %zu\\n", sizeof({sname}));')
        for f, _ in cls._fields_:
            lines.append(f'printf("{sname} {f} %zu\\n", offsetof({sname}, {f}));')
    lines.append("return 0;}")
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    for line in out:
        if not line:
            continue
        sname, field, val = line.split()
        cls = structs[sname]
        if field == "size":
            assert ctypes.sizeof(cls) == int(val), sname
        else:
            assert getattr(cls, field).offset == int(val), (sname, field)


def test_opts_default(lib):
    o = L.muon_plan_opts()
    assert lib.muon_plan_opts_default(ctypes.byref(o)) == L.MUON_OK
    assert (o.precision, o.max_ns_steps, o.small_m_threshold, o.flags, o.wave_bytes) == (0, 16, 64, 0, 0)
    assert abs(o.a - 3.4445) < 1e-6 and abs(o.b + 4.775) < 1e-6 and abs(o.c - 2.0315) < 1e-6
    assert abs(o.eps - 1e-7) < 1e-12
    assert lib.muon_plan_opts_default(None) == L.MUON_ERR_INVALID_ARG
    assert "NULL" in L.last_error()


def _descs(wl):
    return [(m.rows, m.cols, m.param, m.grad) for m in wl.matrices]


@pytest.mark.parametrize("key", WORKLOAD_KEYS)
def test_host_only_plan_of_each_workload(key):
    wl = get_workload(key)
    plan = MuonPlan(_descs(wl), host_only=True)
    info = plan.info()
    assert info["n_matrices"] == wl.n
    assert info["device"] == -1
    assert info["n_waves"] >= 1
    want = sum(R.ns_flops(m.rows, m.cols, 1) for m in wl.matrices)
    assert abs(info["ns_flops_per_ns_step"] - want) <= 1e-9 * want
    assert info["padded_flops_per_ns_step"] >= info["ns_flops_per_ns_step"]
    assert plan.workspace_bytes > 0
    waves = set()
    for i, m in enumerate(wl.matrices):
        mi = plan.matrix_info(i)
        assert mi["m"] == min(m.rows, m.cols) and mi["n"] == max(m.rows, m.cols)
        assert mi["transposed"] == int(m.rows > m.cols)
        # padded to the tile, or (256 tiles) to 128 with a 128-wide edge strip
        for v, pad in ((mi["m"], mi["m_pad"]), (mi["n"], mi["n_pad"])):
            assert pad >= v and (pad % mi["tile"] == 0 or (mi["tile"] == 256 and pad % 128 == 0 and pad - v < 128))
        assert mi["m"] <= mi["m_pad"] < mi["m"] + mi["tile"]
        assert mi["n"] <= mi["n_pad"] < mi["n"] + mi["tile"]
        assert mi["fp32_ns"] == int(mi["m"] <= 64)
        waves.add(mi["wave"])
    assert waves == set(range(info["n_waves"]))
    plan.close()


def test_fp32_precision_uses_fp32_everywhere():
    wl = get_workload("tiny")
    plan = MuonPlan(_descs(wl), precision="fp32", host_only=True)
    assert all(plan.matrix_info(i)["fp32_ns"] == 1 for i in range(wl.n))


def test_fp16_precision_uses_fp16_everywhere():
    # fp16 keeps every size on 16-bit operands (no fp32 fallback for small m)
    # and still takes the Gram-space form for wide matrices
    wl = get_workload("vla")
    plan = MuonPlan(_descs(wl), precision="fp16", host_only=True)
    for i in range(wl.n):
        mi = plan.matrix_info(i)
        assert mi["fp32_ns"] == 0
        assert L.KERNEL_CLASSES[mi["kernel_class"]].startswith("f16_")
        # the fp16 default threshold, and the Gram-space minimum m of 256
        assert mi["gram_space"] == int(mi["n"] >= 1.4 * mi["m"] and mi["m"] >= 256)
    plan.close()


def test_buckets_of_the_8b_set():
    wl = get_workload("8b")
    plan = MuonPlan(_descs(wl), host_only=True)
    assert plan.info()["n_buckets"] == 3
    shapes = {(plan.matrix_info(i)["m"], plan.matrix_info(i)["n"]) for i in range(wl.n)}
    assert shapes == {(4096, 14336), (4096, 4096), (1024, 4096)}


def test_wave_cap_splits_work():
    wl = get_workload("1b")
    one = MuonPlan(_descs(wl), host_only=True, wave_bytes=1 << 40)
    many = MuonPlan(_descs(wl), host_only=True, wave_bytes=1 << 30)
    assert one.info()["n_waves"] == 1
    assert many.info()["n_waves"] > 1
    assert many.workspace_bytes < one.workspace_bytes


def _create(lib, descs, opts=None):
    arr = (L.muon_matrix_desc * max(1, len(descs)))()
    for i, d in enumerate(descs):
        arr[i].rows, arr[i].cols, arr[i].param_dtype, arr[i].grad_dtype, arr[i].momentum_dtype = d
    h = ctypes.c_void_p()
    if opts is None:
        opts = L.muon_plan_opts()
        lib.muon_plan_opts_default(ctypes.byref(opts))
        opts.flags = L.MUON_PLAN_HOST_ONLY
    st = lib.muon_plan_create(arr, len(descs), ctypes.byref(opts), ctypes.byref(h))
    return st, h


@pytest.mark.parametrize("desc,status", [
    ((0, 5, 1, 1, 0), L.MUON_ERR_INVALID_ARG),
    ((5, -1, 1, 1, 0), L.MUON_ERR_INVALID_ARG),
    ((1 << 31, 5, 1, 1, 0), L.MUON_ERR_INVALID_ARG),
    ((5, 5, 7, 1, 0), L.MUON_ERR_UNSUPPORTED),
    ((5, 5, 1, 9, 0), L.MUON_ERR_UNSUPPORTED),
    ((5, 5, 1, 1, 1), L.MUON_ERR_UNSUPPORTED),   # bf16 momentum
])
def test_plan_create_rejects_bad_descriptors(lib, desc, status):
    st, h = _create(lib, [desc])
    assert st == status
    assert h.value is None
    assert L.last_error()


@pytest.mark.parametrize("field,value", [
    ("precision", 3), ("max_ns_steps", 0), ("max_ns_steps", 65), ("eps", -1.0),
    ("small_m_threshold", -1), ("flags", 0x10), ("wave_bytes", -5), ("a", float("nan")),
    ("c", 1e-39),
])
def test_plan_create_rejects_bad_opts(lib, field, value):
    opts = L.muon_plan_opts()
    lib.muon_plan_opts_default(ctypes.byref(opts))
    opts.flags = L.MUON_PLAN_HOST_ONLY
    setattr(opts, field, value)
    st, h = _create(lib, [(8, 8, 1, 1, 0)], opts)
    assert st == L.MUON_ERR_INVALID_ARG
    assert field.split("_")[0] in L.last_error() or "opts" in L.last_error()


def test_plan_create_accepts_cubic_coefficients(lib):
    opts = L.muon_plan_opts()
    lib.muon_plan_opts_default(ctypes.byref(opts))
    opts.flags = L.MUON_PLAN_HOST_ONLY
    opts.a, opts.b, opts.c = 1.5, -0.5, 0.0
    st, h = _create(lib, [(8, 8, 1, 1, 0)], opts)
    assert st == L.MUON_OK
    assert lib.muon_plan_destroy(h) == L.MUON_OK


QUINTIC = (3.4445, -4.7750, 2.0315)
CLASSIC = (15 / 8, -10 / 8, 3 / 8)
CUBIC = (1.5, -0.5, 0.0)


def _schedule_opts(lib, triples):
    opts = L.muon_plan_opts()
    lib.muon_plan_opts_default(ctypes.byref(opts))
    opts.flags = L.MUON_PLAN_HOST_ONLY
    opts.max_ns_steps = len(triples)
    arr = (ctypes.c_float * (3 * len(triples)))(*[v for t in triples for v in t])
    opts.abc_per_step = arr
    return opts, arr


@pytest.mark.parametrize("bad", [(float("nan"), -1.0, 1.0), (1.0, float("inf"), 1.0), (1.0, -1.0, 1e-39)])
def test_schedule_rejects_bad_triples(lib, bad):
    opts, arr = _schedule_opts(lib, [QUINTIC, QUINTIC, bad, QUINTIC])
    st, h = _create(lib, [(8, 8, 1, 1, 0)], opts)
    assert st == L.MUON_ERR_INVALID_ARG
    assert "abc_per_step step 2" in L.last_error()


def _info(lib, h):
    info = L.muon_plan_info()
    assert lib.muon_plan_get_info(h, ctypes.byref(info)) == L.MUON_OK
    return info


def test_schedule_form_choice_and_launch_count(lib):
    # one wide and one square bf16 matrix
    descs = [(256, 1024, 1, 1, 0), (512, 512, 1, 1, 0)]
    opts, arr = _schedule_opts(lib, [QUINTIC, QUINTIC, QUINTIC, CLASSIC, CLASSIC])
    st, h = _create(lib, descs, opts)
    assert st == L.MUON_OK
    info = _info(lib, h)
    # every c != 0: the wide matrix takes the Gram-space form (segments of 2,
    # 2 and 1 steps: 3L + 1 launches for L = 2, 3 for L = 1, 17 in all), the
    # square one Eq. 2 (3 per step)
    assert info.n_gram == 1 and info.gram_restart == 2
    assert info.launches_per_step == 2 + 17 + 15
    # the plan keeps its own copy of the schedule
    arr[3 * 4 + 2] = 0.0
    assert _info(lib, h).launches_per_step == 2 + 17 + 15
    assert lib.muon_plan_destroy(h) == L.MUON_OK
    # a cubic step keeps every matrix on Eq. 2 and drops that step's A*A
    opts, arr = _schedule_opts(lib, [QUINTIC, QUINTIC, QUINTIC, CUBIC, CLASSIC])
    st, h = _create(lib, descs, opts)
    assert st == L.MUON_OK
    info = _info(lib, h)
    assert info.n_gram == 0
    assert info.launches_per_step == 2 + 14
    assert lib.muon_plan_destroy(h) == L.MUON_OK


def test_padded_dimension_limit(lib):
    # rows and cols may be up to 2^31 - 1, but the padded extent must stay
    # below 2^31; tile indices are 32-bit, so 2^22 columns (65536 tiles of 64)
    # plan fine
    st, h = _create(lib, [(1, (1 << 31) - 1, 1, 1, 0)])
    assert st == L.MUON_ERR_UNSUPPORTED and "2^31" in L.last_error()
    st, h = _create(lib, [(1, 1 << 22, 1, 1, 0), ((1 << 22) + 5, 3, 1, 1, 0)])
    assert st == L.MUON_OK
    assert lib.muon_plan_destroy(h) == L.MUON_OK


def test_null_arguments(lib):
    h = ctypes.c_void_p()
    assert lib.muon_plan_create(None, 1, None, ctypes.byref(h)) == L.MUON_ERR_INVALID_ARG
    arr = (L.muon_matrix_desc * 1)()
    assert lib.muon_plan_create(arr, 0, None, ctypes.byref(h)) == L.MUON_ERR_INVALID_ARG
    assert lib.muon_plan_create(arr, 1, None, None) == L.MUON_ERR_INVALID_ARG
    assert lib.muon_plan_destroy(None) == L.MUON_OK
    b = ctypes.c_size_t()
    assert lib.muon_plan_workspace_bytes(None, ctypes.byref(b)) == L.MUON_ERR_INVALID_ARG
    for s in range(6):
        assert lib.muon_status_string(s).decode().startswith("MUON_")


def test_step_on_host_only_plan_is_rejected_before_any_device_call(lib):
    st, h = _create(lib, [(8, 16, 1, 1, 0)])
    assert st == L.MUON_OK
    p = L.ptr_array([16])
    r = lib.muon_step(h, p, p, p, 0.02, 0.95, 0.01, 5, 1, ctypes.c_void_p(256), 1 << 20, None)
    assert r == L.MUON_ERR_INVALID_ARG
    assert "host-only" in L.last_error()
    mi = L.muon_matrix_info()
    assert lib.muon_plan_matrix_info(h, 5, ctypes.byref(mi)) == L.MUON_ERR_INVALID_ARG
    assert lib.muon_plan_set_timing(h, 1) == L.MUON_ERR_INVALID_ARG
    cnt = ctypes.c_int32()
    assert lib.muon_plan_timing_read(h, None, 0, ctypes.byref(cnt), 1) == L.MUON_OK and cnt.value == 0
    assert lib.muon_plan_destroy(h) == L.MUON_OK


def test_tile_choice_prices_the_k_loop_at_the_real_extent():
    # Cost of one Eq. 2 step as issued: m_pad^2 kn + m_pad^2 km + 2 m_pad n_pad km,
    # with km, kn = m, n rounded to the 64-element K slab, over the class
    # efficiency (256: 1.0, 128: 0.8).
    # 1152 x 1152: 256 tile 4 * 1280^2 * 1152 = 7.55e9; 128 tile 4 * 1152^3 / 0.8 = 7.64e9
    # 640 x 640:   256 tile 4 * 768^2 * 640 = 1.51e9;   128 tile 4 * 640^3 / 0.8 = 1.31e9
    # (pricing K at the padded extent, as the loops once ran, chose 128 for 1152)
    # With edge strips a 256-class 640 x 640 matrix pads to 640 only: its
    # 512 x 512 part at 1.0 and the rest (640^2 - 512^2 of the outputs) at the
    # 128 class's 0.8: 2560 * (512^2 + (640^2 - 512^2) / 0.8) = 1.14e9 < 1.31e9.
    plan = MuonPlan([(1152, 1152, "bf16", "bf16"), (3456, 1152, "bf16", "bf16"), (640, 640, "bf16", "bf16"),
                     (4096, 4096, "bf16", "bf16"), (300, 300, "bf16", "bf16")], host_only=True)
    assert [plan.matrix_info(i)["tile"] for i in range(5)] == [256, 256, 256, 256, 256]
    assert [plan.matrix_info(i)["m_pad"] for i in range(5)] == [1152, 1152, 640, 4096, 384]
    plan.close()


def test_step_buffers_are_checked_against_the_plan():
    # the C ABI sees bare pointers, so the binding checks each buffer's shape,
    # dtype, layout and device before they are handed over
    import torch
    from paper_2606_27153_amd.optim import check_step_tensors
    descs = [(4, 8, "bf16", "f32"), (16, 2, "f32", "bf16")]

    def bufs():
        return ([torch.zeros(4, 8, dtype=torch.bfloat16), torch.zeros(16, 2)],
                [torch.zeros(4, 8), torch.zeros(16, 2, dtype=torch.bfloat16)],
                [torch.zeros(4, 8), torch.zeros(16, 2)])

    p, g, m = bufs()
    with pytest.raises(ValueError, match="not on a GPU"):
        check_step_tensors(descs, p, g, m)
    p, g, m = bufs()
    p[1] = torch.zeros(2, 16)
    with pytest.raises(ValueError, match=r"matrix 1 param has shape \(2, 16\)"):
        check_step_tensors(descs, p, g, m)
    p, g, m = bufs()
    g[0] = torch.zeros(4, 8, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="matrix 0 grad has dtype torch.bfloat16, the plan expects float32"):
        check_step_tensors(descs, p, g, m)
    p, g, m = bufs()
    m[1] = torch.zeros(2, 16).t()   # right shape, column-major
    with pytest.raises(ValueError, match="matrix 1 momentum is not contiguous"):
        check_step_tensors(descs, p, g, m)
    p, g, m = bufs()
    with pytest.raises(ValueError, match="matrix 0 update_out has dtype"):
        check_step_tensors(descs, p, g, m, update_out=[torch.zeros(4, 8, dtype=torch.bfloat16), None])
    with pytest.raises(ValueError, match="expected 2 params"):
        check_step_tensors(descs, p[:1], g, m)
    with pytest.raises(TypeError, match="unsupported dtype"):
        check_step_tensors(descs, [torch.zeros(4, 8, dtype=torch.float16), p[1]], g, m)


def test_plan_create_accepts_the_buffer_check_flag(lib):
    opts = L.muon_plan_opts()
    lib.muon_plan_opts_default(ctypes.byref(opts))
    opts.flags = L.MUON_PLAN_HOST_ONLY | L.MUON_PLAN_CHECK_BUFFERS
    st, h = _create(lib, [(8, 8, 1, 1, 0)], opts)
    assert st == L.MUON_OK
    assert lib.muon_plan_destroy(h) == L.MUON_OK


def test_step_path_never_waits_for_the_stream():
    # the step refreshes its pointer table with a stream-ordered copy; no
    # stream or device synchronisation anywhere in the step's code
    src = open(os.path.join(ROOT, "paper_2606_27153_amd", "csrc", "api.cpp")).read()
    body = src[src.index("muon_status step_impl("):src.index("void release_events(")]
    for call in ("hipStreamSynchronize", "hipDeviceSynchronize", "hipMemcpy(", "hipMalloc", "hipHostMalloc",
                 "hipFree"):
        assert call not in body, call


def test_diag_library_exports_the_ceiling_probe():
    """The bench's matrix-core ceiling probe lives in its own library; its
    argument checks run before any HIP call."""
    from paper_2606_27153_amd.build import DIAG_LIB_PATH
    diag = ctypes.CDLL(DIAG_LIB_PATH)
    fn = diag.muon_diag_mfma_ceiling
    fn.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    dummy = ctypes.c_void_p(16)
    assert fn(0, 10, 0, dummy, None) == -1
    assert fn(4, 0, 0, dummy, None) == -1
    assert fn(4, 10, 3, dummy, None) == -1
    assert fn(4, 10, 0, None, None) == -1
