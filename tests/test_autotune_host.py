"""Host-side checks of the measured tile choice: candidates per operand type,
coordinate descent from the cost model's tiles to the fastest set, the
on-disk cache (a second tuning of the same set measures nothing), and the
plan honouring tile hints."""
import ctypes
import json

import pytest

from paper_2606_27153_amd import _lib as L
from paper_2606_27153_amd import autotune as T
from paper_2606_27153_amd.optim import MuonPlan


def test_candidate_tiles():
    assert T.candidate_tiles(4096, 14336, "bf16") == (256, 128, 64)
    assert T.candidate_tiles(32, 512, "bf16") == (128, 64)      # small m runs fp32 under bf16
    assert T.candidate_tiles(32, 512, "fp16") == (256, 128, 64)
    assert T.candidate_tiles(4096, 4096, "fp32") == (128, 64)


def test_tune_descends_to_the_fastest_set_and_caches(tmp_path):
    # a separable cost: each shape has one best tile; the step time is the
    # sum over the reduced set, so one pass of coordinate descent finds it
    best = {(4096, 14336): 128, (512, 32): 64, (1000, 1000): 256}
    calls = []

    def timer(ds):
        calls.append(len(ds))
        return sum(1.0 if d[4] == best[(d[0], d[1])] else 2.0 + d[4] / 256 for d in ds)

    descs = [(4096, 14336, "bf16", "bf16")] * 3 + [(512, 32, "bf16", "bf16")] * 20 + [(1000, 1000, "f32", "f32")]
    path = str(tmp_path / "tiles.json")
    kw = dict(precision="bf16", cache_path=path, timer=timer, device_name="dev", abi=3)
    hints = T.tune(descs, **kw)
    assert hints == [128] * 3 + [64] * 20 + [256]
    # the reduced set keeps at most 16 of a shape; one base measurement plus
    # one per alternative tile of each shape (2 + 1 + 2)
    assert calls == [3 + 16 + 1] * 6
    entry = next(iter(json.load(open(path)).values()))
    assert entry["ms"] < entry["base_ms"]
    calls.clear()
    assert T.tune(descs, **kw) == hints and calls == []
    # another execution mode is another key
    T.tune(descs[:1], **dict(kw, precision="fp16"))
    assert calls == [1] * 3


def test_tune_keeps_the_cost_model_choice_without_a_clear_gain(tmp_path):
    base = T.planner_tiles([(300, 900, "bf16", "bf16")], precision="bf16", gram_min_aspect=2.0)

    def timer(ds):                       # every tile within 0.5 % of the others
        return 10.0 - 0.04 * (ds[0][4] != base[0])
    hints = T.tune([(300, 900, "bf16", "bf16")], precision="bf16", cache_path=str(tmp_path / "c.json"),
                   timer=timer, device_name="dev", abi=3)
    assert hints == base


def test_plan_honours_tile_hints():
    plan = MuonPlan([(300, 900, "bf16", "bf16", 64), (300, 900, "bf16", "bf16", 256),
                     (300, 900, "bf16", "bf16"), (40, 500, "bf16", "bf16", 64)], host_only=True)
    tiles = [plan.matrix_info(i)["tile"] for i in range(4)]
    assert tiles[0] == 64 and tiles[1] == 256 and tiles[3] == 64
    assert plan.matrix_info(3)["fp32_ns"] == 1
    assert plan.info()["n_buckets"] >= 3
    plan.close()


@pytest.mark.parametrize("desc,hint,status", [((300, 900), 100, L.MUON_ERR_INVALID_ARG),
                                              ((300, 900), -64, L.MUON_ERR_INVALID_ARG),
                                              ((40, 500), 256, L.MUON_ERR_UNSUPPORTED)])
def test_bad_tile_hints(lib, desc, hint, status):
    arr = (L.muon_matrix_desc * 1)()
    arr[0].rows, arr[0].cols = desc
    arr[0].param_dtype = arr[0].grad_dtype = L.MUON_BF16
    arr[0].momentum_dtype = L.MUON_F32
    arr[0].tile_hint = hint
    opts = L.muon_plan_opts()
    lib.muon_plan_opts_default(ctypes.byref(opts))
    opts.flags = L.MUON_PLAN_HOST_ONLY
    h = ctypes.c_void_p()
    assert lib.muon_plan_create(arr, 1, ctypes.byref(opts), ctypes.byref(h)) == status
    assert "tile_hint" in L.last_error()
