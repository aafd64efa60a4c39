"""Host logic of bench.py (no GPU): every stage a step variant times has its
algorithmic work, the roofline classification, the stored traffic table,
and the one-GPU rule."""
import functools
import subprocess
import sys
import types

import pytest

import bench
from datagen.clouds import N_CLASSES, make_workload

_workload = functools.lru_cache(maxsize=None)(make_workload)

VARIANTS = [("slice", False), ("deform", False), ("train", False), ("unet", False), ("pointnet", False),
            ("deform", True), ("unet", True), ("pointnet", True)]


def _names(w, tail, backward):
    """Pipeline.stage_names without building a pipeline (it needs a GPU)."""
    fake = types.SimpleNamespace(convs=list(w.convs), tail=tail, backward=backward or tail == "train")
    return bench.Pipeline.stage_names(fake)


@pytest.mark.parametrize("config", [2, 3, 4, 5])
@pytest.mark.parametrize("tail,backward", VARIANTS)
def test_every_stage_has_its_work(config, tail, backward):
    w = _workload(config)
    if tail == "pointnet" and w.convs[0].c_in != 64:
        pytest.skip("the PointNet step needs a first conv with 64 inputs")
    V, Vc = 10_000, 2_000
    n_cls = N_CLASSES[config] if tail == "deform" else 0
    f_raw = 3 if tail == "pointnet" else -1
    work = bench.algorithmic_work(w, V, n_cls, Vc if tail == "unet" else 0, f_raw)
    names = _names(w, tail, backward)
    assert len(names) == len(set(names))
    for n in names:
        assert n in work, (tail, backward, n)
        e = bench.roofline_entry(n, 0.01, work[n])
        assert e["bound"] in ("hbm", "mfma", "alu") and 0 < e["achieved"] and e["peak"] > 0
    if backward or tail == "train":
        assert names[-1] == ("distribute_bwd" if tail == "pointnet" else "splat_bwd")
        assert sum(n.endswith("_bwd_in") for n in names) == len(w.convs)


def test_roofline_classification():
    # a contraction above its ridge is MFMA-bound, below it HBM-bound
    hi = {"bytes": 1e6, "flops": 1e12, "dtype": "bf16"}
    lo = {"bytes": 1e9, "flops": 1e9, "dtype": "bf16"}
    assert bench.roofline_entry("x", 1.0, hi)["bound"] == "mfma"
    assert bench.roofline_entry("x", 1.0, lo)["bound"] == "hbm"
    e = bench.roofline_entry("x", 1.0, {"bytes": 8e9})  # 8 GB in 1 ms
    assert e["bound"] == "hbm" and e["achieved"] == pytest.approx(8e9 / 1e-3 / 1e9)
    assert e["frac"] == pytest.approx(e["achieved"] / bench.HBM_PEAK_GBS)


def test_stored_traffic_matches_the_sources():
    """Each stored counter entry names the kernel sources it was measured on;
    while they are unchanged the bench line reports it, with its origin."""
    import json

    table = json.load(open(bench.TRAFFIC_FILE))
    assert table["calibration"]["fetch_scale"] > 0 and table["calibration"]["write_scale"] > 0
    for key, e in table["entries"].items():
        workload, stage = key.split("/")
        got, why = bench.measured_traffic(workload, stage)
        if e["source_sha1"] == bench.source_hash(stage):
            assert got is not None and got > 0 and "not measured in this run" in why
        else:
            assert got is None and "measured on kernel source" in why


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU only" in r.stderr
