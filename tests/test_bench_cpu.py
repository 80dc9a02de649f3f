"""bench.py's accounting helpers on the CPU (no GPU, no kernel launch): the
roofline entry, the gather figure and the contraction labels of each workload."""

import importlib.util
import os

import pytest

import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("name", list(workloads.CONFIGS))
def test_roofline_and_gather_entries(bench, name):
    from paper_2010_05222_amd import costmodel as cm
    cfg = workloads.config(name)
    K = 1000
    stage_ms = {"fwd_gemm": 1.0, "dx_gemm": 1.0, "dw_update": 2.0}
    dw = bench.roofline_entry("dw_update", cfg, K, 2.0, None)
    assert dw["bound"] in ("hbm", "mfma") and dw["frac"] > 0
    nbytes = cm.update_bytes(K, cfg["d"], cfg["dtype"], cfg["master"])
    if dw["bound"] == "hbm":
        assert dw["achieved"] == pytest.approx(nbytes / 2e-3 / 1e9)
    assert dw["traffic_GBps"] is None
    dwt = bench.roofline_entry("dw_update", cfg, K, 2.0, 3.0e9)
    assert dwt["traffic"] == 3.0e9 and dwt["traffic_GBps"] == pytest.approx(1500.0)
    g = bench.gather_entry(cfg, K, stage_ms, None)
    elt = cm.DTYPE_BYTES[cfg["dtype"]]
    assert g["bytes"] == K * cfg["d"] * elt
    assert g["achieved"] == pytest.approx(K * cfg["d"] * elt / 1e-3 / 1e9)
    assert g["frac"] == pytest.approx(g["achieved"] / cm.PEAK_HBM_GBPS)
    assert g["w_row_read_bytes_per_step"] == 3 * g["bytes"]
    labels = bench.contraction_precision(cfg["dtype"])
    assert set(labels) == {"forward", "dx", "dw"}
    if cfg["dtype"] != "f32":
        assert labels["dw"].startswith("bf16")
