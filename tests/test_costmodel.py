"""The cost model behind the roofline figures reproduces the paper's printed
analytic numbers (tests/golden/paper_analytic.json)."""

import json
import os

from paper_2010_05222_amd import costmodel as cm
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_analytic.json")


def _golden():
    with open(GOLDEN) as fh:
        return json.load(fh)


def test_first_order_traffic_matches_paper():
    g = _golden()
    s = g["traffic_setting"]
    mp = cm.first_order_traffic_elements(s["N"], s["k"], s["d"], s["C"], s["r"], "mp")
    dp = cm.first_order_traffic_elements(s["N"], s["k"], s["d"], s["C"], s["r"], "dp")
    full = cm.first_order_traffic_elements(s["N"], s["k"], s["d"], s["C"], 1.0, "mp")
    want = g["traffic_million_elements"]
    assert round(mp / 1e6, 1) == want["mp_pfc"]
    assert round(dp / 1e6, 1) == want["dp_pfc"]
    assert round(full / 1e6, 1) == want["full_mp"]


def test_aspect_ratios_match_paper():
    g = _golden()
    s = g["traffic_setting"]
    rows_mp = s["N"] * s["k"]
    want = g["aspect_ratios"]
    assert round(s["r"] * s["C"] / s["k"] / rows_mp) == want["mp_pfc"]
    assert round(s["C"] / s["k"] / rows_mp) == want["full_mp"]
    assert round(s["r"] * s["C"] / s["N"]) == want["dp_pfc"]


def test_fc_memory_matches_paper():
    g = _golden()
    s = g["memory_setting"]
    for k, key in ((8, "k8"), (80, "k80")):
        m_w, m_logit, m_fc = cm.fc_memory_bytes(s["N"], k, s["d"], s["classes_per_gpu"])
        assert round(m_fc / 1e9, 1) == g["memory_gb"][key]
        assert round(2 * m_logit / m_fc, 2) == g["logit_share"][key]
    m_w, m_logit, _ = cm.fc_memory_bytes(s["N"], 80, s["d"], s["classes_per_gpu"])
    assert m_logit / m_w == g["logit_to_weight_ratio_k80"]


def test_massive_workload_figures():
    cfg = workloads.config("massive")
    K = 800_000
    assert cm.step_flops(cfg["B"], cfg["d"], K) == 3 * 2 * 1024 * 512 * 800_000
    assert cm.update_bytes(K, cfg["d"], cfg["dtype"], cfg["master"]) == 800_000 * 512 * 12
