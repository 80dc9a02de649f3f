"""Host-side checks of the C ABI: the library loads, exports every symbol the
header declares, sizes its workspace as documented and rejects bad arguments
before touching the GPU (no kernel is ever launched by these tests)."""

import ctypes
import os
import re

import pytest
import torch

from oracle import pfc_oracle as O
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pfc.h")

pfc = pytest.importorskip("paper_2010_05222_amd.pfc", reason="libpfc.so not built")

FAKE = 0x1000        # never dereferenced: every call below fails its checks first


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pfc_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = _declared_functions()
    assert set(names) == set(pfc.EXPORTS)
    lib = ctypes.CDLL(pfc.LIB_PATH)
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings():
    for st in range(7):
        assert pfc.pfc_status_string(st) not in ("", "unknown status")
    assert pfc.pfc_status_string(99) == "unknown status"


@pytest.mark.parametrize("name", list(workloads.CONFIGS))
def test_workspace_and_capacity_of_each_workload(name):
    cfg = workloads.config(name)
    code = {"f32": pfc.PFC_F32, "bf16": pfc.PFC_BF16, "f16": pfc.PFC_F16}[cfg["dtype"]]
    nbytes, cap = pfc.pfc_workspace_bytes(cfg["B"], cfg["d"], cfg["C"], cfg["r"], code)
    b = O.budget(cfg["r"], cfg["C"])
    assert cap == max(b, min(cfg["B"], cfg["C"]))
    # Dominated by the logit store [B x cap] and the sampler's per-class
    # digits (2 B) and candidate keys (8 B).
    elt = 4 if code == pfc.PFC_F32 else 2
    assert nbytes >= cfg["B"] * cap * elt + cfg["C"] * 10
    assert nbytes < 2 * (cfg["B"] * cap * elt + cfg["C"] * 10) + (256 << 20)


def test_batch_limit_matches_header():
    text = open(HEADER).read()
    assert int(re.search(r"#define PFC_MAX_BATCH (\d+)", text).group(1)) == pfc.PFC_MAX_BATCH
    nbytes, cap = pfc.pfc_workspace_bytes(pfc.PFC_MAX_BATCH, 512, 40000, 0.2, pfc.PFC_F16)
    assert cap == 8192 and nbytes > 0


def test_capacity_when_positives_exceed_budget():
    _, cap = pfc.pfc_workspace_bytes(512, 128, 1000, 0.05, pfc.PFC_BF16)
    assert cap == 512                     # max(b = 50, min(B, C) = 512)
    _, cap = pfc.pfc_workspace_bytes(4, 128, 3, 0.5, pfc.PFC_BF16)
    assert cap == 3


@pytest.mark.parametrize("args,status", [
    ((0, 128, 100, 0.1, 1), pfc.PFC_ERR_INVALID_ARG),      # B = 0
    ((8, 0, 100, 0.1, 1), pfc.PFC_ERR_INVALID_ARG),        # d = 0
    ((8, 12, 100, 0.1, 0), pfc.PFC_ERR_INVALID_ARG),       # d not a multiple of 8
    ((8, 128, 0, 0.1, 1), pfc.PFC_ERR_INVALID_ARG),        # C = 0
    ((8, 128, 100, 0.0, 1), pfc.PFC_ERR_INVALID_ARG),      # r = 0
    ((8, 128, 100, 1.5, 1), pfc.PFC_ERR_INVALID_ARG),      # r > 1
    ((8, 128, 100, float("nan"), 1), pfc.PFC_ERR_INVALID_ARG),
    ((8, 128, 100, 0.1, 7), pfc.PFC_ERR_UNSUPPORTED),      # unknown dtype
    ((8, 64, 100, 0.1, 1), pfc.PFC_ERR_UNSUPPORTED),       # 16-bit path needs d % 128 == 0
    ((8, 1024, 100, 0.1, 2), pfc.PFC_ERR_UNSUPPORTED),     # 16-bit path needs d <= 512
    ((8192, 128, 100, 0.1, 0), pfc.PFC_ERR_UNSUPPORTED),   # fp32 path limited to B <= 4096
    ((8193, 512, 100000, 0.1, 2), pfc.PFC_ERR_INVALID_ARG),  # B above PFC_MAX_BATCH
])
def test_workspace_rejects(args, status):
    with pytest.raises(pfc.PfcError) as e:
        pfc.pfc_workspace_bytes(*args)
    assert e.value.status == status


def _sample_args(**kw):
    a = dict(labels=FAKE, B=16, C=1000, class_offset=0, r=0.1, seed=0, active=FAKE,
             active_cap=100, n_active=FAKE, labels_mapped=FAKE, ws=FAKE, ws_bytes=1 << 30,
             stream=0)
    a.update(kw)
    return a


@pytest.mark.parametrize("kw,status", [
    (dict(labels=0), pfc.PFC_ERR_INVALID_ARG),
    (dict(active=0), pfc.PFC_ERR_INVALID_ARG),
    (dict(B=0), pfc.PFC_ERR_INVALID_ARG),
    (dict(B=8193, active_cap=8193, C=100000), pfc.PFC_ERR_INVALID_ARG),   # B > PFC_MAX_BATCH
    (dict(C=-1), pfc.PFC_ERR_INVALID_ARG),
    (dict(class_offset=-5), pfc.PFC_ERR_INVALID_ARG),
    (dict(r=0.0), pfc.PFC_ERR_INVALID_ARG),
    (dict(active_cap=99), pfc.PFC_ERR_CAPACITY),
    (dict(ws=0), pfc.PFC_ERR_WORKSPACE),
    (dict(ws=FAKE + 16), pfc.PFC_ERR_WORKSPACE),          # not 256-byte aligned
    (dict(ws_bytes=1024), pfc.PFC_ERR_WORKSPACE),
])
def test_sample_rejects_before_launch(kw, status):
    with pytest.raises(pfc.PfcError) as e:
        pfc.pfc_sample(**_sample_args(**kw))
    assert e.value.status == status


def _fwd_args(**kw):
    a = dict(X=FAKE, x_dtype=1, B=16, d=128, W=FAKE, w_dtype=1, C=1000, active=FAKE,
             n_active=FAKE, active_cap=100, labels_mapped=FAKE, compute_dtype=1, s=64.0, m=0.5,
             margin=1, tau=2.0, loss=FAKE, row_lse=FAKE, ws=FAKE, ws_bytes=1 << 40, stream=0)
    a.update(kw)
    return a


@pytest.mark.parametrize("kw,status", [
    (dict(X=0), pfc.PFC_ERR_INVALID_ARG),
    (dict(tau=float("nan")), pfc.PFC_ERR_INVALID_ARG),
    (dict(s=0.0), pfc.PFC_ERR_INVALID_ARG),
    (dict(s=float("inf")), pfc.PFC_ERR_INVALID_ARG),
    (dict(m=-0.1), pfc.PFC_ERR_INVALID_ARG),
    (dict(m=3.2), pfc.PFC_ERR_INVALID_ARG),              # ArcFace margin must be < pi
    (dict(margin=5), pfc.PFC_ERR_INVALID_ARG),
    (dict(x_dtype=2), pfc.PFC_ERR_UNSUPPORTED),          # mixed operand types
    (dict(active_cap=0), pfc.PFC_ERR_CAPACITY),
    (dict(active_cap=1001), pfc.PFC_ERR_CAPACITY),
    (dict(ws_bytes=4096), pfc.PFC_ERR_WORKSPACE),
    (dict(ws=FAKE + 128), pfc.PFC_ERR_WORKSPACE),         # not 256-byte aligned
])
def test_forward_rejects_before_launch(kw, status):
    with pytest.raises(pfc.PfcError) as e:
        pfc.pfc_forward_loss(**_fwd_args(**kw))
    assert e.value.status == status


def _bwd_args(**kw):
    a = dict(X=FAKE, x_dtype=1, B=16, d=128, W=FAKE, w_dtype=1, W_master=0, momentum=FAKE,
             C=1000, active=FAKE, n_active=FAKE, active_cap=100, labels_mapped=FAKE,
             compute_dtype=1, s=64.0, m=0.5, margin=1, row_lse=FAKE, lr=0.1, mu=0.9, dX=FAKE,
             ws=FAKE, ws_bytes=1 << 40, stream=0)
    a.update(kw)
    return a


@pytest.mark.parametrize("kw,status", [
    (dict(momentum=0), pfc.PFC_ERR_INVALID_ARG),
    (dict(dX=0), pfc.PFC_ERR_INVALID_ARG),
    (dict(row_lse=0), pfc.PFC_ERR_INVALID_ARG),
    (dict(lr=0.0), pfc.PFC_ERR_INVALID_ARG),
    (dict(mu=1.0), pfc.PFC_ERR_INVALID_ARG),
    (dict(mu=-0.5), pfc.PFC_ERR_INVALID_ARG),
    (dict(d=256, x_dtype=0, w_dtype=1, compute_dtype=1), pfc.PFC_ERR_UNSUPPORTED),
    (dict(ws=0), pfc.PFC_ERR_WORKSPACE),
    (dict(ws=FAKE + 8), pfc.PFC_ERR_WORKSPACE),           # not 256-byte aligned
])
def test_backward_rejects_before_launch(kw, status):
    with pytest.raises(pfc.PfcError) as e:
        pfc.pfc_backward_update(**_bwd_args(**kw))
    assert e.value.status == status


def _stage_args(**kw):
    a = dict(banks=[FAKE], slots=[FAKE + 16], row_bytes=[256], C=1000, next_active=FAKE,
             next_n=FAKE, prev_active=0, prev_n=0, prev2_active=0, prev2_n=0, active_cap=100,
             bank_version=0, row_version=0, version=1, stale=0, stream=0)
    a.update(kw)
    return a


@pytest.mark.parametrize("kw", [
    dict(banks=[0]), dict(slots=[0]), dict(next_active=0), dict(next_n=0),
    dict(C=0), dict(row_bytes=[8]), dict(row_bytes=[24]), dict(row_bytes=[1 << 17]),
    dict(active_cap=0),
    dict(prev_active=FAKE),                   # a previous list without its count
    dict(prev2_n=FAKE),
    dict(bank_version=FAKE),                  # versions come in pairs
    dict(banks=[], slots=[], row_bytes=[]),   # no array
    dict(banks=[FAKE] * 4, slots=[FAKE + 16] * 4, row_bytes=[256] * 4),   # more than three
    dict(banks=[FAKE, 0], slots=[FAKE + 16, FAKE + 32], row_bytes=[256, 512]),
    dict(banks=[FAKE, FAKE + 48], slots=[FAKE + 16, FAKE + 32], row_bytes=[256, 0]),
    dict(slots=[FAKE]),                       # a bank copied onto itself
])
def test_bank_stage_rejects_before_launch(kw):
    with pytest.raises(pfc.PfcError) as e:
        pfc.pfc_bank_stage(**_stage_args(**kw))
    assert e.value.status == pfc.PFC_ERR_INVALID_ARG


def test_bank_array_lists_must_match():
    with pytest.raises(ValueError):
        pfc.pfc_bank_stage(**_stage_args(row_bytes=[256, 512]))


@pytest.mark.parametrize("kw", [
    dict(prev_slots=[0]), dict(next_slots=[0]), dict(prev_active=0), dict(next_n=0),
    dict(next_slots=[FAKE]), dict(row_bytes=[0]),
    dict(prev_slots=[], next_slots=[], row_bytes=[]),
])
def test_bank_patch_rejects_before_launch(kw):
    a = dict(prev_slots=[FAKE], next_slots=[FAKE + 32], row_bytes=[256], prev_active=FAKE,
             prev_n=FAKE, next_active=FAKE, next_n=FAKE, active_cap=100, stream=0)
    a.update(kw)                              # next_slots=[FAKE]: a slot patched onto itself
    with pytest.raises(pfc.PfcError) as e:
        pfc.pfc_bank_patch(**a)
    assert e.value.status == pfc.PFC_ERR_INVALID_ARG


@pytest.mark.parametrize("kw", [dict(slots=[0]), dict(banks=[0]), dict(C=-1),
                                dict(row_bytes=[100]), dict(next_active=FAKE),
                                dict(slots=[FAKE] * 4, banks=[FAKE + 16] * 4,
                                     row_bytes=[256] * 4)])
def test_bank_writeback_rejects_before_launch(kw):
    a = dict(slots=[FAKE], banks=[FAKE + 16], row_bytes=[256], active=FAKE, n_active=FAKE,
             next_active=0, next_n=0, active_cap=100, C=1000, bank_version=0, version=1,
             stream=0)
    a.update(kw)
    with pytest.raises(pfc.PfcError) as e:
        pfc.pfc_bank_writeback(**a)
    assert e.value.status == pfc.PFC_ERR_INVALID_ARG


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="only meaningful without a GPU")
def test_bank_without_device_reports_hip_error():
    with pytest.raises(pfc.PfcError) as e:
        pfc.pfc_bank_stage(**_stage_args())
    assert e.value.status == pfc.PFC_ERR_HIP


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="only meaningful without a GPU")
def test_no_device_reports_hip_error():
    """With no HIP device the launch fails and the ABI reports PFC_ERR_HIP."""
    with pytest.raises(pfc.PfcError) as e:
        pfc.pfc_sample(**_sample_args())
    assert e.value.status == pfc.PFC_ERR_HIP


def _noalloc_args(**kw):
    a = dict(labels=FAKE, B=16, C=1000, class_offset=0, r=0.1, seed=0, active=FAKE,
             active_cap=100, n_active=FAKE, labels_mapped=FAKE, stream=0)
    a.update(kw)
    return a


@pytest.mark.parametrize("kw,status", [
    (dict(labels=0), pfc.PFC_ERR_INVALID_ARG),
    (dict(n_active=0), pfc.PFC_ERR_INVALID_ARG),
    (dict(B=0), pfc.PFC_ERR_INVALID_ARG),
    (dict(B=8193, active_cap=8193, C=100000), pfc.PFC_ERR_INVALID_ARG),
    (dict(r=1.5), pfc.PFC_ERR_INVALID_ARG),
    (dict(active_cap=99), pfc.PFC_ERR_CAPACITY),
    (dict(C=(1 << 21) + 1, active_cap=1 << 21), pfc.PFC_ERR_SCRATCH),   # beyond the static scratch
])
def test_sample_noalloc_rejects_before_launch(kw, status):
    with pytest.raises(pfc.PfcError) as e:
        pfc.pfc_sample_noalloc(**_noalloc_args(**kw))
    assert e.value.status == status


def test_noalloc_limit_matches_header():
    text = open(HEADER).read()
    assert "(1LL << 21)" in re.search(r"#define PFC_NOALLOC_MAX_CLASSES (.*)", text).group(1)
    assert pfc.PFC_NOALLOC_MAX_CLASSES == 1 << 21


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="only meaningful without a GPU")
def test_noalloc_without_device_reports_hip_error():
    with pytest.raises(pfc.PfcError) as e:
        pfc.pfc_sample_noalloc(**_noalloc_args())
    assert e.value.status == pfc.PFC_ERR_HIP
