"""pfc_sample_noalloc (no workspace; static device scratch) against
pfc_sample (caller workspace): bit-identical active sets, |S| and remapped
labels on two calls in a row, the second smaller than the first, both through
the C ABI.  The second call reuses the scratch the first one left behind.
Also captured into a HIP graph and replayed with new labels."""

import numpy as np
import pytest
import torch

from oracle import pfc_oracle as O

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2010_05222_amd import pfc  # noqa: F401  (fails loudly if libpfc.so is missing)
    return torch.device("cuda:0")


def _labels(rng, B, lo, hi, dev):
    return torch.from_numpy(rng.integers(lo, hi, size=B).astype(np.int64)).to(dev)


def _with_workspace(L, B, C, a, r, seed, cap, dev):
    from paper_2010_05222_amd import pfc
    ws_bytes, _ = pfc.pfc_workspace_bytes(B, 128, C, r, pfc.PFC_F32 if B <= 4096 else pfc.PFC_BF16)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    act = torch.full((cap,), -7, dtype=torch.int32, device=dev)
    n = torch.zeros(1, dtype=torch.int32, device=dev)
    mapped = torch.full((B,), -7, dtype=torch.int32, device=dev)
    s = torch.cuda.current_stream(dev).cuda_stream
    pfc.pfc_sample(L.data_ptr(), B, C, a, r, seed, act.data_ptr(), cap, n.data_ptr(),
                   mapped.data_ptr(), ws.data_ptr(), ws_bytes, s)
    return act, n, mapped


def _noalloc(L, B, C, a, r, seed, cap, dev):
    from paper_2010_05222_amd import pfc
    act = torch.full((cap,), -9, dtype=torch.int32, device=dev)
    n = torch.zeros(1, dtype=torch.int32, device=dev)
    mapped = torch.full((B,), -9, dtype=torch.int32, device=dev)
    s = torch.cuda.current_stream(dev).cuda_stream
    pfc.pfc_sample_noalloc(L.data_ptr(), B, C, a, r, seed, act.data_ptr(), cap, n.data_ptr(),
                           mapped.data_ptr(), s)
    return act, n, mapped


def test_noalloc_matches_workspace_entry_point(dev):
    from paper_2010_05222_amd import pfc
    rng = np.random.default_rng(31)
    # Call 1: the largest accepted shard (2^21 classes), 1,024 labels, r = 0.2.
    # Call 2: a smaller shard at an offset, fewer rows, a third of the labels
    # outside the shard; it runs on the scratch call 1 left behind.
    cases = [(1024, 1 << 21, 0, 0.2, 5, (0, 1 << 21)),
             (100, 5000, 1000, 0.1, 6, (0, 7500))]
    for B, C, a, r, seed, span in cases:
        print(f"\nnoalloc case B={B} C={C} offset={a} r={r} seed={seed}", flush=True)
        _, cap = pfc.pfc_workspace_bytes(B, 128, C, r, pfc.PFC_BF16)
        L = _labels(rng, B, *span, dev)
        ref = _with_workspace(L, B, C, a, r, seed, cap, dev)
        got = _noalloc(L, B, C, a, r, seed, cap, dev)
        torch.cuda.synchronize()
        K = int(ref[1].item())
        assert int(got[1].item()) == K
        assert torch.equal(got[0][:K], ref[0][:K])
        assert torch.equal(got[2], ref[2])
        active_ref, mapped_ref, _ = O.sample_active(L.cpu().numpy(), C, a, r, seed)
        assert np.array_equal(got[0][:K].cpu().numpy(), active_ref)
        assert np.array_equal(got[2].cpu().numpy(), mapped_ref)
        print(f"|S|={K} equal to pfc_sample and to the oracle", flush=True)


def test_noalloc_rejects_oversized_shard(dev):
    from paper_2010_05222_amd import pfc
    L = torch.zeros(4, dtype=torch.int64, device=dev)
    out = torch.empty(1 << 21, dtype=torch.int32, device=dev)
    with pytest.raises(pfc.PfcError) as e:
        pfc.pfc_sample_noalloc(L.data_ptr(), 4, (1 << 21) + 1, 0, 0.1, 0, out.data_ptr(),
                               (1 << 21), out.data_ptr(), out.data_ptr(), 0)
    assert e.value.status == pfc.PFC_ERR_SCRATCH


def test_noalloc_under_graph_capture(dev):
    """The entry point allocates and synchronises nothing, so a caller can
    capture it into a HIP graph: replays, with new labels written into the
    captured input between them, each equal a direct call on those labels
    and the oracle."""
    from paper_2010_05222_amd import pfc
    B, C, a, r, seed = 256, 40000, 0, 0.1, 8
    _, cap = pfc.pfc_workspace_bytes(B, 128, C, r, pfc.PFC_BF16)
    rng = np.random.default_rng(33)
    L = _labels(rng, B, 0, C, dev)
    act = torch.full((cap,), -9, dtype=torch.int32, device=dev)
    n = torch.zeros(1, dtype=torch.int32, device=dev)
    mapped = torch.full((B,), -9, dtype=torch.int32, device=dev)
    _noalloc(L, B, C, a, r, seed, cap, dev)   # a direct call first (scratch address looked up)
    torch.cuda.synchronize()
    print(f"\nnoalloc under graph capture: B={B} C={C} r={r} seed={seed}", flush=True)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pfc.pfc_sample_noalloc(L.data_ptr(), B, C, a, r, seed, act.data_ptr(), cap, n.data_ptr(),
                               mapped.data_ptr(), torch.cuda.current_stream(dev).cuda_stream)
    for rep in range(3):
        L.copy_(_labels(rng, B, 0, C, dev))   # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = (act.clone(), n.clone(), mapped.clone())
        ref = _noalloc(L, B, C, a, r, seed, cap, dev)
        torch.cuda.synchronize()
        K = int(ref[1].item())
        assert int(got[1].item()) == K
        assert torch.equal(got[0][:K], ref[0][:K])
        assert torch.equal(got[2], ref[2])
        active_ref, mapped_ref, _ = O.sample_active(L.cpu().numpy(), C, a, r, seed)
        assert np.array_equal(got[0][:K].cpu().numpy(), active_ref)
        assert np.array_equal(got[2].cpu().numpy(), mapped_ref)
        print(f"replay {rep}: |S|={K} equal to a direct call and to the oracle", flush=True)
