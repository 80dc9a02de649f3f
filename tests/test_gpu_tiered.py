"""Tiered class storage: the class bank in pinned host memory, every step on a
device slot of its active rows (Sec. 3.3.3, the paragraph on asynchronous
hierarchical class storage, Fig. async_pipeline).

A tiered step runs the resident step's kernels on a slot that holds the active
rows in S order, so it must reproduce the resident step bit for bit: each
step's loss, row_lse and dX, and, after the last write-back, the bank equals
the resident W, momentum (and master).  The labels are drawn from a narrow
range so that consecutive active sets share many rows (positives and
negatives), which exercises the patch path.  A multi-step fp32 run is also
compared with the oracle applied step after step.  The versions stamped by
staging and write-back name the last step that touched each row, and rows
staged while their update was still unwritten are counted as stale.
"""

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


TDT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}


def _inputs(B, d, C, dtype, T, seed, dev, span):
    rng = np.random.default_rng(seed)
    W = (0.01 * rng.standard_normal((C, d))).astype(np.float32)
    M = (1e-3 * rng.standard_normal((C, d))).astype(np.float32)
    Xs = [torch.from_numpy(rng.standard_normal((B, d)).astype(np.float32)).to(TDT[dtype]).to(dev)
          for _ in range(T)]
    Ls = [torch.from_numpy(rng.integers(0, span, size=B).astype(np.int64)).to(dev)
          for _ in range(T)]
    return W, M, Xs, Ls


@pytest.mark.parametrize("n_slots", [2, 3])
@pytest.mark.parametrize("dtype,B,d,C,r,margin,m,master", [
    ("f32", 64, 128, 10000, 0.1, "cosface", 0.4, False),
    ("bf16", 200, 256, 30000, 0.1, "arcface", 0.5, True),
    ("f16", 300, 512, 40000, 0.2, "arcface", 0.5, False),
])
def test_tiered_equals_resident(dev, dtype, B, d, C, r, margin, m, master, n_slots):
    from paper_2010_05222_amd.head import PfcShard, TieredShard
    T = 6
    print(f"\ntiered dtype={dtype} B={B} d={d} C={C} r={r} master={master} slots={n_slots}",
          flush=True)
    W, M, Xs, Ls = _inputs(B, d, C, dtype, T, 21, dev, span=C // 8)
    seeds = [100 + t for t in range(T)]
    kw = dict(dtype=dtype, s=64.0, m=m, margin=margin, lr=0.1, mu=0.9, device=dev)

    Wd = torch.from_numpy(W).to(TDT[dtype]).to(dev)
    Md = torch.from_numpy(M).to(dev)
    Pd = torch.from_numpy(W).to(dev) if master else None
    res = PfcShard(B, d, C, r, **kw)
    ts = TieredShard(B, d, C, r, master=master, n_slots=n_slots, **kw)
    ts.W_bank.copy_(Wd.cpu())
    ts.M_bank.copy_(Md.cpu())
    if master:
        ts.P_bank.copy_(Pd.cpu())

    ts.begin(Ls[0], seeds[0])
    shared = []
    prev = None
    for t in range(T):
        res.step(Xs[t], Ls[t], Wd, Md, seeds[t], W_master=Pd)
        nxt = Ls[t + 1] if t + 1 < T else None
        out = ts.step(Xs[t], nxt, seeds[t + 1] if nxt is not None else None)
        torch.cuda.synchronize()
        K = int(res.n_active.item())
        assert int(out.n_active.item()) == K
        act = out.active[:K].cpu().numpy()
        assert np.array_equal(act, res.active[:K].cpu().numpy())
        assert torch.equal(out.labels_mapped, res.labels_mapped)
        assert torch.equal(out.loss, res.loss), (t, out.loss.item(), res.loss.item())
        assert torch.equal(out.row_lse, res.row_lse)
        assert torch.equal(out.dX, res.dX)
        if prev is not None:
            shared.append(len(np.intersect1d(prev, act)))
        prev = act
    assert ts.stale_rows() == 0
    torch.cuda.synchronize()
    print("rows shared by consecutive steps:", shared, flush=True)
    assert min(shared) > 0
    assert torch.equal(ts.W_bank, Wd.cpu())
    assert torch.equal(ts.M_bank, Md.cpu())
    if master:
        assert torch.equal(ts.P_bank, Pd.cpu())


@pytest.mark.parametrize("case", ["pfc_star", "offset_unowned"])
def test_tiered_filter_and_offset(dev, case):
    """The PFC* filter (tau = 0.3) and a shard at class offset 5,000 whose
    batch also holds labels of other shards, tiered against resident."""
    from paper_2010_05222_amd.head import PfcShard, TieredShard
    B, d, C, r, T, dtype = 160, 256, 12000, 0.1, 5, "bf16"
    a = 5000 if case == "offset_unowned" else 0
    tau = 0.3 if case == "pfc_star" else None
    rng = np.random.default_rng(24)
    W = (0.01 * rng.standard_normal((C, d))).astype(np.float32)
    M = (1e-3 * rng.standard_normal((C, d))).astype(np.float32)
    Xs, Ls = [], []
    for t in range(T):
        X = rng.standard_normal((B, d)).astype(np.float32)
        lo, hi = (a - 2000, a + C // 6) if case == "offset_unowned" else (0, C // 6)
        L = rng.integers(lo, hi, size=B).astype(np.int64)
        if case == "pfc_star":
            # Rows near a centre of another row's class: negatives above tau.
            for n in range(0, B, 4):
                k = int(L[(n + 1) % B])
                if k != L[n]:
                    X[n] = (W[k] / np.linalg.norm(W[k]) * np.sqrt(d)
                            + 0.5 * rng.standard_normal(d)).astype(np.float32)
        Xs.append(torch.from_numpy(X).to(torch.bfloat16).to(dev))
        Ls.append(torch.from_numpy(L).to(dev))
    kw = dict(dtype=dtype, class_offset=a, s=64.0, m=0.5, margin="arcface", lr=0.1, mu=0.9,
              device=dev, tau=tau)
    Wd = torch.from_numpy(W).to(torch.bfloat16).to(dev)
    Md = torch.from_numpy(M).to(dev)
    res = PfcShard(B, d, C, r, **kw)
    ts = TieredShard(B, d, C, r, **kw)
    ts.W_bank.copy_(Wd.cpu())
    ts.M_bank.copy_(Md.cpu())
    ts.begin(Ls[0], 0)
    for t in range(T):
        res.step(Xs[t], Ls[t], Wd, Md, t)
        out = ts.step(Xs[t], Ls[t + 1] if t + 1 < T else None, t + 1)
        torch.cuda.synchronize()
        assert torch.equal(out.labels_mapped, res.labels_mapped)
        assert torch.equal(out.loss, res.loss), (t, out.loss.item(), res.loss.item())
        assert torch.equal(out.dX, res.dX)
        if case == "offset_unowned":
            assert int((out.labels_mapped < 0).sum().item()) > 0
    assert ts.stale_rows() == 0
    torch.cuda.synchronize()
    assert torch.equal(ts.W_bank, Wd.cpu())
    assert torch.equal(ts.M_bank, Md.cpu())


def test_tiered_fp32_matches_oracle_over_steps(dev):
    """Three fp32 steps on the bank against the oracle's three lazy steps."""
    from paper_2010_05222_amd.head import TieredShard
    B, d, C, r, T = 64, 128, 10000, 0.1, 3
    W, M, Xs, Ls = _inputs(B, d, C, "f32", T, 22, dev, span=C // 10)
    ts = TieredShard(B, d, C, r, dtype="f32", s=64.0, m=0.4, margin="cosface", lr=0.1, mu=0.9,
                     device=dev)
    ts.W_bank.copy_(torch.from_numpy(W))
    ts.M_bank.copy_(torch.from_numpy(M))
    W64, M64 = W.astype(np.float64), M.astype(np.float64)
    ts.begin(Ls[0], 0)
    for t in range(T):
        out = ts.step(Xs[t], Ls[t + 1] if t + 1 < T else None, t + 1)
        loss = float(out.loss.item())
        ref = O.step(Xs[t].double().cpu().numpy(), W64, M64, Ls[t].cpu().numpy(), C, 0, r, t,
                     64.0, 0.4, "cosface", 0.1, 0.9, "f32")
        assert abs(loss - ref["loss"]) <= 1e-3 * abs(ref["loss"]), (t, loss, ref["loss"])
    assert ts.stale_rows() == 0
    Mb = ts.M_bank.double().numpy()
    Wb = ts.W_bank.double().numpy()
    err_m = float(np.max(np.abs(Mb - M64)))
    err_w = float(np.max(np.abs(Wb - W64)))
    print(f"\nfp32 bank after {T} steps: M max-abs {err_m:.3g}, W max-abs {err_w:.3g}", flush=True)
    assert err_m <= 1e-5 and err_w <= 1e-5
    # Rows never active are untouched.
    touched = np.zeros(C, dtype=bool)
    for t in range(T):
        touched[O.sample_active(Ls[t].cpu().numpy(), C, 0, r, t)[0]] = True
    assert np.array_equal(Wb[~touched], W.astype(np.float64)[~touched])
    assert np.array_equal(Mb[~touched], M.astype(np.float64)[~touched])


@pytest.mark.parametrize("n_slots", [2, 3])
def test_versions_and_stale_rows(dev, n_slots):
    from paper_2010_05222_amd.head import TieredShard
    B, d, C, r, T = 128, 128, 20000, 0.1, 4
    W, M, Xs, Ls = _inputs(B, d, C, "bf16", T, 23, dev, span=C // 8)
    ts = TieredShard(B, d, C, r, dtype="bf16", device=dev, n_slots=n_slots)
    ts.W_bank.copy_(torch.from_numpy(W).to(torch.bfloat16))
    ts.M_bank.copy_(torch.from_numpy(M))
    ts.begin(Ls[0], 0)
    sets = []
    for t in range(T):
        out = ts.step(Xs[t], Ls[t + 1] if t + 1 < T else None, t + 1)
        sets.append(out.active[:int(out.n_active.item())].cpu().numpy())
    assert ts.stale_rows() == 0
    expect = np.zeros(C, dtype=np.int32)
    for t, s in enumerate(sets):
        expect[s] = t + 1
    assert np.array_equal(ts.bank_version.numpy(), expect)
    assert np.array_equal(ts.row_version.cpu().numpy(), expect)

    # A row staged while its update is unwritten: raise every row's staged
    # version before step 1's staging of step 2, so that each cold row of
    # S(2) (in no set still held in a slot) finds an older version in the bank.
    ts2 = TieredShard(B, d, C, r, dtype="bf16", device=dev, n_slots=n_slots)
    ts2.W_bank.copy_(torch.from_numpy(W).to(torch.bfloat16))
    ts2.M_bank.copy_(torch.from_numpy(M))
    ts2.begin(Ls[0], 0)
    p0 = ts2.parts[0]
    a0 = None
    ts2.step(Xs[0], Ls[1], 1)
    torch.cuda.synchronize()        # step 1's staging is done before the versions move
    a0 = p0.active[:int(p0.n_active.item())].cpu().numpy()
    ts2.row_version += 1000
    p1, p2 = ts2.parts[1], ts2.parts[2 % n_slots]
    ts2.step(Xs[1], Ls[2], 2)
    torch.cuda.synchronize()
    a1 = p1.active[:int(p1.n_active.item())].cpu().numpy()
    a2 = p2.active[:int(p2.n_active.item())].cpu().numpy()
    ts2.step(Xs[2], None, None)
    n_stale = ts2.stale_rows()
    held = a1 if n_slots == 2 else np.union1d(a1, a0)
    assert n_stale == len(np.setdiff1d(a2, held)) > 0


def test_bank_rejects_pageable_memory(dev):
    from paper_2010_05222_amd import pfc
    cap, d = 64, 128
    pageable = torch.zeros((1000, d), dtype=torch.float32)     # not pinned
    slot = torch.zeros((cap, d), dtype=torch.float32, device=dev)
    ids = torch.arange(cap, dtype=torch.int32, device=dev)
    n = torch.full((1,), cap, dtype=torch.int32, device=dev)
    with pytest.raises(pfc.PfcError) as e:
        pfc.pfc_bank_stage([pageable.data_ptr()], [slot.data_ptr()], [d * 4], 1000,
                           ids.data_ptr(), n.data_ptr(), 0, 0, 0, 0, cap, 0, 0, 1, 0, 0)
    assert e.value.status == pfc.PFC_ERR_INVALID_ARG
    with pytest.raises(pfc.PfcError) as e:
        pfc.pfc_bank_writeback([slot.data_ptr()], [pageable.data_ptr()], [d * 4],
                               ids.data_ptr(), n.data_ptr(), 0, 0, cap, 1000, 0, 1, 0)
    assert e.value.status == pfc.PFC_ERR_INVALID_ARG
    torch.cuda.synchronize()


def test_tiered_full_size_equals_resident(dev):
    """The massive workload (C = 8M, |S| = 800,000, fp16 W, fp32 momentum) with
    its bank in pinned host memory, three steps, against the same steps on the
    resident shard: every step's loss, row_lse and dX bit for bit, and sampled
    bank rows (touched and untouched) against the resident shard afterwards."""
    import workloads
    from paper_2010_05222_amd.head import PfcShard, TieredShard
    cfg = workloads.config("massive")
    B, d, C, r, T = cfg["B"], cfg["d"], cfg["C"], cfg["r"], 3
    tdt = torch.float16
    kw = dict(dtype=cfg["dtype"], class_offset=cfg["a"], s=cfg["s"], m=cfg["m"],
              margin=cfg["margin"], lr=cfg["lr"], mu=cfg["mu"], device=dev)
    print(f"\ntiered full size: B={B} d={d} C={C} r={r}", flush=True)
    W, _ = workloads.make_weights_device(cfg, dev)
    M = torch.zeros((C, d), dtype=torch.float32, device=dev)
    ts = TieredShard(B, d, C, r, **kw)
    ts.W_bank.copy_(W)
    res = PfcShard(B, d, C, r, **kw)
    batches = []
    for t in range(T):
        X, L = workloads.make_batch(cfg, t)
        batches.append((torch.from_numpy(X).to(tdt).to(dev), torch.from_numpy(L).to(dev)))
    torch.cuda.synchronize()
    print("inputs ready", flush=True)
    ts.begin(batches[0][1], 0)
    touched = torch.zeros(C, dtype=torch.bool, device=dev)
    for t in range(T):
        out = ts.step(batches[t][0], batches[t + 1][1] if t + 1 < T else None, t + 1)
        res.step(batches[t][0], batches[t][1], W, M, t)
        torch.cuda.synchronize()
        K = int(res.n_active.item())
        assert int(out.n_active.item()) == K
        assert torch.equal(out.active[:K], res.active[:K])
        assert torch.equal(out.loss, res.loss), (t, out.loss.item(), res.loss.item())
        assert torch.equal(out.row_lse, res.row_lse)
        assert torch.equal(out.dX, res.dX)
        touched[res.active[:K].long()] = True
        print(f"step {t}: |S|={K} loss={out.loss.item():.4f} equal", flush=True)
    assert ts.stale_rows() == 0
    torch.cuda.synchronize()
    rng = np.random.default_rng(5)
    t_ids = torch.nonzero(touched).flatten().cpu().numpy()
    u_ids = torch.nonzero(~touched).flatten().cpu().numpy()
    pick = np.concatenate([rng.choice(t_ids, 20000, replace=False),
                           rng.choice(u_ids, 5000, replace=False)])
    pick_t = torch.from_numpy(pick)
    assert torch.equal(ts.W_bank[pick_t], W[pick_t.to(dev)].cpu())
    assert torch.equal(ts.M_bank[pick_t], M[pick_t.to(dev)].cpu())
    print(f"bank rows equal: {len(pick)} sampled of {len(t_ids)} touched", flush=True)
