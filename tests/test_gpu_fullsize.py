"""GPU parity at the benchmark's full sizes and launch configuration.

One head step of a full-size workload, run exactly as bench.py runs it
(PfcShard on the device, weights drawn on the device, momentum from zero),
checked against the CPU oracle on what the oracle can afford at this size:

  - the active set and remapped labels, bit for bit;
  - row_lse of every row and the batch loss (the oracle's forward over all
    rows and all |S| active classes, in row blocks: rows are independent);
  - dX on a seeded sample of rows;
  - the class gradients (through the momentum rows, M starts at zero so
    M[S_j] = g_j) and the updated weights on a seeded sample of active
    classes together with every positive class of the batch;
  - every row outside S: weights and momentum untouched (checked on the GPU
    over the whole shard).
"""

import numpy as np
import pytest
import torch

import workloads
from oracle import pfc_oracle as O

pytestmark = pytest.mark.gpu

N_ROWS_DX = 32        # sampled batch rows for dX
N_CLASSES_G = 4096    # sampled active classes for the class gradients / update
ROW_BLOCK = 256       # rows per oracle forward call


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2010_05222_amd import pfc  # noqa: F401  (fails loudly if libpfc.so is missing)
    return torch.device("cuda:0")


@pytest.mark.parametrize("name", ["massive", "one_shard", "zipf", "full_softmax"])
def test_full_size_step(dev, name):
    from _gpu_util import MAX_ABS, REL_ROW, row_rel_err
    from paper_2010_05222_amd.head import PfcShard

    cfg = workloads.config(name)
    B, d, C, dt = cfg["B"], cfg["d"], cfg["C"], cfg["dtype"]
    print(f"\nfull-size step {name}: B={B} d={d} C={C} r={cfg['r']} {dt} "
          f"master={cfg['master']} {cfg['margin']}", flush=True)
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dt]
    W, master = workloads.make_weights_device(cfg, dev)
    M = torch.zeros((C, d), dtype=torch.float32, device=dev)
    X, labels = workloads.make_batch(cfg, 0)
    Xd = torch.from_numpy(X).to(tdt).to(dev)
    Ld = torch.from_numpy(labels).to(dev)
    W0 = W.clone()
    P0 = master.clone() if master is not None else None
    shard = PfcShard(B, d, C, cfg["r"], dtype=dt, class_offset=cfg["a"], s=cfg["s"], m=cfg["m"],
                     margin=cfg["margin"], lr=cfg["lr"], mu=cfg["mu"], device=dev)
    seed = 0
    shard.step(Xd, Ld, W, M, seed, master)
    torch.cuda.synchronize()
    print("step done", flush=True)

    # Sampler: bit-exact.
    active_ref, mapped_ref, _ = O.sample_active(labels, C, cfg["a"], cfg["r"], seed)
    K = int(shard.n_active.item())
    assert K == len(active_ref)
    assert np.array_equal(shard.active[:K].cpu().numpy(), active_ref)
    assert np.array_equal(shard.labels_mapped.cpu().numpy(), mapped_ref)

    # Rows outside S: untouched weights, momentum (and master).
    act_d = torch.from_numpy(active_ref.astype(np.int64)).to(dev)
    in_s = torch.zeros(C, dtype=torch.bool, device=dev)
    in_s[act_d] = True
    assert not bool(((W != W0).any(dim=1) & ~in_s).any())
    assert not bool(((M != 0).any(dim=1) & ~in_s).any())
    if master is not None:
        assert not bool(((master != P0).any(dim=1) & ~in_s).any())
    print("untouched rows ok", flush=True)

    # Oracle forward over all rows and all active classes, in row blocks.
    X64 = Xd.double().cpu().numpy()
    Ws = W0[act_d].double().cpu().numpy()
    lse_ref = np.empty(B)
    row_loss = np.empty(B)
    for r0 in range(0, B, ROW_BLOCK):
        fw = O.forward(X64[r0:r0 + ROW_BLOCK], Ws, mapped_ref[r0:r0 + ROW_BLOCK], cfg["s"],
                       cfg["m"], cfg["margin"])
        lse_ref[r0:r0 + ROW_BLOCK] = fw["lse"]
        row_loss[r0:r0 + ROW_BLOCK] = fw["row_loss"]
        del fw
    loss_ref = O.batch_loss(row_loss, B)
    print("oracle forward done", flush=True)

    loss = float(shard.loss.item())
    lse = shard.row_lse.cpu().numpy().astype(np.float64)
    out = {"K": K, "loss_rel": abs(loss - loss_ref) / abs(loss_ref),
           "lse_abs": float(np.max(np.abs(lse - lse_ref)))}
    assert out["loss_rel"] <= 1e-3, out
    assert out["lse_abs"] <= 5e-3, out

    # dX on sampled rows.
    rng = np.random.default_rng([cfg["data_seed"], 7])
    rows = np.sort(rng.choice(B, size=min(N_ROWS_DX, B), replace=False))
    dx_ref = O.grad_x(X64[rows], Ws, mapped_ref[rows], lse_ref[rows], B, cfg["s"], cfg["m"],
                      cfg["margin"])
    dx = shard.dX[torch.from_numpy(rows).to(dev)].double().cpu().numpy()
    out["dx_abs"] = float(np.max(np.abs(dx - dx_ref)))
    out["dx_row_rel"] = float(np.max(row_rel_err(dx, dx_ref)))
    assert out["dx_abs"] <= MAX_ABS[dt], out
    assert out["dx_row_rel"] <= REL_ROW[dt], out

    # Class gradients and the update on sampled active classes, plus every
    # positive class: only those carry the exact target term and the dW
    # kernel's target-row lists.  The Zipf workload's most duplicated classes
    # (the top one is the label of ~12 % of the rows) are among them.
    pos, counts = np.unique(mapped_ref[mapped_ref >= 0], return_counts=True)
    out["n_positive_cols"] = int(len(pos))
    out["max_rows_per_class"] = int(counts.max()) if counts.size else 0
    cols = np.union1d(rng.choice(K, size=min(N_CLASSES_G, K), replace=False), pos)
    g_ref = O.grad_w(X64, Ws[cols], cols, mapped_ref, lse_ref, B, cfg["s"], cfg["m"],
                     cfg["margin"])
    rows_g = torch.from_numpy(active_ref[cols].astype(np.int64)).to(dev)
    g_gpu = M[rows_g].double().cpu().numpy()          # M0 = 0: M1 = fp32(g)
    out["g_abs"] = float(np.max(np.abs(g_gpu - g_ref)))
    out["g_row_rel"] = float(np.max(row_rel_err(g_gpu, g_ref)))
    assert out["g_abs"] <= MAX_ABS[dt], out
    assert out["g_row_rel"] <= REL_ROW[dt], out

    step = cfg["lr"] * g_gpu
    W1 = W[rows_g].double().cpu().numpy()
    if master is not None:
        p0 = P0[rows_g].double().cpu().numpy()
        p1 = master[rows_g].double().cpu().numpy()
        tol = 2.0 ** -22 * (np.abs(p0) + np.abs(step))
        out["master_err_ulps"] = float(np.max(np.abs(p1 - (p0 - step)) / tol))
        assert out["master_err_ulps"] <= 1.0, out
        assert np.array_equal(W1, O.round_to(p1, dt))
    else:
        w0 = W0[rows_g].double().cpu().numpy()
        exp_w = O.round_to(w0 - step, dt)
        ulp = {"f32": 2.0 ** -23, "bf16": 2.0 ** -7, "f16": 2.0 ** -10}[dt]
        tol = ulp * np.abs(exp_w) + 2.0 ** -22 * (np.abs(w0) + np.abs(step))
        if dt == "f16":
            tol = np.maximum(tol, 2.0 ** -24)
        out["w_err_tol"] = float(np.max(np.abs(W1 - exp_w) / tol))
        assert out["w_err_tol"] <= 1.0, out
    print(out, flush=True)
