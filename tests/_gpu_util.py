"""Shared helpers of the GPU parity tests: run one head step through the C ABI
and compare it with the CPU oracle on the same seeded inputs."""

import numpy as np
import torch

from oracle import pfc_oracle as O

TDT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}

# Tolerances.  Stated bar: loss rel <= 1e-3; dX and dW max-abs <= 2e-2 for the
# 16-bit paths and <= 1e-5 for fp32.  The tighter relative bounds below are
# derived from the arithmetic of the kernels:
#  16-bit paths - the logit store keeps E = 2^(f - m) in fp16 (<= 2^-11
#   relative, so each p = E * scale is off by <= 0.05 %); softmax coefficients
#   rounded to bf16 for the backward contractions (<= 2^-9 relative); fp16
#   inputs rounded to bf16 on their way into the backward contractions
#   (<= 2^-9); fp32 accumulation.  Row-wise relative L2 error of dX and of each
#   class gradient stays well below 1e-2.
#  fp32 path - fp32 products and accumulation over d and |S| (<= 1e-6
#   relative per term): row-wise relative L2 error below 1e-4.
REL_ROW = {"f32": 1e-4, "bf16": 1e-2, "f16": 1e-2}
MAX_ABS = {"f32": 1e-5, "bf16": 2e-2, "f16": 2e-2}


def row_rel_err(got, ref):
    num = np.linalg.norm(got - ref, axis=1)
    den = np.maximum(np.linalg.norm(ref, axis=1), 1e-30)
    return num / den


def make_problem(B, d, C, dtype, seed, class_offset=0, label_span=None, random_m=True,
                 master=False, labels=None, device="cuda:0", conflicts=0):
    """Seeded Gaussian problem.  conflicts > 0: every conflicts-th row is
    placed near the centre of the next row's class (a duplicated identity:
    cosine ~0.9 to a negative that is always active, being a positive of the
    batch), the input of the PFC* conflict-filter tests."""
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((B, d)).astype(np.float32)
    W = (0.01 * rng.standard_normal((C, d))).astype(np.float32)
    if labels is None:
        lo, hi = (class_offset, class_offset + C) if label_span is None else label_span
        labels = rng.integers(lo, hi, size=B)
    if conflicts:
        for n in range(0, B, conflicts):
            k = int(labels[(n + 1) % B]) - class_offset
            if 0 <= k < C and labels[(n + 1) % B] != labels[n]:
                w = W[k].astype(np.float64)
                X[n] = (w / np.linalg.norm(w) * np.sqrt(d)
                        + 0.5 * rng.standard_normal(d)).astype(np.float32)
    M = (1e-3 * rng.standard_normal((C, d))).astype(np.float32) if random_m else \
        np.zeros((C, d), dtype=np.float32)
    dev = torch.device(device)
    t = TDT[dtype]
    Xd = torch.from_numpy(X).to(t).to(dev)
    Wd = torch.from_numpy(W).to(t).to(dev)
    Md = torch.from_numpy(M).to(dev)
    Pd = torch.from_numpy(W).to(dev) if master else None
    Ld = torch.from_numpy(np.asarray(labels, dtype=np.int64)).to(dev)
    return Xd, Wd, Md, Pd, Ld


def run_and_compare(shard, Xd, Wd, Md, Pd, Ld, seed, margin_name, check_sampler_only=False,
                    abs_scaled=False, degenerate=False):
    """One step on the GPU and the oracle on the same (rounded) inputs.

    Returns a dict of the error figures; asserts the stated bar and the
    derived bounds.  The max-abs gradient bar is the stated one unless
    `abs_scaled`, which multiplies it by max(1, max |ref|) for a case whose
    gradients are far larger than any workload's (see the single-row test).
    `degenerate`: a case whose references are exactly zero (a one-class
    shard: owned rows have loss 0 and no gradient), where a relative error
    has no meaning: the loss is compared with an absolute bar of 1e-3 when
    |loss| < 1, and dX rows whose reference is zero only with the max-abs
    bar."""
    dt = shard.dtype_name
    X64 = Xd.double().cpu().numpy()
    W0 = Wd.double().cpu().numpy()
    M0 = Md.double().cpu().numpy()
    P0 = Pd.double().cpu().numpy() if Pd is not None else None
    labels = Ld.cpu().numpy()
    Wd0, Md0 = Wd.clone(), Md.clone()

    shard.sample(Ld, seed)
    if not check_sampler_only:
        shard.forward(Xd, Wd)
        shard.backward(Xd, Wd, Md, Pd)
    torch.cuda.synchronize()

    active_ref, mapped_ref, info = O.sample_active(labels, shard.C, shard.class_offset, shard.r,
                                                   seed)
    K = int(shard.n_active.item())
    assert K == len(active_ref), (K, len(active_ref))
    assert np.array_equal(shard.active[:K].cpu().numpy(), active_ref)
    assert np.array_equal(shard.labels_mapped.cpu().numpy(), mapped_ref)
    out = {"K": K, "n_pos": info["n_pos"]}
    if check_sampler_only:
        return out

    B = shard.B
    Ws = W0[active_ref]
    tau = shard.tau
    fw = O.forward(X64, Ws, mapped_ref, shard.s, shard.m, margin_name, tau)
    if tau is not None and tau < 1.0:
        # The filter is a decision on a cosine: the GPU takes it in fp32, the
        # oracle in fp64.  The inputs keep every cosine well away from tau.
        out["n_filtered"] = int(np.sum(~O.conflict_mask(fw["cos"], mapped_ref, tau)))
        assert np.min(np.abs(fw["cos"] - tau)) > 1e-3
    loss_ref = O.batch_loss(fw["row_loss"], B)
    dx_ref = O.grad_x(X64, Ws, mapped_ref, fw["lse"], B, shard.s, shard.m, margin_name, tau)
    g_ref = O.grad_w(X64, Ws, np.arange(K), mapped_ref, fw["lse"], B, shard.s, shard.m,
                     margin_name, tau)

    loss = float(shard.loss.item())
    lse = shard.row_lse.cpu().numpy().astype(np.float64)
    dx = shard.dX.cpu().numpy().astype(np.float64)
    M1 = Md.double().cpu().numpy()
    W1 = Wd.double().cpu().numpy()
    # Class gradients through the momentum rows: M1 = fp32(mu * M0 + g).
    mom_ref = shard.mu * M0[active_ref]
    g_gpu = M1[active_ref] - mom_ref

    out["loss_rel"] = abs(loss - loss_ref) / max(abs(loss_ref), 1.0 if degenerate else 1e-30)
    # A row with an empty denominator has lse = -inf on both sides.
    empty = np.isneginf(fw["lse"])
    assert np.array_equal(np.isneginf(lse), empty), (np.nonzero(np.isneginf(lse))[0],
                                                     np.nonzero(empty)[0])
    out["n_empty_rows"] = int(np.sum(empty))
    out["lse_abs"] = float(np.max(np.abs(lse[~empty] - fw["lse"][~empty]), initial=0.0))
    out["dx_abs"] = float(np.max(np.abs(dx - dx_ref)))
    rows = np.linalg.norm(dx_ref, axis=1) > 0 if degenerate else np.ones(len(dx_ref), bool)
    out["dx_row_rel"] = float(np.max(row_rel_err(dx[rows], dx_ref[rows]), initial=0.0))
    out["g_abs"] = float(np.max(np.abs(g_gpu - g_ref)))
    # Row-wise relative error of g, allowing the fp32 rounding of the momentum sum.
    num = np.linalg.norm(g_gpu - g_ref, axis=1)
    slack = 2.0 ** -22 * np.linalg.norm(M1[active_ref], axis=1)
    den = np.linalg.norm(g_ref, axis=1)
    nz = den > 0
    out["g_row_rel"] = float(np.max(np.maximum(num[nz] - slack[nz], 0) / den[nz])) if nz.any() else 0.0

    assert out["loss_rel"] <= 1e-3, out
    assert out["lse_abs"] <= (1e-4 if dt == "f32" else 5e-3), out
    bar_dx = MAX_ABS[dt] * (max(1.0, np.max(np.abs(dx_ref))) if abs_scaled else 1.0)
    bar_g = MAX_ABS[dt] * (max(1.0, np.max(np.abs(g_ref))) if abs_scaled else 1.0)
    assert out["dx_abs"] <= bar_dx, out
    assert out["g_abs"] <= bar_g, out
    assert out["dx_row_rel"] <= REL_ROW[dt], out
    assert out["g_row_rel"] <= REL_ROW[dt], out

    # W of the active rows: the GPU's fp32 step from its own M, rounded to the
    # storage type.  Allowed: one unit in the last place of the stored result
    # plus the fp32 rounding of the step (which may be fused).
    step = shard.lr * M1[active_ref]
    if Pd is not None:
        P1 = Pd.double().cpu().numpy()
        exp_p = P0[active_ref] - step
        tol = 2.0 ** -22 * (np.abs(P0[active_ref]) + np.abs(step))
        out["master_err_ulps"] = float(np.max(np.abs(P1[active_ref] - exp_p) / tol))
        assert out["master_err_ulps"] <= 1.0, out
        assert np.array_equal(W1[active_ref], O.round_to(P1[active_ref], dt))
    else:
        exact = W0[active_ref] - step
        exp_w = O.round_to(exact, dt)
        ulp = {"f32": 2.0 ** -23, "bf16": 2.0 ** -7, "f16": 2.0 ** -10}[dt]
        tol = ulp * np.abs(exp_w) + 2.0 ** -22 * (np.abs(W0[active_ref]) + np.abs(step))
        if dt == "f16":
            tol = np.maximum(tol, 2.0 ** -24)            # fp16 subnormal spacing
        out["w_err_tol"] = float(np.max(np.abs(W1[active_ref] - exp_w) / tol))
        assert out["w_err_tol"] <= 1.0, out

    # Rows outside S: bit-identical weights, momentum and master.
    mask = torch.ones(shard.C, dtype=torch.bool, device=Wd.device)
    mask[torch.from_numpy(active_ref.astype(np.int64)).to(Wd.device)] = False
    assert torch.equal(Wd[mask], Wd0[mask])
    assert torch.equal(Md[mask], Md0[mask])
    return out
