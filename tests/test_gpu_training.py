"""Training through the library learns: steps on one fixed batch move the
class centres of its labels toward their rows (Eq. pfc_center_update), so the
loss falls well below its starting value, with the negatives redrawn every
step (Sec. 3.3.1).  A functional check beside the per-step parity tests."""

import numpy as np
import pytest
import torch

from paper_2010_05222_amd.head import PfcShard


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_training_reduces_loss(dtype):
    dev = torch.device("cuda:0")
    B, d, C, r, steps = 64, 128, 2000, 0.2, 40
    print(f"\ntraining: {steps} steps of one batch, B={B} d={d} C={C} r={r} {dtype}", flush=True)
    rng = np.random.default_rng(30)
    t = {"bf16": torch.bfloat16, "f16": torch.float16}[dtype]
    X = torch.from_numpy(rng.standard_normal((B, d)).astype(np.float32)).to(t).to(dev)
    W = torch.from_numpy((0.01 * rng.standard_normal((C, d))).astype(np.float32)).to(t).to(dev)
    M = torch.zeros((C, d), dtype=torch.float32, device=dev)
    labels = torch.from_numpy(rng.integers(0, C, size=B)).to(dev)
    shard = PfcShard(B, d, C, r, dtype=dtype, s=64.0, m=0.4, margin="cosface", lr=0.1, mu=0.9,
                     device=dev)
    losses = []
    for step in range(steps):
        shard.step(X, labels, W, M, step)
        losses.append(float(shard.loss.item()))
    print("loss:", " ".join(f"{v:.3f}" for v in losses[::5]), f"... {losses[-1]:.3f}", flush=True)
    assert all(np.isfinite(losses))
    assert losses[-1] < 0.5 * losses[0], losses
