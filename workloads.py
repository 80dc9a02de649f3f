"""Seeded synthetic workloads shaped like the paper's face-recognition heads.

This module only draws random inputs; it holds none of the method's
arithmetic.  Both the CPU oracle's tests and the HIP path's tests and benchmark
take their inputs from here, so both sides see identical data.

Stand-in for the paper's datasets (MS1MV2, Glint360K, WebFace, ...), which are
not available: embeddings are i.i.d. N(0, 1) rows (a backbone's output before
normalisation), class centres are i.i.d. N(0, 0.01^2) (a fresh classifier),
labels are uniform over the shard or, for the long-tail case, a truncated
Zipf(1.1) law over a fixed random permutation of the class ids (the paper's
long-tailed WebFace setting, Sec. 4.4).  Hyper-parameters follow Sec. 4.1:
s = 64, CosFace m = 0.4, ArcFace m = 0.5, learning rate 0.1, momentum 0.9.
"""

import numpy as np

# name -> workload.  C is the shard size, a its first global class id.
CONFIGS = {
    # Parity-scale case: everything in fp32.
    "tiny": dict(B=64, d=128, C=10_000, a=0, r=0.1, dtype="f32", master=False,
                 margin="cosface", s=64.0, m=0.4, lr=0.1, mu=0.9,
                 labels="uniform", data_seed=0),
    # r = 1: the sampled head is the full softmax over one million classes.
    "full_softmax": dict(B=512, d=512, C=1_000_000, a=0, r=1.0, dtype="bf16",
                         master=False, margin="arcface", s=64.0, m=0.5, lr=0.1,
                         mu=0.9, labels="uniform", data_seed=2),
    # One shard of a class-sharded head, bf16 with an fp32 master copy.
    "one_shard": dict(B=1024, d=512, C=1_000_000, a=0, r=0.1, dtype="bf16",
                      master=True, margin="arcface", s=64.0, m=0.5, lr=0.1,
                      mu=0.9, labels="uniform", data_seed=3),
    # Long-tailed labels: heavily duplicated positives.
    "zipf": dict(B=1024, d=512, C=2_000_000, a=0, r=0.2, dtype="bf16",
                 master=False, margin="cosface", s=64.0, m=0.4, lr=0.1, mu=0.9,
                 labels="zipf", data_seed=4),
    # One GPU's share of a 64M-class head (8 shards of 8M), fp16 weights.
    "massive": dict(B=1024, d=512, C=8_000_000, a=0, r=0.1, dtype="f16",
                    master=False, margin="arcface", s=64.0, m=0.5, lr=0.1,
                    mu=0.9, labels="uniform", data_seed=5),
}

ZIPF_ALPHA = 1.1
W_STD = 0.01
MOMENTUM_STD = 1e-3


def config(name, **overrides):
    cfg = dict(CONFIGS[name])
    cfg.update(overrides)
    cfg["name"] = name
    return cfg


def _zipf_labels(rng, B, C, a, perm_seed):
    ranks = np.arange(1, C + 1, dtype=np.float64)
    w = ranks ** (-ZIPF_ALPHA)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    u = rng.random(B)
    rank0 = np.minimum(np.searchsorted(cdf, u, side="right"), C - 1)
    perm = np.random.default_rng([perm_seed, 2**31 - 1]).permutation(C)
    return perm[rank0].astype(np.int64) + a


def make_batch(cfg, step=0):
    """Embeddings X (float32 [B, d]) and global labels (int64 [B]) of one step."""
    rng = np.random.default_rng([cfg["data_seed"], step])
    B, d, C, a = cfg["B"], cfg["d"], cfg["C"], cfg["a"]
    X = rng.standard_normal((B, d)).astype(np.float32)
    if cfg["labels"] == "zipf":
        labels = _zipf_labels(rng, B, C, a, cfg["data_seed"])
    elif cfg["labels"] == "uniform":
        labels = rng.integers(a, a + C, size=B, dtype=np.int64)
    else:
        raise ValueError(cfg["labels"])
    return X, labels


def make_weights_host(cfg, seed=None):
    """Class centres W (float32 [C, d]) drawn on the host (small shards)."""
    seed = cfg["data_seed"] if seed is None else seed
    rng = np.random.default_rng([seed, 2**31 - 2])
    return (W_STD * rng.standard_normal((cfg["C"], cfg["d"]))).astype(np.float32)


def make_momentum_host(cfg, random=False, seed=None):
    if not random:
        return np.zeros((cfg["C"], cfg["d"]), dtype=np.float32)
    seed = cfg["data_seed"] if seed is None else seed
    rng = np.random.default_rng([seed, 2**31 - 3])
    return (MOMENTUM_STD * rng.standard_normal((cfg["C"], cfg["d"]))).astype(np.float32)


def make_weights_device(cfg, device, seed=None, chunk_rows=1 << 20):
    """Class centres drawn on the device with torch's generator (large shards).

    Returns the fp32 draw rounded to the storage type, plus the fp32 draw
    itself when the workload keeps an fp32 master copy (else None).
    """
    import torch
    seed = cfg["data_seed"] if seed is None else seed
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[cfg["dtype"]]
    C, d = cfg["C"], cfg["d"]
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    W = torch.empty((C, d), dtype=tdt, device=device)
    master = torch.empty((C, d), dtype=torch.float32, device=device) if cfg["master"] else None
    for r0 in range(0, C, chunk_rows):
        r1 = min(C, r0 + chunk_rows)
        draw = torch.randn((r1 - r0, d), generator=gen, device=device,
                           dtype=torch.float32) * W_STD
        W[r0:r1] = draw.to(tdt)
        if master is not None:
            master[r0:r1] = draw
    return W, master
