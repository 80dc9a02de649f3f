"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Integer outputs (active set, |S|, remapped labels) must match bit for bit;
floating point within the stated bar and the derived bounds of _gpu_util.
Sizes span several tiles of every kernel and leave ragged tails in the batch
and in |S|.
"""

import numpy as np
import pytest
import torch

import workloads
from oracle import pfc_oracle as O

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2010_05222_amd import pfc  # noqa: F401  (fails loudly if libpfc.so is missing)
    return torch.device("cuda:0")


def _shard(B, d, C, r, dtype, margin, m, class_offset=0, dev="cuda:0", tau=None):
    from paper_2010_05222_amd.head import PfcShard
    return PfcShard(B, d, C, r, dtype=dtype, class_offset=class_offset, s=64.0, m=m,
                    margin=margin, lr=0.1, mu=0.9, device=dev, tau=tau)


def _case(dev, B, d, C, r, dtype, margin, m, seed, class_offset=0, label_span=None,
          random_m=True, master=False, labels=None, tau=None, conflicts=0, abs_scaled=False,
          degenerate=False):
    from _gpu_util import make_problem, run_and_compare
    print(f"\ncase B={B} d={d} C={C} r={r} dtype={dtype} margin={margin} seed={seed} "
          f"offset={class_offset} master={master} tau={tau}", flush=True)
    Xd, Wd, Md, Pd, Ld = make_problem(B, d, C, dtype, seed, class_offset, label_span, random_m,
                                      master, labels, dev, conflicts)
    shard = _shard(B, d, C, r, dtype, margin, m, class_offset, dev, tau)
    out = run_and_compare(shard, Xd, Wd, Md, Pd, Ld, seed, margin, abs_scaled=abs_scaled,
                          degenerate=degenerate)
    print(out, flush=True)
    return out


def test_tiny_workload_fp32(dev):
    """The parity-scale workload (B=64, d=128, C=10,000, r=0.1, fp32, CosFace)."""
    cfg = workloads.config("tiny")
    from _gpu_util import run_and_compare
    X, labels = workloads.make_batch(cfg, 0)
    W = workloads.make_weights_host(cfg)
    Xd = torch.from_numpy(X).to(dev)
    Wd = torch.from_numpy(W).to(dev)
    Ld = torch.from_numpy(labels).to(dev)
    for random_m in (False, True):
        Md = torch.from_numpy(workloads.make_momentum_host(cfg, random=random_m)).to(dev)
        shard = _shard(cfg["B"], cfg["d"], cfg["C"], cfg["r"], "f32", cfg["margin"], cfg["m"],
                       dev=dev)
        out = run_and_compare(shard, Xd, Wd.clone(), Md, None, Ld, 0, cfg["margin"])
        assert out["K"] == 1000
        print(out, flush=True)


@pytest.mark.parametrize("margin,m", [("cosface", 0.4), ("arcface", 0.5)])
def test_bf16_ragged(dev, margin, m):
    # B not a multiple of any tile; |S| = 300 not a multiple of 32/64/128.
    _case(dev, 100, 128, 3000, 0.1, "bf16", margin, m, seed=1)


def test_bf16_master(dev):
    _case(dev, 96, 256, 4000, 0.2, "bf16", "arcface", 0.5, seed=2, master=True)


def test_f16_ragged(dev):
    _case(dev, 70, 256, 5000, 0.2, "f16", "arcface", 0.5, seed=3)


def test_bf16_d512_several_tiles(dev):
    _case(dev, 300, 512, 20000, 0.1, "bf16", "cosface", 0.4, seed=4, random_m=False)


def test_f16_d512_zero_momentum(dev):
    _case(dev, 260, 512, 12000, 0.1, "f16", "arcface", 0.5, seed=5, random_m=False)


def test_f16_d512_master(dev):
    # fp16 weights with an fp32 master at d = 512; |S| = 910, B ragged.
    _case(dev, 190, 512, 9100, 0.1, "f16", "cosface", 0.4, seed=18, master=True)


def test_f16_d128(dev):
    _case(dev, 150, 128, 4100, 0.1, "f16", "cosface", 0.4, seed=19)


@pytest.mark.parametrize("d", [8, 1000, 1024])
def test_f32_feature_widths(dev, d):
    # The fp32 path takes any d that is a multiple of 8 up to 1024: the
    # smallest, one that is not a multiple of 32 or 64, and the largest.
    # At d = 8 the class rows (std 0.01) have norm ~0.028, so 1/||w|| ~ 35
    # and the class gradients reach ~72, where one fp32 ulp is 7.6e-6: the
    # max-abs bar is applied relative to max |ref| there (as for B = 1);
    # the row-relative bound is unchanged.
    _case(dev, 40, d, 1500, 0.2, "f32", "arcface", 0.5, seed=27, abs_scaled=(d == 8))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_single_class_shard(dev, dtype):
    # The smallest shard: one class, taken at r = 1.  Rows labelled with it
    # have a one-term softmax (probability 1, loss 0, no gradient); the
    # others are unowned and their only logit gets the full gradient, so the
    # class gradient reaches ~30.  References that are exactly zero and that
    # magnitude take the degenerate-case and scaled bars.
    labels = np.array([0, 3, 0, 9, 0, 0, 5, 0, 2, 0, 0, 4])
    out = _case(dev, 12, 128, 1, 1.0, dtype, "arcface", 0.5, seed=28, labels=labels,
                abs_scaled=True, degenerate=True)
    assert out["K"] == 1


def test_positives_exceed_budget(dev):
    out = _case(dev, 512, 128, 1000, 0.05, "bf16", "cosface", 0.4, seed=6)
    assert out["K"] == out["n_pos"] > 50


def test_r1_full_softmax(dev):
    out = _case(dev, 64, 128, 2000, 1.0, "bf16", "arcface", 0.5, seed=7)
    assert out["K"] == 2000


def test_unowned_labels_and_offset(dev):
    # Shard [1000, 3000) of a larger head; a third of the labels fall outside it.
    _case(dev, 128, 128, 2000, 0.1, "bf16", "arcface", 0.5, seed=8, class_offset=1000,
          label_span=(0, 4000))


def test_no_owned_labels(dev):
    _case(dev, 32, 128, 2000, 0.1, "bf16", "cosface", 0.4, seed=9, class_offset=5000,
          label_span=(0, 4000))


def test_duplicated_positives(dev):
    rng = np.random.default_rng(10)
    labels = rng.choice(np.array([3, 17, 17, 17, 250, 999]), size=200)
    _case(dev, 200, 128, 1000, 0.1, "bf16", "cosface", 0.4, seed=10, labels=labels)


def test_single_row_and_tiny_shard(dev):
    # B = 1 makes the gradient scale s/B = 64, so |g| reaches ~100 here, two
    # orders of magnitude above any workload's.  The bf16 coefficients carry
    # ~2^-9 relative error, so the max-abs bar is applied relative to the
    # reference magnitude (max(1, max |ref|) times the stated bar) in this
    # case only; the row-relative bound is unchanged.
    _case(dev, 1, 128, 7, 0.5, "bf16", "arcface", 0.5, seed=11, abs_scaled=True)


def test_repeat_is_deterministic(dev):
    """Same inputs twice: bit-identical outputs (no floating-point atomics)."""
    from _gpu_util import make_problem
    outs = []
    for _ in range(2):
        Xd, Wd, Md, Pd, Ld = make_problem(200, 256, 6000, "bf16", 12, device=dev)
        shard = _shard(200, 256, 6000, 0.1, "bf16", "arcface", 0.5, dev=dev)
        shard.step(Xd, Ld, Wd, Md, 12)
        torch.cuda.synchronize()
        outs.append((shard.loss.clone(), shard.dX.clone(), Wd.clone(), Md.clone()))
    for a, b in zip(*outs):
        assert torch.equal(a, b)


@pytest.mark.parametrize("name", ["one_shard", "zipf", "massive"])
def test_sampler_full_size(dev, name):
    """Bit-exact active set and remap at the workloads' full shard sizes."""
    cfg = workloads.config(name)
    _, labels = workloads.make_batch(cfg, 0)
    print(f"\nsampler {name}: B={cfg['B']} C={cfg['C']} r={cfg['r']}", flush=True)
    shard = _shard(cfg["B"], cfg["d"], cfg["C"], cfg["r"], cfg["dtype"], cfg["margin"], cfg["m"],
                   dev=dev)
    Ld = torch.from_numpy(labels).to(dev)
    shard.sample(Ld, 0)
    torch.cuda.synchronize()
    active_ref, mapped_ref, info = O.sample_active(labels, cfg["C"], cfg["a"], cfg["r"], 0)
    K = int(shard.n_active.item())
    assert K == len(active_ref) == max(O.budget(cfg["r"], cfg["C"]), info["n_pos"])
    assert np.array_equal(shard.active[:K].cpu().numpy(), active_ref)
    assert np.array_equal(shard.labels_mapped.cpu().numpy(), mapped_ref)


# Shards that do not start on a Philox block (class_offset not a multiple of
# four), ragged last groups, every selection mode (keys; all classes at r = 1;
# positives only when they exceed the budget), duplicated and unowned labels.
@pytest.mark.parametrize("B,C,a,r,seed", [
    (64, 9001, 3, 0.1, 21),
    (300, 70001, 1000001, 0.05, 22),
    (8, 17, 2, 0.5, 23),
    (256, 5000, 6, 0.01, 24),       # |P| > budget: positives only
    (40, 2003, 5, 1.0, 25),         # every class
    (1000, 12289, 4097, 0.3, 26),   # most labels in one 4,096-class group
    (64, 9001, 2**40 + 3, 0.1, 29), # global ids above 2^32: the counter's high word
])
def test_sampler_offsets_and_modes(dev, B, C, a, r, seed):
    rng = np.random.default_rng(seed)
    labels = rng.integers(max(a - 50, 0), a + C + 50, size=B)  # some outside the shard
    if C > 8192:
        labels[: B // 2] = rng.integers(a + 4096, a + 8192, size=B // 2)
    labels[::7] = labels[0]                                    # duplicates
    print(f"\nsampler B={B} C={C} a={a} r={r} seed={seed}", flush=True)
    shard = _shard(B, 128, C, r, "bf16", "arcface", 0.5, class_offset=a, dev=dev)
    shard.sample(torch.from_numpy(labels.astype(np.int64)).to(dev), seed)
    torch.cuda.synchronize()
    active_ref, mapped_ref, info = O.sample_active(labels, C, a, r, seed)
    K = int(shard.n_active.item())
    assert K == len(active_ref) == max(O.budget(r, C), info["n_pos"])
    assert np.array_equal(shard.active[:K].cpu().numpy(), active_ref)
    assert np.array_equal(shard.labels_mapped.cpu().numpy(), mapped_ref)


def test_sampler_refinement_beyond_lds(dev):
    """A shard of 20M classes: the threshold's top-digit bucket holds more
    candidates than the refinement keeps in LDS (4,096), so it works on them
    in memory.  Bit-exact active set and remap."""
    from oracle import philox
    B, C, a, r, seed = 1024, 20_000_000, 0, 0.01, 31
    rng = np.random.default_rng(seed)
    labels = rng.integers(0, C, size=B)
    active_ref, mapped_ref, info = O.sample_active(labels, C, a, r, seed)
    # The bucket of the n_neg-th smallest non-positive key (12 top bits at this C).
    is_pos = np.zeros(C, dtype=bool)
    is_pos[info["positives"]] = True
    pool = np.nonzero(~is_pos)[0]
    digits = philox.class_keys(seed, pool + a) >> np.uint64(52)
    thresh_digit = np.sort(digits)[info["n_neg"] - 1]
    bucket = int(np.count_nonzero(digits == thresh_digit))
    assert bucket > 4096, bucket
    print(f"\nsampler C={C} r={r}: bucket of {bucket} candidates", flush=True)
    shard = _shard(B, 128, C, r, "bf16", "arcface", 0.5, class_offset=a, dev=dev)
    shard.sample(torch.from_numpy(labels.astype(np.int64)).to(dev), seed)
    torch.cuda.synchronize()
    K = int(shard.n_active.item())
    assert K == len(active_ref) == max(O.budget(r, C), info["n_pos"])
    assert np.array_equal(shard.active[:K].cpu().numpy(), active_ref)
    assert np.array_equal(shard.labels_mapped.cpu().numpy(), mapped_ref)


def test_many_rows_per_class(dev):
    # Every row is labelled with one of three classes of the same 128-class
    # tile: each quarter of the batch holds more target rows of that tile than
    # the class-gradient kernel lists, so it scans the labels instead.
    rng = np.random.default_rng(13)
    labels = rng.choice(np.array([5, 6, 100]), size=2400)
    _case(dev, 2400, 128, 3000, 0.1, "bf16", "arcface", 0.5, seed=13, labels=labels)


# PFC* conflict filter (Sec. 3.3.4, Eq. noise_filtering): some rows sit near
# the centre of another row's class, so their cosine to that (active)
# negative is ~0.9 > tau and the logit leaves the row's denominator.
@pytest.mark.parametrize("dtype,margin,m", [("bf16", "arcface", 0.5), ("f16", "cosface", 0.4)])
def test_conflict_filter(dev, dtype, margin, m):
    out = _case(dev, 300, 512, 20000, 0.1, dtype, margin, m, seed=14, tau=0.4, conflicts=3)
    assert out["n_filtered"] >= 50


def test_conflict_filter_ragged_and_unowned(dev):
    out = _case(dev, 100, 256, 5000, 0.2, "bf16", "arcface", 0.5, seed=15, class_offset=1000,
                label_span=(1000, 6500), tau=0.4, conflicts=2)
    assert out["n_filtered"] >= 20


def test_conflict_filter_fp32(dev):
    out = _case(dev, 64, 128, 2000, 0.1, "f32", "cosface", 0.4, seed=16, tau=0.4, conflicts=2)
    assert out["n_filtered"] >= 20


def test_conflict_filter_full_softmax(dev):
    """FC*-1.0: the filter at r = 1."""
    out = _case(dev, 64, 128, 2000, 1.0, "bf16", "arcface", 0.5, seed=17, tau=0.4, conflicts=2)
    assert out["K"] == 2000 and out["n_filtered"] >= 20


def test_tau_at_least_one_is_pfc(dev):
    """tau >= 1 runs the unfiltered kernels: bit-identical to no filter."""
    from _gpu_util import make_problem
    outs = []
    for tau in (None, 1.0):
        Xd, Wd, Md, Pd, Ld = make_problem(200, 256, 6000, "bf16", 18, device=dev, conflicts=2)
        shard = _shard(200, 256, 6000, 0.1, "bf16", "arcface", 0.5, dev=dev, tau=tau)
        shard.step(Xd, Ld, Wd, Md, 18)
        torch.cuda.synchronize()
        outs.append((shard.loss.clone(), shard.dX.clone(), Wd.clone(), Md.clone()))
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def _empty_row_problem(seed, dtype, dev, B=96, d=128, C=2000, a=1000, n_empty=3, mu=10.0):
    """Class centres sharing a common direction u, and a few rows along u whose
    labels lie outside the shard [a, a + C): every active cosine of such a row
    is ~0.66, above tau = 0.3, so the PFC* filter leaves its denominator empty.
    The other rows are ordinary Gaussian rows with owned labels."""
    rng = np.random.default_rng(seed)
    u = rng.standard_normal(d)
    u /= np.linalg.norm(u)
    W = (0.01 * (rng.standard_normal((C, d)) + mu * u)).astype(np.float32)
    X = rng.standard_normal((B, d)).astype(np.float32)
    labels = rng.integers(a, a + C, size=B)
    for k in range(n_empty):
        n = 7 + 31 * k
        X[n] = (np.sqrt(d) * u + 0.3 * rng.standard_normal(d)).astype(np.float32)
        labels[n] = a + C + 17 * k
    M = (1e-3 * rng.standard_normal((C, d))).astype(np.float32)
    t = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]
    return (torch.from_numpy(X).to(t).to(dev), torch.from_numpy(W).to(t).to(dev),
            torch.from_numpy(M).to(dev), None, torch.from_numpy(labels).to(dev))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_conflict_filter_empty_denominator(dev, dtype):
    """Rows whose label is outside the shard and whose every logit the PFC*
    filter drops: lse = -inf, no probability, no gradient, no NaN anywhere."""
    from _gpu_util import run_and_compare
    seed, tau = 32, 0.3
    print(f"\nempty-denominator rows: dtype={dtype} seed={seed} tau={tau}", flush=True)
    Xd, Wd, Md, Pd, Ld = _empty_row_problem(seed, dtype, dev)
    shard = _shard(96, 128, 2000, 0.2, dtype, "arcface", 0.5, class_offset=1000, dev=dev,
                   tau=tau)
    out = run_and_compare(shard, Xd, Wd, Md, Pd, Ld, seed, "arcface")
    print(out, flush=True)
    assert out["n_empty_rows"] == 3
    assert bool(torch.isfinite(Wd).all()) and bool(torch.isfinite(Md).all())
    empty = torch.isneginf(shard.row_lse)
    assert int(empty.sum()) == 3
    assert bool((shard.dX[empty] == 0).all())


@pytest.mark.parametrize("d,dtype,margin,m,seed", [
    (512, "f16", "arcface", 0.5, 20),
    (256, "bf16", "cosface", 0.4, 22),
    (128, "bf16", "arcface", 0.5, 23),
])
def test_batch_at_limit_16bit(dev, d, dtype, margin, m, seed):
    """The largest batch the ABI accepts (PFC_MAX_BATCH = 8192) at each feature
    width of the 16-bit path; the positives (~7,400 distinct labels) nearly
    fill the budget of 8,000."""
    from paper_2010_05222_amd import pfc
    assert pfc.PFC_MAX_BATCH == 8192
    out = _case(dev, 8192, d, 40000, 0.2, dtype, margin, m, seed=seed, random_m=False)
    assert out["K"] == 8000


def test_batch_at_limit_fp32(dev):
    """The largest batch of the fp32 path (4096 rows); here |P| > b, so S = P."""
    out = _case(dev, 4096, 128, 3000, 0.5, "f32", "cosface", 0.4, seed=21)
    assert out["K"] == out["n_pos"] > 1500


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_mapped_label_past_active_set_is_unowned(dev, dtype):
    """A labels_mapped entry at or past |S| (never produced by the sampler,
    but accepted by the forward and backward calls) counts as an unowned
    label: no target term and a zero loss term, as the oracle computes for a
    label of -1.  The id list is valid past |S| here, so the call reads no
    out-of-range class either way."""
    from _gpu_util import make_problem, row_rel_err, MAX_ABS, REL_ROW
    B, d, C, r, seed = 200, 128, 1000, 0.05, 41
    labels = np.random.default_rng(41).integers(0, 30, size=B)   # 30 classes: |S| = 50 < cap
    print(f"\ncase B={B} d={d} C={C} r={r} dtype={dtype} seed={seed} mapped label past |S|",
          flush=True)
    Xd, Wd, Md, Pd, Ld = make_problem(B, d, C, dtype, seed, labels=labels, device=dev)
    shard = _shard(B, d, C, r, dtype, "arcface", 0.5, 0, dev)
    X64 = Xd.double().cpu().numpy()
    W0 = Wd.double().cpu().numpy()
    M0 = Md.double().cpu().numpy()
    shard.sample(Ld, seed)
    torch.cuda.synchronize()
    K = int(shard.n_active.item())
    assert K + 5 < shard.cap, (K, shard.cap)
    shard.active[K + 5] = 0
    row = 7
    shard.labels_mapped[row] = K + 5
    shard.forward(Xd, Wd)
    shard.backward(Xd, Wd, Md, None)
    torch.cuda.synchronize()

    active = shard.active[:K].cpu().numpy()
    mapped = shard.labels_mapped.cpu().numpy().copy()
    mapped[row] = -1
    Ws = W0[active]
    fw = O.forward(X64, Ws, mapped, shard.s, shard.m, "arcface")
    loss_ref = O.batch_loss(fw["row_loss"], B)
    dx_ref = O.grad_x(X64, Ws, mapped, fw["lse"], B, shard.s, shard.m, "arcface")
    g_ref = O.grad_w(X64, Ws, np.arange(K), mapped, fw["lse"], B, shard.s, shard.m, "arcface")
    loss = float(shard.loss.item())
    dx = shard.dX.cpu().numpy().astype(np.float64)
    g = Md.double().cpu().numpy()[active] - shard.mu * M0[active]
    assert abs(loss - loss_ref) <= 1e-3 * abs(loss_ref), (loss, loss_ref)
    assert np.max(np.abs(dx - dx_ref)) <= MAX_ABS[dtype]
    assert np.max(row_rel_err(dx, dx_ref)) <= REL_ROW[dtype]
    assert np.max(np.abs(g - g_ref)) <= MAX_ABS[dtype]


def test_pipeline_equals_serial_steps(dev):
    """PfcPipeline (each step's active set drawn on a side stream beside the
    previous step) gives the serial steps' loss, row_lse, dX, W and momentum
    bit for bit over four steps with different batches and seeds."""
    from paper_2010_05222_amd.head import PfcPipeline
    from _gpu_util import make_problem
    B, d, C, r, T = 96, 256, 5000, 0.1, 4
    print(f"\ncase B={B} d={d} C={C} r={r} bf16 pipeline vs serial, {T} steps", flush=True)
    Xd, Wd, Md, _, _ = make_problem(B, d, C, "bf16", 51, device=dev)
    rng = np.random.default_rng(52)
    Ls = [torch.from_numpy(rng.integers(0, C, size=B)).to(dev) for _ in range(T)]
    Xs = [torch.roll(Xd, 7 * t, 0).contiguous() for t in range(T)]
    W1, M1, W2, M2 = Wd.clone(), Md.clone(), Wd.clone(), Md.clone()
    shard = _shard(B, d, C, r, "bf16", "arcface", 0.5, 0, dev)
    serial = []
    for t in range(T):
        shard.step(Xs[t], Ls[t], W1, M1, 100 + t)
        serial.append((shard.loss.clone(), shard.row_lse.clone(), shard.dX.clone()))
    pipe = PfcPipeline(B, d, C, r, dtype="bf16", s=64.0, m=0.5, margin="arcface", lr=0.1,
                       mu=0.9, device=dev)
    pipe.begin(Ls[0], 100)
    for t in range(T):
        last = t + 1 == T
        out = pipe.step(Xs[t], W2, M2, None if last else Ls[t + 1], None if last else 101 + t)
        got = (out.loss.clone(), out.row_lse.clone(), out.dX.clone())
        for a, b in zip(got, serial[t]):
            assert torch.equal(a, b), t
    torch.cuda.synchronize()
    assert torch.equal(W1, W2) and torch.equal(M1, M2)
    with pytest.raises(RuntimeError):
        pipe.step(Xs[0], W2, M2)          # no active set drawn for a fifth step
