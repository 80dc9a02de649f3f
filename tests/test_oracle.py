"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test names the passage of Partial FC (arXiv 2010.05222) or the external
definition that fixes the expected value.  None of them re-derives a value by
calling the function under test a second way.
"""

import math
import os

import numpy as np
import pytest
import torch

from oracle import pfc_oracle as O
from oracle.philox import class_keys, philox4x64_blocks, philox4x64_scalar
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------- Philox

def _kat_rows():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x64_10_kat.txt")) as fh:
        for line in fh:
            if line.startswith("#") or not line.strip():
                continue
            v = [int(t, 16) for t in line.split()]
            rows.append((tuple(v[0:4]), tuple(v[4:6]), tuple(v[6:10])))
    return rows


def test_philox_known_answers():
    """Published Philox4x64-10 known-answer vectors (SC'11 reference library)."""
    rows = _kat_rows()
    assert len(rows) == 3
    for ctr, key, out in rows:
        assert philox4x64_scalar(ctr, key) == out


def test_philox_vectorised_matches_scalar():
    rng = np.random.default_rng(1)
    c0 = rng.integers(0, 2**63, size=64, dtype=np.int64).astype(np.uint64) * np.uint64(2)
    for key in [(0, 0), (12345, 0), (2**64 - 1, 2**63 + 7)]:
        got = philox4x64_blocks(c0, key)
        for i in range(len(c0)):
            assert tuple(int(x) for x in got[i]) == philox4x64_scalar((int(c0[i]), 0, 0, 0), key)


@pytest.mark.parametrize("seed", [0, 1, 99, 2**40 + 3])
def test_class_keys_match_numpy_philox(seed):
    """numpy.random.Philox is an independent Philox4x64-10; it increments its
    counter before each block, so a start counter of -1 yields blocks 0, 1, ..."""
    n = 4096
    bitgen = np.random.Philox(key=np.array([seed, 0], dtype=np.uint64),
                              counter=np.array([2**64 - 1] * 4, dtype=np.uint64))
    stream = bitgen.random_raw(n)
    assert np.array_equal(class_keys(seed, np.arange(n)), stream)
    # Keys depend on the global id only: a shard starting at 1001 sees the same keys.
    assert np.array_equal(class_keys(seed, np.arange(1001, 1500)), stream[1001:1500])


# ----------------------------------------------------------------- sampling

def _check_sample(labels, C, a, r, seed):
    S, yhat, info = O.sample_active(labels, C, a, r, seed)
    S = S.astype(np.int64)
    y = np.asarray(labels)
    owned = (y >= a) & (y < a + C)
    P = np.unique(y[owned] - a)
    b = info["b"]
    # Sorted, unique, inside the shard.
    assert np.all(np.diff(S) > 0)
    assert S.size == 0 or (S[0] >= 0 and S[-1] < C)
    # Every positive kept (Sec. 3.3.1); |S| = max(b, |P|) (Eq. local_sampling).
    assert np.all(np.isin(P, S))
    assert S.size == max(b, P.size)
    # Remap (searchsorted): S[yhat] = local label; unowned rows -> -1.
    assert np.all(yhat[~owned] == -1)
    assert np.array_equal(S[yhat[owned]], y[owned] - a)
    # Negatives are the smallest-key non-positives: every chosen negative's
    # (key, id) precedes every unchosen non-positive's (key, id).
    neg = np.setdiff1d(S, P)
    rest = np.setdiff1d(np.arange(C), S)
    if neg.size and rest.size:
        kn, kr = class_keys(seed, neg + a), class_keys(seed, rest + a)
        worst = max(zip(kn.tolist(), neg.tolist()))
        best = min(zip(kr.tolist(), rest.tolist()))
        assert worst < best
    return S, yhat, info


@pytest.mark.parametrize("case", range(40))
def test_sampler_invariants_random(case):
    rng = np.random.default_rng([7, case])
    C = int(rng.integers(1, 400))
    B = int(rng.integers(1, 80))
    a = int(rng.integers(0, 3)) * int(rng.integers(0, 1000))
    r = float(rng.choice([0.01, 0.1, 0.25, 0.5, 1.0, rng.random()]))
    r = max(r, 1e-3)
    # Some labels outside the shard.
    labels = rng.integers(max(0, a - 20), a + C + 20, size=B)
    _check_sample(labels, C, a, r, int(rng.integers(0, 2**40)))


def test_sampler_r1_is_all_classes():
    """r = 1 activates every class: full softmax / full model parallelism (Sec. 3.3.2)."""
    labels = np.array([3, 3, 17, 99])
    S, yhat, _ = _check_sample(labels, 100, 0, 1.0, 5)
    assert np.array_equal(S, np.arange(100))
    assert np.array_equal(yhat, labels)


def test_sampler_positives_exceed_budget():
    """|P| > b keeps all positives and no negatives (Sec. 3.3.2)."""
    labels = np.arange(0, 100, 2)          # 50 distinct positives
    S, _, info = _check_sample(labels, 100, 0, 0.1, 3)    # b = 10
    assert info["b"] == 10 and info["n_neg"] == 0
    assert np.array_equal(S, labels)


def test_sampler_no_owned_labels():
    labels = np.array([500, 600, 700])
    S, yhat, info = _check_sample(labels, 100, 0, 0.2, 11)
    assert info["n_pos"] == 0 and S.size == 20
    assert np.all(yhat == -1)


def test_budget_reading():
    # Every workload's r*C is an integer, so floor and ceil agree.
    expect = {"tiny": 1000, "full_softmax": 1_000_000, "one_shard": 100_000,
              "zipf": 400_000, "massive": 800_000}
    for name, k in expect.items():
        cfg = workloads.config(name)
        assert O.budget(cfg["r"], cfg["C"]) == k
        assert math.floor(cfg["r"] * cfg["C"] + 1e-6) == k
    assert O.budget(0.1, 10001) == 1001       # ceil when r*C is fractional
    assert O.budget(1.0, 7) == 7


def test_sampler_inclusion_probability():
    """A non-positive class is activated with probability n_neg/(C - |P|) ~ r
    (Sec. 3.3.4), positives with probability 1; uniform over classes."""
    C, r, trials = 60, 0.25, 3000
    labels = np.array([0, 5, 5, 9])
    counts = np.zeros(C)
    for t in range(trials):
        S, _, info = O.sample_active(labels, C, 0, r, t)
        counts[S] += 1
    pos = np.array([0, 5, 9])
    assert np.all(counts[pos] == trials)
    neg = np.setdiff1d(np.arange(C), pos)
    p = (O.budget(r, C) - 3) / (C - 3)
    sd = math.sqrt(trials * p * (1 - p))
    z = (counts[neg] - trials * p) / sd
    assert np.max(np.abs(z)) < 4.5          # ~57 classes, Bonferroni-safe
    assert abs(np.mean(counts[neg]) - trials * p) < 0.01 * trials


# ----------------------------------------------------------------- forward

def _unit(a):
    return a / np.linalg.norm(a, axis=1, keepdims=True)


def test_full_softmax_at_r1_matches_library_cross_entropy():
    """At r = 1 (and m = 0) the PFC loss is the plain normalised softmax CE
    (Sec. 3.2.1 matrix form): torch's cross_entropy on the dense logits."""
    rng = np.random.default_rng(3)
    B, d, C, s = 16, 12, 40, 64.0
    X = rng.standard_normal((B, d))
    W = 0.01 * rng.standard_normal((C, d))
    labels = rng.integers(0, C, size=B)
    S, yhat, _ = O.sample_active(labels, C, 0, 1.0, 0)
    assert np.array_equal(S, np.arange(C))
    for margin in (O.COSFACE, O.ARCFACE):
        fw = O.forward(X, W[S], yhat, s, 0.0, margin)
        loss = O.batch_loss(fw["row_loss"], B)
        Z = torch.from_numpy(s * _unit(X) @ _unit(W).T)
        ref = torch.nn.functional.cross_entropy(Z, torch.from_numpy(labels)).item()
        assert abs(loss - ref) < 1e-12 * max(1, abs(ref))
        assert np.allclose(fw["P"].sum(axis=1), 1.0, atol=1e-14, rtol=0)
        Pref = torch.softmax(Z, dim=1).numpy()
        assert np.allclose(fw["P"], Pref, atol=1e-14, rtol=0)


def _orthonormal_case(B, K, d, target_equals_row):
    """W rows = first K basis vectors of R^d (scaled); X rows either the
    target's basis vector or a basis vector orthogonal to every row of W."""
    assert d > K
    W = np.zeros((K, d))
    W[np.arange(K), np.arange(K)] = 0.3
    labels = np.arange(B) % K
    X = np.zeros((B, d))
    if target_equals_row:
        X[np.arange(B), labels] = 2.0
    else:
        X[:, K] = 1.5
    return X, W, labels


@pytest.mark.parametrize("margin,m", [(O.COSFACE, 0.4), (O.ARCFACE, 0.5)])
def test_margin_closed_forms(margin, m):
    """Closed forms: with all cosines 0 the row loss is log(e^{f_y} + K - 1) - f_y
    with f_y = -s m (CosFace) or s cos(pi/2 + m) = -s sin m (ArcFace); with the
    target cosine 1 and all others 0, f_y = s (1 - m) or s cos(m)."""
    s, K, d, B = 64.0, 7, 10, 5
    X, W, labels = _orthonormal_case(B, K, d, False)
    fw = O.forward(X, W, labels, s, m, margin)
    fy = -s * m if margin == O.COSFACE else -s * math.sin(m)
    expect = math.log(math.exp(fy) + K - 1) - fy
    assert np.allclose(fw["row_loss"], expect, rtol=1e-13, atol=0)
    X, W, labels = _orthonormal_case(B, K, d, True)
    fw = O.forward(X, W, labels, s, m, margin)
    fy = s * (1 - m) if margin == O.COSFACE else s * math.cos(m)
    expect = math.log(math.exp(fy) + K - 1) - fy
    assert np.allclose(fw["row_loss"], expect, rtol=1e-12, atol=1e-300)


def test_zero_margin_cosface_equals_arcface_and_scale_invariance():
    rng = np.random.default_rng(4)
    X = rng.standard_normal((9, 16))
    W = rng.standard_normal((30, 16))
    y = rng.integers(0, 30, size=9)
    a = O.forward(X, W, y, 64.0, 0.0, O.COSFACE)["row_loss"]
    b = O.forward(X, W, y, 64.0, 0.0, O.ARCFACE)["row_loss"]
    assert np.allclose(a, b, rtol=1e-12, atol=1e-12)
    # Normalised logits: positive rescaling of rows changes nothing (Sec. 3.1).
    c = O.forward(X * rng.uniform(0.1, 9, (9, 1)), W * rng.uniform(0.1, 9, (30, 1)),
                  y, 64.0, 0.5, O.ARCFACE)["row_loss"]
    d_ = O.forward(X, W, y, 64.0, 0.5, O.ARCFACE)["row_loss"]
    assert np.allclose(c, d_, rtol=1e-12, atol=1e-12)


def test_unowned_rows_have_no_loss_term():
    rng = np.random.default_rng(5)
    X = rng.standard_normal((4, 8))
    W = rng.standard_normal((6, 8))
    y = np.array([1, -1, 3, -1])
    fw = O.forward(X, W, y, 64.0, 0.4, O.COSFACE)
    assert fw["row_loss"][1] == 0 and fw["row_loss"][3] == 0
    assert fw["row_loss"][0] > 0


# ----------------------------------------------------------------- backward

def _loss_fn(X, Ws, y, B, s, m, margin):
    """The shard's differentiable objective.  A row whose label lies outside
    the shard keeps only its log-sum-exp here: its target term belongs to the
    owning shard (Sec. 3.2.1: only the owner contributes the target term), so
    the local gradient of that row is P/B."""
    fw = O.forward(X, Ws, y, s, m, margin)
    return (np.sum(fw["row_loss"]) + np.sum(fw["lse"][np.asarray(y) < 0])) / B


@pytest.mark.parametrize("margin,m", [(O.COSFACE, 0.4), (O.ARCFACE, 0.5), (O.COSFACE, 0.0)])
def test_gradients_match_finite_differences(margin, m):
    """Brute-force central differences of the batch loss (check 4)."""
    rng = np.random.default_rng([8, int(m * 10)])
    B, d, C, r, s = 4, 8, 20, 0.5, 8.0   # smaller s keeps the loss smooth for h = 1e-6
    X = rng.standard_normal((B, d))
    W = rng.standard_normal((C, d))
    labels = np.array([2, 2, 11, 25])      # one row outside the shard
    S, y, _ = O.sample_active(labels, C, 0, r, 4)
    Ws = W[S]
    fw = O.forward(X, Ws, y, s, m, margin)
    dx = O.grad_x(X, Ws, y, fw["lse"], B, s, m, margin)
    gw = O.grad_w(X, Ws, np.arange(len(S)), y, fw["lse"], B, s, m, margin)
    h = 1e-6
    for (arr, grad) in ((X, dx), (Ws, gw)):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            keep = arr[idx]
            arr[idx] = keep + h
            lp = _loss_fn(X, Ws, y, B, s, m, margin)
            arr[idx] = keep - h
            lm = _loss_fn(X, Ws, y, B, s, m, margin)
            arr[idx] = keep
            num[idx] = (lp - lm) / (2 * h)
        err = np.max(np.abs(num - grad)) / max(1e-12, np.max(np.abs(num)))
        assert err < 1e-6, err


@pytest.mark.parametrize("margin,m", [(O.COSFACE, 0.4), (O.ARCFACE, 0.5)])
def test_gradients_match_torch_autograd(margin, m):
    """torch float64 autograd of the same loss, with W[S] as a leaf."""
    rng = np.random.default_rng(9)
    B, d, C, r, s = 12, 16, 60, 0.3, 64.0
    X = rng.standard_normal((B, d))
    W = 0.01 * rng.standard_normal((C, d))
    labels = rng.integers(0, C, size=B)
    labels[0] = C + 3                       # unowned row
    S, y, _ = O.sample_active(labels, C, 0, r, 1)
    Ws = W[S]
    fw = O.forward(X, Ws, y, s, m, margin)
    dx = O.grad_x(X, Ws, y, fw["lse"], B, s, m, margin)
    gw = O.grad_w(X, Ws, np.arange(len(S)), y, fw["lse"], B, s, m, margin)

    tX = torch.tensor(X, requires_grad=True)
    tW = torch.tensor(Ws, requires_grad=True)
    cos = torch.nn.functional.normalize(tX, dim=1) @ torch.nn.functional.normalize(tW, dim=1).T
    ty = torch.tensor(y.astype(np.int64))
    own = ty >= 0
    rows = torch.nonzero(own).flatten()
    ct = cos[rows, ty[rows]]
    if margin == O.COSFACE:
        ft = s * (ct - m)
    else:
        ft = s * torch.cos(torch.acos(ct) + m)
    f = (s * cos).index_put((rows, ty[rows]), ft)
    lse = torch.logsumexp(f, dim=1)
    loss = (lse[rows] - f[rows, ty[rows]]).sum() / B
    # Unowned rows keep only their log-sum-exp in the shard's objective.
    objective = loss + lse[~own].sum() / B
    objective.backward()
    assert abs(loss.item() - O.batch_loss(fw["row_loss"], B)) < 1e-12
    assert np.allclose(dx, tX.grad.numpy(), atol=1e-12, rtol=1e-9)
    assert np.allclose(gw, tW.grad.numpy(), atol=1e-12, rtol=1e-9)


def test_gradient_row_sums_and_tangent_projection():
    """Rows of (P - Y) sum to 0 for owned rows and to 1 for unowned rows (check
    3); the normalisation backward is orthogonal to each row (Sec. 3.1)."""
    rng = np.random.default_rng(10)
    B, d, K, s = 6, 10, 25, 64.0
    X = rng.standard_normal((B, d))
    Ws = rng.standard_normal((K, d))
    y = np.array([0, 4, 4, 24, -1, 7])
    fw = O.forward(X, Ws, y, s, 0.0, O.COSFACE)
    dc = O.cos_grad(fw["cos"], fw["lse"], y, B, s, 0.0, O.COSFACE)
    sums = dc.sum(axis=1) * B / s
    assert np.allclose(sums[y >= 0], 0.0, atol=1e-13)
    assert np.allclose(sums[y < 0], 1.0, atol=1e-13)
    dx = O.grad_x(X, Ws, y, fw["lse"], B, s, 0.5, O.ARCFACE)
    g = O.grad_w(X, Ws, np.arange(K), y, fw["lse"], B, s, 0.5, O.ARCFACE)
    assert np.allclose(np.sum(_unit(X) * dx, axis=1), 0, atol=1e-14)
    assert np.allclose(np.sum(_unit(Ws) * g, axis=1), 0, atol=1e-14)


def test_class_subset_gradient_matches_full():
    rng = np.random.default_rng(11)
    B, d, K = 8, 12, 30
    X = rng.standard_normal((B, d))
    Ws = rng.standard_normal((K, d))
    y = rng.integers(0, K, size=B)
    fw = O.forward(X, Ws, y, 64.0, 0.5, O.ARCFACE)
    full = O.grad_w(X, Ws, np.arange(K), y, fw["lse"], B, 64.0, 0.5, O.ARCFACE)
    cols = np.array([y[0], 3, 17, y[5], 29])
    part = O.grad_w(X, Ws[cols], cols, y, fw["lse"], B, 64.0, 0.5, O.ARCFACE)
    assert np.allclose(part, full[cols], rtol=1e-12, atol=1e-15)


def test_arcface_beyond_pi_is_finite():
    """theta + m > pi: paper silent (parity unpinned); only finiteness checked."""
    X = np.array([[-1.0, 0.01]])
    W = np.array([[1.0, 0.0], [0.0, 1.0]])
    fw = O.forward(X, W, np.array([0]), 64.0, 0.5, O.ARCFACE)
    assert np.all(np.isfinite(fw["row_loss"]))
    dx = O.grad_x(X, W, np.array([0]), fw["lse"], 1, 64.0, 0.5, O.ARCFACE)
    assert np.all(np.isfinite(dx))


# ----------------------------------------------------------------- update

def test_round_bf16_matches_library_on_float32_values():
    rng = np.random.default_rng(12)
    x = (rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 6, 20000)).astype(np.float32)
    ours = O.round_bf16(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ours, ref)


@pytest.mark.parametrize("random_m", [False, True])
def test_momentum_update_matches_torch_sgd(random_m):
    """Lazy momentum SGD on the active rows equals torch.optim.SGD (momentum,
    no dampening/Nesterov/decay) run on the gathered rows; every other row and
    its momentum stay bit-identical (Sec. 3.1, Sec. 3.3.1)."""
    rng = np.random.default_rng(13)
    C, d, lr, mu = 50, 6, 0.1, 0.9
    W = rng.standard_normal((C, d)).astype(np.float32).astype(np.float64)
    M = (rng.standard_normal((C, d)) * 1e-3 if random_m else np.zeros((C, d)))
    M = M.astype(np.float32).astype(np.float64)
    active = np.array([1, 4, 5, 30, 49])
    g = rng.standard_normal((len(active), d))
    W0, M0 = W.copy(), M.copy()
    O.momentum_update(W, M, active, g, lr, mu, "f32")
    p = torch.nn.Parameter(torch.tensor(W0[active]))
    opt = torch.optim.SGD([p], lr=lr, momentum=mu, dampening=0, nesterov=False, weight_decay=0)
    if random_m:
        opt.state[p]["momentum_buffer"] = torch.tensor(M0[active])
    p.grad = torch.tensor(g)
    opt.step()
    assert np.allclose(W[active], p.detach().numpy(), rtol=0, atol=1e-6)
    assert np.allclose(M[active], opt.state[p]["momentum_buffer"].numpy(), rtol=1e-7, atol=1e-12)
    rest = np.setdiff1d(np.arange(C), active)
    assert np.array_equal(W[rest], W0[rest]) and np.array_equal(M[rest], M0[rest])


def test_master_update_rounds_shadow():
    rng = np.random.default_rng(14)
    C, d = 10, 4
    master = rng.standard_normal((C, d)).astype(np.float32).astype(np.float64)
    W = O.round_bf16(master)
    M = np.zeros((C, d))
    active = np.array([2, 7])
    g = rng.standard_normal((2, d))
    master0 = master.copy()
    O.momentum_update(W, M, active, g, 0.1, 0.9, "bf16", master=master)
    # From zero momentum the buffer is g and the master moves by -lr*g (fp32).
    expect = (master0[active] - 0.1 * g).astype(np.float32).astype(np.float64)
    assert np.array_equal(master[active], expect)
    assert np.array_equal(W[active], O.round_bf16(expect))
    rest = np.setdiff1d(np.arange(C), active)
    assert np.array_equal(master[rest], master0[rest])


def test_lazy_step_at_r1_equals_dense_step():
    """r = 1: the sampled step is the dense full-softmax SGD step (Sec. 3.3.2)."""
    rng = np.random.default_rng(15)
    B, d, C = 10, 8, 30
    X = rng.standard_normal((B, d))
    W = (0.01 * rng.standard_normal((C, d))).astype(np.float32).astype(np.float64)
    M = np.zeros((C, d))
    labels = rng.integers(0, C, size=B)
    W1, M1 = W.copy(), M.copy()
    out = O.step(X, W1, M1, labels, C, 0, 1.0, 0, 64.0, 0.4, O.COSFACE, 0.1, 0.9, "f32")
    # Dense reference with torch autograd over the whole classifier.
    tX = torch.tensor(X)
    tW = torch.nn.Parameter(torch.tensor(W))
    cos = torch.nn.functional.normalize(tX, dim=1) @ torch.nn.functional.normalize(tW, dim=1).T
    f = 64.0 * cos - 64.0 * 0.4 * torch.nn.functional.one_hot(torch.tensor(labels), C).double()
    loss = torch.nn.functional.cross_entropy(f, torch.tensor(labels))
    opt = torch.optim.SGD([tW], lr=0.1, momentum=0.9)
    loss.backward()
    opt.step()
    assert abs(out["loss"] - loss.item()) < 1e-12
    assert np.allclose(W1, tW.detach().numpy(), atol=1e-12, rtol=2**-23)   # fp32 storage rounding


# ------------------------------------------------- PFC* conflict filter

def _conflict_problem(seed, B=10, d=12, C=30, r=0.5):
    """Rows of X placed near the centre of an active class other than their
    own label (a duplicated identity), so that some negative cosines exceed
    tau = 0.4, and one row near its own centre (a positive above tau)."""
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((C, d))
    labels = rng.integers(0, C, size=B)
    S, y, _ = O.sample_active(labels, C, 0, r, seed)
    X = rng.standard_normal((B, d))
    for n in range(0, B, 2):                      # conflicts: near another row's class
        k = y[(n + 1) % B]
        if k != y[n]:
            X[n] = W[S[k]] + 0.3 * rng.standard_normal(d)
    X[1] = W[S[y[1]]] + 0.1 * rng.standard_normal(d)   # positive far above tau
    return X, W[S], y


def test_filter_tau_at_least_one_is_pfc():
    """tau >= 1 keeps every logit (cos <= 1), so PFC* reduces to PFC."""
    X, Ws, y = _conflict_problem(21)
    B, s, m = len(y), 64.0, 0.5
    ref = O.forward(X, Ws, y, s, m, O.ARCFACE)
    for tau in (1.0, 1.5):
        fw = O.forward(X, Ws, y, s, m, O.ARCFACE, tau)
        assert np.array_equal(fw["lse"], ref["lse"])
        assert np.array_equal(
            O.grad_x(X, Ws, y, fw["lse"], B, s, m, O.ARCFACE, tau),
            O.grad_x(X, Ws, y, ref["lse"], B, s, m, O.ARCFACE))


def test_filter_matches_brute_force_definition():
    """Loss of Eq. noise_filtering written out with loops: a logit enters row
    n's denominator iff it is the target or its unmargined cosine is <= tau;
    the positive is never filtered; probabilities of the kept logits sum to 1
    and dropped logits have probability 0."""
    tau, s, m = 0.4, 16.0, 0.35
    X, Ws, y = _conflict_problem(22)
    B, K = len(y), len(Ws)
    fw = O.forward(X, Ws, y, s, m, O.COSFACE, tau)
    n_dropped = 0
    for n in range(B):
        xh = X[n] / math.sqrt(sum(v * v for v in X[n]))
        terms, ft = [], None
        for j in range(K):
            wh = Ws[j] / math.sqrt(sum(v * v for v in Ws[j]))
            c = sum(a * b for a, b in zip(xh, wh))
            if j == y[n]:
                ft = s * (c - m)
                terms.append(ft)
            elif c <= tau:
                terms.append(s * c)
            else:
                n_dropped += 1
                assert fw["P"][n, j] == 0.0
        lse = math.log(sum(math.exp(t) for t in terms))
        assert abs(fw["lse"][n] - lse) < 1e-12 * max(1.0, abs(lse))
        assert abs(fw["row_loss"][n] - (lse - ft)) < 1e-11
        assert abs(np.sum(fw["P"][n]) - 1.0) < 1e-12
    assert n_dropped >= B // 2 - 1       # the problem does exercise the filter
    assert fw["cos"][1, y[1]] > tau      # a positive above tau is kept (checked above)


@pytest.mark.parametrize("margin,m", [(O.COSFACE, 0.4), (O.ARCFACE, 0.5)])
def test_filter_gradients_match_torch_autograd(margin, m):
    """torch float64 autograd of the filtered loss (dropped logits masked to
    -inf; the mask is piecewise constant) with W[S] as a leaf."""
    tau, s = 0.4, 32.0
    X, Ws, y = _conflict_problem(23)
    B = len(y)
    fw = O.forward(X, Ws, y, s, m, margin, tau)
    dx = O.grad_x(X, Ws, y, fw["lse"], B, s, m, margin, tau)
    gw = O.grad_w(X, Ws, np.arange(len(Ws)), y, fw["lse"], B, s, m, margin, tau)
    tX = torch.tensor(X, requires_grad=True)
    tW = torch.tensor(Ws, requires_grad=True)
    cos = torch.nn.functional.normalize(tX, dim=1) @ torch.nn.functional.normalize(tW, dim=1).T
    ty = torch.tensor(y.astype(np.int64))
    rows = torch.arange(B)
    ct = cos[rows, ty]
    ft = s * (ct - m) if margin == O.COSFACE else s * torch.cos(torch.acos(ct) + m)
    f = (s * cos).index_put((rows, ty), ft)
    drop = (cos.detach() > tau)
    drop[rows, ty] = False
    assert bool(drop.any())
    f = f.masked_fill(drop, -math.inf)
    loss = (torch.logsumexp(f, dim=1) - f[rows, ty]).sum() / B
    loss.backward()
    assert abs(loss.item() - O.batch_loss(fw["row_loss"], B)) < 1e-12
    assert np.allclose(dx, tX.grad.numpy(), atol=1e-12, rtol=1e-9)
    assert np.allclose(gw, tW.grad.numpy(), atol=1e-12, rtol=1e-9)


def test_filter_step_at_r1_is_fc_star():
    """FC*-1.0 (Sec. 3.3.4): PFC* at r = 1 is the filtered full softmax; the
    step's class gradients match the dense filtered gradient of every class."""
    rng = np.random.default_rng(24)
    B, d, C, tau, s, m = 8, 10, 16, 0.4, 64.0, 0.5
    X = rng.standard_normal((B, d))
    W = rng.standard_normal((C, d))
    labels = rng.integers(0, C, size=B)
    X[0] = W[(labels[0] + 1) % C] + 0.2 * rng.standard_normal(d)
    out = O.step(X, W.copy(), np.zeros((C, d)), labels, C, 0, 1.0, 3, s, m, O.ARCFACE, 0.1,
                 0.9, "f32", tau=tau)
    assert np.array_equal(out["active"], np.arange(C))
    fw = O.forward(X, W, labels, s, m, O.ARCFACE, tau)
    assert abs(out["loss"] - O.batch_loss(fw["row_loss"], B)) < 1e-12
    assert out["P"][0, (labels[0] + 1) % C] == 0.0


def _nearest_f16_brute_force(x):
    """Nearest binary16 value of each float64 x, ties to the even bit pattern,
    by search over the sorted table of every finite binary16 value (the table
    comes from widening bit patterns, which is exact)."""
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    vals = bits.view(np.float16).astype(np.float64)
    ok = np.isfinite(vals) & ~((vals == 0) & (bits >= 0x8000))     # drop inf/nan and -0
    vals, bits = vals[ok], bits[ok]
    order = np.argsort(vals, kind="stable")
    vals, bits = vals[order], bits[order]
    i = np.clip(np.searchsorted(vals, x), 1, len(vals) - 1)
    lo, hi = vals[i - 1], vals[i]
    dlo, dhi = x - lo, hi - x
    pick_hi = (dhi < dlo) | ((dhi == dlo) & (bits[i] % 2 == 0))
    return np.where(pick_hi, hi, lo)


def test_round_f16_matches_brute_force_and_library():
    """The fp16 branch of round_to against (a) a brute-force nearest-value
    search over all binary16 values with ties to even, on float64 inputs that
    include exact midpoints and subnormals, and (b) torch's float32 -> float16
    conversion on float32 inputs."""
    rng = np.random.default_rng(13)
    x = rng.standard_normal(20000) * 10.0 ** rng.integers(-8, 4, 20000)
    # exact midpoints between neighbouring binary16 values (ties), both signs
    grid = np.sort(np.unique(rng.standard_normal(4000).astype(np.float16).astype(np.float64)))
    mids = (grid[:-1] + grid[1:]) / 2.0
    sub = np.arange(1, 2000) * 2.0 ** -25            # around the subnormal spacing 2^-24
    x = np.concatenate([x, mids, -mids, sub, -sub])
    x = x[np.abs(x) < 65504.0]
    assert np.array_equal(O.round_to(x, "f16"), _nearest_f16_brute_force(x))
    x32 = (rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 4, 20000)).astype(np.float32)
    x32 = x32[np.abs(x32) < 65504.0]
    ref = torch.from_numpy(x32).to(torch.float16).to(torch.float64).numpy()
    assert np.array_equal(O.round_to(x32.astype(np.float64), "f16"), ref)


def test_empty_denominator_row_contributes_nothing():
    """A row whose label is outside the shard and whose every logit the PFC*
    filter drops has an empty denominator (reading of Eq. noise_filtering):
    lse = -inf, probability 0 everywhere, no gradient, loss term 0.  Pinned
    against the same batch without that row (same batch size in the mean):
    every other row's lse, dx and every class gradient are unchanged."""
    rng = np.random.default_rng(25)
    B, d, K, tau, s, m = 6, 12, 9, 0.3, 32.0, 0.5
    u = rng.standard_normal(d)
    u /= np.linalg.norm(u)
    Ws = rng.standard_normal((K, d)) + 6.0 * u           # every centre leans along u
    X = rng.standard_normal((B, d))
    y = rng.integers(0, K, size=B)
    X[2] = 4.0 * u + 0.05 * rng.standard_normal(d)
    y[2] = -1                                           # label outside the shard
    for margin in (O.COSFACE, O.ARCFACE):
        fw = O.forward(X, Ws, y, s, m, margin, tau)
        assert np.all(fw["cos"][2] > tau)               # every logit of row 2 is dropped
        assert fw["lse"][2] == -np.inf and np.all(fw["P"][2] == 0.0)
        assert fw["row_loss"][2] == 0.0
        dx = O.grad_x(X, Ws, y, fw["lse"], B, s, m, margin, tau)
        g = O.grad_w(X, Ws, np.arange(K), y, fw["lse"], B, s, m, margin, tau)
        assert np.all(np.isfinite(dx)) and np.all(np.isfinite(g))
        assert np.all(dx[2] == 0.0)
        keep = np.array([n for n in range(B) if n != 2])
        fk = O.forward(X[keep], Ws, y[keep], s, m, margin, tau)
        assert np.array_equal(fw["lse"][keep], fk["lse"])
        assert O.batch_loss(fw["row_loss"], B) == O.batch_loss(fk["row_loss"], B)
        assert np.allclose(dx[keep], O.grad_x(X[keep], Ws, y[keep], fk["lse"], B, s, m, margin,
                                              tau), rtol=1e-13, atol=1e-15)
        assert np.allclose(g, O.grad_w(X[keep], Ws, np.arange(K), y[keep], fk["lse"], B, s, m,
                                       margin, tau), rtol=1e-13, atol=1e-15)
