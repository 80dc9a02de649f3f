"""Plain CPU oracle of the Partial FC classifier-head step on one class shard.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import or call this module.  It shares no
code with the HIP path and imports nothing from it.

Every float computation runs in float64.  Inputs given in a 16-bit format are
expected as float64 arrays holding the exact upcast values.  Each function
cites the passage of Partial FC (arXiv 2010.05222) it follows.  Where the paper
is silent the reading taken is stated next to the code.

Functions that work on a subset of rows (samples) or columns (sampled classes)
evaluate the same definitions on that subset; rows of the forward pass are
independent, and a class gradient needs only the per-row log-sum-exp, so large
problems can be checked on sampled outputs.

Parity status: sampling, remap, forward, backward, the update and the PFC*
conflict filter are pinned (see tests/test_oracle.py).  "Parity unpinned": ArcFace where theta + m > pi
(only finiteness is checked there), and the exact rounding points of the GPU's
16-bit operands (covered by tolerance only).
"""

import math

import numpy as np

from .philox import class_keys

EPS_NORM = 1e-12       # floor of a row norm (paper silent; never reached by Gaussian data)
EPS_SIN2 = 1e-12       # floor of sin^2(theta) in the ArcFace derivative (paper silent)

COSFACE = "cosface"
ARCFACE = "arcface"


# ---------------------------------------------------------------------------
# Sampling and remap (Sec. 3.3.1 and Sec. 3.3.2, Eq. local_sampling)
# ---------------------------------------------------------------------------

def local_labels(labels, C, a):
    """Label masking to local coordinates (Sec. 3.3.2): y - a if owned, else -1."""
    y = np.asarray(labels, dtype=np.int64)
    owned = (y >= a) & (y < a + C)
    return np.where(owned, y - a, -1).astype(np.int64)


def positive_set(y_local):
    """Local positive set: sorted unique owned local labels (Sec. 3.3.2)."""
    y = np.asarray(y_local, dtype=np.int64)
    return np.unique(y[y >= 0])


def budget(r, C):
    """Activation budget b for a shard of C classes at rate r.

    The paper writes floor(r*C) (Sec. 3.3.2); the build target states
    ceil(r*C).  Reading: r*C within 1e-9 relative of an integer is that
    integer (all workloads here), otherwise ceil.
    """
    t = float(r) * float(C)
    rt = round(t)
    if abs(t - rt) <= 1e-9 * max(1.0, t):
        return int(rt)
    return int(math.ceil(t))


def sample_active(labels, C, a, r, seed):
    """Positive-preserving sampling and label remap (Eq. local_sampling).

    S = P  union  Sample([0, C) minus P, max(b - |P|, 0)), sorted ascending;
    labels_mapped = searchsorted(S, y_local) for owned rows, else -1.

    The paper does not say how the draw without replacement is made.  Reading: each
    class c gets the 64-bit key of its global id a + c (see philox.class_keys)
    and the negatives are the max(b - |P|, 0) non-positive classes with the
    smallest (key, c) pairs in lexicographic order.  That is a uniformly random
    subset (keys i.i.d. uniform; ties broken by the lower class id).

    Returns (active int32[K], labels_mapped int32[B], info dict).
    """
    y_loc = local_labels(labels, C, a)
    P = positive_set(y_loc)
    b = budget(r, C)
    n_neg = max(b - len(P), 0)
    is_pos = np.zeros(C, dtype=bool)
    is_pos[P] = True
    pool = np.nonzero(~is_pos)[0]
    if n_neg > 0:
        keys = class_keys(seed, pool + a)
        order = np.lexsort((pool, keys))        # primary: key, secondary: class id
        negatives = pool[order[:n_neg]]
    else:
        negatives = np.zeros(0, dtype=np.int64)
    S = np.sort(np.concatenate([P, negatives]))
    mapped = np.full(y_loc.shape, -1, dtype=np.int64)
    own = y_loc >= 0
    mapped[own] = np.searchsorted(S, y_loc[own], side="left")
    info = {"b": b, "n_pos": len(P), "n_neg": n_neg, "positives": P}
    return S.astype(np.int32), mapped.astype(np.int32), info


# ---------------------------------------------------------------------------
# Normalisation, margins and the sampled softmax (Sec. 3.1, Eq. proxy_softmax,
# Eq. pfc_probability_overview / sampled_probability)
# ---------------------------------------------------------------------------

def row_norms(A):
    """max(||a_n||, eps) for each row (normalised cosine logits, Sec. 3.1)."""
    A = np.asarray(A, dtype=np.float64)
    return np.maximum(np.sqrt(np.sum(A * A, axis=1)), EPS_NORM)


def target_logit(c, s, m, margin):
    """Margined target logit from the unmargined cosine c (Sec. 3.1, Sec. 2.1).

    CosFace (additive cosine margin): s * (c - m).
    ArcFace (additive angular margin): s * cos(arccos(c) + m), c clipped to
    [-1, 1]; no "easy margin" branch for theta + m > pi (paper silent).
    """
    c = np.asarray(c, dtype=np.float64)
    if margin == COSFACE:
        return s * (c - m)
    if margin == ARCFACE:
        return s * np.cos(np.arccos(np.clip(c, -1.0, 1.0)) + m)
    raise ValueError(margin)


def target_logit_slope(c, m, margin):
    """d(target logit)/dc divided by s: 1 (CosFace), sin(theta+m)/sin(theta) (ArcFace)."""
    c = np.asarray(c, dtype=np.float64)
    if margin == COSFACE:
        return np.ones_like(c)
    if margin == ARCFACE:
        theta = np.arccos(np.clip(c, -1.0, 1.0))
        return np.sin(theta + m) / np.sqrt(np.maximum(1.0 - c * c, EPS_SIN2))
    raise ValueError(margin)


def cosines(X, Ws):
    """Unmargined cosines x_hat_n . w_hat_j over the active classes (Sec. 3.1)."""
    X = np.asarray(X, dtype=np.float64)
    Ws = np.asarray(Ws, dtype=np.float64)
    xh = X / row_norms(X)[:, None]
    wh = Ws / row_norms(Ws)[:, None]
    return xh @ wh.T


def conflict_mask(cos, yhat, tau):
    """PFC* filter (Sec. 3.3.4, Eq. noise_filtering): M[n, j] = 1 at the row's target,
    else 1 iff the unmargined cosine is <= tau.

    Reading: tau None or tau >= 1 means no filtering (PFC itself); the cosine
    never exceeds 1, so this only removes the effect of rounding at tau = 1.
    A row whose label is outside the shard has no target column: all its
    columns are negatives.
    """
    cos = np.asarray(cos, dtype=np.float64)
    if tau is None or tau >= 1.0:
        return np.ones(cos.shape, dtype=bool)
    keep = cos <= tau
    yhat = np.asarray(yhat, dtype=np.int64)
    n = np.nonzero(yhat >= 0)[0]
    if n.size:
        keep[n, yhat[n]] = True
    return keep


def logits(cos, yhat, s, m, margin, tau=None):
    """f = s * cos with the margin applied at each owned row's target column;
    -inf where the PFC* filter drops the logit from the row's denominator."""
    f = s * np.asarray(cos, dtype=np.float64)
    n = np.nonzero(np.asarray(yhat) >= 0)[0]
    if n.size:
        j = np.asarray(yhat)[n]
        f[n, j] = target_logit(cos[n, j], s, m, margin)
    if tau is not None and tau < 1.0:
        f = np.where(conflict_mask(cos, yhat, tau), f, -np.inf)
    return f


def log_sum_exp(f):
    """Row log-sum-exp as max + log(sum exp(f - max)) (Sec. 3.2.1 max/sum steps).

    Reading (paper silent): a row with no logit left (every entry -inf, which
    the PFC* filter can cause for a row whose label is outside the shard) has
    an empty denominator and lse = -inf; a log-sum-exp merge across shards
    then ignores it.
    """
    f = np.asarray(f, dtype=np.float64)
    mx = np.max(f, axis=1)
    empty = mx == -np.inf
    ref = np.where(empty, 0.0, mx)
    with np.errstate(divide="ignore"):
        return np.where(empty, -np.inf,
                        mx + np.log(np.sum(np.exp(f - ref[:, None]), axis=1)))


def probabilities(f, lse):
    """Softmax probabilities exp(f - lse) over each row's denominator.

    A logit outside the denominator (-inf: dropped by the PFC* filter) has
    probability 0; so does every entry of a row with an empty denominator
    (lse = -inf), which therefore gets no gradient.
    """
    f = np.asarray(f, dtype=np.float64)
    lse = np.asarray(lse, dtype=np.float64)
    live = np.isfinite(f) & np.isfinite(lse)[:, None]
    out = np.zeros(f.shape)
    out[live] = np.exp((f - np.where(np.isfinite(lse), lse, 0.0)[:, None])[live])
    return out


def forward(X, Ws, yhat, s, m, margin, tau=None):
    """Sampled margin-softmax cross-entropy of the rows given.

    Probabilities are normalised over the active set only (Eq.
    sampled_probability), and with the PFC* filter (tau < 1) over the
    unfiltered logits of each row only (Eq. noise_filtering); filtered logits
    have probability 0.  Row loss l_n = lse_n - f_{n, yhat_n} for owned rows.
    Reading: a row whose label is outside the shard has no target here and
    contributes 0 to the reported loss (its target term belongs to the owning
    shard, Sec. 3.2.1); its gradient is still P/B, the derivative of its
    log-sum-exp.  If the PFC* filter also drops every one of its logits, its
    denominator is empty: lse = -inf, P = 0, no gradient, loss term 0.  The batch mean always divides by the full batch size
    (G = (P - Y)/B, Sec. 3.2.1), which the caller applies.
    Returns dict(cos, f, lse, P, row_loss).
    """
    yhat = np.asarray(yhat, dtype=np.int64)
    cos = cosines(X, Ws)
    f = logits(cos, yhat, s, m, margin, tau)
    lse = log_sum_exp(f)
    P = probabilities(f, lse)
    own = np.nonzero(yhat >= 0)[0]
    row_loss = np.zeros(len(yhat))
    row_loss[own] = lse[own] - f[own, yhat[own]]
    return {"cos": cos, "f": f, "lse": lse, "P": P, "row_loss": row_loss}


def batch_loss(row_loss, B):
    """L = (1/B) * sum of row losses (mean over the batch, Sec. 3.2.1)."""
    return float(np.sum(row_loss) / B)


# ---------------------------------------------------------------------------
# Backward (Eq. proxy_update, Eq. pfc_center_update, Sec. 3.2.1 matrix form)
# ---------------------------------------------------------------------------

def cos_grad(cos, lse, yhat, B, s, m, margin, tau=None):
    """dL/dcos for the rows given, with lse the rows' log-sum-exp.

    dF = (P - Y)/B (Sec. 3.2.1); dcos = s * dF, times the target slope at the
    target column (margin derivative, Sec. 3.1).  Logits dropped by the PFC*
    filter do not enter the loss: their P, and so their gradient, is 0.
    """
    yhat = np.asarray(yhat, dtype=np.int64)
    f = logits(cos, yhat, s, m, margin, tau)
    dF = probabilities(f, lse)
    own = np.nonzero(yhat >= 0)[0]
    dF[own, yhat[own]] -= 1.0
    dF /= B
    dc = s * dF
    if own.size:
        dc[own, yhat[own]] *= target_logit_slope(cos[own, yhat[own]], m, margin)
    return dc


def normalise_backward(A, dAhat):
    """Gradient w.r.t. raw rows of A given the gradient w.r.t. their unit rows.

    d a = (d a_hat - a_hat (a_hat . d a_hat)) / ||a|| : the tangent-space
    projection of differentiating through normalisation (Sec. 3.1).
    """
    A = np.asarray(A, dtype=np.float64)
    nrm = row_norms(A)
    ah = A / nrm[:, None]
    radial = np.sum(ah * dAhat, axis=1)
    return (dAhat - ah * radial[:, None]) / nrm[:, None]


def grad_x(X_rows, Ws, yhat_rows, lse_rows, B, s, m, margin, tau=None):
    """dL/dx for the rows given (raw head input), summed over all active classes."""
    X_rows = np.asarray(X_rows, dtype=np.float64)
    Ws = np.asarray(Ws, dtype=np.float64)
    cos = cosines(X_rows, Ws)
    dc = cos_grad(cos, lse_rows, yhat_rows, B, s, m, margin, tau)
    wh = Ws / row_norms(Ws)[:, None]
    return normalise_backward(X_rows, dc @ wh)


def grad_w(X, Ws_cols, cols, yhat, lse, B, s, m, margin, tau=None):
    """dL/dw for the active classes `cols` (positions in S), raw row gradients.

    Contributions of all batch rows are summed (Eq. pfc_center_update), so a
    class that is the target of several rows accumulates all of them.
    """
    X = np.asarray(X, dtype=np.float64)
    Ws_cols = np.asarray(Ws_cols, dtype=np.float64)
    cols = np.asarray(cols, dtype=np.int64)
    yhat = np.asarray(yhat, dtype=np.int64)
    cos = cosines(X, Ws_cols)
    # Target columns restricted to this column subset: remap yhat into it.
    pos_in_cols = np.full(len(yhat), -1, dtype=np.int64)
    where = {int(c): i for i, c in enumerate(cols)}
    for n, t in enumerate(yhat):
        if t >= 0 and int(t) in where:
            pos_in_cols[n] = where[int(t)]
    # Rows whose target lies outside the subset still owe P/B on these columns.
    f = logits(cos, pos_in_cols, s, m, margin, tau)
    hit = np.nonzero(pos_in_cols >= 0)[0]
    dF = probabilities(f, lse)
    dF[hit, pos_in_cols[hit]] -= 1.0
    dF /= B
    dc = s * dF
    if hit.size:
        dc[hit, pos_in_cols[hit]] *= target_logit_slope(cos[hit, pos_in_cols[hit]], m, margin)
    xh = X / row_norms(X)[:, None]
    return normalise_backward(Ws_cols, dc.T @ xh)


# ---------------------------------------------------------------------------
# Lazy momentum SGD on the active rows (Sec. 3.1: unsampled centres untouched)
# ---------------------------------------------------------------------------

def round_bf16(x):
    """Round float64 values to the nearest bfloat16 (ties to even), as float64.

    8 significant bits; exponent range is not limited here (the values of
    these workloads stay far inside bfloat16's normal range).
    """
    x = np.asarray(x, dtype=np.float64)
    mant, expo = np.frexp(x)                       # x = mant * 2**expo, 0.5 <= |mant| < 1
    return np.ldexp(np.round(mant * 256.0) / 256.0, expo)   # np.round: ties to even


def round_to(x, dtype):
    """Round float64 values to the storage type ("f32", "bf16", "f16")."""
    if dtype == "f32":
        return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)
    if dtype == "f16":
        return np.asarray(x, dtype=np.float64).astype(np.float16).astype(np.float64)
    if dtype == "bf16":
        return round_bf16(x)
    raise ValueError(dtype)


def momentum_update(W, M, active, g, lr, mu, w_dtype, master=None):
    """Momentum SGD applied to the active rows only; all other rows unchanged.

    Reading (paper names momentum SGD, Sec. 4.1, without the convention):
    v <- mu * v + g ; w <- w - lr * v ; no dampening, no Nesterov, no weight
    decay.  With an fp32 master copy the step goes to the master and the
    16-bit W row is its round-to-nearest-even value; without one the new W is
    rounded to W's storage type.  Arrays are updated in place (float64).
    """
    active = np.asarray(active, dtype=np.int64)
    M[active] = mu * M[active] + g
    if master is not None:
        master[active] = round_to(master[active] - lr * M[active], "f32")
        W[active] = round_to(master[active], w_dtype)
    else:
        W[active] = round_to(W[active] - lr * M[active], w_dtype)
    M[active] = round_to(M[active], "f32")


# ---------------------------------------------------------------------------
# One whole head step
# ---------------------------------------------------------------------------

def step(X, W, M, labels, C, a, r, seed, s, m, margin, lr, mu, w_dtype,
         master=None, tau=None):
    """Sample, remap, forward, backward and the lazy update for the whole batch.

    W, M (and master) are float64 arrays updated in place.  tau < 1 turns on
    the PFC* conflict filter.  Returns a dict with active, labels_mapped, lse,
    loss, dx, g (raw-row gradient of each active class, in S order).
    """
    X = np.asarray(X, dtype=np.float64)
    B = X.shape[0]
    active, mapped, info = sample_active(labels, C, a, r, seed)
    Ws = np.asarray(W[active], dtype=np.float64)
    fw = forward(X, Ws, mapped, s, m, margin, tau)
    loss = batch_loss(fw["row_loss"], B)
    dx = grad_x(X, Ws, mapped, fw["lse"], B, s, m, margin, tau)
    g = grad_w(X, Ws, np.arange(len(active)), mapped, fw["lse"], B, s, m, margin, tau)
    momentum_update(W, M, active, g, lr, mu, w_dtype, master)
    return {"active": active, "labels_mapped": mapped, "info": info,
            "lse": fw["lse"], "row_loss": fw["row_loss"], "loss": loss,
            "P": fw["P"], "dx": dx, "g": g}
