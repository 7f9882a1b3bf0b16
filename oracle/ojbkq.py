"""Plain CPU fp64 oracle for OJBKQ's per-layer box-constrained ILS path.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import or call this module.  The GPU
library shares no code with it and never calls it.

It follows the paper step by step, slowly and in float64, on the same float32
inputs the GPU path receives:

  scales/zeros      Sec. 3.2 (Q, S, Z and the dequantised weight), Alg. 1 step 1
  Gram + damping    Alg. 1 step 2: X~^T X~ + lambda^2 I = R^T R
  relaxed solution  Alg. 1 step 3-4: R^T u = A^T t, R v = u, qbar = v / s + z,
                    with A = [X~; lambda I], t = [Y*(mu) w; lambda w] (Eq. new_obj)
                    and Y*(mu) = (1 - mu) X W + mu X~ W (Eq. jta_target)
  Babai path        Alg. 1 steps 6-10 (extended, box-clamped nearest plane)
  Klein paths       Eq. klein_prob / Alg. 3, temperature per the alpha rule
                    stated after Eq. klein_prob (K = (e rho)^(2m/rho))
  selection         Alg. 4 over the Babai path and the K Klein paths
  weight order      optional permutation of the input features (act order),
                    the extension the paper's limitations name as future
                    work, read as GPTQ's largest-diagonal-first order

Layout of the arguments is the storage layout shared with the GPU path:
W is [n, m] (row j = the paper's column w_j), X_ref and X_q are [m, T]
(the paper's X^T and X~^T).  Readings of points the paper leaves open:

  * scale/zero: asymmetric min-max over each group with the range widened to
    contain 0; an all-zero group uses [-1, 1]; the scale is stored in float32
    and that stored value is the one the decode uses; z = rint(-xmin / s).
    The symmetric Absmax variant (the calibration the paper names as an
    example): z = 2^(bits-1) and s = max|w| / (2^(bits-1) - 1) in float32,
    so that the grid s (q - z) holds +max|w| and -max|w| (all-zero group:
    max|w| = 1); it needs bits >= 2.
  * lambda^2 = lambda_rel * mean(diag(X~^T X~)) on the unnormalised Gram.
  * A^T y of Alg. 1 step 3 is A^T t_j = X~^T y*_j + lambda^2 w_j.
  * qbar = v / s + z (Alg. 1 step 4; the derivation text drops the +z).
  * Klein weight exp(-alpha * Rbar_ii^2 * (c - v)^2) over the box, with the
    squared diagonal (the form under which the alpha rule is scale-free) and
    alpha_j = ln(rho) / min_i Rbar_ii^2 taken per column on Rbar_j = R D_j.
  * candidate set: the Babai path (k = 0) plus K Klein paths; scored by the
    reduced residual ||Rbar (q - qbar)||^2 (equal to the JTA score minus the
    column's least-squares floor), first strict minimum wins.
  * rounding is round-half-to-even (numpy.rint).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional

import numpy as np
import scipy.linalg

from .philox import uniform53


class NotPositiveDefinite(ValueError):
    """The damped Gram X~^T X~ + lambda^2 I has a non-positive pivot."""


# ---------------------------------------------------------------------------
# Step 1: scales and zero points (Sec. 3.2 data model; Alg. 1 step 1)
# ---------------------------------------------------------------------------

def group_size(m: int, group: int) -> int:
    """Effective group length: ``group`` <= 0 or >= m means one group per column."""
    return m if (group <= 0 or group >= m) else group


def num_groups(m: int, group: int) -> int:
    g = group_size(m, group)
    return (m + g - 1) // g


def scales_zeros(W: np.ndarray, bits: int, group: int, scheme: str = "asym"):
    """Per (column, group) scale s and zero point z from the float32 weights.

    "asym": W_hat = S * (Q - Z) must be able to represent 0 and the group's
    extreme values, so the range is [min(w, 0), max(w, 0)] spread over the
    2^bits - 1 steps of the box.  "sym" (Absmax): the zero point is the middle
    of the box, 2^(bits-1), and the scale maps max|w| to the 2^(bits-1) - 1
    steps above it.  Returns (S, Z) as float32 [n, groups].
    """
    W = np.asarray(W)
    n, m = W.shape
    qmax = (1 << bits) - 1
    if scheme not in ("asym", "sym") or (scheme == "sym" and bits < 2):
        raise ValueError("scheme must be 'asym', or 'sym' with bits >= 2")
    g = group_size(m, group)
    G = num_groups(m, group)
    S = np.empty((n, G), dtype=np.float32)
    Z = np.empty((n, G), dtype=np.float32)
    for j in range(n):
        for t in range(G):
            w = W[j, t * g:min(m, (t + 1) * g)].astype(np.float64)
            if scheme == "sym":
                a = float(np.abs(w).max())
                if a == 0.0:
                    a = 1.0
                half = 1 << (bits - 1)
                S[j, t] = np.float32(a / (half - 1))
                Z[j, t] = half
                continue
            xmin = min(float(w.min()), 0.0)
            xmax = max(float(w.max()), 0.0)
            if xmax == xmin:
                xmin, xmax = -1.0, 1.0
            s = np.float32((xmax - xmin) / qmax)           # stored precision
            z = np.rint(-xmin / np.float64(s))
            S[j, t] = s
            Z[j, t] = z
    return S, Z


def expand_groups(A: np.ndarray, m: int, group) -> np.ndarray:
    """[n, groups] -> [n, m] by repeating each group's value over its rows.

    ``group`` is the group size, or an array giving the group of every row
    (rows of one group need not be adjacent)."""
    if np.ndim(group) == 1:
        return np.asarray(A, dtype=np.float64)[:, np.asarray(group, dtype=np.int64)]
    g = group_size(m, group)
    return np.repeat(np.asarray(A, dtype=np.float64), g, axis=1)[:, :m]


# ---------------------------------------------------------------------------
# Step 2: damped Gram and its Cholesky factor (Alg. 1 step 2)
# ---------------------------------------------------------------------------

def gram(X_q: np.ndarray) -> np.ndarray:
    """X~^T X~ in float64, with X~ = X_q^T (tokens x features)."""
    Xt = np.asarray(X_q, dtype=np.float64).T
    return Xt.T @ Xt


def damping(Gm: np.ndarray, lambda_rel: float) -> float:
    """lambda^2 = lambda_rel * mean(diag(X~^T X~))."""
    return float(lambda_rel) * float(np.mean(np.diag(Gm)))


def cholesky_upper(H: np.ndarray) -> np.ndarray:
    """Upper-triangular R with R^T R = H (Alg. 1 step 2)."""
    try:
        L = np.linalg.cholesky(H)
    except np.linalg.LinAlgError as exc:
        raise NotPositiveDefinite(str(exc)) from exc
    if not np.all(np.isfinite(L)) or np.any(np.diag(L) <= 0):
        raise NotPositiveDefinite("non-positive pivot")
    return L.T.copy()


# ---------------------------------------------------------------------------
# Steps 3-4: real least-squares solution and the real centre qbar
# ---------------------------------------------------------------------------

def jta_target(W: np.ndarray, X_ref: np.ndarray, X_q: np.ndarray, mu: float) -> np.ndarray:
    """Y*(mu) = (1 - mu) X W + mu X~ W (Eq. jta_target), tokens x n, float64."""
    Wp = np.asarray(W, dtype=np.float64).T                # paper layout: m x n
    X = np.asarray(X_ref, dtype=np.float64).T
    Xt = np.asarray(X_q, dtype=np.float64).T
    return (1.0 - mu) * (X @ Wp) + mu * (Xt @ Wp)


def relaxed_solution(W, X_ref, X_q, mu: float, lam2: float, R: np.ndarray) -> np.ndarray:
    """v_j = (A^T A)^{-1} A^T t_j for every column (Alg. 1 step 3), as [n, m].

    A^T t_j = X~^T y*_j + lambda^2 w_j; the two triangular solves
    R^T u = A^T t and R v = u use the factor of Alg. 1 step 2.
    """
    Wp = np.asarray(W, dtype=np.float64).T
    Xt = np.asarray(X_q, dtype=np.float64).T
    AtT = Xt.T @ jta_target(W, X_ref, X_q, mu) + lam2 * Wp
    U = scipy.linalg.solve_triangular(R, AtT, trans="T", lower=False)   # R^T u = A^T t
    V = scipy.linalg.solve_triangular(R, U, lower=False)                # R v = u
    return V.T.copy()


def centres(V: np.ndarray, S: np.ndarray, Z: np.ndarray, group: int) -> np.ndarray:
    """qbar = v / s + z (Alg. 1 step 4), [n, m] float64."""
    m = V.shape[1]
    return V / expand_groups(S, m, group) + expand_groups(Z, m, group)


# ---------------------------------------------------------------------------
# Klein temperature (the alpha rule stated after Eq. klein_prob)
# ---------------------------------------------------------------------------

def klein_log_rho(m: int, K: int) -> float:
    """ln(rho) where rho > 1 solves K = (e rho)^(2m / rho).

    Taking logs: ln K = (2m / rho)(1 + ln rho).  In x = ln rho the right side
    2m (1 + x) e^{-x} falls strictly from 2m at x = 0 towards 0, so for
    0 < ln K < 2m there is exactly one root; it is found by bisection.
    K <= 1 has no finite root (rho -> infinity, greedy rounding): returns inf.
    ln K >= 2m has no root above 1: returns 0 (rho = 1, flat sampling).
    """
    if K <= 1:
        return math.inf
    lnK = math.log(K)
    if lnK >= 2.0 * m:
        return 0.0

    def f(x):
        return 2.0 * m * (1.0 + x) * math.exp(-x) - lnK

    lo, hi = 0.0, 1.0
    while f(hi) > 0.0:
        lo, hi = hi, 2.0 * hi
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if mid <= lo or mid >= hi:
            break
        if f(mid) > 0.0:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def klein_alpha(R: np.ndarray, S: np.ndarray, group: int, K: int) -> np.ndarray:
    """alpha_j = ln(rho) / min_i (R_ii s_j(i))^2 per column, [n]."""
    m = R.shape[0]
    lr = klein_log_rho(m, K)
    Sx = expand_groups(S, m, group)                      # [n, m]
    rb2 = (np.diag(R)[None, :] * Sx) ** 2
    return lr / rb2.min(axis=1)


# ---------------------------------------------------------------------------
# Steps 6-10: Babai path and Klein paths (Alg. 1, Alg. 3), then Alg. 4
# ---------------------------------------------------------------------------

def klein_pick(c: np.ndarray, kappa: np.ndarray, u: np.ndarray, qmax: int) -> np.ndarray:
    """Draw q in {0..qmax} with Pr(q = v) proportional to exp(-kappa (c - v)^2).

    Inverse-CDF draw with u in [0, 1): the smallest v whose running weight
    sum exceeds u times the total.  Weights are normalised by the largest
    one before exponentiating; kappa = inf means plain nearest-point rounding.
    """
    c = np.asarray(c, dtype=np.float64)
    out = np.empty(c.shape, dtype=np.int64)
    greedy = ~np.isfinite(kappa)
    if np.any(greedy):
        out[greedy] = np.clip(np.rint(c[greedy]), 0, qmax).astype(np.int64)
    sel = ~greedy
    if np.any(sel):
        cs, ks, us = c[sel], kappa[sel], u[sel]
        v = np.arange(qmax + 1, dtype=np.float64)
        logits = -ks[:, None] * (cs[:, None] - v[None, :]) ** 2
        w = np.exp(logits - logits.max(axis=1, keepdims=True))
        cum = np.add.accumulate(w, axis=1)                # running sums, in v order
        total = cum[:, -1]
        hit = (us * total)[:, None] < cum
        first = np.argmax(hit, axis=1)
        none = ~hit.any(axis=1)
        if np.any(none):                                  # rounding corner: last v with weight
            lastpos = qmax - np.argmax((w[:, ::-1] > 0), axis=1)
            first = np.where(none, lastpos, first)
        out[sel] = first
    return out


def decode_column(R: np.ndarray, qbar: np.ndarray, s_row: np.ndarray, bits: int, K: int,
                  alpha: float, seed: int, j: int):
    """All K+1 candidate code vectors of one column.

    R: upper factor [m, m]; qbar: [m]; s_row: per-row scale [m] of this column.
    Path k = 0 rounds to the nearest box point (Alg. 1); paths k = 1..K draw
    from Eq. klein_prob (Alg. 3).  Returns codes [K+1, m] int64.
    """
    m = R.shape[0]
    qmax = (1 << bits) - 1
    Rbar = R * s_row[None, :]                            # Rbar = R D_j (Alg. 1 step 5)
    P = K + 1
    Q = np.zeros((P, m), dtype=np.int64)
    ks = np.arange(P)
    # the uniforms of every (row, Klein path) of this column, drawn up front
    U = uniform53(seed, np.arange(m)[:, None], j, ks[None, 1:]) if K > 0 else None
    for i in range(m - 1, -1, -1):
        # centre of row i from the rows already decided (Alg. 1 step 9)
        diff = qbar[i + 1:][None, :] - Q[:, i + 1:]       # [P, m - i - 1]
        c = qbar[i] + (diff @ Rbar[i, i + 1:]) / Rbar[i, i]
        q = np.clip(np.rint(c), 0, qmax).astype(np.int64)  # Babai (Alg. 1 step 10)
        if K > 0:
            kappa = np.full(K, alpha * Rbar[i, i] ** 2)
            q[1:] = klein_pick(c[1:], kappa, U[i], qmax)
        Q[:, i] = q
    return Q


def reduced_residual(R: np.ndarray, s_row: np.ndarray, q: np.ndarray, qbar: np.ndarray) -> np.ndarray:
    """||Rbar (q - qbar)||^2 for each row of q ([P, m] -> [P])."""
    Rbar = R * s_row[None, :]
    d = (np.asarray(q, dtype=np.float64) - qbar[None, :]).T   # [m, P]
    return np.sum((Rbar @ d) ** 2, axis=0)


def select_best(resid: np.ndarray) -> int:
    """Alg. 4: keep the first candidate with the strictly smallest residual."""
    best, best_r = 0, math.inf
    for k, r in enumerate(resid):
        if r < best_r:
            best, best_r = k, r
    return best


@dataclass
class DecodeResult:
    codes: np.ndarray          # [n, m] uint8, winning candidate
    residuals: np.ndarray      # [n] float64, reduced residual of the winner
    winner: np.ndarray         # [n] int32, candidate index (0 = Babai)
    path_codes: np.ndarray     # [n, K+1, m] uint8
    path_resid: np.ndarray     # [n, K+1] float64
    alpha: np.ndarray          # [n]


def decode(R: np.ndarray, qbar: np.ndarray, S: np.ndarray, bits: int, group: int, K: int,
           seed: int, columns: Optional[np.ndarray] = None) -> DecodeResult:
    """Decode every column (or the listed ``columns``) and select per Alg. 4."""
    R = np.asarray(R, dtype=np.float64)
    qbar = np.asarray(qbar, dtype=np.float64)
    m = R.shape[0]
    n = qbar.shape[0]
    cols = np.arange(n) if columns is None else np.asarray(columns)
    alpha_all = klein_alpha(R, S[cols], group, K)
    Sx = expand_groups(S[cols], m, group)
    nc = len(cols)
    path_codes = np.zeros((nc, K + 1, m), dtype=np.uint8)
    path_resid = np.zeros((nc, K + 1), dtype=np.float64)
    codes = np.zeros((nc, m), dtype=np.uint8)
    res = np.zeros(nc, dtype=np.float64)
    win = np.zeros(nc, dtype=np.int32)
    for t, j in enumerate(cols):
        Q = decode_column(R, qbar[j], Sx[t], bits, K, float(alpha_all[t]), seed, int(j))
        r = reduced_residual(R, Sx[t], Q, qbar[j])
        k = select_best(r)
        path_codes[t] = Q
        path_resid[t] = r
        codes[t] = Q[k]
        res[t] = r[k]
        win[t] = k
    return DecodeResult(codes, res, win, path_codes, path_resid, alpha_all)


# ---------------------------------------------------------------------------
# The whole layer
# ---------------------------------------------------------------------------

@dataclass
class LayerResult:
    codes: np.ndarray
    scales: np.ndarray
    zeros: np.ndarray
    residuals: np.ndarray
    winner: np.ndarray
    lam2: float = 0.0
    G: Optional[np.ndarray] = None
    R: Optional[np.ndarray] = None
    V: Optional[np.ndarray] = None
    qbar: Optional[np.ndarray] = None
    decode: Optional[DecodeResult] = None
    extra: dict = field(default_factory=dict)


def act_order_perm(Gm: np.ndarray) -> np.ndarray:
    """Decode order of the weight permutation the paper's limitations name as
    future work (the GPTQ heuristic: treat the input features with the largest
    Hessian diagonal first).

    Position p of the permuted problem holds input feature perm[p].  The
    features are sorted by increasing diag(X~^T X~), equal values by index, so
    that the decoder, which walks positions from m - 1 down to 0 (Alg. 1),
    decides the largest-diagonal features first and the rest compensate for
    them.  diag(X~^T X~) and diag(H) give the same order (H adds lambda^2 I).
    """
    return np.argsort(np.diag(np.asarray(Gm, dtype=np.float64)), kind="stable")


def feature_groups(perm: np.ndarray, group: int) -> np.ndarray:
    """Scale group of every input feature under the permutation: feature
    perm[p] belongs to group p // g (groups are runs of g decode positions)."""
    perm = np.asarray(perm)
    m = perm.shape[0]
    g = group_size(m, group)
    out = np.empty(m, dtype=np.int64)
    out[perm] = np.arange(m) // g
    return out


def dequantize_by_feature(codes, S, Z, gidx) -> np.ndarray:
    """W_hat [n, m] = s (q - z) with the group of input feature i given by
    gidx[i] (codes in the original feature order)."""
    S = np.asarray(S, dtype=np.float64)
    Z = np.asarray(Z, dtype=np.float64)
    return S[:, gidx] * (np.asarray(codes, dtype=np.float64) - Z[:, gidx])


def quantize_layer(W, X_ref, X_q, mu: float, bits: int, group: int, K: int, seed: int,
                   lambda_rel: float = 0.01, columns=None, G: Optional[np.ndarray] = None,
                   scheme: str = "asym", act_order: bool = False,
                   perm: Optional[np.ndarray] = None, static_groups: bool = False,
                   scales=None) -> LayerResult:
    """The per-layer path end to end.

    ``columns`` restricts the decode (not the scales, Gram or factor) to a
    subset of output channels; ``G`` may pass a Gram the caller already
    formed with :func:`gram` on the same X_q; ``scheme`` picks the scale and
    zero-point rule (see :func:`scales_zeros`).

    ``act_order`` (or an explicit ``perm``) solves the problem with its input
    features reordered: position p holds feature perm[p] (default order:
    :func:`act_order_perm`), scale groups are runs of g positions, and the
    returned codes are put back in the original feature order (codes[j, i]
    is the code of W[j, i]); scales and zeros are per permuted group, and
    ``extra["perm"]`` holds the order.  The other fields (G, R, V, qbar,
    decode) are those of the permuted problem.  With ``static_groups`` the
    groups stay runs of g features in W's order (the scales are those of the
    unpermuted layer) and only the decode order changes: position p then
    uses the group of feature perm[p].

    ``scales`` = (S, Z) replaces the scale rule; ``group`` may then also be
    an array with the group of every row.
    """
    W = np.asarray(W)
    if act_order or perm is not None:
        Gm = gram(X_q) if G is None else np.asarray(G)
        if perm is None:
            perm = act_order_perm(Gm)
        perm = np.asarray(perm, dtype=np.int64)
        if sorted(perm.tolist()) != list(range(W.shape[1])):
            raise ValueError("perm is not a permutation of the input features")
        Xr = None if X_ref is None else np.asarray(X_ref)[perm]
        if static_groups:
            S, Z = scales_zeros(W, bits, group, scheme)
            pos_group = perm // group_size(W.shape[1], group)
            sub = quantize_layer(W[:, perm], Xr, np.asarray(X_q)[perm], mu, bits, pos_group, K,
                                 seed, lambda_rel, columns, Gm[np.ix_(perm, perm)], scheme,
                                 scales=(S, Z))
        else:
            sub = quantize_layer(W[:, perm], Xr, np.asarray(X_q)[perm], mu, bits, group, K, seed,
                                 lambda_rel, columns, Gm[np.ix_(perm, perm)], scheme)
        codes = np.empty_like(sub.codes)
        codes[:, perm] = sub.codes
        sub.codes = codes
        sub.extra["perm"] = perm
        return sub
    S, Z = scales_zeros(W, bits, group, scheme) if scales is None else scales
    Gm = gram(X_q) if G is None else G
    lam2 = damping(Gm, lambda_rel)
    H = Gm + lam2 * np.eye(Gm.shape[0])
    R = cholesky_upper(H)
    V = relaxed_solution(W, X_ref, X_q, mu, lam2, R)
    qb = centres(V, S, Z, group)
    dec = decode(R, qb, S, bits, group, K, seed, columns)
    cols = np.arange(W.shape[0]) if columns is None else np.asarray(columns)
    return LayerResult(codes=dec.codes, scales=S, zeros=Z, residuals=dec.residuals,
                       winner=dec.winner, lam2=lam2, G=Gm, R=R, V=V, qbar=qb, decode=dec,
                       extra={"columns": cols})


def jta_score(W, X_ref, X_q, W_hat, mu: float, lam2: float) -> np.ndarray:
    """Per-column S(W_hat) = ||X~ w_hat - y*||^2 + lambda^2 ||w_hat - w||^2 (Eq. jta_score)."""
    Wp = np.asarray(W, dtype=np.float64).T
    Whp = np.asarray(W_hat, dtype=np.float64).T
    Xt = np.asarray(X_q, dtype=np.float64).T
    Ys = jta_target(W, X_ref, X_q, mu)
    return np.sum((Xt @ Whp - Ys) ** 2, axis=0) + lam2 * np.sum((Whp - Wp) ** 2, axis=0)


def dequantize(codes, S, Z, group: int) -> np.ndarray:
    """W_hat = S * (Q - Z) in the [n, m] layout."""
    m = codes.shape[1]
    return expand_groups(S, m, group) * (np.asarray(codes, dtype=np.float64) - expand_groups(Z, m, group))
