"""Helpers that compare the HIP path with the CPU oracle on the same inputs.

The parity bar (applied element by element):
  * scales and zero points: within 1e-6 relative (the implementation is in
    fact bit-exact: both sides take the same float64 steps);
  * codes: at least 99.9% of entries equal, and every differing path explained
    by a near-tie: replaying the path with the GPU's own earlier codes, the
    GPU's pick at the first difference must be reproducible with the centre
    moved by at most 1e-5 (Babai: |c - floor(c)| within 1e-5 of 0.5; Klein:
    the same shift of c, or u within 1e-6 of a CDF boundary);
  * residuals: within 1e-4 relative for columns with the same winner.
"""

from __future__ import annotations

import math

import numpy as np

from oracle import ojbkq as orc
from oracle.philox import uniform53

CODE_AGREEMENT = 0.999
RESID_RTOL = 1e-4
SCALE_RTOL = 1e-6
TIE_BAND = 1e-5
U_BAND = 1e-6


def np64(t):
    return t.detach().cpu().numpy()


def centres_from_gq(L, gq_rows, S_rows, group):
    """The real centres behind the decoder's input rows.

    Row j of gq is Rbar_j qbar_j = R (s_j qbar_j) written as a row,
    (s_j qbar_j)^T L with L = R^T; so s_j qbar_j = L^-T gq_j (one host
    triangular solve per row) and qbar_j follows by dividing by the scales.
    """
    import scipy.linalg
    m = L.shape[0]
    v = scipy.linalg.solve_triangular(L, np.asarray(gq_rows, dtype=np.float64).T, lower=True,
                                      trans="T", check_finite=False).T
    return v / orc.expand_groups(S_rows, m, group)


def _pick_range(c, kappa, u, qmax):
    """Set of codes reachable by moving c within the tie band or u within U_BAND."""
    picks = set()
    for dc in (-TIE_BAND, 0.0, TIE_BAND):
        for du in (-U_BAND, 0.0, U_BAND):
            uu = min(max(u + du, 0.0), 1.0 - 1e-17)
            if math.isinf(kappa):
                picks.add(int(np.clip(np.rint(c + dc), 0, qmax)))
            else:
                picks.add(int(orc.klein_pick(np.array([c + dc]), np.array([kappa]),
                                             np.array([uu]), qmax)[0]))
    return picks


def first_divergence_is_tie(R, qbar_j, s_row, bits, alpha_j, seed, j, k, gpu_path, oracle_path):
    """Replay one path with the GPU's own codes; True if the first difference is a near-tie."""
    qmax = (1 << bits) - 1
    m = len(qbar_j)
    Rbar = R * s_row[None, :]
    diff = np.nonzero(gpu_path != oracle_path)[0]
    if len(diff) == 0:
        return True
    i = int(diff.max())                      # rows are decided from m-1 down: first difference
    q = gpu_path.astype(np.float64)
    c = qbar_j[i] + (Rbar[i, i + 1:] @ (qbar_j[i + 1:] - q[i + 1:])) / Rbar[i, i]
    kappa = math.inf if k == 0 else alpha_j * Rbar[i, i] ** 2
    u = 0.5 if k == 0 else float(uniform53(seed, i, j, k))
    return int(gpu_path[i]) in _pick_range(c, kappa, u, qmax)


def check_paths(R, qbar, S, group, bits, K, seed, alpha, gpu_paths, oracle_paths, cols=None):
    """Path-by-path code parity.  Returns (agreement fraction, #tie-explained paths)."""
    n, P, m = oracle_paths.shape
    cols = np.arange(n) if cols is None else np.asarray(cols)
    Sx = orc.expand_groups(S, m, group)
    same = gpu_paths == oracle_paths
    frac = float(same.mean())
    ties = 0
    for t in range(n):
        for k in range(P):
            if not same[t, k].all():
                assert first_divergence_is_tie(R, qbar[t], Sx[t], bits, alpha[t], seed,
                                               int(cols[t]), k, gpu_paths[t, k],
                                               oracle_paths[t, k]), \
                    f"column {cols[t]} path {k}: difference is not a near-tie"
                ties += 1
    assert frac >= CODE_AGREEMENT, f"code agreement {frac:.6f} < {CODE_AGREEMENT}"
    return frac, ties


def check_residuals(gpu_res, gpu_win, orc_res, orc_win):
    same = gpu_win == orc_win
    rel = np.abs(gpu_res[same] - orc_res[same]) / np.maximum(np.abs(orc_res[same]), 1e-300)
    worst = float(rel.max()) if rel.size else 0.0
    assert worst <= RESID_RTOL, f"residual rel error {worst:.3e}"
    return worst, int((~same).sum())
