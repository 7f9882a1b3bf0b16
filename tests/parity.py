"""Helpers that compare the HIP path with the CPU oracle on the same inputs.

The parity bar (applied element by element, :func:`check_paths_strict`):
  * scales and zero points: within 1e-6 relative (the implementation is in
    fact bit-exact: both sides take the same float64 steps);
  * codes: at least 99.9% of the entries of every candidate path equal, and
    every differing path explained by a near-tie: replaying the path with the
    GPU's own earlier codes, the GPU's pick at the first difference must be
    reproducible with the centre moved by at most 1e-5 (Babai: |c - floor(c)|
    within 1e-5 of 0.5; Klein: the same shift of c, or u within 1e-6 of a CDF
    boundary);
  * residuals: every GPU candidate residual within 1e-4 relative of the
    oracle's residual formula applied to the GPU's own codes of that
    candidate, and of the oracle's candidate where the codes agree;
  * selection: the GPU's winner is the first strict minimum of its own
    candidate residuals; where it differs from the oracle's winner, one of
    the two paths diverged at a near-tie or their oracle residuals agree to
    1e-4 (a residual tie); the winning residual agrees to 1e-4 unless one of
    the two paths diverged at a near-tie.
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

# Relative error of the token sums X~^T X~ and X~^T (X - X~), and of what
# follows from them to first order (lambda^2, the factor, matrix-free probes,
# the Gram diagonal that orders act-order features), by the arithmetic of the
# Gram stage (ojbkq_params.gram_fp64):
#   int8: every value is kept to 28 bits below its row's power-of-two maximum
#     2^e (error <= 2^(e-28)), so a product x_i x_j loses at most about
#     2^-27 2^(e_i + e_j) per token, with random signs over the tokens: about
#     sqrt(T) 2^-27 2^(e_i + e_j) in all, measured 1e-10 to 5e-10 of
#     sqrt(G_ii G_jj) on these workloads; 1e-8 leaves a 20x margin;
#   fp64: exact products, float64 sums.
GRAM_RTOL = {"int8": 1e-8, "fp64": 1e-11}
# the same for quantities that go through a solve with H (Rbar qbar, whose
# cross-term part is L^-1 E w, the centres, candidate residuals): the above
# amplified by at most the conditioning of H, measured up to 2.3e-8 relative
# for int8
SOLVE_RTOL = {"int8": 1e-6, "fp64": 1e-9}


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


def first_strict_min(r):
    best, br = 0, r[0]
    for k in range(1, len(r)):
        if r[k] < br:
            best, br = k, r[k]
    return best


def check_paths_strict(R, qbar, s_rows, bits, seed, alpha, cols, gpu_paths, gpu_presid,
                       gpu_codes, gpu_res, gpu_win, orc_paths, orc_presid, orc_res, orc_win,
                       tag=""):
    """The full parity rule on every candidate of the given columns.

    R [m, m] upper factor and qbar [c, m], s_rows [c, m] (each row's scale in
    decode order), alpha [c] of the oracle; cols [c] the column indices (for
    the Philox counters); gpu_paths / orc_paths [c, K+1, m] and gpu_codes
    [c, m] in decode order; residuals [c, K+1] and [c]; winners [c].
    Returns a dict of counts and worst errors.
    """
    c, P, m = orc_paths.shape
    same = gpu_paths == orc_paths
    frac = float(same.mean())
    diverged = ~same.all(axis=2)                                  # [c, P]
    ties = 0
    worst_same = 0.0
    worst_eval = 0.0
    win_mis = res_tie = 0
    for t in range(c):
        j = int(cols[t])
        r_eval = orc.reduced_residual(R, s_rows[t], gpu_paths[t], qbar[t])
        rel_e = np.abs(gpu_presid[t] - r_eval) / np.maximum(r_eval, 1e-300)
        worst_eval = max(worst_eval, float(rel_e.max()))
        assert rel_e.max() <= RESID_RTOL, \
            f"{tag} column {j}: GPU candidate residuals off the oracle's formula by {rel_e.max():.2e}"
        for k in range(P):
            if diverged[t, k]:
                assert first_divergence_is_tie(R, qbar[t], s_rows[t], bits, alpha[t], seed, j, k,
                                               gpu_paths[t, k], orc_paths[t, k]), \
                    f"{tag} column {j} path {k}: difference is not a near-tie"
                ties += 1
            else:
                rel = abs(gpu_presid[t, k] - orc_presid[t, k]) / max(orc_presid[t, k], 1e-300)
                worst_same = max(worst_same, rel)
                assert rel <= RESID_RTOL, f"{tag} column {j} path {k}: residual rel err {rel:.2e}"
        kg, ko = int(gpu_win[t]), int(orc_win[t])
        assert kg == first_strict_min(gpu_presid[t]), f"{tag} column {j}: winner is not the first minimum"
        assert np.array_equal(gpu_codes[t], gpu_paths[t, kg]), f"{tag} column {j}: winner codes"
        assert gpu_res[t] == gpu_presid[t, kg], f"{tag} column {j}: winner residual"
        involved = diverged[t, kg] or diverged[t, ko]
        if kg != ko:
            win_mis += 1
            rtie = abs(orc_presid[t, kg] - orc_presid[t, ko]) <= RESID_RTOL * orc_presid[t, ko]
            res_tie += int(rtie)
            assert involved or rtie, \
                f"{tag} column {j}: winner {kg} vs oracle {ko} without a near-tie"
        if not involved:
            rel = abs(gpu_res[t] - orc_res[t]) / max(orc_res[t], 1e-300)
            assert rel <= RESID_RTOL, f"{tag} column {j}: winning residual rel err {rel:.2e}"
    assert frac >= CODE_AGREEMENT, f"{tag} code agreement {frac:.6f} < {CODE_AGREEMENT}"
    out = {"agreement": frac, "tie_paths": ties, "winner_mismatch": win_mis,
           "residual_ties": res_tie, "worst_same": worst_same, "worst_eval": worst_eval}
    print(f"[{tag}] paths {c}x{P}: code agreement {frac:.6f}, near-tie paths {ties}, winner "
          f"mismatches {win_mis} ({res_tie} residual ties), worst candidate residual rel err "
          f"{worst_same:.2e} (same codes), {worst_eval:.2e} (oracle formula on GPU codes)",
          flush=True)
    return out


def check_layer_strict(o, gpu, gpu_paths_w, gpu_presid, bits, seed, group_rows, perm=None,
                       tag=""):
    """check_paths_strict for a whole-layer oracle result ``o`` (every column
    the oracle decoded, o.extra["columns"]).  gpu: a QuantResult; gpu_paths_w
    [n, K+1, m] and gpu_presid [n, K+1] from the staged calls, codes in W's
    feature order; group_rows: the oracle's group argument for the decode
    order (size or per-position array); perm: the decode order or None."""
    cols = np.asarray(o.extra["columns"])
    m = o.R.shape[0]
    codes_w = np64(gpu.codes)[cols]
    paths_w = gpu_paths_w[cols]
    if perm is not None:
        paths = paths_w[:, :, perm]
        codes = codes_w[:, perm]
    else:
        paths, codes = paths_w, codes_w
    s_rows = orc.expand_groups(o.scales[cols], m, group_rows)
    return check_paths_strict(o.R, o.qbar[cols], s_rows, bits, seed, o.decode.alpha, cols,
                              paths, gpu_presid[cols], codes, np64(gpu.residuals)[cols],
                              np64(gpu.winner)[cols], o.decode.path_codes,
                              o.decode.path_resid, o.residuals, o.winner, tag=tag)
