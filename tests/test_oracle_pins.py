"""Pins for the CPU oracle: hand-worked examples, closed forms, brute force and invariants.

Each check is chosen so a plausible slip in the oracle (a dropped term, a sign,
an index, a transposed operand, a missing square) makes at least one fail.
"""

import itertools
import math

import numpy as np
import pytest

from oracle import ojbkq as o


# ---------------------------------------------------------------------------
# helpers written independently of the oracle's decode loop
# ---------------------------------------------------------------------------

def brute_force_opt(Rbar, qbar, qmax):
    """Exact box-constrained ILS optimum by enumerating every box point."""
    m = len(qbar)
    pts = np.array(list(itertools.product(range(qmax + 1), repeat=m)), dtype=np.float64)
    r = np.sum(((pts - qbar[None, :]) @ Rbar.T) ** 2, axis=1)
    k = int(np.argmin(r))
    return pts[k].astype(int), float(r[k])


def centres_from_codes(Rbar, qbar, q):
    """c_i = qbar_i + sum_{l>i} Rbar_il (qbar_l - q_l) / Rbar_ii, for given codes q."""
    m = len(qbar)
    c = np.empty(m)
    for i in range(m):
        acc = 0.0
        for l in range(i + 1, m):
            acc += Rbar[i, l] * (qbar[l] - q[l])
        c[i] = qbar[i] + acc / Rbar[i, i]
    return c


def random_upper(rng, m, cond=1.0):
    A = rng.standard_normal((m + 3, m)) * np.exp(cond * rng.standard_normal(m))[None, :]
    return o.cholesky_upper(A.T @ A + 0.05 * np.eye(m))


# ---------------------------------------------------------------------------
# scales and zeros
# ---------------------------------------------------------------------------

def test_scale_zero_hand_worked(golden):
    g = golden("hand_worked_3x3.txt")
    W = np.array([g["scale_w"]], dtype=np.float32)
    S, Z = o.scales_zeros(W, 2, 128)
    assert S.shape == (1, 1)
    assert abs(S[0, 0] - g["scale_s"][0]) < 1e-7
    assert Z[0, 0] == g["scale_z"][0]


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_scale_zero_properties(bits):
    rng = np.random.default_rng(bits)
    qmax = 2 ** bits - 1
    m, group = 200, 128                      # ragged last group of 72
    W = (rng.standard_normal((9, m)) * 0.02).astype(np.float32)
    W[1] = np.abs(W[1])                      # all >= 0: xmin forced to 0
    W[2] = -np.abs(W[2])                     # all <= 0: xmax forced to 0
    W[3, :128] = 0.0                         # degenerate group
    S, Z = o.scales_zeros(W, bits, group)
    assert S.shape == (9, 2) and S.dtype == np.float32
    assert np.all(Z == np.rint(Z)) and np.all(Z >= 0) and np.all(Z <= qmax)
    assert S[3, 0] == np.float32(2.0 / qmax) and Z[3, 0] == np.rint((1.0) / np.float64(np.float32(2.0 / qmax)))
    for j in range(9):
        for t, (a, b) in enumerate([(0, 128), (128, 200)]):
            w = W[j, a:b].astype(np.float64)
            s, z = float(S[j, t]), float(Z[j, t])
            lo, hi = min(w.min(), 0.0), max(w.max(), 0.0)
            if lo == hi:
                continue
            # the grid s * (v - z), v in the box, covers [lo, hi] to within half a step
            assert s * (0 - z) <= lo + 0.5 * s + 1e-12
            assert s * (qmax - z) >= hi - 0.5 * s - 1e-12
            assert abs(s - (hi - lo) / qmax) <= 1e-7 * s
    S1, _ = o.scales_zeros(W, bits, 0)       # group <= 0: one group per column
    assert S1.shape == (9, 1)
    S2, _ = o.scales_zeros(W, bits, 10 ** 6)
    assert np.array_equal(S1, S2)


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_symmetric_absmax_scale_zero(bits):
    """Absmax: the box middle is the zero point and +-max|w| lie on the grid;
    the rule is odd in w (a sign flip keeps s and z) and commutes with
    power-of-two rescaling."""
    rng = np.random.default_rng(40 + bits)
    half = 2 ** (bits - 1)
    m, group = 200, 128
    W = (rng.standard_normal((7, m)) * 0.02).astype(np.float32)
    W[3, :128] = 0.0
    S, Z = o.scales_zeros(W, bits, group, "sym")
    assert S.dtype == np.float32 and np.all(Z == half)
    assert S[3, 0] == np.float32(1.0 / (half - 1))                  # all-zero group: max|w| = 1
    for j in range(7):
        for t, (a, b) in enumerate([(0, 128), (128, 200)]):
            amax = float(np.abs(W[j, a:b]).max())
            if amax == 0.0:
                continue
            s = float(S[j, t])
            # +max|w| at v = 2 half - 1 and -max|w| at v = 1, to float32 rounding of s
            assert abs(s * (half - 1) - amax) <= (half - 1) * 2.0 ** -24 * s
            # every weight rounds onto the box with at most half a step of error
            v = np.rint(W[j, a:b].astype(np.float64) / s + half)
            assert v.min() >= 0 and v.max() <= 2 * half - 1
            assert np.max(np.abs(s * (v - half) - W[j, a:b])) <= 0.5 * s * (1 + 1e-6)
    Sn, Zn = o.scales_zeros(-W, bits, group, "sym")
    assert np.array_equal(Sn, S) and np.array_equal(Zn, Z)
    S4, _ = o.scales_zeros(4 * W, bits, group, "sym")
    nz = np.abs(W[:, :128]).max(axis=1) > 0
    assert np.array_equal(S4[nz, 0], 4 * S[nz, 0])
    with pytest.raises(ValueError):
        o.scales_zeros(W, 1, group, "sym")


def test_symmetric_scales_through_the_layer():
    """With the problem separated (orthogonal activations, mu = 1) Babai is
    RTN on the symmetric grid as well, and the optimum."""
    rng = np.random.default_rng(5)
    m, n, T = 6, 4, 6
    Xq = np.diag(np.exp(rng.standard_normal(m))).astype(np.float32) @ np.eye(m, T, dtype=np.float32)
    W = (rng.standard_normal((n, m)) * 0.3).astype(np.float32)
    res = o.quantize_layer(W, Xq, Xq, 1.0, 2, 128, 3, 0, lambda_rel=0.0, scheme="sym")
    assert np.all(res.zeros == 2)
    rtn = np.clip(np.rint(W / res.scales.astype(np.float64) + 2), 0, 3)
    assert np.array_equal(res.codes, rtn.astype(np.uint8))
    for j in range(n):
        Rb = res.R * o.expand_groups(res.scales[j:j + 1], m, 128)[0][None, :]
        _, r_opt = brute_force_opt(Rb, res.qbar[j], 3)
        assert abs(res.residuals[j] - r_opt) <= 1e-9 * max(1, r_opt)


# ---------------------------------------------------------------------------
# Klein temperature: K = (e rho)^(2m / rho)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("m,K", [(3, 4), (8, 16), (128, 4), (4096, 5), (4096, 16), (4096, 25),
                                 (5120, 32), (11008, 16), (28672, 16), (2, 50)])
def test_rho_solves_defining_equation(m, K):
    x = o.klein_log_rho(m, K)
    rho = math.exp(x)
    assert rho > 1.0
    # K = (e rho)^(2m/rho)  <=>  ln K = (2m/rho)(1 + ln rho)
    assert abs((2.0 * m / rho) * (1.0 + x) - math.log(K)) <= 1e-12 * math.log(K)


def test_rho_limits():
    assert o.klein_log_rho(100, 1) == math.inf        # K = 1: greedy rounding
    assert o.klein_log_rho(100, 0) == math.inf
    assert o.klein_log_rho(1, 10) == 0.0              # ln K >= 2m: flat sampling
    a = [o.klein_log_rho(512, K) for K in (2, 4, 16, 64, 1024)]
    assert all(x > y for x, y in zip(a, a[1:]))       # more samples -> flatter


def test_alpha_uses_scaled_diagonal():
    R = np.diag([2.0, 1.0, 4.0]) + np.triu(np.ones((3, 3)), 1) * 0.1
    S = np.array([[0.5], [2.0]], dtype=np.float32)
    a = o.klein_alpha(R, S, 128, 4)
    lr = o.klein_log_rho(3, 4)
    # min over i of (R_ii s)^2: column 0 -> (1 * 0.5)^2, column 1 -> (1 * 2)^2
    assert np.allclose(a, [lr / 0.25, lr / 4.0], rtol=1e-15)


# ---------------------------------------------------------------------------
# Babai path: hand-worked, brute force, closed forms
# ---------------------------------------------------------------------------

def test_babai_hand_worked(golden):
    g = golden("hand_worked_3x3.txt")
    R = np.array(g["decode_R"]).reshape(3, 3)
    qbar = np.array(g["decode_qbar"])
    Q = o.decode_column(R, qbar, np.ones(3), 2, 0, 0.0, 0, 0)
    assert Q.tolist() == [[int(v) for v in g["decode_babai"]]]
    r = o.reduced_residual(R, np.ones(3), Q, qbar)
    assert abs(r[0] - g["decode_babai_residual"][0]) < 1e-12
    q_opt, r_opt = brute_force_opt(R, qbar, 3)
    assert q_opt.tolist() == [int(v) for v in g["decode_opt"]]
    assert abs(r_opt - g["decode_opt_residual"][0]) < 1e-12


def test_babai_steps_are_nearest_plane():
    """Every Babai code is the clamped rounding of the centre its predecessors imply."""
    rng = np.random.default_rng(3)
    for trial in range(20):
        m = 12
        R = random_upper(rng, m)
        s = np.exp(rng.standard_normal(m) * 0.3)
        qbar = rng.uniform(-2, 6, m)
        q = o.decode_column(R, qbar, s, 2, 0, 0.0, 0, 0)[0]
        c = centres_from_codes(R * s[None, :], qbar, q)
        assert np.array_equal(q, np.clip(np.rint(c), 0, 3))
        # residual identity: ||Rbar (q - qbar)||^2 = sum_i (Rbar_ii (q_i - c_i))^2
        Rb = R * s[None, :]
        lhs = o.reduced_residual(R, s, q[None, :], qbar)[0]
        rhs = np.sum((np.diag(Rb) * (q - c)) ** 2)
        assert abs(lhs - rhs) <= 1e-10 * max(1.0, rhs)


def test_brute_force_bounds_and_best_of_k():
    rng = np.random.default_rng(7)
    hits, inst = 0, 0
    for trial in range(12):
        m = 6
        R = random_upper(rng, m, cond=0.7)
        s = np.ones(m)
        qbar = rng.uniform(-0.5, 3.5, m)
        q_opt, r_opt = brute_force_opt(R, qbar, 3)
        K = 400
        alpha = o.klein_alpha(R, np.ones((1, 1), np.float32), 128, K)[0]
        Q = o.decode_column(R, qbar, s, 2, K, alpha, 99, trial)
        r = o.reduced_residual(R, s, Q, qbar)
        assert np.all(Q >= 0) and np.all(Q <= 3)
        assert np.all(r >= r_opt - 1e-12)                  # nothing beats the optimum
        assert r[0] >= r_opt - 1e-12
        k = o.select_best(r)
        assert r[k] <= r[0]                                 # chosen never worse than Babai
        inst += 1
        hits += int(abs(r[k] - r_opt) <= 1e-12)
    assert hits >= 9, f"best of 400 Klein samples found the optimum on {hits}/{inst} instances"


def test_diagonal_gram_babai_is_rtn_and_optimal():
    """Orthogonal activation columns + mu = 1: the problem separates, Babai = RTN = optimum."""
    rng = np.random.default_rng(2)
    m, n, T = 6, 5, 6
    Xq = np.diag(np.exp(rng.standard_normal(m))).astype(np.float32) @ np.eye(m, T, dtype=np.float32)
    W = (rng.standard_normal((n, m)) * 0.3).astype(np.float32)
    res = o.quantize_layer(W, Xq, Xq, 1.0, 2, 128, 0, 0, lambda_rel=0.0)
    S, Z = res.scales, res.zeros
    rtn = np.clip(np.rint(W / S.astype(np.float64) + Z), 0, 3)
    assert np.array_equal(res.codes, rtn.astype(np.uint8))
    for j in range(n):
        Rb = res.R * o.expand_groups(S[j:j + 1], m, 128)[0][None, :]
        _, r_opt = brute_force_opt(Rb, res.qbar[j], 3)
        assert abs(res.residuals[j] - r_opt) <= 1e-9 * max(1, r_opt)


# ---------------------------------------------------------------------------
# Klein paths: the sampler draws from Eq. klein_prob
# ---------------------------------------------------------------------------

def exact_path_probs(Rbar, qbar, kappa_scale, qmax):
    """Probability of every code vector under sequential Klein sampling (enumerated)."""
    m = len(qbar)
    probs = {}
    for q in itertools.product(range(qmax + 1), repeat=m):
        q = np.array(q)
        p = 1.0
        for i in range(m - 1, -1, -1):
            c = qbar[i] + sum(Rbar[i, l] * (qbar[l] - q[l]) for l in range(i + 1, m)) / Rbar[i, i]
            w = np.array([math.exp(-kappa_scale * Rbar[i, i] ** 2 * (c - v) ** 2) for v in range(qmax + 1)])
            p *= w[q[i]] / w.sum()
        probs[tuple(q)] = p
    return probs


def test_klein_distribution_matches_eq_klein_prob(golden):
    g = golden("hand_worked_3x3.txt")
    R = np.array(g["decode_R"]).reshape(3, 3)
    qbar = np.array(g["decode_qbar"])
    K = 4
    alpha = o.klein_log_rho(3, K) / 1.0       # min Rbar_ii^2 = 1
    exact = exact_path_probs(R, qbar, alpha, 3)
    assert abs(sum(exact.values()) - 1.0) < 1e-12
    N = 20000
    counts = {}
    for t in range(N // 50):
        Q = o.decode_column(R, qbar, np.ones(3), 2, 50, alpha, 1000 + t, 0)[1:]
        for q in map(tuple, Q):
            counts[q] = counts.get(q, 0) + 1
    # chi-square over the cells with expected count >= 20, rest pooled
    chi2, dof, pooled_e, pooled_o = 0.0, -1, 0.0, 0
    for q, p in exact.items():
        e = p * N
        if e >= 20:
            chi2 += (counts.get(q, 0) - e) ** 2 / e
            dof += 1
        else:
            pooled_e += e
            pooled_o += counts.get(q, 0)
    if pooled_e > 0:
        chi2 += (pooled_o - pooled_e) ** 2 / pooled_e
        dof += 1
    # 99.9% quantile of chi2 with ~dof degrees of freedom is below dof + 4.5 sqrt(2 dof) + 10
    assert chi2 < dof + 4.5 * math.sqrt(2 * dof) + 10, (chi2, dof)
    # the most likely path is the Babai point
    assert max(exact, key=exact.get) == (0, 0, 1)


def test_klein_greedy_limit_is_babai():
    rng = np.random.default_rng(4)
    R = random_upper(rng, 10)
    qbar = rng.uniform(-1, 4, 10)
    Q = o.decode_column(R, qbar, np.ones(10), 2, 6, math.inf, 5, 0)
    assert all(np.array_equal(Q[0], Q[k]) for k in range(1, 7))
    # K = 1 gives alpha = inf through the rho rule (the paper's greedy limit)
    assert np.all(~np.isfinite(o.klein_alpha(R, np.ones((1, 1), np.float32), 128, 1)))


def test_klein_flat_limit_is_uniform():
    u = np.linspace(0, 1, 64, endpoint=False) + 1.0 / 128
    q = o.klein_pick(np.full(64, 1.3), np.zeros(64), u, 3)
    assert np.bincount(q, minlength=4).tolist() == [16, 16, 16, 16]


def test_klein_pick_far_outside_box():
    q = o.klein_pick(np.array([-50.0, 80.0]), np.array([3.0, 3.0]), np.array([0.999, 0.5]), 7)
    assert q.tolist() == [0, 7]
    # u = 0 takes the first value with a non-zero weight: here v = 6 (weight e^-441 vs 1)
    assert o.klein_pick(np.array([80.0]), np.array([3.0]), np.array([0.0]), 7).tolist() == [6]


# ---------------------------------------------------------------------------
# whole layer: relaxed solution, JTA score and selection
# ---------------------------------------------------------------------------

def small_layer(seed, m=10, n=4, T=40, mu=0.5):
    rng = np.random.default_rng(seed)
    sig = np.exp(rng.standard_normal(m))
    Xr = (rng.standard_normal((m, T)) * sig[:, None]).astype(np.float32)
    Xq = (Xr + 0.1 * rng.standard_normal((m, T)) * sig[:, None]).astype(np.float32)
    W = (0.05 * rng.standard_normal((n, m))).astype(np.float32)
    return W, Xr, Xq


def test_layer_hand_worked(golden):
    g = golden("hand_worked_3x3.txt")
    W = np.array([g["layer_W"]], dtype=np.float32)
    Xq = np.array(g["layer_Xq"], dtype=np.float32).reshape(3, 3)
    res = o.quantize_layer(W, Xq, Xq, 1.0, 2, 128, 0, 0, lambda_rel=0.0)
    assert np.allclose(res.qbar[0], g["layer_qbar"], atol=5e-7)
    assert res.codes[0].tolist() == [int(v) for v in g["layer_codes"]]
    assert abs(res.residuals[0] - g["layer_residual"][0]) < 5e-7


@pytest.mark.parametrize("tag,mu", [("mu05", 0.5), ("mu0", 0.0)])
def test_damped_layer_hand_worked(golden, tag, mu):
    """The 3x3 layer with damping (lambda_rel = 0.01) and a cross term
    (X_ref = X_q + 0.1 I), worked by hand in the golden file: lambda^2 as
    lambda_rel times the mean Gram diagonal (Alg. 1 step 2), the factor, the
    relaxed solution through A^T t (Alg. 1 steps 3-4), the Babai codes and the
    reduced residual, and the JTA score minus its floor.  A damping taken from
    the trace, from lambda_rel^2 or from a 1/T-normalised Gram moves lambda^2
    and the residual far outside these tolerances."""
    g = golden("hand_worked_3x3.txt")
    W = np.array([g["layer_W"]], dtype=np.float32)
    Xq = np.array(g["layer_Xq"], dtype=np.float32).reshape(3, 3)
    Xr = (Xq + np.float32(g["damped_delta"][0]) * np.eye(3, dtype=np.float32)).astype(np.float32)
    res = o.quantize_layer(W, Xr, Xq, mu, 2, 128, 0, 0, lambda_rel=0.01)
    assert abs(res.lam2 - g["damped_lam2"][0]) <= 1e-9
    assert np.allclose(res.R, np.array(g["damped_R"]).reshape(3, 3), atol=5e-7, rtol=0)
    assert np.allclose(res.V[0], g[f"damped_{tag}_v"], atol=5e-7, rtol=0)
    assert np.allclose(res.qbar[0], g[f"damped_{tag}_qbar"], atol=5e-7, rtol=0)
    assert res.codes[0].tolist() == [int(v) for v in g[f"damped_{tag}_codes"]]
    assert abs(res.residuals[0] - g[f"damped_{tag}_residual"][0]) < 5e-7
    What = o.dequantize(res.codes, res.scales, res.zeros, 128)
    full = o.jta_score(W, Xr, Xq, What, mu, res.lam2)[0]
    floor = o.jta_score(W, Xr, Xq, res.V, mu, res.lam2)[0]
    assert abs(full - g[f"damped_{tag}_jta"][0]) < 5e-7
    assert abs(floor - g[f"damped_{tag}_floor"][0]) < 5e-8


def test_select_best_strict_minimum():
    """Alg. 4 keeps a candidate only when its residual is strictly smaller, so
    among equal minima the lowest index wins."""
    assert o.select_best(np.array([0.5, 0.3, 0.3, 0.4])) == 1
    assert o.select_best(np.array([0.2, 0.2, 0.2])) == 0
    assert o.select_best(np.array([0.9, 0.4, 0.7, 0.4, 0.1, 0.1])) == 4
    assert o.select_best(np.array([7.0])) == 0


def test_exact_residual_tie_keeps_babai(golden):
    """m = 1, qbar = 1.5 on the box {0..3}: Babai (half-to-even) gives 2, and
    every Klein draw of 1 or 2 ties with it exactly at 0.25; the winner is the
    Babai candidate."""
    g = golden("hand_worked_3x3.txt")
    R = np.ones((1, 1))
    qbar = np.array([[g["tie_qbar"][0]]])
    dec = o.decode(R, qbar, np.ones((1, 1), np.float32), 2, 128, 8, 5)
    r = dec.path_resid[0]
    assert dec.path_codes[0, 0, 0] == 2
    assert r[0] == g["tie_residual"][0]
    ties = [k for k in range(1, 9) if r[k] == r[0]]
    assert ties, "no Klein candidate tied with Babai"
    assert any(dec.path_codes[0, k, 0] == 1 for k in ties)       # a different point, same residual
    assert dec.winner[0] == int(g["tie_winner"][0]) and dec.residuals[0] == 0.25


@pytest.mark.parametrize("mu", [0.0, 0.3, 1.0])
def test_relaxed_solution_is_stacked_least_squares(mu):
    """v_j minimises ||[X~; lambda I] v - [y*_j; lambda w_j]|| (Eq. new_obj), via lstsq."""
    W, Xr, Xq = small_layer(1, mu=mu)
    lam2 = o.damping(o.gram(Xq), 0.01)
    R = o.cholesky_upper(o.gram(Xq) + lam2 * np.eye(W.shape[1]))
    V = o.relaxed_solution(W, Xr, Xq, mu, lam2, R)
    Xt = Xq.astype(np.float64).T
    A = np.vstack([Xt, math.sqrt(lam2) * np.eye(W.shape[1])])
    Ys = (1 - mu) * (Xr.astype(np.float64).T @ W.T.astype(np.float64)) + mu * (Xt @ W.T.astype(np.float64))
    Tm = np.vstack([Ys, math.sqrt(lam2) * W.T.astype(np.float64)])
    V_ls = np.linalg.lstsq(A, Tm, rcond=None)[0].T
    assert np.allclose(V, V_ls, rtol=1e-9, atol=1e-12)
    if mu == 1.0:
        assert np.allclose(V, W.astype(np.float64), rtol=1e-10, atol=1e-13)


def test_jta_score_minus_floor_is_reduced_residual():
    W, Xr, Xq = small_layer(2)
    mu, K = 0.5, 5
    res = o.quantize_layer(W, Xr, Xq, mu, 3, 4, K, 17, lambda_rel=0.01)
    What = o.dequantize(res.codes, res.scales, res.zeros, 4)
    full = o.jta_score(W, Xr, Xq, What, mu, res.lam2)
    floor = o.jta_score(W, Xr, Xq, res.V, mu, res.lam2)
    assert np.allclose(full - floor, res.residuals, rtol=1e-7, atol=1e-12)
    # and over every candidate: the argmin of the full JTA score is the chosen one
    for j in range(W.shape[0]):
        scores = [o.jta_score(W[j:j + 1], Xr, Xq,
                              o.dequantize(res.decode.path_codes[j, k][None, :], res.scales[j:j + 1],
                                           res.zeros[j:j + 1], 4), mu, res.lam2)[0] for k in range(K + 1)]
        assert int(np.argmin(scores)) == res.winner[j] or np.isclose(min(scores), scores[res.winner[j]])


def test_invariants_layer():
    W, Xr, Xq = small_layer(3, m=24, n=6, T=60)
    base = o.quantize_layer(W, Xr, Xq, 0.5, 4, 8, 0, 1)
    assert np.all(base.winner == 0)
    babai = base.decode.path_codes[:, 0]
    assert np.array_equal(base.codes, babai)
    res = o.quantize_layer(W, Xr, Xq, 0.5, 4, 8, 12, 1)
    assert np.array_equal(res.decode.path_codes[:, 0], babai)        # path 0 is Babai
    assert np.all(res.residuals <= res.decode.path_resid[:, 0])      # chosen <= Babai
    assert res.codes.max() <= 15
    # X_q == X_ref: the target no longer depends on mu
    a = o.quantize_layer(W, Xq, Xq, 0.0, 4, 8, 5, 1)
    b = o.quantize_layer(W, Xq, Xq, 1.0, 4, 8, 5, 1)
    assert np.array_equal(a.codes, b.codes) and np.allclose(a.residuals, b.residuals, rtol=1e-9)


def test_k_sweep_invariants():
    """Across the K values of the paper's ablation: path 0 is the same Babai
    point for every K, K = 1 is greedy (alpha = inf) and so repeats it, and
    no K selects a candidate worse than that path (residuals compared to a
    relative 1e-12: the oracle sums a path's residual in an order that
    depends on how many paths it evaluates together)."""
    W, Xr, Xq = small_layer(6, m=40, n=6, T=120)
    runs = {K: o.quantize_layer(W, Xr, Xq, 0.6, 4, 16, K, 3) for K in (0, 1, 5, 25)}
    babai = runs[0].codes
    r0 = runs[0].residuals
    for K, r in runs.items():
        assert np.array_equal(r.decode.path_codes[:, 0], babai), K
        assert np.all(r.residuals <= r0 * (1 + 1e-12)), K
    assert np.array_equal(runs[1].codes, babai)
    assert np.allclose(runs[1].residuals, r0, rtol=1e-12, atol=0)
    assert np.all(runs[1].winner == 0)
    assert runs[25].residuals.sum() < runs[0].residuals.sum()


def test_scale_invariance():
    """X -> 2X scales the residuals by 4 with the same codes; W -> 2W scales s exactly."""
    W, Xr, Xq = small_layer(4, m=16, n=5, T=50)
    a = o.quantize_layer(W, Xr, Xq, 0.5, 3, 8, 6, 2)
    b = o.quantize_layer(W, 2 * Xr, 2 * Xq, 0.5, 3, 8, 6, 2)
    assert np.array_equal(a.codes, b.codes)
    assert np.allclose(b.residuals, 4 * a.residuals, rtol=1e-9)
    c = o.quantize_layer(2 * W, Xr, Xq, 0.5, 3, 8, 6, 2)
    assert np.array_equal(c.scales, 2 * a.scales) and np.array_equal(c.zeros, a.zeros)
    assert np.array_equal(a.codes, c.codes)
    assert np.allclose(c.residuals, 4 * a.residuals, rtol=1e-9)


def test_not_positive_definite():
    W, Xr, Xq = small_layer(5, m=8, n=2, T=20)
    Xq = Xq.copy()
    Xq[3] = 0.0
    with pytest.raises(o.NotPositiveDefinite):
        o.quantize_layer(W, Xr, Xq, 0.5, 4, 128, 2, 0, lambda_rel=0.0)
    o.quantize_layer(W, Xr, Xq, 0.5, 4, 128, 2, 0, lambda_rel=0.01)   # damping fixes it


def test_column_subset_matches_full():
    W, Xr, Xq = small_layer(6, m=12, n=7, T=30)
    full = o.quantize_layer(W, Xr, Xq, 0.5, 4, 5, 3, 9)
    cols = np.array([5, 0, 3])
    sub = o.quantize_layer(W, Xr, Xq, 0.5, 4, 5, 3, 9, columns=cols)
    assert np.array_equal(sub.codes, full.codes[cols])
    assert np.array_equal(sub.residuals, full.residuals[cols])
