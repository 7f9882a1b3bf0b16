"""Pins for the oracle's weight permutation (act order): the decode order that
the paper's limitations name as future work, taken as the GPTQ heuristic
(largest Hessian diagonal decided first).

Each check fixes the order, the groups or the way codes are put back by
something other than the oracle's own permutation code: a hand-worked order,
closed-form rounding on a diagonal Gram, the JTA score evaluated feature by
feature in the original order, and equivariance under a relabelling of the
input features.
"""

import itertools

import numpy as np
import pytest

from oracle import ojbkq as o


def layer(seed, m=12, n=5, T=48):
    rng = np.random.default_rng(seed)
    sig = np.exp(rng.standard_normal(m))
    Xr = (rng.standard_normal((m, T)) * sig[:, None]).astype(np.float32)
    Xq = (Xr + 0.1 * rng.standard_normal((m, T)) * sig[:, None]).astype(np.float32)
    W = (0.05 * rng.standard_normal((n, m))).astype(np.float32)
    return W, Xr, Xq


def test_perm_hand_worked():
    """Rows with squared norms 4, 1, 9, 1, 0.25: increasing order with equal
    values by index is features 4, 1, 3, 0, 2 (worked by hand)."""
    Xq = np.zeros((5, 5), dtype=np.float32)
    for i, v in enumerate([2.0, 1.0, 3.0, 1.0, 0.5]):
        Xq[i, i] = v
    assert o.act_order_perm(o.gram(Xq)).tolist() == [4, 1, 3, 0, 2]
    # groups of 2 positions: features 4, 1 -> group 0; 3, 0 -> group 1; 2 -> group 2
    assert o.feature_groups([4, 1, 3, 0, 2], 2).tolist() == [1, 0, 2, 1, 0]


def test_sorted_input_is_unchanged():
    """Features whose diagonal already increases: act order is the identity
    and the result is the plain path's, bit for bit."""
    W, Xr, Xq = layer(1)
    order = np.argsort(np.sum(Xq.astype(np.float64) ** 2, axis=1))
    W, Xr, Xq = W[:, order], Xr[order], Xq[order]
    a = o.quantize_layer(W, Xr, Xq, 0.5, 4, 4, 5, 3)
    b = o.quantize_layer(W, Xr, Xq, 0.5, 4, 4, 5, 3, act_order=True)
    assert b.extra["perm"].tolist() == list(range(W.shape[1]))
    for f in ("codes", "scales", "zeros", "residuals", "winner"):
        assert np.array_equal(getattr(a, f), getattr(b, f)), f


@pytest.mark.parametrize("group", [0, 3])
def test_diagonal_gram_rounds_to_nearest_in_original_order(group):
    """X~ = X with orthogonal rows of distinct norms: H is diagonal, so every
    candidate's centres are the real solution and Babai is plain rounding of
    w / s + z, which needs no decode order.  Norms fall with the index, so
    the order is the reversal (hand-worked), and with groups of 3 positions
    feature i sits in group (m - 1 - i) // 3."""
    m, n = 8, 4
    rng = np.random.default_rng(5)
    Xq = np.zeros((m, m), dtype=np.float32)
    for i in range(m):
        Xq[i, i] = 8.0 - i
    W = (0.05 * rng.standard_normal((n, m))).astype(np.float32)
    res = o.quantize_layer(W, Xq, Xq, 0.5, 3, group, 0, 0, lambda_rel=0.0, act_order=True)
    assert res.extra["perm"].tolist() == list(range(m - 1, -1, -1))
    g = m if group <= 0 else group
    for j in range(n):
        for i in range(m):
            grp = (m - 1 - i) // g
            s, z = float(res.scales[j, grp]), float(res.zeros[j, grp])
            q = min(max(np.rint(float(W[j, i]) / s + z), 0), 7)
            assert res.codes[j, i] == q, (j, i)
    # the scales are those of the permuted groups: group 0 holds features 7, 6, 5
    if group == 3:
        Wg = W[:, [7, 6, 5]].astype(np.float64)
        lo, hi = np.minimum(Wg.min(1), 0), np.maximum(Wg.max(1), 0)
        assert np.allclose(res.scales[:, 0], (hi - lo) / 7, rtol=1e-6)


def test_score_in_original_order_minus_floor_is_residual():
    """The JTA score (Eq. jta_score) of W_hat rebuilt feature by feature in
    the original order, with feature i dequantized on the scale of the group
    its decode position falls in, minus the least-squares floor, equals the
    reported residual; a slip in putting codes back or in the groups breaks
    it."""
    W, Xr, Xq = layer(2, m=14, n=6, T=60)
    mu, g = 0.5, 4
    res = o.quantize_layer(W, Xr, Xq, mu, 3, g, 6, 11, act_order=True)
    perm = res.extra["perm"]
    m = W.shape[1]
    W_hat = np.zeros(W.shape)
    V = np.zeros(W.shape)
    for p in range(m):
        i = int(perm[p])
        grp = p // g
        W_hat[:, i] = res.scales[:, grp] * (res.codes[:, i].astype(np.float64) - res.zeros[:, grp])
        V[:, i] = res.V[:, p]
    full = o.jta_score(W, Xr, Xq, W_hat, mu, res.lam2)
    floor = o.jta_score(W, Xr, Xq, V, mu, res.lam2)
    assert np.allclose(full - floor, res.residuals, rtol=1e-7, atol=1e-12)
    assert np.allclose(W_hat, o.dequantize_by_feature(res.codes, res.scales, res.zeros,
                                                      o.feature_groups(perm, g)), rtol=0, atol=0)


def test_equivariant_under_relabelled_features():
    """Relabelling the input features (W's columns, X's rows) by sigma and
    solving with act order gives the same decode: codes relabelled alike,
    the same scales, zeros and residuals, and perm' = sigma^-1 o perm."""
    W, Xr, Xq = layer(3, m=16, n=5, T=64)
    sigma = np.random.default_rng(9).permutation(W.shape[1])
    a = o.quantize_layer(W, Xr, Xq, 0.6, 4, 4, 8, 2, act_order=True)
    b = o.quantize_layer(W[:, sigma], Xr[sigma], Xq[sigma], 0.6, 4, 4, 8, 2, act_order=True)
    inv = np.argsort(sigma)
    assert b.extra["perm"].tolist() == inv[a.extra["perm"]].tolist()
    assert np.array_equal(b.codes, a.codes[:, sigma])
    assert np.array_equal(b.scales, a.scales) and np.array_equal(b.zeros, a.zeros)
    assert np.allclose(b.residuals, a.residuals, rtol=1e-9)


def test_bounds_against_brute_force():
    """m = 6, b = 2: the chosen candidate is never worse than Babai and never
    better than the exact box optimum of the permuted problem, enumerated over
    all 4^6 points in the original feature order."""
    W, Xr, Xq = layer(4, m=6, n=3, T=30)
    res = o.quantize_layer(W, Xr, Xq, 0.5, 2, 0, 12, 5, act_order=True)
    perm = res.extra["perm"]
    Rbar_p = None
    for j in range(W.shape[0]):
        s = float(res.scales[j, 0])
        Rbar_p = res.R * s
        best = np.inf
        for pt in itertools.product(range(4), repeat=6):
            q = np.array(pt, dtype=np.float64)
            r = float(np.sum((Rbar_p @ (q[perm] - res.qbar[j])) ** 2))
            best = min(best, r)
        assert res.residuals[j] >= best * (1 - 1e-12)
        assert res.residuals[j] <= res.decode.path_resid[j, 0] * (1 + 1e-12)


def test_explicit_perm_must_be_a_permutation():
    W, Xr, Xq = layer(6, m=5, n=2, T=20)
    with pytest.raises(ValueError):
        o.quantize_layer(W, Xr, Xq, 0.5, 4, 0, 1, 0, perm=np.array([0, 1, 1, 3, 4]))
    r = o.quantize_layer(W, Xr, Xq, 0.5, 4, 0, 1, 0, perm=np.array([4, 3, 2, 1, 0]))
    assert r.extra["perm"].tolist() == [4, 3, 2, 1, 0]


# ---------------------------------------------------------------------------
# static groups: only the decode order changes, the groups stay runs of g
# features in W's order
# ---------------------------------------------------------------------------

def test_static_groups_keep_the_layer_scales():
    W, Xr, Xq = layer(7, m=14, n=4, T=50)
    plain = o.quantize_layer(W, Xr, Xq, 0.5, 3, 4, 4, 1)
    st = o.quantize_layer(W, Xr, Xq, 0.5, 3, 4, 4, 1, act_order=True, static_groups=True)
    assert np.array_equal(st.scales, plain.scales) and np.array_equal(st.zeros, plain.zeros)
    assert st.extra["perm"].tolist() == o.act_order_perm(o.gram(Xq)).tolist()


@pytest.mark.parametrize("group", [3, 0])
def test_static_groups_diagonal_gram_rounds_on_the_original_groups(group):
    """Diagonal H (orthogonal rows of falling norms, so the order is the
    reversal): Babai is plain rounding with feature i on group i // g of W's
    own order."""
    m, n = 8, 4
    rng = np.random.default_rng(8)
    Xq = np.zeros((m, m), dtype=np.float32)
    for i in range(m):
        Xq[i, i] = 8.0 - i
    W = (0.05 * rng.standard_normal((n, m))).astype(np.float32)
    res = o.quantize_layer(W, Xq, Xq, 0.5, 3, group, 0, 0, lambda_rel=0.0, act_order=True,
                           static_groups=True)
    assert res.extra["perm"].tolist() == list(range(m - 1, -1, -1))
    g = m if group <= 0 else group
    for j in range(n):
        for i in range(m):
            s, z = float(res.scales[j, i // g]), float(res.zeros[j, i // g])
            assert res.codes[j, i] == min(max(np.rint(float(W[j, i]) / s + z), 0), 7), (j, i)


def test_static_groups_score_minus_floor_is_residual():
    """The JTA score of W_hat dequantized in W's order on W's groups (the
    plain layout), minus the floor, equals the reported residual."""
    W, Xr, Xq = layer(9, m=14, n=5, T=60)
    mu, g = 0.5, 4
    res = o.quantize_layer(W, Xr, Xq, mu, 3, g, 6, 13, act_order=True, static_groups=True)
    perm = res.extra["perm"]
    V = np.zeros(W.shape)
    V[:, perm] = res.V
    W_hat = o.dequantize(res.codes, res.scales, res.zeros, g)
    full = o.jta_score(W, Xr, Xq, W_hat, mu, res.lam2)
    floor = o.jta_score(W, Xr, Xq, V, mu, res.lam2)
    assert np.allclose(full - floor, res.residuals, rtol=1e-7, atol=1e-12)


def test_static_groups_equivariant_under_group_preserving_relabelling():
    """Relabel features inside each group and the groups among themselves:
    scales follow the group relabelling, codes the feature relabelling."""
    W, Xr, Xq = layer(10, m=16, n=4, T=64)
    rng = np.random.default_rng(11)
    gperm = rng.permutation(4)
    sigma = np.concatenate([4 * gg + rng.permutation(4) for gg in gperm])
    a = o.quantize_layer(W, Xr, Xq, 0.6, 4, 4, 6, 2, act_order=True, static_groups=True)
    b = o.quantize_layer(W[:, sigma], Xr[sigma], Xq[sigma], 0.6, 4, 4, 6, 2, act_order=True,
                         static_groups=True)
    assert np.array_equal(b.scales, a.scales[:, gperm])
    assert np.array_equal(b.codes, a.codes[:, sigma])
    assert np.allclose(b.residuals, a.residuals, rtol=1e-9)


def test_static_groups_brute_force_bound():
    W, Xr, Xq = layer(12, m=6, n=3, T=30)
    res = o.quantize_layer(W, Xr, Xq, 0.5, 2, 3, 12, 5, act_order=True, static_groups=True)
    perm = res.extra["perm"]
    Sx = o.expand_groups(res.scales, 6, 3)           # W's order
    for j in range(W.shape[0]):
        Rbar_p = res.R * Sx[j, perm][None, :]
        best = np.inf
        for pt in itertools.product(range(4), repeat=6):
            q = np.array(pt, dtype=np.float64)
            best = min(best, float(np.sum((Rbar_p @ (q[perm] - res.qbar[j])) ** 2)))
        assert best * (1 - 1e-12) <= res.residuals[j] <= res.decode.path_resid[j, 0] * (1 + 1e-12)
