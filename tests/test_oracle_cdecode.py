"""The oracle's C decode (oracle/decode.c) against its pinned Python decode
(oracle/ojbkq.py): same codes for every candidate and residuals to 1e-12 on
random problems spanning box widths, ragged groups, the greedy and flat
Klein limits, and the hand-worked 3x3 example."""

import math

import numpy as np
import pytest

from oracle import cdecode
from oracle import ojbkq as o


def problem(seed, m, n, ngroups):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((m + 5, m)) * np.exp(0.5 * rng.standard_normal(m))[None, :]
    R = o.cholesky_upper(A.T @ A + 0.05 * np.eye(m))
    S = np.exp(0.3 * rng.standard_normal((n, ngroups))).astype(np.float32)
    return R, S, rng


@pytest.mark.parametrize("m,n,bits,group,K,seed", [
    (1, 3, 2, 128, 4, 1),
    (7, 4, 2, 128, 6, 2),
    (50, 6, 3, 16, 7, 3),        # ragged groups
    (97, 5, 4, 32, 16, 4),
    (64, 3, 8, 0, 3, 5),         # 256-value box, one group
    (130, 4, 1, 64, 5, 6),       # 1-bit box
])
def test_c_decode_matches_python(m, n, bits, group, K, seed):
    G = o.num_groups(m, group)
    R, S, rng = problem(seed, m, n, G)
    qmax = (1 << bits) - 1
    qbar = rng.uniform(-0.7, qmax + 0.7, (n, m))
    a = o.decode(R, qbar, S, bits, group, K, seed)
    b = cdecode.decode(R, qbar, S, bits, group, K, seed)
    assert np.array_equal(a.path_codes, b.path_codes)
    assert np.allclose(a.path_resid, b.path_resid, rtol=1e-12, atol=0)
    assert np.array_equal(a.winner, b.winner) and np.array_equal(a.codes, b.codes)


def test_c_decode_limits_and_columns():
    """A column subset in any order, with the greedy (alpha = inf: every
    candidate is the Babai point) and flat (alpha = 0) temperatures."""
    R, S, rng = problem(9, 40, 6, 1)
    qbar = rng.uniform(-1, 16, (6, 40))
    cols = np.array([4, 1, 5])
    for alpha in (np.full(3, math.inf), np.zeros(3)):
        ref = [o.decode_column(R, qbar[j], o.expand_groups(S[j:j + 1], 40, 128)[0], 4, 5,
                               float(alpha[t]), 7, int(j)) for t, j in enumerate(cols)]
        b = cdecode.decode(R, qbar, S, 4, 128, 5, 7, columns=cols, alpha=alpha)
        assert np.array_equal(np.stack(ref), b.path_codes)
        if math.isinf(alpha[0]):
            assert all(np.array_equal(b.path_codes[t, 0], b.path_codes[t, k])
                       for t in range(3) for k in range(6))


def test_c_decode_hand_worked(golden):
    g = golden("hand_worked_3x3.txt")
    R = np.array(g["decode_R"]).reshape(3, 3)
    qbar = np.array([g["decode_qbar"]])
    b = cdecode.decode(R, qbar, np.ones((1, 1), np.float32), 2, 128, 0, 0)
    assert b.codes[0].tolist() == [int(v) for v in g["decode_babai"]]
    assert abs(b.residuals[0] - g["decode_babai_residual"][0]) < 1e-12


def test_c_decode_wide_column():
    """One column at m = 700 with K = 9 on a heavy-tailed factor."""
    R, S, rng = problem(12, 700, 2, 6)
    qbar = rng.uniform(0, 15, (2, 700))
    a = o.decode(R, qbar, S, 4, 128, 9, 3)
    b = cdecode.decode(R, qbar, S, 4, 128, 9, 3)
    assert np.array_equal(a.path_codes, b.path_codes)
    assert np.allclose(a.path_resid, b.path_resid, rtol=1e-12, atol=0)
