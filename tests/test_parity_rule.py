"""CPU checks of the parity rule itself (tests/parity.py): the oracle
compared with itself passes, and each kind of mistake the rule exists to
catch -- a code flip away from a near-tie, a winner swap without a tie, a
candidate residual off by more than 1e-4 -- makes it fail."""

import numpy as np
import pytest

from oracle import ojbkq as orc
from parity import check_paths_strict


def _case():
    rng = np.random.default_rng(11)
    m, n, T = 40, 6, 160
    sig = np.exp(rng.standard_normal(m))
    Xr = (rng.standard_normal((m, T)) * sig[:, None]).astype(np.float32)
    Xq = (Xr + 0.05 * rng.standard_normal((m, T)) * sig[:, None]).astype(np.float32)
    W = (0.05 * rng.standard_normal((n, m))).astype(np.float32)
    o = orc.quantize_layer(W, Xr, Xq, 0.5, 3, 16, 5, 4)
    s_rows = orc.expand_groups(o.scales, m, 16)
    d = o.decode
    base = dict(R=o.R, qbar=o.qbar, s_rows=s_rows, bits=3, seed=4, alpha=d.alpha,
                cols=np.arange(n), gpu_paths=d.path_codes.copy(), gpu_presid=d.path_resid.copy(),
                gpu_codes=o.codes.copy(), gpu_res=o.residuals.copy(), gpu_win=o.winner.copy(),
                orc_paths=d.path_codes, orc_presid=d.path_resid, orc_res=o.residuals,
                orc_win=o.winner)
    return o, base


def test_oracle_against_itself_passes():
    _, base = _case()
    st = check_paths_strict(**base, tag="self")
    assert st["agreement"] == 1.0 and st["tie_paths"] == 0 and st["winner_mismatch"] == 0


def test_code_flip_away_from_a_tie_fails():
    o, base = _case()
    R, qbar, s = o.R, o.qbar, base["s_rows"]
    # the Babai row of column 0 whose centre is farthest from a rounding boundary
    q = o.decode.path_codes[0, 0].astype(np.float64)
    Rb = R * s[0][None, :]
    m = len(q)
    c = np.array([qbar[0, i] + Rb[i, i + 1:] @ (qbar[0, i + 1:] - q[i + 1:]) / Rb[i, i]
                  for i in range(m)])
    far = int(np.argmin(np.abs(np.abs(c - np.floor(c)) - 0.5) * -1))
    paths = base["gpu_paths"]
    paths[0, 0, far] = paths[0, 0, far] + 1 if paths[0, 0, far] < 7 else paths[0, 0, far] - 1
    base["gpu_presid"][0, 0] = orc.reduced_residual(R, s[0], paths[0, :1], qbar[0])[0]
    with pytest.raises(AssertionError, match="not a near-tie"):
        check_paths_strict(**base)


def test_winner_swap_without_a_tie_fails():
    o, base = _case()
    t = int(np.argmax([np.ptp(r) for r in o.decode.path_resid]))
    k_other = int(np.argmax(o.decode.path_resid[t]))
    base["gpu_presid"][t, k_other] = 0.0           # a wrong residual makes another candidate win
    base["gpu_win"][t] = k_other
    with pytest.raises(AssertionError):
        check_paths_strict(**base)


def test_candidate_residual_error_fails():
    _, base = _case()
    base["gpu_presid"][2, 3] *= 1.0 + 3e-4
    with pytest.raises(AssertionError, match="residual"):
        check_paths_strict(**base)
