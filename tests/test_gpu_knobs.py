"""Per-layer knobs on one staged context (ojbkq_set_knobs): a new damping is
a re-factor of the kept Gram, a smaller K a different candidate count.  Both
must give exactly what a fresh call with those knobs gives (same token sums,
same kernels), and that agrees with the oracle."""

import numpy as np
import pytest
import torch

import paper_2602_08376_amd as ok
from oracle import ojbkq as orc
from parity import check_layer_strict, np64
from synth import LayerConfig, make_layer

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ok.library()


def cfg_of(m, n, T, K, seed):
    return LayerConfig(key=f"k{m}x{n}", title="knobs", n=n, m=m, T=T, bits=4, group=64, K=K,
                       mus=(0.5,), w_std=0.02, kind="heavy", data_seed=seed, klein_seed=seed + 1,
                       outliers=2, outlier_gain=20.0, noise=0.02)


def same(a, b):
    for f in ("codes", "scales", "zeros", "residuals", "winner"):
        assert torch.equal(getattr(a, f), getattr(b, f)), f
    if a.perm is not None or b.perm is not None:
        assert torch.equal(a.perm, b.perm)


@pytest.mark.parametrize("m,n,act", [(260, 90, False), (200, 150, True)])
def test_knobs_equal_fresh_calls(m, n, act):
    cfg = cfg_of(m, n, 1200, 8, 81 + m)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    s = ok.LayerSolver(m, n, cfg.bits, cfg.group, 8, cfg.klein_seed, 0.01, device=DEV,
                       act_order=act, keep_gram=True)
    s.set_weights(W)                      # the one-shot call binds W too: same routes
    s.accumulate(Xr, Xq)
    for lam, K, mu in ((0.01, 8, 0.5), (0.1, 3, 0.5), (0.001, 0, 0.2), (0.01, 8, 0.5)):
        s.set_knobs(lam, K)
        g = s.solve(W, mu)
        f = ok.quantize_layer(W, Xr, Xq, mu, cfg.bits, cfg.group, K, cfg.klein_seed, lam,
                              act_order=act)
        torch.cuda.synchronize()
        same(g, f)
        assert g.winner.max().item() <= K
        assert float(s.inspect("lam2")[0]) > 0
    # the oracle on one of the settings
    s.set_knobs(0.1, 3)
    g = s.solve(W, 0.5)
    pc, pr = np64(s.path_codes()), np64(s.inspect("path_resid"))
    assert pc.shape == (n, 4, m) and pr.shape == (n, 4)
    perm = None if not act else np64(g.perm).astype(np.int64)
    o = orc.quantize_layer(np64(W), np64(Xr), np64(Xq), 0.5, cfg.bits, cfg.group, 3,
                           cfg.klein_seed, lambda_rel=0.1, perm=perm)
    assert np.array_equal(np64(g.scales), o.scales) and np.array_equal(np64(g.zeros), o.zeros)
    st = check_layer_strict(o, g, pc, pr, cfg.bits, cfg.klein_seed, cfg.group, perm=perm,
                            tag=f"knobs m={m} act={act} lambda 0.1 K 3")
    assert st["agreement"] >= 0.999
    with pytest.raises(ok.OjbkqError) as ei:
        s.set_knobs(0.1, 9)               # more candidates than the context was carved for
    assert ei.value.code == "EINVAL"
    s.close()


def test_knob_errors_and_recovery_from_a_bad_pivot():
    cfg = cfg_of(96, 20, 300, 4, 91)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    Xq = Xq.clone()
    Xq[7] = 0.0                           # a dead channel: undamped Gram is singular
    # without a kept Gram, only K may change after the first solve
    s = ok.LayerSolver(96, 20, 4, 64, 4, cfg.klein_seed, 0.01, device=DEV)
    s.accumulate(Xr, Xq)
    s.solve(W, 0.5)
    s.set_knobs(0.01, 2)
    assert s.solve(W, 0.5).winner.max().item() <= 2
    with pytest.raises(ok.OjbkqError) as ei:
        s.set_knobs(0.02, 2)
    assert ei.value.code == "ESTATE"
    s.close()
    # with it: lambda = 0 fails at the pivot, a positive lambda then succeeds
    s = ok.LayerSolver(96, 20, 4, 64, 4, cfg.klein_seed, 0.0, device=DEV, keep_gram=True)
    s.set_weights(W)
    s.accumulate(Xr, Xq)
    with pytest.raises(ok.OjbkqError) as ei:
        s.solve(W, 0.5)
    assert ei.value.code == "ENOTPD"
    s.set_knobs(0.01, 4)
    g = s.solve(W, 0.5)
    f = ok.quantize_layer(W, Xr, Xq, 0.5, 4, 64, 4, cfg.klein_seed, 0.01)
    torch.cuda.synchronize()
    assert torch.equal(g.codes, f.codes) and torch.equal(g.residuals, f.residuals)
    s.close()
