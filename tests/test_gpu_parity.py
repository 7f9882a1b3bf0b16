"""GPU parity: the HIP path (through the C ABI) against the CPU fp64 oracle.

Every input is seeded and synthetic; the oracle receives host copies of the
very arrays the GPU consumed.  Sizes are chosen so that the oracle finishes in
seconds while the GPU kernels still span several GEMM tiles (128), Cholesky
panels (64), decoder blocks (32) and decoder workgroups (256 paths), with
ragged tails everywhere.
"""

import math

import numpy as np
import pytest
import torch

import paper_2602_08376_amd as ok
from oracle import ojbkq as orc
from parity import (GRAM_RTOL, SCALE_RTOL, SOLVE_RTOL, centres_from_gq, check_layer_strict,
                    check_paths, np64)

GRAMS = ["int8", "fp64"]
from synth import CONFIGS, LayerConfig, make_layer, make_triangular_problem

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ok.library()          # fails loudly if the HIP library is missing
    torch.cuda.init()


def small_cfg(m, n, T, bits, group, K, seed, kind="heavy", sparsity=0.0, mu=0.5):
    return LayerConfig(key=f"t{m}x{n}", title="test", n=n, m=m, T=T, bits=bits, group=group, K=K,
                       mus=(mu,), w_std=0.02, kind=kind, data_seed=seed, klein_seed=seed + 7,
                       outliers=2, outlier_gain=20.0, noise=0.05 if kind == "tiny" else 0.02,
                       sparsity=sparsity)


def paths_of(s):
    """Every candidate of a staged context's last solve: codes [n, K+1, m] in
    W's order and residuals [n, K+1]."""
    return np64(s.path_codes()), np64(s.inspect("path_resid"))


def staged(cfg, W, Xr, Xq, mu, lam=None, K=None, **kw):
    """One staged solve with W bound and all tokens in one chunk (the calls
    the one-shot entry point makes); returns (result, paths, path residuals)."""
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K if K is None else K,
                       cfg.klein_seed, cfg.lambda_rel if lam is None else lam, device=DEV,
                       **kw)
    s.set_weights(W)
    s.accumulate(None if mu == 1.0 else Xr, Xq)   # the one-shot call reads no X_ref at mu = 1
    g = s.solve(W, mu)
    pc, pr = paths_of(s)
    s.close()
    return g, pc, pr


def same_result(a, b):
    for f in ("codes", "scales", "zeros", "residuals", "winner"):
        assert torch.equal(getattr(a, f), getattr(b, f)), f


def run_pair(cfg, mu=None, lambda_rel=None, gram="int8"):
    """The one-shot call and the same solve through the staged calls (which
    must agree bit for bit), and the oracle on the same arrays."""
    mu = cfg.mu if mu is None else mu
    lam = cfg.lambda_rel if lambda_rel is None else lambda_rel
    W, Xr, Xq = make_layer(cfg, device=DEV)
    g = ok.quantize_layer(W, Xr, Xq, mu, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, lam,
                          gram=gram)
    st, pc, pr = staged(cfg, W, Xr, Xq, mu, lam, gram=gram)
    torch.cuda.synchronize()
    same_result(g, st)
    o = orc.quantize_layer(np64(W), np64(Xr), np64(Xq), mu, cfg.bits, cfg.group, cfg.K,
                           cfg.klein_seed, lambda_rel=lam)
    return (W, Xr, Xq), g, o, (pc, pr)


def check_layer(cfg, g, o, mu, paths):
    """Scales and zero points bit-equal, then the full rule on every
    candidate of every column (tests/parity.py)."""
    S, Z = np64(g.scales), np64(g.zeros)
    assert np.array_equal(S, o.scales), "scales differ"
    assert np.array_equal(Z, o.zeros), "zero points differ"
    assert np.all(np.abs(S - o.scales) <= SCALE_RTOL * np.abs(o.scales))
    codes = np64(g.codes)
    assert codes.max() <= (1 << cfg.bits) - 1
    pc, pr = paths
    st = check_layer_strict(o, g, pc, pr, cfg.bits, cfg.klein_seed, cfg.group,
                            tag=f"{cfg.key} mu={mu}")
    return st["agreement"]


# ---------------------------------------------------------------------------
# hand-worked example (the 3x3 layer worked out by hand in tests/golden)
# ---------------------------------------------------------------------------

def test_hand_worked_layer(golden):
    gd = golden("hand_worked_3x3.txt")
    W = torch.tensor([gd["layer_W"]], dtype=torch.float32, device=DEV)
    Xq = torch.tensor(gd["layer_Xq"], dtype=torch.float32, device=DEV).reshape(3, 3)
    g = ok.quantize_layer(W, Xq, Xq, 1.0, 2, 128, 0, 0, lambda_rel=0.0)
    assert np64(g.codes)[0].tolist() == [int(v) for v in gd["layer_codes"]]
    assert abs(float(g.residuals[0]) - gd["layer_residual"][0]) < 5e-7
    assert int(g.winner[0]) == 0


def test_hand_worked_decode(golden):
    gd = golden("hand_worked_3x3.txt")
    R = torch.tensor(gd["decode_R"], dtype=torch.float64, device=DEV).reshape(3, 3)
    qbar = torch.tensor([gd["decode_qbar"]], dtype=torch.float64, device=DEV)
    S = torch.ones(1, 1, dtype=torch.float32, device=DEV)
    codes, res, win, _, _ = ok.decode_stage(R, qbar, S, 2, 128, 0, 0)
    assert np64(codes)[0].tolist() == [int(v) for v in gd["decode_babai"]]
    assert abs(float(res[0]) - gd["decode_babai_residual"][0]) < 1e-12


@pytest.mark.parametrize("tag,mu", [("mu05", 0.5), ("mu0", 0.0)])
def test_hand_worked_damped_layer(golden, tag, mu):
    """The 3x3 layer with damping and a cross term, worked by hand: lambda^2,
    the factor, the codes and the reduced residual."""
    gd = golden("hand_worked_3x3.txt")
    W = torch.tensor([gd["layer_W"]], dtype=torch.float32, device=DEV)
    Xq = torch.tensor(gd["layer_Xq"], dtype=torch.float32, device=DEV).reshape(3, 3)
    Xr = Xq + gd["damped_delta"][0] * torch.eye(3, dtype=torch.float32, device=DEV)
    s = ok.LayerSolver(3, 1, 2, 128, 0, 0, lambda_rel=0.01, device=DEV)
    s.accumulate(Xr, Xq)
    g = s.solve(W, mu)
    lam2 = float(s.inspect("lam2")[0])
    L = np64(s.inspect("L"))
    s.close()
    assert abs(lam2 - gd["damped_lam2"][0]) <= 1e-9
    assert np.allclose(L.T, np.array(gd["damped_R"]).reshape(3, 3), atol=5e-7, rtol=0)
    assert np64(g.codes)[0].tolist() == [int(v) for v in gd[f"damped_{tag}_codes"]]
    assert abs(float(g.residuals[0]) - gd[f"damped_{tag}_residual"][0]) < 5e-7
    one = ok.quantize_layer(W, Xr, Xq, mu, 2, 128, 0, 0, lambda_rel=0.01)
    assert torch.equal(one.codes, g.codes)


def test_exact_residual_tie_keeps_babai(golden):
    """Alg. 4's strict "<": candidates whose residual equals the Babai one
    exactly (m = 1, qbar = 1.5) do not replace it."""
    gd = golden("hand_worked_3x3.txt")
    R = torch.ones(1, 1, dtype=torch.float64, device=DEV)
    qbar = torch.full((1, 1), gd["tie_qbar"][0], dtype=torch.float64, device=DEV)
    S = torch.ones(1, 1, dtype=torch.float32, device=DEV)
    codes, res, win, pc, pr = ok.decode_stage(R, qbar, S, 2, 128, 8, 5, want_paths=True)
    pr, pc = np64(pr)[0], np64(pc)[0, :, 0]
    assert pc[0] == 2 and pr[0] == gd["tie_residual"][0]
    ties = [k for k in range(1, 9) if pr[k] == pr[0]]
    assert ties and any(pc[k] == 1 for k in ties)
    assert int(win[0]) == int(gd["tie_winner"][0]) and float(res[0]) == 0.25
    dec = orc.decode(np64(R), np64(qbar), np64(S), 2, 128, 8, 5)
    assert np.array_equal(pc, dec.path_codes[0, :, 0])


# ---------------------------------------------------------------------------
# the decoder alone, on the oracle's own factor and centres
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("decode", ["int8", "fp64"])
@pytest.mark.parametrize("m,n,bits,group,K,seed", [
    (7, 5, 2, 128, 6, 1),          # tiny, one partial block
    (100, 23, 3, 40, 9, 2),        # ragged groups and blocks, several workgroups (int8: not
                                   # whole 64-row pairs, so the fp64 update runs)
    (257, 40, 4, 128, 16, 3),      # > 256 paths, 9 blocks, 3 groups (ragged)
    (64, 300, 4, 0, 0, 4),         # Babai only, 2 workgroups
    (96, 11, 8, 32, 3, 5),         # 8-bit box (256 values): the fp64 update
    (990, 17, 7, 64, 5, 6),        # 7-bit box (int8 codes up to 127), one pair per group,
                                   # 31 blocks (the code segments padded to 32)
    (1100, 9, 4, 256, 4, 7),       # four pairs per group, ragged last group and block
    (2900, 3, 3, 0, 2, 8),         # one group: scale flushes every 32 pairs
])
def test_decode_stage_matches_oracle(m, n, bits, group, K, seed, decode):
    R, qbar, S = make_triangular_problem(m, n, orc.num_groups(m, group), seed)
    if bits >= 7:
        qbar = qbar * (2.0 ** (bits - 4))
    Rn, qn, Sn = R.numpy(), qbar.numpy(), S.numpy()
    codes, res, win, pc, pr = ok.decode_stage(R.to(DEV), qbar.to(DEV), S.to(DEV), bits, group, K,
                                              seed, want_paths=True, decode=decode)
    dec = orc.decode(Rn, qn, Sn, bits, group, K, seed)
    frac, ties = check_paths(Rn, qn, Sn, group, bits, K, seed, dec.alpha, np64(pc),
                             dec.path_codes)
    rel = np.abs(np64(pr) - dec.path_resid) / np.abs(dec.path_resid)
    print(f"[decode {decode} m={m} n={n} b={bits} K={K}] agreement {frac:.6f} ties {ties} "
          f"max path resid rel err {rel.max():.2e}")
    assert rel.max() <= 1e-9
    assert np.array_equal(np64(win), dec.winner)
    assert np.array_equal(np64(codes), dec.codes)
    assert np.all(np64(res) == np64(pr)[np.arange(n), np64(win)])


def test_decode_brute_force_small():
    """m = 6, b = 2: nothing beats the exact optimum, the choice never loses to Babai, and the
    GPU reaches the optimum on exactly the instances where the oracle's own draws do."""
    import itertools
    hits = orc_hits = 0
    pts = np.array(list(itertools.product(range(4), repeat=6)), dtype=np.float64)
    for trial in range(6):
        R, qbar, S = make_triangular_problem(6, 4, 1, 100 + trial, coupling=1.0, qbar_lo=-0.5,
                                             qbar_hi=3.5)
        S = torch.ones_like(S)
        codes, res, win, pc, pr = ok.decode_stage(R.to(DEV), qbar.to(DEV), S.to(DEV), 2, 128, 300,
                                                  trial, want_paths=True)
        Rn, qn = R.numpy(), qbar.numpy()
        dec = orc.decode(Rn, qn, S.numpy(), 2, 128, 300, trial)
        for j in range(4):
            r_opt = np.sum(((pts - qn[j][None, :]) @ Rn.T) ** 2, axis=1).min()
            assert float(res[j]) >= r_opt - 1e-9
            assert float(res[j]) <= float(pr[j, 0]) + 1e-15          # never worse than Babai
            hits += int(abs(float(res[j]) - r_opt) <= 1e-9 * max(1.0, r_opt))
            orc_hits += int(abs(dec.residuals[j] - r_opt) <= 1e-9 * max(1.0, r_opt))
    print(f"[brute force] optimum reached on {hits}/24 columns (oracle {orc_hits}/24)")
    assert hits == orc_hits
    assert hits >= 12


# ---------------------------------------------------------------------------
# whole layer through the one-shot entry point
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("gram", GRAMS)
def test_tiny_config_c1(gram):
    cfg = CONFIGS["c1"]
    _, g, o, paths = run_pair(cfg, gram=gram)
    frac = check_layer(cfg, g, o, cfg.mu, paths)
    assert frac == 1.0


@pytest.mark.parametrize("m,n,T,bits,group,K,seed,mu", [
    (200, 37, 300, 3, 128, 3, 11, 0.5),     # ragged group (72), ragged tiles
    (130, 5, 257, 4, 0, 0, 12, 0.0),        # one group per column, Babai only, mu = 0
    (300, 150, 700, 4, 128, 8, 13, 1.0),    # several tiles / panels / blocks, mu = 1
    (1, 3, 5, 2, 128, 2, 14, 0.5),          # single input feature
    (33, 2, 40, 8, 16, 5, 15, 0.25),        # 8-bit box
    (96, 80, 400, 4, 32, 6, 16, 0.5),       # n > m / 2: Rbar qbar through Q = L + (1 - mu) (L^-1 E)^T
    (150, 40, 500, 3, 64, 4, 17, 0.0),      # n < m / 2: Rbar qbar through W E^T and L^-T, mu = 0
])
def test_layer_matches_oracle(m, n, T, bits, group, K, seed, mu):
    cfg = small_cfg(m, n, T, bits, group, K, seed)
    _, g, o, paths = run_pair(cfg, mu=mu)
    frac = check_layer(cfg, g, o, mu, paths)
    assert frac >= 0.999


@pytest.mark.parametrize("gram", GRAMS)
def test_heavy_tailed_layer_m1024(gram):
    """A slice of the 4096x4096 attention workload: heavy-tailed channels, 1% outliers x50."""
    cfg = small_cfg(1024, 48, 4096, 4, 128, 16, 21)
    _, g, o, paths = run_pair(cfg, gram=gram)
    frac = check_layer(cfg, g, o, cfg.mu, paths)
    assert frac >= 0.999


def gq_error(gq, o, W, m, group):
    """Largest error of the decoder's input rows Rbar_j qbar_j against the
    oracle's, each entry relative to the size of the terms summed into it:
    (|s qbar| + |w| + |s z|) |R^T| (the centre s qbar = w + s z + the
    cross-term correction can cancel to almost nothing, as in a group of one
    negative weight)."""
    Sx = orc.expand_groups(o.scales, m, group)
    Zx = orc.expand_groups(o.zeros, m, group)
    scale = (np.abs(Sx * o.qbar) + np.abs(W) + np.abs(Sx * Zx)) @ np.abs(o.R.T)
    return float(np.max(np.abs(gq - (Sx * o.qbar) @ o.R.T) / scale))


@pytest.mark.parametrize("m,n,mu", [
    (64, 40, 0.5),      # one tile; n > m / 2: the whole L^-1
    (65, 20, 0.5),      # a ragged second tile of one row; n < m / 2: triangular solve
    (127, 100, 0.0),
    (191, 60, 0.5),     # three tiles, the last ragged; solve leaves of 128 and 63
    (257, 200, 1.0),    # no cross term
    (700, 120, 0.25),   # eleven tiles (ragged 60), six solve leaves
    (700, 500, 0.5),
])
def test_factor_and_solve_routes(m, n, mu):
    """The one-launch tiled factor and its inverse tiles (whole, or the
    128-wide diagonal blocks the triangular solve multiplies by) against the
    oracle's R and centres, on both routes to Rbar qbar."""
    cfg = small_cfg(m, n, max(2 * m, 256), 4, 128, 2, 40 + m % 17)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, device=DEV)
    s.accumulate(Xr, Xq)
    g = s.solve(W, mu)
    o = orc.quantize_layer(np64(W), np64(Xr), np64(Xq), mu, cfg.bits, cfg.group, cfg.K,
                           cfg.klein_seed)
    L = np64(s.inspect("L"))
    assert np.all(np.triu(L, 1) == 0.0), "upper triangle of the factor not cleared"
    colnorm = np.sqrt(np.sum(o.R ** 2, axis=0))
    errR = float(np.max(np.abs(L.T - o.R) / colnorm[None, :]))
    gq = np64(s.inspect("gq"))
    errg = gq_error(gq, o, np64(W), cfg.m, cfg.group)
    print(f"[factor m={m} n={n} mu={mu}] R err {errR:.2e}, Rbar qbar err {errg:.2e}")
    assert errR < GRAM_RTOL["int8"], errR
    assert errg < SOLVE_RTOL["int8"], errg
    assert check_layer(cfg, g, o, mu, paths_of(s)) >= 0.999
    s.close()


def test_blocked_factor_beyond_tiled_range():
    """m = 12300, above the size the one-launch tiled factor takes: the
    blocked factor (64-wide steps in 256-wide outer panels, ragged last panel
    of 12 columns), its 128-wide inverse blocks and the triangular solve."""
    cfg = small_cfg(12300, 6, 1024, 4, 128, 2, 24)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, device=DEV)
    s.accumulate(Xr, Xq)
    g = s.solve(W, cfg.mu)
    L = np64(s.inspect("L"))
    gq = np64(s.inspect("gq"))
    paths = paths_of(s)
    s.close()
    o = orc.quantize_layer(np64(W), np64(Xr), np64(Xq), cfg.mu, cfg.bits, cfg.group, cfg.K,
                           cfg.klein_seed)
    colnorm = np.sqrt(np.sum(o.R ** 2, axis=0))
    errR = float(np.max(np.abs(L.T - o.R) / colnorm[None, :]))
    errg = gq_error(gq, o, np64(W), cfg.m, cfg.group)
    print(f"[t12300] R err {errR:.2e}, Rbar qbar err {errg:.2e}")
    assert errR < GRAM_RTOL["int8"], errR
    assert errg < SOLVE_RTOL["int8"], errg
    assert check_layer(cfg, g, o, cfg.mu, paths) >= 0.999


def test_wide_layer_two_level_factor():
    """m = 6200 in the one-launch tiled factor: 97 tiles per side, the last
    of 56 rows."""
    cfg = small_cfg(6200, 6, 8192, 4, 128, 2, 23)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, device=DEV)
    s.accumulate(Xr, Xq)
    g = s.solve(W, cfg.mu)
    L = np64(s.inspect("L"))
    paths = paths_of(s)
    s.close()
    o = orc.quantize_layer(np64(W), np64(Xr), np64(Xq), cfg.mu, cfg.bits, cfg.group, cfg.K,
                           cfg.klein_seed)
    colnorm = np.sqrt(np.sum(o.R ** 2, axis=0))
    errR = float(np.max(np.abs(L.T - o.R) / colnorm[None, :]))
    print(f"[t6200] R err {errR:.2e}")
    assert errR < GRAM_RTOL["int8"], errR
    assert check_layer(cfg, g, o, cfg.mu, paths) >= 0.999


def test_sparse_mlp_layer_3bit():
    """Post-SiLU-like activations (60% near-zero), 3-bit box, as the down_proj workload."""
    cfg = small_cfg(640, 40, 2048, 3, 128, 16, 22, sparsity=0.6)
    _, g, o, paths = run_pair(cfg)
    frac = check_layer(cfg, g, o, cfg.mu, paths)
    assert frac >= 0.999


# ---------------------------------------------------------------------------
# intermediates of the staged entry points
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("gram", GRAMS)
def test_staged_intermediates_and_chunks(gram):
    cfg = small_cfg(300, 60, 1200, 4, 128, 8, 31)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, device=DEV,
                       gram=gram)
    for c0 in range(0, cfg.T, 400):          # three token chunks (views with row stride T)
        s.accumulate(Xr[:, c0:c0 + 400], Xq[:, c0:c0 + 400])
    g = s.solve(W, 0.5)
    o = orc.quantize_layer(np64(W), np64(Xr), np64(Xq), 0.5, cfg.bits, cfg.group, cfg.K,
                           cfg.klein_seed)
    L = np64(s.inspect("L"))
    colnorm = np.sqrt(np.sum(o.R ** 2, axis=0))          # sqrt(H_ll)
    errR = np.max(np.abs(L.T - o.R) / colnorm[None, :])
    assert errR < GRAM_RTOL[gram], errR
    lam2 = float(s.inspect("lam2")[0])
    assert abs(lam2 - o.lam2) <= GRAM_RTOL[gram] * o.lam2
    # the decoder's input rows Rbar_j qbar_j against the oracle's centres and
    # factor, and the centres recovered from them
    gq = np64(s.inspect("gq"))
    Sx = orc.expand_groups(o.scales, cfg.m, cfg.group)
    gq_o = (Sx * o.qbar) @ o.R.T
    gq_scale = np.abs(Sx * o.qbar) @ np.abs(o.R.T)
    errg = np.max(np.abs(gq - gq_o) / gq_scale)
    assert errg < SOLVE_RTOL[gram], errg
    qb = centres_from_gq(L, gq, o.scales, cfg.group)
    errq = np.max(np.abs(qb - o.qbar))
    assert errq < 1e-7, errq
    al = np64(s.inspect("alpha"))
    assert np.allclose(al, o.decode.alpha, rtol=GRAM_RTOL[gram])
    pr = np64(s.inspect("path_resid"))
    assert np.allclose(pr, o.decode.path_resid, rtol=SOLVE_RTOL[gram])
    print(f"[staged] R err {errR:.2e}, qbar err {errq:.2e}")
    check_layer(cfg, g, o, 0.5, paths_of(s))
    # the one-shot call on the whole token set gives the same codes
    one = ok.quantize_layer(W, Xr, Xq, 0.5, cfg.bits, cfg.group, cfg.K, cfg.klein_seed,
                            gram=gram)
    assert torch.equal(one.codes, g.codes)
    assert np.allclose(np64(one.residuals), np64(g.residuals), rtol=SOLVE_RTOL[gram])
    s.close()


def _chunked_reference(Xr, Xq, bounds, cross):
    """X_ref as the oracle sees it: chunks accumulated without a cross term
    have X_ref = X_q."""
    xr = Xr.clone()
    for (a, b), c in zip(bounds, cross):
        if not c:
            xr[:, a:b] = Xq[:, a:b]
    return xr


@pytest.mark.parametrize("m,n,bind,gram", [
    (300, 40, True, "fp64"),    # 5 n <= 2 m with W bound: cross term accumulated as W E^T
    (300, 40, False, "fp64"),   # same layer, mixed product route
    (120, 100, True, "fp64"),   # n > m / 2: W only bound, mixed product route
    (300, 25, True, "int8"),    # 10 n <= m with W bound: W E^T accumulated
    (300, 40, True, "int8"),    # the cross term itself, chunk by chunk
    (120, 100, False, "int8"),
])
def test_mixed_chunks_and_bound_weights(m, n, bind, gram):
    """Chunks with and without a cross term in any order, and the projected
    route, whose token steps (2240 tokens at m = 300, n = 40) split the
    second chunk with a ragged tail."""
    cfg = small_cfg(m, n, 3600, 4, 128, 6, 35)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    bounds = [(0, 400), (400, 2600), (2600, 3000), (3000, 3600)]
    cross = [False, True, False, True]
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, device=DEV,
                       gram=gram)
    if bind:
        s.set_weights(W)
    for (a, b), c in zip(bounds, cross):
        s.accumulate(Xr[:, a:b] if c else None, Xq[:, a:b])
    xr_o = np64(_chunked_reference(Xr, Xq, bounds, cross))
    for mu in (0.5, 0.0):
        g = s.solve(W, mu)
        torch.cuda.synchronize()
        o = orc.quantize_layer(np64(W), xr_o, np64(Xq), mu, cfg.bits, cfg.group, cfg.K,
                               cfg.klein_seed)
        gq = np64(s.inspect("gq"))
        Sx = orc.expand_groups(o.scales, cfg.m, cfg.group)
        gq_o = (Sx * o.qbar) @ o.R.T
        errg = np.max(np.abs(gq - gq_o) / (np.abs(Sx * o.qbar) @ np.abs(o.R.T)))
        print(f"[mixed m={m} n={n} bind={bind} {gram} mu={mu}] Rbar qbar rel err {errg:.2e}")
        assert errg < SOLVE_RTOL[gram], errg
        assert check_layer(cfg, g, o, mu, paths_of(s)) >= 0.999
    if bind:
        with pytest.raises(ok.OjbkqError) as ei:
            s.solve(W.clone(), 0.5)          # another buffer than the bound one
        assert ei.value.code == "EINVAL"
    s.close()
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, device=DEV,
                       gram=gram)
    s.accumulate(Xr, Xq)
    with pytest.raises(ok.OjbkqError) as ei:
        s.set_weights(W)                     # only before the first chunk
    assert ei.value.code == "ESTATE"
    s.close()


def test_large_k_and_k_sweep_invariants():
    """K = 25 and 50, the top of the paper's K ablation, against the oracle;
    and across the sweep: K = 1 draws greedily (alpha = inf), so it returns
    the Babai point, and no K selects a worse candidate than that path."""
    cfg = small_cfg(512, 12, 2048, 4, 128, 0, 51, mu=0.6)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    runs = {}
    for K in (0, 1, 25, 50):
        g = ok.quantize_layer(W, Xr, Xq, 0.6, cfg.bits, cfg.group, K, cfg.klein_seed)
        torch.cuda.synchronize()
        runs[K] = g
        if K >= 25:
            st, pc, pr = staged(cfg, W, Xr, Xq, 0.6, K=K)
            same_result(g, st)
            o = orc.quantize_layer(np64(W), np64(Xr), np64(Xq), 0.6, cfg.bits, cfg.group, K,
                                   cfg.klein_seed)
            assert check_layer(cfg, g, o, 0.6, (pc, pr)) >= 0.999
    r0 = np64(runs[0].residuals)
    assert np.array_equal(np64(runs[1].codes), np64(runs[0].codes))
    assert np.allclose(np64(runs[1].residuals), r0, rtol=1e-13, atol=0)
    assert np.all(np64(runs[1].winner) == 0)
    for K in (25, 50):
        assert np.all(np64(runs[K].residuals) <= r0 * (1 + 1e-13)), K
    print(f"[k sweep] mean residual K=0 {r0.mean():.4e}, K=25 {np64(runs[25].residuals).mean():.4e}, "
          f"K=50 {np64(runs[50].residuals).mean():.4e}")


@pytest.mark.parametrize("m,n,bits,group,K,mu", [
    (300, 40, 4, 128, 6, 0.6),    # projected cross term, ragged group
    (130, 70, 3, 0, 4, 0.5),      # one group per column, mixed-product route
    (96, 8, 2, 32, 3, 1.0),       # 2-bit box (z = 2, s = max|w|), no cross term
])
def test_symmetric_absmax_scales(m, n, bits, group, K, mu):
    """The symmetric Absmax scales and zero points end to end against the oracle."""
    cfg = small_cfg(m, n, 4 * m + 17, bits, group, K, 61 + bits)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    g = ok.quantize_layer(W, Xr, Xq, mu, bits, group, K, cfg.klein_seed, scheme="sym")
    torch.cuda.synchronize()
    o = orc.quantize_layer(np64(W), np64(Xr), np64(Xq), mu, bits, group, K, cfg.klein_seed,
                           scheme="sym")
    assert np.all(np64(g.zeros) == 2 ** (bits - 1))
    s = ok.LayerSolver(m, n, bits, group, K, cfg.klein_seed, device=DEV, scheme="sym")
    s.accumulate(Xr, Xq)
    st = s.solve(W, mu)
    paths = paths_of(s)
    s.close()
    assert torch.equal(st.codes, g.codes) and torch.equal(st.scales, g.scales)
    assert check_layer(cfg, st, o, mu, paths) >= 0.999


@pytest.mark.parametrize("gram", GRAMS)
def test_gram_load_paths_agree(gram):
    """The token sums read 16-byte runs of tokens when rows are 16-byte
    aligned (and, for fp64, T % 4 == 0), else single tokens; both paths stage
    the same values, so the factor they lead to is bit-identical, and it
    matches the oracle's."""
    cfg = small_cfg(200, 24, 1200, 4, 128, 4, 33)
    W, Xr, Xq = make_layer(cfg, device=DEV)

    def factor(xr, xq):
        s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, device=DEV,
                           gram=gram)
        s.accumulate(xr, xq)
        s.solve(W, 0.5)
        L = s.inspect("L")
        s.close()
        return L

    L16 = factor(Xr, Xq)
    # the same tokens as views at a 4-byte offset with an odd row stride
    br = torch.zeros(cfg.m, cfg.T + 5, dtype=torch.float32, device=DEV)
    bq = torch.zeros_like(br)
    br[:, 1:cfg.T + 1] = Xr
    bq[:, 1:cfg.T + 1] = Xq
    L4 = factor(br[:, 1:cfg.T + 1], bq[:, 1:cfg.T + 1])
    assert torch.equal(L16, L4)
    o = orc.quantize_layer(np64(W), np64(Xr), np64(Xq), 0.5, cfg.bits, cfg.group, cfg.K,
                           cfg.klein_seed)
    colnorm = np.sqrt(np.sum(o.R ** 2, axis=0))
    assert np.max(np.abs(np64(L16).T - o.R) / colnorm[None, :]) < GRAM_RTOL[gram]


def test_alpha_sweep_reuses_factor():
    cfg = small_cfg(160, 20, 600, 3, 32, 5, 41)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, device=DEV)
    s.accumulate(Xr, Xq)
    for mu in (0.0, 0.5, 1.0):
        g = s.solve(W, mu)
        one = ok.quantize_layer(W, Xr, Xq, mu, cfg.bits, cfg.group, cfg.K, cfg.klein_seed)
        assert torch.equal(one.codes, g.codes)
        o = orc.quantize_layer(np64(W), np64(Xr), np64(Xq), mu, cfg.bits, cfg.group, cfg.K,
                               cfg.klein_seed)
        check_layer(cfg, g, o, mu, paths_of(s))
    with pytest.raises(ok.OjbkqError) as ei:
        s.accumulate(Xr, Xq)
    assert ei.value.code == "ESTATE"
    s.close()


def test_degenerate_groups_and_channels():
    """Weight groups that are all zero, all positive or all negative, two equal
    columns, and a dead input channel (zero Gram row: only the damping keeps
    H positive definite)."""
    cfg = small_cfg(160, 24, 600, 4, 32, 6, 71)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    W[0, :32] = 0.0
    W[1, 32:64] = W[1, 32:64].abs()
    W[2] = -W[2].abs()
    W[4] = W[3]
    Xr[5] = 0.0
    Xq[5] = 0.0
    g = ok.quantize_layer(W, Xr, Xq, 0.5, cfg.bits, cfg.group, cfg.K, cfg.klein_seed)
    st, pc, pr = staged(cfg, W, Xr, Xq, 0.5)
    torch.cuda.synchronize()
    same_result(g, st)
    o = orc.quantize_layer(np64(W), np64(Xr), np64(Xq), 0.5, cfg.bits, cfg.group, cfg.K,
                           cfg.klein_seed)
    assert check_layer(cfg, g, o, 0.5, (pc, pr)) >= 0.999
    # the degenerate group's grid is [-1, 1]: zero point in the middle of the box
    assert float(g.scales[0, 0]) == float(o.scales[0, 0]) == float(np.float32(2.0 / 15.0))
    assert float(g.zeros[0, 0]) == float(o.zeros[0, 0])
    # equal columns share scales and zero points
    assert torch.equal(g.scales[3], g.scales[4]) and torch.equal(g.zeros[3], g.zeros[4])


def test_same_activations_make_mu_irrelevant():
    cfg = small_cfg(96, 12, 300, 4, 32, 4, 51)
    W, _, Xq = make_layer(cfg, device=DEV)
    a = ok.quantize_layer(W, Xq, Xq, 0.0, cfg.bits, cfg.group, cfg.K, 3)
    b = ok.quantize_layer(W, None, Xq, 1.0, cfg.bits, cfg.group, cfg.K, 3)
    assert torch.equal(a.codes, b.codes)
    assert torch.equal(a.residuals, b.residuals)


# ---------------------------------------------------------------------------
# invariants, determinism, failure path
# ---------------------------------------------------------------------------

def test_invariants_and_determinism():
    cfg = small_cfg(256, 64, 1024, 4, 128, 12, 61)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    a = ok.quantize_layer(W, Xr, Xq, 0.5, 4, 128, 12, 9)
    b = ok.quantize_layer(W, Xr, Xq, 0.5, 4, 128, 12, 9)
    assert torch.equal(a.codes, b.codes) and torch.equal(a.residuals, b.residuals)
    z = ok.quantize_layer(W, Xr, Xq, 0.5, 4, 128, 0, 9)           # K = 0: Babai only
    assert torch.all(z.winner == 0)
    assert torch.all(a.residuals <= z.residuals)                   # chosen <= Babai
    one = ok.quantize_layer(W, Xr, Xq, 0.5, 4, 128, 1, 9)          # K = 1: alpha = inf
    assert torch.equal(one.codes, z.codes) and torch.all(one.winner == 0)
    c = ok.quantize_layer(W, Xr, Xq, 0.5, 4, 128, 12, 10)          # another seed, other draws
    assert not torch.equal(a.codes, c.codes)


def test_not_positive_definite_reported():
    cfg = small_cfg(40, 4, 100, 4, 128, 2, 71)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    Xq = Xq.clone()
    Xq[17] = 0.0
    with pytest.raises(ok.OjbkqError) as ei:
        ok.quantize_layer(W, Xr, Xq, 0.5, 4, 128, 2, 0, lambda_rel=0.0)
    assert ei.value.code == "ENOTPD" and "17" in str(ei.value)
    ok.quantize_layer(W, Xr, Xq, 0.5, 4, 128, 2, 0, lambda_rel=0.01)   # damping repairs it


def test_stage_timing():
    cfg = small_cfg(256, 64, 1024, 4, 128, 8, 81)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, device=DEV)
    s.set_timing(True)
    s.accumulate(Xr, Xq)
    g1 = s.solve(W, 0.5)
    t1 = s.stage_times()
    assert set(t1) == set(ok.STAGES)
    assert all(v > 0.0 for v in t1.values()), t1
    g2 = s.solve(W, 0.0)             # the factor is reused: no second factor stage
    t2 = s.stage_times()
    assert t2["factor"] == t1["factor"] and t2["decode"] > t1["decode"]
    s.set_timing(False)
    assert all(v == 0.0 for v in s.stage_times().values())
    one = ok.quantize_layer(W, Xr, Xq, 0.5, cfg.bits, cfg.group, cfg.K, cfg.klein_seed)
    assert torch.equal(one.codes, g1.codes)     # timing changes nothing
    s.close()
