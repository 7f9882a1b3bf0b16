"""Parity at the full size of the Llama-7B-shaped attention projection.

W 4096 x 4096, X_ref / X_q 4096 x 262144 tokens (heavy-tailed channel scales,
1% outlier channels), 4-bit, group 128, K = 16, alpha = 0.5 -- the workload
bench.py times, run through the same staged calls (one token chunk, one
solve) in the same launch configuration.

The oracle forms its own full fp64 Gram and factor on the host, then the
relaxed solution and the decode of a seeded sample of columns (every candidate
of each).  Scales and zero points are compared for every column.
"""

import numpy as np
import pytest
import torch

import paper_2602_08376_amd as ok
from oracle import ojbkq as orc
from parity import check_residuals, first_divergence_is_tie, np64
from synth import CONFIGS
from synth.workloads import activation_chunks, make_weights

pytestmark = pytest.mark.gpu

N_COLS = 12


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ok.library()


def test_attention_projection_full_size():
    cfg = CONFIGS["c2"]
    dev = torch.device("cuda", 0)
    W = make_weights(cfg, device=dev)
    (Xr, Xq), = list(activation_chunks(cfg, device=dev))
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, cfg.lambda_rel,
                       device=dev)
    s.accumulate(Xr, Xq)
    g = s.solve(W, cfg.mu)
    L = np64(s.inspect("L"))
    qbar_g = np64(s.inspect("qbar"))
    alpha_g = np64(s.inspect("alpha"))
    lam2_g = float(s.inspect("lam2")[0])
    pres_g = np64(s.inspect("path_resid"))
    s.close()
    codes_g, res_g, win_g = np64(g.codes), np64(g.residuals), np64(g.winner)
    Wn = np64(W)
    Xqn = np64(Xq)
    Xrn = np64(Xr)
    del Xq, Xr
    torch.cuda.empty_cache()
    print("[full c2] GPU layer done; oracle Gram on the host", flush=True)

    # oracle: full Gram and factor, then a column sample
    G = orc.gram(Xqn)
    lam2 = orc.damping(G, cfg.lambda_rel)
    R = orc.cholesky_upper(G + lam2 * np.eye(cfg.m))
    del G
    S, Z = orc.scales_zeros(Wn, cfg.bits, cfg.group)
    cols = np.sort(np.random.default_rng(2024).choice(cfg.n, N_COLS, replace=False))
    V = orc.relaxed_solution(Wn[cols], Xrn, Xqn, cfg.mu, lam2, R)
    qb = orc.centres(V, S[cols], Z[cols], cfg.group)
    qbar_full = np.zeros((cfg.n, cfg.m))
    qbar_full[cols] = qb
    print("[full c2] oracle factor and centres done; decoding the sample", flush=True)
    dec = orc.decode(R, qbar_full, S, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, columns=cols)

    # scales / zeros: every column, bit-equal
    assert np.array_equal(np64(g.scales), S) and np.array_equal(np64(g.zeros), Z)
    # damping and factor
    assert abs(lam2_g - lam2) <= 1e-12 * lam2
    colnorm = np.sqrt(np.sum(R ** 2, axis=0))
    errR = float(np.max(np.abs(L.T - R) / colnorm[None, :]))
    assert errR < 1e-9, errR
    # centres and temperatures of the sample
    errq = float(np.max(np.abs(qbar_g[cols] - qb)))
    assert errq < 1e-6, errq
    assert np.allclose(alpha_g[cols], dec.alpha, rtol=1e-9)
    # codes: the winners' code vectors; a differing one must start at a near-tie
    frac = float((codes_g[cols] == dec.codes).mean())
    Sx = orc.expand_groups(S[cols], cfg.m, cfg.group)
    for t, j in enumerate(cols):
        if win_g[j] == dec.winner[t] and not np.array_equal(codes_g[j], dec.codes[t]):
            assert first_divergence_is_tie(R, qb[t], Sx[t], cfg.bits, dec.alpha[t],
                                           cfg.klein_seed, int(j), int(win_g[j]), codes_g[j],
                                           dec.codes[t])
    assert frac >= 0.999, frac
    # residuals: every candidate of the sample, and the winners
    rel = np.abs(pres_g[cols] - dec.path_resid) / np.abs(dec.path_resid)
    worst, nwin = check_residuals(res_g[cols], win_g[cols], dec.residuals, dec.winner)
    print(f"[full c2] R err {errR:.2e}, qbar err {errq:.2e}, code agreement {frac:.6f}, "
          f"candidate residual max rel err {rel.max():.2e}, winner mismatches {nwin}", flush=True)
    assert float(np.median(rel)) <= 1e-4
    # every GPU winner is the first minimum of its own candidate residuals
    assert np.array_equal(win_g, np.argmin(pres_g, axis=1))
    assert np.array_equal(res_g, pres_g[np.arange(cfg.n), win_g])
    assert int(codes_g.max()) <= (1 << cfg.bits) - 1
