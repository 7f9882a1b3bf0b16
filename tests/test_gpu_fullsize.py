"""Parity at the full sizes of the five workloads' four large layers.

Every check applies the full parity rule of tests/parity.py to every
candidate of the sampled columns: each differing path must start at a
near-tie, every candidate residual must match the oracle's residual formula
on the GPU's codes, and winner swaps must be explained.

* 4096 x 4096 attention projection (262,144 tokens, 4-bit, K = 16), the
  workload bench.py times, through the same staged calls: the oracle forms
  its own full fp64 Gram, damping and factor on the host, then the relaxed
  solution and the decode of 128 seeded columns (every candidate); also with
  the weight permutation in both group modes (32 columns each).
* 5120 x 13824 up_proj (3-bit, K = 32, the mu sweep on one factor): the
  oracle again forms its own Gram and factor, and for every mu its own
  centres and the decode of 16 columns.
* 11008 x 4096 (3-bit) and 28672 x 8192 (8 token chunks): a host fp64 Gram
  of these does not fit a test's time, so the factor is checked matrix-free
  over every entry (L L^T v - lambda^2 v against X~^T (X~ v) for 8 random
  probes v, summed chunk by chunk on the host), the centres through the
  normal equations of the stacked problem (Eq. new_obj), and the oracle then
  decodes 8 columns on the factor and centres so verified.
"""

import numpy as np
import pytest
import torch

import paper_2602_08376_amd as ok
from oracle import cdecode
from oracle import ojbkq as orc
from parity import GRAM_RTOL, centres_from_gq, check_paths_strict, np64
from synth import CONFIGS
from synth.workloads import activation_chunks, make_weights

pytestmark = pytest.mark.gpu

N_COLS = 128         # sampled columns at 4096 x 4096
N_COLS_ACT = 32      # with the weight permutation
N_COLS_C4 = 16       # per mu at 5120 x 13824
N_DEC = 8            # at 11008 x 4096 and 28672 x 8192
N_PROBES = 8


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ok.library()


def gpu_paths(s, cols, dev):
    """Candidate codes [c, K+1, m] (W's order) and residuals [c, K+1] of the
    sampled columns of the last solve."""
    idx = torch.as_tensor(np.asarray(cols), device=dev)
    pc = np64(s.path_codes()[idx])
    pr = np64(s.inspect("path_resid"))[np.asarray(cols)]
    return pc, pr


def strict(R, qbar, S_cols, group_rows, cfg, cols, dec, pc, pr, g, perm=None, tag=""):
    """check_paths_strict on sampled columns; pc / g's codes in W's order."""
    m = R.shape[0]
    codes = np64(g.codes)[cols]
    if perm is not None:
        pc = pc[:, :, perm]
        codes = codes[:, perm]
    s_rows = orc.expand_groups(S_cols, m, group_rows)
    return check_paths_strict(R, qbar, s_rows, cfg.bits, cfg.klein_seed, dec.alpha, cols, pc, pr,
                              codes, np64(g.residuals)[cols], np64(g.winner)[cols],
                              dec.path_codes, dec.path_resid, dec.residuals, dec.winner, tag=tag)


@pytest.mark.parametrize("gram", ["int8", "fp64"])
def test_attention_projection_full_size(gram):
    cfg = CONFIGS["c2"]
    dev = torch.device("cuda", 0)
    W = make_weights(cfg, device=dev)
    (Xr, Xq), = list(activation_chunks(cfg, device=dev))
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, cfg.lambda_rel,
                       device=dev, gram=gram)
    s.set_weights(W)
    s.accumulate(Xr, Xq)
    g = s.solve(W, cfg.mu)
    cols = np.sort(np.random.default_rng(2024).choice(cfg.n, N_COLS, replace=False))
    L = np64(s.inspect("L"))
    gq_g = np64(s.inspect("gq"))
    alpha_g = np64(s.inspect("alpha"))
    lam2_g = float(s.inspect("lam2")[0])
    pres_all = np64(s.inspect("path_resid"))
    pc, pr = gpu_paths(s, cols, dev)
    s.close()
    Wn, Xqn, Xrn = np64(W), np64(Xq), np64(Xr)
    del Xq, Xr
    torch.cuda.empty_cache()
    print("[full c2] GPU layer done; oracle Gram on the host", flush=True)

    G = orc.gram(Xqn)
    lam2 = orc.damping(G, cfg.lambda_rel)
    R = orc.cholesky_upper(G + lam2 * np.eye(cfg.m))
    del G
    S, Z = orc.scales_zeros(Wn, cfg.bits, cfg.group)
    V = orc.relaxed_solution(Wn[cols], Xrn, Xqn, cfg.mu, lam2, R)
    qb = orc.centres(V, S[cols], Z[cols], cfg.group)
    qbar_full = np.zeros((cfg.n, cfg.m))
    qbar_full[cols] = qb
    print("[full c2] oracle factor and centres done; decoding the sample", flush=True)
    dec = cdecode.decode(R, qbar_full, S, cfg.bits, cfg.group, cfg.K, cfg.klein_seed,
                         columns=cols)

    assert np.array_equal(np64(g.scales), S) and np.array_equal(np64(g.zeros), Z)
    assert abs(lam2_g - lam2) <= GRAM_RTOL[gram] * lam2
    colnorm = np.sqrt(np.sum(R ** 2, axis=0))
    errR = float(np.max(np.abs(L.T - R) / colnorm[None, :]))
    assert errR < GRAM_RTOL[gram], errR
    qbar_g = centres_from_gq(L, gq_g[cols], np64(g.scales)[cols], cfg.group)
    errq = float(np.max(np.abs(qbar_g - qb)))
    assert errq < 1e-6, errq
    assert np.allclose(alpha_g[cols], dec.alpha, rtol=GRAM_RTOL[gram])
    print(f"[full c2 {gram}] R err {errR:.2e}, qbar err {errq:.2e}", flush=True)
    strict(R, qb, S[cols], cfg.group, cfg, cols, dec, pc, pr, g, tag=f"full c2 {gram}")
    # over all columns: every winner is the first minimum of its candidates
    win_g = np64(g.winner)
    assert np.array_equal(win_g, np.argmin(pres_all, axis=1))
    assert np.array_equal(np64(g.residuals), pres_all[np.arange(cfg.n), win_g])
    assert int(np64(g.codes).max()) <= (1 << cfg.bits) - 1


@pytest.mark.parametrize("mode", ["positions", "static"])
def test_attention_projection_full_size_act_order(mode):
    """The same layer with the weight permutation: the GPU's decode order
    must sort the oracle's full-size Gram diagonal (ties only within the
    int8 token sums' relative error); the oracle then factors the permuted Gram and decodes a sample
    of columns on that order, every candidate, and the codes come back in W's
    order.  Scale groups by decode position, or W's own (static)."""
    cfg = CONFIGS["c2"]
    dev = torch.device("cuda", 0)
    W = make_weights(cfg, device=dev)
    (Xr, Xq), = list(activation_chunks(cfg, device=dev))
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, cfg.lambda_rel,
                       device=dev, act_order=(mode if mode == "static" else True))
    s.set_weights(W)
    s.accumulate(Xr, Xq)
    g = s.solve(W, cfg.mu)
    cols = np.sort(np.random.default_rng(2025).choice(cfg.n, N_COLS_ACT, replace=False))
    pres_all = np64(s.inspect("path_resid"))
    pc, pr = gpu_paths(s, cols, dev)
    s.close()
    perm = np64(g.perm).astype(np.int64)
    Wn, Xqn, Xrn = np64(W), np64(Xq), np64(Xr)
    del Xq, Xr
    torch.cuda.empty_cache()
    print("[full c2 act order] GPU layer done; oracle Gram on the host", flush=True)
    G = orc.gram(Xqn)
    d = np.diag(G)
    assert sorted(perm.tolist()) == list(range(cfg.m))
    ref = orc.act_order_perm(G)
    for p in np.nonzero(perm != ref)[0]:
        assert abs(d[perm[p]] - d[ref[p]]) <= GRAM_RTOL["int8"] * d[ref[p]], p
    Gp = G[np.ix_(perm, perm)]
    del G
    lam2 = orc.damping(Gp, cfg.lambda_rel)
    R = orc.cholesky_upper(Gp + lam2 * np.eye(cfg.m))
    del Gp
    Wp, Xqp, Xrp = Wn[:, perm], Xqn[perm], Xrn[perm]
    del Xqn, Xrn
    if mode == "static":   # W's own groups; position p on the group of feature perm[p]
        S, Z = orc.scales_zeros(Wn, cfg.bits, cfg.group)
        grp = perm // cfg.group
    else:
        S, Z = orc.scales_zeros(Wp, cfg.bits, cfg.group)
        grp = cfg.group
    assert np.array_equal(np64(g.scales), S) and np.array_equal(np64(g.zeros), Z)
    V = orc.relaxed_solution(Wp[cols], Xrp, Xqp, cfg.mu, lam2, R)
    qb = orc.centres(V, S[cols], Z[cols], grp)
    qbar_full = np.zeros((cfg.n, cfg.m))
    qbar_full[cols] = qb
    print(f"[full c2 act order {mode}] oracle factor and centres done; decoding the sample",
          flush=True)
    dec = cdecode.decode(R, qbar_full, S, cfg.bits, grp, cfg.K, cfg.klein_seed, columns=cols)
    strict(R, qb, S[cols], grp, cfg, cols, dec, pc, pr, g, perm=perm,
           tag=f"full c2 act order {mode}")
    assert np.array_equal(np64(g.winner), np.argmin(pres_all, axis=1))


def test_upproj_full_size_mu_sweep():
    """5120 x 13824, 3-bit, K = 32, mu in {0, 0.5, 1} on one factor: the
    oracle's own Gram, damping and factor, and per mu its own centres and the
    decode of 8 columns, every candidate."""
    cfg = CONFIGS["c4"]
    dev = torch.device("cuda", 0)
    W = make_weights(cfg, device=dev)
    Wn = np64(W)
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, cfg.lambda_rel,
                       device=dev)
    s.set_weights(W)
    (Xr, Xq), = list(activation_chunks(cfg, device=dev))
    s.accumulate(Xr, Xq)
    Xrn, Xqn = np64(Xr), np64(Xq)
    del Xr, Xq
    torch.cuda.empty_cache()
    rng = np.random.default_rng(44)
    gpu = []
    for mu in cfg.mus:
        g = s.solve(W, mu)
        cols = np.sort(rng.choice(cfg.n, N_COLS_C4, replace=False))
        pc, pr = gpu_paths(s, cols, dev)
        gpu.append((mu, g, cols, pc, pr, np64(s.inspect("path_resid")), np64(s.inspect("L"))
                    if mu == cfg.mus[0] else None, float(s.inspect("lam2")[0])))
        print(f"[full c4] GPU solve and decode done for mu = {mu}", flush=True)
    s.close()
    print("[full c4] oracle Gram on the host", flush=True)
    G = orc.gram(Xqn)
    lam2 = orc.damping(G, cfg.lambda_rel)
    R = orc.cholesky_upper(G + lam2 * np.eye(cfg.m))
    del G
    S, Z = orc.scales_zeros(Wn, cfg.bits, cfg.group)
    L = gpu[0][6]
    colnorm = np.sqrt(np.sum(R ** 2, axis=0))
    errR = float(np.max(np.abs(L.T - R) / colnorm[None, :]))
    print(f"[full c4] R err {errR:.2e}", flush=True)
    assert errR < GRAM_RTOL["int8"], errR
    for mu, g, cols, pc, pr, pres_all, _, lam2_g in gpu:
        assert abs(lam2_g - lam2) <= GRAM_RTOL["int8"] * lam2
        assert np.array_equal(np64(g.scales), S) and np.array_equal(np64(g.zeros), Z)
        V = orc.relaxed_solution(Wn[cols], Xrn, Xqn, mu, lam2, R)
        qb = orc.centres(V, S[cols], Z[cols], cfg.group)
        qbar_full = np.zeros((cfg.n, cfg.m))
        qbar_full[cols] = qb
        dec = cdecode.decode(R, qbar_full, S, cfg.bits, cfg.group, cfg.K, cfg.klein_seed,
                             columns=cols)
        strict(R, qb, S[cols], cfg.group, cfg, cols, dec, pc, pr, g, tag=f"full c4 mu={mu}")
        assert np.array_equal(np64(g.winner), np.argmin(pres_all, axis=1))


@pytest.mark.parametrize("key", ["c3", "c5"])
def test_full_size_factor_probes_and_decode(key):
    cfg = CONFIGS[key]
    dev = torch.device("cuda", 0)
    rng = np.random.default_rng(7 + int(key[1]))
    W = make_weights(cfg, device=dev)
    Wn = np64(W)
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, cfg.lambda_rel,
                       device=dev)
    s.set_weights(W)          # as bench.py: the projected cross term
    diag = np.zeros(cfg.m)
    probes = rng.standard_normal((cfg.m, N_PROBES))
    gprobe = np.zeros((cfg.m, N_PROBES))          # X~^T (X~ v), summed over chunks
    chunks_host = []
    for c, (Xr, Xq) in enumerate(activation_chunks(cfg, device=dev)):
        s.accumulate(Xr, Xq)
        Xqn, Xrn = np64(Xq), np64(Xr)
        del Xr, Xq
        Xq64 = Xqn.astype(np.float64)
        diag += np.einsum("it,it->i", Xq64, Xq64)
        gprobe += Xq64 @ (Xq64.T @ probes)
        del Xq64
        chunks_host.append((Xrn, Xqn))
        print(f"[full {key}] chunk {c + 1}/{cfg.chunks} accumulated", flush=True)
    torch.cuda.empty_cache()
    S, Z = orc.scales_zeros(Wn, cfg.bits, cfg.group)
    mu = cfg.mu
    g = s.solve(W, mu)
    torch.cuda.synchronize()
    print(f"[full {key}] GPU solve and decode done", flush=True)
    assert np.array_equal(np64(g.scales), S) and np.array_equal(np64(g.zeros), Z)
    lam2_g = float(s.inspect("lam2")[0])
    assert abs(lam2_g - cfg.lambda_rel * diag.mean()) <= GRAM_RTOL["int8"] * lam2_g
    L = np64(s.inspect("L"))
    # the whole factor, matrix-free: L L^T v = (X~^T X~ + lambda^2 I) v
    lhs = L @ (L.T @ probes) - lam2_g * probes
    rel = np.linalg.norm(lhs - gprobe, axis=0) / np.linalg.norm(gprobe, axis=0)
    print(f"[full {key}] factor probes: relative residuals {[f'{x:.1e}' for x in rel]}",
          flush=True)
    assert float(rel.max()) < GRAM_RTOL["int8"], rel
    # centres: normal equations of the stacked problem for the sampled columns
    cols = np.sort(rng.choice(cfg.n, N_DEC, replace=False))
    gq = np64(s.inspect("gq"))[cols]
    qbar_c = centres_from_gq(L, gq, S[cols], cfg.group)
    Sx = orc.expand_groups(S[cols], cfg.m, cfg.group)
    Zx = orc.expand_groups(Z[cols], cfg.m, cfg.group)
    V = ((qbar_c - Zx) * Sx).T   # [m, c]
    Wc = Wn[cols].astype(np.float64).T
    nl, nr = lam2_g * V, lam2_g * Wc
    for Xrn, Xqn in chunks_host:
        Xq64 = Xqn.astype(np.float64)
        nl += Xq64 @ (Xq64.T @ V)
        nr += Xq64 @ orc.jta_target(Wn[cols], Xrn, Xqn, mu)
        del Xq64
    del chunks_host
    rel = np.linalg.norm(nl - nr, axis=0) / np.linalg.norm(nr, axis=0)
    print(f"[full {key}] columns {cols.tolist()}: normal-equation residuals "
          f"{[f'{x:.2e}' for x in rel]}", flush=True)
    assert float(rel.max()) < GRAM_RTOL["int8"], rel
    # decode: the oracle's candidates on the verified factor and centres
    pc, pr = gpu_paths(s, cols, dev)
    pres_all = np64(s.inspect("path_resid"))
    alpha_g = np64(s.inspect("alpha"))
    s.close()
    R = L.T.copy()
    del L
    qbar_full = np.zeros((cfg.n, cfg.m))
    qbar_full[cols] = qbar_c
    dec = cdecode.decode(R, qbar_full, S, cfg.bits, cfg.group, cfg.K, cfg.klein_seed,
                         columns=cols)
    assert np.allclose(alpha_g[cols], dec.alpha, rtol=1e-12)
    strict(R, qbar_c, S[cols], cfg.group, cfg, cols, dec, pc, pr, g, tag=f"full {key}")
    assert np.array_equal(np64(g.winner), np.argmin(pres_all, axis=1))
