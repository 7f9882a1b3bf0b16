"""GPU parity of the weight permutation (act order) through the C ABI.

The decode order is a sort of diag(X~^T X~); the GPU and the oracle form
that diagonal with different summation orders, so features whose diagonals
agree to rounding may be ordered either way.  The tests therefore check the
GPU's order against the oracle's diagonal (a valid increasing order, equal to
the oracle's own wherever the keys are apart), then run the oracle on the
GPU's order and compare codes, scales, zeros and residuals element by element
to the usual bar.
"""

import numpy as np
import pytest
import torch

import paper_2602_08376_amd as ok
from oracle import infer as oi
from oracle import ojbkq as orc
from parity import GRAM_RTOL, SCALE_RTOL, check_layer_strict, np64
from synth import LayerConfig, make_layer

pytestmark = pytest.mark.gpu
DEV = "cuda"
# diagonal entries this close may be ordered either way: the GPU sorts its
# own Gram diagonal, whose relative error is that of the int8 token sums
KEY_RTOL = GRAM_RTOL["int8"]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ok.library()


def cfg_of(m, n, T, bits, group, K, seed, mu=0.5, sparsity=0.0):
    return LayerConfig(key=f"a{m}x{n}", title="act order", n=n, m=m, T=T, bits=bits, group=group,
                       K=K, mus=(mu,), w_std=0.02, kind="heavy", data_seed=seed,
                       klein_seed=seed + 3, outliers=2, outlier_gain=20.0, noise=0.02,
                       sparsity=sparsity)


def check_perm(perm, G_o):
    """perm is a permutation that sorts diag(G_o) increasingly; where it
    differs from the oracle's order, the keys involved are equal to rounding."""
    d = np.diag(G_o)
    m = d.shape[0]
    assert sorted(perm.tolist()) == list(range(m)), "not a permutation"
    dp = d[perm]
    assert np.all(dp[1:] >= dp[:-1] - KEY_RTOL * np.abs(dp[1:])), "not an increasing order"
    ref = orc.act_order_perm(G_o)
    bad = np.nonzero(perm != ref)[0]
    for p in bad:
        assert abs(d[perm[p]] - d[ref[p]]) <= KEY_RTOL * abs(d[ref[p]]), \
            f"position {p}: feature {perm[p]} vs {ref[p]} with distinct keys"
    return len(bad)


def paths_of(s):
    return np64(s.path_codes()), np64(s.inspect("path_resid"))


def staged(cfg, W, Xr, Xq, mu, mode, one_shot):
    """The solve of a one-shot act-order call through the staged calls (W
    bound, one chunk): bit-equal results, and every candidate's codes."""
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, cfg.lambda_rel,
                       device=DEV, act_order=mode)
    s.set_weights(W)
    s.accumulate(None if mu == 1.0 else Xr, Xq)
    g = s.solve(W, mu)
    paths = paths_of(s)
    s.close()
    for f in ("codes", "scales", "zeros", "residuals", "winner", "perm"):
        assert torch.equal(getattr(g, f), getattr(one_shot, f)), f
    return paths


def check_against_oracle(cfg, g, W, Xr, Xq, mu, paths, G_o=None, static=False):
    perm = np64(g.perm).astype(np.int64)
    Xq_np = np64(Xq)
    G_o = orc.gram(Xq_np) if G_o is None else G_o
    moved = check_perm(perm, G_o)
    o = orc.quantize_layer(np64(W), np64(Xr), Xq_np, mu, cfg.bits, cfg.group, cfg.K,
                           cfg.klein_seed, lambda_rel=cfg.lambda_rel, G=G_o, perm=perm,
                           static_groups=static)
    S, Z = np64(g.scales), np64(g.zeros)
    assert np.array_equal(S, o.scales), "scales differ"
    assert np.array_equal(Z, o.zeros), "zero points differ"
    assert np.all(np.abs(S - o.scales) <= SCALE_RTOL * np.abs(o.scales))
    codes = np64(g.codes)
    assert codes.max() <= (1 << cfg.bits) - 1
    grp = perm // orc.group_size(cfg.m, cfg.group) if static else cfg.group
    tag = (f"act order{' static' if static else ''} {cfg.key} b{cfg.bits} g{cfg.group} K{cfg.K} "
           f"mu={mu}, order moved at {moved} positions")
    st = check_layer_strict(o, g, paths[0], paths[1], cfg.bits, cfg.klein_seed, grp, perm=perm,
                            tag=tag)
    assert st["agreement"] >= 0.999
    return o


@pytest.mark.parametrize("m,n,T,bits,group,K,seed,mu", [
    (200, 150, 700, 4, 128, 6, 61, 0.5),    # 2 n > m: Q = L + (1 - mu) (L^-1 E)^T route
    (300, 140, 900, 3, 64, 4, 62, 0.0),     # direct route, U = W E^T formed from E
    (300, 40, 900, 4, 128, 5, 63, 0.5),     # 5 n <= 2 m: U accumulated projected
    (33, 2, 80, 8, 16, 5, 64, 0.25),        # ragged groups of 16, 8-bit box
    (130, 5, 300, 2, 0, 3, 65, 1.0),        # one group per column, no cross term
    (1, 3, 9, 2, 128, 2, 66, 0.5),          # a single feature
])
def test_act_order_layer_matches_oracle(m, n, T, bits, group, K, seed, mu):
    cfg = cfg_of(m, n, T, bits, group, K, seed, mu)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    g = ok.quantize_layer(W, Xr, Xq, mu, bits, group, K, cfg.klein_seed, cfg.lambda_rel,
                          act_order=True)
    paths = staged(cfg, W, Xr, Xq, mu, True, g)
    check_against_oracle(cfg, g, W, Xr, Xq, mu, paths)


def test_act_order_heavy_tailed_m1024():
    """A slice of the attention workload (heavy-tailed channels), K = 16."""
    cfg = cfg_of(1024, 40, 4096, 4, 128, 16, 67)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    g = ok.quantize_layer(W, Xr, Xq, 0.5, 4, 128, 16, cfg.klein_seed, cfg.lambda_rel,
                          act_order=True)
    paths = staged(cfg, W, Xr, Xq, 0.5, True, g)
    o = check_against_oracle(cfg, g, W, Xr, Xq, 0.5, paths)
    plain = orc.quantize_layer(np64(W), np64(Xr), np64(Xq), 0.5, 4, 128, 16, cfg.klein_seed,
                               lambda_rel=cfg.lambda_rel)
    print(f"[act order m1024] mean residual {o.residuals.mean():.4e} vs plain order "
          f"{plain.residuals.mean():.4e}")


def test_act_order_staged_sweep_and_chunks():
    """Token chunks with and without a cross term, then two knobs on one
    factor: the order is fixed at the first solve and reused."""
    cfg = cfg_of(260, 90, 1500, 4, 64, 4, 68)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, device=DEV,
                       act_order=True)
    s.accumulate(Xr[:, :700], Xq[:, :700])
    s.accumulate(None, Xq[:, 700:1100])
    s.accumulate(Xr[:, 1100:], Xq[:, 1100:])
    xr = Xr.clone()
    xr[:, 700:1100] = Xq[:, 700:1100]       # the chunk without a cross term has X = X~
    G_o = orc.gram(np64(Xq))
    perms = []
    for mu in (0.5, 0.0):
        g = s.solve(W, mu)
        torch.cuda.synchronize()
        assert torch.equal(s.inspect("perm"), g.perm)
        perms.append(np64(g.perm))
        check_against_oracle(cfg, g, W, xr, Xq, mu, paths_of(s), G_o=G_o)
    assert np.array_equal(perms[0], perms[1])
    s.close()
    plain = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, device=DEV)
    plain.accumulate(Xr, Xq)
    plain.solve(W, 0.5)
    with pytest.raises(ok.OjbkqError) as ei:
        plain.inspect("perm")
    assert ei.value.code == "EINVAL"
    plain.close()


@pytest.mark.parametrize("n,m,T,bits,group", [
    (96, 256, 300, 4, 128),     # act-order codes of a quantize call
    (70, 200, 133, 3, 32),      # ragged channels, features and tokens, 3-bit fields
    (256, 512, 512, 4, 128),    # whole 256 x 256 tiles: every stage gathered by the kernels'
                                #   own loads (rows of the next stage read a step ahead)
    (320, 640, 300, 3, 64),     # one whole tile beside ragged ones
])
def test_packed_product_in_decode_order(n, m, T, bits, group):
    """Codes packed in decode order (position p holds feature perm[p]) and
    multiplied with the rows of X gathered alike: the packing is bit-exact and
    the product within the fp32 summation bound of W_hat X in either order."""
    cfg = cfg_of(m, n, T, bits, group, 2, 69 + bits)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    q = ok.quantize_layer(W, Xr, Xq, 0.5, bits, group, 2, cfg.klein_seed, cfg.lambda_rel,
                          act_order=True)
    P = ok.pack_codes(q.codes, bits, q.perm)
    X16 = Xq.half()
    Y = ok.dequant_matmul(P, q.scales, q.zeros, m, bits, group, X16, q.perm)
    Y_tiles = ok.dequant_matmul(P, q.scales, q.zeros, m, bits, group, X16, q.perm,
                                workspace=False)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y_tiles)              # W_hat once or per tile: the same bits
    perm = np64(q.perm).astype(np.int64)
    codes = np64(q.codes)
    assert np.array_equal(P.cpu().numpy().view(np.uint32), oi.pack_codes(codes[:, perm], bits))
    W16 = oi.dequantize_fp16(codes[:, perm], np64(q.scales), np64(q.zeros), group)
    x16 = X16.cpu().numpy()[perm]
    ref = oi.dequant_matmul(W16, x16)
    bound = oi.summation_bound(W16, x16)
    err = np.abs(Y.cpu().numpy().astype(np.float64) - ref)
    print(f"[act order product {n}x{m}x{T} b{bits}] max err / bound "
          f"{np.max(err / (bound + 1e-300)):.3f}")
    assert np.all(err <= bound + 1e-30)
    # the same weights in W's order: feature i on the group of its position
    gidx = orc.feature_groups(perm, group)
    W_orig = orc.dequantize_by_feature(codes, np64(q.scales), np64(q.zeros), gidx)
    assert np.array_equal(W_orig.astype(np.float32).astype(np.float16)[:, perm], W16)


@pytest.mark.parametrize("m,n,T,bits,group,K,seed,mu", [
    (200, 150, 700, 4, 64, 6, 71, 0.5),     # Q route, groups of 64 scattered over positions
    (300, 140, 900, 3, 128, 4, 72, 0.0),    # direct route, ragged last group
    (300, 40, 900, 4, 32, 5, 73, 0.5),      # projected route
    (33, 2, 80, 8, 16, 5, 74, 0.25),        # ragged groups of 16
    (130, 5, 300, 2, 0, 3, 75, 1.0),        # one group: the same as position groups
])
def test_static_groups_layer_matches_oracle(m, n, T, bits, group, K, seed, mu):
    """act_order = "static": the scale groups stay runs of g features in W's
    order, so the decoder reads each row's scale through the group index of
    its position, and the scales equal those of the plain call."""
    cfg = cfg_of(m, n, T, bits, group, K, seed, mu)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    g = ok.quantize_layer(W, Xr, Xq, mu, bits, group, K, cfg.klein_seed, cfg.lambda_rel,
                          act_order="static")
    plain = ok.quantize_layer(W, Xr, Xq, mu, bits, group, K, cfg.klein_seed, cfg.lambda_rel)
    paths = staged(cfg, W, Xr, Xq, mu, "static", g)
    assert torch.equal(g.scales, plain.scales) and torch.equal(g.zeros, plain.zeros)
    check_against_oracle(cfg, g, W, Xr, Xq, mu, paths, static=True)


def test_static_groups_staged_and_plain_product():
    """Static groups through the staged calls (chunks, two knobs on one
    factor), then the plain packed product (no perm) against the oracle."""
    cfg = cfg_of(256, 96, 1200, 4, 64, 4, 76)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed, device=DEV,
                       act_order="static")
    s.accumulate(Xr[:, :500], Xq[:, :500])
    s.accumulate(Xr[:, 500:], Xq[:, 500:])
    G_o = orc.gram(np64(Xq))
    for mu in (0.5, 0.0):
        q = s.solve(W, mu)
        torch.cuda.synchronize()
        check_against_oracle(cfg, q, W, Xr, Xq, mu, paths_of(s), G_o=G_o, static=True)
    s.close()
    X16 = Xq.half()
    P = ok.pack_codes(q.codes, cfg.bits)
    Y = ok.dequant_matmul(P, q.scales, q.zeros, cfg.m, cfg.bits, cfg.group, X16)
    torch.cuda.synchronize()
    W16 = oi.dequantize_fp16(np64(q.codes), np64(q.scales), np64(q.zeros), cfg.group)
    x16 = X16.cpu().numpy()
    err = np.abs(Y.cpu().numpy().astype(np.float64) - oi.dequant_matmul(W16, x16))
    assert np.all(err <= oi.summation_bound(W16, x16) + 1e-30)


@pytest.mark.parametrize("mode", [True, "static"])
def test_act_order_ties_and_degenerate_channels(mode):
    """Equal keys and degenerate channels: two duplicated activation rows
    (equal diagonals, which the GPU may order either way), a dead channel
    (zero diagonal, decided last), an all-zero weight group, 1-bit codes and
    K = 0 (Babai only)."""
    cfg = cfg_of(96, 12, 400, 1, 32, 0, 77)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    Xq, Xr, W = Xq.clone(), Xr.clone(), W.clone()
    Xq[9] = Xq[5]
    Xr[9] = Xr[5]
    Xq[40] = 0.0
    Xr[40] = 0.0
    W[3, 32:64] = 0.0
    g = ok.quantize_layer(W, Xr, Xq, 0.5, 1, 32, 0, cfg.klein_seed, cfg.lambda_rel,
                          act_order=mode)
    paths = staged(cfg, W, Xr, Xq, 0.5, mode, g)
    perm = np64(g.perm)
    assert perm[0] == 40                   # the zero diagonal comes first: decided last
    assert abs(int(np.nonzero(perm == 5)[0][0]) - int(np.nonzero(perm == 9)[0][0])) == 1
    assert int(g.winner.max()) == 0
    check_against_oracle(cfg, g, W, Xr, Xq, 0.5, paths, static=(mode == "static"))
