"""GPU parity of the quantized layer in use: packed codes (bit-exact) and the
dequantize-and-multiply product against the CPU oracle (``oracle/infer.py``),
through the C ABI."""

import numpy as np
import pytest
import torch

import paper_2602_08376_amd as ok
from oracle import infer as oi
from oracle import ojbkq as orc
from parity import np64
from synth import LayerConfig, make_layer

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ok.library()


@pytest.mark.parametrize("bits", range(1, 9))
def test_pack_codes_bit_exact(bits):
    rng = np.random.default_rng(100 + bits)
    codes = rng.integers(0, 1 << bits, size=(37, 301), dtype=np.uint8)
    g = ok.pack_codes(torch.from_numpy(codes).to(DEV), bits)
    torch.cuda.synchronize()
    got = g.cpu().numpy().view(np.uint32)
    assert np.array_equal(got, oi.pack_codes(codes, bits))


def _random_quantized(n, m, bits, group, seed):
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((n, m)) * 0.02).astype(np.float32)
    S, Z = orc.scales_zeros(W, bits, group)
    codes = rng.integers(0, 1 << bits, size=(n, m), dtype=np.uint8)
    return codes, S, Z


@pytest.mark.parametrize("n,m,T,bits,group", [
    (300, 200, 257, 4, 32),     # ragged channels, features (one ragged k step) and tokens
    (130, 512, 300, 3, 128),    # 3-bit fields straddling words
    (64, 96, 128, 8, 32),       # 8-bit fields, a ragged 64-deep stage (and products whose
                                #   one-step fp16 rounding differs from the two-step one)
    (64, 96, 128, 8, 16),       # groups of 16
    (70, 160, 90, 1, 32),       # 1-bit fields: a 16-code run starts at bit 0 or 16
    (100, 192, 200, 5, 64),     # 5-, 6-, 7-bit fields straddling words
    (33, 320, 77, 6, 32),
    (48, 224, 130, 7, 32),
    (256, 256, 256, 4, 32),     # exactly one tile, interior stages only
    (512, 1024, 768, 4, 128),   # several whole tiles in both directions
    (768, 512, 512, 3, 64),
    (257, 129, 33, 2, 0),       # one group per column, m not a multiple of 16
    (16, 4096, 1000, 4, 128),   # a long contraction
])
def test_dequant_matmul_matches_oracle(n, m, T, bits, group):
    codes, S, Z = _random_quantized(n, m, bits, group, n + m + T)
    rng = np.random.default_rng(7)
    scale = np.exp(rng.standard_normal((m, 1))).astype(np.float32)
    X16 = (rng.standard_normal((m, T)).astype(np.float32) * scale).astype(np.float16)
    P = ok.pack_codes(torch.from_numpy(codes).to(DEV), bits)
    args = (P, torch.from_numpy(S).to(DEV), torch.from_numpy(Z).to(DEV), m, bits, group,
            torch.from_numpy(X16).to(DEV))
    # W_hat formed once in a workspace, and dequantized tile by tile: the same
    # weights and the same sums in the same order, so the same bits
    Y = ok.dequant_matmul(*args, workspace=True)
    Y_tiles = ok.dequant_matmul(*args, workspace=False)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y_tiles)
    W16 = oi.dequantize_fp16(codes, S, Z, group)
    ref = oi.dequant_matmul(W16, X16)
    bound = oi.summation_bound(W16, X16)
    err = np.abs(Y.cpu().numpy().astype(np.float64) - ref)
    print(f"[dequant {n}x{m}x{T} b{bits} g{group}] max err / bound {np.max(err / (bound + 1e-300)):.3f}")
    assert np.all(err <= bound + 1e-30)


@pytest.mark.parametrize("n,m,bits,group", [
    (70, 200, 4, 32),    # a ragged last stage: a run cut at m, runs wholly past it
    (33, 96, 8, 16),
    (50, 160, 1, 32),
    (40, 192, 3, 64),
    (300, 100, 2, 0),    # m not a multiple of 16, channels past one tile
    (64, 256, 6, 128),
])
def test_dequant_matmul_identity_gives_w_hat(n, m, bits, group):
    # X = I: every output element is one weight times 1 plus zeros, so Y is
    # W_hat itself and both forms of the product must reproduce the oracle's
    # fp16(fp32(s (q - z))) bit for bit
    codes, S, Z = _random_quantized(n, m, bits, group, 3 * n + m + bits)
    P = ok.pack_codes(torch.from_numpy(codes).to(DEV), bits)
    X16 = torch.eye(m, dtype=torch.float16, device=DEV)
    args = (P, torch.from_numpy(S).to(DEV), torch.from_numpy(Z).to(DEV), m, bits, group, X16)
    want = oi.dequantize_fp16(codes, S, Z, group).astype(np.float32)
    for ws in (True, False):
        Y = ok.dequant_matmul(*args, workspace=ws)
        torch.cuda.synchronize()
        assert np.array_equal(Y.cpu().numpy(), want), f"workspace={ws}"


def test_dequant_matmul_codes_past_the_end_stay_out():
    # the last group's grid overflows fp16 at code 0 (5000 (0 - 15) = -75000)
    # while its real codes 13..15 give finite weights: the packing's zero
    # bits past m, dequantized with that group, would be -inf, and -inf times
    # a zero activation is NaN.  Both forms must leave them out.
    n, m, T, bits, group = 40, 100, 64, 4, 32
    codes, S, Z = _random_quantized(n, m, bits, group, 17)
    rng = np.random.default_rng(18)
    codes[:, 96:] = rng.integers(13, 16, size=(n, 4), dtype=np.uint8)
    S[:, 3] = 5000.0
    Z[:, 3] = 15.0
    X16 = rng.standard_normal((m, T)).astype(np.float16)
    P = ok.pack_codes(torch.from_numpy(codes).to(DEV), bits)
    args = (P, torch.from_numpy(S).to(DEV), torch.from_numpy(Z).to(DEV), m, bits, group,
            torch.from_numpy(X16).to(DEV))
    W16 = oi.dequantize_fp16(codes, S, Z, group)
    assert np.all(np.isfinite(W16))
    ref = oi.dequant_matmul(W16, X16)
    bound = oi.summation_bound(W16, X16)
    for ws in (True, False):
        Y = ok.dequant_matmul(*args, workspace=ws).cpu().numpy()
        assert np.all(np.isfinite(Y)), f"workspace={ws}"
        assert np.all(np.abs(Y.astype(np.float64) - ref) <= bound + 1e-30), f"workspace={ws}"


def test_dequant_matmul_workspace_errors():
    codes, S, Z = _random_quantized(40, 96, 4, 32, 5)
    P = ok.pack_codes(torch.from_numpy(codes).to(DEV), 4)
    X16 = torch.zeros(96, 50, dtype=torch.float16, device=DEV)
    args = (P, torch.from_numpy(S).to(DEV), torch.from_numpy(Z).to(DEV), 96, 4, 32, X16)
    need = ok.library().ojbkq_dequant_matmul_workspace_bytes(40, 96)
    assert need == 40 * 128 * 2                  # rows padded to a whole 64-feature stage
    small = torch.empty(need - 1, dtype=torch.uint8, device=DEV)
    with pytest.raises(ok.OjbkqError) as ei:
        ok.dequant_matmul(*args, workspace=small)
    assert ei.value.status == -2                  # OJBKQ_ENOSPACE
    buf = torch.empty(need + 16, dtype=torch.uint8, device=DEV)
    with pytest.raises(ok.OjbkqError) as ei:
        ok.dequant_matmul(*args, workspace=buf[1:])   # misaligned
    assert ei.value.status == -1                  # OJBKQ_EINVAL
    assert torch.equal(ok.dequant_matmul(*args, workspace=buf[16:]),
                       ok.dequant_matmul(*args, workspace=False))


def test_quantized_layer_forward():
    """Codes, scales and zeros from the quantize call, packed, applied to X~."""
    cfg = LayerConfig(key="t", title="t", n=96, m=256, T=640, bits=4, group=128, K=4,
                      mus=(0.5,), w_std=0.02, kind="heavy", data_seed=71, klein_seed=3, noise=0.02)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    q = ok.quantize_layer(W, Xr, Xq, 0.5, cfg.bits, cfg.group, cfg.K, cfg.klein_seed)
    X16 = Xq.half()
    P = ok.pack_codes(q.codes, cfg.bits)
    Y = ok.dequant_matmul(P, q.scales, q.zeros, cfg.m, cfg.bits, cfg.group, X16)
    torch.cuda.synchronize()
    W16 = oi.dequantize_fp16(q.codes.cpu().numpy(), np64(q.scales), np64(q.zeros), cfg.group)
    x16 = X16.cpu().numpy()
    ref = oi.dequant_matmul(W16, x16)
    assert np.all(np.abs(Y.cpu().numpy() - ref) <= oi.summation_bound(W16, x16) + 1e-30)
    ones = torch.ones(cfg.n, ok.num_groups(cfg.m, 40), dtype=torch.float32, device=DEV)
    with pytest.raises(ok.OjbkqError) as ei:     # groups of 40: not a multiple of 16
        ok.dequant_matmul(P, ones, ones, cfg.m, cfg.bits, 40, X16)
    assert ei.value.code == "EINVAL"
