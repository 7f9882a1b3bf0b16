"""ojbkq_quantize_layer_noalloc (the one-shot call on the library's static
scratch) against ojbkq_quantize_layer with a torch workspace: two calls in a
row on one GPU, the second on a smaller layer, must each equal the
workspace call bit for bit (same kernels on the same inputs); a layer too
large for the scratch is rejected before anything is enqueued."""

import ctypes

import pytest
import torch

import paper_2602_08376_amd as ok
from synth import CONFIGS, LayerConfig, make_layer

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ok.library()


def small(m, n, T, bits, group, K, seed):
    return LayerConfig(key=f"na{m}x{n}", title="no-alloc", n=n, m=m, T=T, bits=bits,
                       group=group, K=K, mus=(0.5,), w_std=0.02, kind="heavy", data_seed=seed,
                       klein_seed=seed + 5, noise=0.02)


def same(a, b):
    for f in ("codes", "scales", "zeros", "residuals", "winner"):
        assert torch.equal(getattr(a, f), getattr(b, f)), f


def test_noalloc_equals_workspace_call_twice():
    for cfg, mu in ((small(600, 300, 2000, 4, 128, 8, 91), 0.5), (CONFIGS["c1"], 0.5),
                    (small(97, 33, 250, 3, 32, 5, 92), 0.0)):
        W, Xr, Xq = make_layer(cfg, device=DEV)
        print(f"[noalloc] {cfg.key} mu={mu}", flush=True)
        a = ok.quantize_layer_noalloc(W, Xr, Xq, mu, cfg.bits, cfg.group, cfg.K, cfg.klein_seed,
                                      cfg.lambda_rel)
        b = ok.quantize_layer(W, Xr, Xq, mu, cfg.bits, cfg.group, cfg.K, cfg.klein_seed,
                              cfg.lambda_rel)
        torch.cuda.synchronize()
        same(a, b)
    # act order through the static scratch as well
    cfg = small(200, 90, 700, 4, 64, 4, 93)
    W, Xr, Xq = make_layer(cfg, device=DEV)
    a = ok.quantize_layer_noalloc(W, Xr, Xq, 0.5, 4, 64, 4, cfg.klein_seed, act_order=True)
    b = ok.quantize_layer(W, Xr, Xq, 0.5, 4, 64, 4, cfg.klein_seed, act_order=True)
    torch.cuda.synchronize()
    same(a, b)
    assert torch.equal(a.perm, b.perm)


def test_noalloc_rejects_layers_beyond_the_scratch():
    lib = ok.library()
    p = ok._params(4096, 4096, 4, 128, 16, 0.5, 0.01, 0)
    assert lib.ojbkq_workspace_bytes(ctypes.byref(p)) > ok.NOALLOC_SCRATCH_BYTES
    rc = lib.ojbkq_quantize_layer_noalloc(ctypes.byref(p), 1, None, 1, 10, 10, None, 1, 1, 1, 1,
                                          None, None)
    assert rc == -1
    assert "static scratch" in lib.ojbkq_last_error().decode()
