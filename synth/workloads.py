"""Synthetic layers shaped like the LLM workloads the paper quantizes.

The paper calibrates on 128 sequences x 2048 tokens of C4 text drawn through
Llama/Qwen/Mistral layers (Experiments section).  Neither the text nor the
weights are available here, so these generators stand in for them: random
weights with the stated spread, and activations with heavy-tailed per-channel
scales, a few outlier channels and a small perturbation playing the part of the
runtime activations of a partially quantized network.

Layout (as stored and passed over the C ABI): W is [n, m] (output channels x
input features, the nn.Linear layout); X_ref and X_q are [m, T] (features x
tokens).  Everything is float32.  Generation is seeded through torch.Generator
on the device the tensors are made on, so a GPU run and the CPU oracle see the
same arrays when the oracle receives host copies of the GPU tensors.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Iterator, Optional, Sequence, Tuple

import torch


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    key: str
    title: str
    n: int                # output channels = independent box-constrained ILS problems
    m: int                # input features = lattice dimension
    T: int                # calibration tokens
    bits: int
    group: int
    K: int                # Klein samples; K + 1 candidates per column
    mus: Tuple[float, ...]  # JTA knob value(s)
    w_std: float
    kind: str             # "tiny" or "heavy"
    data_seed: int
    klein_seed: int = 0
    lambda_rel: float = 0.01
    chunks: int = 1       # token chunks the Gram is accumulated over
    outliers: int = 0     # tiny kind: number of outlier channels
    outlier_gain: float = 1.0
    noise: float = 0.0    # X_q - X_ref noise, relative to the channel scale
    sparsity: float = 0.0  # fraction of near-zero activations (post-SiLU-like)

    @property
    def mu(self) -> float:
        return self.mus[0]

    @property
    def paths(self) -> int:
        return self.n * (self.K + 1)


CONFIGS = {
    "c1": LayerConfig(
        key="c1", title="tiny BILS layer 64x128, 512 tokens",
        n=64, m=128, T=512, bits=4, group=128, K=4, mus=(0.5,), w_std=0.02,
        kind="tiny", data_seed=0, klein_seed=0, outliers=4, outlier_gain=20.0, noise=0.05),
    "c2": LayerConfig(
        key="c2", title="Llama-7B-shaped attention projection 4096x4096, 262144 tokens",
        n=4096, m=4096, T=262144, bits=4, group=128, K=16, mus=(0.5,), w_std=0.02,
        kind="heavy", data_seed=2, noise=0.02),
    "c3": LayerConfig(
        key="c3", title="Llama-7B-shaped MLP down_proj 4096x11008, 262144 tokens",
        n=4096, m=11008, T=262144, bits=3, group=128, K=16, mus=(0.5,), w_std=0.015,
        kind="heavy", data_seed=3, noise=0.02, sparsity=0.6),
    "c4": LayerConfig(
        key="c4", title="Llama-13B-shaped up_proj 13824x5120, 262144 tokens",
        n=13824, m=5120, T=262144, bits=3, group=128, K=32, mus=(0.0, 0.5, 1.0), w_std=0.02,
        kind="heavy", data_seed=4, noise=0.02),
    "c5": LayerConfig(
        key="c5", title="70B-shaped MLP down_proj shard 8192x28672, 131072 tokens in 8 chunks",
        n=8192, m=28672, T=131072, bits=4, group=128, K=16, mus=(0.5,), w_std=0.01,
        kind="heavy", data_seed=5, noise=0.02, chunks=8),
}


# The four linear-layer shapes of a Llama-3-8B block (hidden 4096, eight
# key/value heads of 128, MLP 14336), calibrated as in the paper's
# experiments (128 sequences x 2048 tokens, 4-bit, group 128) with the JTA
# knob mu = 0.6 that its main experiments fix.  K is the default the
# ablations settle on (5); the K sweep of bench.py overrides it.
LLAMA3_8B = {
    "l3_qo": LayerConfig(
        key="l3_qo", title="Llama-3-8B-shaped q/o_proj 4096x4096, 262144 tokens",
        n=4096, m=4096, T=262144, bits=4, group=128, K=5, mus=(0.6,), w_std=0.02,
        kind="heavy", data_seed=11, noise=0.02),
    "l3_kv": LayerConfig(
        key="l3_kv", title="Llama-3-8B-shaped k/v_proj 1024x4096, 262144 tokens",
        n=1024, m=4096, T=262144, bits=4, group=128, K=5, mus=(0.6,), w_std=0.02,
        kind="heavy", data_seed=12, noise=0.02),
    "l3_gate_up": LayerConfig(
        key="l3_gate_up", title="Llama-3-8B-shaped gate/up_proj 14336x4096, 262144 tokens",
        n=14336, m=4096, T=262144, bits=4, group=128, K=5, mus=(0.6,), w_std=0.02,
        kind="heavy", data_seed=13, noise=0.02),
    "l3_down": LayerConfig(
        key="l3_down", title="Llama-3-8B-shaped down_proj 4096x14336, 262144 tokens",
        n=4096, m=14336, T=262144, bits=4, group=128, K=5, mus=(0.6,), w_std=0.015,
        kind="heavy", data_seed=14, noise=0.02, sparsity=0.6),
}


def config_by_name(name: str) -> LayerConfig:
    return CONFIGS[name] if name in CONFIGS else LLAMA3_8B[name]


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def channel_scales(cfg: LayerConfig, m: Optional[int] = None, device="cpu") -> torch.Tensor:
    """Per-input-channel activation scale sigma_c (float32, [m])."""
    m = cfg.m if m is None else m
    g = _gen(device, cfg.data_seed * 7919 + 11)
    if cfg.kind == "tiny":
        sig = torch.ones(m, dtype=torch.float32, device=device)
        idx = torch.randperm(m, generator=g, device=device)[: cfg.outliers]
        sig[idx] = cfg.outlier_gain
        return sig
    # heavy-tailed: log-normal(0, 1) scales, 1% of channels (rounded) boosted x50
    sig = torch.exp(torch.randn(m, generator=g, device=device, dtype=torch.float32))
    n_out = int(round(0.01 * m))
    idx = torch.randperm(m, generator=g, device=device)[:n_out]
    sig[idx] = sig[idx] * 50.0
    return sig


def make_weights(cfg: LayerConfig, n: Optional[int] = None, m: Optional[int] = None,
                 device="cpu") -> torch.Tensor:
    n = cfg.n if n is None else n
    m = cfg.m if m is None else m
    g = _gen(device, cfg.data_seed * 7919 + 1)
    return torch.randn(n, m, generator=g, device=device, dtype=torch.float32) * cfg.w_std


def activation_chunks(cfg: LayerConfig, m: Optional[int] = None, T: Optional[int] = None,
                      chunks: Optional[int] = None, device="cpu",
                      rows_per_draw: int = 1024) -> Iterator[Tuple[torch.Tensor, torch.Tensor]]:
    """Yield (X_ref_c, X_q_c) token chunks, each [m, T / chunks] float32.

    Rows are drawn in slabs of ``rows_per_draw`` channels so that the
    temporaries stay small for the 11008- and 28672-channel layers.
    """
    m = cfg.m if m is None else m
    T = cfg.T if T is None else T
    chunks = cfg.chunks if chunks is None else chunks
    if T % chunks:
        raise ValueError("token count must split evenly into chunks")
    Tc = T // chunks
    sig = channel_scales(cfg, m, device)
    for c in range(chunks):
        g = _gen(device, cfg.data_seed * 7919 + 1000 + c)
        X = torch.empty(m, Tc, dtype=torch.float32, device=device)
        Xq = torch.empty(m, Tc, dtype=torch.float32, device=device)
        for r0 in range(0, m, rows_per_draw):
            r1 = min(m, r0 + rows_per_draw)
            s = sig[r0:r1, None]
            base = torch.randn(r1 - r0, Tc, generator=g, device=device, dtype=torch.float32)
            noise = torch.randn(r1 - r0, Tc, generator=g, device=device, dtype=torch.float32)
            if cfg.kind == "tiny":
                x = base * s
                xq = x + noise * cfg.noise
            else:
                x = base * s
                dn = noise * (s * cfg.noise)
                if cfg.sparsity > 0.0:
                    keep = torch.rand(r1 - r0, Tc, generator=g, device=device) >= cfg.sparsity
                    shrink = torch.where(keep, torch.ones((), device=device),
                                         torch.full((), 0.01, device=device))
                    x = x * shrink
                    dn = dn * shrink
                xq = x + dn
            X[r0:r1] = x
            Xq[r0:r1] = xq
            del base, noise, x, xq
        yield X, Xq


def make_layer(cfg: LayerConfig, n: Optional[int] = None, m: Optional[int] = None,
               T: Optional[int] = None, device="cpu"):
    """Return (W [n,m], X_ref [m,T], X_q [m,T]) for ``cfg`` (one token chunk)."""
    W = make_weights(cfg, n, m, device)
    (X, Xq), = list(activation_chunks(cfg, m, T, 1, device))
    return W, X, Xq


def make_triangular_problem(m: int, n: int, groups: int, seed: int, device="cpu",
                            spread: float = 1.0, coupling: float = 0.3,
                            qbar_lo: float = -1.5, qbar_hi: float = 16.5):
    """Random inputs for the decode stage alone.

    Returns (R [m,m] float64 upper triangular with a positive diagonal,
    qbar [n,m] float64 real-valued centres, S [n,groups] float32 positive scales).
    R = diag(d) (I + U) with log-normal d and a dense strictly upper U of
    size ``coupling / sqrt(m)``: shaped like the factor of a damped Gram of
    heavy-tailed activations, without computing one.
    """
    g = _gen(device, 104729 * seed + 17)
    d = torch.exp(spread * torch.randn(m, generator=g, device=device, dtype=torch.float64))
    U = torch.randn(m, m, generator=g, device=device, dtype=torch.float64) * (coupling / math.sqrt(max(m, 1)))
    U = torch.triu(U, diagonal=1)
    R = d[:, None] * (torch.eye(m, dtype=torch.float64, device=device) + U)
    qbar = qbar_lo + (qbar_hi - qbar_lo) * torch.rand(n, m, generator=g, device=device, dtype=torch.float64)
    S = torch.exp(0.5 * torch.randn(n, groups, generator=g, device=device, dtype=torch.float64) - 4.0)
    return R, qbar, S.to(torch.float32)
