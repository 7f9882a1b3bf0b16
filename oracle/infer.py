"""Plain CPU oracle for the quantized layer in use: packed codes and the
product with the dequantized weight W_hat = S (Q - Z) (the Q, S, Z data model
of Sec. 3.2), which forms the activations X~ that layer-by-layer quantization
feeds to the next layer (Sec. 3.1).

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import or call this module.  The GPU
library shares no code with it and never calls it.

Storage conventions (the library's; parity unpinned against the paper, which
fixes no storage format):
  * a packed row is the little-endian bit stream of the row's codes, code i
    at bits [i b, (i + 1) b) counted from bit 0 of 32-bit word 0, zero past
    the last code;
  * W_hat is rounded to float16 as fp16(fp32(s (q - z))): the product in
    float32, then float16, both to nearest even.
"""

from __future__ import annotations

import numpy as np

from .ojbkq import expand_groups, group_size


def packed_words(m: int, bits: int) -> int:
    return (m * bits + 31) // 32


def pack_codes(codes: np.ndarray, bits: int) -> np.ndarray:
    """codes [n, m] (integers < 2^bits) -> [n, packed_words(m, bits)] uint32."""
    codes = np.asarray(codes)
    n, m = codes.shape
    out = np.zeros((n, packed_words(m, bits)), dtype=np.uint32)
    mask = (1 << bits) - 1
    for j in range(n):
        stream = 0                       # the row as one Python integer
        for i in range(m):
            stream |= (int(codes[j, i]) & mask) << (i * bits)
        for w in range(out.shape[1]):
            out[j, w] = (stream >> (32 * w)) & 0xFFFFFFFF
    return out


def unpack_codes(packed: np.ndarray, m: int, bits: int) -> np.ndarray:
    """Inverse of :func:`pack_codes`."""
    packed = np.asarray(packed, dtype=np.uint32)
    n = packed.shape[0]
    out = np.zeros((n, m), dtype=np.uint8)
    mask = (1 << bits) - 1
    for j in range(n):
        stream = 0
        for w in range(packed.shape[1]):
            stream |= int(packed[j, w]) << (32 * w)
        for i in range(m):
            out[j, i] = (stream >> (i * bits)) & mask
    return out


def dequantize_fp16(codes: np.ndarray, S: np.ndarray, Z: np.ndarray, group: int) -> np.ndarray:
    """W_hat [n, m] as float16: fp16(fp32(s (q - z)))."""
    codes = np.asarray(codes)
    m = codes.shape[1]
    Sx = expand_groups(S, m, group).astype(np.float32)
    Zx = expand_groups(Z, m, group).astype(np.float32)
    d = (codes.astype(np.float32) - Zx)          # small integers: exact in float32
    return (Sx * d).astype(np.float32).astype(np.float16)


def dequant_matmul(W16: np.ndarray, X16: np.ndarray) -> np.ndarray:
    """Y = W_hat X from float16 operands, summed exactly enough in float64
    (every product of two float16 values is exact there)."""
    return np.asarray(W16, dtype=np.float64) @ np.asarray(X16, dtype=np.float64)


def summation_bound(W16: np.ndarray, X16: np.ndarray) -> np.ndarray:
    """Elementwise bound on the float32 accumulation error of W_hat X in any
    order: m u |W_hat| |X| with u = 2^-24 (each of the m - 1 additions
    rounds once to float32; the products themselves are exact)."""
    m = np.asarray(W16).shape[1]
    return m * 2.0 ** -24 * (np.abs(np.asarray(W16, dtype=np.float64)) @
                             np.abs(np.asarray(X16, dtype=np.float64)))


__all__ = ["packed_words", "pack_codes", "unpack_codes", "dequantize_fp16", "dequant_matmul",
           "summation_bound", "group_size"]
