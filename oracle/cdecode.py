"""ctypes wrapper of the oracle's C decode (oracle/decode.c).

TEST INFRASTRUCTURE: only ``tests/`` loads it.  It computes exactly what
:func:`oracle.ojbkq.decode` computes (the same steps of Alg. 1, Eq.
klein_prob, Alg. 3 and Alg. 4, the same draws), in plain C loops so that
full-size layers can be checked on many columns; the CPU tests compare the
two on random problems.  Built by :func:`build` (gcc, OpenMP).
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from . import ojbkq as orc

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "decode.c")
LIB = os.path.join(HERE, "liboracle_decode.so")
_lib = None


def build() -> str:
    """Compile decode.c into liboracle_decode.so (IEEE float64 semantics:
    no fast-math, no contraction into fused multiply-adds)."""
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-shared", "-fPIC",
           SRC, "-o", tmp, "-lm"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"gcc failed on oracle/decode.c:\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


def _library():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        lib = ctypes.CDLL(LIB)
        i64, dp, vp = ctypes.c_int64, ctypes.POINTER(ctypes.c_double), ctypes.c_void_p
        lib.oracle_decode.restype = ctypes.c_int
        lib.oracle_decode.argtypes = [i64, i64, vp, vp, vp, ctypes.c_int, ctypes.c_int, vp,
                                      ctypes.c_uint64, vp, ctypes.c_int, vp, vp]
        _lib = lib
    return _lib


def decode(R, qbar, S, bits: int, group, K: int, seed: int, columns=None,
           alpha=None) -> "orc.DecodeResult":
    """Same arguments and result as :func:`oracle.ojbkq.decode` (``alpha``
    may pass the per-column temperatures instead of the rule's)."""
    R = np.ascontiguousarray(R, dtype=np.float64)
    qbar = np.asarray(qbar, dtype=np.float64)
    m = R.shape[0]
    n = qbar.shape[0]
    cols = np.arange(n) if columns is None else np.asarray(columns)
    al = orc.klein_alpha(R, S[cols], group, K) if alpha is None else np.asarray(alpha, np.float64)
    al = np.ascontiguousarray(al, dtype=np.float64)
    s_rows = np.ascontiguousarray(orc.expand_groups(S[cols], m, group))
    qb = np.ascontiguousarray(qbar[cols])
    c64 = np.ascontiguousarray(cols, dtype=np.int64)
    nc = len(cols)
    P = K + 1
    codes = np.zeros((nc, P, m), dtype=np.uint8)
    resid = np.zeros((nc, P), dtype=np.float64)
    threads = max(1, len(os.sched_getaffinity(0)))
    grp = max(1, min(P, (P * nc + threads - 1) // threads if nc < threads else P))
    rc = _library().oracle_decode(m, nc, R.ctypes.data, qb.ctypes.data, s_rows.ctypes.data,
                                  int(bits), int(K), al.ctypes.data, int(seed) & (2 ** 64 - 1),
                                  c64.ctypes.data, int(grp), codes.ctypes.data, resid.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_decode rejected its arguments")
    win = np.array([orc.select_best(r) for r in resid], dtype=np.int32)
    best = codes[np.arange(nc), win]
    return orc.DecodeResult(best, resid[np.arange(nc), win], win, codes, resid, al)
