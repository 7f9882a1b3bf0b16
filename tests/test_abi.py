"""CPU-only checks of the C ABI: the library loads, exports every declared
symbol, rejects bad arguments before touching a GPU, and its host-side Klein
temperature solver satisfies the defining equation."""

import ctypes
import math
import os
import re

import pytest

import paper_2602_08376_amd as ok
from conftest import ROOT
from oracle import ojbkq as orc

HEADER = os.path.join(ROOT, "include", "ojbkq.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ojbkq_[a-z_]+)\s*\(", text)))


def test_library_builds_and_loads():
    assert os.path.exists(ok.library_path), "run __graft_entry__.build() first"
    ok.library()


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) == 22
    assert sorted(ok.ABI_FUNCTIONS) == names
    lib = ctypes.CDLL(ok.library_path)
    for name in names:
        assert hasattr(lib, name), name


def _p(**kw):
    base = dict(m=128, n=64, bits=4, group=128, K=4, alpha=0.5, lambda_rel=0.01, seed=0)
    base.update(kw)
    return ok._params(**base)


@pytest.mark.parametrize("bad", [dict(m=0), dict(n=0), dict(bits=0), dict(bits=9), dict(K=-1),
                                 dict(alpha=1.5), dict(alpha=-0.1), dict(alpha=float("nan")),
                                 dict(lambda_rel=-1.0), dict(lambda_rel=float("inf"))])
def test_bad_params_rejected(bad):
    lib = ok.library()
    p = _p(**bad)
    assert lib.ojbkq_workspace_bytes(ctypes.byref(p)) == 0
    assert lib.ojbkq_decode_workspace_bytes(ctypes.byref(p)) == 0
    rc = lib.ojbkq_quantize_layer(ctypes.byref(p), 1, 1, 1, 10, 10, 256, 1 << 30, None, 1, 1, 1, 1,
                                  None, None)
    assert rc == -1
    assert lib.ojbkq_last_error().decode()


def test_gram_mode_values():
    lib = ok.library()
    for v, good in ((0, True), (1, True), (2, False), (-1, False)):
        p = _p()
        p.gram_fp64 = v
        assert (lib.ojbkq_workspace_bytes(ctypes.byref(p)) > 0) == good, v
    # the int8 token sums carve their split digits (about 64 m^2 bytes) from
    # the workspace; their partial-tile scratch is half the fp64 kernel's
    i8 = ok.workspace_bytes(4096, 4096, 4, 128, 16, gram="int8")
    f64 = ok.workspace_bytes(4096, 4096, 4, 128, 16, gram="fp64")
    assert i8 - f64 >= 64 * 4096 ** 2 - 64 * 2 ** 20


def test_decode_mode_values():
    lib = ok.library()
    for v, good in ((0, True), (1, True), (2, False), (-1, False)):
        p = _p()
        p.decode_fp64 = v
        assert (lib.ojbkq_workspace_bytes(ctypes.byref(p)) > 0) == good, v
    with pytest.raises(ValueError):
        ok._params(128, 64, 4, 128, 4, 0.5, 0.01, 0, decode="fp32")


def test_scheme_values():
    lib = ok.library()
    for scheme, bits, ok_ in ((0, 4, True), (1, 4, True), (1, 2, True), (1, 1, False),
                              (0, 1, True), (2, 4, False), (-1, 4, False)):
        p = _p(bits=bits)
        p.scheme = scheme
        assert (lib.ojbkq_workspace_bytes(ctypes.byref(p)) > 0) == ok_, (scheme, bits)
    with pytest.raises(ValueError):
        ok._params(128, 64, 4, 128, 4, 0.5, 0.01, 0, "absmax")


def test_act_order_values():
    """act_order is 0, 1 or 2; 1 adds the decode order and the permuted
    weights (m int32 + n m float32) to the workspace, 2 also the inverse order
    and the group of every position; keep_gram is 0 or 1."""
    lib = ok.library()

    def perm_ws(m, n):
        return ok.workspace_bytes(m, n, 4, 128, 4, act_order=True)

    for v, ok_ in ((0, True), (1, True), (2, True), (3, False), (-1, False)):
        p = _p()
        p.act_order = v
        assert (lib.ojbkq_workspace_bytes(ctypes.byref(p)) > 0) == ok_, v
    for v, ok_ in ((0, True), (1, True), (2, False), (-1, False)):
        p = _p()
        p.keep_gram = v
        assert (lib.ojbkq_workspace_bytes(ctypes.byref(p)) > 0) == ok_, v
    # static groups add the inverse order and the group of every position
    assert ok.workspace_bytes(300, 70, 4, 128, 4, act_order="static") >= perm_ws(300, 70) + 2 * 300 * 4
    with pytest.raises(ValueError):
        ok._params(128, 64, 4, 128, 4, 0.5, 0.01, 0, act_order="desc")
    assert ok.workspace_bytes(300, 70, 4, 128, 4, keep_gram=True) >= \
        ok.workspace_bytes(300, 70, 4, 128, 4) + 300 * 300 * 8
    plain = ok.workspace_bytes(300, 70, 4, 128, 4)
    assert perm_ws(300, 70) >= plain + 300 * 4 + 70 * 300 * 4


def test_null_and_shape_errors_before_any_launch():
    lib = ok.library()
    p = _p()
    ws = lib.ojbkq_workspace_bytes(ctypes.byref(p))
    assert ws > 0
    # missing outputs / inputs
    assert lib.ojbkq_quantize_layer(ctypes.byref(p), None, None, 1, 10, 10, 256, ws, None, 1, 1, 1,
                                    1, None, None) == -1
    assert lib.ojbkq_quantize_layer(ctypes.byref(p), 1, None, 1, 10, 10, 256, ws, None, None, 1, 1,
                                    1, None, None) == -1
    # bad token count / stride
    assert lib.ojbkq_quantize_layer(ctypes.byref(p), 1, None, 1, 0, 10, 256, ws, None, 1, 1, 1, 1,
                                    None, None) == -1
    assert lib.ojbkq_quantize_layer(ctypes.byref(p), 1, None, 1, 10, 9, 256, ws, None, 1, 1, 1, 1,
                                    None, None) == -1
    assert lib.ojbkq_quantize_layer(ctypes.byref(p), 1, None, 1, 10, (1 << 27) + 1, 256, ws, None,
                                    1, 1, 1, 1, None, None) == -1
    assert "2^27" in lib.ojbkq_last_error().decode()
    # misaligned or missing workspace
    assert lib.ojbkq_quantize_layer(ctypes.byref(p), 1, None, 1, 10, 10, 0, ws, None, 1, 1, 1, 1,
                                    None, None) == -1
    assert lib.ojbkq_quantize_layer(ctypes.byref(p), 1, None, 1, 10, 10, 8, ws, None, 1, 1, 1, 1,
                                    None, None) == -1
    # workspace too small
    assert lib.ojbkq_quantize_layer(ctypes.byref(p), 1, None, 1, 10, 10, 256, ws - 1, None, 1, 1,
                                    1, 1, None, None) == -2
    assert "needs" in lib.ojbkq_last_error().decode()
    # staged calls on a NULL handle
    h = ctypes.c_void_p()
    assert lib.ojbkq_create(ctypes.byref(p), None, ws, None, ctypes.byref(h)) == -1
    assert lib.ojbkq_create(ctypes.byref(p), 256, ws, None, None) == -1
    assert lib.ojbkq_accumulate(None, None, 1, 10, 10) == -1
    assert lib.ojbkq_solve(None, 1, 0.5, 1, 1, 1, 1, None, None) == -1
    assert lib.ojbkq_set_knobs(None, 0.01, 1) == -1
    ptr = ctypes.c_void_p()
    assert lib.ojbkq_inspect(None, 0, ctypes.byref(ptr)) == -1
    assert lib.ojbkq_path_codes(None, 1) == -1
    assert lib.ojbkq_destroy(None) == 0
    assert lib.ojbkq_set_timing(None, 1) == -1
    ms = (ctypes.c_double * 6)()
    assert lib.ojbkq_stage_times(None, ms) == -1
    # decode stage
    dws = lib.ojbkq_decode_workspace_bytes(ctypes.byref(p))
    assert dws > 0
    assert lib.ojbkq_decode_stage(ctypes.byref(p), None, 1, 1, 256, dws, None, 1, 1, None, None,
                                  None) == -1
    assert lib.ojbkq_decode_stage(ctypes.byref(p), 1, 1, 1, 256, dws - 1, None, 1, 1, None, None,
                                  None) == -2


def test_workspace_size_grows_with_shape():
    small = ok.workspace_bytes(128, 64, 4, 128, 4)
    big = ok.workspace_bytes(4096, 4096, 4, 128, 16)
    # G, E, L^-1 and Q (m^2 doubles each), one n*m double array, codes of n(K+1) padded paths
    paths = ((4096 * 17 + 255) // 256) * 256
    assert big >= 4 * 4096 * 4096 * 8 + 4096 * 4096 * 8 + paths * 4096
    assert small < big


@pytest.mark.parametrize("m,K", [(3, 4), (8, 16), (128, 4), (4096, 5), (4096, 16), (5120, 32),
                                 (11008, 16), (28672, 16), (2, 50)])
def test_klein_log_rho_defining_equation(m, K):
    x = ok.klein_log_rho(m, K)
    rho = math.exp(x)
    assert rho > 1.0
    assert abs((2.0 * m / rho) * (1.0 + x) - math.log(K)) <= 1e-12 * math.log(K)
    # the oracle solves the same equation independently
    assert abs(x - orc.klein_log_rho(m, K)) <= 1e-13 * x


def test_klein_log_rho_limits():
    assert ok.klein_log_rho(100, 1) == math.inf
    assert ok.klein_log_rho(100, 0) == math.inf
    assert ok.klein_log_rho(1, 10) == 0.0
    assert math.isnan(ok.klein_log_rho(0, 10))
