"""MI355X (gfx950) implementation of OJBKQ's per-layer quantisation path.

A thin Python binding over the C ABI of ``include/ojbkq.h`` (``libojbkq.so``
in this directory).  Only argument marshalling happens here: torch supplies
device memory and the current stream, every step of the path runs in the HIP
kernels of the library.  There is no fallback: without the built library
every call raises.
"""

from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass
from typing import Optional

import torch

__all__ = [
    "OjbkqError", "Params", "library", "library_path", "quantize_layer", "LayerSolver",
    "decode_stage", "klein_log_rho", "workspace_bytes", "decode_workspace_bytes",
    "ABI_FUNCTIONS", "QuantResult", "STAGES",
]

_PKG = os.path.dirname(os.path.abspath(__file__))
library_path = os.path.join(_PKG, "libojbkq.so")

# every entry point of include/ojbkq.h
ABI_FUNCTIONS = (
    "ojbkq_workspace_bytes", "ojbkq_quantize_layer", "ojbkq_create", "ojbkq_accumulate",
    "ojbkq_solve", "ojbkq_destroy", "ojbkq_inspect", "ojbkq_decode_workspace_bytes",
    "ojbkq_decode_stage", "ojbkq_klein_log_rho", "ojbkq_last_error", "ojbkq_set_timing",
    "ojbkq_stage_times", "ojbkq_set_weights", "ojbkq_packed_words", "ojbkq_pack_codes",
    "ojbkq_dequant_matmul", "ojbkq_set_knobs", "ojbkq_path_codes",
    "ojbkq_quantize_layer_noalloc", "ojbkq_dequant_matmul_workspace_bytes",
    "ojbkq_dequant_matmul_ws",
)

NOALLOC_SCRATCH_BYTES = 256 * 1024 * 1024   # OJBKQ_NOALLOC_SCRATCH_BYTES

STAGES = ("gram", "factor", "solve", "centres", "decode", "select")

_STATUS = {0: "OK", -1: "EINVAL", -2: "ENOSPACE", -3: "ENOTPD", -4: "EHIP", -5: "ESTATE"}


class OjbkqError(RuntimeError):
    """A library call returned a non-zero status."""

    def __init__(self, status: int, message: str):
        super().__init__(f"ojbkq {_STATUS.get(status, status)}: {message}")
        self.status = status
        self.code = _STATUS.get(status, str(status))


class Params(ctypes.Structure):
    _fields_ = [
        ("m", ctypes.c_int64), ("n", ctypes.c_int64), ("bits", ctypes.c_int32),
        ("group", ctypes.c_int32), ("K", ctypes.c_int32), ("scheme", ctypes.c_int32),
        ("alpha", ctypes.c_double), ("lambda_rel", ctypes.c_double), ("seed", ctypes.c_uint64),
        ("act_order", ctypes.c_int32), ("keep_gram", ctypes.c_int32),
        ("gram_fp64", ctypes.c_int32), ("decode_fp64", ctypes.c_int32),
    ]


_lib = None


def library() -> ctypes.CDLL:
    """The loaded HIP library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(library_path):
        raise RuntimeError(f"HIP library {library_path} is not built; run "
                           "`python -m paper_2602_08376_amd.build` (no CPU fallback exists)")
    lib = ctypes.CDLL(library_path)
    P, vp, i64, dp = ctypes.POINTER(Params), ctypes.c_void_p, ctypes.c_int64, ctypes.c_double
    sig = {
        "ojbkq_workspace_bytes": (ctypes.c_size_t, [P]),
        "ojbkq_decode_workspace_bytes": (ctypes.c_size_t, [P]),
        "ojbkq_quantize_layer": (ctypes.c_int, [P, vp, vp, vp, i64, i64, vp, ctypes.c_size_t, vp,
                                                vp, vp, vp, vp, vp, vp]),
        "ojbkq_quantize_layer_noalloc": (ctypes.c_int, [P, vp, vp, vp, i64, i64, vp, vp, vp,
                                                        vp, vp, vp, vp]),
        "ojbkq_create": (ctypes.c_int, [P, vp, ctypes.c_size_t, vp, ctypes.POINTER(vp)]),
        "ojbkq_set_weights": (ctypes.c_int, [vp, vp]),
        "ojbkq_set_knobs": (ctypes.c_int, [vp, dp, ctypes.c_int32]),
        "ojbkq_packed_words": (i64, [i64, ctypes.c_int32]),
        "ojbkq_pack_codes": (ctypes.c_int, [vp, i64, i64, ctypes.c_int32, vp, vp, vp]),
        "ojbkq_dequant_matmul": (ctypes.c_int, [vp, vp, vp, i64, i64, ctypes.c_int32,
                                                ctypes.c_int32, vp, i64, i64, vp, vp, i64, vp]),
        "ojbkq_dequant_matmul_workspace_bytes": (ctypes.c_size_t, [i64, i64]),
        "ojbkq_dequant_matmul_ws": (ctypes.c_int, [vp, vp, vp, i64, i64, ctypes.c_int32,
                                                   ctypes.c_int32, vp, i64, i64, vp, vp, i64, vp,
                                                   ctypes.c_size_t, vp]),
        "ojbkq_accumulate": (ctypes.c_int, [vp, vp, vp, i64, i64]),
        "ojbkq_solve": (ctypes.c_int, [vp, vp, dp, vp, vp, vp, vp, vp, vp]),
        "ojbkq_destroy": (ctypes.c_int, [vp]),
        "ojbkq_inspect": (ctypes.c_int, [vp, ctypes.c_int, ctypes.POINTER(vp)]),
        "ojbkq_path_codes": (ctypes.c_int, [vp, vp]),
        "ojbkq_decode_stage": (ctypes.c_int, [P, vp, vp, vp, vp, ctypes.c_size_t, vp, vp, vp, vp,
                                              vp, vp]),
        "ojbkq_klein_log_rho": (ctypes.c_double, [i64, i64]),
        "ojbkq_set_timing": (ctypes.c_int, [vp, ctypes.c_int]),
        "ojbkq_stage_times": (ctypes.c_int, [vp, ctypes.POINTER(ctypes.c_double)]),
        "ojbkq_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(rc: int):
    if rc != 0:
        msg = library().ojbkq_last_error().decode(errors="replace")
        raise OjbkqError(rc, msg)


SCHEMES = {"asym": 0, "sym": 1}   # scale / zero-point rule (ojbkq_params.scheme)


ACT_ORDER = {False: 0, True: 1, "static": 2}   # ojbkq_params.act_order


def _act_order(v) -> int:
    if isinstance(v, int) and not isinstance(v, bool) and v in (0, 1, 2):
        return v
    if v not in ACT_ORDER:
        raise ValueError('act_order must be False, True or "static"')
    return ACT_ORDER[v]


GRAMS = {"int8": 0, "fp64": 1}     # arithmetic of the token sums (ojbkq_params.gram_fp64)
DECODES = {"int8": 0, "fp64": 1}   # the decoder's lazy update (ojbkq_params.decode_fp64)


def _params(m, n, bits, group, K, alpha, lambda_rel, seed, scheme="asym",
            act_order=False, keep_gram=False, gram="int8", decode="int8") -> Params:
    if scheme not in SCHEMES:
        raise ValueError(f"scheme must be one of {sorted(SCHEMES)}")
    if gram not in GRAMS:
        raise ValueError(f"gram must be one of {sorted(GRAMS)}")
    if decode not in DECODES:
        raise ValueError(f"decode must be one of {sorted(DECODES)}")
    return Params(int(m), int(n), int(bits), int(group), int(K), SCHEMES[scheme], float(alpha),
                  float(lambda_rel), int(seed) & 0xFFFFFFFFFFFFFFFF, _act_order(act_order),
                  1 if keep_gram else 0, GRAMS[gram], DECODES[decode])


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _need(t: torch.Tensor, name: str, dtype, shape=None, device=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU (got {t.device})")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (got {t.dtype})")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)} (got {tuple(t.shape)})")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")


def _rows_view(X: torch.Tensor, name: str, m: int):
    """(T, row stride) of an [m, T] float32 tensor whose rows are contiguous."""
    if X.dim() != 2 or X.shape[0] != m:
        raise ValueError(f"{name} must be [m={m}, T] (got {tuple(X.shape)})")
    if X.stride(1) != 1:
        raise ValueError(f"{name} rows must be contiguous")
    T = X.shape[1]
    ld = X.stride(0) if X.shape[0] > 1 else T
    return T, max(ld, T)


def projects_cross_term(m: int, n: int, gram: str = "int8") -> bool:
    """Whether a context with bound weights accumulates the cross term as
    W E^T instead of forming E (the rule stated at ojbkq_set_weights)."""
    return 10 * n <= m if gram == "int8" else 5 * n <= 2 * m


def num_groups(m: int, group: int) -> int:
    g = m if (group <= 0 or group >= m) else group
    return (m + g - 1) // g


def workspace_bytes(m, n, bits, group, K, alpha=0.5, lambda_rel=0.01, seed=0,
                    act_order=False, keep_gram=False, gram="int8", decode="int8") -> int:
    p = _params(m, n, bits, group, K, alpha, lambda_rel, seed, act_order=act_order,
                keep_gram=keep_gram, gram=gram, decode=decode)
    nb = library().ojbkq_workspace_bytes(ctypes.byref(p))
    if nb == 0:
        _check(-1)
    return int(nb)


def decode_workspace_bytes(m, n, bits, group, K, seed=0, decode="int8") -> int:
    p = _params(m, n, bits, group, K, 0.5, 0.0, seed, decode=decode)
    nb = library().ojbkq_decode_workspace_bytes(ctypes.byref(p))
    if nb == 0:
        _check(-1)
    return int(nb)


def _workspace(nbytes: int, device) -> torch.Tensor:
    # torch's allocator returns 512-byte aligned blocks
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)


@dataclass
class QuantResult:
    codes: torch.Tensor       # [n, m] uint8
    scales: torch.Tensor      # [n, G] float32
    zeros: torch.Tensor       # [n, G] float32
    residuals: torch.Tensor   # [n] float64
    winner: torch.Tensor      # [n] int32
    perm: Optional[torch.Tensor] = None   # [m] int32 decode order (act order only)


def _outputs(n, m, G, device, act_order=False):
    return QuantResult(
        codes=torch.empty(n, m, dtype=torch.uint8, device=device),
        scales=torch.empty(n, G, dtype=torch.float32, device=device),
        zeros=torch.empty(n, G, dtype=torch.float32, device=device),
        residuals=torch.empty(n, dtype=torch.float64, device=device),
        winner=torch.empty(n, dtype=torch.int32, device=device),
        perm=torch.empty(m, dtype=torch.int32, device=device) if act_order else None,
    )


def quantize_layer(W, X_ref, X_q, alpha, bits, group, K, seed, lambda_rel=0.01,
                   workspace: Optional[torch.Tensor] = None, scheme="asym",
                   act_order=False, gram="int8", decode="int8") -> QuantResult:
    """One-shot ``ojbkq_quantize_layer`` on device tensors.

    W [n, m] float32; X_ref, X_q [m, T] float32 (X_ref may be None or X_q);
    scheme: "asym" (min-max) or "sym" (Absmax) scales and zero points;
    act_order: decode the features with the largest Hessian diagonal first
    (codes stay in W's order, ``perm`` holds the decode order); True groups
    the scales by decode position, "static" keeps W's own groups;
    gram: "int8" (digit products on the int8 matrix cores) or "fp64";
    decode: "int8" (the decoder's lazy update on the int8 matrix cores where
    the codes have at most 7 bits and the scale groups are whole 64-row
    pairs) or "fp64".
    """
    n, m = W.shape
    dev = W.device
    _need(W, "W", torch.float32, device=dev)
    if not W.is_contiguous():
        raise ValueError("W must be contiguous")
    _need(X_q, "X_q", torch.float32, device=dev)
    T, ld = _rows_view(X_q, "X_q", m)
    if X_ref is not None and X_ref is not X_q:
        _need(X_ref, "X_ref", torch.float32, device=dev)
        if tuple(X_ref.shape) != tuple(X_q.shape) or X_ref.stride() != X_q.stride():
            raise ValueError("X_ref must have the shape and strides of X_q")
    p = _params(m, n, bits, group, K, alpha, lambda_rel, seed, scheme, act_order, gram=gram,
                decode=decode)
    lib = library()
    need = lib.ojbkq_workspace_bytes(ctypes.byref(p))
    if need == 0:
        _check(-1)
    ws = workspace if workspace is not None else _workspace(need, dev)
    out = _outputs(n, m, num_groups(m, group), dev, act_order)
    rc = lib.ojbkq_quantize_layer(ctypes.byref(p), _ptr(W), _ptr(X_ref), _ptr(X_q), T, ld,
                                  _ptr(ws), ws.numel(), _stream(dev), _ptr(out.codes),
                                  _ptr(out.scales), _ptr(out.zeros), _ptr(out.residuals),
                                  _ptr(out.winner), _ptr(out.perm))
    _check(rc)
    return out


def quantize_layer_noalloc(W, X_ref, X_q, alpha, bits, group, K, seed, lambda_rel=0.01,
                           scheme="asym", act_order=False, gram="int8", decode="int8",
                           out: Optional[QuantResult] = None) -> QuantResult:
    """``ojbkq_quantize_layer_noalloc``: the one-shot call on the library's
    static scratch (no workspace).  ``out`` may pass preallocated outputs
    (then nothing at all is allocated on the device for the call)."""
    n, m = W.shape
    dev = W.device
    _need(W, "W", torch.float32, device=dev)
    if not W.is_contiguous():
        raise ValueError("W must be contiguous")
    _need(X_q, "X_q", torch.float32, device=dev)
    T, ld = _rows_view(X_q, "X_q", m)
    if X_ref is not None and X_ref is not X_q:
        _need(X_ref, "X_ref", torch.float32, device=dev)
        if tuple(X_ref.shape) != tuple(X_q.shape) or X_ref.stride() != X_q.stride():
            raise ValueError("X_ref must have the shape and strides of X_q")
    p = _params(m, n, bits, group, K, alpha, lambda_rel, seed, scheme, act_order, gram=gram,
                decode=decode)
    if out is None:
        out = _outputs(n, m, num_groups(m, group), dev, act_order)
    rc = library().ojbkq_quantize_layer_noalloc(
        ctypes.byref(p), _ptr(W), _ptr(X_ref), _ptr(X_q), T, ld, _stream(dev), _ptr(out.codes),
        _ptr(out.scales), _ptr(out.zeros), _ptr(out.residuals), _ptr(out.winner), _ptr(out.perm))
    _check(rc)
    return out


class LayerSolver:
    """Staged form: accumulate token chunks, then solve for one or more knobs."""

    def __init__(self, m, n, bits, group, K, seed, lambda_rel=0.01, device="cuda",
                 workspace: Optional[torch.Tensor] = None, scheme="asym", act_order=False,
                 keep_gram=False, gram="int8", decode="int8"):
        self.m, self.n, self.bits, self.group, self.K = int(m), int(n), bits, group, K
        _act_order(act_order)
        self.act_order = act_order
        self.lambda_rel = float(lambda_rel)
        self.device = torch.device(device)
        if self.device.index is None:
            self.device = torch.device("cuda", torch.cuda.current_device())
        self.p = _params(m, n, bits, group, K, 0.5, lambda_rel, seed, scheme, act_order,
                         keep_gram, gram, decode)
        lib = library()
        need = lib.ojbkq_workspace_bytes(ctypes.byref(self.p))
        if need == 0:
            _check(-1)
        self.ws = workspace if workspace is not None else _workspace(need, self.device)
        h = ctypes.c_void_p()
        _check(lib.ojbkq_create(ctypes.byref(self.p), _ptr(self.ws), self.ws.numel(),
                                _stream(self.device), ctypes.byref(h)))
        self.h = h

    def set_weights(self, W):
        """Bind W before the first chunk (see ojbkq_set_weights); every solve
        must then be given this same tensor, which is kept alive here."""
        _need(W, "W", torch.float32, (self.n, self.m), self.device)
        if not W.is_contiguous():
            raise ValueError("W must be contiguous")
        _check(library().ojbkq_set_weights(self.h, _ptr(W)))
        self.W = W

    def set_knobs(self, lambda_rel=None, K=None):
        """``ojbkq_set_knobs``: damping and Klein samples for the next solves
        (a new lambda_rel after a solve needs keep_gram=True)."""
        lam = self.lambda_rel if lambda_rel is None else float(lambda_rel)
        k = self.K if K is None else int(K)
        _check(library().ojbkq_set_knobs(self.h, lam, k))
        self.lambda_rel, self.K = lam, k

    def accumulate(self, X_ref_c, X_q_c):
        _need(X_q_c, "X_q_c", torch.float32, device=self.device)
        T, ld = _rows_view(X_q_c, "X_q_c", self.m)
        if X_ref_c is not None and X_ref_c is not X_q_c:
            _need(X_ref_c, "X_ref_c", torch.float32, device=self.device)
            if tuple(X_ref_c.shape) != tuple(X_q_c.shape) or X_ref_c.stride() != X_q_c.stride():
                raise ValueError("X_ref_c must have the shape and strides of X_q_c")
        _check(library().ojbkq_accumulate(self.h, _ptr(X_ref_c), _ptr(X_q_c), T, ld))

    def solve(self, W, alpha) -> QuantResult:
        _need(W, "W", torch.float32, (self.n, self.m), self.device)
        if not W.is_contiguous():
            raise ValueError("W must be contiguous")
        out = _outputs(self.n, self.m, num_groups(self.m, self.group), self.device,
                       self.act_order)
        _check(library().ojbkq_solve(self.h, _ptr(W), float(alpha), _ptr(out.codes),
                                     _ptr(out.scales), _ptr(out.zeros), _ptr(out.residuals),
                                     _ptr(out.winner), _ptr(out.perm)))
        self._solved_K = self.K
        return out

    def inspect(self, which: str) -> torch.Tensor:
        """A copy of an intermediate of the last solve: 'L', 'gq' (rows Rbar_j qbar_j),
        'alpha', 'lam2', 'path_resid', 'perm' (act order)."""
        idx = {"L": 0, "gq": 1, "alpha": 2, "lam2": 3, "path_resid": 4, "perm": 5}[which]
        ptr = ctypes.c_void_p()
        _check(library().ojbkq_inspect(self.h, idx, ctypes.byref(ptr)))
        shape = {"L": (self.m, self.m), "gq": (self.n, self.m), "alpha": (self.n,),
                 "lam2": (1,), "path_resid": (self.n, self.K + 1), "perm": (self.m,)}[which]
        off = ptr.value - self.ws.data_ptr()
        count = int(math.prod(shape))
        if which == "perm":
            return self.ws[off:off + 4 * count].view(torch.int32).clone()
        flat = self.ws[off:off + 8 * count].view(torch.float64)
        return flat.reshape(shape).clone()

    def path_codes(self) -> torch.Tensor:
        """``ojbkq_path_codes``: every candidate of the last solve, [n, K + 1, m]
        uint8 in W's feature order (K of that solve)."""
        k = getattr(self, "_solved_K", self.K)
        out = torch.empty(self.n, k + 1, self.m, dtype=torch.uint8, device=self.device)
        _check(library().ojbkq_path_codes(self.h, _ptr(out)))
        return out

    def set_timing(self, enable: bool = True):
        """Record per-stage device times from now on (see ojbkq_stage_times)."""
        _check(library().ojbkq_set_timing(self.h, 1 if enable else 0))

    def stage_times(self) -> dict:
        """Device milliseconds per stage since timing was enabled."""
        arr = (ctypes.c_double * len(STAGES))()
        _check(library().ojbkq_stage_times(self.h, arr))
        return {name: float(arr[i]) for i, name in enumerate(STAGES)}

    def close(self):
        if getattr(self, "h", None) is not None and self.h.value:
            library().ojbkq_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def decode_stage(R, qbar, scales, bits, group, K, seed, want_paths=False, decode="int8"):
    """``ojbkq_decode_stage``: decode + select on a given upper factor R (float64)."""
    m = R.shape[0]
    n = qbar.shape[0]
    dev = R.device
    _need(R, "R", torch.float64, (m, m), dev)
    _need(qbar, "qbar", torch.float64, (n, m), dev)
    _need(scales, "scales", torch.float32, (n, num_groups(m, group)), dev)
    for t, nm in ((R, "R"), (qbar, "qbar"), (scales, "scales")):
        if not t.is_contiguous():
            raise ValueError(f"{nm} must be contiguous")
    p = _params(m, n, bits, group, K, 0.5, 0.0, seed, decode=decode)
    lib = library()
    need = lib.ojbkq_decode_workspace_bytes(ctypes.byref(p))
    if need == 0:
        _check(-1)
    ws = _workspace(need, dev)
    codes = torch.empty(n, m, dtype=torch.uint8, device=dev)
    resid = torch.empty(n, dtype=torch.float64, device=dev)
    winner = torch.empty(n, dtype=torch.int32, device=dev)
    pc = torch.empty(n, K + 1, m, dtype=torch.uint8, device=dev) if want_paths else None
    pr = torch.empty(n, K + 1, dtype=torch.float64, device=dev) if want_paths else None
    _check(lib.ojbkq_decode_stage(ctypes.byref(p), _ptr(R), _ptr(qbar), _ptr(scales), _ptr(ws),
                                  ws.numel(), _stream(dev), _ptr(codes), _ptr(resid), _ptr(winner),
                                  _ptr(pc), _ptr(pr)))
    return codes, resid, winner, pc, pr


def klein_log_rho(m: int, K: int) -> float:
    """Host-side ``ojbkq_klein_log_rho`` (no GPU needed)."""
    return float(library().ojbkq_klein_log_rho(int(m), int(K)))


# ---------------------------------------------------------------------------
# the quantized layer in use: packed codes and W_hat X
# ---------------------------------------------------------------------------

def packed_words(m: int, bits: int) -> int:
    """32-bit words per packed row (``ojbkq_packed_words``)."""
    w = library().ojbkq_packed_words(int(m), int(bits))
    if w <= 0:
        raise ValueError("need m >= 1 and bits in [1, 8]")
    return int(w)


def _perm_arg(perm, m, dev):
    if perm is None:
        return None
    _need(perm, "perm", torch.int32, (m,), dev)
    if not perm.is_contiguous():
        raise ValueError("perm must be contiguous")
    return perm


def pack_codes(codes: torch.Tensor, bits: int, perm: Optional[torch.Tensor] = None) -> torch.Tensor:
    """``ojbkq_pack_codes``: codes [n, m] uint8 -> [n, words] int32 holding the
    uint32 bit streams (position p holds codes[:, perm[p]] when perm is given)."""
    _need(codes, "codes", torch.uint8)
    if codes.dim() != 2 or not codes.is_contiguous():
        raise ValueError("codes must be a contiguous [n, m] tensor")
    n, m = codes.shape
    perm = _perm_arg(perm, m, codes.device)
    out = torch.empty(n, packed_words(m, bits), dtype=torch.int32, device=codes.device)
    _check(library().ojbkq_pack_codes(_ptr(codes), n, m, int(bits), _ptr(perm), _ptr(out),
                                      _stream(codes.device)))
    return out


def dequant_matmul(packed: torch.Tensor, scales: torch.Tensor, zeros: torch.Tensor, m: int,
                   bits: int, group: int, X: torch.Tensor,
                   perm: Optional[torch.Tensor] = None, workspace=True) -> torch.Tensor:
    """Y [n, T] float32 = W_hat [n, m] X [m, T] with X float16 (rows
    contiguous) and W_hat from the packed codes (packed with ``perm`` when one
    is given).  ``workspace``: True (a device buffer of
    ``ojbkq_dequant_matmul_workspace_bytes`` is allocated here and W_hat formed
    there once, ``ojbkq_dequant_matmul_ws``), a uint8 device tensor to use as
    that buffer, or False (``ojbkq_dequant_matmul``: dequantized per tile, no
    buffer)."""
    dev = packed.device
    _need(packed, "packed", torch.int32, device=dev)
    n = packed.shape[0]
    G = num_groups(m, group)
    _need(scales, "scales", torch.float32, (n, G), dev)
    _need(zeros, "zeros", torch.float32, (n, G), dev)
    _need(X, "X", torch.float16, device=dev)
    if packed.shape != (n, packed_words(m, bits)) or not packed.is_contiguous():
        raise ValueError("packed must be [n, packed_words(m, bits)] and contiguous")
    if not (scales.is_contiguous() and zeros.is_contiguous()):
        raise ValueError("scales and zeros must be contiguous")
    T, ld = _rows_view(X, "X", m)
    perm = _perm_arg(perm, m, dev)
    Y = torch.empty(n, T, dtype=torch.float32, device=dev)
    if workspace is False:
        _check(library().ojbkq_dequant_matmul(_ptr(packed), _ptr(scales), _ptr(zeros), n, m,
                                              int(bits), int(group), _ptr(X), T, ld, _ptr(perm),
                                              _ptr(Y), T, _stream(dev)))
        return Y
    need = int(library().ojbkq_dequant_matmul_workspace_bytes(n, m))
    if workspace is True:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    else:
        ws = workspace
        _need(ws, "workspace", torch.uint8, device=dev)
        if not ws.is_contiguous():
            raise ValueError("workspace must be contiguous")
    _check(library().ojbkq_dequant_matmul_ws(_ptr(packed), _ptr(scales), _ptr(zeros), n, m,
                                             int(bits), int(group), _ptr(X), T, ld, _ptr(perm),
                                             _ptr(Y), T, _ptr(ws), ws.numel(), _stream(dev)))
    return Y

