"""Python binding of liblogbq (ctypes): argument marshalling only.

Every step of the computation runs in the library: ``fit`` in its host code, ``encode``,
``linear`` and ``dequantize`` in its gfx950 kernels. PyTorch provides device memory and the
current stream; nothing here computes on the data. If the library is not built, every call
raises ``LogbqUnavailable``: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_double, c_float, c_int32, c_int64, c_uint8, c_uint16, c_void_p

import numpy as np

# LOGBQ_LIBRARY selects another build of the library (e.g. a sanitizer build for CPU tests).
LIB_PATH = os.environ.get("LOGBQ_LIBRARY") or \
    os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblogbq.so")

OK, ERR_INVALID_ARG, ERR_NONFINITE, ERR_DEGENERATE, ERR_UNSUPPORTED, ERR_HIP, ERR_HOST_RESOURCE = \
    range(7)


class LogbqUnavailable(RuntimeError):
    pass


class LogbqError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_str(status)} (status {status})")


class Params(ctypes.Structure):
    """Mirror of ``logbq_params`` (include/logbq.h)."""
    _fields_ = [
        ("bits", c_int32), ("qmax", c_int32), ("eps", c_double), ("wmin", c_double),
        ("wmax", c_double), ("base", c_double), ("shift", c_int32), ("reserved", c_int32),
        ("wmin_index", c_int64), ("codebook", c_float * 256), ("thresholds", c_float * 128),
    ]

    def codebook_array(self) -> np.ndarray:
        """The 2^bits codebook entries (16 for 4-bit, 256 for 8-bit codes)."""
        return np.ctypeslib.as_array(self.codebook)[: 1 << self.bits].copy()

    def thresholds_array(self) -> np.ndarray:
        """thresholds[0 .. qmax - 1] followed by +inf padding up to 2^(bits-1) entries."""
        return np.ctypeslib.as_array(self.thresholds)[: 1 << (self.bits - 1)].copy()


class Uniform(ctypes.Structure):
    """logbq_uniform: parameters of the asymmetric linear baseline (4-bit)."""
    _fields_ = [("bits", c_int32), ("zero", c_int32), ("wmin", c_double), ("wmax", c_double),
                ("scale", c_double), ("codebook", c_float * 16), ("thresholds", c_float * 15),
                ("reserved", c_float)]

    def codebook_array(self) -> np.ndarray:
        return np.ctypeslib.as_array(self.codebook).copy()

    def thresholds_array(self) -> np.ndarray:
        return np.ctypeslib.as_array(self.thresholds).copy()


_lib = None

SIGNATURES = {
    "logbq_abi_version": (c_int32, []),
    "logbq_status_str": (ctypes.c_char_p, [c_int32]),
    "logbq_fit": (c_int32, [POINTER(c_float), c_int64, c_int32, c_double, POINTER(Params)]),
    "logbq_encode": (c_int32, [c_void_p, c_int64, c_int64, POINTER(Params), c_void_p,
                               POINTER(c_float), c_void_p]),
    "logbq_linear": (c_int32, [c_void_p, c_int64, c_int64, c_void_p, c_int64, POINTER(c_float),
                               c_void_p, c_void_p]),
    "logbq_dequantize": (c_int32, [c_void_p, c_int64, c_int64, POINTER(c_float), c_void_p,
                                   c_void_p]),
    "logbq_linear_multi": (c_int32, [c_void_p, c_int64, c_int64, c_int32, POINTER(c_void_p),
                                     POINTER(c_int64), POINTER(POINTER(c_float)),
                                     POINTER(c_void_p), c_void_p]),
    "logbq_linear8": (c_int32, [c_void_p, c_int64, c_int64, c_void_p, c_int64, POINTER(c_float),
                                c_void_p, c_void_p]),
    "logbq_dequantize8": (c_int32, [c_void_p, c_int64, c_int64, POINTER(c_float), c_void_p,
                                    c_void_p]),
    "logbq_linear_path": (c_int32, [c_int32, c_int64, c_int64, c_int64, POINTER(c_int32)]),
    "logbq_linear_kernel": (c_int32, [c_int32, c_int64, c_int64, c_int64, POINTER(c_float),
                                      ctypes.c_char_p, c_int64]),
    "logbq_fit_uniform": (c_int32, [POINTER(c_float), c_int64, c_int32, POINTER(Uniform)]),
    "logbq_encode_uniform": (c_int32, [c_void_p, c_int64, c_int64, POINTER(Uniform), c_void_p,
                                       c_void_p]),
    "logbq_gptq": (c_int32, [c_void_p, c_int64, c_int64, c_void_p, POINTER(Params),
                             POINTER(Uniform), c_void_p, c_void_p, c_void_p]),
    "logbq_gptq_noalloc": (c_int32, [c_void_p, c_int64, c_int64, c_void_p, POINTER(Params),
                                     POINTER(Uniform), c_void_p, c_void_p]),
    "logbq_fit_device": (c_int32, [c_void_p, c_int64, c_int32, c_double, c_void_p,
                                   POINTER(Params), c_void_p]),
    "logbq_fit_exact": (c_int32, [POINTER(c_float), c_int64, c_int32, c_double, POINTER(Params)]),
}

FIT_WORKSPACE_BYTES = 110600

ABI_VERSION = 2


def lib() -> ctypes.CDLL:
    """The loaded liblogbq.so (raises LogbqUnavailable if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise LogbqUnavailable(
                f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        h = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        if h.logbq_abi_version() != ABI_VERSION:
            raise LogbqUnavailable(f"{LIB_PATH} has ABI {h.logbq_abi_version()}, "
                                   f"the binding expects {ABI_VERSION}; rebuild it")
        _lib = h
    return _lib


def status_str(status: int) -> str:
    return lib().logbq_status_str(int(status)).decode()


def _check(status: int, where: str):
    if status != OK:
        raise LogbqError(status, where)


def _stream(stream):
    if stream is None:
        import torch
        return c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return c_void_p(stream)
    return c_void_p(stream.cuda_stream)


def _cb_ptr(codebook, entries=16):
    if isinstance(codebook, Params):
        if (1 << codebook.bits) != entries:
            raise ValueError(f"parameters of a {codebook.bits}-bit fit, call needs {entries} entries")
        return codebook.codebook, codebook
    arr = np.ascontiguousarray(np.asarray(codebook, dtype=np.float32))
    if arr.shape != (entries,):
        raise ValueError(f"codebook must hold {entries} float32 values")
    return arr.ctypes.data_as(POINTER(c_float)), arr


def fit(w, bits: int = 4, eps: float = 4e-3) -> Params:
    """logbq_fit on host float32 weights (numpy array or CPU torch tensor)."""
    if hasattr(w, "detach"):
        w = w.detach().cpu().numpy()
    w = np.ascontiguousarray(w, dtype=np.float32)
    p = Params()
    _check(lib().logbq_fit(w.ctypes.data_as(POINTER(c_float)), w.size, bits, eps,
                           ctypes.byref(p)), "logbq_fit")
    return p


def fit_exact(w, bits: int = 4, eps: float = 4e-3) -> Params:
    """logbq_fit_exact on host float32 weights: the device fit's parameters, computed on the host."""
    if hasattr(w, "detach"):
        w = w.detach().cpu().numpy()
    w = np.ascontiguousarray(w, dtype=np.float32)
    p = Params()
    _check(lib().logbq_fit_exact(w.ctypes.data_as(POINTER(c_float)), w.size, bits, eps,
                                 ctypes.byref(p)), "logbq_fit_exact")
    return p


def fit_device(w, bits: int = 4, eps: float = 4e-3, workspace=None, stream=None) -> Params:
    """logbq_fit_device on a contiguous float32 device tensor (Eq. 5 with exact sums). Blocks
    until the fit's passes have run on `stream`."""
    import torch
    if w.dtype != torch.float32 or not w.is_contiguous() or w.device.type != "cuda":
        raise ValueError("w must be a contiguous float32 device tensor")
    if workspace is None:
        workspace = torch.empty(FIT_WORKSPACE_BYTES, dtype=torch.uint8, device=w.device)
    elif workspace.numel() * workspace.element_size() < FIT_WORKSPACE_BYTES:
        raise ValueError(f"workspace must hold {FIT_WORKSPACE_BYTES} bytes")
    p = Params()
    _check(lib().logbq_fit_device(c_void_p(w.data_ptr()), w.numel(), bits, eps,
                                  c_void_p(workspace.data_ptr()), ctypes.byref(p),
                                  _stream(stream)), "logbq_fit_device")
    return p


def encode(w, p: Params, out=None, stream=None):
    """logbq_encode: float32 [N][K] device tensor -> (uint8 codes, float32 codebook).

    Codes are [N][K/2] for a 4-bit fit, [N][K] for an 8-bit one; the codebook has 2^bits
    entries."""
    import torch
    if w.dtype != torch.float32 or w.dim() != 2 or not w.is_contiguous():
        raise ValueError("w must be a contiguous 2-D float32 device tensor")
    n, k = w.shape
    if out is None:
        cols = k // 2 if p.bits == 4 else k
        out = torch.empty((n, cols), dtype=torch.uint8, device=w.device)
    cb = np.zeros(1 << p.bits, dtype=np.float32)
    _check(lib().logbq_encode(c_void_p(w.data_ptr()), n, k, ctypes.byref(p),
                              c_void_p(out.data_ptr()), cb.ctypes.data_as(POINTER(c_float)),
                              _stream(stream)), "logbq_encode")
    return out, cb


def linear(x, codes, codebook, out=None, stream=None):
    """logbq_linear: y[M][N] = x[M][K] . W_hat^T (x float16, y float32) on packed codes."""
    import torch
    if x.dtype != torch.float16 or x.dim() != 2 or not x.is_contiguous():
        raise ValueError("x must be a contiguous 2-D float16 device tensor")
    if codes.dtype != torch.uint8 or codes.dim() != 2 or not codes.is_contiguous():
        raise ValueError("codes must be a contiguous 2-D uint8 device tensor")
    m, k = x.shape
    n = codes.shape[0]
    if codes.shape[1] * 2 != k:
        raise ValueError("codes must be [N][K/2]")
    if out is None:
        out = torch.empty((m, n), dtype=torch.float32, device=x.device)
    cbp, _keep = _cb_ptr(codebook)
    _check(lib().logbq_linear(c_void_p(x.data_ptr()), m, k, c_void_p(codes.data_ptr()), n, cbp,
                              c_void_p(out.data_ptr()), _stream(stream)), "logbq_linear")
    return out


def linear_multi(x, codes_list, codebooks, outs=None, stream=None):
    """logbq_linear_multi: y_i = x . W_hat_i^T for up to 4 linears sharing x (one launch)."""
    import torch
    if x.dtype != torch.float16 or x.dim() != 2 or not x.is_contiguous():
        raise ValueError("x must be a contiguous 2-D float16 device tensor")
    m, k = x.shape
    count = len(codes_list)
    if not 1 <= count <= 4 or len(codebooks) != count:
        raise ValueError("need 1..4 linears with one codebook each")
    for c in codes_list:
        if c.dtype != torch.uint8 or c.dim() != 2 or not c.is_contiguous() or c.shape[1] * 2 != k:
            raise ValueError("codes must be contiguous uint8 [N][K/2] device tensors")
    if outs is None:
        outs = [torch.empty((m, c.shape[0]), dtype=torch.float32, device=x.device)
                for c in codes_list]
    keep = [_cb_ptr(cb) for cb in codebooks]
    cptr = (c_void_p * count)(*[c.data_ptr() for c in codes_list])
    ns = (c_int64 * count)(*[c.shape[0] for c in codes_list])
    cbs = (POINTER(c_float) * count)(*[p for p, _ in keep])
    ys = (c_void_p * count)(*[y.data_ptr() for y in outs])
    _check(lib().logbq_linear_multi(c_void_p(x.data_ptr()), m, k, count, cptr, ns, cbs, ys,
                                    _stream(stream)), "logbq_linear_multi")
    return outs


def dequantize(codes, codebook, out=None, stream=None):
    """logbq_dequantize: uint8 [N][K/2] -> float32 [N][K], bit-exact codebook lookup."""
    import torch
    if codes.dtype != torch.uint8 or codes.dim() != 2 or not codes.is_contiguous():
        raise ValueError("codes must be a contiguous 2-D uint8 device tensor")
    n, h = codes.shape
    k = 2 * h
    if out is None:
        out = torch.empty((n, k), dtype=torch.float32, device=codes.device)
    cbp, _keep = _cb_ptr(codebook)
    _check(lib().logbq_dequantize(c_void_p(codes.data_ptr()), n, k, cbp, c_void_p(out.data_ptr()),
                                  _stream(stream)), "logbq_dequantize")
    return out


def linear8(x, codes, codebook, out=None, stream=None):
    """logbq_linear8: y[M][N] = x[M][K] . W_hat^T on 8-bit codes [N][K] (x float16, y float32)."""
    import torch
    if x.dtype != torch.float16 or x.dim() != 2 or not x.is_contiguous():
        raise ValueError("x must be a contiguous 2-D float16 device tensor")
    if codes.dtype != torch.uint8 or codes.dim() != 2 or not codes.is_contiguous():
        raise ValueError("codes must be a contiguous 2-D uint8 device tensor")
    m, k = x.shape
    n = codes.shape[0]
    if codes.shape[1] != k:
        raise ValueError("8-bit codes must be [N][K]")
    if out is None:
        out = torch.empty((m, n), dtype=torch.float32, device=x.device)
    cbp, _keep = _cb_ptr(codebook, 256)
    _check(lib().logbq_linear8(c_void_p(x.data_ptr()), m, k, c_void_p(codes.data_ptr()), n, cbp,
                               c_void_p(out.data_ptr()), _stream(stream)), "logbq_linear8")
    return out


def dequantize8(codes, codebook, out=None, stream=None):
    """logbq_dequantize8: uint8 [N][K] 8-bit codes -> float32 [N][K], bit-exact lookup."""
    import torch
    if codes.dtype != torch.uint8 or codes.dim() != 2 or not codes.is_contiguous():
        raise ValueError("codes must be a contiguous 2-D uint8 device tensor")
    n, k = codes.shape
    if out is None:
        out = torch.empty((n, k), dtype=torch.float32, device=codes.device)
    cbp, _keep = _cb_ptr(codebook, 256)
    _check(lib().logbq_dequantize8(c_void_p(codes.data_ptr()), n, k, cbp, c_void_p(out.data_ptr()),
                                   _stream(stream)), "logbq_dequantize8")
    return out


PATH_NAMES = {0: "none", 1: "gemv", 2: "mfma", 3: "splitk", 4: "mfma_kq"}


def linear_path(bits: int, m: int, k: int, n: int) -> str:
    """logbq_linear_path: name of the kernel ("none", "gemv", "mfma", "splitk" or "mfma_kq") that
    linear (bits 4) or linear8 (bits 8) runs for an [m][k] x [n][k] call. Host only."""
    out = c_int32(0)
    _check(lib().logbq_linear_path(int(bits), int(m), int(k), int(n), ctypes.byref(out)),
           "logbq_linear_path")
    return PATH_NAMES[out.value]


def linear_kernel(bits: int, m: int, k: int, n: int, codebook=None) -> str:
    """logbq_linear_kernel: the kernel instance (e.g. "k_gemv<4, 1, 4, false, 2>") that the first
    launch of a linear / linear8 call of that shape runs; codebook None stands for a fitted
    (sign-symmetric) one. Host only."""
    buf = ctypes.create_string_buffer(96)
    cb = None
    if codebook is not None:
        arr = np.ascontiguousarray(getattr(codebook, "codebook_array", lambda: codebook)(),
                                   dtype=np.float32)
        if arr.size != 1 << bits:
            raise ValueError(f"codebook of {arr.size} entries for {bits}-bit codes")
        cb = arr.ctypes.data_as(POINTER(c_float))
    _check(lib().logbq_linear_kernel(int(bits), int(m), int(k), int(n), cb, buf, len(buf)),
           "logbq_linear_kernel")
    return buf.value.decode()


def fit_uniform(w, bits: int = 4) -> Uniform:
    """logbq_fit_uniform on host float32 weights (numpy array or CPU torch tensor)."""
    if hasattr(w, "detach"):
        w = w.detach().cpu().numpy()
    w = np.ascontiguousarray(w, dtype=np.float32)
    u = Uniform()
    _check(lib().logbq_fit_uniform(w.ctypes.data_as(POINTER(c_float)), w.size, bits,
                                   ctypes.byref(u)), "logbq_fit_uniform")
    return u


def encode_uniform(w, u: Uniform, out=None, stream=None):
    """logbq_encode_uniform: float32 [N][K] device tensor -> packed uint8 [N][K/2] codes."""
    import torch
    if w.dtype != torch.float32 or w.dim() != 2 or not w.is_contiguous():
        raise ValueError("w must be a contiguous 2-D float32 device tensor")
    n, k = w.shape
    if out is None:
        out = torch.empty((n, k // 2), dtype=torch.uint8, device=w.device)
    _check(lib().logbq_encode_uniform(c_void_p(w.data_ptr()), n, k, ctypes.byref(u),
                                      c_void_p(out.data_ptr()), _stream(stream)),
           "logbq_encode_uniform")
    return out


GPTQ_BLOCK = 128


def gptq(w, u, params, out_codes=None, workspace=None, stream=None):
    """logbq_gptq: GPTQ calibration of the float32 [N][K] device tensor `w` (updated in place to
    the error-compensated weights) with the upper factor `u` ([K][K] float32 device tensor of
    the damped inverse Hessian) and a fixed codebook: `params` is a Params (LogbQuant, from
    fit) or a Uniform (the asymmetric linear baseline, from fit_uniform). Returns packed uint8
    [N][K/2] codes."""
    import torch
    if w.dtype != torch.float32 or w.dim() != 2 or not w.is_contiguous():
        raise ValueError("w must be a contiguous 2-D float32 device tensor")
    n, k = w.shape
    if u.dtype != torch.float32 or tuple(u.shape) != (k, k) or not u.is_contiguous():
        raise ValueError("u must be a contiguous [K][K] float32 device tensor")
    if out_codes is None:
        out_codes = torch.empty((n, k // 2), dtype=torch.uint8, device=w.device)
    if workspace is None:
        workspace = torch.empty((n, GPTQ_BLOCK), dtype=torch.float32, device=w.device)
    pp = ctypes.byref(params) if isinstance(params, Params) else None
    up = ctypes.byref(params) if isinstance(params, Uniform) else None
    if pp is None and up is None:
        raise ValueError("params must be a Params or a Uniform")
    _check(lib().logbq_gptq(c_void_p(w.data_ptr()), n, k, c_void_p(u.data_ptr()), pp, up,
                            c_void_p(workspace.data_ptr()), c_void_p(out_codes.data_ptr()),
                            _stream(stream)), "logbq_gptq")
    return out_codes
