"""Thin ctypes binding of ``libawe.so`` (declared in include/awe.h).

Names follow the C ABI.  This module only marshals arguments: device buffers
are torch tensors (or raw integer device pointers), the stream defaults to
torch's current stream, and every step of the computation runs in the HIP
library.  If the library has not been built, ``lib()`` raises; nothing here
falls back to another implementation.
"""
import ctypes
import os
import re

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libawe.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "awe.h")

# awe_status
OK, ERR_INVALID_VALUE, ERR_UNSUPPORTED, ERR_OVERFLOW, ERR_WORKSPACE, ERR_HIP, ERR_TABLE = range(7)
_FORMATS = ("e2m1", "e4m3", "e2m3")  # element format codes of awe_encoding_info
# awe_encoding
ENC_B13, ENC_AWE6, ENC_AWE6ALT, ENC_AWE4, ENC_MOD, ENC_TERNARY, ENC_FP16, ENC_FP8FP4, ENC_FP6K3, \
    ENC_FP6P4 = 1, 2, 3, 4, 5, 6, 7, 8, 9, 10
ENCODINGS = {"b13": ENC_B13, "awe6": ENC_AWE6, "awe6_alt": ENC_AWE6ALT, "awe4": ENC_AWE4, "mod": ENC_MOD,
             "ternary": ENC_TERNARY, "fp16_12": ENC_FP16, "fp8fp4": ENC_FP8FP4,
             "fp6k3": ENC_FP6K3, "fp6p4": ENC_FP6P4}
# awe_side, awe_dtype
SIDE_A, SIDE_B = 0, 1
I32, I64 = 0, 1

MAX_LIMBS, MAX_PLANES, MAX_PRODUCTS = 4, 8, 16
K_PAD = 256  # AWE_K_PAD: stored planes pad the reduction length to a multiple of this
NOALLOC_MAX_BYTES = 64 << 20  # AWE_NOALLOC_MAX_BYTES: the planes array of gemm_exact_noalloc


class EncodingInfo(ctypes.Structure):
    _fields_ = [
        ("r", ctypes.c_int32),
        ("limbs_a", ctypes.c_int32), ("limbs_b", ctypes.c_int32),
        ("planes_a", ctypes.c_int32), ("planes_b", ctypes.c_int32),
        ("log2_D", ctypes.c_int32),
        ("c_a", ctypes.c_int32), ("c_b", ctypes.c_int32),
        ("n_g", ctypes.c_int32),
        ("modulus", ctypes.c_int32),
        ("xmin_a", ctypes.c_int32), ("xmax_a", ctypes.c_int32),
        ("xmin_b", ctypes.c_int32), ("xmax_b", ctypes.c_int32),
        ("coverage_a", ctypes.c_int32), ("coverage_b", ctypes.c_int32),
        ("w", ctypes.c_int32 * MAX_LIMBS), ("v", ctypes.c_int32 * MAX_LIMBS),
        ("alpha", (ctypes.c_int32 * MAX_LIMBS) * MAX_PLANES),
        ("beta", (ctypes.c_int32 * MAX_LIMBS) * MAX_PLANES),
        ("pair_a", ctypes.c_int32 * MAX_PRODUCTS), ("pair_b", ctypes.c_int32 * MAX_PRODUCTS),
        ("ell", ctypes.c_int64 * MAX_PRODUCTS),
        ("group", ctypes.c_int32 * MAX_PRODUCTS),
        ("k_star", ctypes.c_int64), ("k_seg", ctypes.c_int64),
        ("format_a", ctypes.c_int32 * MAX_PLANES), ("format_b", ctypes.c_int32 * MAX_PLANES),
    ]


class AweError(RuntimeError):
    def __init__(self, status, where, detail):
        self.status = status
        super().__init__("%s: %s (%d)%s" % (where, _status_string(status), status,
                                            (": " + detail) if detail else ""))


_lib = None
_I32, _I64, _SZ, _P = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p


def lib():
    """The loaded library; raises if it has not been built (no fallback exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libawe.so is not built: run `python -m paper_2609_24519_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.awe_get_encoding_info.argtypes = [_I32, _I32, ctypes.POINTER(EncodingInfo)]
        L.awe_get_plane_table.argtypes = [_I32, _I32, _I32, _P, _I64]
        L.awe_plane_bytes.argtypes = [_I32, _I32, _I32, _I64, _I64, ctypes.POINTER(_SZ)]
        L.awe_encode.argtypes = [_I32, _I32, _I32, _P, _I64, _I64, _I64, _P, _P, _P]
        L.awe_gemm_planes.argtypes = [_I32, _I32, _I64, _I64, _I64, _P, _P, _P, _I64, _I32, _I64, _P]
        L.awe_workspace_bytes.argtypes = [_I32, _I32, _I64, _I64, _I64, ctypes.POINTER(_SZ)]
        L.awe_gemm_exact.argtypes = [_I32, _I64, _I64, _I64, _P, _I64, _P, _I64, _P, _I64, _I32,
                                     _P, _SZ, _P, _P]
        L.awe_gemm_mod.argtypes = [_I32, _I64, _I64, _I64, _P, _I64, _P, _I64, _P, _I64,
                                   _P, _SZ, _P, _P]
        L.awe_gemm_exact_noalloc.argtypes = [_I32, _I64, _I64, _I64, _P, _I64, _P, _I64, _P, _I64, _I32,
                                             _P, _P]
        L.awe_residues.argtypes = [_P, _I64, _I64, _I64, _I64, _P, _I32, _P, _I64, _P, _P]
        L.awe_crt.argtypes = [_P, _I64, _I64, _I64, _I64, _P, _I32, _P, _P, _I64, _P]
        L.awe_crt_workspace_bytes.argtypes = [_P, _I32, _I64, _I64, _I64, ctypes.POINTER(_SZ)]
        L.awe_gemm_crt.argtypes = [_I64, _I64, _I64, _P, _I64, _P, _I64, _I64, _I64, _P, _I32,
                                   _P, _P, _I64, _P, _SZ, _P, _P]
        L.awe_status_string.argtypes = [_I32]
        L.awe_status_string.restype = ctypes.c_char_p
        L.awe_last_error.argtypes = []
        L.awe_last_error.restype = ctypes.c_char_p
        for name in ("awe_get_encoding_info", "awe_get_plane_table", "awe_plane_bytes", "awe_encode",
                     "awe_gemm_planes", "awe_workspace_bytes", "awe_gemm_exact", "awe_gemm_exact_noalloc",
                     "awe_gemm_mod",
                     "awe_residues", "awe_crt", "awe_crt_workspace_bytes", "awe_gemm_crt"):
            getattr(L, name).restype = _I32
        _lib = L
    return _lib


def header_symbols():
    """Names of the functions include/awe.h declares."""
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(awe_[a-z_0-9]+)\s*\(", text)))


def _status_string(st):
    try:
        return lib().awe_status_string(st).decode()
    except Exception:  # noqa: BLE001 - message only
        return "status"


def _check(st, where):
    if st != OK:
        raise AweError(st, where, lib().awe_last_error().decode())


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ---- host queries -----------------------------------------------------------
def get_encoding_info(enc, modulus=0):
    info = EncodingInfo()
    _check(lib().awe_get_encoding_info(enc, modulus, ctypes.byref(info)), "awe_get_encoding_info")
    r = info.r
    return {
        "r": r, "limbs_a": info.limbs_a, "limbs_b": info.limbs_b,
        "planes_a": info.planes_a, "planes_b": info.planes_b, "log2_D": info.log2_D,
        "c_a": info.c_a, "c_b": info.c_b, "n_g": info.n_g, "modulus": info.modulus,
        "range_a": (info.xmin_a, info.xmax_a), "range_b": (info.xmin_b, info.xmax_b),
        "coverage_a": info.coverage_a, "coverage_b": info.coverage_b,
        "w": tuple(info.w[:info.limbs_a]), "v": tuple(info.v[:info.limbs_b]),
        "alpha": [tuple(info.alpha[k][:info.limbs_a]) for k in range(info.planes_a)],
        "beta": [tuple(info.beta[k][:info.limbs_b]) for k in range(info.planes_b)],
        "pair_a": list(info.pair_a[:r]), "pair_b": list(info.pair_b[:r]),
        "ell": list(info.ell[:r]), "group": list(info.group[:r]),
        "k_star": info.k_star, "k_seg": info.k_seg,
        "formats_a": [_FORMATS[f] for f in info.format_a[:info.planes_a]],
        "formats_b": [_FORMATS[f] for f in info.format_b[:info.planes_b]],
    }


def get_plane_table(enc, modulus, side):
    """(xmin, T) with T[x - xmin, k] the stored value of plane k for input x."""
    info = get_encoding_info(enc, modulus)
    lo, hi = info["range_a"] if side == SIDE_A else info["range_b"]
    npl = info["planes_a"] if side == SIDE_A else info["planes_b"]
    T = np.zeros((hi - lo + 1, npl), dtype=np.int32)
    _check(lib().awe_get_plane_table(enc, modulus, side, T.ctypes.data, T.size), "awe_get_plane_table")
    return lo, T


def plane_bytes(enc, modulus, side, rows, K):
    n = _SZ()
    _check(lib().awe_plane_bytes(enc, modulus, side, rows, K, ctypes.byref(n)), "awe_plane_bytes")
    return n.value


def workspace_bytes(enc, modulus, M, N, K):
    n = _SZ()
    _check(lib().awe_workspace_bytes(enc, modulus, M, N, K, ctypes.byref(n)), "awe_workspace_bytes")
    return n.value


# ---- device calls (same argument order as the C ABI) ----------------------------
def encode(enc, modulus, side, x, rows, K, ld, planes, d_range_flag=None, stream=None):
    _check(lib().awe_encode(enc, modulus, side, _ptr(x), rows, K, ld, _ptr(planes),
                            _ptr(d_range_flag), _stream(stream)), "awe_encode")


def gemm_planes(enc, modulus, M, N, K, planes_a, planes_b, C, ldc, c_type, k_seg=0, stream=None):
    _check(lib().awe_gemm_planes(enc, modulus, M, N, K, _ptr(planes_a), _ptr(planes_b), _ptr(C),
                                 ldc, c_type, k_seg, _stream(stream)), "awe_gemm_planes")


def gemm_exact(enc, M, N, K, A, lda, B, ldb, C, ldc, c_type, workspace, ws_bytes,
               d_range_flag=None, stream=None):
    _check(lib().awe_gemm_exact(enc, M, N, K, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc, c_type,
                                _ptr(workspace), ws_bytes, _ptr(d_range_flag), _stream(stream)),
           "awe_gemm_exact")


def gemm_exact_noalloc(enc, M, N, K, A, lda, B, ldb, C, ldc, c_type, d_range_flag=None, stream=None):
    _check(lib().awe_gemm_exact_noalloc(enc, M, N, K, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc, c_type,
                                        _ptr(d_range_flag), _stream(stream)), "awe_gemm_exact_noalloc")


def gemm_mod(m, M, N, K, A, lda, B, ldb, C, ldc, workspace, ws_bytes, d_range_flag=None, stream=None):
    _check(lib().awe_gemm_mod(m, M, N, K, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc, _ptr(workspace),
                              ws_bytes, _ptr(d_range_flag), _stream(stream)), "awe_gemm_mod")


# ---- residue number system (moduli: a sequence of ints, passed as a host int32 array) ----
def _moduli(moduli):
    arr = (ctypes.c_int32 * len(moduli))(*[int(m) for m in moduli])
    return arr, len(moduli)


def residues(x, rows, cols, ld, bound, moduli, out, out_stride, d_range_flag=None, stream=None):
    arr, n = _moduli(moduli)
    _check(lib().awe_residues(_ptr(x), rows, cols, ld, bound, arr, n, _ptr(out), out_stride,
                              _ptr(d_range_flag), _stream(stream)), "awe_residues")


def crt(res, res_stride, rows, cols, ld_res, moduli, c128=None, c64=None, ldc=None, stream=None):
    arr, n = _moduli(moduli)
    _check(lib().awe_crt(_ptr(res), res_stride, rows, cols, ld_res, arr, n, _ptr(c128), _ptr(c64),
                         cols if ldc is None else ldc, _stream(stream)), "awe_crt")


def crt_workspace_bytes(moduli, M, N, K):
    arr, n = _moduli(moduli)
    out = _SZ(0)
    _check(lib().awe_crt_workspace_bytes(arr, n, M, N, K, ctypes.byref(out)), "awe_crt_workspace_bytes")
    return out.value


def gemm_crt(M, N, K, A, lda, B, ldb, bound_a, bound_b, moduli, c128, c64, ldc, workspace, ws_bytes,
             d_range_flag=None, stream=None):
    arr, n = _moduli(moduli)
    _check(lib().awe_gemm_crt(M, N, K, _ptr(A), lda, _ptr(B), ldb, bound_a, bound_b, arr, n,
                              _ptr(c128), _ptr(c64), ldc, _ptr(workspace), ws_bytes,
                              _ptr(d_range_flag), _stream(stream)), "awe_gemm_crt")


# ---- torch conveniences (allocation with torch, then the calls above) -------------
def matmul_exact(A, B, enc=ENC_AWE6, out_dtype=None, d_range_flag=None):
    """C = A B exactly for int8 CUDA tensors A (M x K) and B (K x N)."""
    import torch
    M, K = A.shape
    K2, N = B.shape
    if K != K2:
        raise ValueError("inner dimensions differ")
    out_dtype = out_dtype or torch.int32
    c_type = I64 if out_dtype == torch.int64 else I32
    C = torch.empty((M, N), dtype=out_dtype, device=A.device)
    ws_n = workspace_bytes(enc, 0, M, N, K)
    ws = torch.empty(max(ws_n, 1), dtype=torch.uint8, device=A.device)
    gemm_exact(enc, M, N, K, A, A.stride(0), B, B.stride(0), C, C.stride(0), c_type, ws, ws_n,
               d_range_flag)
    return C


def matmul_mod(m, A, B, d_range_flag=None):
    """(A B) mod m for uint8 residue CUDA tensors."""
    import torch
    M, K = A.shape
    _, N = B.shape
    C = torch.empty((M, N), dtype=torch.int32, device=A.device)
    ws_n = workspace_bytes(ENC_MOD, m, M, N, K)
    ws = torch.empty(max(ws_n, 1), dtype=torch.uint8, device=A.device)
    gemm_mod(m, M, N, K, A, A.stride(0), B, B.stride(0), C, C.stride(0), ws, ws_n, d_range_flag)
    return C


def matmul_crt(A, B, moduli, bound_a, bound_b, d_range_flag=None):
    """Exact A B for int64 CUDA tensors through residues; returns (c128, c64): the integer as
    an int64 tensor of shape (M, N, 2) holding (low, high) words, and its nearest double."""
    import torch
    M, K = A.shape
    _, N = B.shape
    c128 = torch.empty((M, N, 2), dtype=torch.int64, device=A.device)
    c64 = torch.empty((M, N), dtype=torch.float64, device=A.device)
    ws_n = crt_workspace_bytes(moduli, M, N, K)
    ws = torch.empty(max(ws_n, 1), dtype=torch.uint8, device=A.device)
    gemm_crt(M, N, K, A, A.stride(0), B, B.stride(0), bound_a, bound_b, moduli, c128, c64, N, ws, ws_n,
             d_range_flag)
    return c128, c64
