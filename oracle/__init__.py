"""CPU oracle for the AF1 binary-factorized linear layer (fp64, plain C).

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check of the build entry
point and the benchmark's cpu_baseline leg may import this package.  The HIP
library never imports, links or calls it, and it never calls the library.

This module only marshals numpy arrays into ``liboracle.so`` (built from
``af1_oracle.c`` by ``build_oracle.py``).  Every function cites, in the C
source, the passage of the paper it follows:

- ``forward``: the factorised product of App. A.2.1 (Diag form) / Sec. 4.1,
  y = s_out .* (Bu (s_mid .* (Bv (s_in .* x)))), all in fp64.
- ``what_dense`` / ``what_packed``: the entry-wise path sum of App. A.2.1.
- ``storage_bits`` / ``bpw``: the deployable-storage count of App. A.3.
- ``budget_rank``: the largest rank (multiple of 32) within 1.0 BPW.
- ``paper_rank``: the budget-to-rank rounding rule of App. A.1.3.
- ``transpose_packed``: the packed storage of a sign matrix's transpose.
- ``backward``: the gradients of the scale-only reconstruction of Sec. 4.1
  (sign matrices frozen) with respect to s_out, s_mid, s_in and x.

The NABF building blocks (surrogate, SVID, null-space projector, ADMM
proxies, scale fits, one iteration of Algorithm nabf) are in ``nabf.py``,
fp64 numpy.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

SRC_F32, SRC_BF16, SRC_F16, SRC_I8 = 0, 1, 2, 3
_DTYPE_CODES = {np.dtype(np.float32): SRC_F32, np.dtype(np.float16): SRC_F16,
                np.dtype(np.int8): SRC_I8}


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build_oracle
        build_oracle.build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    lib.oracle_f16_to_f64.argtypes = [ctypes.c_uint16]
    lib.oracle_f16_to_f64.restype = ctypes.c_double
    lib.oracle_bf16_to_f64.argtypes = [ctypes.c_uint16]
    lib.oracle_bf16_to_f64.restype = ctypes.c_double
    lib.oracle_pack.argtypes = [P, ctypes.c_int, I64, I64, P]
    lib.oracle_unpack.argtypes = [P, I64, I64, P]
    lib.oracle_forward.argtypes = [I64, I64, I64, P, P, P, P, P, P, I64, P]
    lib.oracle_transpose_packed.argtypes = [P, I64, I64, P]
    lib.oracle_backward.argtypes = [I64, I64, I64, P, P, P, P, P, P, P, I64,
                                    P, P, P, P]
    lib.oracle_what_dense.argtypes = [I64, I64, I64, P, P, P, P, P, P]
    lib.oracle_what_packed.argtypes = [I64, I64, I64, P, P, P, P, P, P]
    lib.oracle_storage_bits.argtypes = [I64, I64, I64]
    lib.oracle_storage_bits.restype = I64
    lib.oracle_bpw.argtypes = [I64, P, P, P]
    lib.oracle_bpw.restype = ctypes.c_double
    lib.oracle_budget_rank.argtypes = [I64, I64, I64]
    lib.oracle_budget_rank.restype = I64
    lib.oracle_paper_rank.argtypes = [ctypes.c_double, I64, I64]
    lib.oracle_paper_rank.restype = I64
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    _lib = lib
    return lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    a = np.ascontiguousarray(a)
    if a.dtype != np.dtype(dtype):
        raise TypeError(f"expected {np.dtype(dtype)}, got {a.dtype}")
    return a


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} failed with code {rc}")


def f16_to_f64(h: int) -> float:
    return _load().oracle_f16_to_f64(int(h))


def bf16_to_f64(h: int) -> float:
    return _load().oracle_bf16_to_f64(int(h))


def pack(src: np.ndarray, bf16_bits: bool = False) -> np.ndarray:
    """Pack a rows x cols matrix of signs into rows x cols/32 uint32 words.

    ``src`` is float32, float16, int8, or uint16 bfloat16 patterns (pass
    ``bf16_bits=True`` for the latter)."""
    src = np.ascontiguousarray(src)
    if bf16_bits:
        src = _c(src, np.uint16)
        code = SRC_BF16
    else:
        code = _DTYPE_CODES[src.dtype]
    rows, cols = src.shape
    out = np.empty((rows, cols // 32), dtype=np.uint32)
    _check(_load().oracle_pack(_ptr(src), code, rows, cols, _ptr(out)), "pack")
    return out


def unpack(words: np.ndarray, cols: int) -> np.ndarray:
    words = _c(words, np.uint32)
    rows = words.shape[0]
    out = np.empty((rows, cols), dtype=np.int8)
    _check(_load().oracle_unpack(_ptr(words), rows, cols, _ptr(out)), "unpack")
    return out


def forward(m, n, r, Bu, Bv, s_out, s_mid, s_in, x) -> np.ndarray:
    """fp64 y[b, m] for packed factors, binary16 scales and bfloat16 x[b, n]."""
    Bu = _c(Bu, np.uint32); Bv = _c(Bv, np.uint32)
    s_out = _c(s_out, np.uint16); s_mid = _c(s_mid, np.uint16)
    s_in = _c(s_in, np.uint16); x = _c(x, np.uint16)
    b = x.shape[0]
    y = np.empty((b, m), dtype=np.float64)
    _check(_load().oracle_forward(m, n, r, _ptr(Bu), _ptr(Bv), _ptr(s_out),
                                  _ptr(s_mid), _ptr(s_in), _ptr(x), b, _ptr(y)),
           "forward")
    return y


def transpose_packed(words: np.ndarray, cols: int) -> np.ndarray:
    """Packed cols x rows storage of the transpose of a packed rows x cols
    sign matrix."""
    words = _c(words, np.uint32)
    rows = words.shape[0]
    out = np.empty((cols, rows // 32), dtype=np.uint32)
    _check(_load().oracle_transpose_packed(_ptr(words), rows, cols, _ptr(out)),
           "transpose_packed")
    return out


def backward(m, n, r, Bu, Bv, s_out, s_mid, s_in, x, dy):
    """fp64 (dx[b, n], ds_out[m], ds_mid[r], ds_in[n]) for the upstream
    gradient dy[b, m] (bfloat16 patterns), sign matrices frozen."""
    Bu = _c(Bu, np.uint32); Bv = _c(Bv, np.uint32)
    s_out = _c(s_out, np.uint16); s_mid = _c(s_mid, np.uint16)
    s_in = _c(s_in, np.uint16); x = _c(x, np.uint16); dy = _c(dy, np.uint16)
    b = x.shape[0]
    if dy.shape != (b, m) or x.shape != (b, n):
        raise ValueError("x must be b x n and dy b x m")
    dx = np.empty((b, n), dtype=np.float64)
    ds_out = np.empty(m, dtype=np.float64)
    ds_mid = np.empty(r, dtype=np.float64)
    ds_in = np.empty(n, dtype=np.float64)
    _check(_load().oracle_backward(m, n, r, _ptr(Bu), _ptr(Bv), _ptr(s_out),
                                   _ptr(s_mid), _ptr(s_in), _ptr(x), _ptr(dy), b,
                                   _ptr(dx), _ptr(ds_out), _ptr(ds_mid), _ptr(ds_in)),
           "backward")
    return dx, ds_out, ds_mid, ds_in


def what_dense(A, B, a, lam, bvec) -> np.ndarray:
    """Reconstructed matrix from dense +-1 factors and double scales."""
    A = _c(A, np.int8); B = _c(B, np.int8)
    a = _c(a, np.float64); lam = _c(lam, np.float64); bvec = _c(bvec, np.float64)
    m, r = A.shape
    n = B.shape[1]
    W = np.empty((m, n), dtype=np.float64)
    _check(_load().oracle_what_dense(m, n, r, _ptr(A), _ptr(B), _ptr(a),
                                     _ptr(lam), _ptr(bvec), _ptr(W)), "what_dense")
    return W


def what_packed(m, n, r, Bu, Bv, s_out, s_mid, s_in) -> np.ndarray:
    Bu = _c(Bu, np.uint32); Bv = _c(Bv, np.uint32)
    s_out = _c(s_out, np.uint16); s_mid = _c(s_mid, np.uint16)
    s_in = _c(s_in, np.uint16)
    W = np.empty((m, n), dtype=np.float64)
    _check(_load().oracle_what_packed(m, n, r, _ptr(Bu), _ptr(Bv), _ptr(s_out),
                                      _ptr(s_mid), _ptr(s_in), _ptr(W)),
           "what_packed")
    return W


def storage_bits(m, n, r) -> int:
    return int(_load().oracle_storage_bits(m, n, r))


def bpw(ms, ns, rs) -> float:
    ms = np.ascontiguousarray(ms, dtype=np.int64)
    ns = np.ascontiguousarray(ns, dtype=np.int64)
    rs = np.ascontiguousarray(rs, dtype=np.int64)
    return float(_load().oracle_bpw(len(ms), _ptr(ms), _ptr(ns), _ptr(rs)))


def budget_rank(m, n, multiple=32) -> int:
    return int(_load().oracle_budget_rank(m, n, multiple))


def paper_rank(bits_per_weight, m, n) -> int:
    return int(_load().oracle_paper_rank(float(bits_per_weight), m, n))


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(t: int) -> None:
    _load().oracle_set_num_threads(int(t))
