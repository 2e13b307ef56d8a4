"""ctypes binding of libaf1_nabf.so (include/af1_nabf.h): the NABF building
blocks (Sec. 4.1, Algorithm nabf, App. A.1.4, App. A.2.2-A.2.5).  Argument
marshalling only; every step runs in the library.  Loading raises when the
library has not been built: there is no fallback path."""
import ctypes
import os

from .af1 import _addr, _stream, _check, af1_factorized_linear  # noqa: F401

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libaf1_nabf.so")
AF1_NABF_MAX_DIM = 65536
AF1_NABF_MAX_TOKENS = 1 << 20
AF1_NABF_MAX_POWER_ITERS = 1000
_lib = None


class af1_nabf_state(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int64), ("n", ctypes.c_int64), ("r", ctypes.c_int64),
                ("A", ctypes.c_void_p), ("B", ctypes.c_void_p), ("UA", ctypes.c_void_p),
                ("UB", ctypes.c_void_p), ("A_bits", ctypes.c_void_p), ("B_bits", ctypes.c_void_p),
                ("a", ctypes.c_void_p), ("m1", ctypes.c_void_p), ("m2", ctypes.c_void_p),
                ("b", ctypes.c_void_p)]


def lib():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(there is no fallback path)")
    L = ctypes.CDLL(LIB_PATH)
    P, I64, I32, SZ, F = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t,
                          ctypes.c_float)
    S = ctypes.POINTER(af1_nabf_state)
    L.af1_nabf_workspace_bytes.argtypes = [I64, I64, I64, I64]
    L.af1_nabf_workspace_bytes.restype = SZ
    L.af1_nabf_surrogate.argtypes = [P, I64, I64, P, P, I64, P, P, P, P, SZ, P]
    L.af1_svid.argtypes = [P, I64, I64, I32, P, P, P, P, SZ, P]
    L.af1_nullspace_projector.argtypes = [P, I64, F, P, P, P, SZ, P]
    L.af1_admm_proxy.argtypes = [I32, P, I64, I64, I64, P, P, P, F, P, P, SZ, P]
    L.af1_scale_fit.argtypes = [I32, P, P, P, P, I64, I64, P, P, P, SZ, P]
    L.af1_nabf_iteration.argtypes = [P, S, F, F, I32, P, SZ, P]
    L.af1_nabf_export.argtypes = [S, P, P, P, P, P, P]
    for fn in ("af1_nabf_surrogate", "af1_svid", "af1_nullspace_projector", "af1_admm_proxy",
               "af1_scale_fit", "af1_nabf_iteration", "af1_nabf_export"):
        getattr(L, fn).restype = I32
    _lib = L
    return L


def _ret(st, name, check):
    if check:
        _check(st, name)
    return st


def make_state(m, n, r, A, B, UA, UB, A_bits, B_bits, a, m1, m2, b) -> af1_nabf_state:
    return af1_nabf_state(m, n, r, *[_addr(t) for t in (A, B, UA, UB, A_bits, B_bits, a, m1, m2, b)])


def af1_nabf_workspace_bytes(m, n, r, T=0) -> int:
    return int(lib().af1_nabf_workspace_bytes(m, n, r, T))


def af1_nabf_surrogate(W, m, n, X, G, T, Wp, i_vec, o_vec, ws, ws_bytes, stream=None, check=True):
    return _ret(lib().af1_nabf_surrogate(_addr(W), m, n, _addr(X), _addr(G), T, _addr(Wp),
                                         _addr(i_vec), _addr(o_vec), _addr(ws), ws_bytes,
                                         _stream(stream)), "af1_nabf_surrogate", check)


def af1_svid(Z, rows, cols, iters, bits, left, right, ws, ws_bytes, stream=None, check=True):
    return _ret(lib().af1_svid(_addr(Z), rows, cols, iters, _addr(bits), _addr(left),
                               _addr(right), _addr(ws), ws_bytes, _stream(stream)),
                "af1_svid", check)


def af1_nullspace_projector(C, r, eta, P, k_out, ws, ws_bytes, stream=None, check=True):
    return _ret(lib().af1_nullspace_projector(_addr(C), r, eta, _addr(P), _addr(k_out),
                                              _addr(ws), ws_bytes, _stream(stream)),
                "af1_nullspace_projector", check)


def af1_admm_proxy(side, Wp, m, n, r, A, B, U, rho, out, ws, ws_bytes, stream=None, check=True):
    return _ret(lib().af1_admm_proxy(side, _addr(Wp), m, n, r, _addr(A), _addr(B), _addr(U), rho,
                                     _addr(out), _addr(ws), ws_bytes, _stream(stream)),
                "af1_admm_proxy", check)


def af1_scale_fit(side, hat, bits, left, right, rows, cols, P, fit, ws, ws_bytes, stream=None,
                  check=True):
    return _ret(lib().af1_scale_fit(side, _addr(hat), _addr(bits), _addr(left), _addr(right),
                                    rows, cols, _addr(P), _addr(fit), _addr(ws), ws_bytes,
                                    _stream(stream)), "af1_scale_fit", check)


def af1_nabf_iteration(Wp, state, rho, eta, power_iters, ws, ws_bytes, stream=None, check=True):
    ref = ctypes.byref(state) if state is not None else None
    return _ret(lib().af1_nabf_iteration(_addr(Wp), ref, rho, eta, power_iters, _addr(ws),
                                         ws_bytes, _stream(stream)), "af1_nabf_iteration", check)


def af1_nabf_export(state, i_vec, o_vec, s_out, s_mid, s_in, stream=None, check=True):
    ref = ctypes.byref(state) if state is not None else None
    return _ret(lib().af1_nabf_export(ref, _addr(i_vec), _addr(o_vec), _addr(s_out),
                                      _addr(s_mid), _addr(s_in), _stream(stream)),
                "af1_nabf_export", check)
