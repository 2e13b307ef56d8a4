"""Python binding of ``libaf1.so`` (C ABI in include/af1.h).

Argument marshalling only: every function forwards to the C entry point of
the same name, passing device pointers taken from torch tensors (or plain
integers) and the current HIP stream.  No computation happens here, and there
is no fallback: if the library is missing, every call raises.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libaf1.so")

AF1_OK = 0
AF1_ERR_NULL = 1
AF1_ERR_SHAPE = 2
AF1_ERR_BATCH = 3
AF1_ERR_ALIGN = 4
AF1_ERR_WORKSPACE = 5
AF1_ERR_ALIAS = 6
AF1_ERR_HIP = 7
AF1_ERR_DTYPE = 8
AF1_ERR_PLAN = 9

AF1_SRC_F32, AF1_SRC_BF16, AF1_SRC_F16, AF1_SRC_I8 = 0, 1, 2, 3
AF1_GEMV_MAX_BATCH = 16
AF1_GEMV_MULTI_MAX = 4
AF1_GEMV_SCRATCH_BYTES = 4 << 20
AF1_MAX_DIM = 1 << 20

AF1_STREAM_MAX_ITEMS = 4096

_lib = None


class Af1Error(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


class af1_factorized_linear(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int64), ("n", ctypes.c_int64), ("r", ctypes.c_int64),
                ("Bu", ctypes.c_void_p), ("Bv", ctypes.c_void_p),
                ("s_out", ctypes.c_void_p), ("s_mid", ctypes.c_void_p),
                ("s_in", ctypes.c_void_p)]


class af1_stream_item(ctypes.Structure):
    _fields_ = [("L", af1_factorized_linear), ("x", ctypes.c_void_p), ("y", ctypes.c_void_p),
                ("wait", ctypes.c_int32), ("reserved", ctypes.c_int32)]


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(there is no fallback path)")
    L = ctypes.CDLL(LIB_PATH)
    P, I64, I32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    L.af1_pack.argtypes = [P, I32, I64, I64, P, P]
    L.af1_unpack.argtypes = [P, I64, I64, P, P]
    L.af1_gemv_workspace_bytes.argtypes = [I64, I64, I64, I64]
    L.af1_gemv_workspace_bytes.restype = SZ
    L.af1_linear_gemv.argtypes = [ctypes.POINTER(af1_factorized_linear), P, I64, P, P, SZ, P]
    L.af1_gemv_multi_workspace_bytes.argtypes = [ctypes.POINTER(af1_factorized_linear), I32, I64]
    L.af1_gemv_multi_workspace_bytes.restype = SZ
    L.af1_linear_gemv_multi.argtypes = [ctypes.POINTER(af1_factorized_linear), I32, P, I64,
                                        ctypes.POINTER(P), P, SZ, P]
    L.af1_gemm_workspace_bytes.argtypes = [I64, I64, I64, I64]
    L.af1_gemm_workspace_bytes.restype = SZ
    L.af1_linear_gemm.argtypes = [ctypes.POINTER(af1_factorized_linear), P, I64, P, P, SZ, P]
    L.af1_pack_transpose.argtypes = [P, I64, I64, P, P]
    L.af1_train_saved_bytes.argtypes = [I64, I64, I64, I64]
    L.af1_train_saved_bytes.restype = SZ
    L.af1_train_workspace_bytes.argtypes = [I64, I64, I64, I64]
    L.af1_train_workspace_bytes.restype = SZ
    L.af1_linear_forward_train.argtypes = [ctypes.POINTER(af1_factorized_linear), P, I64, P, P,
                                           SZ, P, SZ, P]
    L.af1_linear_backward.argtypes = [ctypes.POINTER(af1_factorized_linear), P, P, P, P, I64, P,
                                      SZ, P, P, P, P, I32, P, SZ, P]
    SI = ctypes.POINTER(af1_stream_item)
    L.af1_stream_workspace_bytes.argtypes = [SI, I32, I64]
    L.af1_stream_workspace_bytes.restype = SZ
    L.af1_stream_plan_bytes.argtypes = [SI, I32, I64]
    L.af1_stream_plan_bytes.restype = SZ
    L.af1_stream_plan.argtypes = [SI, I32, I64, P, SZ, P, SZ]
    L.af1_linear_stream.argtypes = [P, P, P]
    L.af1_storage_bits.argtypes = [I64, I64, I64]
    L.af1_storage_bits.restype = I64
    L.af1_budget_rank.argtypes = [I64, I64, ctypes.c_double, I64]
    L.af1_budget_rank.restype = I64
    L.af1_paper_rank.argtypes = [I64, I64, ctypes.c_double]
    L.af1_paper_rank.restype = I64
    L.af1_linear_gemv_noalloc.argtypes = [ctypes.POINTER(af1_factorized_linear), P, I64, P, P]
    L.af1_status_string.argtypes = [I32]
    L.af1_status_string.restype = ctypes.c_char_p
    L.af1_version.restype = ctypes.c_char_p
    for fn in ("af1_pack", "af1_unpack", "af1_linear_gemv", "af1_linear_gemv_noalloc",
               "af1_linear_gemv_multi",
               "af1_linear_gemm", "af1_pack_transpose", "af1_linear_forward_train",
               "af1_linear_backward", "af1_stream_plan", "af1_linear_stream"):
        getattr(L, fn).restype = I32
    _lib = L
    return L


def _addr(t):
    """Device address of a torch tensor, or an integer address as is."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status, where):
    if status != AF1_OK:
        raise Af1Error(status, where)


def status_string(status: int) -> str:
    return lib().af1_status_string(int(status)).decode()


def af1_version() -> str:
    return lib().af1_version().decode()


def make_layer(m, n, r, Bu, Bv, s_out, s_mid, s_in) -> af1_factorized_linear:
    """The C descriptor of one factorized layer (device arrays)."""
    return af1_factorized_linear(m, n, r, _addr(Bu), _addr(Bv), _addr(s_out),
                                 _addr(s_mid), _addr(s_in))


def af1_pack(src, src_dtype: int, rows: int, cols: int, dst, stream=None, check=True) -> int:
    st = lib().af1_pack(_addr(src), src_dtype, rows, cols, _addr(dst), _stream(stream))
    if check:
        _check(st, "af1_pack")
    return st


def af1_unpack(words, rows: int, cols: int, dst, stream=None, check=True) -> int:
    st = lib().af1_unpack(_addr(words), rows, cols, _addr(dst), _stream(stream))
    if check:
        _check(st, "af1_unpack")
    return st


def af1_gemv_workspace_bytes(m, n, r, b) -> int:
    return int(lib().af1_gemv_workspace_bytes(m, n, r, b))


def af1_linear_gemv(layer, x, b: int, y, ws, ws_bytes: int, stream=None, check=True) -> int:
    ref = ctypes.byref(layer) if layer is not None else None
    st = lib().af1_linear_gemv(ref, _addr(x), b, _addr(y), _addr(ws), ws_bytes, _stream(stream))
    if check:
        _check(st, "af1_linear_gemv")
    return st


def af1_linear_gemv_noalloc(layer, x, b: int, y, stream=None, check=True) -> int:
    ref = ctypes.byref(layer) if layer is not None else None
    st = lib().af1_linear_gemv_noalloc(ref, _addr(x), b, _addr(y), _stream(stream))
    if check:
        _check(st, "af1_linear_gemv_noalloc")
    return st


def _layer_array(layers):
    arr = (af1_factorized_linear * len(layers))()
    for i, L in enumerate(layers):
        arr[i] = L
    return arr


def af1_gemv_multi_workspace_bytes(layers, b) -> int:
    return int(lib().af1_gemv_multi_workspace_bytes(_layer_array(layers), len(layers), b))


def af1_linear_gemv_multi(layers, x, b: int, ys, ws, ws_bytes: int, stream=None,
                          check=True) -> int:
    """layers: list of af1_factorized_linear; ys: list of outputs (tensors or
    addresses), one per layer.  The count passed is len(layers)."""
    arr = _layer_array(layers) if layers is not None else None
    yarr = (ctypes.c_void_p * len(ys))(*[_addr(y) for y in ys]) if ys is not None else None
    st = lib().af1_linear_gemv_multi(arr, len(layers) if layers is not None else 0, _addr(x), b,
                                     yarr, _addr(ws), ws_bytes, _stream(stream))
    if check:
        _check(st, "af1_linear_gemv_multi")
    return st


def af1_gemm_workspace_bytes(m, n, r, T) -> int:
    return int(lib().af1_gemm_workspace_bytes(m, n, r, T))


def af1_linear_gemm(layer, x, T: int, y, ws, ws_bytes: int, stream=None, check=True) -> int:
    ref = ctypes.byref(layer) if layer is not None else None
    st = lib().af1_linear_gemm(ref, _addr(x), T, _addr(y), _addr(ws), ws_bytes, _stream(stream))
    if check:
        _check(st, "af1_linear_gemm")
    return st


def af1_pack_transpose(src, rows: int, cols: int, dst, stream=None, check=True) -> int:
    st = lib().af1_pack_transpose(_addr(src), rows, cols, _addr(dst), _stream(stream))
    if check:
        _check(st, "af1_pack_transpose")
    return st


def af1_train_saved_bytes(m, n, r, T) -> int:
    return int(lib().af1_train_saved_bytes(m, n, r, T))


def af1_train_workspace_bytes(m, n, r, T) -> int:
    return int(lib().af1_train_workspace_bytes(m, n, r, T))


def af1_linear_forward_train(layer, x, T: int, y, saved, saved_bytes: int, ws, ws_bytes: int,
                             stream=None, check=True) -> int:
    ref = ctypes.byref(layer) if layer is not None else None
    st = lib().af1_linear_forward_train(ref, _addr(x), T, _addr(y), _addr(saved), saved_bytes,
                                        _addr(ws), ws_bytes, _stream(stream))
    if check:
        _check(st, "af1_linear_forward_train")
    return st


def af1_linear_backward(layer, BuT, BvT, x, dy, T: int, saved, saved_bytes: int, dx, ds_out,
                        ds_mid, ds_in, accumulate: int, ws, ws_bytes: int, stream=None,
                        check=True) -> int:
    ref = ctypes.byref(layer) if layer is not None else None
    st = lib().af1_linear_backward(ref, _addr(BuT), _addr(BvT), _addr(x), _addr(dy), T,
                                   _addr(saved), saved_bytes, _addr(dx), _addr(ds_out),
                                   _addr(ds_mid), _addr(ds_in), int(accumulate), _addr(ws),
                                   ws_bytes, _stream(stream))
    if check:
        _check(st, "af1_linear_backward")
    return st


def stream_items(entries):
    """A ctypes array of af1_stream_item from (layer descriptor, x, y, wait)
    tuples (x and y tensors or addresses)."""
    arr = (af1_stream_item * len(entries))()
    for i, (desc, x, y, wait) in enumerate(entries):
        arr[i] = af1_stream_item(desc, _addr(x), _addr(y), int(bool(wait)), 0)
    return arr


def af1_stream_workspace_bytes(items, b) -> int:
    return int(lib().af1_stream_workspace_bytes(items, len(items), b))


def af1_stream_plan_bytes(items, b) -> int:
    return int(lib().af1_stream_plan_bytes(items, len(items), b))


def af1_stream_plan(items, b: int, ws, ws_bytes: int, plan, plan_bytes: int, count=None,
                    check=True) -> int:
    """plan: a host buffer (an int address, or a numpy uint8 array)."""
    addr = plan if isinstance(plan, int) or plan is None else plan.ctypes.data
    n = len(items) if count is None else count
    st = lib().af1_stream_plan(items, n, b, _addr(ws), ws_bytes, addr, plan_bytes)
    if check:
        _check(st, "af1_stream_plan")
    return st


def af1_linear_stream(plan, plan_dev, stream=None, check=True) -> int:
    """plan: the host plan (numpy uint8 array or address); plan_dev: its
    device copy."""
    addr = plan if isinstance(plan, int) or plan is None else plan.ctypes.data
    st = lib().af1_linear_stream(addr, _addr(plan_dev), _stream(stream))
    if check:
        _check(st, "af1_linear_stream")
    return st


def af1_storage_bits(m, n, r) -> int:
    return int(lib().af1_storage_bits(m, n, r))


def af1_budget_rank(m, n, bpw=1.0, multiple=32) -> int:
    return int(lib().af1_budget_rank(m, n, float(bpw), multiple))


def af1_paper_rank(m, n, bpw) -> int:
    return int(lib().af1_paper_rank(m, n, float(bpw)))
