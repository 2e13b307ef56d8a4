"""Device-resident factorized layer: the packed signs and fp16 scales held as
torch CUDA tensors (plumbing only), plus the C descriptor that points at them.
"""
import contextlib

import numpy as np
import torch

from . import af1

_VIEW = {np.dtype(np.uint32): np.int32, np.dtype(np.uint16): np.int16,
         np.dtype(np.uint8): np.uint8, np.dtype(np.int8): np.int8,
         np.dtype(np.float32): np.float32, np.dtype(np.float16): np.float16}


def to_device(a: np.ndarray, device="cuda") -> torch.Tensor:
    """Copy a host array to the device byte for byte (unsigned 32/16-bit
    patterns travel as signed views of the same bits)."""
    a = np.ascontiguousarray(a)
    return torch.from_numpy(a.view(_VIEW[a.dtype])).to(device)


def on_stream(stream):
    """Context in which the helpers below allocate their outputs and
    workspaces: the stream the kernels are launched on (torch's current one
    when stream is None), so a zero-fill is ordered before the kernels and
    the caching allocator does not hand the memory to other work while they
    may still use it."""
    if stream is None or isinstance(stream, int):
        # an integer stream handle: the caller owns ordering and lifetimes
        return contextlib.nullcontext()
    return torch.cuda.stream(stream)


def bf16_bits_to_f64(t: torch.Tensor) -> np.ndarray:
    """Host float64 values of a tensor of bfloat16 bit patterns."""
    u = t.detach().cpu().numpy().view(np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


class DeviceLayer:
    def __init__(self, m, n, r, Bu, Bv, s_out, s_mid, s_in, device="cuda"):
        self.m, self.n, self.r = int(m), int(n), int(r)
        self.Bu = to_device(Bu, device)
        self.Bv = to_device(Bv, device)
        self.s_out = to_device(s_out, device)
        self.s_mid = to_device(s_mid, device)
        self.s_in = to_device(s_in, device)
        self.desc = af1.make_layer(self.m, self.n, self.r, self.Bu, self.Bv,
                                   self.s_out, self.s_mid, self.s_in)

    @classmethod
    def from_host(cls, lin, device="cuda"):
        return cls(lin.m, lin.n, lin.r, lin.Bu, lin.Bv, lin.s_out, lin.s_mid, lin.s_in, device)

    def storage_bytes(self) -> int:
        return af1.af1_storage_bits(self.m, self.n, self.r) // 8

    def gemv(self, x: torch.Tensor, y: torch.Tensor = None, ws: torch.Tensor = None, stream=None):
        b = x.shape[0]
        with on_stream(stream):
            if y is None:
                y = torch.empty((b, self.m), dtype=torch.int16, device=x.device)
            need = af1.af1_gemv_workspace_bytes(self.m, self.n, self.r, b)
            if ws is None:
                # zero-filled: the decode path keeps arrival counters here
                ws = torch.zeros(max(need, 256), dtype=torch.uint8, device=x.device)
            af1.af1_linear_gemv(self.desc, x, b, y, ws, ws.numel(), stream)
        return y

    def gemm(self, x: torch.Tensor, y: torch.Tensor = None, ws: torch.Tensor = None, stream=None):
        T = x.shape[0]
        with on_stream(stream):
            if y is None:
                y = torch.empty((T, self.m), dtype=torch.int16, device=x.device)
            need = af1.af1_gemm_workspace_bytes(self.m, self.n, self.r, T)
            if ws is None:
                ws = torch.empty(max(need, 256), dtype=torch.uint8, device=x.device)
            af1.af1_linear_gemm(self.desc, x, T, y, ws, ws.numel(), stream)
        return y

    # -- scale-only reconstruction: signs frozen, scales trained -----------

    def transposed(self, stream=None):
        """(Bu^T, Bv^T) in the packed format, made once on the device."""
        if getattr(self, "_T", None) is None:
            BuT = torch.empty((self.r, self.m // 32), dtype=torch.int32, device=self.Bu.device)
            BvT = torch.empty((self.n, self.r // 32), dtype=torch.int32, device=self.Bu.device)
            af1.af1_pack_transpose(self.Bu, self.m, self.r, BuT, stream)
            af1.af1_pack_transpose(self.Bv, self.r, self.n, BvT, stream)
            self._T = (BuT, BvT)
        return self._T

    def forward_train(self, x, y=None, saved=None, ws=None, stream=None):
        T = x.shape[0]
        with on_stream(stream):
            if y is None:
                y = torch.empty((T, self.m), dtype=torch.int16, device=x.device)
            if saved is None:
                saved = torch.empty(af1.af1_train_saved_bytes(self.m, self.n, self.r, T),
                                    dtype=torch.uint8, device=x.device)
            if ws is None:
                ws = torch.empty(af1.af1_train_workspace_bytes(self.m, self.n, self.r, T),
                                 dtype=torch.uint8, device=x.device)
            af1.af1_linear_forward_train(self.desc, x, T, y, saved, saved.numel(), ws,
                                         ws.numel(), stream)
        return y, saved

    def backward(self, x, dy, saved, dx=None, grads=None, accumulate=False, ws=None,
                 stream=None, want_dx=True):
        """dx ([T, n] bf16 patterns, or None) and the fp32 scale gradients
        (ds_out, ds_mid, ds_in)."""
        T = x.shape[0]
        with on_stream(stream):
            BuT, BvT = self.transposed(stream)
            if dx is None and want_dx:
                dx = torch.empty((T, self.n), dtype=torch.int16, device=x.device)
            if grads is None:
                grads = tuple(torch.empty(k, dtype=torch.float32, device=x.device)
                              for k in (self.m, self.r, self.n))
            if ws is None:
                ws = torch.empty(af1.af1_train_workspace_bytes(self.m, self.n, self.r, T),
                                 dtype=torch.uint8, device=x.device)
            af1.af1_linear_backward(self.desc, BuT, BvT, x, dy, T, saved, saved.numel(), dx,
                                    grads[0], grads[1], grads[2], int(bool(accumulate)), ws,
                                    ws.numel(), stream)
        return dx, grads


def gemv_multi(layers, x: torch.Tensor, ys=None, ws: torch.Tensor = None, stream=None):
    """One decode step of several layers that read the same x (same n)."""
    b = x.shape[0]
    with on_stream(stream):
        if ys is None:
            ys = [torch.empty((b, L.m), dtype=torch.int16, device=x.device) for L in layers]
        descs = [L.desc for L in layers]
        need = af1.af1_gemv_multi_workspace_bytes(descs, b)
        if ws is None:
            ws = torch.zeros(max(need, 256), dtype=torch.uint8, device=x.device)
        af1.af1_linear_gemv_multi(descs, x, b, ys, ws, ws.numel(), stream)
    return ys


class LayerStream:
    """A decode pass over a sequence of layers in one persistent launch.

    entries: (DeviceLayer, x, y, wait) tuples, x / y device tensors of bf16
    patterns ([b, n] and [b, m]); wait=True makes an item start after every
    earlier item has finished (it may read their outputs).  The plan is built
    once here, bound to these buffers and to the zero-filled workspace, and
    copied to the device; run() launches one pass."""

    def __init__(self, entries, b, device="cuda"):
        self.entries = list(entries)
        self.b = int(b)
        self.items = af1.stream_items([(L.desc, x, y, w) for L, x, y, w in self.entries])
        ws_bytes = af1.af1_stream_workspace_bytes(self.items, self.b)
        plan_bytes = af1.af1_stream_plan_bytes(self.items, self.b)
        if ws_bytes == 0 or plan_bytes == 0:
            # report the argument error through the plan call
            af1.af1_stream_plan(self.items, self.b, None, 0, None, 0)
        self.ws = torch.zeros(ws_bytes, dtype=torch.uint8, device=device)
        # 16-byte aligned host buffer (numpy aligns large arrays further)
        self._plan_buf = np.zeros(plan_bytes + 16, np.uint8)
        off = (-self._plan_buf.ctypes.data) % 16
        self.plan = self._plan_buf[off:off + plan_bytes]
        af1.af1_stream_plan(self.items, self.b, self.ws, ws_bytes, self.plan, plan_bytes)
        self.plan_dev = torch.from_numpy(self.plan.copy()).to(device)

    def run(self, stream=None):
        af1.af1_linear_stream(self.plan, self.plan_dev, stream)

    def error_word(self) -> int:
        """Non-zero when a barrier of an earlier pass timed out."""
        return int(self.ws[4:8].view(torch.int32).item())
