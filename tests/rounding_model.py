"""First-order model of the error that the scale-only reconstruction path's
fp16 roundings put into its three scale gradients (Sec. 4.1), and a numpy
emulation of those roundings, for the tolerance of the training parity
tests.

The path rounds five quantities to binary16 (each at a power-of-two scale
that keeps it in the normal range, so the rounding is relative):
s_in.x and s_mid.v in the forward, the saved v, and s_out.dy and s_mid.dt in
the backward.  Modelled as independent relative errors of variance
(2^-11)^2 / 3, carried to first order through Bu, Bv and
W = Bu diag(s_mid) Bv, they give the predicted 2-norm error of ds_out, ds_mid
and ds_in.  Test infrastructure only."""
import numpy as np

U2 = (2.0 ** -11) ** 2 / 3   # variance of one round-to-nearest fp16 relative error


def f16_bits(h):
    return np.asarray(h, np.uint16).view(np.float16).astype(np.float64)


def bf16_bits(h):
    return (np.asarray(h, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _dense(oracle, lin, dy):
    Bu = oracle.unpack(lin.Bu, lin.r).astype(np.float64)
    Bv = oracle.unpack(lin.Bv, lin.n).astype(np.float64)
    return (Bu, Bv, f16_bits(lin.s_out), f16_bits(lin.s_mid), f16_bits(lin.s_in),
            bf16_bits(lin.x), bf16_bits(dy))


def rounding_noise(oracle, lin, dy):
    """Predicted 2-norm errors of (ds_out, ds_mid, ds_in)."""
    Bu, Bv, s_out, s_mid, s_in, x, g = _dense(oracle, lin, dy)
    sx = x * s_in
    v = sx @ Bv.T
    a = g * s_out
    dt = a @ Bu
    W2 = ((Bu * s_mid) @ Bv) ** 2

    def row(t):
        return (t ** 2).sum(1, keepdims=True)

    var_out = (g ** 2 * (row(v * s_mid) + (sx ** 2) @ W2.T)).sum()
    var_mid = (dt ** 2 * (row(sx) + v ** 2) + v ** 2 * row(a)).sum()
    var_in = (x ** 2 * ((a ** 2) @ W2 + row(dt * s_mid))).sum()
    return [float(np.sqrt(U2 * t)) for t in (var_out, var_mid, var_in)]


def _round_f16(t):
    """binary16 rounding of each row of t at the power of two that puts the
    row's largest magnitude in [2^13, 2^14)."""
    mx = np.abs(t).max(axis=1, keepdims=True)
    e = np.where(mx > 0, 13 - np.floor(np.log2(np.where(mx > 0, mx, 1.0))), 0.0)
    return (t * 2.0 ** e).astype(np.float16).astype(np.float64) * 2.0 ** -e


def emulate_gradients(oracle, lin, dy):
    """(ds_out, ds_mid, ds_in) with exactly the five roundings of the model
    and exact arithmetic everywhere else."""
    Bu, Bv, s_out, s_mid, s_in, x, g = _dense(oracle, lin, dy)
    v = _round_f16(x * s_in) @ Bv.T
    z = _round_f16(v * s_mid) @ Bu.T
    dt = _round_f16(g * s_out) @ Bu
    du = _round_f16(dt * s_mid) @ Bv
    return (g * z).sum(0), (dt * _round_f16(v)).sum(0), (x * du).sum(0)
