"""GPU parity of the forward paths across the input range bf16 allows.

The layer is defined for any x (App. A.2.1, Diag form), but the prefill
contractions run on fp16 operands (2^-24 .. 65504).  Both fp16 operands
carry a per-token power-of-two scale that is undone in fp32, so activations
far above and far below fp16's range give the oracle's result.  These tests
multiply the seeded N(0,1) x (with 1% x20 outlier channels) by powers of two
(exact in bf16) and by per-token factors spanning 10^12, then compare every
token with the fp64 oracle at the usual bars: relative L2 5e-3 per token,
plus an element-wise bound.  The decode path (fp32 intermediates) and the
training forward/backward (whose saved intermediate keeps the forward's
per-token scale) are checked on the same inputs."""
import numpy as np
import pytest
import torch

from paper_2609_06161_amd import synth
from paper_2609_06161_amd.layer import DeviceLayer, bf16_bits_to_f64, to_device

pytestmark = pytest.mark.gpu

TOL = 5e-3
GRAD_TOL = 1e-3


def bf16_to_f32(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)


def scaled_x(x_bits, factor):
    """x * factor (factor a scalar or a per-token column), rounded once to
    bf16; a power-of-two factor is exact."""
    v = bf16_to_f32(x_bits).astype(np.float64) * factor
    return synth.f32_to_bf16_bits(v.astype(np.float32))


def token_factors(seed, T, decades=12.0):
    """Per-token factors 10^u, u uniform in [-decades/2, decades/2], with the
    extremes present: consecutive tokens (inside one 64-token group) differ
    by up to 10^12."""
    rng = np.random.default_rng(seed)
    u = rng.uniform(-decades / 2, decades / 2, size=T)
    u[0], u[-1] = -decades / 2, decades / 2
    if T > 2:
        u[1] = decades / 2
    return (10.0 ** u)[:, None]


def max_row_rel_l2(y, ref):
    worst = 0.0
    for a, e in zip(np.asarray(y, np.float64), np.asarray(ref, np.float64)):
        ne = np.linalg.norm(e)
        if ne == 0.0:
            assert np.all(a == 0.0)
            continue
        worst = max(worst, np.linalg.norm(a - e) / ne)
    return worst


def elementwise_ok(y, ref, rel=2 ** -6, abs_rms=6e-3):
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.sqrt(np.mean(ref ** 2, axis=1, keepdims=True))
    bad = np.abs(y - ref) > rel * np.abs(ref) + abs_rms * scale
    return not bad.any(), np.argwhere(bad)[:5]


def oracle_y(oracle, lin, x):
    return oracle.forward(lin.m, lin.n, lin.r, lin.Bu, lin.Bv, lin.s_out, lin.s_mid, lin.s_in, x)


def run(kind, lin, x):
    print(f"{kind} m={lin.m} n={lin.n} r={lin.r} rows={x.shape[0]}", flush=True)
    L = DeviceLayer.from_host(lin)
    y = (L.gemm if kind == "gemm" else L.gemv)(to_device(x))
    torch.cuda.synchronize()
    return bf16_bits_to_f64(y)


def check(oracle, lin, x, y, idx=None):
    idx = np.arange(x.shape[0]) if idx is None else idx
    ref = oracle_y(oracle, lin, x[idx])
    assert np.all(np.isfinite(ref))
    got = y[idx]
    assert np.all(np.isfinite(got)), "inf or NaN in the output"
    err = max_row_rel_l2(got, ref)
    ok, where = elementwise_ok(got, ref)
    print(f"  max token rel-L2 {err:.3e}", flush=True)
    assert err <= TOL and ok, (err, where)


FACTORS = [2.0 ** 17, 2.0 ** 20, 2.0 ** -30]


@pytest.mark.parametrize("factor", FACTORS, ids=["x2^17", "x2^20", "x2^-30"])
@pytest.mark.parametrize("m,n,r,T", [(4096, 4096, 2016, 17), (4096, 4096, 2016, 64),
                                     (1056, 2080, 4064, 3)])
def test_gemm_scaled_activations(oracle, factor, m, n, r, T):
    """T = 17 and 3 split K (their reduction applies the token shifts); T = 64
    runs the plain tile epilogue."""
    lin = synth.make_linear(4100 + T, m, n, r, T)
    x = scaled_x(lin.x, factor)
    check(oracle, lin, x, run("gemm", lin, x))


@pytest.mark.parametrize("factor", FACTORS, ids=["x2^17", "x2^20", "x2^-30"])
def test_gemm_scaled_activations_mixed_grid_2048_tokens(oracle, factor):
    """28672x8192 at 2048 tokens: the mixed grid (whole tiles plus K-split
    tiles added by their own reduction); a seeded sample of 12 tokens, the
    first and last included, against the oracle."""
    m, n, r = synth.SHAPES["mlp_up28672x8192"]
    T = 2048
    lin = synth.make_linear(4200, m, n, r, T)
    x = scaled_x(lin.x, factor)
    y = run("gemm", lin, x)
    idx = np.sort(np.random.default_rng(3).choice(np.arange(1, T - 1), 10, replace=False))
    idx = np.concatenate([[0], idx, [T - 1]])
    check(oracle, lin, x, y, idx)


@pytest.mark.parametrize("m,n,r,T", [(4096, 4096, 2016, 17), (4096, 4096, 2016, 128),
                                     (1024, 1024, 480, 300)])
def test_gemm_token_scales_spanning_1e12(oracle, m, n, r, T):
    """Tokens whose magnitudes differ by up to 10^12 inside one 64-token
    group: each token keeps its own digits."""
    lin = synth.make_linear(4300 + T, m, n, r, T)
    x = scaled_x(lin.x, token_factors(4301 + T, T))
    check(oracle, lin, x, run("gemm", lin, x))


def test_gemm_token_scales_spanning_1e12_mixed_grid(oracle):
    m, n, r = synth.SHAPES["mlp_up28672x8192"]
    T = 2048
    lin = synth.make_linear(4400, m, n, r, T)
    x = scaled_x(lin.x, token_factors(4401, T))
    y = run("gemm", lin, x)
    idx = np.sort(np.random.default_rng(4).choice(np.arange(2, T - 1), 10, replace=False))
    idx = np.concatenate([[0, 1], idx, [T - 1]])
    check(oracle, lin, x, y, idx)


def test_gemm_zero_and_extreme_tokens(oracle):
    """An all-zero token gives exact zeros; a token with a single nonzero
    entry and tokens near the ends of bf16's normal range stay exact to the
    bar."""
    m, n, r, T = 1056, 2080, 480, 6
    lin = synth.make_linear(4500, m, n, r, T)
    xf = bf16_to_f32(lin.x).astype(np.float64)
    xf[0] = 0.0
    xf[1] = 0.0
    xf[1, 77] = 3.0
    xf[2] *= 2.0 ** 100
    xf[3] *= 2.0 ** -100
    xf[4] *= 2.0 ** 60
    x = synth.f32_to_bf16_bits(xf.astype(np.float32))
    y = run("gemm", lin, x)
    assert np.all(y[0] == 0.0)
    check(oracle, lin, x, y, np.arange(1, T))


@pytest.mark.parametrize("factor", FACTORS + [2.0 ** 60, 2.0 ** -90],
                         ids=["x2^17", "x2^20", "x2^-30", "x2^60", "x2^-90"])
@pytest.mark.parametrize("m,n,r,b", [(4096, 4096, 2016, 1), (4096, 4096, 2016, 8),
                                     (14336, 4096, 3136, 16)])
def test_gemv_scaled_activations(oracle, factor, m, n, r, b):
    """The decode path keeps s_in .* x and the intermediate in fp32."""
    lin = synth.make_linear(4600 + b, m, n, r, b)
    x = scaled_x(lin.x, factor)
    check(oracle, lin, x, run("gemv", lin, x))


@pytest.mark.parametrize("factor", [2.0 ** 20, 2.0 ** -30, "tokens"],
                         ids=["x2^20", "x2^-30", "token_scales_1e12"])
@pytest.mark.parametrize("m,n,r,T", [(1056, 2080, 160, 130), (4096, 4096, 2016, 65)])
def test_training_scaled_activations(oracle, factor, m, n, r, T):
    """The training forward saves the first product at the token's scale;
    the backward's s_mid gradient undoes it.  y is bit-identical to the
    inference forward's, dx and the three scale gradients match the oracle."""
    lin = synth.make_linear(4700 + T, m, n, r, T)
    f = token_factors(4701, T) if factor == "tokens" else factor
    lin.x = scaled_x(lin.x, f)
    dy = synth.make_output_grad(4702 + T, T, m)
    print(f"train m={m} n={n} r={r} T={T}", flush=True)
    L = DeviceLayer.from_host(lin)
    x = to_device(lin.x)
    y, saved = L.forward_train(x)
    y_inf = L.gemm(x)
    dx, grads = L.backward(x, to_device(dy), saved)
    torch.cuda.synchronize()
    assert torch.equal(y, y_inf)
    check(oracle, lin, lin.x, bf16_bits_to_f64(y))
    rdx, rout, rmid, rin = oracle.backward(m, n, r, lin.Bu, lin.Bv, lin.s_out, lin.s_mid,
                                           lin.s_in, lin.x, dy)
    rel = lambda a, e: float(np.linalg.norm(a - e) / np.linalg.norm(e))
    g = [t.detach().cpu().numpy().astype(np.float64) for t in grads]
    e = max_row_rel_l2(bf16_bits_to_f64(dx), rdx)
    eo, em, ei = rel(g[0], rout), rel(g[1], rmid), rel(g[2], rin)
    print(f"  dx {e:.2e} ds_out {eo:.2e} ds_mid {em:.2e} ds_in {ei:.2e}", flush=True)
    assert e <= TOL and eo <= GRAD_TOL and em <= GRAD_TOL and ei <= GRAD_TOL


@pytest.mark.parametrize("n,T", [(33024, 5), (32768, 3)])
def test_gemm_wide_rows_scaled(oracle, n, T):
    """Rows wider than the preparation keeps in registers (more than 2048
    units of 16 columns, read three times) and the widest that it keeps
    (2048 units), with token scales spanning 10^12."""
    m, r = 96, 64
    lin = synth.make_linear(4800 + n, m, n, r, T)
    x = scaled_x(lin.x, token_factors(4801, T))
    check(oracle, lin, x, run("gemm", lin, x))


@pytest.mark.parametrize("n,T", [(4096, 3077), (8192, 4101), (16384, 1800), (24576, 900)],
                         ids=["units256", "units512", "units1024", "units1536"])
def test_gemm_prep_several_tokens_per_worker(oracle, n, T):
    """The persistent preparation (one row in registers, the next one
    loading) at token counts where each worker takes three to five tokens
    and the last round is ragged (on 256 compute units: 1024, 1024, 512 and
    256 workers for these widths), with token scales spanning 10^12 so that
    a token prepared with another token's range-guard shift fails.  Every
    token against the oracle."""
    m, r = 96, 64
    lin = synth.make_linear(4900 + n, m, n, r, T)
    x = scaled_x(lin.x, token_factors(4901 + n, T))
    check(oracle, lin, x, run("gemm", lin, x))


def biased_words(seed, rows, cols, p):
    """Packed sign words whose bits are set with probability p (bit j of word
    w is column 32 w + j)."""
    bits = np.random.default_rng(seed).random((rows, cols)) < p
    return np.packbits(bits, axis=1, bitorder="little").view(np.uint32).reshape(rows, cols // 32)


@pytest.mark.parametrize("offset", [40.0, 1000.0], ids=["mean40sd", "mean1000sd"])
@pytest.mark.parametrize("p", [0.5, 0.1, 0.9], ids=["fair", "bits0.1", "bits0.9"])
@pytest.mark.parametrize("m,n,r,T", [(4096, 4096, 2016, 64), (4096, 4096, 2016, 17)])
def test_gemm_offset_activations_and_biased_signs(oracle, offset, p, m, n, r, T):
    """Activations with a common offset far above their spread (x = offset +
    N(0,1), every entry positive) and sign matrices with biased bits.  The
    forward forms each signed sum as R - 2 acc from the operand's row sum R
    and the sum over set bits acc; with fair signs both are about sqrt(K)
    times the result, the case where fp32 cancellation would show."""
    lin = synth.make_linear(4800 + T, m, n, r, T)
    lin.Bv = biased_words(4801, r, n, p)
    lin.Bu = biased_words(4802, m, r, p)
    z = np.random.default_rng(4803).standard_normal((T, n))
    x = synth.f32_to_bf16_bits((offset + z).astype(np.float32))
    check(oracle, lin, x, run("gemm", lin, x))


@pytest.mark.parametrize("offset", [40.0, 1000.0], ids=["mean40sd", "mean1000sd"])
def test_gemm_offset_activations_8192(oracle, offset):
    """The same offset activations through 8192x8192 at 2048 tokens (K =
    8192 in the first product, 64-token tiles), fair signs, on a seeded
    sample of tokens."""
    m, n, r = synth.SHAPES["sq8192"]
    T = 2048
    lin = synth.make_linear(4900, m, n, r, T)
    z = np.random.default_rng(4901).standard_normal((T, n))
    x = synth.f32_to_bf16_bits((offset + z).astype(np.float32))
    y = run("gemm", lin, x)
    idx = np.sort(np.random.default_rng(4902).choice(np.arange(1, T - 1), 6, replace=False))
    idx = np.concatenate([[0], idx, [T - 1]])
    check(oracle, lin, x, y, idx)
