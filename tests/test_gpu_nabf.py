"""GPU parity of the NABF building blocks (libaf1_nabf.so, include/af1_nabf.h)
against the fp64 oracle (oracle/nabf.py) on the same seeded fp32 inputs.

Bars: SVID signs bit-exact; the null-space cutoff index equal; every other
output within the relative Frobenius error stated per test (fp32 products
and factorisations on the GPU against fp64 on the CPU, same inputs).  In a
whole iteration the signs of entries whose magnitude is within float32
rounding of zero may differ; they are compared only where the oracle's
value is clear of zero."""
import numpy as np
import pytest
import torch

import oracle
from oracle import nabf as onabf
from paper_2609_06161_amd import nabf, synth
from paper_2609_06161_amd.layer import DeviceLayer, bf16_bits_to_f64, to_device

pytestmark = pytest.mark.gpu


def dev(a):
    return to_device(np.ascontiguousarray(a))


def host(t, dtype=np.float64):
    return t.detach().cpu().numpy().astype(dtype)


def rel(a, e):
    a = np.asarray(a, np.float64)
    e = np.asarray(e, np.float64)
    return float(np.linalg.norm(a - e) / np.linalg.norm(e))


def ws_for(m, n, r, T=0):
    return torch.empty(nabf.af1_nabf_workspace_bytes(m, n, r, T), dtype=torch.uint8,
                       device="cuda")


def f32(rng, *shape, scale=1.0):
    return (rng.standard_normal(shape) * scale).astype(np.float32)


# --------------------------------------------------------------------------
# surrogate
# --------------------------------------------------------------------------

def test_surrogate_matches_oracle():
    m, n, T = 256, 320, 200
    rng = np.random.default_rng(1)
    W = f32(rng, m, n)
    X = synth.make_activations(2, T, n)
    G = synth.make_output_grad(3, T, m)
    print(f"surrogate m={m} n={n} T={T}", flush=True)
    d_Wp = torch.empty((m, n), dtype=torch.float32, device="cuda")
    d_i = torch.empty(n, dtype=torch.float32, device="cuda")
    d_o = torch.empty(m, dtype=torch.float32, device="cuda")
    ws = ws_for(m, n, 32, T)
    nabf.af1_nabf_surrogate(dev(W), m, n, dev(X), dev(G), T, d_Wp, d_i, d_o, ws, ws.numel())
    torch.cuda.synchronize()
    Wp, i, o = onabf.surrogate(W, bf16_bits_to_f64(torch.from_numpy(X.view(np.int16))),
                               bf16_bits_to_f64(torch.from_numpy(G.view(np.int16))))
    assert rel(host(d_i), i) < 1e-6 and rel(host(d_o), o) < 1e-6
    assert rel(host(d_Wp), Wp) < 1e-6


# --------------------------------------------------------------------------
# SVID
# --------------------------------------------------------------------------

@pytest.mark.parametrize("rows,cols,iters", [(64, 96, 0), (256, 320, 1), (256, 320, 30),
                                             (2016, 4096, 20), (4096, 2016, 20)])
def test_svid_matches_oracle(rows, cols, iters):
    rng = np.random.default_rng(rows + cols + iters)
    Z = f32(rng, rows, cols) * rng.uniform(0.2, 3.0, (rows, 1)).astype(np.float32)
    Z[0, 0] = -0.0
    print(f"svid {rows}x{cols} iters={iters}", flush=True)
    bits = torch.empty((rows, cols // 32), dtype=torch.int32, device="cuda")
    left = torch.empty(rows, dtype=torch.float32, device="cuda")
    right = torch.empty(cols, dtype=torch.float32, device="cuda")
    ws = ws_for(rows, cols, cols)
    nabf.af1_svid(dev(Z), rows, cols, iters, bits, left, right, ws, ws.numel())
    torch.cuda.synchronize()
    rb, ra, rv = onabf.svid(Z, iters)
    assert np.array_equal(bits.cpu().numpy().view(np.uint32), rb)
    assert rel(host(left), ra) < 1e-5 and rel(host(right), rv) < 1e-5


# --------------------------------------------------------------------------
# null-space projector
# --------------------------------------------------------------------------

@pytest.mark.parametrize("r,n,eta", [(64, 96, 0.01), (256, 512, 0.01), (256, 512, 0.1),
                                     (2016, 4096, 0.01)])
def test_projector_matches_oracle(r, n, eta):
    rng = np.random.default_rng(r + n)
    B = f32(rng, r, n) * rng.uniform(0.1, 2.0, (r, 1)).astype(np.float32)
    C = (B.astype(np.float64) @ B.T.astype(np.float64)).astype(np.float32)
    print(f"projector r={r} eta={eta}", flush=True)
    P = torch.empty((r, r), dtype=torch.float32, device="cuda")
    k = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    ws = ws_for(32, 32, r)
    nabf.af1_nullspace_projector(dev(C), r, eta, P, k, ws, ws.numel())
    torch.cuda.synchronize()
    rP, rk = onabf.nullspace_projector(C.astype(np.float64), eta)
    assert int(k.item()) == rk
    assert rel(host(P), rP) < 1e-5


# --------------------------------------------------------------------------
# ADMM proxies
# --------------------------------------------------------------------------

@pytest.mark.parametrize("side", [0, 1])
@pytest.mark.parametrize("m,n,r", [(128, 192, 64), (1056, 544, 256), (4096, 4096, 2016)])
def test_admm_proxy_matches_oracle(side, m, n, r):
    rng = np.random.default_rng(m + n + r + side)
    Wp, A, B = f32(rng, m, n), f32(rng, m, r, scale=0.1), f32(rng, r, n, scale=0.1)
    U = f32(rng, m, r, scale=0.01) if side == 0 else f32(rng, r, n, scale=0.01)
    rho = 0.5
    print(f"admm side={side} m={m} n={n} r={r}", flush=True)
    out = torch.empty(U.shape, dtype=torch.float32, device="cuda")
    ws = ws_for(m, n, r)
    nabf.af1_admm_proxy(side, dev(Wp), m, n, r, dev(A), dev(B), dev(U), rho, out, ws, ws.numel())
    torch.cuda.synchronize()
    f = onabf.admm_left if side == 0 else onabf.admm_right
    ref = f(Wp.astype(np.float64), A.astype(np.float64), B.astype(np.float64),
            U.astype(np.float64), rho)
    assert rel(host(out), ref) < 1e-4


# --------------------------------------------------------------------------
# compensation and scale fits
# --------------------------------------------------------------------------

@pytest.mark.parametrize("side", [0, 1])
def test_scale_fit_matches_oracle(side):
    rng = np.random.default_rng(40 + side)
    r, other = 96, 320
    rows, cols = (other, r) if side == 0 else (r, other)
    hat = f32(rng, rows, cols)
    bits_h, left_h, right_h = onabf.svid(hat + f32(rng, rows, cols, scale=0.05), 10)
    left_h, right_h = left_h.astype(np.float32), right_h.astype(np.float32)
    Q, _ = np.linalg.qr(rng.standard_normal((r, r)))
    P = (Q[:, 60:] @ Q[:, 60:].T).astype(np.float32)
    print(f"scale fit side={side}", flush=True)
    fit = torch.empty(r, dtype=torch.float32, device="cuda")
    ws = ws_for(other, other, r)
    nabf.af1_scale_fit(side, dev(hat), dev(bits_h), dev(left_h), dev(right_h), rows, cols,
                       dev(P), fit, ws, ws.numel())
    torch.cuda.synchronize()
    Qd = onabf.binary_scaled(bits_h, left_h, right_h, cols)
    f = onabf.compensate_left if side == 0 else onabf.compensate_right
    ref = f(hat.astype(np.float64), Qd, P.astype(np.float64))
    assert rel(host(fit), ref) < 1e-5


# --------------------------------------------------------------------------
# one iteration, and the exported layer
# --------------------------------------------------------------------------

def initial_state(seed, m, n, r, noise=0.3):
    """A surrogate W' = A* B* + noise and a start from SVID of perturbed
    factors (float32 host arrays)."""
    rng = np.random.default_rng(seed)
    As = f32(rng, m, r) * 0.2
    Bs = f32(rng, r, n) * 0.2
    Wp = (As.astype(np.float64) @ Bs + noise * rng.standard_normal((m, n)) * 0.1).astype(np.float32)
    A0 = (As + f32(rng, m, r, scale=0.05))
    B0 = (Bs + f32(rng, r, n, scale=0.05))
    Ab, a, m1 = onabf.svid(A0, 30)
    Bb, m2, b = onabf.svid(B0, 30)
    S = dict(A_bits=Ab, B_bits=Bb, a=a.astype(np.float32), m1=m1.astype(np.float32),
             m2=m2.astype(np.float32), b=b.astype(np.float32),
             UA=np.zeros((m, r), np.float32), UB=np.zeros((r, n), np.float32))
    S["A"] = onabf.binary_scaled(Ab, S["a"], S["m1"], r).astype(np.float32)
    S["B"] = onabf.binary_scaled(Bb, S["m2"], S["b"], n).astype(np.float32)
    return Wp, S


def device_state(S, m, n, r):
    D = {k: dev(v) for k, v in S.items()}
    st = nabf.make_state(m, n, r, D["A"], D["B"], D["UA"], D["UB"], D["A_bits"], D["B_bits"],
                         D["a"], D["m1"], D["m2"], D["b"])
    return D, st


@pytest.mark.parametrize("m,n,r", [(256, 320, 96), (1024, 1024, 480)])
def test_iteration_matches_oracle(m, n, r):
    Wp, S = initial_state(50 + r, m, n, r)
    D, st = device_state(S, m, n, r)
    ws = ws_for(m, n, r)
    rho, eta, iters = 0.5, 0.01, 30
    print(f"nabf iteration m={m} n={n} r={r}", flush=True)
    nabf.af1_nabf_iteration(dev(Wp), st, rho, eta, iters, ws, ws.numel())
    torch.cuda.synchronize()
    S64 = {k: (v.astype(np.float64) if v.dtype == np.float32 else v) for k, v in S.items()}
    T = onabf.nabf_iteration(Wp.astype(np.float64), S64, rho, eta, iters)
    # signs of A_hat + UA (and B_hat + UB): equal wherever the value is clear
    # of zero; the dense factors and duals are compared where the two sides
    # took the same sign decision (a flip near zero is a different but valid
    # rounding of the same projection)
    agree = {}
    for bits, hat, U, cols, key in (("A_bits", "Ahat", "UA", r, "A"), ("B_bits", "Bhat", "UB", n, "B")):
        z = T[hat] + S64[U]
        clear = np.abs(z) > 1e-4 * np.sqrt(np.mean(z * z))
        got = oracle.unpack(D[bits].cpu().numpy().view(np.uint32), cols)
        want = oracle.unpack(T[bits], cols)
        assert np.array_equal(got[clear], want[clear])
        agree[key] = got == want
        print(f"  {key}: {int((~agree[key]).sum())} sign(s) differ near zero", flush=True)
    for key in ("a", "m1", "m2", "b"):
        e = rel(host(D[key]), T[key])
        print(f"  {key}: {e:.2e}", flush=True)
        assert e < 2e-3, key
    for key, mask in (("A", agree["A"]), ("UA", agree["A"]), ("B", agree["B"]), ("UB", agree["B"])):
        e = rel(host(D[key])[mask], T[key][mask])
        print(f"  {key}: {e:.2e}", flush=True)
        assert e < 2e-3, key


def test_iteration_repeats_bit_for_bit():
    m, n, r = 256, 320, 96
    Wp, S = initial_state(61, m, n, r)
    outs = []
    for _ in range(2):
        D, st = device_state(S, m, n, r)
        ws = ws_for(m, n, r)
        d_Wp = dev(Wp)
        for _ in range(3):
            nabf.af1_nabf_iteration(d_Wp, st, 0.5, 0.01, 20, ws, ws.numel())
        torch.cuda.synchronize()
        outs.append({k: v.clone() for k, v in D.items()})
    for k in outs[0]:
        assert torch.equal(outs[0][k], outs[1][k]), k


def test_calibrated_layer_runs_through_the_forward():
    """Surrogate -> NABF iterations -> export -> af1_linear_gemv: the layer's
    output equals x (A B / (o i^T))^T computed from the calibrated dense
    factors, within the fp16 rounding of the exported scales."""
    m, n, r, T = 256, 320, 96, 256
    rng = np.random.default_rng(70)
    W = f32(rng, m, n, scale=0.05)
    X = synth.make_activations(71, T, n)
    G = synth.make_output_grad(72, T, m)
    d_Wp = torch.empty((m, n), dtype=torch.float32, device="cuda")
    d_i = torch.empty(n, dtype=torch.float32, device="cuda")
    d_o = torch.empty(m, dtype=torch.float32, device="cuda")
    ws = ws_for(m, n, r, T)
    nabf.af1_nabf_surrogate(dev(W), m, n, dev(X), dev(G), T, d_Wp, d_i, d_o, ws, ws.numel())
    torch.cuda.synchronize()
    Wp = host(d_Wp, np.float32)
    _, S = initial_state(73, m, n, r)
    U, s, Vt = np.linalg.svd(Wp.astype(np.float64), full_matrices=False)
    A0 = (U[:, :r] * np.sqrt(s[:r])).astype(np.float32)
    B0 = (np.sqrt(s[:r])[:, None] * Vt[:r]).astype(np.float32)
    Ab, a, m1 = onabf.svid(A0, 30)
    Bb, m2, b = onabf.svid(B0, 30)
    S.update(A_bits=Ab, B_bits=Bb, a=a.astype(np.float32), m1=m1.astype(np.float32),
             m2=m2.astype(np.float32), b=b.astype(np.float32))
    S["A"] = onabf.binary_scaled(Ab, S["a"], S["m1"], r).astype(np.float32)
    S["B"] = onabf.binary_scaled(Bb, S["m2"], S["b"], n).astype(np.float32)
    D, st = device_state(S, m, n, r)
    for _ in range(5):
        nabf.af1_nabf_iteration(d_Wp, st, 0.5, 0.01, 20, ws, ws.numel())
    s_out = torch.empty(m, dtype=torch.int16, device="cuda")
    s_mid = torch.empty(r, dtype=torch.int16, device="cuda")
    s_in = torch.empty(n, dtype=torch.int16, device="cuda")
    nabf.af1_nabf_export(st, d_i, d_o, s_out, s_mid, s_in)
    torch.cuda.synchronize()
    # the exported scales are the fp16 roundings of the folded fp32 values
    a_, m1_, m2_, b_ = (host(D[k], np.float32) for k in ("a", "m1", "m2", "b"))
    i_, o_ = host(d_i, np.float32), host(d_o, np.float32)
    assert np.array_equal(s_out.cpu().numpy().view(np.uint16),
                          (a_ / o_).astype(np.float16).view(np.uint16))
    assert np.array_equal(s_mid.cpu().numpy().view(np.uint16),
                          (m1_ * m2_).astype(np.float16).view(np.uint16))
    assert np.array_equal(s_in.cpu().numpy().view(np.uint16),
                          (b_ / i_).astype(np.float16).view(np.uint16))
    # the deployable layer reproduces the calibrated factors
    L = DeviceLayer(m, n, r, D["A_bits"].cpu().numpy().view(np.uint32),
                    D["B_bits"].cpu().numpy().view(np.uint32),
                    s_out.cpu().numpy().view(np.uint16), s_mid.cpu().numpy().view(np.uint16),
                    s_in.cpu().numpy().view(np.uint16))
    xs = X[:4]
    y = bf16_bits_to_f64(L.gemv(dev(xs)))
    What = (host(D["A"]) @ host(D["B"])) / (o_[:, None].astype(np.float64) * i_[None, :])
    ref = bf16_bits_to_f64(torch.from_numpy(xs.view(np.int16))) @ What.T
    assert rel(y, ref) < 5e-3
    # and approximates the original weight (reported, loosely bounded)
    err = rel(What, W)
    print(f"  calibrated relative weight error {err:.3f}", flush=True)
    assert err < 1.0
