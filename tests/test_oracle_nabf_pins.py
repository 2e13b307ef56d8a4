"""Pins for the oracle's NABF building blocks (Sec. 4.1, Algorithm nabf,
App. A.1.4, App. A.2.2-A.2.5): each is tied to a hand computation, a closed
form, an independent library routine or an exact invariant."""
import numpy as np
import pytest
import scipy.linalg

from oracle import nabf


def _signs_to_words(S):
    bits = (np.asarray(S) < 0).astype(np.uint8)
    rows, cols = bits.shape
    by = np.packbits(bits, axis=1, bitorder="little")
    return np.ascontiguousarray(by).view("<u4").reshape(rows, cols // 32).astype(np.uint32)


def _orthogonal(rng, r):
    Q, R = np.linalg.qr(rng.standard_normal((r, r)))
    return Q * np.sign(np.diag(R))


# --------------------------------------------------------------------------
# surrogate reparameterization
# --------------------------------------------------------------------------

def test_surrogate_hand_example():
    W = np.array([[1.0, -2.0], [3.0, 0.5], [-1.0, 4.0]])
    X = np.array([[1.0, 2.0], [3.0, -4.0]])            # tokens x n
    G = np.array([[2.0, 0.0, 1.0], [0.0, 2.0, -3.0]])   # tokens x m
    Wp, i, o = nabf.surrogate(W, X, G)
    np.testing.assert_allclose(i, [np.sqrt(5.0), np.sqrt(10.0)], rtol=1e-15)
    np.testing.assert_allclose(o, [np.sqrt(2.0), np.sqrt(2.0), np.sqrt(5.0)], rtol=1e-15)
    expect = np.array([[np.sqrt(2) * 1 * np.sqrt(5), np.sqrt(2) * -2 * np.sqrt(10)],
                       [np.sqrt(2) * 3 * np.sqrt(5), np.sqrt(2) * 0.5 * np.sqrt(10)],
                       [np.sqrt(5) * -1 * np.sqrt(5), np.sqrt(5) * 4 * np.sqrt(10)]])
    np.testing.assert_allclose(Wp, expect, rtol=1e-14)


# --------------------------------------------------------------------------
# SVID
# --------------------------------------------------------------------------

def test_svid_signs_match_numpy():
    Z = np.random.default_rng(1).standard_normal((40, 96)).astype(np.float32)
    Z[0, 3] = -0.0
    bits, _, _ = nabf.svid(Z, 5)
    assert np.array_equal(bits, _signs_to_words(np.where(np.signbit(Z), -1, 1)))


def test_svid_converges_to_top_singular_pair():
    Z = np.random.default_rng(2).standard_normal((64, 160)).astype(np.float32)
    _, a, v = nabf.svid(Z, 300)
    U, s, Vt = np.linalg.svd(np.abs(Z.astype(np.float64)))
    u1, v1 = U[:, 0] * np.sign(U[0, 0]), Vt[0] * np.sign(Vt[0, 0])
    np.testing.assert_allclose(v, v1, rtol=0, atol=1e-10)
    np.testing.assert_allclose(a, s[0] * u1, rtol=1e-10)


def test_svid_exact_on_rank_one_magnitudes():
    rng = np.random.default_rng(3)
    p = rng.integers(1, 9, 32) / 4.0      # products exact in float32
    q = rng.integers(1, 9, 64) / 4.0
    S = np.where(rng.random((32, 64)) < 0.5, -1.0, 1.0)
    Z = (S * np.outer(p, q)).astype(np.float32)
    _, a, v = nabf.svid(Z, 3)
    np.testing.assert_allclose(np.outer(a, v), np.abs(Z.astype(np.float64)), rtol=1e-12)


def test_svid_zero_iterations_uses_the_start_vector():
    Z = np.random.default_rng(4).standard_normal((8, 32)).astype(np.float32)
    _, a, v = nabf.svid(Z, 0)
    np.testing.assert_allclose(v, np.full(32, 32 ** -0.5), rtol=1e-15)
    np.testing.assert_allclose(a, np.abs(Z.astype(np.float64)).sum(axis=1) / np.sqrt(32), rtol=1e-14)


# --------------------------------------------------------------------------
# null-space projector
# --------------------------------------------------------------------------

def test_projector_on_a_constructed_spectrum():
    rng = np.random.default_rng(5)
    lam = np.array([50.0, 20.0, 10.0, 5.0, 0.3, 0.2, 0.1, 0.0])
    Q = _orthogonal(rng, 8)
    C = Q @ np.diag(lam) @ Q.T
    P, k = nabf.nullspace_projector(C, eta=0.01)
    # tail sums 0, 0.1, 0.3, 0.6 (<= 0.856), then 5.6 (> 0.856): four trailing
    # eigenvectors, cut after the fourth largest eigenvalue
    assert k == 4
    tail = Q[:, 4:]
    np.testing.assert_allclose(P, tail @ tail.T, atol=1e-12)


def test_projector_properties_on_a_factor():
    rng = np.random.default_rng(6)
    r, n = 96, 160
    B = rng.standard_normal((r, n)) * rng.uniform(0.1, 3.0, (r, 1))
    C = B @ B.T
    P, k = nabf.nullspace_projector(C, eta=0.01)
    np.testing.assert_allclose(P @ P, P, atol=1e-10)
    np.testing.assert_allclose(P, P.T, atol=1e-12)
    assert abs(np.trace(P) - (r - k)) < 1e-9
    lam = scipy.linalg.eigvalsh(C)[::-1]
    total = lam.sum()
    # ||P B||_F^2 equals the residual energy, within the cutoff; one fewer
    # eigenvector kept would exceed it
    resid = np.linalg.norm(P @ B) ** 2
    np.testing.assert_allclose(resid, lam[k:].sum(), rtol=1e-8, atol=1e-9 * total)
    assert resid <= 0.01 * total
    assert lam[k - 1:].sum() > 0.01 * total


def test_projector_is_scale_invariant():
    rng = np.random.default_rng(7)
    B = rng.standard_normal((64, 96))
    P1, k1 = nabf.nullspace_projector(B @ B.T)
    P2, k2 = nabf.nullspace_projector(1e4 * (B @ B.T))
    assert k1 == k2
    np.testing.assert_allclose(P1, P2, atol=1e-9)


# --------------------------------------------------------------------------
# ADMM proxies
# --------------------------------------------------------------------------

def _admm_case(seed, m=48, n=80, r=32):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((m, n)), rng.standard_normal((m, r)), rng.standard_normal((r, n)),
            0.1 * rng.standard_normal((m, r)), 0.1 * rng.standard_normal((r, n)))


def test_admm_left_satisfies_its_normal_equations():
    Wp, A, B, UA, _ = _admm_case(8)
    rho = 0.7
    X = nabf.admm_left(Wp, A, B, UA, rho)
    lhs = X @ (B @ B.T + rho * np.eye(B.shape[0]))
    np.testing.assert_allclose(lhs, Wp @ B.T + rho * (A - UA), rtol=1e-10, atol=1e-10)


def test_admm_left_without_penalty_is_least_squares():
    Wp, A, B, UA, _ = _admm_case(9)
    X = nabf.admm_left(Wp, A, B, UA, 1e-12)
    ref = np.linalg.lstsq(B.T, Wp.T, rcond=None)[0].T     # argmin ||X B - W'||
    np.testing.assert_allclose(X, ref, rtol=1e-7, atol=1e-8)


def test_admm_right_is_the_transposed_left_proxy():
    Wp, A, B, _, UB = _admm_case(10)
    rho = 0.3
    X = nabf.admm_right(Wp, A, B, UB, rho)
    ref = nabf.admm_left(Wp.T, B.T, A.T, UB.T, rho).T
    np.testing.assert_allclose(X, ref, rtol=1e-11, atol=1e-11)
    G = A.T @ A + rho * np.eye(A.shape[1])
    np.testing.assert_allclose(G @ X, A.T @ Wp + rho * (B - UB), rtol=1e-10, atol=1e-10)


# --------------------------------------------------------------------------
# compensation and scale fits
# --------------------------------------------------------------------------

def test_gamma_is_columnwise_least_squares():
    rng = np.random.default_rng(11)
    m, r = 50, 24
    Ahat = rng.standard_normal((m, r))
    Aq = rng.standard_normal((m, r))
    Q = _orthogonal(rng, r)[:, :7]
    P = Q @ Q.T
    g = nabf.compensate_left(Ahat, Aq, P)
    target = Ahat - (Ahat - Aq) @ P
    for k in range(r):
        ref = np.linalg.lstsq(Aq[:, k:k + 1], target[:, k], rcond=None)[0][0]
        assert abs(g[k] - ref) <= 1e-10 * max(1.0, abs(ref))


def test_gamma_limits():
    rng = np.random.default_rng(12)
    Ahat = rng.standard_normal((30, 16))
    Aq = rng.standard_normal((30, 16))
    np.testing.assert_allclose(nabf.compensate_left(Ahat, Aq, np.eye(16)), 1.0, atol=1e-10)
    g0 = nabf.compensate_left(Ahat, Aq, np.zeros((16, 16)))
    np.testing.assert_allclose(g0, (Aq * Ahat).sum(0) / (Aq * Aq).sum(0), rtol=1e-10)


def test_eta_is_rowwise_least_squares():
    rng = np.random.default_rng(13)
    r, n = 20, 44
    Bhat = rng.standard_normal((r, n))
    Bq = rng.standard_normal((r, n))
    Q = _orthogonal(rng, r)[:, :5]
    P = Q @ Q.T
    e = nabf.compensate_right(Bhat, Bq, P)
    target = Bhat - P @ (Bhat - Bq)
    for k in range(r):
        ref = np.linalg.lstsq(Bq[k][:, None], target[k], rcond=None)[0][0]
        assert abs(e[k] - ref) <= 1e-10 * max(1.0, abs(ref))
    np.testing.assert_allclose(nabf.compensate_right(Bhat, Bq, np.eye(r)), 1.0, atol=1e-10)


# --------------------------------------------------------------------------
# one NABF iteration
# --------------------------------------------------------------------------

def _exact_state(seed, m=64, n=96, r=32):
    """A layer W' = A* B* that is exactly binary-scaled with rank-1 magnitudes."""
    import oracle
    rng = np.random.default_rng(seed)
    a, m1 = rng.uniform(0.5, 2, m), rng.uniform(0.5, 2, r)
    m2, b = rng.uniform(0.5, 2, r), rng.uniform(0.5, 2, n)
    SA = np.where(rng.random((m, r)) < 0.5, -1.0, 1.0)
    SB = np.where(rng.random((r, n)) < 0.5, -1.0, 1.0)
    A = a[:, None] * SA * m1[None, :]
    B = m2[:, None] * SB * b[None, :]
    S = dict(A_bits=oracle.pack(SA.astype(np.float32)), B_bits=oracle.pack(SB.astype(np.float32)),
             a=a, m1=m1, m2=m2, b=b, A=A, B=B, UA=np.zeros((m, r)), UB=np.zeros((r, n)))
    return A @ B, S


def test_iteration_keeps_an_exact_factorization_fixed():
    Wp, S = _exact_state(14)
    T = nabf.nabf_iteration(Wp, S, rho=0.5, eta=0.01, iters=20)
    assert np.array_equal(T["A_bits"], S["A_bits"]) and np.array_equal(T["B_bits"], S["B_bits"])
    # SVID sees its input in float32 (the precision both sides use), so the
    # fixed point holds to float32 rounding
    np.testing.assert_allclose(T["A"], S["A"], rtol=1e-6)
    np.testing.assert_allclose(T["B"], S["B"], rtol=1e-6)
    np.testing.assert_allclose(T["A"] @ T["B"], Wp, rtol=1e-6, atol=1e-6)
    assert np.abs(T["UA"]).max() < 1e-6 and np.abs(T["UB"]).max() < 1e-6
    np.testing.assert_allclose(T["gamma"], 1.0, atol=1e-6)
    np.testing.assert_allclose(T["eta"], 1.0, atol=1e-6)


def test_iteration_output_structure():
    """The carried factors stay binary-scaled: A = a . sign(A_hat + U_A) . m1^T
    with the scale fit folded into m1 (same for B and m2), and the duals
    move by A_hat - A."""
    Wp0, S = _exact_state(15)
    rng = np.random.default_rng(16)
    Wp = Wp0 + 0.3 * rng.standard_normal(Wp0.shape)
    T = nabf.nabf_iteration(Wp, S, rho=0.5, eta=0.01, iters=30)
    signs = np.where(np.signbit((T["Ahat"] + S["UA"]).astype(np.float32)), -1.0, 1.0)
    np.testing.assert_allclose(T["A"], T["a"][:, None] * signs * T["m1"][None, :], rtol=1e-12)
    signs = np.where(np.signbit((T["Bhat"] + S["UB"]).astype(np.float32)), -1.0, 1.0)
    np.testing.assert_allclose(T["B"], T["m2"][:, None] * signs * T["b"][None, :], rtol=1e-12)
    # the left proxy uses the incoming B; the right proxy the updated A
    rho, r = 0.5, S["B"].shape[0]
    np.testing.assert_allclose(T["Ahat"] @ (S["B"] @ S["B"].T + rho * np.eye(r)),
                               Wp @ S["B"].T + rho * (S["A"] - S["UA"]), rtol=1e-9, atol=1e-9)
    np.testing.assert_allclose((T["A"].T @ T["A"] + rho * np.eye(r)) @ T["Bhat"],
                               T["A"].T @ Wp + rho * (S["B"] - S["UB"]), rtol=1e-9, atol=1e-9)
    np.testing.assert_allclose(T["UA"], S["UA"] + T["Ahat"] - T["A"], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(T["UB"], S["UB"] + T["Bhat"] - T["B"], rtol=1e-12, atol=1e-12)
