"""NABF building blocks in fp64 numpy -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check of the build entry point and the benchmark's
cpu_baseline leg may import this module; the HIP library never calls it and
it never calls the library.  Library primitives (matrix products, a linear
solve, a symmetric eigendecomposition) serve as steps; everything else is
written out in the paper's order and notation (paper: "All for 1-Bit",
Sec. 4.1 "Null-space-Aware Binary Factorization", Algorithm nabf in App. A.1,
App. A.1.4 "ADMM-SVID Framework in DBF", App. A.2.2-A.2.5).

Dense matrices are row-major float64 arrays.  A sign matrix is stored packed
as in the rest of the project (bit 1 = -1, LSB first); the sign of a value
is its IEEE sign bit, taken from the float32 value both sides see.

Readings where the paper is silent (also listed in the design notes):
  * SVID's rank-1 magnitude fit: `iters` power-iteration passes on |Z| from
    the all-ones right vector, v <- |Z|^T |Z| v / ||.||; the left factor is
    a = |Z| v (least squares given unit v) and the right factor is v.
  * epsilon of the residual-energy fraction and of the scale fits: 1e-12.
  * the scaled dual update uses the factor the iteration carries after the
    scale fold: U <- U + A_hat - A.
  * the surrogate statistics are means over the calibration tokens.
"""
import numpy as np

from . import pack as _pack

EPS = 1e-12


def surrogate(W, X, G):
    """Hessian-aware surrogate (Sec. 4.1, first paragraph of NABF; Algorithm
    nabf, first two steps): i_j = sqrt(E[x_j^2]) over the calibration tokens,
    o_u = sqrt(E[g_u^2]) over the output gradients, W' = o . W . i^T."""
    X = np.asarray(X, np.float64)
    G = np.asarray(G, np.float64)
    i = np.sqrt(np.mean(X * X, axis=0))
    o = np.sqrt(np.mean(G * G, axis=0))
    return o[:, None] * np.asarray(W, np.float64) * i[None, :], i, o


def svid(Z, iters):
    """SVID projection (App. A.1.4): the signs of Z and a rank-1 fit of |Z|.

    Z is a float32 array (its sign bits are the stored signs).  Returns
    (packed signs, a, v) with |Z| ~ a v^T, v of unit norm."""
    Z = np.asarray(Z, np.float32)
    rows, cols = Z.shape
    S = np.abs(Z.astype(np.float64))
    v = np.full(cols, 1.0 / np.sqrt(cols))
    for _ in range(iters):
        u = S @ v
        w = S.T @ u
        nw = np.linalg.norm(w)
        if nw > 0:
            v = w / nw
    a = S @ v
    return _pack(Z), a, v


def binary_scaled(bits, left, right, cols):
    """left . B_pm1 . right^T as a dense float64 matrix."""
    from . import unpack as _unpack
    return np.asarray(left)[:, None] * _unpack(bits, cols).astype(np.float64) * np.asarray(right)[None, :]


def nullspace_projector(C, eta=0.01, eps=EPS):
    """Approximate null-space projector of a PSD matrix (App. A.2.2, A.2.3,
    eqs. app_residual_energy_fraction / app_residual_energy_condition,
    A.2.4): C = U diag(lam) U^T with lam descending; the first k with
    rho_k = sum_{i>k} lam_i / (sum lam + eps) <= eta; U_hat = the trailing
    r - k eigenvectors; P = U_hat U_hat^T.  Returns (P, k)."""
    C = np.asarray(C, np.float64)
    lam, U = np.linalg.eigh(C)          # ascending
    lam = lam[::-1]
    U = U[:, ::-1]
    r = len(lam)
    total = lam.sum()
    k = r
    for kk in range(r + 1):
        if lam[kk:].sum() / (total + eps) <= eta:
            k = kk
            break
    Uh = U[:, k:]
    return Uh @ Uh.T, k


def admm_left(Wp, A, B, U, rho):
    """Left proxy (App. A.1.4): A_hat = (W' B^T + rho (A - U)) (B B^T + rho I)^-1."""
    r = B.shape[0]
    G = B @ B.T + rho * np.eye(r)
    R = Wp @ B.T + rho * (A - U)
    return np.linalg.solve(G, R.T).T     # X G = R with G symmetric


def admm_right(Wp, A, B, U, rho):
    """Right proxy (App. A.1.4): B_hat = (A^T A + rho I)^-1 (A^T W' + rho (B - U))."""
    r = A.shape[1]
    G = A.T @ A + rho * np.eye(r)
    return np.linalg.solve(G, A.T @ Wp + rho * (B - U))


def compensate_left(Ahat, Aq, P, eps=EPS):
    """Null-space compensation and column scale fit (Sec. 4.1, eqs.
    gamma_lstsq and gamma_solution; App. A.2.5): E = A_hat - A_q,
    A_target = A_hat - E P, gamma = diag(A_q^T A_target) / (diag(A_q^T A_q) + eps)."""
    E = Ahat - Aq
    target = Ahat - E @ P
    return np.sum(Aq * target, axis=0) / (np.sum(Aq * Aq, axis=0) + eps)


def compensate_right(Bhat, Bq, P, eps=EPS):
    """The symmetric right-factor form (App. A.2.5): E = B_hat - B_q,
    B_target = B_hat - P E, eta = diag(B_target B_q^T) / (diag(B_q B_q^T) + eps)."""
    E = Bhat - Bq
    target = Bhat - P @ E
    return np.sum(Bq * target, axis=1) / (np.sum(Bq * Bq, axis=1) + eps)


def nabf_iteration(Wp, S, rho, eta, iters, eps=EPS):
    """One pass of the loop of Algorithm nabf: left-factor update, right-factor
    update, dual updates.  S is a dict with the packed signs A_bits (m x r),
    B_bits (r x n), the scales a (m), m1 (r), m2 (r), b (n), the dense
    scaled factors A, B and the scaled duals UA, UB; a new dict is
    returned."""
    Wp = np.asarray(Wp, np.float64)
    m, n = Wp.shape
    r = S["B"].shape[0]
    A, B = S["A"], S["B"]
    # left-factor update
    Ahat = admm_left(Wp, A, B, S["UA"], rho)
    A_bits, a, m1 = svid((Ahat + S["UA"]).astype(np.float32), iters)
    Aq = binary_scaled(A_bits, a, m1, r)
    PB, kB = nullspace_projector(B @ B.T, eta, eps)
    gamma = compensate_left(Ahat, Aq, PB, eps)
    m1 = m1 * gamma
    A = binary_scaled(A_bits, a, m1, r)
    # right-factor update (with the updated left factor)
    Bhat = admm_right(Wp, A, B, S["UB"], rho)
    B_bits, m2, b = svid((Bhat + S["UB"]).astype(np.float32), iters)
    Bq = binary_scaled(B_bits, m2, b, n)
    PA, kA = nullspace_projector(A.T @ A, eta, eps)
    etav = compensate_right(Bhat, Bq, PA, eps)
    m2 = etav * m2
    B = binary_scaled(B_bits, m2, b, n)
    # scaled dual updates
    UA = S["UA"] + Ahat - A
    UB = S["UB"] + Bhat - B
    return dict(A_bits=A_bits, B_bits=B_bits, a=a, m1=m1, m2=m2, b=b, A=A, B=B, UA=UA, UB=UB,
                Ahat=Ahat, Bhat=Bhat, gamma=gamma, eta=etav, kB=kB, kA=kA)
