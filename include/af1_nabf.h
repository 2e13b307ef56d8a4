/*
 * af1_nabf.h -- C ABI of the NABF building blocks on AMD MI355X (gfx950),
 * built as libaf1_nabf.so.
 *
 * NABF (paper "All for 1-Bit", Sec. 4.1 "Null-space-Aware Binary
 * Factorization", Algorithm nabf in App. A.1, App. A.1.4, App. A.2.2-A.2.5)
 * is the offline calibration that produces the sign factors and scales of
 * one factorised linear from its weight W, calibration inputs and output
 * gradients.  For the surrogate weight W' (m x n) it alternates over the
 * scaled factors
 *
 *     A = a . A_pm1 . m1^T   (m x r)       B = m2 . B_pm1 . b^T   (r x n)
 *
 * an ADMM proxy, an SVID projection, a null-space-compensated scale fit and
 * a scaled dual update.  The deployable layer of af1.h is then Bu = A_pm1,
 * Bv = B_pm1, s_out = a / o, s_mid = m1 . m2, s_in = b / i.
 *
 * Conventions (beyond those of af1.h)
 * -----------------------------------
 * Dense matrices are fp32, row-major, contiguous, device memory, 16-byte
 *   aligned; sign matrices use the packed format of af1.h.
 * Dimensions m, n, r are multiples of 32 in [32, AF1_NABF_MAX_DIM].
 * Matrix products run on rocBLAS (fp32) and the Cholesky and symmetric
 *   eigen factorisations on rocSOLVER (the eigenproblem in fp64).  The
 *   library keeps one rocBLAS handle per device, created on first use and
 *   kept until the process ends; rocBLAS allocates its own device scratch
 *   through that handle.  Calls on one device are serialised on the host
 *   while they enqueue work.  Unlike af1.h, these entry points are an
 *   offline path: they may synchronise internally where rocSOLVER does.
 * Workspace: every call takes a device workspace; af1_nabf_workspace_bytes
 *   (m, n, r, T) bytes cover every entry point for a layer of those
 *   dimensions (af1_svid of its m x r or r x n factor included).
 * Errors: as in af1.h (argument errors before any work, AF1_ERR_HIP when
 *   HIP, rocBLAS or rocSOLVER reject a call).
 */
#ifndef AF1_NABF_H
#define AF1_NABF_H

#include "af1.h"

#ifdef __cplusplus
extern "C" {
#endif

#define AF1_NABF_MAX_DIM 65536
#define AF1_NABF_MAX_TOKENS (1 << 20)
#define AF1_NABF_MAX_POWER_ITERS 1000

/* The factor state one NABF iteration reads and updates in place (all
 * device arrays).  A and B must equal their binary-scaled forms
 * a . A_pm1 . m1^T and m2 . B_pm1 . b^T. */
typedef struct af1_nabf_state {
    int64_t m, n, r;
    float *A;          /* m x r scaled left factor */
    float *B;          /* r x n scaled right factor */
    float *UA;         /* m x r scaled dual of the left update */
    float *UB;         /* r x n scaled dual of the right update */
    uint32_t *A_bits;  /* m x r signs, m * (r/32) words (the deployable Bu) */
    uint32_t *B_bits;  /* r x n signs, r * (n/32) words (the deployable Bv) */
    float *a;          /* m */
    float *m1;         /* r */
    float *m2;         /* r */
    float *b;          /* n */
} af1_nabf_state;

/* Workspace bytes for layers up to m x n, rank r, and T calibration tokens
 * (T may be 0 when af1_nabf_surrogate is not called).  0 for invalid
 * arguments. */
AF1_API size_t af1_nabf_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t T);

/*
 * af1_nabf_surrogate -- Hessian-aware surrogate (Sec. 4.1, first NABF
 * paragraph): i_j = sqrt(mean_t X[t][j]^2), o_u = sqrt(mean_t G[t][u]^2),
 * Wp = o . W . i^T.
 *   W : m x n fp32.   X : [T, n] bfloat16 calibration inputs.
 *   G : [T, m] bfloat16 output gradients.
 *   Wp (m x n), i_vec (n), o_vec (m): fp32, written.
 * Means over the T tokens in fp32, summed per 64-token tile and then over
 * tiles in a fixed order.  Wp must not be W (AF1_ERR_ALIAS).
 */
AF1_API af1_status af1_nabf_surrogate(const float *W, int64_t m, int64_t n, const uint16_t *X,
                                      const uint16_t *G, int64_t T, float *Wp, float *i_vec,
                                      float *o_vec, void *ws, size_t ws_bytes, void *stream);

/*
 * af1_svid -- SVID projection (App. A.1.4): the signs of Z packed into bits
 * (rows x cols, the IEEE sign bit of each entry, as af1_pack), and a rank-1
 * fit |Z| ~ left right^T by `iters` power-iteration passes from the
 * all-ones right vector: each pass forms u = |Z| v, w = |Z|^T u and
 * v = w / ||w|| (v is kept when w is zero); then left = |Z| v and right = v
 * (unit norm).  fp32 throughout.  iters in [0, AF1_NABF_MAX_POWER_ITERS].
 *   Z : rows x cols fp32.  bits: rows * (cols/32) words.  left: rows.
 *   right: cols.
 */
AF1_API af1_status af1_svid(const float *Z, int64_t rows, int64_t cols, int32_t iters,
                            uint32_t *bits, float *left, float *right, void *ws, size_t ws_bytes,
                            void *stream);

/*
 * af1_nullspace_projector -- approximate null-space projector of a PSD
 * matrix (App. A.2.2-A.2.4): C = U diag(lambda) U^T with lambda descending,
 * k the first index with sum_{i>k} lambda_i / (sum lambda + 1e-12) <= eta
 * (eq. app_residual_energy_condition; the paper uses eta = 0.01), and
 * P = U_hat U_hat^T over the trailing r - k eigenvectors.
 *   C : r x r fp32 (symmetric; its upper triangle is read).
 *   P : r x r fp32, written.
 *   k_out : device int32, written with k (may be NULL).
 * The eigenproblem and the cutoff are in fp64; P is rounded to fp32.
 */
AF1_API af1_status af1_nullspace_projector(const float *C, int64_t r, float eta, float *P,
                                           int32_t *k_out, void *ws, size_t ws_bytes,
                                           void *stream);

/*
 * af1_admm_proxy -- the closed-form ADMM proxies (App. A.1.4):
 *   side 0: out (m x r) = (Wp B^T + rho (A - U)) (B B^T + rho I)^-1
 *   side 1: out (r x n) = (A^T A + rho I)^-1 (A^T Wp + rho (B - U))
 * with U the scaled dual of that side (m x r or r x n).  rho > 0 keeps the
 * Gram matrix positive definite; the solve is a Cholesky factorisation.
 */
AF1_API af1_status af1_admm_proxy(int32_t side, const float *Wp, int64_t m, int64_t n, int64_t r,
                                  const float *A, const float *B, const float *U, float rho,
                                  float *out, void *ws, size_t ws_bytes, void *stream);

/*
 * af1_scale_fit -- null-space compensation and scale fit (Sec. 4.1, eqs.
 * gamma_lstsq / gamma_solution; App. A.2.5).  Q = left . S . right^T is the
 * binary-scaled SVID projection given by its signs and scales, E = hat - Q.
 *   side 0 (left factor, rows = m, cols = r): target = hat - E P,
 *     fit[k] = sum_i Q[i][k] target[i][k] / (sum_i Q[i][k]^2 + 1e-12)  (gamma)
 *   side 1 (right factor, rows = r, cols = n): target = hat - P E,
 *     fit[k] = sum_j Q[k][j] target[k][j] / (sum_j Q[k][j]^2 + 1e-12)  (eta)
 *   P : r x r fp32 projector.  fit: r fp32, written.
 */
AF1_API af1_status af1_scale_fit(int32_t side, const float *hat, const uint32_t *bits,
                                 const float *left, const float *right, int64_t rows,
                                 int64_t cols, const float *P, float *fit, void *ws,
                                 size_t ws_bytes, void *stream);

/*
 * af1_nabf_iteration -- one pass of the loop of Algorithm nabf on state S:
 *   A_hat = proxy(side 0);  (A_bits, a, m1) = SVID(A_hat + UA);
 *   P_B = projector(B B^T, eta);  m1 .= gamma(A_hat, A_q, P_B);
 *   A = a . A_bits . m1^T;  UA += A_hat - A;
 *   then the same for the right factor with the new A:
 *   B_hat = proxy(side 1);  (B_bits, m2, b) = SVID(B_hat + UB);
 *   P_A = projector(A^T A, eta);  m2 .= eta(B_hat, B_q, P_A);
 *   B = m2 . B_bits . b^T;  UB += B_hat - B.
 * power_iters is SVID's pass count.  Every array of S is updated in place;
 * Wp (m x n) is read.  The arrays must not overlap each other, Wp or ws.
 */
AF1_API af1_status af1_nabf_iteration(const float *Wp, const af1_nabf_state *S, float rho,
                                      float eta, int32_t power_iters, void *ws, size_t ws_bytes,
                                      void *stream);

/*
 * af1_nabf_export -- the deployable scales of the calibrated layer (the
 * surrogate scalings folded back, Sec. 4.1; m = m1 . m2 merged, App. A.1.4):
 *   s_out = fp16(a / o), s_mid = fp16(m1 . m2), s_in = fp16(b / i)
 * (round to nearest even; a zero o or i gives an infinite scale).  i_vec
 * and o_vec may be NULL (no surrogate: W' = W).  The signs S->A_bits and
 * S->B_bits are already the layer's Bu and Bv.
 */
AF1_API af1_status af1_nabf_export(const af1_nabf_state *S, const float *i_vec,
                                   const float *o_vec, uint16_t *s_out, uint16_t *s_mid,
                                   uint16_t *s_in, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* AF1_NABF_H */
