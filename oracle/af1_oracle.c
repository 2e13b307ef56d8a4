/*
 * af1_oracle.c -- plain, slow, obviously-correct CPU oracle for the AF1
 * binary-factorized linear layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may include, link,
 * load or call this file.  Its only users are the tests, the smoke check of
 * the build entry point and the cpu_baseline leg of the benchmark.  It shares
 * no code, header, table or helper with the HIP library: every convention it
 * needs (bit order, half-precision widening) is written out again here.
 *
 * What it computes (paper: "All for 1-Bit", App. A.2.1, the Diag form of the
 * double-factor parameterisation, label eq:double_factor_equiv, and the
 * deployable form of Sec. 4.1, label eq:final_reconstruction):
 *
 *     W_hat = Diag(a) * A_pm1 * Diag(m) * B_pm1 * Diag(b)
 *     y     = W_hat x  =  a .* ( A_pm1 * ( m .* ( B_pm1 * ( b .* x ) ) ) )
 *
 * with A_pm1 in {-1,+1}^{d_out x r}, B_pm1 in {-1,+1}^{r x d_in} and three
 * 16-bit scale vectors a (d_out), m = m1 .* m2 (r), b (d_in).  In the code
 * below the library's names are used: Bu = A_pm1, Bv = B_pm1, s_out = a,
 * s_mid = m, s_in = b, and m = d_out, n = d_in.
 *
 * Storage format read here (the paper fixes the bit count but not the layout;
 * this is the reading the whole project uses):
 *   - bit value 1 encodes -1, bit value 0 encodes +1;
 *   - a rows x cols sign matrix is stored row-major as rows * (cols/32)
 *     uint32 words; column j of a row is bit (j mod 32) of word (j div 32);
 *   - cols must be a multiple of 32 (no padding bits exist);
 *   - scales are IEEE binary16 bit patterns, activations bfloat16 patterns.
 *
 * It also computes the gradients of the scale-only reconstruction (Sec. 4.1,
 * labels eq:final_reconstruction and eq:scale_only_kl): with the two sign
 * matrices frozen, the vector-Jacobian product of the layer with respect to
 * s_out, s_mid, s_in and x, and the bit transpose of the packed storage that
 * the transposed products use.
 *
 * Arithmetic: every value is widened exactly to double and every product and
 * sum is taken in double, in the factorised order written above.  The entry
 * -wise path sum of App. A.2.1 (label eq:binary_paths) is provided as an
 * independent brute-force route to the same matrix.
 *
 * Parity pins (tests that tie this file to the paper and to mathematics, not
 * to itself): the paper's 2x2 worked example in App. A.2.1 (stored in
 * tests/golden with its citation), its Kronecker embedding into a packable
 * layer, the Sylvester-Hadamard identity H*H = n*I, one-hot probes against
 * the brute-force matrix, single-bit-flip deltas, sign-gauge invariance,
 * linearity, the storage-bit count of App. A.3 against hand-computed
 * integers, and the half-precision widenings against numpy's own.  The
 * gradients are pinned by one-hot probes of the brute-force path sum (the
 * layer is linear in each scale vector and in x, so a one-hot scale vector
 * gives one gradient entry exactly), by dx against dy times the brute-force
 * matrix, by the four homogeneity identities sum(s .* ds) = sum(dy .* y),
 * and by dx against the forward of the transposed layer.  The transpose is
 * pinned against numpy's unpackbits/packbits and a single-bit probe.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_OK 0
#define OR_ERR_ARG 1
#define OR_ERR_NOMEM 2

/* ---------------------------------------------------------------------- */
/* Half-precision widening, from the format definitions.                   */
/* ---------------------------------------------------------------------- */

/* IEEE 754 binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction
 * bits.  Exponent 0 holds zero and subnormals (value = f * 2^-24); exponent
 * 31 holds infinities and NaNs. */
double oracle_f16_to_f64(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int f = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);
    else if (e == 31)
        v = (f == 0) ? INFINITY : NAN;
    else
        v = ldexp((double)(1024 + f), e - 25);
    return sign ? -v : v;
}

/* bfloat16: the upper 16 bits of an IEEE binary32.  1 sign bit, 8 exponent
 * bits (bias 127), 7 fraction bits. */
double oracle_bf16_to_f64(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 7) & 0xff;
    int f = h & 0x7f;
    double v;
    if (e == 0)
        v = ldexp((double)f, -133);
    else if (e == 255)
        v = (f == 0) ? INFINITY : NAN;
    else
        v = ldexp((double)(128 + f), e - 134);
    return sign ? -v : v;
}

/* ---------------------------------------------------------------------- */
/* Sign packing and unpacking (storage of A_pm1 / B_pm1, App. A.3).         */
/* ---------------------------------------------------------------------- */

/* Source element types accepted by oracle_pack. */
#define OR_SRC_F32 0
#define OR_SRC_BF16 1
#define OR_SRC_F16 2
#define OR_SRC_I8 3

/* The bit of one source element: the IEEE sign bit for floating types (so
 * +0 packs as +1, -0 as -1, a NaN as its own sign bit), v < 0 for int8. */
static int src_sign_bit(const void *src, int dtype, size_t idx)
{
    switch (dtype) {
    case OR_SRC_F32: {
        uint32_t u;
        memcpy(&u, (const char *)src + 4 * idx, 4);
        return (int)(u >> 31);
    }
    case OR_SRC_BF16:
    case OR_SRC_F16: {
        uint16_t u;
        memcpy(&u, (const char *)src + 2 * idx, 2);
        return (int)(u >> 15);
    }
    default: {
        int8_t v = ((const int8_t *)src)[idx];
        return v < 0 ? 1 : 0;
    }
    }
}

int oracle_pack(const void *src, int dtype, int64_t rows, int64_t cols,
                uint32_t *dst)
{
    if (!src || !dst || rows < 0 || cols < 0 || cols % 32 != 0 ||
        dtype < OR_SRC_F32 || dtype > OR_SRC_I8)
        return OR_ERR_ARG;
    int64_t wpr = cols / 32;
    for (int64_t i = 0; i < rows; ++i)
        for (int64_t w = 0; w < wpr; ++w) {
            uint32_t word = 0;
            for (int bit = 0; bit < 32; ++bit) {
                size_t idx = (size_t)(i * cols + w * 32 + bit);
                if (src_sign_bit(src, dtype, idx))
                    word |= (uint32_t)1 << bit;
            }
            dst[i * wpr + w] = word;
        }
    return OR_OK;
}

/* Dense +-1 (int8) from packed words. */
int oracle_unpack(const uint32_t *words, int64_t rows, int64_t cols,
                  int8_t *dst)
{
    if (!words || !dst || rows < 0 || cols < 0 || cols % 32 != 0)
        return OR_ERR_ARG;
    int64_t wpr = cols / 32;
    for (int64_t i = 0; i < rows; ++i)
        for (int64_t j = 0; j < cols; ++j) {
            uint32_t word = words[i * wpr + j / 32];
            int bit = (int)((word >> (j % 32)) & 1u);
            dst[i * cols + j] = bit ? -1 : 1;
        }
    return OR_OK;
}

/* ---------------------------------------------------------------------- */
/* Factorised forward in fp64 (App. A.2.1, Diag form; Sec. 4.1).            */
/* ---------------------------------------------------------------------- */

/*
 * y[beta, i] = s_out[i] * sum_k Bu[i,k] * ( s_mid[k] * sum_j Bv[k,j] *
 *              ( s_in[j] * x[beta, j] ) )
 *
 * Bu: m x r packed, Bv: r x n packed, s_*: binary16 patterns, x: b x n
 * bfloat16 patterns, y: b x m doubles (caller-allocated).
 */
int oracle_forward(int64_t m, int64_t n, int64_t r, const uint32_t *Bu,
                   const uint32_t *Bv, const uint16_t *s_out,
                   const uint16_t *s_mid, const uint16_t *s_in,
                   const uint16_t *x, int64_t b, double *y)
{
    if (m <= 0 || n <= 0 || r <= 0 || b < 0 || m % 32 || n % 32 || r % 32 ||
        !Bu || !Bv || !s_out || !s_mid || !s_in || (b > 0 && (!x || !y)))
        return OR_ERR_ARG;
    if (b == 0)
        return OR_OK;

    int8_t *U = (int8_t *)malloc((size_t)(m * r));
    int8_t *V = (int8_t *)malloc((size_t)(r * n));
    double *u = (double *)malloc(sizeof(double) * (size_t)n);
    double *t = (double *)malloc(sizeof(double) * (size_t)r);
    if (!U || !V || !u || !t) {
        free(U); free(V); free(u); free(t);
        return OR_ERR_NOMEM;
    }
    oracle_unpack(Bu, m, r, U);
    oracle_unpack(Bv, r, n, V);

    for (int64_t beta = 0; beta < b; ++beta) {
        /* step 1: input scaling u = s_in .* x */
        for (int64_t j = 0; j < n; ++j)
            u[j] = oracle_f16_to_f64(s_in[j]) *
                   oracle_bf16_to_f64(x[beta * n + j]);
        /* step 2: first binary product and the middle scale */
#pragma omp parallel for schedule(static)
        for (int64_t k = 0; k < r; ++k) {
            double acc = 0.0;
            const int8_t *row = V + k * n;
            for (int64_t j = 0; j < n; ++j)
                acc += (double)row[j] * u[j];
            t[k] = oracle_f16_to_f64(s_mid[k]) * acc;
        }
        /* step 3: second binary product and the output scale */
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < m; ++i) {
            double acc = 0.0;
            const int8_t *row = U + i * r;
            for (int64_t k = 0; k < r; ++k)
                acc += (double)row[k] * t[k];
            y[beta * m + i] = oracle_f16_to_f64(s_out[i]) * acc;
        }
    }
    free(U); free(V); free(u); free(t);
    return OR_OK;
}

/* ---------------------------------------------------------------------- */
/* Transposed sign storage (for the products with B_u^T and B_v^T).        */
/* ---------------------------------------------------------------------- */

/*
 * dst is the cols x rows sign matrix whose entry (j, i) is the sign of
 * src(i, j), in the same packed format.  Both dimensions must be multiples
 * of 32 so that source and destination rows are whole words.  Written bit
 * by bit from the format definition above.
 */
int oracle_transpose_packed(const uint32_t *src, int64_t rows, int64_t cols,
                            uint32_t *dst)
{
    if (!src || !dst || rows < 0 || cols < 0 || rows % 32 || cols % 32)
        return OR_ERR_ARG;
    int64_t swords = cols / 32, dwords = rows / 32;
    for (int64_t j = 0; j < cols; ++j)
        for (int64_t w = 0; w < dwords; ++w) {
            uint32_t word = 0;
            for (int bit = 0; bit < 32; ++bit) {
                int64_t i = 32 * w + bit;
                uint32_t s = (src[i * swords + j / 32] >> (j % 32)) & 1u;
                word |= s << bit;
            }
            dst[j * dwords + w] = word;
        }
    return OR_OK;
}

/* ---------------------------------------------------------------------- */
/* Scale-only reconstruction: gradients with the sign matrices frozen      */
/* (Sec. 4.1, paragraph on scale-only global reconstruction, labels        */
/* eq:final_reconstruction and eq:scale_only_kl).                          */
/* ---------------------------------------------------------------------- */

/*
 * The paper trains only the three scale vectors (a, m, b here s_out, s_mid,
 * s_in) after freezing A_pm1 and B_pm1, through the unchanged factorised
 * graph.  For an upstream gradient dy of one linear's output this is the
 * chain rule through the four steps of the forward, per token beta:
 *
 *   forward   u = s_in .* x,  v = Bv u,  t = s_mid .* v,  z = Bu t,
 *             y = s_out .* z
 *   backward  dz = s_out .* dy          ds_out += dy .* z
 *             dt = Bu^T dz              ds_mid += dt .* v
 *             dv = s_mid .* dt
 *             du = Bv^T dv              ds_in  += du .* x
 *             dx = s_in .* du
 *
 * The scale gradients are summed over the b tokens.  Bu: m x r packed,
 * Bv: r x n packed (the forward factors themselves; the transposed products
 * read them column-wise), s_*: binary16 patterns, x: b x n and dy: b x m
 * bfloat16 patterns.  Outputs (caller-allocated doubles, overwritten):
 * dx b x n, ds_out m, ds_mid r, ds_in n.
 */
int oracle_backward(int64_t m, int64_t n, int64_t r, const uint32_t *Bu,
                    const uint32_t *Bv, const uint16_t *s_out,
                    const uint16_t *s_mid, const uint16_t *s_in,
                    const uint16_t *x, const uint16_t *dy, int64_t b,
                    double *dx, double *ds_out, double *ds_mid, double *ds_in)
{
    if (m <= 0 || n <= 0 || r <= 0 || b < 0 || m % 32 || n % 32 || r % 32 ||
        !Bu || !Bv || !s_out || !s_mid || !s_in || !ds_out || !ds_mid ||
        !ds_in || (b > 0 && (!x || !dy || !dx)))
        return OR_ERR_ARG;
    for (int64_t i = 0; i < m; ++i) ds_out[i] = 0.0;
    for (int64_t k = 0; k < r; ++k) ds_mid[k] = 0.0;
    for (int64_t j = 0; j < n; ++j) ds_in[j] = 0.0;
    if (b == 0)
        return OR_OK;

    int8_t *U = (int8_t *)malloc((size_t)(m * r));
    int8_t *V = (int8_t *)malloc((size_t)(r * n));
    double *u = (double *)malloc(sizeof(double) * (size_t)n);
    double *v = (double *)malloc(sizeof(double) * (size_t)r);
    double *t = (double *)malloc(sizeof(double) * (size_t)r);
    double *z = (double *)malloc(sizeof(double) * (size_t)m);
    double *dz = (double *)malloc(sizeof(double) * (size_t)m);
    double *dt = (double *)malloc(sizeof(double) * (size_t)r);
    double *dv = (double *)malloc(sizeof(double) * (size_t)r);
    if (!U || !V || !u || !v || !t || !z || !dz || !dt || !dv) {
        free(U); free(V); free(u); free(v); free(t); free(z); free(dz);
        free(dt); free(dv);
        return OR_ERR_NOMEM;
    }
    oracle_unpack(Bu, m, r, U);
    oracle_unpack(Bv, r, n, V);

    for (int64_t beta = 0; beta < b; ++beta) {
        const uint16_t *xb = x + beta * n;
        const uint16_t *dyb = dy + beta * m;
        double *dxb = dx + beta * n;
        /* forward intermediates of this token */
        for (int64_t j = 0; j < n; ++j)
            u[j] = oracle_f16_to_f64(s_in[j]) * oracle_bf16_to_f64(xb[j]);
#pragma omp parallel for schedule(static)
        for (int64_t k = 0; k < r; ++k) {
            double acc = 0.0;
            for (int64_t j = 0; j < n; ++j)
                acc += (double)V[k * n + j] * u[j];
            v[k] = acc;
            t[k] = oracle_f16_to_f64(s_mid[k]) * acc;
        }
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < m; ++i) {
            double acc = 0.0;
            for (int64_t k = 0; k < r; ++k)
                acc += (double)U[i * r + k] * t[k];
            z[i] = acc;
        }
        /* output scale: its gradient and the gradient entering Bu */
        for (int64_t i = 0; i < m; ++i) {
            double g = oracle_bf16_to_f64(dyb[i]);
            ds_out[i] += g * z[i];
            dz[i] = oracle_f16_to_f64(s_out[i]) * g;
        }
        /* dt = Bu^T dz: column k of Bu against dz */
#pragma omp parallel for schedule(static)
        for (int64_t k = 0; k < r; ++k) {
            double acc = 0.0;
            for (int64_t i = 0; i < m; ++i)
                acc += (double)U[i * r + k] * dz[i];
            dt[k] = acc;
        }
        /* middle scale */
        for (int64_t k = 0; k < r; ++k) {
            ds_mid[k] += dt[k] * v[k];
            dv[k] = oracle_f16_to_f64(s_mid[k]) * dt[k];
        }
        /* du = Bv^T dv: column j of Bv against dv; then the input scale */
#pragma omp parallel for schedule(static)
        for (int64_t j = 0; j < n; ++j) {
            double acc = 0.0;
            for (int64_t k = 0; k < r; ++k)
                acc += (double)V[k * n + j] * dv[k];
            dxb[j] = oracle_f16_to_f64(s_in[j]) * acc;
            ds_in[j] += acc * oracle_bf16_to_f64(xb[j]);
        }
    }
    free(U); free(V); free(u); free(v); free(t); free(z); free(dz);
    free(dt); free(dv);
    return OR_OK;
}

/* ---------------------------------------------------------------------- */
/* Brute-force reconstructed matrix, entry by entry (App. A.2.1, the        */
/* path-sum equation, label eq:binary_paths).                               */
/* ---------------------------------------------------------------------- */

/*
 * W[i,j] = a[i] * b[j] * sum_k lam[k] * A[i,k] * B[k,j]
 *
 * A: m x r dense +-1 (int8), B: r x n dense +-1 (int8), a/lam/bv: doubles.
 * Taking dense signs and double scales lets the paper's own 2x2 example be
 * evaluated without the packed format.
 */
int oracle_what_dense(int64_t m, int64_t n, int64_t r, const int8_t *A,
                      const int8_t *B, const double *a, const double *lam,
                      const double *bv, double *W)
{
    if (m <= 0 || n <= 0 || r <= 0 || !A || !B || !a || !lam || !bv || !W)
        return OR_ERR_ARG;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i)
        for (int64_t j = 0; j < n; ++j) {
            double paths = 0.0;
            for (int64_t k = 0; k < r; ++k)
                paths += lam[k] * (double)A[i * r + k] * (double)B[k * n + j];
            W[i * n + j] = a[i] * bv[j] * paths;
        }
    return OR_OK;
}

/* The same brute force, reading the packed storage format and the 16-bit
 * scale patterns. */
int oracle_what_packed(int64_t m, int64_t n, int64_t r, const uint32_t *Bu,
                       const uint32_t *Bv, const uint16_t *s_out,
                       const uint16_t *s_mid, const uint16_t *s_in, double *W)
{
    if (m <= 0 || n <= 0 || r <= 0 || m % 32 || n % 32 || r % 32 || !Bu ||
        !Bv || !s_out || !s_mid || !s_in || !W)
        return OR_ERR_ARG;
    int8_t *A = (int8_t *)malloc((size_t)(m * r));
    int8_t *B = (int8_t *)malloc((size_t)(r * n));
    double *a = (double *)malloc(sizeof(double) * (size_t)m);
    double *lam = (double *)malloc(sizeof(double) * (size_t)r);
    double *bv = (double *)malloc(sizeof(double) * (size_t)n);
    int rc = OR_ERR_NOMEM;
    if (A && B && a && lam && bv) {
        oracle_unpack(Bu, m, r, A);
        oracle_unpack(Bv, r, n, B);
        for (int64_t i = 0; i < m; ++i) a[i] = oracle_f16_to_f64(s_out[i]);
        for (int64_t k = 0; k < r; ++k) lam[k] = oracle_f16_to_f64(s_mid[k]);
        for (int64_t j = 0; j < n; ++j) bv[j] = oracle_f16_to_f64(s_in[j]);
        rc = oracle_what_dense(m, n, r, A, B, a, lam, bv, W);
    }
    free(A); free(B); free(a); free(lam); free(bv);
    return rc;
}

/* ---------------------------------------------------------------------- */
/* Storage accounting (App. A.3, labels eq:app_af1_memory, eq:app_af1_bpw)  */
/* ---------------------------------------------------------------------- */

/* Deployable bits of one factorised linear: r*(d_out + d_in) sign bits plus
 * three 16-bit scale vectors of lengths d_out, r and d_in. */
int64_t oracle_storage_bits(int64_t m, int64_t n, int64_t r)
{
    return r * (m + n) + 16 * (m + n + r);
}

/* Model-level effective bits per weight: total deployable bits over total
 * dense weights of all linears. */
double oracle_bpw(int64_t count, const int64_t *m, const int64_t *n,
                  const int64_t *r)
{
    int64_t bits = 0, weights = 0;
    for (int64_t i = 0; i < count; ++i) {
        bits += oracle_storage_bits(m[i], n[i], r[i]);
        weights += m[i] * n[i];
    }
    return weights ? (double)bits / (double)weights : 0.0;
}

/* Strict 1.0-BPW rank: the largest r, a multiple of `multiple`, whose
 * storage_bits(m, n, r) does not exceed m*n.  Found by counting down from
 * the bound given by the sign bits alone, so no closed-form rearrangement
 * is involved. */
int64_t oracle_budget_rank(int64_t m, int64_t n, int64_t multiple)
{
    if (m <= 0 || n <= 0 || multiple <= 0)
        return 0;
    int64_t r = (m * n) / (m + n);
    r -= r % multiple;
    while (r > 0 && oracle_storage_bits(m, n, r) > m * n)
        r -= multiple;
    return r;
}

/* The paper's budget-to-rank conversion (App. A.1.3): r = Round(bits *
 * d_out * d_in / (d_out + d_in)), counting only the sign bits.  Rounding is
 * half away from zero; the clipping the paper mentions is left to callers. */
int64_t oracle_paper_rank(double bits_per_weight, int64_t m, int64_t n)
{
    if (m <= 0 || n <= 0)
        return 0;
    return (int64_t)llround(bits_per_weight * (double)m * (double)n /
                            (double)(m + n));
}

/* Threads OpenMP will use for the parallel loops above (1 without OpenMP). */
#ifdef _OPENMP
#include <omp.h>
int oracle_num_threads(void) { return omp_get_max_threads(); }
void oracle_set_num_threads(int t) { if (t > 0) omp_set_num_threads(t); }
#else
int oracle_num_threads(void) { return 1; }
void oracle_set_num_threads(int t) { (void)t; }
#endif
