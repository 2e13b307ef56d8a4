// NABF building blocks on the GPU (paper Sec. 4.1 "Null-space-Aware Binary
// Factorization", Algorithm nabf in App. A.1, App. A.1.4 "ADMM-SVID Framework
// in DBF", App. A.2.2-A.2.5).  Offline calibration math for one linear:
//
//   surrogate      W' = o . W . i^T with i, o the RMS of calibration inputs
//                  and output gradients
//   SVID           signs of Z and a rank-1 fit |Z| ~ a v^T (power iteration)
//   null space     P = U_hat U_hat^T from the trailing eigenvectors of a PSD
//                  C that carry at most eta of its spectral energy
//   ADMM proxies   A_hat = (W' B^T + rho (A - U)) (B B^T + rho I)^-1 and
//                  B_hat = (A^T A + rho I)^-1 (A^T W' + rho (B - U))
//   scale fits     gamma, eta of the null-space-compensated targets
//   iteration      one pass of the NABF loop over both factors
//
// Dense matrices are fp32 row-major.  Plain matrix products go to rocBLAS,
// the Cholesky and symmetric eigen factorisations to rocSOLVER (the
// eigenproblem in fp64: the cutoff compares sums of eigenvalues); every
// other step -- the power iteration, the sign packing, the energy cutoff,
// the compensation and scale fits, the factor rebuilds and dual updates,
// the surrogate statistics -- is a kernel here.  Reductions take partial
// sums per tile and add them in a fixed order, so results repeat bit for
// bit.
#include <math.h>
#include <mutex>

#include <rocblas/rocblas.h>
#include <rocsolver/rocsolver.h>

#include "af1_device.h"
#include "af1_internal.h"
#include "af1_nabf.h"

namespace af1n {
namespace {

using af1::bf16_to_f32;
using af1::f32_to_f16;
using af1::wave_sum;

constexpr double kEps = 1e-12;   // residual-energy fraction and scale fits
constexpr int kChunk = 64;       // rows per partial-sum tile

// ---------------------------------------------------------------------------
// Device kernels
// ---------------------------------------------------------------------------

// part[chunk][j] = sum over tokens of the chunk of X[t][j]^2 (bf16 input).
__global__ __launch_bounds__(256) void colsq_kernel(const uint16_t *__restrict__ X, int T, int n,
                                                    float *__restrict__ part) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= n) return;
  const int t0 = blockIdx.y * kChunk;
  const int t1 = min(T, t0 + kChunk);
  float s = 0.f;
  for (int t = t0; t < t1; ++t) {
    const float v = bf16_to_f32(X[(size_t)t * n + j]);
    s += v * v;
  }
  part[(size_t)blockIdx.y * n + j] = s;
}

// out[j] = sqrt(sum over chunks of part[chunk][j] / T), chunks added in order.
__global__ __launch_bounds__(256) void rms_finish_kernel(const float *__restrict__ part, int chunks,
                                                         int n, int T, float *__restrict__ out) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= n) return;
  float s = 0.f;
  for (int c = 0; c < chunks; ++c) s += part[(size_t)c * n + j];
  out[j] = sqrtf(s / (float)T);
}

// Wp[u][j] = o[u] * W[u][j] * i[j].
__global__ __launch_bounds__(256) void surrogate_scale_kernel(const float *__restrict__ W, int64_t m,
                                                              int n, const float *__restrict__ o,
                                                              const float *__restrict__ iv,
                                                              float *__restrict__ Wp) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= n) return;
  const float ij = iv[j];
  for (int64_t u = blockIdx.y; u < m; u += gridDim.y)
    Wp[u * n + j] = o[u] * W[u * n + j] * ij;
}

__global__ __launch_bounds__(256) void fill_kernel(float *__restrict__ v, int n, float val) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j < n) v[j] = val;
}

// u[i] = sum_j |Z[i][j]| v[j]: one wave per row, 16-byte loads (cols % 32 == 0).
__global__ __launch_bounds__(256) void abs_rowdot_kernel(const float *__restrict__ Z, int64_t rows,
                                                         int cols, const float *__restrict__ v,
                                                         float *__restrict__ u) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= rows) return;
  const float4 *zr = reinterpret_cast<const float4 *>(Z + i * cols);
  const float4 *v4 = reinterpret_cast<const float4 *>(v);
  float s = 0.f;
  for (int q = lane; q < cols / 4; q += 64) {
    const float4 z = zr[q], w = v4[q];
    s += fabsf(z.x) * w.x + fabsf(z.y) * w.y + fabsf(z.z) * w.z + fabsf(z.w) * w.w;
  }
  s = wave_sum(s);
  if (lane == 0) u[i] = s;
}

// part[chunk][j] = sum over the chunk's rows i of |Z[i][j]| u[i].
__global__ __launch_bounds__(256) void abs_coldot_kernel(const float *__restrict__ Z, int64_t rows,
                                                         int cols, const float *__restrict__ u,
                                                         float *__restrict__ part) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= cols) return;
  const int64_t i0 = (int64_t)blockIdx.y * kChunk;
  const int64_t i1 = min(rows, i0 + kChunk);
  float s = 0.f;
  for (int64_t i = i0; i < i1; ++i) s += fabsf(Z[i * cols + j]) * u[i];
  part[(size_t)blockIdx.y * cols + j] = s;
}

// w[j] = sum over chunks of part[chunk][j] (in order); sq[block] = the
// block's sum of w^2 (lane order, then wave order).
__global__ __launch_bounds__(256) void coldot_finish_kernel(const float *__restrict__ part,
                                                            int chunks, int cols,
                                                            float *__restrict__ w,
                                                            float *__restrict__ sq) {
  __shared__ float red[4];
  const int j = blockIdx.x * 256 + threadIdx.x;
  float s = 0.f;
  if (j < cols) {
    for (int c = 0; c < chunks; ++c) s += part[(size_t)c * cols + j];
    w[j] = s;
  }
  const float q = wave_sum(s * s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = q;
  __syncthreads();
  if (threadIdx.x == 0) sq[blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}

// v = w / ||w|| (||w||^2 = the block partials added in order); v is kept
// when w is zero.
__global__ __launch_bounds__(256) void normalize_kernel(const float *__restrict__ w,
                                                        const float *__restrict__ sq, int nsq,
                                                        int cols, float *__restrict__ v) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= cols) return;
  float s = 0.f;
  for (int k = 0; k < nsq; ++k) s += sq[k];
  if (s > 0.f) v[j] = w[j] / sqrtf(s);
}

__global__ __launch_bounds__(256) void to_f64_kernel(const float *__restrict__ s,
                                                     double *__restrict__ d, int64_t n) {
  for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < n; k += (int64_t)gridDim.x * 256)
    d[k] = (double)s[k];
}

__global__ __launch_bounds__(256) void to_f32_kernel(const double *__restrict__ s,
                                                     float *__restrict__ d, int64_t n) {
  for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < n; k += (int64_t)gridDim.x * 256)
    d[k] = (float)s[k];
}

// Residual-energy cutoff (App. A.2.3) on the ascending eigenvalues D of a
// PSD matrix.  With lambda in descending order, rho_k is the sum of the
// r - k smallest eigenvalues over (total + eps); the first k (from 0 up)
// with rho_k <= eta is the largest count c = r - k of smallest eigenvalues
// whose sum stays within eta (total + eps).  One thread, in fp64.
__global__ void cutoff_kernel(const double *__restrict__ D, int r, double eta, double eps,
                              double *__restrict__ pre, int *__restrict__ count,
                              int *__restrict__ k_out) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  double s = 0.0;
  pre[0] = 0.0;
  for (int c = 0; c < r; ++c) {
    s += D[c];
    pre[c + 1] = s;
  }
  const double thr = eta * (s + eps);
  int c = 0;
  for (int cc = r; cc >= 0; --cc)
    if (pre[cc] <= thr) {
      c = cc;
      break;
    }
  *count = c;
  if (k_out) *k_out = r - c;
}

// Zero the eigenvector columns past the selected count (column-major U).
__global__ __launch_bounds__(256) void mask_columns_kernel(double *__restrict__ U, int r,
                                                           const int *__restrict__ count) {
  const int c = *count;
  const int64_t n = (int64_t)r * r;
  for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < n; k += (int64_t)gridDim.x * 256)
    if (k / r >= c) U[k] = 0.0;
}

// G = C + rho I (copy), both r x r.
__global__ __launch_bounds__(256) void shift_copy_kernel(const float *__restrict__ C,
                                                         float *__restrict__ G, int r, float rho) {
  const int64_t n = (int64_t)r * r;
  for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < n; k += (int64_t)gridDim.x * 256)
    G[k] = C[k] + ((k / r == k % r) ? rho : 0.f);
}

// out = alpha (x - y) or x + y, elementwise.
__global__ __launch_bounds__(256) void scaled_diff_kernel(const float *__restrict__ x,
                                                          const float *__restrict__ y, float alpha,
                                                          float *__restrict__ out, int64_t n) {
  for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < n; k += (int64_t)gridDim.x * 256)
    out[k] = alpha * (x[k] - y[k]);
}
__global__ __launch_bounds__(256) void add_kernel(const float *__restrict__ x,
                                                  const float *__restrict__ y,
                                                  float *__restrict__ out, int64_t n) {
  for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < n; k += (int64_t)gridDim.x * 256)
    out[k] = x[k] + y[k];
}

// The binary-scaled matrix left . S . right^T at (i, j); bit 1 is -1.
__device__ __forceinline__ float bscaled(const uint32_t *__restrict__ bits,
                                         const float *__restrict__ left,
                                         const float *__restrict__ right, int64_t i, int j,
                                         int cols) {
  const uint32_t word = bits[i * (cols / 32) + (j >> 5)];
  const float v = left[i] * right[j];
  return ((word >> (j & 31)) & 1u) ? -v : v;
}

// E = hat - (left . S . right^T).
__global__ __launch_bounds__(256) void residual_kernel(const float *__restrict__ hat,
                                                       const uint32_t *__restrict__ bits,
                                                       const float *__restrict__ left,
                                                       const float *__restrict__ right,
                                                       int64_t rows, int cols,
                                                       float *__restrict__ E) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= cols) return;
  for (int64_t i = blockIdx.y; i < rows; i += gridDim.y)
    E[i * cols + j] = hat[i * cols + j] - bscaled(bits, left, right, i, j, cols);
}

// dense = left . S . right^T, and U += hat - dense (when U is given).
__global__ __launch_bounds__(256) void rebuild_kernel(const uint32_t *__restrict__ bits,
                                                      const float *__restrict__ left,
                                                      const float *__restrict__ right,
                                                      int64_t rows, int cols,
                                                      const float *__restrict__ hat,
                                                      float *__restrict__ dense,
                                                      float *__restrict__ U) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= cols) return;
  for (int64_t i = blockIdx.y; i < rows; i += gridDim.y) {
    const float q = bscaled(bits, left, right, i, j, cols);
    dense[i * cols + j] = q;
    if (U) U[i * cols + j] += hat[i * cols + j] - q;
  }
}

// Column fit partials: num = sum_i q (hat - HP), den = sum_i q^2 over a chunk
// of rows, q the binary-scaled entry.
__global__ __launch_bounds__(256) void colfit_kernel(const float *__restrict__ hat,
                                                     const float *__restrict__ HP,
                                                     const uint32_t *__restrict__ bits,
                                                     const float *__restrict__ left,
                                                     const float *__restrict__ right, int64_t rows,
                                                     int cols, float *__restrict__ pnum,
                                                     float *__restrict__ pden) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= cols) return;
  const int64_t i0 = (int64_t)blockIdx.y * kChunk;
  const int64_t i1 = min(rows, i0 + kChunk);
  float num = 0.f, den = 0.f;
  for (int64_t i = i0; i < i1; ++i) {
    const float q = bscaled(bits, left, right, i, j, cols);
    num += q * (hat[i * cols + j] - HP[i * cols + j]);
    den += q * q;
  }
  pnum[(size_t)blockIdx.y * cols + j] = num;
  pden[(size_t)blockIdx.y * cols + j] = den;
}

__global__ __launch_bounds__(256) void colfit_finish_kernel(const float *__restrict__ pnum,
                                                            const float *__restrict__ pden,
                                                            int chunks, int cols, float eps,
                                                            float *__restrict__ fit) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= cols) return;
  float num = 0.f, den = 0.f;
  for (int c = 0; c < chunks; ++c) {
    num += pnum[(size_t)c * cols + j];
    den += pden[(size_t)c * cols + j];
  }
  fit[j] = num / (den + eps);
}

// Row fit: one block per row k, fit[k] = sum_j q (hat - HP) / (sum_j q^2 + eps).
__global__ __launch_bounds__(256) void rowfit_kernel(const float *__restrict__ hat,
                                                     const float *__restrict__ HP,
                                                     const uint32_t *__restrict__ bits,
                                                     const float *__restrict__ left,
                                                     const float *__restrict__ right, int cols,
                                                     float eps, float *__restrict__ fit) {
  __shared__ float rn[4], rd[4];
  const int64_t k = blockIdx.x;
  float num = 0.f, den = 0.f;
  for (int j = threadIdx.x; j < cols; j += 256) {
    const float q = bscaled(bits, left, right, k, j, cols);
    num += q * (hat[k * cols + j] - HP[k * cols + j]);
    den += q * q;
  }
  num = wave_sum(num);
  den = wave_sum(den);
  if ((threadIdx.x & 63) == 0) {
    rn[threadIdx.x >> 6] = num;
    rd[threadIdx.x >> 6] = den;
  }
  __syncthreads();
  if (threadIdx.x == 0)
    fit[k] = (((rn[0] + rn[1]) + rn[2]) + rn[3]) / ((((rd[0] + rd[1]) + rd[2]) + rd[3]) + eps);
}

// X[i + j * ld] /= (D[j or i] + rho): dim 0 scales the rows of a
// column-major block (index i), dim 1 its columns (index j).
__global__ __launch_bounds__(256) void inv_shift_scale_kernel(float *__restrict__ X, int64_t rows,
                                                              int64_t cols,
                                                              const double *__restrict__ D,
                                                              float rho, int dim) {
  const int64_t n = rows * cols;
  for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < n; k += (int64_t)gridDim.x * 256) {
    const int64_t e = dim == 0 ? k % rows : k / rows;
    X[k] = (float)((double)X[k] / (D[e] + (double)rho));
  }
}

__global__ __launch_bounds__(256) void mul_kernel(float *__restrict__ x, const float *__restrict__ y,
                                                  int n) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j < n) x[j] *= y[j];
}

// Deployable scales: s_out = a / o, s_mid = m1 . m2, s_in = b / i (binary16,
// round to nearest even).
__global__ __launch_bounds__(256) void export_kernel(const float *__restrict__ a,
                                                     const float *__restrict__ m1,
                                                     const float *__restrict__ m2,
                                                     const float *__restrict__ b,
                                                     const float *__restrict__ iv,
                                                     const float *__restrict__ o, int m, int n,
                                                     int r, uint16_t *__restrict__ s_out,
                                                     uint16_t *__restrict__ s_mid,
                                                     uint16_t *__restrict__ s_in) {
  int k = blockIdx.x * 256 + threadIdx.x;
  if (k < m) {
    s_out[k] = f32_to_f16(o ? a[k] / o[k] : a[k]);
    return;
  }
  k -= m;
  if (k < r) {
    s_mid[k] = f32_to_f16(m1[k] * m2[k]);
    return;
  }
  k -= r;
  if (k < n) s_in[k] = f32_to_f16(iv ? b[k] / iv[k] : b[k]);
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------

unsigned blocks_for(int64_t n) { return (unsigned)((n + 255) / 256); }
unsigned grid_cap(int64_t n) {
  const int64_t b = (n + 255) / 256;
  return (unsigned)(b < 4096 ? (b > 0 ? b : 1) : 4096);
}
unsigned rows_grid(int64_t rows) { return (unsigned)(rows < 65535 ? rows : 65535); }
int64_t chunks_of(int64_t rows) { return (rows + kChunk - 1) / kChunk; }
size_t al(size_t v) { return (v + 255) & ~(size_t)255; }

// One rocBLAS handle per device, created on first use.  The mutex is held
// for a whole entry point call, so concurrent calls on one device take turns
// setting the handle's stream.
struct DeviceHandle {
  std::mutex mu;
  rocblas_handle h = nullptr;
};
DeviceHandle g_handles[64];

struct Handle {
  std::unique_lock<std::mutex> lock;
  rocblas_handle h = nullptr;
  bool ok = false;
  explicit Handle(hipStream_t s) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return;
    lock = std::unique_lock<std::mutex>(g_handles[dev].mu);
    if (!g_handles[dev].h && rocblas_create_handle(&g_handles[dev].h) != rocblas_status_success) {
      g_handles[dev].h = nullptr;
      return;
    }
    h = g_handles[dev].h;
    ok = rocblas_set_stream(h, s) == rocblas_status_success;
  }
};

#define CHECK_HIP(x)                              \
  do {                                            \
    if ((x) != hipSuccess) return AF1_ERR_HIP;    \
  } while (0)
#define CHECK_LAUNCH() CHECK_HIP(hipGetLastError())
#define CHECK_RB(x)                                          \
  do {                                                       \
    if ((x) != rocblas_status_success) return AF1_ERR_HIP;   \
  } while (0)

const rocblas_operation kN = rocblas_operation_none, kT = rocblas_operation_transpose;

// C (m x n, column-major, ldc) = alpha op(A) op(B) + beta C.
af1_status sgemm(rocblas_handle h, rocblas_operation ta, rocblas_operation tb, int64_t m, int64_t n,
                 int64_t k, const float *A, int64_t lda, const float *B, int64_t ldb, float beta,
                 float *C, int64_t ldc) {
  const float alpha = 1.f;
  CHECK_RB(rocblas_sgemm(h, ta, tb, (rocblas_int)m, (rocblas_int)n, (rocblas_int)k, &alpha, A,
                         (rocblas_int)lda, B, (rocblas_int)ldb, &beta, C, (rocblas_int)ldc));
  return AF1_OK;
}

// ---- workspace layout (one query covers every entry point) ----------------

struct Ws {
  float *hat_a, *hat_b, *z, *e, *ep, *c, *g, *p, *svid_part, *svid_w, *svid_sq, *fit, *pnum, *pden,
      *rms_part;
  double *c64, *p64, *d, *e64, *pre;
  int *count, *info, *k;
};

size_t ws_layout(int64_t m, int64_t n, int64_t r, int64_t T, uint8_t *base, Ws *w) {
  const int64_t big = (m > n ? m : n) * r;
  const int64_t maxdim = m > n ? (m > r ? m : r) : (n > r ? n : r);
  const int64_t rows_max = maxdim;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    uint8_t *p = base ? base + off : nullptr;
    off += al(bytes);
    return p;
  };
  Ws t;
  t.hat_a = (float *)take((size_t)m * r * 4);
  t.hat_b = (float *)take((size_t)r * n * 4);
  t.z = (float *)take((size_t)big * 4);
  t.e = (float *)take((size_t)big * 4);
  t.ep = (float *)take((size_t)big * 4);
  t.c = (float *)take((size_t)r * r * 4);
  t.g = (float *)take((size_t)r * r * 4);
  t.p = (float *)take((size_t)r * r * 4);
  t.svid_part = (float *)take((size_t)chunks_of(rows_max) * maxdim * 4);
  t.svid_w = (float *)take((size_t)maxdim * 4);
  t.svid_sq = (float *)take((size_t)blocks_for(maxdim) * 4);
  t.fit = (float *)take((size_t)maxdim * 4);
  t.pnum = (float *)take((size_t)chunks_of(rows_max) * r * 4);
  t.pden = (float *)take((size_t)chunks_of(rows_max) * r * 4);
  t.rms_part = (float *)take((size_t)chunks_of(T > 0 ? T : 1) * (m + n) * 4);
  t.c64 = (double *)take((size_t)r * r * 8);
  t.p64 = (double *)take((size_t)r * r * 8);
  t.d = (double *)take((size_t)r * 8);
  t.e64 = (double *)take((size_t)r * 8);
  t.pre = (double *)take((size_t)(r + 1) * 8);
  t.count = (int *)take(4);
  t.info = (int *)take(4);
  t.k = (int *)take(4);
  if (w) *w = t;
  return off;
}

// The scratch of a stand-alone SVID of a rows x cols matrix (the power
// iteration's partial sums), laid out from the start of the workspace; it
// never exceeds the layout above for a layer that has such a factor.
size_t svid_layout(int64_t rows, int64_t cols, uint8_t *base, Ws *w) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    uint8_t *p = base ? base + off : nullptr;
    off += al(bytes);
    return p;
  };
  Ws t{};
  t.svid_part = (float *)take((size_t)chunks_of(rows) * cols * 4);
  t.svid_w = (float *)take((size_t)cols * 4);
  t.svid_sq = (float *)take((size_t)blocks_for(cols) * 4);
  if (w) *w = t;
  return off;
}

// ---- building blocks (arguments already validated) ------------------------

af1_status run_svid(const float *Z, int64_t rows, int64_t cols, int iters, uint32_t *bits,
                    float *left, float *right, const Ws &w, hipStream_t s) {
  const unsigned cb = blocks_for(cols);
  const int64_t chunks = chunks_of(rows);
  fill_kernel<<<cb, 256, 0, s>>>(right, (int)cols, 1.0f / sqrtf((float)cols));
  CHECK_LAUNCH();
  const unsigned rowblocks = (unsigned)((rows + 3) / 4);
  for (int it = 0; it < iters; ++it) {
    abs_rowdot_kernel<<<rowblocks, 256, 0, s>>>(Z, rows, (int)cols, right, left);
    CHECK_LAUNCH();
    abs_coldot_kernel<<<dim3(cb, (unsigned)chunks), 256, 0, s>>>(Z, rows, (int)cols, left,
                                                                  w.svid_part);
    CHECK_LAUNCH();
    coldot_finish_kernel<<<cb, 256, 0, s>>>(w.svid_part, (int)chunks, (int)cols, w.svid_w,
                                            w.svid_sq);
    CHECK_LAUNCH();
    normalize_kernel<<<cb, 256, 0, s>>>(w.svid_w, w.svid_sq, (int)cb, (int)cols, right);
    CHECK_LAUNCH();
  }
  abs_rowdot_kernel<<<rowblocks, 256, 0, s>>>(Z, rows, (int)cols, right, left);
  CHECK_LAUNCH();
  CHECK_HIP(af1::launch_pack(Z, 0, rows, cols, bits, s));
  return AF1_OK;
}

// C = U diag(D) U^T in fp64 (U column-major in w.c64, D ascending in w.d).
af1_status run_eig(rocblas_handle h, const float *C, int64_t r, const Ws &w, hipStream_t s) {
  const int64_t rr = r * r;
  to_f64_kernel<<<grid_cap(rr), 256, 0, s>>>(C, w.c64, rr);
  CHECK_LAUNCH();
  CHECK_RB(rocsolver_dsyevd(h, rocblas_evect_original, rocblas_fill_upper, (rocblas_int)r, w.c64,
                            (rocblas_int)r, w.d, w.e64, w.info));
  return AF1_OK;
}

// P from the decomposition in w.c64 / w.d (the eigenvectors are masked in
// place, so any other use of them comes first).
af1_status projector_from_eig(rocblas_handle h, int64_t r, float eta, float *P, int *k_out,
                              const Ws &w, hipStream_t s) {
  const int64_t rr = r * r;
  cutoff_kernel<<<1, 64, 0, s>>>(w.d, (int)r, (double)eta, kEps, w.pre, w.count, k_out);
  CHECK_LAUNCH();
  mask_columns_kernel<<<grid_cap(rr), 256, 0, s>>>(w.c64, (int)r, w.count);
  CHECK_LAUNCH();
  const double one = 1.0, zero = 0.0;
  CHECK_RB(rocblas_dgemm(h, kN, kT, (rocblas_int)r, (rocblas_int)r, (rocblas_int)r, &one, w.c64,
                         (rocblas_int)r, w.c64, (rocblas_int)r, &zero, w.p64, (rocblas_int)r));
  to_f32_kernel<<<grid_cap(rr), 256, 0, s>>>(w.p64, P, rr);
  CHECK_LAUNCH();
  return AF1_OK;
}

af1_status run_projector(rocblas_handle h, const float *C, int64_t r, float eta, float *P,
                         int *k_out, const Ws &w, hipStream_t s) {
  af1_status st = run_eig(h, C, r, w, s);
  if (st != AF1_OK) return st;
  return projector_from_eig(h, r, eta, P, k_out, w, s);
}

// Left proxy into out (m x r).  The Gram matrix B B^T is left in w.c.
af1_status run_admm_left(rocblas_handle h, const float *Wp, int64_t m, int64_t n, int64_t r,
                         const float *A, const float *B, const float *U, float rho, float *out,
                         const Ws &w, hipStream_t s) {
  // B row-major r x n is column-major n x r: B B^T = B_c^T B_c.
  af1_status st = sgemm(h, kT, kN, r, r, n, B, n, B, n, 0.f, w.c, r);
  if (st != AF1_OK) return st;
  shift_copy_kernel<<<grid_cap(r * r), 256, 0, s>>>(w.c, w.g, (int)r, rho);
  CHECK_LAUNCH();
  scaled_diff_kernel<<<grid_cap(m * r), 256, 0, s>>>(A, U, rho, out, m * r);
  CHECK_LAUNCH();
  // out^T (r x m, column-major) += B W'^T = B_c^T W'_c
  st = sgemm(h, kT, kN, r, m, n, B, n, Wp, n, 1.f, out, r);
  if (st != AF1_OK) return st;
  // X G = R  <=>  G X^T = R^T: a left solve on the column-major view
  CHECK_RB(rocsolver_spotrf(h, rocblas_fill_lower, (rocblas_int)r, w.g, (rocblas_int)r, w.info));
  CHECK_RB(rocsolver_spotrs(h, rocblas_fill_lower, (rocblas_int)r, (rocblas_int)m, w.g,
                            (rocblas_int)r, out, (rocblas_int)r));
  return AF1_OK;
}

// Right proxy into out (r x n).  The Gram matrix A^T A is left in w.c.
af1_status run_admm_right(rocblas_handle h, const float *Wp, int64_t m, int64_t n, int64_t r,
                          const float *A, const float *B, const float *U, float rho, float *out,
                          const Ws &w, hipStream_t s) {
  // A row-major m x r is column-major r x m: A^T A = A_c A_c^T.
  af1_status st = sgemm(h, kN, kT, r, r, m, A, r, A, r, 0.f, w.c, r);
  if (st != AF1_OK) return st;
  shift_copy_kernel<<<grid_cap(r * r), 256, 0, s>>>(w.c, w.g, (int)r, rho);
  CHECK_LAUNCH();
  scaled_diff_kernel<<<grid_cap(r * n), 256, 0, s>>>(B, U, rho, out, r * n);
  CHECK_LAUNCH();
  // out^T (n x r, column-major) += W'^T A = W'_c A_c^T
  st = sgemm(h, kN, kT, n, r, m, Wp, n, A, r, 1.f, out, n);
  if (st != AF1_OK) return st;
  // G X = R  <=>  X^T G = R^T: two right-side triangular solves with G = L L^T
  CHECK_RB(rocsolver_spotrf(h, rocblas_fill_lower, (rocblas_int)r, w.g, (rocblas_int)r, w.info));
  const float one = 1.f;
  CHECK_RB(rocblas_strsm(h, rocblas_side_right, rocblas_fill_lower, kT, rocblas_diagonal_non_unit,
                         (rocblas_int)n, (rocblas_int)r, &one, w.g, (rocblas_int)r, out,
                         (rocblas_int)n));
  CHECK_RB(rocblas_strsm(h, rocblas_side_right, rocblas_fill_lower, kN, rocblas_diagonal_non_unit,
                         (rocblas_int)n, (rocblas_int)r, &one, w.g, (rocblas_int)r, out,
                         (rocblas_int)n));
  return AF1_OK;
}

// gamma (side 0: hat is rows x r, P acts on the right) or eta (side 1: hat is
// r x cols, P acts on the left) into fit.
af1_status run_fit(rocblas_handle h, int side, const float *hat, const uint32_t *bits,
                   const float *left, const float *right, int64_t rows, int64_t cols,
                   const float *P, float *fit, const Ws &w, hipStream_t s) {
  const unsigned cb = blocks_for(cols);
  residual_kernel<<<dim3(cb, rows_grid(rows)), 256, 0, s>>>(hat, bits, left, right, rows,
                                                             (int)cols, w.e);
  CHECK_LAUNCH();
  if (side == 0) {
    // EP = E P (rows x r): column-major EP^T = P E^T (P symmetric)
    af1_status st = sgemm(h, kN, kN, cols, rows, cols, P, cols, w.e, cols, 0.f, w.ep, cols);
    if (st != AF1_OK) return st;
    const int64_t chunks = chunks_of(rows);
    colfit_kernel<<<dim3(cb, (unsigned)chunks), 256, 0, s>>>(hat, w.ep, bits, left, right, rows,
                                                              (int)cols, w.pnum, w.pden);
    CHECK_LAUNCH();
    colfit_finish_kernel<<<cb, 256, 0, s>>>(w.pnum, w.pden, (int)chunks, (int)cols, (float)kEps,
                                            fit);
    CHECK_LAUNCH();
  } else {
    // PE = P E (r x cols): column-major PE^T = E^T P
    af1_status st = sgemm(h, kN, kN, cols, rows, rows, w.e, cols, P, rows, 0.f, w.ep, cols);
    if (st != AF1_OK) return st;
    rowfit_kernel<<<(unsigned)rows, 256, 0, s>>>(hat, w.ep, bits, left, right, (int)cols,
                                                 (float)kEps, fit);
    CHECK_LAUNCH();
  }
  return AF1_OK;
}

// The proxies of one iteration, solved with the eigendecomposition of the
// Gram matrix that the null-space projector needs anyway:
// (C + rho I)^-1 = U diag(1 / (D + rho)) U^T.  w.c holds C on entry; on
// exit w.c64 / w.d hold its decomposition and w.g the fp32 eigenvectors.
af1_status proxy_by_eig(rocblas_handle h, int side, const float *Wp, int64_t m, int64_t n,
                        int64_t r, const float *A, const float *B, const float *U, float rho,
                        float *out, const Ws &w, hipStream_t s) {
  af1_status st = run_eig(h, w.c, r, w, s);
  if (st != AF1_OK) return st;
  to_f32_kernel<<<grid_cap(r * r), 256, 0, s>>>(w.c64, w.g, r * r);
  CHECK_LAUNCH();
  if (side == 0) {
    scaled_diff_kernel<<<grid_cap(m * r), 256, 0, s>>>(A, U, rho, out, m * r);
    CHECK_LAUNCH();
    st = sgemm(h, kT, kN, r, m, n, B, n, Wp, n, 1.f, out, r);   // R^T += B W'^T
    if (st != AF1_OK) return st;
    // X^T = U diag U^T R^T (column-major r x m)
    st = sgemm(h, kT, kN, r, m, r, w.g, r, out, r, 0.f, w.ep, r);
    if (st != AF1_OK) return st;
    inv_shift_scale_kernel<<<grid_cap(m * r), 256, 0, s>>>(w.ep, r, m, w.d, rho, 0);
    CHECK_LAUNCH();
    return sgemm(h, kN, kN, r, m, r, w.g, r, w.ep, r, 0.f, out, r);
  }
  scaled_diff_kernel<<<grid_cap(r * n), 256, 0, s>>>(B, U, rho, out, r * n);
  CHECK_LAUNCH();
  st = sgemm(h, kN, kT, n, r, m, Wp, n, A, r, 1.f, out, n);      // R^T += W'^T A
  if (st != AF1_OK) return st;
  // X^T = R^T U diag U^T (column-major n x r)
  st = sgemm(h, kN, kN, n, r, r, out, n, w.g, r, 0.f, w.ep, n);
  if (st != AF1_OK) return st;
  inv_shift_scale_kernel<<<grid_cap(n * r), 256, 0, s>>>(w.ep, n, r, w.d, rho, 1);
  CHECK_LAUNCH();
  return sgemm(h, kN, kT, n, r, r, w.ep, n, w.g, r, 0.f, out, n);
}

af1_status run_iteration(rocblas_handle h, const float *Wp, const af1_nabf_state *S, float rho,
                         float eta, int iters, const Ws &w, hipStream_t s) {
  const int64_t m = S->m, n = S->n, r = S->r;
  // left-factor update: C_B = B B^T gives both the proxy's solve and P_B
  af1_status st = sgemm(h, kT, kN, r, r, n, S->B, n, S->B, n, 0.f, w.c, r);
  if (st != AF1_OK) return st;
  st = proxy_by_eig(h, 0, Wp, m, n, r, S->A, S->B, S->UA, rho, w.hat_a, w, s);
  if (st != AF1_OK) return st;
  add_kernel<<<grid_cap(m * r), 256, 0, s>>>(w.hat_a, S->UA, w.z, m * r);
  CHECK_LAUNCH();
  st = run_svid(w.z, m, r, iters, S->A_bits, S->a, S->m1, w, s);
  if (st != AF1_OK) return st;
  st = projector_from_eig(h, r, eta, w.p, nullptr, w, s);   // null space of B B^T
  if (st != AF1_OK) return st;
  st = run_fit(h, 0, w.hat_a, S->A_bits, S->a, S->m1, m, r, w.p, w.fit, w, s);
  if (st != AF1_OK) return st;
  mul_kernel<<<blocks_for(r), 256, 0, s>>>(S->m1, w.fit, (int)r);
  CHECK_LAUNCH();
  rebuild_kernel<<<dim3(blocks_for(r), rows_grid(m)), 256, 0, s>>>(S->A_bits, S->a, S->m1, m,
                                                                   (int)r, w.hat_a, S->A, S->UA);
  CHECK_LAUNCH();
  // right-factor update with the new left factor: C_A = A^T A
  st = sgemm(h, kN, kT, r, r, m, S->A, r, S->A, r, 0.f, w.c, r);
  if (st != AF1_OK) return st;
  st = proxy_by_eig(h, 1, Wp, m, n, r, S->A, S->B, S->UB, rho, w.hat_b, w, s);
  if (st != AF1_OK) return st;
  add_kernel<<<grid_cap(r * n), 256, 0, s>>>(w.hat_b, S->UB, w.z, r * n);
  CHECK_LAUNCH();
  st = run_svid(w.z, r, n, iters, S->B_bits, S->m2, S->b, w, s);
  if (st != AF1_OK) return st;
  st = projector_from_eig(h, r, eta, w.p, nullptr, w, s);   // null space of A^T A
  if (st != AF1_OK) return st;
  st = run_fit(h, 1, w.hat_b, S->B_bits, S->m2, S->b, r, n, w.p, w.fit, w, s);
  if (st != AF1_OK) return st;
  mul_kernel<<<blocks_for(r), 256, 0, s>>>(S->m2, w.fit, (int)r);
  CHECK_LAUNCH();
  rebuild_kernel<<<dim3(blocks_for(n), rows_grid(r)), 256, 0, s>>>(S->B_bits, S->m2, S->b, r,
                                                                   (int)n, w.hat_b, S->B, S->UB);
  CHECK_LAUNCH();
  return AF1_OK;
}

// ---- validation helpers ---------------------------------------------------

bool dim_ok(int64_t d) { return d >= 32 && d <= AF1_NABF_MAX_DIM && d % 32 == 0; }

struct Span {
  uintptr_t lo, hi;
};
Span span(const void *p, uint64_t bytes) {
  const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
  return Span{lo, lo + (uintptr_t)bytes};
}
// true when any two of the non-empty spans overlap
bool any_overlap(const Span *s, int count) {
  for (int i = 0; i < count; ++i)
    for (int j = i + 1; j < count; ++j)
      if (s[i].lo != s[i].hi && s[j].lo != s[j].hi && s[i].lo < s[j].hi && s[j].lo < s[i].hi)
        return true;
  return false;
}
// rocBLAS takes 32-bit dimensions and leading dimensions; keep every matrix
// below 2^31 elements as well.
bool counts_ok(int64_t a, int64_t b) { return a * b <= (int64_t)INT32_MAX; }
bool a16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
hipStream_t as_stream(void *s) { return static_cast<hipStream_t>(s); }

}  // namespace
}  // namespace af1n

using namespace af1n;

extern "C" {

size_t af1_nabf_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t T) {
  if (!dim_ok(m) || !dim_ok(n) || !dim_ok(r) || T < 0 || T > AF1_NABF_MAX_TOKENS) return 0;
  return ws_layout(m, n, r, T, nullptr, nullptr);
}

af1_status af1_nabf_surrogate(const float *W, int64_t m, int64_t n, const uint16_t *X,
                              const uint16_t *G, int64_t T, float *Wp, float *i_vec, float *o_vec,
                              void *ws, size_t ws_bytes, void *stream) {
  if (!W || !X || !G || !Wp || !i_vec || !o_vec) return AF1_ERR_NULL;
  if (!dim_ok(m) || !dim_ok(n) || !counts_ok(m, n)) return AF1_ERR_SHAPE;
  if (T < 1 || T > AF1_NABF_MAX_TOKENS) return AF1_ERR_BATCH;
  if (!a16(W) || !a16(X) || !a16(G) || !a16(Wp) || !a16(i_vec) || !a16(o_vec) || (ws && !a16(ws)))
    return AF1_ERR_ALIGN;
  Ws w;
  const size_t need = ws_layout(m, n, 32, T, static_cast<uint8_t *>(ws), &w);
  if (!ws || ws_bytes < need) return AF1_ERR_WORKSPACE;
  if (W == Wp) return AF1_ERR_ALIAS;
  hipStream_t s = as_stream(stream);
  const int64_t chunks = chunks_of(T);
  float *px = w.rms_part, *pg = w.rms_part + chunks * n;
  colsq_kernel<<<dim3(blocks_for(n), (unsigned)chunks), 256, 0, s>>>(X, (int)T, (int)n, px);
  CHECK_LAUNCH();
  colsq_kernel<<<dim3(blocks_for(m), (unsigned)chunks), 256, 0, s>>>(G, (int)T, (int)m, pg);
  CHECK_LAUNCH();
  rms_finish_kernel<<<blocks_for(n), 256, 0, s>>>(px, (int)chunks, (int)n, (int)T, i_vec);
  CHECK_LAUNCH();
  rms_finish_kernel<<<blocks_for(m), 256, 0, s>>>(pg, (int)chunks, (int)m, (int)T, o_vec);
  CHECK_LAUNCH();
  surrogate_scale_kernel<<<dim3(blocks_for(n), rows_grid(m)), 256, 0, s>>>(W, m, (int)n, o_vec,
                                                                           i_vec, Wp);
  CHECK_LAUNCH();
  return AF1_OK;
}

af1_status af1_svid(const float *Z, int64_t rows, int64_t cols, int32_t iters, uint32_t *bits,
                    float *left, float *right, void *ws, size_t ws_bytes, void *stream) {
  if (!Z || !bits || !left || !right) return AF1_ERR_NULL;
  if (!dim_ok(rows) || !dim_ok(cols) || !counts_ok(rows, cols) || iters < 0 ||
      iters > AF1_NABF_MAX_POWER_ITERS)
    return AF1_ERR_SHAPE;
  if (!a16(Z) || !a16(bits) || !a16(left) || !a16(right) || (ws && !a16(ws))) return AF1_ERR_ALIGN;
  Ws w;
  const size_t need = svid_layout(rows, cols, static_cast<uint8_t *>(ws), &w);
  if (!ws || ws_bytes < need) return AF1_ERR_WORKSPACE;
  return run_svid(Z, rows, cols, iters, bits, left, right, w, as_stream(stream));
}

af1_status af1_nullspace_projector(const float *C, int64_t r, float eta, float *P, int32_t *k_out,
                                   void *ws, size_t ws_bytes, void *stream) {
  if (!C || !P) return AF1_ERR_NULL;
  if (!dim_ok(r) || !(eta >= 0.f && eta <= 1.f)) return AF1_ERR_SHAPE;
  if (!a16(C) || !a16(P) || (ws && !a16(ws))) return AF1_ERR_ALIGN;
  Ws w;
  const size_t need = ws_layout(32, 32, r, 0, static_cast<uint8_t *>(ws), &w);
  if (!ws || ws_bytes < need) return AF1_ERR_WORKSPACE;
  if (C == P) return AF1_ERR_ALIAS;
  hipStream_t s = as_stream(stream);
  Handle h(s);
  if (!h.ok) return AF1_ERR_HIP;
  return run_projector(h.h, C, r, eta, P, k_out, w, s);
}

af1_status af1_admm_proxy(int32_t side, const float *Wp, int64_t m, int64_t n, int64_t r,
                          const float *A, const float *B, const float *U, float rho, float *out,
                          void *ws, size_t ws_bytes, void *stream) {
  if (side != 0 && side != 1) return AF1_ERR_SHAPE;
  if (!Wp || !A || !B || !U || !out) return AF1_ERR_NULL;
  if (!dim_ok(m) || !dim_ok(n) || !dim_ok(r) || !counts_ok(m, n) || !counts_ok(m, r) ||
      !counts_ok(r, n) || !(rho > 0.f))
    return AF1_ERR_SHAPE;
  if (!a16(Wp) || !a16(A) || !a16(B) || !a16(U) || !a16(out) || (ws && !a16(ws)))
    return AF1_ERR_ALIGN;
  Ws w;
  const size_t need = ws_layout(m, n, r, 0, static_cast<uint8_t *>(ws), &w);
  if (!ws || ws_bytes < need) return AF1_ERR_WORKSPACE;
  if (out == Wp || out == A || out == B || out == U) return AF1_ERR_ALIAS;
  hipStream_t s = as_stream(stream);
  Handle h(s);
  if (!h.ok) return AF1_ERR_HIP;
  return side == 0 ? run_admm_left(h.h, Wp, m, n, r, A, B, U, rho, out, w, s)
                   : run_admm_right(h.h, Wp, m, n, r, A, B, U, rho, out, w, s);
}

af1_status af1_scale_fit(int32_t side, const float *hat, const uint32_t *bits, const float *left,
                         const float *right, int64_t rows, int64_t cols, const float *P, float *fit,
                         void *ws, size_t ws_bytes, void *stream) {
  if (side != 0 && side != 1) return AF1_ERR_SHAPE;
  if (!hat || !bits || !left || !right || !P || !fit) return AF1_ERR_NULL;
  if (!dim_ok(rows) || !dim_ok(cols) || !counts_ok(rows, cols)) return AF1_ERR_SHAPE;
  if (!a16(hat) || !a16(bits) || !a16(left) || !a16(right) || !a16(P) || !a16(fit) ||
      (ws && !a16(ws)))
    return AF1_ERR_ALIGN;
  Ws w;
  // side 0: rows = m, cols = r; side 1: rows = r, cols = n
  const size_t need = side == 0 ? ws_layout(rows, 32, cols, 0, static_cast<uint8_t *>(ws), &w)
                                : ws_layout(32, cols, rows, 0, static_cast<uint8_t *>(ws), &w);
  if (!ws || ws_bytes < need) return AF1_ERR_WORKSPACE;
  hipStream_t s = as_stream(stream);
  Handle h(s);
  if (!h.ok) return AF1_ERR_HIP;
  return run_fit(h.h, side, hat, bits, left, right, rows, cols, P, fit, w, s);
}

af1_status af1_nabf_iteration(const float *Wp, const af1_nabf_state *S, float rho, float eta,
                              int32_t power_iters, void *ws, size_t ws_bytes, void *stream) {
  if (!Wp || !S) return AF1_ERR_NULL;
  if (!S->A || !S->B || !S->UA || !S->UB || !S->A_bits || !S->B_bits || !S->a || !S->m1 ||
      !S->m2 || !S->b)
    return AF1_ERR_NULL;
  if (!dim_ok(S->m) || !dim_ok(S->n) || !dim_ok(S->r) || !counts_ok(S->m, S->n) ||
      !counts_ok(S->m, S->r) || !counts_ok(S->r, S->n) || !(rho > 0.f) ||
      !(eta >= 0.f && eta <= 1.f) || power_iters < 0 || power_iters > AF1_NABF_MAX_POWER_ITERS)
    return AF1_ERR_SHAPE;
  const void *ptrs[] = {Wp, S->A, S->B, S->UA, S->UB, S->A_bits, S->B_bits, S->a, S->m1, S->m2,
                        S->b};
  for (const void *p : ptrs)
    if (!a16(p)) return AF1_ERR_ALIGN;
  if (ws && !a16(ws)) return AF1_ERR_ALIGN;
  Ws w;
  const size_t need = ws_layout(S->m, S->n, S->r, 0, static_cast<uint8_t *>(ws), &w);
  if (!ws || ws_bytes < need) return AF1_ERR_WORKSPACE;
  const uint64_t m = S->m, n = S->n, r = S->r;
  const Span spans[] = {span(Wp, m * n * 4),     span(S->A, m * r * 4),   span(S->B, r * n * 4),
                        span(S->UA, m * r * 4),  span(S->UB, r * n * 4),  span(S->A_bits, m * r / 8),
                        span(S->B_bits, r * n / 8), span(S->a, m * 4),    span(S->m1, r * 4),
                        span(S->m2, r * 4),      span(S->b, n * 4),       span(ws, need)};
  if (any_overlap(spans, (int)(sizeof(spans) / sizeof(spans[0])))) return AF1_ERR_ALIAS;
  hipStream_t s = as_stream(stream);
  Handle h(s);
  if (!h.ok) return AF1_ERR_HIP;
  return run_iteration(h.h, Wp, S, rho, eta, power_iters, w, s);
}

af1_status af1_nabf_export(const af1_nabf_state *S, const float *i_vec, const float *o_vec,
                           uint16_t *s_out, uint16_t *s_mid, uint16_t *s_in, void *stream) {
  if (!S || !S->a || !S->m1 || !S->m2 || !S->b || !s_out || !s_mid || !s_in) return AF1_ERR_NULL;
  if (!dim_ok(S->m) || !dim_ok(S->n) || !dim_ok(S->r)) return AF1_ERR_SHAPE;
  hipStream_t s = as_stream(stream);
  export_kernel<<<blocks_for(S->m + S->r + S->n), 256, 0, s>>>(
      S->a, S->m1, S->m2, S->b, i_vec, o_vec, (int)S->m, (int)S->n, (int)S->r, s_out, s_mid, s_in);
  CHECK_LAUNCH();
  return AF1_OK;
}

}  // extern "C"
