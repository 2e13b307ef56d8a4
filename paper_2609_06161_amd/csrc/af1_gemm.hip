// Prefill-regime forward of the factorized binary linear on the gfx950
// matrix cores (paper App. A.2.1, Diag form; Sec. 4.1):
//
//   G1:  Z[t, k] = fp16( sum_j x[t, j] * (Bv[k, j] * s_in[j]) )
//   G2:  y[t, i] = bf16( s_out[i] * sum_k Z[t, k] * (Bu[i, k] * s_mid[k]) )
//
// Both are "activations x signed column scale" contractions,
//   C[t, n] = rowscale[n] * sum_c A[t, c] * (sign(W[n, c]) * colscale[c]),
// with A fp16 (G1 converts the bf16 input on load) and W bit-packed.  Folding
// the column scale into the +-1 operand keeps both MFMA operands exact fp16
// values; accumulation is fp32.
//
// Tiling: a 256-thread workgroup computes a 128 x 128 tile of C with four
// waves in a 2 x 2 arrangement (64 x 64 each, 2 x 2 MFMA 32x32x16 blocks).
// Per 32-wide K step the A tile is staged to LDS as fp16 and the 128 weight
// words are expanded to fp16 (+-colscale) into LDS, so the bit expansion is
// done once per workgroup and shared by all four waves.
#include "af1_device.h"
#include "af1_internal.h"

namespace af1 {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int BK = 32;
constexpr int LDH = BK + 8;  // LDS row stride in halves (80 B)

__device__ __forceinline__ uint32_t bf16x2_to_f16x2(uint32_t v) {
  const _Float16 lo = (_Float16)bf16_to_f32(v & 0xffffu);
  const _Float16 hi = (_Float16)bf16_to_f32(v >> 16);
  return (uint32_t)__builtin_bit_cast(uint16_t, lo) |
         ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
}

template <bool kABf16, bool kOutBf16>
__global__ __launch_bounds__(256) void bingemm_kernel(
    const uint16_t *__restrict__ A, int T, int K, const uint32_t *__restrict__ W, int N,
    const uint16_t *__restrict__ colscale, const uint16_t *__restrict__ rowscale,
    uint16_t *__restrict__ C) {
  __shared__ __attribute__((aligned(16))) _Float16 As[BM * LDH];
  __shared__ __attribute__((aligned(16))) _Float16 Bs[BN * LDH];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int t0 = blockIdx.y * BM;
  const int n0 = blockIdx.x * BN;
  const int kw = K / 32;

  floatx16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  for (int kb = 0; kb < kw; ++kb) {
    // A tile: BM rows x 32 halves, four 16-byte pieces per row.
#pragma unroll
    for (int it = 0; it < (BM * 4) / 256; ++it) {
      const int i = tid + it * 256;
      const int row = i >> 2, part = i & 3;
      const int t = t0 + row;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (t < T) v = *reinterpret_cast<const uint4 *>(A + (size_t)t * K + kb * 32 + part * 8);
      if constexpr (kABf16) {
        v.x = bf16x2_to_f16x2(v.x);
        v.y = bf16x2_to_f16x2(v.y);
        v.z = bf16x2_to_f16x2(v.z);
        v.w = bf16x2_to_f16x2(v.w);
      }
      *reinterpret_cast<uint4 *>(&As[row * LDH + part * 8]) = v;
    }
    // W tile: BN words -> BN x 32 halves of +-colscale.
    if (tid < BN) {
      const int n = n0 + tid;
      const uint32_t w = (n < N) ? W[(size_t)n * kw + kb] : 0u;
      const uint4 *cs = reinterpret_cast<const uint4 *>(colscale + kb * 32);
      uint32_t d[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint4 c = cs[q];
        d[4 * q + 0] = c.x;
        d[4 * q + 1] = c.y;
        d[4 * q + 2] = c.z;
        d[4 * q + 3] = c.w;
      }
#pragma unroll
      for (int p = 0; p < 16; ++p) {
        const uint32_t lo = (w >> (2 * p)) & 1u;
        const uint32_t hi = (w >> (2 * p + 1)) & 1u;
        d[p] ^= (lo << 15) | (hi << 31);
      }
      uint4 *dst = reinterpret_cast<uint4 *>(&Bs[tid * LDH]);
#pragma unroll
      for (int q = 0; q < 4; ++q) dst[q] = make_uint4(d[4 * q], d[4 * q + 1], d[4 * q + 2], d[4 * q + 3]);
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      half8 a[2], bb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = *reinterpret_cast<const half8 *>(
            &As[(wm * 64 + i * 32 + (lane & 31)) * LDH + ks * 16 + 8 * (lane >> 5)]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bb[j] = *reinterpret_cast<const half8 *>(
            &Bs[(wn * 64 + j * 32 + (lane & 31)) * LDH + ks * 16 + 8 * (lane >> 5)]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[i], bb[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }

  // Epilogue.  32x32 accumulator layout: lane l holds column (l mod 32) and
  // rows 8*(e/4) + 4*(l/32) + (e mod 4) for e = 0..15.
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int n = n0 + wn * 64 + j * 32 + (lane & 31);
    if (n >= N) continue;
    const float rs = rowscale ? f16_to_f32(rowscale[n]) : 1.0f;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int t = t0 + wm * 64 + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (t < T) {
          const float v = acc[i][j][e] * rs;
          C[(size_t)t * N + n] = kOutBf16 ? f32_to_bf16(v) : f32_to_f16(v);
        }
      }
    }
  }
}

}  // namespace

size_t gemm_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t T) {
  (void)m;
  (void)n;
  const size_t z = (size_t)T * (size_t)r * sizeof(uint16_t);
  return (z + 255) & ~(size_t)255;
}

hipError_t launch_gemm(int64_t m, int64_t n, int64_t r, const uint32_t *Bu,
                       const uint32_t *Bv, const uint16_t *s_out,
                       const uint16_t *s_mid, const uint16_t *s_in,
                       const uint16_t *x, int64_t T, uint16_t *y, void *ws,
                       hipStream_t s) {
  uint16_t *Z = static_cast<uint16_t *>(ws);
  const int gy = (int)((T + BM - 1) / BM);
  dim3 g1((unsigned)((r + BN - 1) / BN), (unsigned)gy);
  bingemm_kernel<true, false><<<g1, 256, 0, s>>>(x, (int)T, (int)n, Bv, (int)r, s_in, nullptr, Z);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 g2((unsigned)((m + BN - 1) / BN), (unsigned)gy);
  bingemm_kernel<false, true><<<g2, 256, 0, s>>>(Z, (int)T, (int)r, Bu, (int)m, s_mid, s_out, y);
  return hipGetLastError();
}

}  // namespace af1
