// Prefill-regime forward of the factorized binary linear on the gfx950
// matrix cores (paper App. A.2.1, Diag form; Sec. 4.1):
//
//   G1:  Z[t, k] = fp16( sum_j x[t, j] * (Bv[k, j] * s_in[j]) )
//   G2:  y[t, i] = bf16( s_out[i] * sum_k Z[t, k] * (Bu[i, k] * s_mid[k]) )
//
// Both are "activations x signed column scale" contractions,
//   C[t, n] = rowscale[n] * sum_c A[t, c] * (sign(W[n, c]) * colscale[c]),
// with A fp16 (G1 converts the bf16 input on the way into LDS, exact for
// |x| < 65504) and W bit-packed.  Flipping the sign bit of the fp16 column
// scale keeps both MFMA operands exact; accumulation is fp32.
//
// Tiling.  A 256-thread workgroup computes a 128 (tokens) x 256 (weight
// rows) tile of C over K steps of 64 columns.  The activation tile is the
// only large operand (sign bits are 1/16 of its bytes per element), so the
// tile is wide in weight rows.  Each of the four waves owns 64 weight rows
// for all 128 tokens (4 x 2 blocks of v_mfma_f32_32x32x16_f16), so every
// sign bit is expanded exactly once, in registers, straight into an MFMA
// operand: within a 32-bit word, columns p and p+16 form one operand dword,
// so one shift and one three-input bit operation produce two fp16 operands
// (column-scale pair XOR the two sign bits).  The activation tile is stored
// in LDS in the same (p, p+16) pair order, and so is the column scale.
//
// Pipeline.  LDS holds two activation tiles; each K step issues the global
// loads of the next step (activations, sign words, column scale) before its
// own MFMAs, then converts and stores the next tile and meets one barrier.
// Tiles are assigned so that the workgroups on one XCD (blockIdx mod 8) work
// on a contiguous range of tiles and share activation rows in their L2.
#include "af1_device.h"
#include "af1_internal.h"

namespace af1 {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float float2v __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128;          // tokens per tile
constexpr int BN = 256;          // weight rows per tile
constexpr int BK = 64;           // columns per K step (two sign words)
constexpr int kThreads = 256;
constexpr int kRowBytes = 144;   // LDS bytes per token row: 64 fp16 + 16 pad
constexpr int kATile = BM * kRowBytes;
constexpr int kCsBytes = 128;    // column-scale pairs of one K step
constexpr int kOob = (int)0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *base, int64_t bytes) {
  const int n = bytes > 0x7fffffff ? 0x7fffffff : (bytes < 0 ? 0 : (int)bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, n, 0x00020000);
}

// Two fp32 -> packed fp16 (round to nearest even).
__device__ __forceinline__ uint32_t pack_f16x2(float lo_half, float hi_half) {
  const float2v f = {lo_half, hi_half};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, half2v));
}

// Pair dwords (column c+d, column c+16+d), d = 0..7, from the 16-byte loads
// of columns c..c+7 (lo) and c+16..c+23 (hi).  bf16 input is converted to
// fp16; fp16 input only has its halves interleaved.
template <bool kBf16>
__device__ __forceinline__ void make_pairs(const u32x4 &lo, const u32x4 &hi, uint32_t (&d)[8]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t a = lo[e], b = hi[e];
    if constexpr (kBf16) {
      d[2 * e] = pack_f16x2(__uint_as_float(a << 16), __uint_as_float(b << 16));
      d[2 * e + 1] = pack_f16x2(__uint_as_float(a & 0xffff0000u), __uint_as_float(b & 0xffff0000u));
    } else {
      d[2 * e] = __builtin_amdgcn_perm(b, a, 0x05040100u);      // (a.lo, b.lo)
      d[2 * e + 1] = __builtin_amdgcn_perm(b, a, 0x07060302u);  // (a.hi, b.hi)
    }
  }
}

template <bool kABf16, bool kOutBf16>
__global__ __launch_bounds__(kThreads, 2) void bingemm_kernel(
    const uint16_t *__restrict__ A, int T, int K, const uint32_t *__restrict__ W, int N,
    const uint16_t *__restrict__ colscale, const uint16_t *__restrict__ rowscale,
    uint16_t *__restrict__ C) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * kATile + 2 * kCsBytes];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // Tile assignment: consecutive workgroups land on consecutive XCDs; give
  // each XCD a contiguous range of tiles (weight-row tiles fastest).
  const int nN = gridDim.x, nT = gridDim.y, total = nN * nT;
  int L = blockIdx.y * nN + blockIdx.x;
  if ((total & 7) == 0) L = (L & 7) * (total >> 3) + (L >> 3);
  const int t0 = (L / nN) * BM;
  const int n0 = (L % nN) * BN;

  const int kw = K / 32;                // sign words per row
  const int nk = (kw + 1) / 2;          // K steps (the last may hold one word)
  const __amdgpu_buffer_rsrc_t ares = buffer_rsrc(A, (int64_t)T * K * 2);
  const __amdgpu_buffer_rsrc_t wres = buffer_rsrc(W, (int64_t)N * kw * 4);
  const __amdgpu_buffer_rsrc_t cres = buffer_rsrc(colscale, (int64_t)K * 2);

  // Staging roles.  Activation units: (token, word wi, half h) -> columns
  // 32wi+8h .. +7 and +16 .. +23; thread tid handles units tid and tid+256.
  // Column scale: threads 0..7 each build 4 pair dwords.
  int a_tok[2], a_col[2], a_dst[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int u = tid + kThreads * k;
    const int tok = u >> 2, wi = (u >> 1) & 1, h = u & 1;
    a_tok[k] = t0 + tok;
    a_col[k] = 32 * wi + 8 * h;
    a_dst[k] = tok * kRowBytes + (16 * wi + 8 * h) * 4;
  }
  const int cs_wi = tid >> 2, cs_part = tid & 3;  // valid for tid < 8

  u32x4 a_raw[2][2];
  u32x2 cs_raw[2];
  auto load_stage = [&](int step) {
    const int k0 = step * BK;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int col = k0 + a_col[k];
      const bool ok = a_tok[k] < T && col < K;
      const int off = ok ? (a_tok[k] * K + col) * 2 : kOob;
      a_raw[k][0] = __builtin_amdgcn_raw_buffer_load_b128(ares, off, 0, 0);
      a_raw[k][1] = __builtin_amdgcn_raw_buffer_load_b128(ares, ok ? off + 32 : kOob, 0, 0);
    }
    if (tid < 8) {
      const int c = k0 + 32 * cs_wi + 4 * cs_part;
      cs_raw[0] = __builtin_amdgcn_raw_buffer_load_b64(cres, c * 2, 0, 0);        // c..c+3
      cs_raw[1] = __builtin_amdgcn_raw_buffer_load_b64(cres, (c + 16) * 2, 0, 0); // c+16..
    }
  };
  auto store_stage = [&](int buf) {
    uint8_t *at = lds + buf * kATile;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      uint32_t d[8];
      make_pairs<kABf16>(a_raw[k][0], a_raw[k][1], d);
      uint4 *dst = reinterpret_cast<uint4 *>(at + a_dst[k]);
      dst[0] = make_uint4(d[0], d[1], d[2], d[3]);
      dst[1] = make_uint4(d[4], d[5], d[6], d[7]);
    }
    if (tid < 8) {
      uint32_t d[4];
      d[0] = __builtin_amdgcn_perm(cs_raw[1].x, cs_raw[0].x, 0x05040100u);
      d[1] = __builtin_amdgcn_perm(cs_raw[1].x, cs_raw[0].x, 0x07060302u);
      d[2] = __builtin_amdgcn_perm(cs_raw[1].y, cs_raw[0].y, 0x05040100u);
      d[3] = __builtin_amdgcn_perm(cs_raw[1].y, cs_raw[0].y, 0x07060302u);
      reinterpret_cast<uint4 *>(lds + 2 * kATile + buf * kCsBytes)[tid] =
          make_uint4(d[0], d[1], d[2], d[3]);
    }
  };

  // Sign words of this wave's rows: lane l, block j -> row n0 + 64*wave +
  // 32*j + (l mod 32); both words of the K step.
  const int wrow0 = n0 + 64 * wave + (lane & 31);
  auto load_w = [&](int step, u32x2 (&wb)[2]) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int row = wrow0 + 32 * j;
      const int w0 = 2 * step;
      // Two 4-byte loads, each range-checked on its own: with an odd word
      // count the second word of the last step lies past the row (and, for
      // the last row, past the buffer); it reads as zero.
      const int off = row < N ? (row * kw + w0) * 4 : kOob;
      wb[j].x = __builtin_amdgcn_raw_buffer_load_b32(wres, off, 0, 0);
      wb[j].y = __builtin_amdgcn_raw_buffer_load_b32(wres, (row < N && w0 + 1 < kw) ? off + 4 : kOob,
                                                     0, 0);
    }
  };

  floatx16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  uint32_t kSignMask;
  asm volatile("v_mov_b32 %0, 0x80008000" : "=v"(kSignMask));

  u32x2 wcur[2], wnext[2];
  load_stage(0);
  load_w(0, wcur);
  store_stage(0);
  __syncthreads();

  const int g = lane >> 5;  // K half of an MFMA operand (slots 8g .. 8g+7)
  for (int step = 0; step < nk; ++step) {
    const int buf = step & 1;
    const bool more = step + 1 < nk;
    if (more) {
      load_stage(step + 1);
      load_w(step + 1, wnext);
    }
    const uint8_t *at = lds + buf * kATile;
    const uint4 *cs = reinterpret_cast<const uint4 *>(lds + 2 * kATile + buf * kCsBytes);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int wi = ks >> 1, s = ks & 1;
      // column-scale pairs and activation fragments of this MFMA K step:
      // pair dwords 16wi + 8s + 4g .. +3
      const uint4 c4 = cs[4 * wi + 2 * s + g];
      half8 af[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const half8 *>(
            at + (32 * i + (lane & 31)) * kRowBytes + (16 * wi + 8 * s + 4 * g) * 4);
      const uint32_t cpair[4] = {c4.x, c4.y, c4.z, c4.w};
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const uint32_t w = wi ? wcur[j].y : wcur[j].x;
        uint32_t bd[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int p = 8 * s + 4 * g + e;  // g is lane-dependent: variable shift
          bd[e] = cpair[e] ^ ((w << (15 - p)) & kSignMask);
        }
        const half8 bf = __builtin_bit_cast(half8, make_uint4(bd[0], bd[1], bd[2], bd[3]));
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[i], bf, acc[i][j], 0, 0, 0);
      }
    }
    if (more) {
      store_stage(buf ^ 1);
      wcur[0] = wnext[0];
      wcur[1] = wnext[1];
    }
    __syncthreads();
  }

  // Epilogue.  32x32 accumulator layout: lane l holds column (l mod 32) and
  // rows 8*(e/4) + 4*(l/32) + (e mod 4), e = 0..15.
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int n = wrow0 + 32 * j;
    if (n >= N) continue;
    const float rs = rowscale ? f16_to_f32(rowscale[n]) : 1.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int t = t0 + 32 * i + 8 * (e >> 2) + 4 * g + (e & 3);
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
  // 32-bit element offsets inside the buffer resources
  if (T * n > 0x3fffffff || T * r > 0x3fffffff || T * m > 0x7fffffff ||
      m * (r / 32) > 0x1fffffff || r * (n / 32) > 0x1fffffff)
    return hipErrorInvalidValue;
  uint16_t *Z = static_cast<uint16_t *>(ws);
  const unsigned gy = (unsigned)((T + BM - 1) / BM);
  dim3 g1((unsigned)((r + BN - 1) / BN), gy);
  bingemm_kernel<true, false><<<g1, kThreads, 0, s>>>(x, (int)T, (int)n, Bv, (int)r, s_in,
                                                      nullptr, Z);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 g2((unsigned)((m + BN - 1) / BN), gy);
  bingemm_kernel<false, true><<<g2, kThreads, 0, s>>>(Z, (int)T, (int)r, Bu, (int)m, s_mid,
                                                      s_out, y);
  return hipGetLastError();
}

}  // namespace af1
