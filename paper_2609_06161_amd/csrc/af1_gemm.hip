// Prefill-regime forward of the factorized binary linear on the gfx950
// matrix cores (paper App. A.2.1, Diag form; Sec. 4.1):
//
//   G1:  Z[t, k] = fp16( sum_j x[t, j] * (Bv[k, j] * s_in[j]) )
//   G2:  y[t, i] = bf16( s_out[i] * sum_k Z[t, k] * (Bu[i, k] * s_mid[k]) )
//
// Both are "activations x signed column scale" contractions,
//   C[t, n] = rowscale[n] * sum_c A[t, c] * (sign(W[n, c]) * colscale[c]),
// with A fp16 and W bit-packed.  Flipping the sign bit of the fp16 column
// scale keeps both MFMA operands exact (x is converted bf16 -> fp16, exact
// for |x| < 65504); accumulation is fp32.
//
// Pair order.  Within a 32-bit sign word, columns p and p+16 (p = 0..15)
// form one MFMA operand dword, so one shift and one three-input bit
// operation produce two fp16 operands (column-scale pair XOR the two sign
// bits).  The activations are kept in the same order: inside every group
// of 32 columns, column p sits at position 2p and column p+16 at 2p+1.  A
// pre-pass writes x in that order (converting bf16 to fp16 once, instead
// of once per weight-row tile), and G1 writes Z in that order, so both GEMMs
// stage their activation tiles with plain copies.
//
// Tiling.  A 256-thread workgroup computes a 128 (tokens) x 256 (weight
// rows) tile of C over K steps of 128 columns.  The activation tile is the
// only large operand (sign bits are 1/16 of its bytes per element), so the
// tile is wide in weight rows.  Each of the four waves owns 64 weight rows
// for all 128 tokens (4 x 2 blocks of v_mfma_f32_32x32x16_f16), so every
// sign bit is expanded exactly once, in registers, straight into an MFMA
// operand.
//
// Pipeline.  LDS holds two sets of (activation tile, column-scale pairs,
// sign words); each K step issues the global loads of the next step before
// its own MFMAs, consumes them only after the MFMAs, and meets one barrier.
// Per-step addresses move the scalar buffer base.  Columns past K
// read a zero column scale, so they contribute nothing whatever the
// activation or sign data they meet.  Tiles are assigned so that the
// workgroups of one XCD (blockIdx mod 8) work on a contiguous range of
// tiles and share activation rows in their L2.
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
constexpr int kWords = 4;        // sign words per K step
constexpr int BK = 32 * kWords;  // columns per K step
constexpr int kThreads = 256;
constexpr int kRowBytes = BK * 2 + 16;             // LDS bytes per token row (+16 pad)
constexpr int kATile = BM * kRowBytes;
constexpr int kCsBytes = kWords * 16 * 4;          // column-scale pairs of one K step
constexpr int kWBytes = BN * kWords * 4;           // sign words of one K step
constexpr int kAChunks = BM * BK * 2 / 16 / kThreads;  // 16-byte activation chunks per thread
constexpr int kLdsBytes = 2 * (kATile + kCsBytes + kWBytes);
constexpr int kOob = (int)0x80000000u;
static_assert(kAChunks * kThreads * 16 == BM * BK * 2, "activation chunks");
static_assert(4 * kWords <= kThreads, "column-scale staging");

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *base, int64_t bytes) {
  const int n = bytes > 0x7fffffff ? 0x7fffffff : (bytes < 0 ? 0 : (int)bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, n, 0x00020000);
}

// Two fp32 -> packed fp16 (round to nearest even).
__device__ __forceinline__ uint32_t pack_f16x2(float lo_half, float hi_half) {
  const float2v f = {lo_half, hi_half};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, half2v));
}

// Position of column c inside its 32-column group in pair order.
__device__ __forceinline__ int pair_pos(int c) {
  return (c & ~31) + 2 * (c & 15) + ((c >> 4) & 1);
}

// x (bf16, [T][K]) -> xp (fp16, [T][K], pair order).  One thread per 16
// columns: 8 columns c .. c+7 and their partners c+16 .. c+23 become the
// pair dwords 8h .. 8h+7 of their group.
__global__ __launch_bounds__(256) void pair_order_kernel(const uint16_t *__restrict__ x,
                                                         uint16_t *__restrict__ xp, int T, int K) {
  const int units_per_row = K / 16;
  const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (u >= (int64_t)T * units_per_row) return;
  const int t = (int)(u / units_per_row);
  const int ur = (int)(u % units_per_row);
  const int c = (ur >> 1) * 32 + 8 * (ur & 1);
  const uint16_t *src = x + (size_t)t * K + c;
  const u32x4 lo = *reinterpret_cast<const u32x4 *>(src);
  const u32x4 hi = *reinterpret_cast<const u32x4 *>(src + 16);
  uint32_t d[8];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    d[2 * e] = pack_f16x2(__uint_as_float(lo[e] << 16), __uint_as_float(hi[e] << 16));
    d[2 * e + 1] = pack_f16x2(__uint_as_float(lo[e] & 0xffff0000u), __uint_as_float(hi[e] & 0xffff0000u));
  }
  uint4 *dst = reinterpret_cast<uint4 *>(xp + (size_t)t * K + (c & ~31) + 2 * (c & 15));
  dst[0] = make_uint4(d[0], d[1], d[2], d[3]);
  dst[1] = make_uint4(d[4], d[5], d[6], d[7]);
}

// C = rowscale * (A_pairorder x (sign(W) * colscale)^T).  kOutBf16: C is
// bf16 in natural column order (y); otherwise fp16 in pair order (Z).
template <bool kOutBf16>
__global__ __launch_bounds__(kThreads, 2) void bingemm_kernel(
    const uint16_t *__restrict__ A, int T, int K, const uint32_t *__restrict__ W, int N,
    const uint16_t *__restrict__ colscale, const uint16_t *__restrict__ rowscale,
    uint16_t *__restrict__ C) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
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

  const int kw = K / 32;                       // sign words per row
  const int nk = (kw + kWords - 1) / kWords;   // K steps (the last may be partial)

  // Staging roles (fixed per thread; a step only adds a scalar offset).
  // Activations: 16-byte chunk q = tid + 256k of the tile -> token q / 16,
  // byte 16 (q mod 16) of the token's K-step slice (already in pair order).
  // Column scale: threads 0 .. 4*kWords-1 load columns c .. c+3 and c+16 ..
  // c+19 of word tid/4 and build 4 pair dwords.  Sign words: thread tid
  // stages row n0 + tid.
  int a_off[kAChunks], a_dst[kAChunks];
#pragma unroll
  for (int k = 0; k < kAChunks; ++k) {
    const int q = tid + kThreads * k;
    const int tok = q / (BK * 2 / 16), part = q % (BK * 2 / 16);
    a_off[k] = t0 + tok < T ? ((t0 + tok) * K) * 2 + 16 * part : kOob;
    a_dst[k] = tok * kRowBytes + 16 * part;
  }
  const bool cs_thread = tid < 4 * kWords;
  const int cs_off = cs_thread ? (32 * (tid >> 2) + 4 * (tid & 3)) * 2 : kOob;
  const int w_off = n0 + tid < N ? (n0 + tid) * kw * 4 : kOob;

  u32x4 a_raw[kAChunks];
  u32x2 cs_raw[2];
  uint32_t w_raw[kWords];
  // All of a step's loads are consumed only by store_stage, after the MFMAs
  // of the previous step, so the MFMAs never wait on global memory.  Every
  // thread issues every load (out-of-range offsets where there is nothing
  // to load), so the count of outstanding loads never depends on a branch.
  //  The step offset moves the (scalar) resource base rather than being a
  //  scalar offset: range checking covers the vector offset only, so every
  //  access is checked against what remains of its buffer from the base.
  auto load_stage = [&](int step) {
    const int ka = step * BK * 2;   // byte offset of the step in an A row / colscale
    const int kwb = step * kWords * 4;
    const __amdgpu_buffer_rsrc_t as = buffer_rsrc(A + step * BK, (int64_t)T * K * 2 - ka);
    const __amdgpu_buffer_rsrc_t cs = buffer_rsrc(colscale + step * BK, (int64_t)K * 2 - ka);
    const __amdgpu_buffer_rsrc_t ws = buffer_rsrc(W + step * kWords, (int64_t)N * kw * 4 - kwb);
#pragma unroll
    for (int k = 0; k < kAChunks; ++k)
      a_raw[k] = __builtin_amdgcn_raw_buffer_load_b128(as, a_off[k], 0, 0);
    cs_raw[0] = __builtin_amdgcn_raw_buffer_load_b64(cs, cs_off, 0, 0);
    cs_raw[1] = __builtin_amdgcn_raw_buffer_load_b64(cs, cs_off == kOob ? kOob : cs_off + 32, 0, 0);
#pragma unroll
    for (int i = 0; i < kWords; ++i)
      w_raw[i] = __builtin_amdgcn_raw_buffer_load_b32(ws, w_off == kOob ? kOob : w_off + 4 * i, 0, 0);
  };
  auto store_stage = [&](int buf) {
    uint8_t *at = lds + buf * kATile;
#pragma unroll
    for (int k = 0; k < kAChunks; ++k)
      *reinterpret_cast<u32x4 *>(at + a_dst[k]) = a_raw[k];
    if (cs_thread) {
      uint32_t d[4];
      d[0] = __builtin_amdgcn_perm(cs_raw[1].x, cs_raw[0].x, 0x05040100u);
      d[1] = __builtin_amdgcn_perm(cs_raw[1].x, cs_raw[0].x, 0x07060302u);
      d[2] = __builtin_amdgcn_perm(cs_raw[1].y, cs_raw[0].y, 0x05040100u);
      d[3] = __builtin_amdgcn_perm(cs_raw[1].y, cs_raw[0].y, 0x07060302u);
      reinterpret_cast<uint4 *>(lds + 2 * kATile + buf * kCsBytes)[tid] =
          make_uint4(d[0], d[1], d[2], d[3]);
    }
    uint32_t *wdst =
        reinterpret_cast<uint32_t *>(lds + 2 * kATile + 2 * kCsBytes + buf * kWBytes) + tid * kWords;
#pragma unroll
    for (int i = 0; i < kWords; ++i) wdst[i] = w_raw[i];
  };

  // This lane's weight rows: block j -> tile row 64*wave + 32*j + (l mod 32).
  const int wrow_l = 64 * wave + (lane & 31);
  const int wrow0 = n0 + wrow_l;

  floatx16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  uint32_t kSignMask;
  asm volatile("v_mov_b32 %0, 0x80008000" : "=v"(kSignMask));

  load_stage(0);
  store_stage(0);
  __syncthreads();

  const int g = lane >> 5;  // K half of an MFMA operand (slots 8g .. 8g+7)
  for (int step = 0; step < nk; ++step) {
    const int buf = step & 1;
    const bool more = step + 1 < nk;
    if (more) load_stage(step + 1);
    const uint8_t *at = lds + buf * kATile + (lane & 31) * kRowBytes + 16 * g;
    const uint4 *cs = reinterpret_cast<const uint4 *>(lds + 2 * kATile + buf * kCsBytes);
    const uint32_t *ws =
        reinterpret_cast<const uint32_t *>(lds + 2 * kATile + 2 * kCsBytes + buf * kWBytes);
    uint32_t wj[2][kWords];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < kWords; ++i) wj[j][i] = ws[(wrow_l + 32 * j) * kWords + i];
#pragma unroll
    for (int ks = 0; ks < 2 * kWords; ++ks) {
      const int wi = ks >> 1, s = ks & 1;
      // column-scale pairs and activation fragments of this MFMA K step:
      // pair dwords 16wi + 8s + 4g .. +3
      const uint4 c4 = cs[4 * wi + 2 * s + g];
      half8 af[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const half8 *>(at + 32 * i * kRowBytes + (16 * wi + 8 * s) * 4);
      const uint32_t cpair[4] = {c4.x, c4.y, c4.z, c4.w};
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const uint32_t w = wj[j][wi];
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
    if (more) store_stage(buf ^ 1);
    __syncthreads();
  }

  // Epilogue.  32x32 accumulator layout: lane l holds column (l mod 32) and
  // rows 8*(e/4) + 4*(l/32) + (e mod 4), e = 0..15.
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int n = wrow0 + 32 * j;
    if (n >= N) continue;
    const float rs = rowscale ? f16_to_f32(rowscale[n]) : 1.0f;
    const int cpos = kOutBf16 ? n : pair_pos(n);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int t = t0 + 32 * i + 8 * (e >> 2) + 4 * g + (e & 3);
        if (t < T) {
          const float v = acc[i][j][e] * rs;
          C[(size_t)t * N + cpos] = kOutBf16 ? f32_to_bf16(v) : f32_to_f16(v);
        }
      }
    }
  }
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

}  // namespace

size_t gemm_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t T) {
  (void)m;
  // fp16 x in pair order, then the fp16 intermediate Z (pair order)
  return align256((size_t)T * (size_t)n * 2) + align256((size_t)T * (size_t)r * 2);
}

hipError_t launch_gemm(int64_t m, int64_t n, int64_t r, const uint32_t *Bu,
                       const uint32_t *Bv, const uint16_t *s_out,
                       const uint16_t *s_mid, const uint16_t *s_in,
                       const uint16_t *x, int64_t T, uint16_t *y, void *ws,
                       hipStream_t s) {
  // byte offsets inside the buffer resources are 32-bit
  if (T * n * 2 > 0x7fffffff || T * r * 2 > 0x7fffffff || m * (r / 32) * 4 > 0x7fffffff ||
      r * (n / 32) * 4 > 0x7fffffff)
    return hipErrorInvalidValue;
  uint16_t *xp = static_cast<uint16_t *>(ws);
  uint16_t *Z = reinterpret_cast<uint16_t *>(static_cast<uint8_t *>(ws) + align256((size_t)T * n * 2));
  const int64_t units = T * (n / 16);
  pair_order_kernel<<<(unsigned)((units + 255) / 256), 256, 0, s>>>(x, xp, (int)T, (int)n);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const unsigned gy = (unsigned)((T + BM - 1) / BM);
  dim3 g1((unsigned)((r + BN - 1) / BN), gy);
  bingemm_kernel<false><<<g1, kThreads, kLdsBytes, s>>>(xp, (int)T, (int)n, Bv, (int)r, s_in,
                                                        nullptr, Z);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 g2((unsigned)((m + BN - 1) / BN), gy);
  bingemm_kernel<true><<<g2, kThreads, kLdsBytes, s>>>(Z, (int)T, (int)r, Bu, (int)m, s_mid,
                                                       s_out, y);
  return hipGetLastError();
}

}  // namespace af1
