// Sign <-> bit packing of the binary factors (paper App. A.3: each sign of
// A_pm1 / B_pm1 is stored in one bit), and the bit transpose of the packed
// storage.
//
// Layout: word w of the flat row-major matrix holds elements 32w .. 32w+31,
// element 32w+j in bit j; bit 1 means -1.  Because cols is a multiple of 32,
// row boundaries fall on word boundaries and the flat view is exact.
//
// One thread builds one word from 32 consecutive source elements with
// 16-byte loads (the 32 elements of a word are contiguous and 16-byte
// aligned), and writes it with a coalesced 4-byte store.
#include "af1_device.h"
#include "af1_internal.h"

namespace af1 {
namespace {

// Element bytes -> number of uint4 loads per word, and the sign bit of each
// element inside a 32-bit lane of the loaded data.
template <int ElemBytes>
__device__ __forceinline__ uint32_t word_from_src(const uint4 *p) {
  constexpr int kLoads = ElemBytes * 32 / 16;
  uint32_t word = 0;
#pragma unroll
  for (int q = 0; q < kLoads; ++q) {
    uint4 v = p[q];
    uint32_t d[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if constexpr (ElemBytes == 4) {
        word |= (d[e] >> 31) << (q * 4 + e);
      } else if constexpr (ElemBytes == 2) {
        const int base = (q * 4 + e) * 2;
        word |= ((d[e] >> 15) & 1u) << base;
        word |= (d[e] >> 31) << (base + 1);
      } else {
        const int base = (q * 4 + e) * 4;
#pragma unroll
        for (int t = 0; t < 4; ++t) word |= ((d[e] >> (8 * t + 7)) & 1u) << (base + t);
      }
    }
  }
  return word;
}

template <int ElemBytes>
__global__ __launch_bounds__(256) void pack_kernel(const uint4 *__restrict__ src,
                                                   uint32_t *__restrict__ dst,
                                                   int64_t nwords) {
  constexpr int kLoads = ElemBytes * 32 / 16;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; w < nwords; w += stride)
    dst[w] = word_from_src<ElemBytes>(src + w * kLoads);
}

__global__ __launch_bounds__(256) void unpack_kernel(const uint32_t *__restrict__ words,
                                                     uint4 *__restrict__ dst,
                                                     int64_t nwords) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; w < nwords; w += stride) {
    const uint32_t word = words[w];
    uint32_t out[8];
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      uint32_t v = 0;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const uint32_t bit = (word >> (4 * d + t)) & 1u;
        v |= (bit ? 0xffu : 0x01u) << (8 * t);   // int8 -1 or +1
      }
      out[d] = v;
    }
    dst[2 * w] = make_uint4(out[0], out[1], out[2], out[3]);
    dst[2 * w + 1] = make_uint4(out[4], out[5], out[6], out[7]);
  }
}

// ---------------------------------------------------------------------------
// Bit transpose of the packed storage.  The gradients of the scale-only
// reconstruction (Sec. 4.1) multiply by Bu^T and Bv^T; with the signs
// frozen, each factor is transposed once into the same row-major packed
// format and the backward products then read whole words along K exactly
// as the forward ones do.
//
// A workgroup transposes a tile of 512 source rows x 16 source words (512
// columns).  Thread (rb, w) loads the 32 x 32 bit block of source rows
// 32 rb .. 32 rb + 31 and word w (lanes of consecutive w read 64
// contiguous bytes of a row), transposes it in registers, and parks the 32
// result words in LDS; the tile then leaves row by row, 16 consecutive
// destination words (64 bytes) per row.
// ---------------------------------------------------------------------------

constexpr int kTrRows = 512;   // source rows per tile
constexpr int kTrWords = 16;   // source words per tile

// In-register transpose of a 32 x 32 bit matrix: on entry bit j of a[i] is
// entry (i, j), on exit entry (j, i).  Each round s = 16, 8, 4, 2, 1 swaps
// the two off-diagonal s x s blocks inside every 2s x 2s diagonal block:
// rows i and i + s (bit s of i clear) exchange the columns of row i whose
// index has bit s set for the columns of row i + s whose index has it clear.
template <int S, uint32_t kKeep>
__device__ __forceinline__ void transpose_round(uint32_t (&a)[32]) {
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    if (i & S) continue;
    const uint32_t lo = a[i], hi = a[i + S];
    a[i] = (lo & kKeep) | ((hi << S) & ~kKeep);
    a[i + S] = ((lo >> S) & kKeep) | (hi & ~kKeep);
  }
}

__device__ __forceinline__ void transpose32(uint32_t (&a)[32]) {
  transpose_round<16, 0x0000ffffu>(a);
  transpose_round<8, 0x00ff00ffu>(a);
  transpose_round<4, 0x0f0f0f0fu>(a);
  transpose_round<2, 0x33333333u>(a);
  transpose_round<1, 0x55555555u>(a);
}

// LDS position of word c of tile row R (512 rows x 16 words).  Rows are
// permuted (low two bits XOR bits 5-6) and words XORed with a multiple of 4
// taken from bits 7-8, so that both the register-to-LDS writes (16 rows 32
// apart, 4 words each) and the row-wise reads of a wave hit 64 distinct
// banks.
__device__ __forceinline__ int tr_pos(int R, int c) {
  const int w = R >> 5;
  return ((R ^ (w & 3)) << 4) + (c ^ ((w >> 2) << 2));
}

__global__ __launch_bounds__(256) void transpose_kernel(const uint32_t *__restrict__ src,
                                                        int64_t rows, int64_t cols,
                                                        uint32_t *__restrict__ dst) {
  __shared__ uint32_t tile[kTrRows * kTrWords];
  const int tid = threadIdx.x;
  const int w = tid & 15, rb = tid >> 4;
  const int64_t swords = cols / 32, dwords = rows / 32;
  const int64_t row0 = (int64_t)blockIdx.y * kTrRows;
  const int64_t cw0 = (int64_t)blockIdx.x * kTrWords;
  const int64_t cw = cw0 + w, rbase = row0 + 32 * rb;
  uint32_t a[32];
  if (cw < swords && rbase < rows) {  // rows is a multiple of 32: whole blocks
    const uint32_t *p = src + rbase * swords + cw;
#pragma unroll
    for (int i = 0; i < 32; ++i) a[i] = p[(int64_t)i * swords];
  } else {
#pragma unroll
    for (int i = 0; i < 32; ++i) a[i] = 0u;
  }
  transpose32(a);
  // a[k]: destination row 32 cw + k (tile row 32 w + k), word row0/32 + rb
#pragma unroll
  for (int k = 0; k < 32; ++k) tile[tr_pos(32 * w + k, rb)] = a[k];
  __syncthreads();
  const int c = tid & 15;
  const int64_t oword = row0 / 32 + c;
#pragma unroll 4
  for (int q = 0; q < 32; ++q) {
    const int R = (tid >> 4) + 16 * q;
    const int64_t orow = 32 * cw0 + R;
    if (orow < cols && oword < dwords) dst[orow * dwords + oword] = tile[tr_pos(R, c)];
  }
}

int grid_for(int64_t nwords) {
  int64_t blocks = (nwords + 255) / 256;
  const int64_t cap = 256 * 64;  // grid-stride beyond this
  return (int)(blocks < cap ? (blocks > 0 ? blocks : 1) : cap);
}

}  // namespace

hipError_t launch_pack(const void *src, int dtype, int64_t rows, int64_t cols,
                       uint32_t *dst, hipStream_t s) {
  const int64_t nwords = rows * (cols / 32);
  if (nwords == 0) return hipSuccess;
  const uint4 *p = static_cast<const uint4 *>(src);
  const int g = grid_for(nwords);
  switch (dtype) {
    case 0: pack_kernel<4><<<g, 256, 0, s>>>(p, dst, nwords); break;
    case 1:
    case 2: pack_kernel<2><<<g, 256, 0, s>>>(p, dst, nwords); break;
    default: pack_kernel<1><<<g, 256, 0, s>>>(p, dst, nwords); break;
  }
  return hipGetLastError();
}

hipError_t launch_unpack(const uint32_t *words, int64_t rows, int64_t cols,
                         int8_t *dst, hipStream_t s) {
  const int64_t nwords = rows * (cols / 32);
  if (nwords == 0) return hipSuccess;
  unpack_kernel<<<grid_for(nwords), 256, 0, s>>>(words, reinterpret_cast<uint4 *>(dst), nwords);
  return hipGetLastError();
}

hipError_t launch_transpose(const uint32_t *src, int64_t rows, int64_t cols, uint32_t *dst,
                            hipStream_t s) {
  if (rows == 0 || cols == 0) return hipSuccess;
  const dim3 g((unsigned)((cols / 32 + kTrWords - 1) / kTrWords),
               (unsigned)((rows + kTrRows - 1) / kTrRows));
  transpose_kernel<<<g, 256, 0, s>>>(src, rows, cols, dst);
  return hipGetLastError();
}

}  // namespace af1
