// Sign <-> bit packing of the binary factors (paper App. A.3: each sign of
// A_pm1 / B_pm1 is stored in one bit).
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

}  // namespace af1
