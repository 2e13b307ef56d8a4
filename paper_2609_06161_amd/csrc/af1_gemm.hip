// Prefill-regime forward of the factorized binary linear on the gfx950
// matrix cores (paper App. A.2.1, Diag form; Sec. 4.1), and the contractions
// of its scale-only reconstruction (Sec. 4.1: sign matrices frozen, the
// gradients of the three scale vectors and of x through the transposed
// factors; the modes are listed under Mode below):
//
//   G1:  Z[t, k] = fp16( s_mid[k] * sum_j xs[t, j] * Bv[k, j] ),
//        xs = fp16(s_in .* x)
//   G2:  y[t, i] = bf16( s_out[i] * sum_k Z[t, k] * Bu[i, k] )
//
// Every contraction has the form
//   C[t, n] = rowscale[n] * sum_c A[t, c] * sign(W[n, c]),
// with A fp16 (the column scales already folded in, each product rounded
// once to fp16) and W bit-packed, so the B operand of the matrix cores is
// exactly +-1.  The other placement, the signed column scale as B and the
// activations exact, costs the same instructions but draws more power per
// MFMA (the B mantissas toggle); under the chip's power limit it ran 5-8%
// slower on the 70B-shaped layers.  Accumulation is fp32.
//
// Pair order.  Within a 32-bit sign word, columns p and p+16 (p = 0..15)
// form one MFMA operand dword, so one shift and one three-input bit
// operation produce two fp16 operands (the +1 pair XOR the two sign bits).
// The activations are kept in the same order: inside every group of 32
// columns, column p sits at position 2p and column p+16 at 2p+1.  A
// preparation pass writes fp16(s_in .* x) in that order, and G1 writes Z in
// that order, so the GEMMs stage their operands with plain copies.
//
// Tiling.  A 256-thread workgroup computes a 128 (tokens) x 256 (weight
// rows) tile of C over K steps of 128 columns.  The activation tile is the
// only large operand (sign bits are 1/16 of its bytes per element), so the
// tile is wide in weight rows.  Each of the four waves owns 64 weight rows
// for all 128 tokens (4 x 2 blocks of v_mfma_f32_32x32x16_f16), so every
// sign bit is expanded exactly once, in registers, straight into an MFMA
// operand.
//
// Staging.  Operands go from global memory straight into LDS (buffer loads
// with the LDS destination), double-buffered: a K step issues the copies of
// the next step, runs its MFMAs, waits for its copies and meets one
// barrier (a three-buffer variant, two steps ahead, is a template option;
// it measured slower).  No staging registers are needed, which leaves room
// to read the next MFMA step's operands from LDS while the current one
// runs.  An LDS
// copy instruction writes 64 consecutive 16-byte chunks, one per lane, but
// each lane chooses its source: the chunk of token row t holding columns
// 8c .. 8c+7 of the step is stored at chunk position c XOR (t mod 16) of the
// row, so that the MFMA operand reads (16 bytes per lane, consecutive
// tokens) fall in distinct LDS banks.  Tiles are assigned so that the
// workgroups of one XCD (blockIdx mod 8) work on a contiguous range of
// tiles and share activation rows in their L2.  The 16-bit output tile is
// assembled in LDS and leaves in 16-byte rows.
//
// Few tokens.  When the tile grid leaves compute units idle, a forward
// contraction splits its K steps over grid z and a reduction launch adds
// the fp32 partials in split order (see plan_contraction).
#include <utility>

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

// What one launch of the contraction computes (the A operand, the sign
// words and the tiling are the same in all of them).  acc is the signed
// product: in the forward modes R - 2 x (the MFMA sum over set sign bits,
// see the sign operands below), scaled by the token's range-guard shift; in
// the backward modes the MFMA sum against +-1 operands.
//   kMid     forward G1: C = fp16(rowscale * acc) times the column factors,
//            pair order, and the per-tile row sums of C into RS.
//   kMidSave kMid, and V = fp16(acc) (pair order) for the backward.
//   kOut     forward G2: C = bf16(rowscale * acc).
//   kOutSave kOut, and F = acc (fp32, natural order) for the backward.
//   kBwdMid  backward, first product: acc times gscale[2G] (G = the token's
//            64-token group) is dt; C = fp16(rowscale * acc *
//            gscale[2G + 1]), pair order; F = per-tile token sums of dt * S,
//            S fp16 in pair order.
//   kBwdIn   backward, second product: acc gscale[2G] / gscale[2G + 1] is
//            du; C = bf16(rowscale * du) when C is given; F = per-tile token
//            sums of du * S, S bf16 in natural order.
// The backward's A operands also carry a power-of-two scale per 64-token
// group (see bwd_prep_kernel).  With a split K (grid z > 1) a workgroup
// instead writes the fp32 partial of its K steps to P and
// splitk_reduce_kernel (forward modes) or splitk_bwd_reduce_kernel
// produces the mode's outputs.
enum Mode : int { kMid = 0, kMidSave = 1, kOut = 2, kOutSave = 3, kBwdMid = 4, kBwdIn = 5 };

constexpr int BM = 128;          // tokens per tile
constexpr int BN = 256;          // weight rows per tile
constexpr int kWords = 4;        // sign words per K step
constexpr int BK = 32 * kWords;  // columns per K step
constexpr int kThreads = 256;
constexpr int kARow = BK * 2;                // bytes of one token row of a K step
constexpr int kATile = BM * kARow;           // 32 KiB
constexpr int kWTile = BN * kWords * 4;      // 4 KiB
// LDS map: A0 .. A(S-1) | W0 .. W(S-1) for S pipeline stages (the
// activation buffers first, so operand reads are immediate offsets from one
// address), then the forward's per-token tables (the range-guard shift and
// the row sum R of each of the tile's tokens), for a token tile of kBM rows
// (128, or 64 for grids that would give each compute unit at most one
// workgroup).
template <int kBM, int kStages>
struct Lds {
  static constexpr int kATileT = kBM * kARow;
  static constexpr int kA0 = 0;
  static constexpr int kW0 = kStages * kATileT;
  static constexpr int kTab = kW0 + kStages * kWTile;
  static constexpr int kBytes = kTab + 8 * kBM;
};
constexpr int kOob = (int)0x80000000u;
static_assert(BM * kARow == 32 * 1024 && kThreads == 256, "eight 1 KiB copies per wave at BM");
static_assert(kATile + 3 * 32 * kARow + kARow < 65536, "immediate LDS offsets");

typedef __attribute__((address_space(3))) void lds_void;
typedef int i32x4 __attribute__((ext_vector_type(4)));

// The same raw buffer resource (stride 0, raw dword access) as four scalar
// dwords, for the copy instructions below.
__device__ __forceinline__ i32x4 copy_rsrc(const void *base, int64_t bytes) {
  const int n = bytes > 0x7fffffff ? 0x7fffffff : (bytes < 0 ? 0 : (int)bytes);
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return i32x4{(int)(uint32_t)a, (int)((a >> 32) & 0xffffu), n, 0x00020000};
}

// Global -> LDS copies: lane l of the wave writes `bytes` bytes at
// dst + bytes * l (dst wave-uniform, passed in M0), read from voff of the
// resource (zero when out of range).  Written as inline assembly so that the
// compiler does not wait for them before every LDS read (it cannot tell
// that they target the other buffer); wait_copies() is the only wait.
__device__ __forceinline__ void copy16(i32x4 r, uint8_t *dst, int voff) {
  const uint32_t m = (uint32_t)(size_t)(lds_void *)dst;
  asm volatile("buffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(voff), "s"(r), "{m0}"(m) : "memory");
}
__device__ __forceinline__ void copy4(i32x4 r, uint8_t *dst, int voff) {
  const uint32_t m = (uint32_t)(size_t)(lds_void *)dst;
  asm volatile("buffer_load_dword %0, %1, 0 offen lds" ::"v"(voff), "s"(r), "{m0}"(m) : "memory");
}

__device__ __forceinline__ void wait_copies() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Wait until at most N vector memory operations of this wave are in flight
// (s_waitcnt with the expcnt and lgkmcnt fields at their maxima).
template <int N>
__device__ __forceinline__ void wait_copies_but() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Two fp32 -> packed fp16 (round to nearest even).
__device__ __forceinline__ uint32_t pack_f16x2(float lo_half, float hi_half) {
  const float2v f = {lo_half, hi_half};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, half2v));
}

// The low and high fp16 halves of a dword, as floats.  (Reading a dword
// element of a vector through a bit cast to a half pair is avoided: the
// compiler in use then reads element 0 whatever the index.)
__device__ __forceinline__ float f16_lo(uint32_t w) { return f16_to_f32((uint16_t)(w & 0xffffu)); }
__device__ __forceinline__ float f16_hi(uint32_t w) { return f16_to_f32((uint16_t)(w >> 16)); }

// Position of column c inside its 32-column group in pair order.
__device__ __forceinline__ int pair_pos(int c) {
  return (c & ~31) + 2 * (c & 15) + ((c >> 4) & 1);
}

// Range guard of the forward's fp16 operands, per token t (one row of x).
// The layer is defined for any input (App. A.2.1), but fp16 holds only
// 2^-24 .. 65504, so both fp16 operands carry a power-of-two scale that is
// undone in fp32:
//   xp[t]  = fp16(s_in .* x[t] * 2^e_t), e_t putting the row's largest entry
//            in [2^-1, 1);
//   Z[t]   = fp16(s_mid .* (Bv xp[t]) * 2^-c_t), where L_t = sum_j |s_in_j
//            x_tj| 2^e_t bounds every |(Bv xp[t])_k| (the signs are +-1),
//            and c_t makes L_t * max|s_mid| * 2^-c_t < 1;
//   y[t]   = bf16(s_out .* (Bu Z[t]) * 2^(c_t - e_t)).
// Both operands are stored with a further exact power-of-two factor per
// column, 2^slot_exp(column mod 4) <= 2^14 (see the sign operands below), so
// every stored fp16 value stays under 2^14: each rounding to fp16 is a plain
// 2^-11 relative rounding with no overflow, whatever the magnitude of x
// (entries far below a row's largest one, under about 2^-20 of it, keep
// fewer digits, as in any fp16 rounding).  Scaling by a power of two is
// exact, so for inputs inside fp16's range the results differ from unscaled
// operands only where they would have been subnormal.  The per-token record
// is
//   tinfo[2t] = L_t (fp32),  tinfo[2t + 1] = e_t (int32 bits),
//   tinfo[2T] = max_k |s_mid_k|,
//   tinfo[2T + 4 + t] = R1_t, tinfo[3T + 4 + t] = R2_t (the row sums of
//   the two products' operands, see the sign operands below).
// `tinfo_floats(T)` floats hold it.
__host__ __device__ constexpr int64_t tinfo_floats(int64_t T) { return 4 * T + 4; }
template <typename F>
__device__ __forceinline__ F *tinfo_r1(F *tinfo, int T) { return tinfo + 2 * T + 4; }
template <typename F>
__device__ __forceinline__ F *tinfo_r2(F *tinfo, int T) { return tinfo + 3 * T + 4; }

// Sign operands of the forward products.  The MFMA's sign operand is built
// from the packed words with a rotation and a mask: a set bit (sign -1)
// becomes a single fp16 exponent bit, the value 2^-slot_exp(e) with e the
// operand register's index in its quad (bits 10 .. 13: 2^-14, 2^-13,
// 2^-11, 2^-7), a clear bit zero.  The activation operand of column j
// carries the matching factor 2^slot_exp(j mod 4) (the column's register
// index in pair order is j mod 4), so the product accumulates
// acc = sum_j a_j b_j, with a_j the activation as stored times
// 2^-slot_exp and b_j the sign bit, and the signed product is
// sum_j (1 - 2 b_j) a_j = R - 2 acc with the row sum R = sum_j a_j.  R1_t
// (the G1 operand's, from the preparation) and R2_t (the intermediate's,
// from G1's per-tile sums) are in the record above.  The mask keeps single
// exponent bits because the matrix cores multiply normal fp16 powers of two
// exactly, while single-bit subnormals lose precision.  (The backward keeps
// the +-1 operands.)
__host__ __device__ constexpr int slot_exp(int e) {
  return e == 0 ? 14 : e == 1 ? 13 : e == 2 ? 11 : 7;
}
// G1's per-tile row sums of the intermediate: RS[t][b] = sum of a_k over the
// 256 columns of tile b (the second product adds them up into R2_t), rows
// of rs_ld(r) floats.
__host__ __device__ constexpr int rs_ld(int64_t r) { return (int)((((r + 255) / 256) + 3) & ~3); }

// Exponent c_t of the intermediate's scale: 2^-c_t L_t smax' < 1, with
// smax' = max|s_mid| (1 when every s_mid is zero).  0 for an all-zero row.
__device__ __forceinline__ int mid_exp(float L, float smax) {
  const float b = L * (smax > 0.f ? smax : 1.f);
  if (!(b > 0.f) || !__builtin_isfinite(b)) return 0;
  int k;
  frexpf(b, &k);  // b = f 2^k, f in [0.5, 1): b < 2^k
  return k;
}

// Scale exponent of the training forward's saved v: smax' < 2^(es - 14)
// (so 2^(es - c_t) L_t < 2^15).
__device__ __forceinline__ int smax_exp(float smax) {
  int k;
  frexpf(smax > 0.f && __builtin_isfinite(smax) ? smax : 1.f, &k);
  return k + 14;
}

// The training forward saves V = fp16(v 2^(e_t - c_t + es)) (v = Bv (s_in
// .* x), es = smax_exp); v = V 2^shift with this shift.
__device__ __forceinline__ int saved_v_shift(const float *__restrict__ tinfo, int T, int t) {
  const float2 ti = reinterpret_cast<const float2 *>(tinfo)[t];
  return mid_exp(ti.x, tinfo[2 * T]) - smax_exp(tinfo[2 * T]) - __float_as_int(ti.y);
}

// The forward's preparation and range guard.  Each token row is prepared by
// one workgroup: x (bf16, [T][K]) and s (fp16, [K]) -> xp = fp16(x .* s
// 2^e_t) ([T][K], pair order) and the token's record.  Three steps, each
// ending in a reduction over the workgroup:
//  1. the largest |x| (bf16 magnitudes compare as integers), whose binary
//     exponent gives a first shift e1 with |x 2^e1| < 1 (so x 2^e1 s_in is
//     finite and exact for any bf16 x and fp16 s_in);
//  2. p = x 2^e1 s_in: the largest |p| and sum |p|, which give e2;
//  3. xp = fp16(p 2^(e2 + slot_exp(column mod 4))), e_t = e1 + e2, and the
//     thread's part of R1_t, the sum of the stored values over their column
//     factors (see the sign operands above), reduced with the next step 1
//     of the workgroup (or on its own after its last token).
// Rows of up to 2048 units (1024 threads, two units each) are loaded once
// and kept in registers through the three steps (prep_stream_kernel); wider
// rows are read three times (prep_kernel, the later passes hit the caches).
// One more workgroup stores max |s_mid|.  A unit is 16 columns: 8 columns
// c .. c+7 and their partners c+16 .. c+23, which become the pair dwords
// 8h .. 8h+7 of their group.
__device__ __forceinline__ void load_x_unit(const uint16_t *__restrict__ row, int c, u32x4 &lo,
                                            u32x4 &hi) {
  lo = *reinterpret_cast<const u32x4 *>(row + c);
  hi = *reinterpret_cast<const u32x4 *>(row + c + 16);
}

__device__ __forceinline__ int unit_col(int u) { return (u >> 1) * 32 + 8 * (u & 1); }

// Sum and maximum over the workgroup (fixed order: lanes by butterfly, then
// the waves in order), every thread receives both.  red holds 32 floats.
__device__ __forceinline__ void block_sum_max(float &sum, float &mx, float *red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int waves = blockDim.x >> 6;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    sum += __shfl_xor(sum, off, 64);
    mx = fmaxf(mx, __shfl_xor(mx, off, 64));
  }
  __syncthreads();  // red may still be read from a previous call
  if (lane == 0) {
    red[wave] = sum;
    red[16 + wave] = mx;
  }
  __syncthreads();
  sum = red[0];
  mx = red[16];
  for (int w = 1; w < waves; ++w) {
    sum += red[w];
    mx = fmaxf(mx, red[16 + w]);
  }
}

// The same reduction for workgroups that keep global loads in flight across
// it (the next token's prefetch): the barriers wait for LDS operations only,
// and the lanes are combined by DPP within 16-lane rows, then the four rows
// through lanes 0, 16, 32, 48 (a fixed order).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
template <int kCtrl>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), kCtrl, 0xF, 0xF, false));
}
__device__ __forceinline__ float lane_f32(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
// Sum of the 16 lanes of each DPP row, in every lane of the row.
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_f32<0xB1>(v);
  v += dpp_f32<0x4E>(v);
  v += dpp_f32<0x124>(v);
  v += dpp_f32<0x128>(v);
  return v;
}
// The sum of v over the 32 lanes of each half wave (all 64 lanes active),
// in every lane: the DPP rows of 16, then the two rows of the half.
__device__ __forceinline__ float half_wave_sum(float v) {
  const float h = row16_sum(v);
  return (threadIdx.x & 32) == 0 ? lane_f32(h, 0) + lane_f32(h, 16)
                                 : lane_f32(h, 32) + lane_f32(h, 48);
}
template <int kWaves>
__device__ __forceinline__ void block_sum_max_async(float &sum, float &mx, float *red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  sum = row16_sum(sum);
  mx = fmaxf(mx, dpp_f32<0xB1>(mx));
  mx = fmaxf(mx, dpp_f32<0x4E>(mx));
  mx = fmaxf(mx, dpp_f32<0x124>(mx));
  mx = fmaxf(mx, dpp_f32<0x128>(mx));
  sum = (lane_f32(sum, 0) + lane_f32(sum, 16)) + (lane_f32(sum, 32) + lane_f32(sum, 48));
  mx = fmaxf(fmaxf(lane_f32(mx, 0), lane_f32(mx, 16)), fmaxf(lane_f32(mx, 32), lane_f32(mx, 48)));
  lds_barrier();  // red may still be read from a previous call
  if (lane == 0) {
    red[wave] = sum;
    red[16 + wave] = mx;
  }
  lds_barrier();
  sum = red[0];
  mx = red[16];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) {
    sum += red[w];
    mx = fmaxf(mx, red[16 + w]);
  }
}

// The largest |s_mid[k]| over this thread's share of the r entries (r a
// multiple of 8, s_mid 16-byte aligned): 16-byte loads, eight in flight per
// round, so a rank of up to 64 * threads entries costs one memory round trip
// (a load per entry and iteration would wait for each in turn: r / threads
// round trips).
__device__ __forceinline__ float smid_absmax_part(const uint16_t *__restrict__ s_mid, int r,
                                                  int threads) {
  float mx = 0.f;
  for (int c0 = (int)threadIdx.x * 8; c0 < r; c0 += 64 * threads) {
    u32x4 v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int c = c0 + 8 * threads * q;
      v[q] = c < r ? *reinterpret_cast<const u32x4 *>(s_mid + c) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int q = 0; q < 8; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        mx = fmaxf(mx, fmaxf(fabsf(f16_lo(v[q][e])), fabsf(f16_hi(v[q][e]))));
  }
  return mx;
}

// Block T: max |s_mid| into tinfo[2T].
__device__ __forceinline__ void prep_smax(const uint16_t *__restrict__ s_mid, int r, int T,
                                          float *__restrict__ tinfo, float *red) {
  float sum = 0.f, mx = smid_absmax_part(s_mid, r, (int)blockDim.x);
  block_sum_max(sum, mx, red);
  if (threadIdx.x == 0) tinfo[2 * T] = mx;
}

// e1 from the row's largest bf16 magnitude pattern: |x 2^e1| < 1.
__device__ __forceinline__ int prep_e1(uint32_t mb) {
  const float xmax = bf16_to_f32(mb);
  int e1 = 0;
  if (xmax > 0.f && __builtin_isfinite(xmax)) {
    frexpf(xmax, &e1);  // xmax < 2^e1
    e1 = -e1;
  }
  return e1;
}

// e2 from the largest |p|: pmax 2^e2 in [2^-1, 1).
__device__ __forceinline__ int prep_e2(float pmax) {
  int e2 = 0;
  if (pmax > 0.f && __builtin_isfinite(pmax)) {
    frexpf(pmax, &e2);  // pmax = f 2^k, f in [0.5, 1)
    e2 = -e2;
  }
  return e2;
}

// Pair-order dwords of one unit from its 16 values (v[d] = column c + d,
// v[8 + d] = column c + 16 + d, c a multiple of 8, so both have the column
// factor of d mod 4), stored at the unit's place in xp; returns the sum of
// the stored values over their column factors.
__device__ __forceinline__ float prep_store(uint16_t *__restrict__ xp, int t, int K, int c,
                                            const float (&v)[16], int e2) {
  uint32_t d[8];
  float r1 = 0.f;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int sc = e2 + slot_exp(k & 3);
    d[k] = pack_f16x2(ldexpf(v[k], sc), ldexpf(v[8 + k], sc));
    const _Float16 f = (_Float16)(1.0f / (float)(1 << slot_exp(k & 3)));  // exact
    r1 = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2v, d[k]), half2v{f, f}, r1, false);
  }
  uint4 *dst = reinterpret_cast<uint4 *>(xp + (size_t)t * K + (c & ~31) + 2 * (c & 15));
  dst[0] = make_uint4(d[0], d[1], d[2], d[3]);
  dst[1] = make_uint4(d[4], d[5], d[6], d[7]);
  return r1;
}

// p values of one unit: x 2^e1 s_in, v[d] = column c + d, v[8 + d] = c + 16 + d.
__device__ __forceinline__ void prep_values(const u32x4 &lo, const u32x4 &hi, const u32x4 &slo,
                                            const u32x4 &shi, int e1, float (&v)[16]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[2 * e] = ldexpf(__uint_as_float(lo[e] << 16), e1) * f16_lo(slo[e]);
    v[2 * e + 1] = ldexpf(__uint_as_float(lo[e] & 0xffff0000u), e1) * f16_hi(slo[e]);
    v[8 + 2 * e] = ldexpf(__uint_as_float(hi[e] << 16), e1) * f16_lo(shi[e]);
    v[8 + 2 * e + 1] = ldexpf(__uint_as_float(hi[e] & 0xffff0000u), e1) * f16_hi(shi[e]);
  }
}

__device__ __forceinline__ uint32_t unit_maxbits(const u32x4 &lo, const u32x4 &hi) {
  uint32_t mb = 0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    mb = max(mb, max(lo[e] & 0x7fffu, (lo[e] >> 16) & 0x7fffu));
    mb = max(mb, max(hi[e] & 0x7fffu, (hi[e] >> 16) & 0x7fffu));
  }
  return mb;
}

// Any row width: three passes over the row, one token a workgroup.
__global__ __launch_bounds__(256) void prep_kernel(
    const uint16_t *__restrict__ x, const uint16_t *__restrict__ s_in,
    uint16_t *__restrict__ xp, int T, int K, float *__restrict__ tinfo,
    const uint16_t *__restrict__ s_mid, int r) {
  __shared__ float red[32];
  const int t = blockIdx.x;
  if (t == T) {
    prep_smax(s_mid, r, T, tinfo, red);
    return;
  }
  const int units = K / 16;
  const uint16_t *row = x + (size_t)t * K;
  uint32_t mb = 0;
  for (int u = threadIdx.x; u < units; u += 256) {
    u32x4 lo, hi;
    load_x_unit(row, unit_col(u), lo, hi);
    mb = max(mb, unit_maxbits(lo, hi));
  }
  float sum = 0.f, mx = __uint_as_float(mb);  // a non-negative pattern orders as its value
  block_sum_max(sum, mx, red);
  const int e1 = prep_e1(__float_as_uint(mx));
  float l1 = 0.f, pmax = 0.f;
  for (int u = threadIdx.x; u < units; u += 256) {
    const int c = unit_col(u);
    u32x4 lo, hi;
    load_x_unit(row, c, lo, hi);
    float v[16];
    prep_values(lo, hi, *reinterpret_cast<const u32x4 *>(s_in + c),
                *reinterpret_cast<const u32x4 *>(s_in + c + 16), e1, v);
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      pmax = fmaxf(pmax, fabsf(v[k]));
      l1 += fabsf(v[k]);
    }
  }
  block_sum_max(l1, pmax, red);
  const int e2 = prep_e2(pmax);
  float r1 = 0.f, unused = 0.f;
  for (int u = threadIdx.x; u < units; u += 256) {
    const int c = unit_col(u);
    u32x4 lo, hi;
    load_x_unit(row, c, lo, hi);
    float v[16];
    prep_values(lo, hi, *reinterpret_cast<const u32x4 *>(s_in + c),
                *reinterpret_cast<const u32x4 *>(s_in + c + 16), e1, v);
    r1 += prep_store(xp, t, K, c, v, e2);
  }
  block_sum_max(r1, unused, red);
  if (threadIdx.x == 0) {
    reinterpret_cast<float2 *>(tinfo)[t] = make_float2(ldexpf(l1, e2), __int_as_float(e1 + e2));
    tinfo_r1(tinfo, T)[t] = r1;
  }
}

// The same preparation for rows of up to kU * kThreads units, persistent:
// workgroup w < W takes tokens w, w + W, w + 2W, ... and loads the next
// token's row while it reduces and stores the current one, so the row loads
// and the xp stores of different tokens overlap.  s_in is loaded once.  The
// two row buffers alternate in a loop unrolled by two (the first pair
// peeled, so the loop is entered with the same memory operations in flight
// as it is repeated with); a thread whose unit index passes the row's end
// holds a copy of the row's last unit, kept out of the reductions and
// stored back unchanged, so that no load or store sits in a branch.  The
// arithmetic and the order of each token's results are those of
// prep_kernel except the order in which the reductions add.  Workgroup W
// stores max |s_mid|.
template <int kU>
struct PrepRow {
  u32x4 lo[kU], hi[kU];
};

template <int kU, int kThreads>
__device__ __forceinline__ void prep_row_load(const uint16_t *__restrict__ x, int t, int K,
                                              int units, PrepRow<kU> &b) {
  const uint16_t *row = x + (size_t)t * K;
#pragma unroll
  for (int i = 0; i < kU; ++i)
    load_x_unit(row, unit_col(min((int)threadIdx.x + kThreads * i, units - 1)), b.lo[i], b.hi[i]);
}

// carry: in, this thread's part of the previous token tp's R1 (tp < 0:
// none), added up in the first reduction and stored; out, the part of this
// token's.
template <int kU, int kThreads>
__device__ __forceinline__ void prep_row_token(const PrepRow<kU> &b, const u32x4 (&sl)[kU],
                                               const u32x4 (&sh)[kU], uint16_t *__restrict__ xp,
                                               float *__restrict__ tinfo, int t, int T,
                                               int K, int units, float *red, float &carry,
                                               int tp) {
  uint32_t mb = 0;
#pragma unroll
  for (int i = 0; i < kU; ++i) {
    const uint32_t m = unit_maxbits(b.lo[i], b.hi[i]);
    mb = max(mb, (int)threadIdx.x + kThreads * i < units ? m : 0u);
  }
  float mx = __uint_as_float(mb);
  block_sum_max_async<kThreads / 64>(carry, mx, red);
  if (tp >= 0) tinfo_r1(tinfo, T)[tp] = carry;  // the same value in every lane
  const int e1 = prep_e1(__float_as_uint(mx));
  float v[kU][16], l1 = 0.f, pmax = 0.f;
#pragma unroll
  for (int i = 0; i < kU; ++i) {
    prep_values(b.lo[i], b.hi[i], sl[i], sh[i], e1, v[i]);
    const float keep = (int)threadIdx.x + kThreads * i < units ? 1.f : 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      pmax = fmaxf(pmax, keep * fabsf(v[i][k]));
      l1 += keep * fabsf(v[i][k]);
    }
  }
  block_sum_max_async<kThreads / 64>(l1, pmax, red);
  const int e2 = prep_e2(pmax);
  carry = 0.f;
#pragma unroll
  for (int i = 0; i < kU; ++i) {
    const float r1 = prep_store(xp, t, K, unit_col(min((int)threadIdx.x + kThreads * i, units - 1)),
                                v[i], e2);
    carry += (int)threadIdx.x + kThreads * i < units ? r1 : 0.f;
  }
  // every lane stores the token's record (the same value, one write a wave)
  reinterpret_cast<float2 *>(tinfo)[t] = make_float2(ldexpf(l1, e2), __int_as_float(e1 + e2));
}

// The last token's R1 (see prep_row_token).
template <int kThreads>
__device__ __forceinline__ void prep_r1_flush(float *__restrict__ tinfo, int T, int tp,
                                              float carry, float *red) {
  float unused = 0.f;
  block_sum_max_async<kThreads / 64>(carry, unused, red);
  tinfo_r1(tinfo, T)[tp] = carry;
}

template <int kU, int kThreads>
__global__ __launch_bounds__(kThreads) void prep_stream_kernel(
    const uint16_t *__restrict__ x, const uint16_t *__restrict__ s_in,
    uint16_t *__restrict__ xp, int T, int K, float *__restrict__ tinfo,
    const uint16_t *__restrict__ s_mid, int r) {
  __shared__ float red[32];
  const int W = (int)gridDim.x - 1;
  if ((int)blockIdx.x == W) {
    prep_smax(s_mid, r, T, tinfo, red);
    return;
  }
  const int units = K / 16;
  u32x4 sl[kU], sh[kU];
#pragma unroll
  for (int i = 0; i < kU; ++i) {
    const int c = unit_col(min((int)threadIdx.x + kThreads * i, units - 1));
    sl[i] = *reinterpret_cast<const u32x4 *>(s_in + c);
    sh[i] = *reinterpret_cast<const u32x4 *>(s_in + c + 16);
  }
  PrepRow<kU> a, b;
  float carry = 0.f;  // R1 part of the last token prepared
  int t = blockIdx.x;  // < T: the grid has at most T workers
  prep_row_load<kU, kThreads>(x, t, K, units, a);
  prep_row_load<kU, kThreads>(x, min(t + W, T - 1), K, units, b);
  prep_row_token<kU, kThreads>(a, sl, sh, xp, tinfo, t, T, K, units, red, carry, -1);
  t += W;
  if (t >= T) {
    prep_r1_flush<kThreads>(tinfo, T, t - W, carry, red);
    return;
  }
  prep_row_load<kU, kThreads>(x, min(t + W, T - 1), K, units, a);
  prep_row_token<kU, kThreads>(b, sl, sh, xp, tinfo, t, T, K, units, red, carry, t - W);
  for (t += W; t < T; t += 2 * W) {
    prep_row_load<kU, kThreads>(x, min(t + W, T - 1), K, units, b);
    prep_row_token<kU, kThreads>(a, sl, sh, xp, tinfo, t, T, K, units, red, carry, t - W);
    if (t + W >= T) {
      prep_r1_flush<kThreads>(tinfo, T, t, carry, red);
      return;
    }
    prep_row_load<kU, kThreads>(x, min(t + 2 * W, T - 1), K, units, a);
    prep_row_token<kU, kThreads>(b, sl, sh, xp, tinfo, t + W, T, K, units, red, carry, t);
  }
  // the loop ended after a token pair: t - W was prepared last
  prep_r1_flush<kThreads>(tinfo, T, t - W, carry, red);
}

// C = rowscale * (A_pairorder x sign(W)^T), in the forms listed under Mode.
template <int kMode, int kBM, int kStages>
__global__ __launch_bounds__(kThreads, 2) void bingemm_kernel(
    const uint16_t *__restrict__ A, int T, int K, const uint32_t *__restrict__ W, int N,
    const uint16_t *__restrict__ rowscale, uint16_t *__restrict__ C, uint16_t *__restrict__ V,
    const uint16_t *__restrict__ S, float *__restrict__ F, const float *__restrict__ gscale,
    int split_steps, float *__restrict__ P, int mix_full, int mix_splits, int mix_nN,
    float *__restrict__ tinfo, float *__restrict__ RS) {
  constexpr bool kPairOut = kMode == kMid || kMode == kMidSave || kMode == kBwdMid;
  constexpr bool kBwd = kMode == kBwdMid || kMode == kBwdIn;
  constexpr bool kFirst = kMode == kMid || kMode == kMidSave;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  using LM = Lds<kBM, kStages>;
  static_assert(kStages == 2 || kStages == 3, "pipeline depth");
  constexpr int kA0 = LM::kA0, kW0 = LM::kW0, kATile = LM::kATileT;
  constexpr int kLdsBytes = LM::kBytes;
  constexpr int kTokBlocks = kBM / 32;          // 32-token MFMA blocks per wave
  constexpr int kACopies = kBM * kARow / 1024 / 4;  // 1 KiB copies per wave per step
  // Copy instructions per wave per step (the same in every wave, so one
  // s_waitcnt leaves exactly the newest step's copies in flight).
  constexpr int kCopiesPerStep = kACopies + 4;

  const int kw = K / 32;                       // sign words per row
  const int nk_row = (kw + kWords - 1) / kWords;  // the last step may be partial
  // Tile and K steps of this workgroup.
  //  Plain grid: consecutive workgroups land on consecutive XCDs; each XCD
  //  takes a contiguous range of tiles (weight-row tiles fastest); all K
  //  steps, or with a split K (grid z > 1) the range of split blockIdx.z.
  //  Mixed grid (mix_full > 0, forward modes, 1-D): workgroups below
  //  mix_full take whole tiles (one per compute unit: workgroups are placed
  //  one per unit before any unit gets a second), each remaining tile is cut
  //  into mix_splits K ranges written as partials (pslot).
  int nN, L, k0, nk, pslot = -1;
  if (mix_full > 0) {
    nN = mix_nN;
    const int bid = (int)blockIdx.x;
    if (bid < mix_full) {
      L = bid;
      if ((mix_full & 7) == 0) L = (L & 7) * (mix_full >> 3) + (L >> 3);
      k0 = 0;
      nk = nk_row;
    } else {
      pslot = bid - mix_full;
      const int cut = (int)gridDim.x - mix_full;
      if ((cut & 7) == 0) pslot = (pslot & 7) * (cut >> 3) + (pslot >> 3);
      const int h = pslot / mix_splits;
      L = mix_full + h;
      k0 = (pslot - h * mix_splits) * split_steps;
      nk = min(nk_row, k0 + split_steps);
    }
  } else {
    nN = gridDim.x;
    const int total = nN * gridDim.y;
    L = blockIdx.y * nN + blockIdx.x;
    if ((total & 7) == 0) L = (L & 7) * (total >> 3) + (L >> 3);
    k0 = gridDim.z > 1 ? (int)blockIdx.z * split_steps : 0;
    nk = gridDim.z > 1 ? min(nk_row, k0 + split_steps) : nk_row;
  }
  const int t0 = (L / nN) * kBM;
  const int n0 = (L % nN) * BN;

  // Copy roles, fixed per lane (a step only moves the resources' bases).
  //  Activations: wave w issues copies j = kACopies*w + jj, each covering
  //  token rows 4j .. 4j+3 of the tile; lane l fills chunk position l mod 16
  //  of row 4j + l/16 with the chunk whose index is that position XOR the
  //  row's low four bits.  Columns past K read the next row or zeros; they
  //  meet zero B operands (sign words past the row end).
  int a_off[kACopies];
#pragma unroll
  for (int jj = 0; jj < kACopies; ++jj) {
    const int tok = 4 * (kACopies * wave + jj) + (lane >> 4);
    const int part = (lane & 15) ^ (tok & 15);
    a_off[jj] = t0 + tok < T ? (t0 + tok) * K * 2 + 16 * part : kOob;
  }
  //  Sign words: copy i of wave w covers tile rows 64w + 16i .. +15, four
  //  words (16 bytes) per row.
  int w_off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = n0 + 64 * wave + 16 * i + (lane >> 2);
    w_off[i] = row < N ? row * kw * 4 + 4 * (lane & 3) : kOob;
  }

  auto issue = [&](int step, int buf) {
    const i32x4 as = copy_rsrc(A + step * BK, (int64_t)T * K * 2 - (int64_t)step * BK * 2);
    const i32x4 ws = copy_rsrc(W + step * kWords, (int64_t)N * kw * 4 - (int64_t)step * kWords * 4);
#pragma unroll
    for (int jj = 0; jj < kACopies; ++jj)
      copy16(as, lds + kA0 + buf * kATile + (kACopies * wave + jj) * 1024, a_off[jj]);
#pragma unroll
    for (int i = 0; i < 4; ++i) copy4(ws, lds + kW0 + buf * kWTile + (64 * wave + 16 * i) * 16, w_off[i]);
  };

  // No stale LDS pattern (possibly a NaN) may ever meet an MFMA, even in
  // rows or columns that are never stored.
  for (int o = tid * 16; o < kLdsBytes; o += kThreads * 16)
    *reinterpret_cast<uint4 *>(lds + o) = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  issue(k0, 0);
  if (kStages == 3 && k0 + 1 < nk) issue(k0 + 1, 1);
  // The forward's per-token tables, loaded while the first copies travel:
  // the range-guard shift of the output (see prep_stream_kernel; the first
  // product's accumulator is scaled by 2^-c_t, the second's by 2^(c_t - e_t),
  // which leaves the unscaled value) and the operand's row sum R (R1 from the preparation for the first product; for
  // the second, R2 added up from G1's per-tile sums in tile order, which the
  // workgroups of the first column tile and K range also store in the
  // record for the split and mixed reductions).
  int tab_sh = 0;
  float tab_r = 0.f;
  if constexpr (!kBwd) {
    const int q = tid < kBM ? tid : kBM - 1;
    const int t = min(t0 + q, T - 1);
    const float2 ti = reinterpret_cast<const float2 *>(tinfo)[t];
    const float smax = tinfo[2 * T];
    if constexpr (kFirst) {
      tab_r = tinfo_r1(tinfo, T)[t];
    } else {
      const int nb = (K + 255) / 256, ld = rs_ld(K);
      const float4 *rr = reinterpret_cast<const float4 *>(RS + (size_t)t * ld);
      for (int b0 = 0; b0 < nb; b0 += 16) {
        float4 v[4];
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) v[q4] = rr[min(b0 / 4 + q4, ld / 4 - 1)];
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int b = b0 + 4 * q4;
          tab_r += b < nb ? v[q4].x : 0.f;
          tab_r += b + 1 < nb ? v[q4].y : 0.f;
          tab_r += b + 2 < nb ? v[q4].z : 0.f;
          tab_r += b + 3 < nb ? v[q4].w : 0.f;
        }
      }
      if (L % nN == 0 && k0 == 0 && tid < kBM && t0 + q < T) tinfo_r2(tinfo, T)[t] = tab_r;
    }
    const int c = mid_exp(ti.x, smax);
    tab_sh = kFirst ? -c : c - __float_as_int(ti.y);
    if (t0 + q >= T) {
      tab_sh = 0;
      tab_r = 0.f;
    }
  }

  // This lane's weight rows: block j -> tile row 64*wave + 32*j + (l mod 32).
  const int wrow_l = 64 * wave + (lane & 31);
  const int wrow0 = n0 + wrow_l;
  const int g = lane >> 5;  // K half of an MFMA operand (slots 8g .. 8g+7)
  // Activation operand of MFMA step ks (columns 16ks .. 16ks+15 of the K
  // step): chunk 2ks + g of token row (l mod 32) + 32i, swizzled.
  int a_rd[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) a_rd[ks] = (lane & 31) * kARow + (((2 * ks + g) ^ (lane & 15)) << 4);
  // Shift that moves sign bit p = 8s + 4g + e of a word to bit 15 (the
  // backward's +-1 operands); the forward's rotation right that moves bits
  // 8s + 4g .. 8s + 4g + 3 (and the same 16 higher) to bits 10 .. 13 (and
  // 26 .. 29).
  int sh[2][4];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int e = 0; e < 4; ++e) sh[s][e] = 15 - (8 * s + 4 * g + e);
  const uint32_t rot[2] = {(uint32_t)(4 * g - 10) & 31u, (uint32_t)(8 + 4 * g - 10) & 31u};

  floatx16 acc[kTokBlocks][2];
#pragma unroll
  for (int i = 0; i < kTokBlocks; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  uint32_t kSignMask;
  asm volatile("v_mov_b32 %0, 0x80008000" : "=v"(kSignMask));
  constexpr uint32_t kOnePair = 0x3c003c00u;  // fp16 +1, +1

  if (kStages == 3 && k0 + 1 < nk)
    wait_copies_but<kCopiesPerStep>();
  else
    wait_copies();
  if constexpr (!kBwd) {
    if (tid < kBM) {
      reinterpret_cast<int *>(lds + LM::kTab)[tid] = tab_sh;
      reinterpret_cast<float *>(lds + LM::kTab + 4 * kBM)[tid] = tab_r;
    }
  }
  __syncthreads();

  auto run_step = [&](int step, auto BUF) {
    constexpr int buf = decltype(BUF)::value;
    if constexpr (kStages == 2) {
      if (step + 1 < nk) issue(step + 1, buf ^ 1);
    } else {
      // the buffer of step + 2 held step - 1, which every wave finished
      // before the last barrier
      if (step + 2 < nk) issue(step + 2, (buf + 2) % 3);
    }
    const uint8_t *abase = lds + kA0 + buf * kATile;
    const uint4 *wt = reinterpret_cast<const uint4 *>(lds + kW0 + buf * kWTile);
    const uint4 wq0 = wt[wrow_l], wq1 = wt[wrow_l + 32];
    const uint32_t wj[2][kWords] = {{wq0.x, wq0.y, wq0.z, wq0.w}, {wq1.x, wq1.y, wq1.z, wq1.w}};
    half8 af[2][kTokBlocks];
    auto read_ops = [&](int ks, int slot) {
#pragma unroll
      for (int i = 0; i < kTokBlocks; ++i)
        af[slot][i] = *reinterpret_cast<const half8 *>(abase + a_rd[ks] + 32 * i * kARow);
    };
    // Sign operand of MFMA step ks for weight-row block j.  Forward: the
    // word rotated so that register e's two sign bits sit on bits 10 + e and
    // 26 + e, masked to them (fp16 2^-slot_exp(e) or 0 in each half).
    // Backward: the fp16 pair (+1, +1) XOR the sign bits moved to bits 15
    // and 31.  Words past the row end (a partial last K step) meet zeros.
    auto expand = [&](int ks, int j) {
      const bool live = step * kWords + (ks >> 1) < kw;
      const uint32_t w = wj[j][ks >> 1];
      uint32_t bd[4];
      if constexpr (kBwd) {
        const uint32_t one = live ? kOnePair : 0u;
#pragma unroll
        for (int e = 0; e < 4; ++e) bd[e] = one ^ ((w << sh[ks & 1][e]) & kSignMask);
      } else {
        const uint32_t wr = __builtin_amdgcn_alignbit(w, w, rot[ks & 1]);
#pragma unroll
        for (int e = 0; e < 4; ++e) bd[e] = wr & (live ? 0x04000400u << e : 0u);
      }
      return make_uint4(bd[0], bd[1], bd[2], bd[3]);
    };
    // Each group of MFMAs uses sign operands expanded one group earlier, and
    // the next step's LDS reads are issued ahead too; the scheduling
    // barriers keep that order, so no MFMA waits on the instructions just
    // before it.  128-token tiles: both blocks' operands of step ks are
    // ready before its first MFMA, those of ks + 1 are expanded between its
    // two halves, and the MFMAs go token block by token block, so each
    // activation operand meets both sign operands back to back (0.3-1.7%
    // faster than block by block under the power limit; slower with
    // 64-token tiles).  64-token tiles: block 1's operand of step ks is
    // expanded while block 0's MFMAs of ks run, block 0's of ks + 1 while
    // block 1's run.
    auto mfma = [&](int i, int j, int slot, const uint4 &b) {
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(
          af[slot][i], __builtin_bit_cast(half8, b), acc[i][j], 0, 0, 0);
    };
    read_ops(0, 0);
    if constexpr (kTokBlocks == 4) {
      uint4 b0 = expand(0, 0), b1 = expand(0, 1), n0, n1;
      static_for<2 * kWords>([&](auto KS) {
        constexpr int ks = decltype(KS)::value;
        constexpr int cur = ks & 1;
        if constexpr (ks + 1 < 2 * kWords) read_ops(ks + 1, cur ^ 1);
        __builtin_amdgcn_sched_barrier(0);
        mfma(0, 0, cur, b0);
        mfma(0, 1, cur, b1);
        mfma(1, 0, cur, b0);
        mfma(1, 1, cur, b1);
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (ks + 1 < 2 * kWords) {
          n0 = expand(ks + 1, 0);
          n1 = expand(ks + 1, 1);
        }
        __builtin_amdgcn_sched_barrier(0);
        mfma(2, 0, cur, b0);
        mfma(2, 1, cur, b1);
        mfma(3, 0, cur, b0);
        mfma(3, 1, cur, b1);
        if constexpr (ks + 1 < 2 * kWords) {
          b0 = n0;
          b1 = n1;
        }
      });
    } else {
      uint4 b0 = expand(0, 0), b1;
      static_for<2 * kWords>([&](auto KS) {
        constexpr int ks = decltype(KS)::value;
        constexpr int cur = ks & 1;
        if constexpr (ks + 1 < 2 * kWords) read_ops(ks + 1, cur ^ 1);
        b1 = expand(ks, 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < kTokBlocks; ++i) mfma(i, 0, cur, b0);
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (ks + 1 < 2 * kWords) b0 = expand(ks + 1, 0);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < kTokBlocks; ++i) mfma(i, 1, cur, b1);
      });
    }
    // the next step's copies must have landed; with three stages the
    // copies of the step after it may stay in flight
    if (kStages == 3 && step + 2 < nk)
      wait_copies_but<kCopiesPerStep>();
    else
      wait_copies();
    __syncthreads();
  };

  if constexpr (kStages == 2) {
    for (int step = k0; step < nk; step += 2) {
      run_step(step, std::integral_constant<int, 0>{});
      if (step + 1 < nk) run_step(step + 1, std::integral_constant<int, 1>{});
    }
  } else {
    for (int step = k0; step < nk; step += 3) {
      run_step(step, std::integral_constant<int, 0>{});
      if (step + 1 < nk) run_step(step + 1, std::integral_constant<int, 1>{});
      if (step + 2 < nk) run_step(step + 2, std::integral_constant<int, 2>{});
    }
  }

  // Epilogue.  32x32 accumulator layout: lane l holds column (l mod 32) and
  // rows 8*(e/4) + 4*(l/32) + (e mod 4), e = 0..15.
  if constexpr (!kBwd) {
    if (pslot >= 0) {
      // Mixed grid: the fp32 partial of this tile over the workgroup's K
      // range, tile-local [token][column], for mixed_reduce_kernel.
      float *__restrict__ Pt = P + (size_t)pslot * (kBM * BN);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int nl = wrow_l + 32 * j;
#pragma unroll
        for (int i = 0; i < kTokBlocks; ++i)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            Pt[(32 * i + 8 * (e >> 2) + 4 * g + (e & 3)) * BN + nl] = acc[i][j][e];
      }
      return;
    }
  }
  // The forward's per-token tables (filled in the prologue, past every
  // staging area below): the 16 range-guard shifts and row sums of token
  // block i for this lane's rows 8(e/4) + 4(l/32) + (e mod 4).  A forward
  // output is (R - 2 acc) 2^shift (see the sign operands).
  constexpr int kRowF = 128 + 4;  // floats per staged fp32 token row
  static_assert(kBM * kRowF * 4 <= LM::kTab && kBM * 512 <= LM::kTab, "staging clear of the tables");
  auto load_tabs = [&](int i, int (&sv)[16], float (&rv)[16]) {
    const int *shl = reinterpret_cast<const int *>(lds + LM::kTab);
    const float *rtl = reinterpret_cast<const float *>(lds + LM::kTab + 4 * kBM);
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4) {
      const int4 s4 = *reinterpret_cast<const int4 *>(shl + 32 * i + 8 * e4 + 4 * g);
      const float4 r4 = *reinterpret_cast<const float4 *>(rtl + 32 * i + 8 * e4 + 4 * g);
      sv[4 * e4] = s4.x;
      sv[4 * e4 + 1] = s4.y;
      sv[4 * e4 + 2] = s4.z;
      sv[4 * e4 + 3] = s4.w;
      rv[4 * e4] = r4.x;
      rv[4 * e4 + 1] = r4.y;
      rv[4 * e4 + 2] = r4.z;
      rv[4 * e4 + 3] = r4.w;
    }
  };
  // A fp32 [T][N] output of the whole tile (a split partial, or the saved
  // pre-scale output z): each half of the tile's columns (the j-th 32 of
  // every wave's 64) is transposed through the idle LDS buffers and leaves
  // in 16-byte stores along the columns.  Stored from the accumulator
  // layout (one column per lane) it took 64-128 single-float stores a lane,
  // whose issue alone cost about 2 us per workgroup.  The LDS buffers must
  // be idle on entry.  shifted: the forward output (R - 2 acc) 2^shift (the
  // saved z) or the raw accumulator (a split partial, finished by its
  // reduction).
  auto store_f32_tile = [&](float *__restrict__ dst, auto shifted) {
    constexpr bool kShift = decltype(shifted)::value;
    float *stg = reinterpret_cast<float *>(lds);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (j > 0) __syncthreads();  // the previous half has been read
#pragma unroll
      for (int i = 0; i < kTokBlocks; ++i) {
        int sv[16] = {};
        float rv[16] = {};
        if constexpr (kShift) load_tabs(i, sv, rv);
#pragma unroll
        for (int e = 0; e < 16; ++e)
          stg[(32 * i + 8 * (e >> 2) + 4 * g + (e & 3)) * kRowF + 32 * wave + (lane & 31)] =
              kShift ? ldexpf(fmaf(-2.f, acc[i][j][e], rv[e]), sv[e]) : acc[i][j][e];
      }
      __syncthreads();
#pragma unroll
      for (int q = 0; q < kBM * 32 / kThreads; ++q) {
        const int idx = q * kThreads + tid;
        const int row = idx >> 5, c4 = idx & 31;  // token row, float4 of the half
        const int n = n0 + 64 * (c4 >> 3) + 32 * j + 4 * (c4 & 7);
        if (t0 + row < T && n < N)
          *reinterpret_cast<float4 *>(dst + (size_t)(t0 + row) * N + n) =
              *reinterpret_cast<const float4 *>(stg + row * kRowF + 4 * c4);
      }
    }
  };
  // (a split K only occurs with 64-token tiles: a grid of 128-token tiles
  // that leaves compute units idle switches to 64-token tiles first, and
  // the 128-token kernels carry no second epilogue)
  if constexpr (kBM == 64) {
    if (gridDim.z > 1) {
      // Split K: the fp32 partial of this tile over the workgroup's K steps,
      // natural column order; the reduction kernel adds the partials and
      // applies the mode's epilogue.
      store_f32_tile(P + (size_t)blockIdx.z * T * N, std::false_type{});
      return;
    }
  }
  // A 16-bit output tile (kBM tokens x 256 columns, 512 bytes a token) is
  // assembled in the idle activation buffers and leaves in 16-byte stores,
  // 512 contiguous bytes per token row; a token row's 16-byte chunk c sits
  // at position c XOR 4 * ((row / 4) mod 2), so that the two lane halves
  // (tokens four apart) write distinct banks.  kMidSave
  // passes its second output V through the same buffer after C.
  // rs: the row scale of the lane's column in each block; the first
  // product's fp16 output also takes the column factor 2^slot_exp(n mod 4)
  // of the second product's operand (n mod 4 = l mod 4).
  float rs[2];
  int cpos[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int n = wrow0 + 32 * j;
    rs[j] = n < N ? (rowscale ? f16_to_f32(rowscale[n]) : 1.0f) : 0.f;
    if constexpr (kFirst) rs[j] = ldexpf(rs[j], slot_exp(lane & 3));
    cpos[j] = (kPairOut ? pair_pos(n) : n) - n0;
  }
  auto stage_tile = [&](auto value) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int cbyte = 2 * (cpos[j] & 7), chunk = (cpos[j] >> 3) ^ (4 * g);
#pragma unroll
      for (int i = 0; i < kTokBlocks; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = 32 * i + 8 * (e >> 2) + 4 * g + (e & 3);
          *reinterpret_cast<uint16_t *>(lds + row * 512 + chunk * 16 + cbyte) = value(i, j, e);
        }
    }
    __syncthreads();
  };
  // store_tile(dst, sums): with sums, also the first product's per-tile row
  // sums of a_k (the stored fp16 value over its column factor; dword e of a
  // chunk holds columns with factor index e) into RS, a token row's 32
  // chunks being the 32 lanes of a half wave.
  auto store_tile = [&](uint16_t *__restrict__ dst, auto sums) {
    constexpr bool kSums = decltype(sums)::value;
    const int chunk = tid & 31;
    const bool col_ok = n0 + 8 * chunk < N;
#pragma unroll 4
    for (int it = 0; it < kBM / (kThreads / 32); ++it) {
      const int row = (tid >> 5) + it * (kThreads / 32);
      const uint4 v = *reinterpret_cast<const uint4 *>(lds + row * 512 +
                                                       ((chunk ^ (4 * ((row >> 2) & 1))) << 4));
      if (col_ok && t0 + row < T)
        *reinterpret_cast<uint4 *>(dst + (size_t)(t0 + row) * N + n0 + 8 * chunk) = v;
      if constexpr (kSums) {
        const uint32_t d[4] = {v.x, v.y, v.z, v.w};
        float a = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const _Float16 f = (_Float16)(1.0f / (float)(1 << slot_exp(e)));  // exact
          a = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2v, d[e]), half2v{f, f}, a, false);
        }
        const float rsum = half_wave_sum(a);
        if (chunk == 0 && t0 + row < T) RS[(size_t)(t0 + row) * rs_ld(N) + n0 / BN] = rsum;
      }
    }
  };
  if constexpr (kBwd) {
    // The S block of this tile (kBM tokens x 256 weight rows, 512 bytes a
    // token) goes into the idle activation buffers with LDS copies, two
    // token rows per copy instruction; a row's 16-byte chunk c lands at
    // position c XOR 4 * ((row / 4) mod 2), so the two lane halves below
    // (tokens four apart) read distinct banks.  Tokens past T read zeros.
    constexpr int kSCopies = kBM / 8;  // per wave
    const i32x4 srs = copy_rsrc(S, (int64_t)T * N * 2);
#pragma unroll
    for (int jj = 0; jj < kSCopies; ++jj) {
      const int row = 2 * (kSCopies * wave + jj) + (lane >> 5);
      const int chunk = (lane & 31) ^ (((row >> 2) & 1) << 2);
      const int off = t0 + row < T ? (t0 + row) * N * 2 + n0 * 2 + 16 * chunk : kOob;
      copy16(srs, lds + (kSCopies * wave + jj) * 1024, off);
    }
    // kBwdMid: S is the saved intermediate, stored with the forward's
    // per-token scale; vsl holds each token's shift back to v (idle sign
    // buffers).
    int *vsl = reinterpret_cast<int *>(lds + kW0);
    if constexpr (kMode == kBwdMid) {
      for (int q = tid; q < kBM; q += kThreads) vsl[q] = t0 + q < T ? saved_v_shift(tinfo, T, t0 + q) : 0;
    }
    wait_copies();
    __syncthreads();
    // The 32-token block i lies in 64-token group (t0 + 32 i) / 64; its
    // factors are uniform over the wave (zero past T).
    float fg[kTokBlocks], fz[kTokBlocks];
#pragma unroll
    for (int i = 0; i < kTokBlocks; ++i) {
      const int tb = t0 + 32 * i;
      const float2 gs = tb < T ? reinterpret_cast<const float2 *>(gscale)[tb >> 6]
                               : make_float2(0.f, 1.f);
      fg[i] = kMode == kBwdMid ? gs.x : gs.x / gs.y;
      fz[i] = gs.y;
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int n = wrow0 + 32 * j;
      // Token sum of gradient * S for weight row n: the lane's sixteen
      // tokens per block, then its partner half (lane XOR 32).  Tokens past
      // T have zero accumulators and zero S.
      const int lpos = (kMode == kBwdMid ? pair_pos(n) : n) - n0;
      const int cbyte = 2 * (lpos & 7);
      float part = 0.f;
#pragma unroll
      for (int i = 0; i < kTokBlocks; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = 32 * i + 8 * (e >> 2) + 4 * g + (e & 3);
          const int pos = ((lpos >> 3) ^ (((row >> 2) & 1) << 2)) * 16 + cbyte;
          const uint16_t sv = *reinterpret_cast<const uint16_t *>(lds + row * 512 + pos);
          if constexpr (kMode == kBwdMid)
            part += ldexpf(acc[i][j][e] * fg[i] * f16_to_f32(sv), vsl[row]);
          else
            part += acc[i][j][e] * fg[i] * bf16_to_f32(sv);
        }
      part += __shfl_xor(part, 32, 64);
      if (g == 0 && n < N) F[(size_t)(t0 / kBM) * N + n] = part;
    }
    if (C) {  // uniform: dx may be skipped
      __syncthreads();  // every wave is done with the S block
      stage_tile([&](int i, int j, int e) {
        if constexpr (kMode == kBwdMid) return f32_to_f16(acc[i][j][e] * rs[j] * fz[i]);
        else return f32_to_bf16(acc[i][j][e] * fg[i] * rs[j]);
      });
      store_tile(C, std::false_type{});
    }
    return;
  }
  // stage_tile of the forward output: value(v, j) of v = (R - 2 acc) 2^shift,
  // a token block at a time (its tables read once for both column blocks).
  // The shifts are applied to each value on its way into the staging
  // (before any rounding), never to the accumulators in place: shifting in
  // place kept old and new accumulators live together and spilled registers
  // to scratch.
  auto stage_shifted = [&](auto value) {
#pragma unroll
    for (int i = 0; i < kTokBlocks; ++i) {
      int sv[16];
      float rv[16];
      load_tabs(i, sv, rv);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int cbyte = 2 * (cpos[j] & 7), chunk = (cpos[j] >> 3) ^ (4 * g);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = 32 * i + 8 * (e >> 2) + 4 * g + (e & 3);
          *reinterpret_cast<uint16_t *>(lds + row * 512 + chunk * 16 + cbyte) =
              value(ldexpf(fmaf(-2.f, acc[i][j][e], rv[e]), sv[e]), j);
        }
      }
    }
    __syncthreads();
  };
  stage_shifted([&](float v, int j) {
    v *= rs[j];
    return kPairOut ? f32_to_f16(v) : f32_to_bf16(v);
  });
  store_tile(C, std::integral_constant<bool, kFirst>{});
  if constexpr (kMode == kMidSave) {
    __syncthreads();
    const int es = smax_exp(tinfo[2 * T]);
    stage_shifted([&](float v, int) { return f32_to_f16(ldexpf(v, es)); });
    store_tile(V, std::false_type{});
  }
  if constexpr (kMode == kOutSave) {
    __syncthreads();  // every wave is done reading the staged C tile
    store_f32_tile(F, std::true_type{});
  }
}

// Backward operand statistics, one launch.  Block t < T takes token t:
// tstat[2t] = max_i |dy[t][i] s_out[i]| and tstat[2t + 1] = sum_i
// |dy[t][i] s_out[i]|, each thread reading 8 columns of every 2048 (four
// such loads in flight).  Block T stores max_k |s_mid[k]| in tstat[2T].
constexpr int kExpClamp = 100;
__global__ __launch_bounds__(256) void bwd_rowstat_kernel(const uint16_t *__restrict__ dy,
                                                          const uint16_t *__restrict__ s_out,
                                                          int T, int m, float *__restrict__ tstat,
                                                          const uint16_t *__restrict__ s_mid,
                                                          int r) {
  __shared__ float rmx[4], rl1[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int t = blockIdx.x;
  float mx = 0.f, l1 = 0.f;
  if (t == T) {
    mx = smid_absmax_part(s_mid, r, 256);
  } else {
    const uint16_t *row = dy + (size_t)t * m;
    for (int c0 = threadIdx.x * 8; c0 < m; c0 += 4 * 2048) {
      u32x4 v[4], so[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = c0 + q * 2048;
        v[q] = c < m ? *reinterpret_cast<const u32x4 *>(row + c) : u32x4{0u, 0u, 0u, 0u};
        so[q] = c < m ? *reinterpret_cast<const u32x4 *>(s_out + c) : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t sp = so[q][e];
          const float a = fabsf(__uint_as_float(v[q][e] << 16) * f16_lo(sp));
          const float b = fabsf(__uint_as_float(v[q][e] & 0xffff0000u) * f16_hi(sp));
          mx = fmaxf(mx, fmaxf(a, b));
          l1 += a + b;
        }
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    l1 += __shfl_xor(l1, off, 64);
  }
  if (lane == 0) {
    rmx[wave] = mx;
    rl1[wave] = l1;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const float m4 = fmaxf(fmaxf(rmx[0], rmx[1]), fmaxf(rmx[2], rmx[3]));
    if (t == T) {
      tstat[2 * T] = m4;
    } else {
      tstat[2 * t] = m4;
      tstat[2 * t + 1] = ((rl1[0] + rl1[1]) + rl1[2]) + rl1[3];
    }
  }
}

// Backward preparation, one launch.  Block row tb is the 64-token group G.
// From the statistics of dy * s_out, with M the group's largest entry,
// L_t the per-token sums of |entries| and S the largest |s_mid|: e
// (M 2^e in [2^13, 2^14)) puts fp16(dy s_out 2^e) at full fp16 precision
// down to M 2^-27, and c (2^e L_t S < 2^(14 + c) for every token of the
// group) bounds the first product's scaled outputs, |acc s_mid| <=
// 2^e L_t S, so fp16(acc s_mid 2^-c) cannot overflow; e and c are clamped
// to +-100 and are 0 for an all-zero group.  Block column 0 stores
// gscale[2G] = 2^-e and gscale[2G + 1] = 2^-c.  Every block then writes
// A1 = fp16(dy s_out 2^e) in pair order (the A operand of the first
// backward product) and the per-group partial sums of dy * z (z = the
// saved pre-scale forward output, fp32 [T][m]) for the gradient of s_out.
// Thread (ty, ux) handles the 16 columns of unit ux (as in pair_order_unit)
// for tokens t0 + ty + 16 q; the 16 ty partials of a column are added in a
// fixed order through LDS.
constexpr int kPrepTokens = 64;
__global__ __launch_bounds__(256) void bwd_prep_kernel(const uint16_t *__restrict__ dy,
                                                       const uint16_t *__restrict__ s_out,
                                                       const float *__restrict__ z, int T, int m,
                                                       const float *__restrict__ tstat,
                                                       float *__restrict__ gscale,
                                                       uint16_t *__restrict__ A1,
                                                       float *__restrict__ part) {
  __shared__ float red[16][256 + 4];
  __shared__ int gexp[2];
  const int ux = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int ur = blockIdx.x * 16 + ux;                       // unit within the row
  const int c = (ur >> 1) * 32 + 8 * (ur & 1);               // first of its columns
  const int tb = blockIdx.y;
  const bool live = c < m;
  const int cl = live ? c : 0;  // loads stay inside the arrays; results unused
  // Every load is issued before any is waited for: wave 0's group
  // statistics first (its wait then leaves the rows in flight), then s_out
  // and the thread's four token rows of dy and z (rows past T load row T-1
  // again and add nothing), so a block costs one memory round trip.
  float st_mx = 0.f, st_l1 = 0.f, st_smax = 0.f;
  const int ts = tb * kPrepTokens + (int)threadIdx.x;
  if (threadIdx.x < 64) {  // wave-uniform
    const int tc = min(ts, T - 1);
    st_mx = tstat[2 * tc];
    st_l1 = tstat[2 * tc + 1];
    st_smax = tstat[2 * T];
  }
  const u32x4 so_lo = *reinterpret_cast<const u32x4 *>(s_out + cl);
  const u32x4 so_hi = *reinterpret_cast<const u32x4 *>(s_out + cl + 16);
  constexpr int kRows = kPrepTokens / 16;
  u32x4 dlo[kRows], dhi[kRows];
  float4 zq[kRows][4];
#pragma unroll
  for (int q4 = 0; q4 < kRows; ++q4) {
    const int tc = min(tb * kPrepTokens + ty + 16 * q4, T - 1);
    const uint16_t *src = dy + (size_t)tc * m + cl;
    dlo[q4] = *reinterpret_cast<const u32x4 *>(src);
    dhi[q4] = *reinterpret_cast<const u32x4 *>(src + 16);
    const float *zr = z + (size_t)tc * m + cl;
    zq[q4][0] = *reinterpret_cast<const float4 *>(zr);
    zq[q4][1] = *reinterpret_cast<const float4 *>(zr + 4);
    zq[q4][2] = *reinterpret_cast<const float4 *>(zr + 16);
    zq[q4][3] = *reinterpret_cast<const float4 *>(zr + 20);
  }
  // group exponents: wave 0 reduces the 64 tokens' statistics
  if (threadIdx.x < 64) {
    const bool tok = ts < T;
    float mx = tok ? st_mx : 0.f;
    for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    int e = 0, c = 0;
    if (mx > 0.f) {
      int k;
      frexpf(mx, &k);  // mx = f 2^k, f in [0.5, 1)
      e = 14 - k;
      e = e > kExpClamp ? kExpClamp : (e < -kExpClamp ? -kExpClamp : e);
      float bound = tok ? ldexpf(st_l1, e) * st_smax : 0.f;
      for (int off = 32; off > 0; off >>= 1) bound = fmaxf(bound, __shfl_xor(bound, off, 64));
      frexpf(bound, &k);  // every 2^e L_t < 2^k
      c = k - 14;
      c = c > kExpClamp ? kExpClamp : (c < -kExpClamp ? -kExpClamp : c);
    }
    if (threadIdx.x == 0) {
      gexp[0] = e;
      gexp[1] = c;
      if (blockIdx.x == 0) {
        gscale[2 * tb] = ldexpf(1.f, -e);
        gscale[2 * tb + 1] = ldexpf(1.f, -c);
      }
    }
  }
  lds_barrier();  // gexp written; the row loads stay in flight
  const float up = ldexpf(1.f, gexp[0]);  // 2^e, exact
  float so[16];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    so[2 * e] = f16_lo(so_lo[e]);
    so[2 * e + 1] = f16_hi(so_lo[e]);
    so[8 + 2 * e] = f16_lo(so_hi[e]);
    so[8 + 2 * e + 1] = f16_hi(so_hi[e]);
  }
  float acc[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) acc[q] = 0.f;
#pragma unroll
  for (int q4 = 0; q4 < kRows; ++q4) {
    const int t = tb * kPrepTokens + ty + 16 * q4;
    const bool use = live && t < T;
    const float zl[8] = {zq[q4][0].x, zq[q4][0].y, zq[q4][0].z, zq[q4][0].w,
                         zq[q4][1].x, zq[q4][1].y, zq[q4][1].z, zq[q4][1].w};
    const float zh[8] = {zq[q4][2].x, zq[q4][2].y, zq[q4][2].z, zq[q4][2].w,
                         zq[q4][3].x, zq[q4][3].y, zq[q4][3].z, zq[q4][3].w};
    const u32x4 lo = dlo[q4], hi = dhi[q4];
    uint32_t d[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float g0 = __uint_as_float(lo[e] << 16), g1 = __uint_as_float(lo[e] & 0xffff0000u);
      const float h0 = __uint_as_float(hi[e] << 16), h1 = __uint_as_float(hi[e] & 0xffff0000u);
      // rows past T (and units past m) add +0: a sum that started at +0 stays
      acc[2 * e] += use ? g0 * zl[2 * e] : 0.f;
      acc[2 * e + 1] += use ? g1 * zl[2 * e + 1] : 0.f;
      acc[8 + 2 * e] += use ? h0 * zh[2 * e] : 0.f;
      acc[8 + 2 * e + 1] += use ? h1 * zh[2 * e + 1] : 0.f;
      // pair dword: column c+k (low half) with its partner c+16+k (high)
      d[2 * e] = pack_f16x2(g0 * so[2 * e] * up, h0 * so[8 + 2 * e] * up);
      d[2 * e + 1] = pack_f16x2(g1 * so[2 * e + 1] * up, h1 * so[8 + 2 * e + 1] * up);
    }
    if (use) {
      uint4 *dst = reinterpret_cast<uint4 *>(A1 + (size_t)t * m + (c & ~31) + 2 * (c & 15));
      dst[0] = make_uint4(d[0], d[1], d[2], d[3]);
      dst[1] = make_uint4(d[4], d[5], d[6], d[7]);
    }
  }
  // columns of this block: unit ux covers local columns lc .. lc+7 and
  // lc+16 .. lc+23 of the block's 256
  const int lc = (ux >> 1) * 32 + 8 * (ux & 1);
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    red[ty][lc + q] = acc[q];
    red[ty][lc + 16 + q] = acc[8 + q];
  }
  __syncthreads();
  const int col = blockIdx.x * 256 + threadIdx.x;
  if (col < m) {
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k) sum += red[k][threadIdx.x];
    part[(size_t)tb * m + col] = sum;
  }
}

// ds[c] = (accumulate ? ds[c] : 0) + sum over tiles of part[tile][c], for
// the three scale gradients in one launch.  A block takes 64 columns; wave
// w adds tiles w, w+4, w+8, ... in order (all its loads in flight at
// once), and wave 0 adds the four wave sums in order, so the result does
// not depend on timing.
constexpr int kFinishCols = 64;
__global__ __launch_bounds__(256) void bwd_finish_kernel(
    const float *__restrict__ p_out, int n_out_tiles, float *__restrict__ ds_out, int m,
    const float *__restrict__ p_mid, int n_mid_tiles, float *__restrict__ ds_mid, int r,
    const float *__restrict__ p_in, int n_in_tiles, float *__restrict__ ds_in, int n,
    int accumulate) {
  __shared__ float quarter[4][kFinishCols];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int idx = blockIdx.x * kFinishCols + lane;
  const float *p = nullptr;
  float *ds = nullptr;
  int tiles = 0, len = 0;
  if (idx < m) {
    p = p_out; ds = ds_out; tiles = n_out_tiles; len = m;
  } else if ((idx -= m) < r) {
    p = p_mid; ds = ds_mid; tiles = n_mid_tiles; len = r;
  } else if ((idx -= r) < n) {
    p = p_in; ds = ds_in; tiles = n_in_tiles; len = n;
  }
  float tot = 0.f, old = 0.f;
  if (p) {
    if (wave == 0 && accumulate) old = ds[idx];
    // Unconditional loads (indices clamped into the array, surplus values
    // dropped afterwards), so all sixteen are in flight together.
    float v[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int k = wave + 4 * q;
      v[q] = p[(size_t)(k < tiles ? k : tiles - 1) * len + idx];
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) tot += wave + 4 * q < tiles ? v[q] : 0.f;
    for (int k = wave + 64; k < tiles; k += 4) tot += p[(size_t)k * len + idx];
  }
  quarter[wave][lane] = tot;
  __syncthreads();
  if (wave == 0 && p) {
    const float s4 = ((quarter[0][lane] + quarter[1][lane]) + quarter[2][lane]) + quarter[3][lane];
    ds[idx] = old + s4;
  }
}

// Adds the S fp32 partials of two float4 runs (columns cl and ch of row
// base, partial s at base + s * stride) in split order.  The loads of a
// batch are all issued before any add: indices past S load the last
// partial again and add zero (an add of +0 leaves a sum that started at +0
// unchanged), so no branch sits between a load and the next one (behind a
// conditional add the compiler moves each load next to its use, one memory
// round trip per split).  The launch picks the batch from S (4, 8 or 16):
// a batch far above S would load the last partial many times over and hold
// registers that limit the waves in flight.
template <int kBatch>
__device__ __forceinline__ void sum_partials(const float *__restrict__ base, size_t stride, int S,
                                             int cl, int ch, float4 &lo, float4 &hi) {
  lo = make_float4(0.f, 0.f, 0.f, 0.f);
  hi = lo;
  for (int s0 = 0; s0 < S; s0 += kBatch) {
    float4 a[kBatch], b[kBatch];
#pragma unroll
    for (int q = 0; q < kBatch; ++q) {
      const int sp = min(s0 + q, S - 1);
      a[q] = *reinterpret_cast<const float4 *>(base + (size_t)sp * stride + cl);
      b[q] = *reinterpret_cast<const float4 *>(base + (size_t)sp * stride + ch);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int q = 0; q < kBatch; ++q) {
      const bool use = s0 + q < S;
      lo.x += use ? a[q].x : 0.f;
      lo.y += use ? a[q].y : 0.f;
      lo.z += use ? a[q].z : 0.f;
      lo.w += use ? a[q].w : 0.f;
      hi.x += use ? b[q].x : 0.f;
      hi.y += use ? b[q].y : 0.f;
      hi.z += use ? b[q].z : 0.f;
      hi.w += use ? b[q].w : 0.f;
    }
  }
}

// What finish8 reads besides the sums: the token's range-guard record, max
// |s_mid| and the operand's row sum R (kRecord, the forward modes; the
// kBwdIn reduction has no record and passes no tinfo), and the row scales
// of the 8 positions (cl .. cl+3 and ch .. ch+3, each run 8-byte aligned).
// Loaded before the partial sums and kept raw (nothing computed from them
// until the sums have arrived), so that their round trip overlaps the sums'
// instead of following it.
struct Fin8In {
  float2 ti;
  float smax, rt;
  uint2 rlo, rhi;
};
// kR: the row sum to load (0 none, 1 R1, 2 R2).
template <bool kRecord, int kR>
__device__ __forceinline__ Fin8In finish8_load(int cl, int ch, int t, int T,
                                               const uint16_t *__restrict__ rowscale,
                                               const float *__restrict__ tinfo) {
  Fin8In in;
  in.ti = make_float2(0.f, 0.f);
  in.smax = in.rt = 0.f;
  if constexpr (kRecord) {
    in.ti = reinterpret_cast<const float2 *>(tinfo)[t];
    in.smax = tinfo[2 * T];
  }
  if constexpr (kR > 0) in.rt = (kR == 1 ? tinfo_r1(tinfo, T) : tinfo_r2(tinfo, T))[t];
  in.rlo = *reinterpret_cast<const uint2 *>(rowscale + cl);
  in.rhi = *reinterpret_cast<const uint2 *>(rowscale + ch);
  return in;
}

// The forward modes' outputs for 8 consecutive output positions p .. p+7 of
// token t from their fp32 accumulator sums: lo holds columns cl .. cl+3, hi
// columns ch .. ch+3 (pair order interleaves the two runs, natural order
// concatenates them).  The first product's modes return the sum of their
// 8 values a_k (the stored fp16 over its column factor) for the row sums
// of the second product's operand; the others return 0.
template <int kMode>
__device__ __forceinline__ float finish8(const float4 &lo, const float4 &hi, const Fin8In &in,
                                         int p, int t, int N, uint16_t *__restrict__ C,
                                         uint16_t *__restrict__ V, float *__restrict__ F,
                                         bool live = true) {
  constexpr bool kPairOut = kMode == kMid || kMode == kMidSave;
  // the token's range-guard shift (see prep_stream_kernel), applied to the
  // signed product R - 2 acc before any rounding
  const int c_t = mid_exp(in.ti.x, in.smax);
  const int sh = kPairOut ? -c_t : c_t - __float_as_int(in.ti.y);
  const int es = kMode == kMidSave ? smax_exp(in.smax) : 0;
  auto fin = [&](float a) { return ldexpf(fmaf(-2.f, a, in.rt), sh); };
  const float l4[4] = {fin(lo.x), fin(lo.y), fin(lo.z), fin(lo.w)};
  const float h4[4] = {fin(hi.x), fin(hi.y), fin(hi.z), fin(hi.w)};
  float acc[8];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    acc[kPairOut ? 2 * k : k] = l4[k];
    acc[kPairOut ? 2 * k + 1 : 4 + k] = h4[k];
  }
  // row scales of columns cl .. cl+3 (rs[0..3]) and ch .. ch+3 (rs[4..7])
  const uint32_t rw[4] = {in.rlo.x, in.rlo.y, in.rhi.x, in.rhi.y};
  float rs[8];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    rs[2 * k] = f16_lo(rw[k]);
    rs[2 * k + 1] = f16_hi(rw[k]);
  }
  uint32_t c[4], v[4];
  float asum = 0.f;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    // pair order: columns (cl + k, ch + k), column factor index k (cl is a
    // multiple of 4); natural: (p + 2k, p + 2k + 1) with cl = p, ch = p + 4
    const float r0 = kPairOut ? ldexpf(rs[k], slot_exp(k)) : rs[2 * k];
    const float r1 = kPairOut ? ldexpf(rs[4 + k], slot_exp(k)) : rs[2 * k + 1];
    const float a0 = acc[2 * k] * r0, a1 = acc[2 * k + 1] * r1;
    c[k] = kPairOut ? (uint32_t)f32_to_f16(a0) | ((uint32_t)f32_to_f16(a1) << 16)
                    : (uint32_t)f32_to_bf16(a0) | ((uint32_t)f32_to_bf16(a1) << 16);
    v[k] = (uint32_t)f32_to_f16(ldexpf(acc[2 * k], es)) |
           ((uint32_t)f32_to_f16(ldexpf(acc[2 * k + 1], es)) << 16);
    if constexpr (kPairOut) asum += ldexpf(f16_lo(c[k]) + f16_hi(c[k]), -slot_exp(k));
  }
  if (!live) return 0.f;
  const size_t o = (size_t)t * N + p;
  *reinterpret_cast<uint4 *>(C + o) = make_uint4(c[0], c[1], c[2], c[3]);
  if constexpr (kMode == kMidSave)
    *reinterpret_cast<uint4 *>(V + o) = make_uint4(v[0], v[1], v[2], v[3]);
  if constexpr (kMode == kOutSave) {
    *reinterpret_cast<float4 *>(F + o) = make_float4(l4[0], l4[1], l4[2], l4[3]);
    *reinterpret_cast<float4 *>(F + o + 4) = make_float4(h4[0], h4[1], h4[2], h4[3]);
  }
  return asum;
}


// Output units (8 positions) per token row of a split-K reduction: the
// first product's rows are padded to whole 256-column tiles (32 units, a
// half wave, whose row sum goes to RS), the second's are not.
__host__ __device__ constexpr int64_t reduce_units_per_row(bool first, int64_t N) {
  return first ? (N + 255) / 256 * 32 : N / 8;
}

// The reduction of a split-K contraction (forward modes): C and its
// companions from the S fp32 partials of the workgroups along K, added in
// split order.  A thread takes 8 consecutive output positions of one token:
// in pair order (kMid, kMidSave) positions 8u .. 8u+7 of a 32-column group
// hold columns c0 .. c0+3 and c0+16 .. c0+19, interleaved; there the 32
// threads of a 256-column tile also add their values a_k for the tile's row
// sum in RS (threads past N add zero and store nothing).
template <int kMode, int kBatch>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float *__restrict__ P, int S,
                                                            int T, int N,
                                                            const uint16_t *__restrict__ rowscale,
                                                            uint16_t *__restrict__ C,
                                                            uint16_t *__restrict__ V,
                                                            float *__restrict__ F,
                                                            float *__restrict__ tinfo,
                                                            float *__restrict__ RS) {
  constexpr bool kPairOut = kMode == kMid || kMode == kMidSave;
  const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int upr = (int)reduce_units_per_row(kPairOut, N);
  if (u >= (int64_t)T * upr) return;  // whole half waves (upr is a multiple of 32 in pair order)
  const int t = (int)(u / upr);
  const int p = (int)(u % upr) * 8;  // first output position
  const bool live = p < N;
  const int pc = live ? p : 0;       // loads stay inside the arrays
  int cl, ch;                        // columns of the two float4 runs
  if (kPairOut) {
    cl = (pc & ~31) + ((pc & 31) >> 1);
    ch = cl + 16;
  } else {
    cl = pc;
    ch = pc + 4;
  }
  const Fin8In in = finish8_load<true, kPairOut ? 1 : 2>(cl, ch, t, T, rowscale, tinfo);
  float4 lo, hi;
  sum_partials<kBatch>(P + (size_t)t * N, (size_t)T * N, S, cl, ch, lo, hi);
  const float a = finish8<kMode>(lo, hi, in, pc, t, N, C, V, F, live);
  if constexpr (kPairOut) {
    const float rsum = half_wave_sum(a);
    if ((u & 31) == 0) RS[(size_t)t * rs_ld(N) + p / 256] = rsum;
  }
}

// The reduction of a mixed grid (forward modes): for each tile cut into
// S K ranges (tiles full .. full + H - 1), the partials of slots h S ..
// h S + S - 1 (tile-local [token][column], fp32) added in range order, then
// the mode's outputs.  16 workgroups per tile; a thread takes 8 consecutive
// output positions of one token row of the tile.
template <int kMode>
__global__ __launch_bounds__(256) void mixed_reduce_kernel(const float *__restrict__ P, int S,
                                                           int full, int nN, int T, int N,
                                                           const uint16_t *__restrict__ rowscale,
                                                           uint16_t *__restrict__ C,
                                                           uint16_t *__restrict__ V,
                                                           float *__restrict__ F,
                                                           float *__restrict__ tinfo,
                                                           float *__restrict__ RS) {
  constexpr bool kPairOut = kMode == kMid || kMode == kMidSave;
  const int h = blockIdx.x >> 4;
  const int unit = ((blockIdx.x & 15) << 8) + threadIdx.x;  // 0 .. 4095
  const int row = unit >> 5, ps = (unit & 31) * 8;          // token row, first position
  const int L = full + h;
  const int t = (L / nN) * BM + row;
  const int n0 = (L % nN) * BN;
  if (t >= T) return;  // a whole half wave (one token row)
  // positions past N add zero to the row sum and store nothing
  const bool live = n0 + ps < N;
  const int pl = live ? ps : 0;
  int cl, ch;  // tile-local columns of the two float4 runs
  if (kPairOut) {
    cl = (pl & ~31) + ((pl & 31) >> 1);
    ch = cl + 16;
  } else {
    cl = pl;
    ch = pl + 4;
  }
  const Fin8In in = finish8_load<true, kPairOut ? 1 : 2>(n0 + cl, n0 + ch, t, T, rowscale, tinfo);
  float4 lo = make_float4(0.f, 0.f, 0.f, 0.f), hi = lo;
  float4 a[4], b[4];
  const float *base = P + (size_t)h * S * (BM * BN) + row * BN;
#pragma unroll
  for (int q = 0; q < 4; ++q) {  // S <= 4; past S: the last partial again, added as zero
    const int sp = q < S ? q : S - 1;
    a[q] = *reinterpret_cast<const float4 *>(base + (size_t)sp * (BM * BN) + cl);
    b[q] = *reinterpret_cast<const float4 *>(base + (size_t)sp * (BM * BN) + ch);
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const bool use = q < S;
    lo.x += use ? a[q].x : 0.f;
    lo.y += use ? a[q].y : 0.f;
    lo.z += use ? a[q].z : 0.f;
    lo.w += use ? a[q].w : 0.f;
    hi.x += use ? b[q].x : 0.f;
    hi.y += use ? b[q].y : 0.f;
    hi.z += use ? b[q].z : 0.f;
    hi.w += use ? b[q].w : 0.f;
  }
  const float asum = finish8<kMode>(lo, hi, in, n0 + pl, t, N, C, V, F, live);
  if constexpr (kPairOut) {
    const float rsum = half_wave_sum(asum);
    if ((unit & 31) == 0) RS[(size_t)t * rs_ld(N) + L % nN] = rsum;
  }
}

// The reduction of a split-K backward contraction.  A workgroup takes 64
// tokens (one 64-token scale group) and 32 output positions: thread (tk, u)
// adds the S partials of positions 8u .. 8u+7 of token tk in split order,
// forms the mode's C values (scaled as in bingemm_kernel's epilogue), and
// the workgroup adds gradient * S over its 64 tokens in token order for the
// per-tile sums F (one row per 64 tokens).
constexpr int kBwdReduceCols = 32;
template <int kMode, int kBatch>
__global__ __launch_bounds__(256) void splitk_bwd_reduce_kernel(
    const float *__restrict__ P, int S, int T, int N, const uint16_t *__restrict__ rowscale,
    const float *__restrict__ gscale, uint16_t *__restrict__ C, const uint16_t *__restrict__ Sv,
    float *__restrict__ F, const float *__restrict__ tinfo) {
  constexpr bool kPairOut = kMode == kBwdMid;
  __shared__ float red[64][kBwdReduceCols + 1];
  const int u = threadIdx.x & 3, tk = threadIdx.x >> 2;
  const int tile = blockIdx.y;
  const int t = tile * 64 + tk;
  const int p = blockIdx.x * kBwdReduceCols + 8 * u;  // first output position
  int cl, ch;                                         // columns of the two float4 runs
  if (kPairOut) {
    cl = (p & ~31) + ((p & 31) >> 1);
    ch = cl + 16;
  } else {
    cl = p;
    ch = p + 4;
  }
  float g[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) g[k] = 0.f;
  if (t < T && p < N) {
    // the operands of the epilogue first (their round trip overlaps the sums')
    const float2 gs = reinterpret_cast<const float2 *>(gscale)[t >> 6];
    const uint4 sq = *reinterpret_cast<const uint4 *>(Sv + (size_t)t * N + p);
    const Fin8In in = finish8_load<kMode == kBwdMid, 0>(cl, ch, t, T, rowscale, tinfo);
    float4 lo, hi;
    sum_partials<kBatch>(P + (size_t)t * N, (size_t)T * N, S, cl, ch, lo, hi);
    const float fg = kMode == kBwdMid ? gs.x : gs.x / gs.y;
    // kBwdMid: S is the saved intermediate at the forward's per-token scale
    // (saved_v_shift from the prefetched record)
    const int vsh = kMode == kBwdMid ? mid_exp(in.ti.x, in.smax) - smax_exp(in.smax) -
                                           __float_as_int(in.ti.y)
                                     : 0;
    // row scales of columns cl .. cl+3 (rsv[0..3]) and ch .. ch+3 (rsv[4..7])
    const uint32_t rw[4] = {in.rlo.x, in.rlo.y, in.rhi.x, in.rhi.y};
    float rsv[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      rsv[2 * k] = f16_lo(rw[k]);
      rsv[2 * k + 1] = f16_hi(rw[k]);
    }
    const float l4[4] = {lo.x, lo.y, lo.z, lo.w}, h4[4] = {hi.x, hi.y, hi.z, hi.w};
    float acc[8], rse[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      acc[kPairOut ? 2 * k : k] = l4[k];
      acc[kPairOut ? 2 * k + 1 : 4 + k] = h4[k];
      rse[kPairOut ? 2 * k : k] = rsv[k];          // column cl + k
      rse[kPairOut ? 2 * k + 1 : 4 + k] = rsv[4 + k];  // column ch + k
    }
    // S is stored like C: fp16 in pair order (kBwdMid), bf16 natural (kBwdIn)
    const uint32_t sw[4] = {sq.x, sq.y, sq.z, sq.w};
    uint32_t c[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float o[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int e = 2 * k + h;
        const uint32_t sbits = h ? sw[k] >> 16 : sw[k] & 0xffffu;
        const float sval = kMode == kBwdMid ? f16_to_f32((uint16_t)sbits) : bf16_to_f32(sbits);
        g[e] = kMode == kBwdMid ? ldexpf(acc[e] * fg * sval, vsh) : acc[e] * fg * sval;
        const float rs = rse[e];
        o[h] = kMode == kBwdMid ? acc[e] * rs * gs.y : acc[e] * fg * rs;
      }
      c[k] = kMode == kBwdMid
                 ? (uint32_t)f32_to_f16(o[0]) | ((uint32_t)f32_to_f16(o[1]) << 16)
                 : (uint32_t)f32_to_bf16(o[0]) | ((uint32_t)f32_to_bf16(o[1]) << 16);
    }
    if (C) *reinterpret_cast<uint4 *>(C + (size_t)t * N + p) = make_uint4(c[0], c[1], c[2], c[3]);
  }
  // token sums: red[token][position in block], then one thread per position
  // adds the 64 tokens in order and writes the column's sum
#pragma unroll
  for (int k = 0; k < 8; ++k) red[tk][8 * u + k] = g[k];
  __syncthreads();
  if (threadIdx.x < kBwdReduceCols) {
    const int pos = threadIdx.x;
    const int pp = blockIdx.x * kBwdReduceCols + pos;
    float sum = 0.f;
    for (int k = 0; k < 64; ++k) sum += red[k][pos];
    if (pp < N) {
      // column of output position pp
      const int n = kPairOut ? (pp & ~31) + ((pp & 31) >> 1) + 16 * (pp & 1) : pp;
      F[(size_t)tile * N + n] = sum;
    }
  }
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// Copy pipeline depth per token-tile height.
#ifndef AF1_GEMM_STAGES_128
#define AF1_GEMM_STAGES_128 2
#endif
#ifndef AF1_GEMM_STAGES_64
#define AF1_GEMM_STAGES_64 2
#endif
constexpr int kStages128 = AF1_GEMM_STAGES_128;
constexpr int kStages64 = AF1_GEMM_STAGES_64;

// How one contraction is launched.  A grid of 128-token tiles that gives
// each compute unit at most one workgroup (one wave per SIMD) uses 64-token
// tiles instead: twice the workgroups, each expanding its signs for half as
// many tokens (measured on 8192x8192 G1: +2%; grids between one and two
// workgroups per unit were slower with it; at 64 tokens or fewer the
// shorter tile also computes fewer empty rows: 4096^2 G1 at T=32, 12.0 ->
// 9.2 us).  A forward grid that still
// leaves compute units idle (few tokens) may split its K steps over grid z
// (at least kMinSplitSteps steps per split); splitk_reduce_kernel then adds
// the fp32 partials in split order.  The split count minimises a simple
// cost: K steps per workgroup times the waves of workgroups (two per unit),
// plus, when split, the partials written and read back and one more launch.
// The constants are measured: a K step of a workgroup with the unit nearly
// to itself takes about 1.5 us at these grid sizes, partials move at about
// 4 TB/s, and the reduction launch costs about 3 us.
constexpr int kMinSplitSteps = 2;
constexpr double kStepUs = 1.5, kPartialBytesPerUs = 4.0e6, kLaunchUs = 3.0;
struct ContractionPlan {
  int bm;                // token-tile height
  unsigned gx, gy;       // weight-row tiles, token tiles
  int splits, split_steps;
  int mix_full, mix_splits;  // mixed grid (mix_full > 0): whole tiles, K ranges per other tile
};

// A forward grid of 128-token tiles with between one and 1.75 tiles per
// compute unit (28672x8192 and 8192x28672 G1 at T=2048: 400 tiles) leaves
// the units that got one tile idle for the last part of the launch.  Mixed
// grid: one whole tile per unit (the first workgroups, placed one per unit),
// and the remaining tiles each cut into kMixSplits K ranges that run beside
// them as partials; mixed_reduce_kernel adds them.  The busiest unit then
// carries 1 + 2/3 tile instead of 2.  Only for K of at least kMixMinSteps
// steps, where the partials' traffic is small against the kernel.
constexpr int kMixSplits = 3;
constexpr int kMixMinSteps = 24;

ContractionPlan plan_contraction(int64_t T, int64_t K, int64_t N, bool allow_split, int cus,
                                 bool allow_mixed = false) {
  ContractionPlan p;
  p.mix_full = p.mix_splits = 0;
  p.gx = (unsigned)((N + BN - 1) / BN);
  const int64_t tiles128 = (int64_t)p.gx * ((T + BM - 1) / BM);
  p.bm = tiles128 <= (int64_t)cus ? 64 : BM;
  p.gy = (unsigned)((T + p.bm - 1) / p.bm);
  const int64_t nk = (K / 32 + kWords - 1) / kWords;
  p.splits = 1;
  p.split_steps = (int)nk;
  const int64_t tiles = (int64_t)p.gx * p.gy;
  if (allow_split && tiles < cus) {
    auto cost = [&](int64_t sp) {
      const int64_t steps = (nk + sp - 1) / sp;
      const int64_t waves = (tiles * sp + 2 * cus - 1) / (2 * cus);
      double us = (double)(steps * waves) * kStepUs;
      if (sp > 1) us += 2.0 * (double)sp * T * N * 4 / kPartialBytesPerUs + kLaunchUs;
      return us;
    };
    int64_t best = 1;
    for (int64_t sp = 2; sp <= nk / kMinSplitSteps; ++sp)
      if (cost(sp) < cost(best)) best = sp;
    if (best > 1) {
      p.split_steps = (int)((nk + best - 1) / best);
      p.splits = (int)((nk + p.split_steps - 1) / p.split_steps);
    }
  }
  if (allow_mixed && p.bm == BM && tiles > cus && tiles * 4 < (int64_t)cus * 7 &&
      nk >= kMixMinSteps) {
    p.mix_full = cus;
    p.split_steps = (int)((nk + kMixSplits - 1) / kMixSplits);
    p.mix_splits = (int)((nk + p.split_steps - 1) / p.split_steps);
  }
  return p;
}

size_t mixed_bytes(const ContractionPlan &p, int64_t T, int64_t N) {
  if (p.mix_full == 0) return 0;
  const int64_t cut = (int64_t)p.gx * p.gy - p.mix_full;
  return align256((size_t)cut * p.mix_splits * BM * BN * 4);
}

size_t split_bytes(const ContractionPlan &p, int64_t T, int64_t N) {
  return p.splits > 1 ? align256((size_t)p.splits * T * N * 4) : 0;
}

// One contraction C[T, N] over K on the stream.  P: fp32 workspace for a
// split K (nullptr never splits).  *tile_tokens receives the token count
// per row of F's per-tile sums (the token-tile height, or 64 when split).
// Forward modes: tinfo is the range-guard record (the second product
// stores R2 into it) and RS the first product's per-tile row sums, written
// by the first product and read by the second.  The backward only reads
// tinfo.
template <int kMode>
hipError_t contraction(const uint16_t *A, int64_t T, int64_t K, const uint32_t *W, int64_t N,
                       const uint16_t *rs, uint16_t *C, uint16_t *V, const uint16_t *S,
                       float *F, hipStream_t s, int *tile_tokens = nullptr,
                       const float *gscale = nullptr, float *P = nullptr,
                       const float *tinfo_in = nullptr, float *RS = nullptr) {
  float *tinfo = const_cast<float *>(tinfo_in);
  constexpr bool kFwd = kMode == kMid || kMode == kMidSave || kMode == kOut || kMode == kOutSave;
  const ContractionPlan p = plan_contraction(T, K, N, P != nullptr, device_cus(), kFwd && P);
  if (p.splits > 1 && p.bm != 64) return hipErrorInvalidValue;  // see bingemm_kernel
  const int64_t tiles = (int64_t)p.gx * p.gy;
  const dim3 g = p.mix_full > 0
                     ? dim3((unsigned)(p.mix_full + (tiles - p.mix_full) * p.mix_splits))
                     : dim3(p.gx, p.gy, (unsigned)p.splits);
  if (p.bm == 64)
    bingemm_kernel<kMode, 64, kStages64><<<g, kThreads, Lds<64, kStages64>::kBytes, s>>>(
        A, (int)T, (int)K, W, (int)N, rs, C, V, S, F, gscale, p.split_steps, P, p.mix_full,
        p.mix_splits, (int)p.gx, tinfo, RS);
  else
    bingemm_kernel<kMode, BM, kStages128><<<g, kThreads, Lds<BM, kStages128>::kBytes, s>>>(
        A, (int)T, (int)K, W, (int)N, rs, C, V, S, F, gscale, p.split_steps, P, p.mix_full,
        p.mix_splits, (int)p.gx, tinfo, RS);
  if (tile_tokens) *tile_tokens = p.splits > 1 ? 64 : p.bm;
  if (p.mix_full > 0) {
    if constexpr (kFwd) {
      const unsigned blocks = (unsigned)((tiles - p.mix_full) * 16);
      mixed_reduce_kernel<kMode><<<blocks, 256, 0, s>>>(P, p.mix_splits, p.mix_full, (int)p.gx,
                                                         (int)T, (int)N, rs, C, V, F, tinfo, RS);
    } else {
      return hipErrorInvalidValue;  // planned for the forward modes only
    }
  }
  if (p.splits > 1) {
    if constexpr (kMode == kBwdMid || kMode == kBwdIn) {
      const dim3 gr((unsigned)((N + kBwdReduceCols - 1) / kBwdReduceCols),
                    (unsigned)((T + 63) / 64));
      auto go = [&](auto kernel) {
        kernel<<<gr, 256, 0, s>>>(P, p.splits, (int)T, (int)N, rs, gscale, C, S, F, tinfo);
      };
      if (p.splits <= 4)
        go(splitk_bwd_reduce_kernel<kMode, 4>);
      else if (p.splits <= 8)
        go(splitk_bwd_reduce_kernel<kMode, 8>);
      else
        go(splitk_bwd_reduce_kernel<kMode, 16>);
    } else {
      // A reduction that would occupy at most half the compute units with
      // 256-thread blocks runs 64-thread blocks: the partial loads of a few
      // blocks are limited per unit (4096^2 at 64 tokens: 30.5 us a call
      // against 33.7 with 256-thread blocks throughout).
      const int64_t units = T * reduce_units_per_row(kMode == kMid || kMode == kMidSave, N);
      const int rt = (units + 255) / 256 <= device_cus() / 2 ? 64 : 256;
      auto go = [&](auto kernel) {
        kernel<<<(unsigned)((units + rt - 1) / rt), rt, 0, s>>>(P, p.splits, (int)T, (int)N, rs,
                                                               C, V, F, tinfo, RS);
      };
      if (p.splits <= 4)
        go(splitk_reduce_kernel<kMode, 4>);
      else if (p.splits <= 8)
        go(splitk_reduce_kernel<kMode, 8>);
      else
        go(splitk_reduce_kernel<kMode, 16>);
    }
  }
  return hipGetLastError();
}

// Worker waves of the preparation a compute unit: with a row and the next
// one in registers (107 to 126 VGPRs) the register file holds four waves a
// SIMD.
constexpr int kPrepWavesPerCU = 16;

// fp16(s_in .* x 2^e_t) in pair order, the A operand of G1, and the
// per-token range-guard record (see prep_stream_kernel).
hipError_t prepare_forward(int64_t n, const uint16_t *s_in, const uint16_t *x, int64_t T,
                           uint16_t *xp, float *tinfo, const uint16_t *s_mid, int64_t r,
                           hipStream_t s) {
  // a row in registers: at most two units a thread, 256 to 1024 threads
  const int64_t units = n / 16;
  if (T == 0) {
    prep_kernel<<<1, 256, 0, s>>>(x, s_in, xp, 0, (int)n, tinfo, s_mid, (int)r);
    return hipGetLastError();
  }
  const auto grid = [&](int threads) {
    const int64_t w = (int64_t)device_cus() * std::max(1, kPrepWavesPerCU * 64 / threads);
    return dim3((unsigned)(std::min<int64_t>(T, w) + 1));
  };
  if (units <= 256)
    prep_stream_kernel<1, 256><<<grid(256), 256, 0, s>>>(x, s_in, xp, (int)T, (int)n, tinfo,
                                                          s_mid, (int)r);
  else if (units <= 512)
    prep_stream_kernel<2, 256><<<grid(256), 256, 0, s>>>(x, s_in, xp, (int)T, (int)n, tinfo,
                                                          s_mid, (int)r);
  else if (units <= 1024)
    prep_stream_kernel<2, 512><<<grid(512), 512, 0, s>>>(x, s_in, xp, (int)T, (int)n, tinfo,
                                                          s_mid, (int)r);
  else if (units <= 2048)
    prep_stream_kernel<2, 1024><<<grid(1024), 1024, 0, s>>>(x, s_in, xp, (int)T, (int)n, tinfo,
                                                             s_mid, (int)r);
  else
    prep_kernel<<<dim3((unsigned)(T + 1)), 256, 0, s>>>(x, s_in, xp, (int)T, (int)n, tinfo,
                                                        s_mid, (int)r);
  return hipGetLastError();
}

size_t tinfo_bytes(int64_t T) { return align256((size_t)tinfo_floats(T) * 4); }

size_t rowsum_bytes(int64_t r, int64_t T) { return align256((size_t)T * rs_ld(r) * 4); }

struct FwdWs {
  uint16_t *xp, *Z;
  float *tinfo;  // the per-token range-guard record
  float *RS;     // G1's per-tile row sums of Z
  float *P;      // split-K partials of G1 or G2 (one at a time)
};

FwdWs forward_ws(void *ws, int64_t n, int64_t r, int64_t T) {
  uint8_t *base = static_cast<uint8_t *>(ws);
  FwdWs w;
  w.xp = reinterpret_cast<uint16_t *>(base);
  base += align256((size_t)T * n * 2);
  w.Z = reinterpret_cast<uint16_t *>(base);
  base += align256((size_t)T * r * 2);
  w.tinfo = reinterpret_cast<float *>(base);
  base += tinfo_bytes(T);
  w.RS = reinterpret_cast<float *>(base);
  base += rowsum_bytes(r, T);
  w.P = reinterpret_cast<float *>(base);
  return w;
}

int64_t tiles64(int64_t T) { return (T + 63) / 64; }

struct BwdWs {
  uint16_t *A1, *Zb;
  float *p_out, *p_mid, *p_in, *tstat, *gscale, *P;
};

BwdWs backward_ws(void *ws, int64_t m, int64_t n, int64_t r, int64_t T) {
  uint8_t *base = static_cast<uint8_t *>(ws);
  BwdWs w;
  w.A1 = reinterpret_cast<uint16_t *>(base);
  base += align256((size_t)T * m * 2);
  w.Zb = reinterpret_cast<uint16_t *>(base);
  base += align256((size_t)T * r * 2);
  w.p_out = reinterpret_cast<float *>(base);
  base += align256((size_t)tiles64(T) * m * 4);
  w.p_mid = reinterpret_cast<float *>(base);
  base += align256((size_t)tiles64(T) * r * 4);
  w.p_in = reinterpret_cast<float *>(base);
  base += align256((size_t)tiles64(T) * n * 4);
  w.tstat = reinterpret_cast<float *>(base);
  base += align256((size_t)T * 8 + 4);
  w.gscale = reinterpret_cast<float *>(base);
  base += align256((size_t)tiles64(T) * 8);
  w.P = reinterpret_cast<float *>(base);
  return w;
}

size_t backward_ws_bytes(int64_t m, int64_t n, int64_t r, int64_t T) {
  // ... and the fp32 partials of whichever backward contraction splits K
  const int cus = device_cus();
  const size_t p1 = split_bytes(plan_contraction(T, m, r, true, cus), T, r);
  const size_t p2 = split_bytes(plan_contraction(T, r, n, true, cus), T, n);
  return align256((size_t)T * m * 2) + align256((size_t)T * r * 2) +
         align256((size_t)tiles64(T) * m * 4) + align256((size_t)tiles64(T) * r * 4) +
         align256((size_t)tiles64(T) * n * 4) + align256((size_t)T * 8 + 4) +
         align256((size_t)tiles64(T) * 8) + (p1 > p2 ? p1 : p2);
}

}  // namespace

size_t gemm_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t T) {
  // fp16(s_in .* x) and the fp16 intermediate Z, both in pair order, and the
  // fp32 partials of whichever contraction splits its K steps
  const int cus = device_cus();
  const ContractionPlan g1 = plan_contraction(T, n, r, true, cus, true);
  const ContractionPlan g2 = plan_contraction(T, r, m, true, cus, true);
  const size_t p1 = split_bytes(g1, T, r) > mixed_bytes(g1, T, r) ? split_bytes(g1, T, r)
                                                                   : mixed_bytes(g1, T, r);
  const size_t p2 = split_bytes(g2, T, m) > mixed_bytes(g2, T, m) ? split_bytes(g2, T, m)
                                                                   : mixed_bytes(g2, T, m);
  return align256((size_t)T * (size_t)n * 2) + align256((size_t)T * (size_t)r * 2) +
         tinfo_bytes(T) + rowsum_bytes(r, T) + (p1 > p2 ? p1 : p2);
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
  const FwdWs w = forward_ws(ws, n, r, T);
  hipError_t e = prepare_forward(n, s_in, x, T, w.xp, w.tinfo, s_mid, r, s);
  if (e != hipSuccess) return e;
  e = contraction<kMid>(w.xp, T, n, Bv, r, s_mid, w.Z, nullptr, nullptr, nullptr, s, nullptr,
                        nullptr, w.P, w.tinfo, w.RS);
  if (e != hipSuccess) return e;
  return contraction<kOut>(w.Z, T, r, Bu, m, s_out, y, nullptr, nullptr, nullptr, s, nullptr,
                           nullptr, w.P, w.tinfo, w.RS);
}

size_t train_saved_bytes(int64_t m, int64_t n, int64_t r, int64_t T) {
  (void)n;
  // the pre-scale intermediate v = Bv (s_in .* x), fp16 in pair order at a
  // per-token scale, the pre-scale output z = Bu (s_mid .* v), fp32, and the
  // per-token range-guard record that gives v's scale
  return align256((size_t)T * r * 2) + align256((size_t)T * m * 4) + tinfo_bytes(T);
}

size_t train_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t T) {
  const size_t f = gemm_workspace_bytes(m, n, r, T), b = backward_ws_bytes(m, n, r, T);
  return f > b ? f : b;
}

hipError_t launch_forward_train(int64_t m, int64_t n, int64_t r, const uint32_t *Bu,
                                const uint32_t *Bv, const uint16_t *s_out,
                                const uint16_t *s_mid, const uint16_t *s_in,
                                const uint16_t *x, int64_t T, uint16_t *y, void *saved,
                                void *ws, hipStream_t s) {
  if (T * n * 2 > 0x7fffffff || T * r * 2 > 0x7fffffff || m * (r / 32) * 4 > 0x7fffffff ||
      r * (n / 32) * 4 > 0x7fffffff)
    return hipErrorInvalidValue;
  const FwdWs w = forward_ws(ws, n, r, T);
  uint16_t *v = static_cast<uint16_t *>(saved);
  float *z = reinterpret_cast<float *>(static_cast<uint8_t *>(saved) + align256((size_t)T * r * 2));
  float *tinfo = reinterpret_cast<float *>(static_cast<uint8_t *>(saved) +
                                           align256((size_t)T * r * 2) +
                                           align256((size_t)T * m * 4));
  hipError_t e = prepare_forward(n, s_in, x, T, w.xp, tinfo, s_mid, r, s);
  if (e != hipSuccess) return e;
  // the same G1 as the inference forward, which also keeps fp16(v) at the
  // token's scale
  e = contraction<kMidSave>(w.xp, T, n, Bv, r, s_mid, w.Z, v, nullptr, nullptr, s, nullptr,
                            nullptr, w.P, tinfo, w.RS);
  if (e != hipSuccess) return e;
  return contraction<kOutSave>(w.Z, T, r, Bu, m, s_out, y, nullptr, nullptr, z, s, nullptr,
                               nullptr, w.P, tinfo, w.RS);
}

hipError_t launch_backward(int64_t m, int64_t n, int64_t r, const uint32_t *BuT,
                           const uint32_t *BvT, const uint16_t *s_out, const uint16_t *s_mid,
                           const uint16_t *s_in, const uint16_t *x, const uint16_t *dy,
                           int64_t T, const void *saved, uint16_t *dx, float *ds_out,
                           float *ds_mid, float *ds_in, int accumulate, void *ws,
                           hipStream_t s) {
  if (T * m * 2 > 0x7fffffff || T * r * 2 > 0x7fffffff || r * (m / 32) * 4 > 0x7fffffff ||
      n * (r / 32) * 4 > 0x7fffffff)
    return hipErrorInvalidValue;
  const BwdWs w = backward_ws(ws, m, n, r, T);
  const uint16_t *v = static_cast<const uint16_t *>(saved);
  const float *z = reinterpret_cast<const float *>(static_cast<const uint8_t *>(saved) +
                                                   align256((size_t)T * r * 2));
  const float *tinfo = reinterpret_cast<const float *>(
      static_cast<const uint8_t *>(saved) + align256((size_t)T * r * 2) +
      align256((size_t)T * m * 4));
  // per-token statistics of dy * s_out, and the largest |s_mid|
  bwd_rowstat_kernel<<<(unsigned)(T + 1), 256, 0, s>>>(dy, s_out, (int)T, (int)m, w.tstat, s_mid,
                                                       (int)r);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 gp((unsigned)((m + 255) / 256), (unsigned)tiles64(T));
  bwd_prep_kernel<<<gp, 256, 0, s>>>(dy, s_out, z, (int)T, (int)m, w.tstat, w.gscale, w.A1,
                                     w.p_out);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // dt 2^e = Bu^T (s_out .* dy 2^e): weight rows are the r rows of Bu^T;
  // the output fp16(s_mid .* dt 2^(e - c)) in pair order is the next A
  // operand; sums dt .* v.
  int tm = 0, ti = 0;
  e = contraction<kBwdMid>(w.A1, T, m, BuT, r, s_mid, w.Zb, nullptr, v, w.p_mid, s, &tm,
                           w.gscale, w.P, tinfo);
  if (e != hipSuccess) return e;
  // du 2^(e - c) = Bv^T (s_mid .* dt 2^(e - c)): dx = s_in .* du; sums du .* x.
  e = contraction<kBwdIn>(w.Zb, T, r, BvT, n, s_in, dx, nullptr, x, w.p_in, s, &ti, w.gscale,
                          w.P);
  if (e != hipSuccess) return e;
  const int total = (int)(m + r + n);
  bwd_finish_kernel<<<(unsigned)((total + kFinishCols - 1) / kFinishCols), 256, 0, s>>>(
      w.p_out, (int)tiles64(T), ds_out, (int)m, w.p_mid, (int)((T + tm - 1) / tm), ds_mid,
      (int)r, w.p_in, (int)((T + ti - 1) / ti), ds_in, (int)n, accumulate);
  return hipGetLastError();
}

}  // namespace af1
