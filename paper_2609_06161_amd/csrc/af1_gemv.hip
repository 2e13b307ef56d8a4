// Decode-regime forward of the factorized binary linear (paper App. A.2.1,
// Diag form, evaluated right to left; Sec. 4.1 deployable form):
//
//   stage 1:  t[b, k] = s_mid[k] * sum_j Bv[k, j] * (s_in[j] * x[b, j])
//   stage 2:  y[b, i] = bf16( s_out[i] * sum_k Bu[i, k] * t[b, k] )
//
// Both stages are one kernel template: a +-1 row product against a vector
// staged in LDS, then a per-row scale.  The products run on the gfx950
// matrix cores (v_mfma_f32_16x16x32_bf16): rows of the sign matrix are the
// M dimension, the batch is N (lanes with no batch row read zeros), the
// input columns are K.
//
// Exactness.  A sign becomes the bf16 value +-1 (exact).  The fp32 input
// (s_in*x is exact in fp32: 8 x 11 significant bits) is split into
// hi = bf16(v) and lo = bf16(v - hi); two MFMAs per tile consume hi and lo,
// so the operand error is below 2^-17 relative, and accumulation is fp32.
//
// Sign expansion.  Within a 32-bit word, columns p and p+16 (p = 0..15) are
// paired: one shift moves bit p to bit 15 and bit p+16 to bit 31, and one
// three-input bit operation merges those two sign bits into 0x3F80 (bf16
// 1.0) -- two VALU ops per two operands.  The MFMA K order is free as long
// as the A (signs) and B (inputs) operands agree, so the LDS copy of the
// input is stored in the same (p, p+16) pairs.
//
// Workgroups.  A 512-thread workgroup owns 16 * 2^k output rows (k = 0..3,
// chosen per stage from the batch and the row count: more rows per
// workgroup share one staged copy of the input as the batch grows).  Its 8
// waves are split over the 16-row tiles, and the waves of a tile split its
// columns into groups of 8 words.
//
// Latency.  A decode-size call is bound by launch and memory latency, not
// bandwidth.  Every wave first issues the loads of its sign words (buffer
// loads: out-of-range lanes read zeros, no branches, so no early waits),
// then the input is loaded and converted to bf16 hi/lo pairs in LDS (with
// one tile per workgroup each wave stages only the columns it uses and no
// barrier is needed), and the MFMAs run with the LDS operand reads
// double-buffered.  The 16x16 results of a tile's waves are added through
// LDS.  When b * K is too large for one LDS slab the columns are split over
// workgroups ("slabs"); each slab writes a partial sum and the last slab of
// a row group to finish (atomic counter) adds the partials in slab order,
// so the result is deterministic.
#include <atomic>
#include <cstring>
#include <mutex>
#include <utility>
#include <vector>

#include "af1_device.h"
#include "af1_internal.h"

namespace af1 {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float float2v __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kTileRows = 16;        // MFMA M
constexpr int kGroupWords = 8;       // one 8-byte load per lane covers 16 rows x 8 words
constexpr int kMaxGroups = 8;        // groups per wave (single pass)
// LDS bytes per (batch row, word): for each half h of the word's 16 pairs,
// 32 bytes of hi then 32 of lo, then 16 bytes of pad.  A staging unit (one
// half) is 64 contiguous bytes, so the units of consecutive lanes (word w,
// half h at 9w + 4h sixteen-byte lines) never share a bank group.
constexpr int kSlot = 144;

// LDS bytes between the staged slots of consecutive batch rows: the words
// of one row, plus 16 bytes when needed to make the stride an odd multiple
// of 16 bytes, so that the lanes of an MFMA operand read (different batch
// rows, same word) fall in distinct 16-byte bank groups.
__host__ __device__ constexpr int row_stride(int w_count) {
  return w_count * kSlot + ((w_count & 1) ? 0 : 16);
}
constexpr int kLdsPerCu = 160 * 1024;  // LDS of one gfx950 compute unit
// Dynamic LDS a stage workgroup may request: the compute unit's LDS less a
// reserve for the kernels' own __shared__ variables (16 bytes in the stage
// kernels, 32 in the stream kernel), which the launch adds to the dynamic
// size.  launch_fits() checks the sum before every launch.
constexpr int kStaticLdsReserve = 256;
constexpr int kLdsBudget = kLdsPerCu - kStaticLdsReserve;
// Cross-wave sums: each wave's 64 lanes x 16 bytes, one 16-byte pad after
// every 16 lanes, so that the 4 rows x 16 columns read by consecutive
// output threads spread over the banks.
constexpr int kRedLanes = 68;
constexpr int kRedBytes = kWaves * kRedLanes * 16;
constexpr int kMaxOutPerThread = 4;  // outputs (row, batch row) written per thread
constexpr int kMaxSlabsLoaded = 8;   // partial sums loaded at once by the last slab
constexpr int kDeviceScope = 16;     // buffer cache policy sc1: coherent across XCDs
// Staging passes.  Shared staging: a slab holds at most (kLdsBudget - kSlot)
// / kSlot words over all batch rows (2 units per word), taken two per thread
// per pass.  Per-wave staging: 128 units per wave per pass; the plan keeps a
// wave's units (groups x b x 16) within kStageIters passes.
constexpr int kStageIters = 3;
static_assert(kStageIters * 2 * kThreads >= 2 * ((kLdsBudget - kSlot) / kSlot), "staging passes");
constexpr int kWaveStageUnits = kStageIters * 128;
constexpr int kOob = (int)0x80000000u;  // a buffer offset past any resource

// The last-slab reduction hands partial sums between workgroups of one
// launch with device-scope stores and loads (coherent across the XCDs' L2
// caches) and relaxed atomics, ordered by waiting for this wave's memory
// operations to complete.  A release/acquire fence at device scope would
// write back and invalidate the whole L2 per workgroup, which costs tens of
// microseconds at these grid sizes.
__device__ __forceinline__ void wait_memory() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ void store_device(float *p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void store_device_u16(uint16_t *p, uint16_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Calls f(std::integral_constant<int, I>) for I = 0 .. N-1, fully unrolled,
// so that register arrays indexed by I stay in registers.
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Buffer resource over [base, base + bytes): loads at offsets beyond `bytes`
// return zero instead of faulting.  Word 3 selects raw 32-bit dword access.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *base, int64_t bytes) {
  const int n = bytes > 0x7fffffff ? 0x7fffffff : (bytes < 0 ? 0 : (int)bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, n, 0x00020000);
}

// Two fp32 -> packed bf16 (round to nearest even), one instruction on gfx950.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo_half, float hi_half) {
  const float2v f = {lo_half, hi_half};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

struct UnitRaw {
  u32x4 a, b, c, d;
};

// Raw data of one staging unit: columns c0 .. c0+7 and c0+16 .. c0+23 of one
// batch row (x and s_in for the first stage, fp32 t for the second).  `off`
// is the element offset of column c0 in the input, kOob for no unit.
template <bool kInX, int kAux>
__device__ __forceinline__ UnitRaw load_unit(__amdgpu_buffer_rsrc_t xres,
                                             __amdgpu_buffer_rsrc_t sres, int off, int col,
                                             int part_off = 0) {
  UnitRaw r;
  if constexpr (kInX) {
    const int xo = off == kOob ? kOob : off * 2;
    const int so = off == kOob ? kOob : col * 2;
    r.a = __builtin_amdgcn_raw_buffer_load_b128(xres, xo, 0, kAux);
    r.b = __builtin_amdgcn_raw_buffer_load_b128(xres, xo + 32, 0, kAux);
    r.c = __builtin_amdgcn_raw_buffer_load_b128(sres, so, 0, 0);
    r.d = __builtin_amdgcn_raw_buffer_load_b128(sres, so + 32, 0, 0);
  } else {
    const int to = off == kOob ? kOob : (off + part_off) * 4;
    r.a = __builtin_amdgcn_raw_buffer_load_b128(xres, to, 0, kAux);
    r.b = __builtin_amdgcn_raw_buffer_load_b128(xres, to + 16, 0, kAux);
    r.c = __builtin_amdgcn_raw_buffer_load_b128(xres, to + 64, 0, kAux);
    r.d = __builtin_amdgcn_raw_buffer_load_b128(xres, to + 80, 0, kAux);
  }
  return r;
}

// fp32 values of a unit: v[d] = column c0+d, v[8+d] = column c0+16+d.  For
// the fp32 input a second set of raw data (a second partial sum) is added.
template <bool kInX>
__device__ __forceinline__ void unit_values(const UnitRaw &r, float (&v)[16],
                                            const UnitRaw *r2 = nullptr) {
  if constexpr (kInX) {
    const uint32_t xd[8] = {r.a.x, r.a.y, r.a.z, r.a.w, r.b.x, r.b.y, r.b.z, r.b.w};
    const uint32_t sd[8] = {r.c.x, r.c.y, r.c.z, r.c.w, r.d.x, r.d.y, r.d.z, r.d.w};
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      v[2 * d] = bf16_to_f32(xd[d] & 0xffffu) * f16_to_f32((uint16_t)(sd[d] & 0xffffu));
      v[2 * d + 1] = bf16_to_f32(xd[d] >> 16) * f16_to_f32((uint16_t)(sd[d] >> 16));
    }
  } else {
    const u32x4 q4[4] = {r.a, r.b, r.c, r.d};
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int e = 0; e < 4; ++e) v[4 * k + e] = __uint_as_float(q4[k][e]);
    if (r2) {
      const u32x4 p4[4] = {r2->a, r2->b, r2->c, r2->d};
#pragma unroll
      for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int e = 0; e < 4; ++e) v[4 * k + e] += __uint_as_float(p4[k][e]);
    }
  }
}

// Store a unit as hi/lo pair dwords (pair 8h+d = columns c0+d and c0+16+d):
// hi = bf16(v), lo = bf16(v - hi).
__device__ __forceinline__ void store_unit(uint8_t *slot_base, int h, const float (&v)[16]) {
  uint32_t hi[8], lo[8];
#pragma unroll
  for (int d = 0; d < 8; ++d) {
    hi[d] = pack_bf16x2(v[d], v[8 + d]);
    lo[d] = pack_bf16x2(v[d] - bf16_to_f32(hi[d] & 0xffffu), v[8 + d] - bf16_to_f32(hi[d] >> 16));
  }
  uint4 *slot = reinterpret_cast<uint4 *>(slot_base);
  slot[4 * h] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
  slot[4 * h + 1] = make_uint4(hi[4], hi[5], hi[6], hi[7]);
  slot[4 * h + 2] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
  slot[4 * h + 3] = make_uint4(lo[4], lo[5], lo[6], lo[7]);
}

// Output modes of a stage launch.
constexpr int kModeFinal = 0;     // one slab: write the scaled result
constexpr int kModeLastSlab = 1;  // several slabs: the last one to finish adds them
constexpr int kModePartial = 2;   // several slabs: each writes its scaled partial sum
                                  // (the next stage adds them while staging)

// Output rows handled by one workgroup: rt_count tiles of 16 rows.  The 8
// waves are split evenly over the tiles; the waves of one tile split its
// columns into groups of 8 words (group g of the slab goes to wave g mod
// waves_per_tile of that tile).
struct Role {
  int rt_log2;     // log2(tiles per workgroup)
  int wpt;         // waves per tile
  int rt;          // this wave's tile within the workgroup
  int cw;          // this wave's column share within its tile
  int tile;        // global 16-row tile of this wave
  int row0;
  int w_begin, w_count;
  int my_groups;
};

__device__ __forceinline__ Role make_role(int wave, int group, int slab, int rt_log2, int wpr,
                                         int slab_words) {
  Role r;
  r.rt_log2 = rt_log2;
  r.wpt = kWaves >> rt_log2;
  r.rt = wave >> (3 - rt_log2);
  r.cw = wave & (r.wpt - 1);
  r.tile = (group << rt_log2) + r.rt;
  r.row0 = r.tile * kTileRows;
  r.w_begin = slab * slab_words;
  r.w_count = min(slab_words, wpr - r.w_begin);
  const int ngroups = (r.w_count + kGroupWords - 1) / kGroupWords;
  r.my_groups = ngroups > r.cw ? (ngroups - r.cw + r.wpt - 1) >> (3 - rt_log2) : 0;
  return r;
}

// One stage: a +-1 product of 16 * 2^rt_log2 rows of M against the staged
// input columns of one slab, then the per-row scale.
//
// kHiLoCols (b <= 8): the bf16 hi and lo parts of batch row beta occupy MFMA
// columns 2*beta and 2*beta+1, so one MFMA per tile covers both; otherwise
// (b up to 16) columns are batch rows and hi and lo take one MFMA each.
//
// Arguments are scalars, most urgent first, so that they are preloaded into
// SGPRs at wave launch instead of being fetched from the kernarg segment.
//
// kMulti: several row tiles per workgroup (rt_log2 > 0, staging shared by
// the workgroup); otherwise one tile, and rt_log2 is ignored.
//
// kCoherent: the input may have been written by other workgroups of the
// same launch and the output may be read by them (the persistent stream
// kernel): input loads and output stores then use device scope, coherent
// across the XCDs' L2 caches.
// Row scales of the outputs thread tid writes at the end of a stage:
// outputs o = tid + kThreads * k, row (o mod rows_wg) of the workgroup's
// rows, batch row o / rows_wg.
__device__ __forceinline__ void load_row_scales(uint32_t (&rs)[kMaxOutPerThread],
                                                const uint16_t *__restrict__ row_scale, int rows,
                                                int group, int rt_log2, int b, int nk_out) {
  const int rows_wg = 16 << rt_log2;
  const int row_wg0 = group * rows_wg;
  const int nout = rows_wg * b;
  const __amdgpu_buffer_rsrc_t rres = buffer_rsrc(row_scale, (int64_t)rows * 2);
#pragma unroll
  for (int k = 0; k < kMaxOutPerThread; ++k) {
    // the first load is unconditional (and so is its use below): a load
    // whose only use sits in a branch is moved there, behind every wait
    rs[k] = 0u;
    if (k > 0 && k >= nk_out) break;
    const int o = (int)threadIdx.x + kThreads * k;
    const int orow = row_wg0 + (o & (rows_wg - 1));
    rs[k] = __builtin_amdgcn_raw_buffer_load_b16(rres, o < nout ? orow * 2 : kOob, 0, 0);
  }
}

// Sign words of one wave's groups (step 1 below) and the row scales of a
// stage, loaded ahead of the rest by the stream kernel.
struct SignRegs {
  u32x2 wv[kMaxGroups];
  uint32_t rs[kMaxOutPerThread];
};

__device__ __forceinline__ void stage_signs(SignRegs &sg, const uint32_t *__restrict__ M, int rows,
                                            int wpr, int slab_words, int rt_log2, int group,
                                            int slab, const uint16_t *__restrict__ row_scale,
                                            int b) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const Role R = make_role(wave, group, slab, rt_log2, wpr, slab_words);
  const int nout = (16 << rt_log2) * b;
  load_row_scales(sg.rs, row_scale, rows, group, rt_log2, b,
                  rt_log2 > 0 ? (nout + kThreads - 1) / kThreads : 1);
  const int64_t left = (int64_t)(rows - R.row0) * wpr * 4;
  const __amdgpu_buffer_rsrc_t mres = buffer_rsrc(M + (size_t)R.row0 * wpr, left);
#pragma unroll
  for (int i = 0; i < kMaxGroups; ++i) {
    sg.wv[i] = u32x2{0u, 0u};
    if (i < R.my_groups) {  // uniform
      const int wl = (R.cw + R.wpt * i) * kGroupWords + 2 * (lane >> 4);
      sg.wv[i] = __builtin_amdgcn_raw_buffer_load_b64(
          mres, ((lane & 15) * wpr + R.w_begin + wl) * 4, 0, 0);
    }
  }
}

// kLoop: a wave may own more than kMaxGroups groups; they are taken in
// chunks of kMaxGroups, the next chunk's sign words loading while the
// current chunk's products run (the stream kernel, whose persistent
// workgroups cover long rows without splitting them into slabs).
template <bool kInX, bool kOutY, bool kHiLoCols, bool kMulti, bool kCoherent = false,
          bool kLoop = false>
__device__ __forceinline__ void stage_body(
    const uint32_t *__restrict__ M, const void *__restrict__ in,
    const uint16_t *__restrict__ s_in, const uint16_t *__restrict__ row_scale, int rows,
    int wpr, int slab_words, int b, int rt_log2_arg, int nslabs, int mode, int in_parts,
    void *__restrict__ out, float *__restrict__ part, uint32_t *__restrict__ cnt, int group,
    int slab, int red_off = 0, const SignRegs *pre = nullptr) {
  constexpr int kInAux = kCoherent ? kDeviceScope : 0;
  const int rt_log2 = kMulti ? rt_log2_arg : 0;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // scalar: wave-uniform
  const Role R = make_role(wave, group, slab, rt_log2, wpr, slab_words);
  const size_t K = (size_t)wpr * 32;
  const int w_begin = R.w_begin;
  const int w_count = R.w_count;

  // 1. Sign words of this wave's groups, one 8-byte load per lane and
  //    group, issued right after the input loads of step 2 (which mostly hit
  //    the caches; loads complete in order, so the conversion of the input
  //    need not wait for the signs to arrive from HBM), or first when the
  //    input is staged pass by pass.  Lanes past the last row or the
  //    slab's last word read data that never reaches a stored output: a
  //    ragged group's tail meets the zero slot on the B side, and rows past
  //    `rows` are not written.  Buffer range checking applies per dword, so
  //    a pair whose second word lies past the buffer still returns its first
  //    word (a second word past the row but inside the buffer is an
  //    out-of-slab word and meets the zero slot).  Only the wave's own
  //    groups are loaded, under a uniform branch: issuing out-of-range loads
  //    for the other groups instead (to avoid the branch) still sent them
  //    through the load path and cost 0.5 us of the 4096^2 layer at b=1.
  const int rho = lane & 15;
  const int q = lane >> 4;
  u32x2 wv[kMaxGroups];
  // sign words of groups c0 .. c0 + kMaxGroups - 1 into dst
  auto load_chunk = [&](u32x2 (&dst)[kMaxGroups], int c0) {
    const int64_t left = (int64_t)(rows - R.row0) * wpr * 4;
    const __amdgpu_buffer_rsrc_t mres = buffer_rsrc(M + (size_t)R.row0 * wpr, left);
#pragma unroll
    for (int i = 0; i < kMaxGroups; ++i) {
      dst[i] = u32x2{0u, 0u};
      if (c0 + i < R.my_groups) {  // uniform
        const int wl = (R.cw + R.wpt * (c0 + i)) * kGroupWords + 2 * q;
        dst[i] = __builtin_amdgcn_raw_buffer_load_b64(mres, (rho * wpr + w_begin + wl) * 4, 0, 0);
      }
    }
  };
  auto load_signs = [&]() {
    if (pre) {  // loaded ahead (same addresses as load_chunk(wv, 0))
#pragma unroll
      for (int i = 0; i < kMaxGroups; ++i) wv[i] = pre->wv[i];
      return;
    }
    load_chunk(wv, 0);
  };

  // 2. Stage the input columns as bf16 hi/lo (p, p+16) pairs, one 144-byte
  //    slot per (batch row, word); slot 0 holds zeros for lanes with no
  //    batch row and for the tail of a ragged group.  A unit is 8 columns
  //    (and their partners 16 on) of one batch row.  With one row tile per
  //    workgroup every wave stages exactly the columns of its own groups
  //    (and reads only what it wrote, the zero slot included, so no
  //    barrier is needed); with
  //    several, the waves of different tiles share columns and the
  //    workgroup stages the slab once, then meets a barrier.  A wave with
  //    no unit in a pass issues no load (out-of-range loads still occupy the
  //    load path); lanes without a unit in a wave that has some store to a
  //    scratch slot instead of branching, so that no load is moved behind
  //    another unit's wait.
  uint8_t *xs = lds + kSlot;
  // Every wave writes the zero slot itself: with one tile per workgroup no
  // barrier separates staging from the products, and a wave whose ragged
  // group tail points at the slot must see zeros written in its own program
  // order (the stores of other waves carry the same zeros).
  if (lane < kSlot / 16) reinterpret_cast<uint4 *>(lds)[lane] = make_uint4(0u, 0u, 0u, 0u);
  {
    constexpr bool shared = kMulti;
    const int per_group = b * kGroupWords * 2;  // units of one group
    const int nunits = shared ? b * 2 * w_count : R.my_groups * per_group;
    const int span = shared ? 2 * w_count : per_group;
    const float inv_span = 1.0f / (float)span;
    const int part_elems = b * (int)K;  // stride between partial input arrays
    const __amdgpu_buffer_rsrc_t xres =
        buffer_rsrc(in, (int64_t)b * K * (kInX ? 2 : 4) * (kInX ? 1 : in_parts));
    const __amdgpu_buffer_rsrc_t sres = buffer_rsrc(s_in, kInX ? (int64_t)K * 2 : 0);
    const bool two_parts = !kInX && in_parts > 1;
    const int bstride = row_stride(w_count);
    uint8_t *junk = xs + (size_t)b * bstride + (tid & 15) * kSlot;
    if (kHiLoCols && !shared && b == 1) {
      // One batch row: the 64 lanes share a group's 16 units, a quarter
      // unit each (columns c, c+1 and their partners c+16, c+17), so the
      // conversion costs a quarter of the per-lane instructions of whole
      // units.  Same values and layout as load_unit / store_unit.
      const int rem = lane >> 2, qq = lane & 3;
      const int qgroups = kLoop ? R.my_groups : kMaxGroups;
      for (int c0 = 0; c0 < qgroups; c0 += kMaxGroups) {
      u32x2 ra[kMaxGroups], rb[kMaxGroups], rc[kMaxGroups], rd[kMaxGroups];
      int dst_off[kMaxGroups];
#pragma unroll
      for (int i = 0; i < kMaxGroups; ++i) {
        if (c0 + i >= R.my_groups) break;  // uniform
        const int wl = (R.cw + R.wpt * (c0 + i)) * kGroupWords + (rem >> 1);
        const int col = (w_begin + wl) * 32 + 8 * (rem & 1) + 2 * qq;
        const bool valid = wl < w_count;
        dst_off[i] = valid ? wl * kSlot + 64 * (rem & 1) + 8 * qq : -1;
        if constexpr (kInX) {
          const int xo = valid ? col * 2 : kOob;
          ra[i][0] = __builtin_amdgcn_raw_buffer_load_b32(xres, xo, 0, kInAux);
          rb[i][0] = __builtin_amdgcn_raw_buffer_load_b32(xres, xo + 32, 0, kInAux);
          rc[i][0] = __builtin_amdgcn_raw_buffer_load_b32(sres, xo, 0, 0);
          rd[i][0] = __builtin_amdgcn_raw_buffer_load_b32(sres, xo + 32, 0, 0);
        } else {
          const int to = valid ? col * 4 : kOob;
          ra[i] = __builtin_amdgcn_raw_buffer_load_b64(xres, to, 0, kInAux);
          rb[i] = __builtin_amdgcn_raw_buffer_load_b64(xres, to + 64, 0, kInAux);
          if (two_parts) {
            const int to2 = valid ? (col + part_elems) * 4 : kOob;
            rc[i] = __builtin_amdgcn_raw_buffer_load_b64(xres, to2, 0, kInAux);
            rd[i] = __builtin_amdgcn_raw_buffer_load_b64(xres, to2 + 64, 0, kInAux);
          }
        }
      }
      if (c0 == 0) load_signs();
#pragma unroll
      for (int i = 0; i < kMaxGroups; ++i) {
        if (c0 + i >= R.my_groups) break;  // uniform
        float v[4];  // columns c, c+1, c+16, c+17
        if constexpr (kInX) {
          v[0] = bf16_to_f32(ra[i][0] & 0xffffu) * f16_to_f32((uint16_t)(rc[i][0] & 0xffffu));
          v[1] = bf16_to_f32(ra[i][0] >> 16) * f16_to_f32((uint16_t)(rc[i][0] >> 16));
          v[2] = bf16_to_f32(rb[i][0] & 0xffffu) * f16_to_f32((uint16_t)(rd[i][0] & 0xffffu));
          v[3] = bf16_to_f32(rb[i][0] >> 16) * f16_to_f32((uint16_t)(rd[i][0] >> 16));
        } else {
          v[0] = __uint_as_float(ra[i][0]);
          v[1] = __uint_as_float(ra[i][1]);
          v[2] = __uint_as_float(rb[i][0]);
          v[3] = __uint_as_float(rb[i][1]);
          if (two_parts) {
            v[0] += __uint_as_float(rc[i][0]);
            v[1] += __uint_as_float(rc[i][1]);
            v[2] += __uint_as_float(rd[i][0]);
            v[3] += __uint_as_float(rd[i][1]);
          }
        }
        const uint32_t h0 = pack_bf16x2(v[0], v[2]), h1 = pack_bf16x2(v[1], v[3]);
        const uint32_t l0 =
            pack_bf16x2(v[0] - bf16_to_f32(h0 & 0xffffu), v[2] - bf16_to_f32(h0 >> 16));
        const uint32_t l1 =
            pack_bf16x2(v[1] - bf16_to_f32(h1 & 0xffffu), v[3] - bf16_to_f32(h1 >> 16));
        uint8_t *dst = dst_off[i] >= 0 ? xs + dst_off[i] : junk + 64 * (rem & 1) + 8 * qq;
        *reinterpret_cast<uint2 *>(dst) = make_uint2(h0, h1);
        *reinterpret_cast<uint2 *>(dst + 32) = make_uint2(l0, l1);
      }
      }
    } else {
      load_signs();
      // pass stride and this thread's first unit
      const int stride = shared ? 2 * kThreads : 128;
      const int first = shared ? tid : lane;
      const int wave_first = shared ? 64 * wave : 0;
#pragma unroll
      for (int it = 0; it < (kLoop ? 1 << 20 : kStageIters); ++it) {
        const int base = it * stride;
        if (base >= nunits) break;  // uniform
        int slot_off[2], half[2], off[2], col[2];
        bool has[2];
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const int u = base + (stride >> 1) * k + first;
          has[k] = base + (stride >> 1) * k + wave_first < nunits;  // wave-uniform
          const bool ok = u < nunits;
          // u / span for u < 2^12: a float estimate, corrected by one step
          int q0 = (int)((float)u * inv_span);
          q0 -= q0 * span > u;
          q0 += (q0 + 1) * span <= u;
          q0 = ok ? q0 : 0;
          const int rem = u - q0 * span;
          int bb, wl;
          if (shared) {
            bb = q0;
            wl = rem >> 1;
            half[k] = rem & 1;
          } else {
            // q0 = the wave's group index i, rem = (batch row, word, half)
            bb = rem >> 4;
            wl = (R.cw + R.wpt * q0) * kGroupWords + ((rem & 15) >> 1);
            half[k] = rem & 1;
          }
          const bool valid = ok && wl < w_count;
          col[k] = (w_begin + wl) * 32 + 8 * half[k];
          off[k] = valid ? (int)(bb * K) + col[k] : kOob;
          slot_off[k] = valid ? bb * bstride + wl * kSlot : -1;
        }
        UnitRaw raw[2], rawb[2];
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          if (has[k]) {
            raw[k] = load_unit<kInX, kInAux>(xres, sres, off[k], col[k]);
            if (two_parts)
              rawb[k] = load_unit<kInX, kInAux>(xres, sres, off[k], col[k], part_elems);
          }
        }
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          if (has[k]) {
            float v[16];
            unit_values<kInX>(raw[k], v, two_parts ? &rawb[k] : nullptr);
            store_unit(slot_off[k] >= 0 ? xs + slot_off[k] : junk, half[k], v);
          }
        }
      }
    }
  }
  // Row scales of the outputs this thread writes at the end (loaded after
  // the staging loads so that waiting for them waits for nothing else).
  // Outputs o = tid + kThreads * k: row (o mod rows_per_wg) of the
  // workgroup's rows, batch row o / rows_per_wg.
  const int rows_log2 = 4 + rt_log2;
  const int rows_wg = 1 << rows_log2;
  const int row_wg0 = group * rows_wg;
  const int nout = rows_wg * b;
  // uniform, <= kMaxOutPerThread (one tile: 16 b <= 256 outputs)
  const int nk_out = kMulti ? (nout + kThreads - 1) / kThreads : 1;
  uint32_t rscale_bits[kMaxOutPerThread];
  if (pre) {
#pragma unroll
    for (int k = 0; k < kMaxOutPerThread; ++k) rscale_bits[k] = pre->rs[k];
  } else {
    load_row_scales(rscale_bits, row_scale, rows, group, rt_log2, b, nk_out);
  }
  if constexpr (kMulti)
    __syncthreads();  // the staged slab is complete
  else
    __builtin_amdgcn_wave_barrier();

  // 3. Products.  Step s = (group i = s / 2, word u = s % 2); independent
  //    accumulator chains per pair quad t (and per hi/lo when they are not
  //    in columns); the B operands of the next step are read from LDS while
  //    this step's MFMAs run.  Only lanes whose column carries a batch row
  //    read LDS; the others keep zero operands.
  const int ncol = lane & 15;
  const int beta = kHiLoCols ? (ncol >> 1) : ncol;
  const int hl_col = kHiLoCols ? (ncol & 1) : 0;
  uint32_t kSignMask, kOne;
  asm volatile("v_mov_b32 %0, 0x80008000" : "=v"(kSignMask));
  asm volatile("v_mov_b32 %0, 0x3f803f80" : "=v"(kOne));
  constexpr int kChains = kHiLoCols ? 1 : 2;
  constexpr int kReads = 4 * kChains;
  floatx4 acc[4][kChains];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int hl = 0; hl < kChains; ++hl) acc[t][hl] = floatx4{0.f, 0.f, 0.f, 0.f};
  const bool b_lane = beta < b;
  // LDS offset of B operand k = 4 * hl + t (pair quad t of the hi or lo part)
  // within a slot: quads 0, 1 are half 0 and quads 2, 3 half 1
  auto b_off = [](int k) {
    const int hl = kHiLoCols ? 0 : (k >> 2), t = k & 3;
    return 16 * (4 * (t >> 1) + 2 * hl + (t & 1));
  };
  // the products of the wave's groups c0 .. c0 + kMaxGroups - 1 (sign words w)
  auto products = [&](const u32x2 (&w)[kMaxGroups], int c0, int nsteps) {
    auto b_ptr = [&](int st) -> const uint8_t * {
      const int wl = (R.cw + R.wpt * (c0 + (st >> 1))) * kGroupWords + 2 * q + (st & 1);
      return wl < w_count ? xs + (size_t)beta * row_stride(w_count) + wl * kSlot + 32 * hl_col
                          : lds;
    };
    uint4 bop[2][kReads];
#pragma unroll
    for (int k = 0; k < kReads; ++k) bop[0][k] = bop[1][k] = make_uint4(0u, 0u, 0u, 0u);
    if (nsteps > 0 && b_lane) {
      const uint8_t *bs = b_ptr(0);
#pragma unroll
      for (int k = 0; k < kReads; ++k) bop[0][k] = *reinterpret_cast<const uint4 *>(bs + b_off(k));
    }
    static_for<kMaxGroups * 2>([&](auto ST) {
      constexpr int st = decltype(ST)::value;
      constexpr int cur = st & 1;
      if (st < nsteps) {  // wave-uniform
        if (st + 1 < nsteps && b_lane) {
          const uint8_t *bs = b_ptr(st + 1);
#pragma unroll
          for (int k = 0; k < kReads; ++k)
            bop[cur ^ 1][k] = *reinterpret_cast<const uint4 *>(bs + b_off(k));
        }
        const uint32_t wd = w[st >> 1][st & 1];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          uint4 a;
          a.x = ((wd << (15 - (4 * t + 0))) & kSignMask) | (kOne & ~kSignMask);
          a.y = ((wd << (15 - (4 * t + 1))) & kSignMask) | (kOne & ~kSignMask);
          a.z = ((wd << (15 - (4 * t + 2))) & kSignMask) | (kOne & ~kSignMask);
          a.w = ((wd << (15 - (4 * t + 3))) & kSignMask) | (kOne & ~kSignMask);
          const bf16x8 av = __builtin_bit_cast(bf16x8, a);
#pragma unroll
          for (int hl = 0; hl < kChains; ++hl)
            acc[t][hl] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                av, __builtin_bit_cast(bf16x8, bop[cur][4 * hl + t]), acc[t][hl], 0, 0, 0);
        }
      }
    });
  };
  if constexpr (kLoop) {
    const int nchunks = (R.my_groups + kMaxGroups - 1) / kMaxGroups;
    for (int chunk = 0; chunk < nchunks; ++chunk) {
      const int c0 = chunk * kMaxGroups;
      u32x2 wnext[kMaxGroups];
      if (chunk + 1 < nchunks) load_chunk(wnext, c0 + kMaxGroups);
      products(wv, c0, min(R.my_groups - c0, kMaxGroups) * 2);
      if (chunk + 1 < nchunks) {
#pragma unroll
        for (int i = 0; i < kMaxGroups; ++i) wv[i] = wnext[i];
      }
    }
  } else {
    products(wv, 0, R.my_groups * 2);
  }
  floatx4 tot = acc[0][0];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int hl = 0; hl < kChains; ++hl)
      if (t | hl) tot += acc[t][hl];

  // 4. Add the 16x16 tiles of the waves that share a row tile, through LDS
  //    (after every wave is done reading the staged input).  Accumulator
  //    layout: lane l holds rows 4*(l/16) + i (i = 0..3) of column l mod 16.
  //    With red_off > 0 the tiles go to their own LDS region past the staged
  //    input, and only one barrier is needed.
  if (red_off == 0) __syncthreads();  // uniform
  reinterpret_cast<float4 *>(lds + red_off)[wave * kRedLanes + lane + (lane >> 4)] =
      make_float4(tot[0], tot[1], tot[2], tot[3]);
  __syncthreads();
  const float *redf = reinterpret_cast<const float *>(lds + red_off);
  float sum[kMaxOutPerThread];
#pragma unroll
  for (int k = 0; k < kMaxOutPerThread; ++k) {
    sum[k] = 0.f;
    if (k >= nk_out) break;
    const int o = tid + kThreads * k;
    if (o < nout) {
      const int r_wg = o & (rows_wg - 1);
      const int obeta = o >> rows_log2;
      const int rt = r_wg >> 4, orow_l = r_wg & 15;
      const int c0 = kHiLoCols ? 2 * obeta : obeta;
      const int l0 = 16 * (orow_l >> 2) + (c0 & 15);
#pragma unroll
      for (int c = 0; c < kWaves; ++c) {
        if (c >= R.wpt) break;
        const int wv2 = rt * R.wpt + c;
        const int ri = (wv2 * kRedLanes + l0 + (l0 >> 4)) * 4 + (orow_l & 3);
        sum[k] += redf[ri];
        if constexpr (kHiLoCols) sum[k] += redf[ri + 4];  // column l0 + 1, same 16 lanes
      }
    }
  }

  if (mode == kModeLastSlab) {
    // Publish this slab's partial sums; the last slab of the workgroup's
    // rows to arrive adds all partials in slab order and resets the counter.
#pragma unroll
    for (int k = 0; k < kMaxOutPerThread; ++k) {
      if (k >= nk_out) break;
      const int o = tid + kThreads * k;
      const int orow = row_wg0 + (o & (rows_wg - 1));
      if (o < nout && orow < rows)
        store_device(&part[((size_t)slab * b + (o >> rows_log2)) * rows + orow], sum[k]);
    }
    wait_memory();
    __syncthreads();
    __shared__ uint32_t s_last;
    if (tid == 0)
      s_last = __hip_atomic_fetch_add(&cnt[group], 1u, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT) == (uint32_t)(nslabs - 1);
    __syncthreads();
    if (!s_last) return;
    // Device-scope loads of every slab's partial, issued before any is
    // added (the slab count is small: at most kMaxSlabsLoaded per pass).
    const __amdgpu_buffer_rsrc_t pres = buffer_rsrc(part, (int64_t)nslabs * b * rows * 4);
#pragma unroll
    for (int k = 0; k < kMaxOutPerThread; ++k) {
      if (k >= nk_out) break;
      const int o = tid + kThreads * k;
      const int orow = row_wg0 + (o & (rows_wg - 1));
      const bool mine = o < nout && orow < rows;
      const int off0 = mine ? ((o >> rows_log2) * rows + orow) * 4 : kOob;
      float acc_s = 0.f;
      for (int sl0 = 0; sl0 < nslabs; sl0 += kMaxSlabsLoaded) {
        float pv[kMaxSlabsLoaded];
#pragma unroll
        for (int q = 0; q < kMaxSlabsLoaded; ++q) {
          const int sl = sl0 + q;
          const int off = (sl < nslabs && off0 != kOob) ? off0 + sl * b * rows * 4 : kOob;
          pv[q] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(pres, off, 0,
                                                                                 kDeviceScope));
        }
#pragma unroll
        for (int q = 0; q < kMaxSlabsLoaded; ++q) acc_s += pv[q];
      }
      sum[k] = acc_s;
    }
    if (tid == 0) __hip_atomic_store(&cnt[group], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
#pragma unroll
  for (int k = 0; k < kMaxOutPerThread; ++k) {
    if (k > 0 && k >= nk_out) break;
    const int o = tid + kThreads * k;
    const int orow = row_wg0 + (o & (rows_wg - 1));
    const float v = sum[k] * f16_to_f32((uint16_t)rscale_bits[k]);
    if (o < nout && orow < rows) {
      size_t oi = (size_t)(o >> rows_log2) * rows + orow;
      if (mode == kModePartial) oi += (size_t)slab * b * rows;
      if constexpr (kCoherent) {
        if constexpr (kOutY)
          store_device_u16(static_cast<uint16_t *>(out) + oi, f32_to_bf16(v));
        else
          store_device(static_cast<float *>(out) + oi, v);
      } else {
        if constexpr (kOutY)
          static_cast<uint16_t *>(out)[oi] = f32_to_bf16(v);
        else
          static_cast<float *>(out)[oi] = v;
      }
    }
  }
}

// One stage of one layer: row group (blockIdx.x), slab (blockIdx.y).
// Arguments are scalars, most urgent first, so that they are preloaded into
// SGPRs at wave launch instead of being fetched from the kernarg segment.
template <bool kInX, bool kOutY, bool kHiLoCols, bool kMulti>
__global__ __launch_bounds__(kThreads) void gemv_stage_kernel(
    const uint32_t *__restrict__ M, const void *__restrict__ in,
    const uint16_t *__restrict__ s_in, const uint16_t *__restrict__ row_scale, int rows,
    int wpr, int slab_words, int b, int rt_log2, int nslabs, int mode, int in_parts,
    void *__restrict__ out, float *__restrict__ part, uint32_t *__restrict__ cnt, int red_off) {
  stage_body<kInX, kOutY, kHiLoCols, kMulti>(M, in, s_in, row_scale, rows, wpr, slab_words, b,
                                             rt_log2, nslabs, mode, in_parts, out, part, cnt,
                                             (int)blockIdx.x, (int)blockIdx.y, red_off);
}

// One stage of several layers that share the input width (the segments):
// the row groups of segment s are blockIdx.x in [group_end[s-1],
// group_end[s]).  Each layer keeps its own sign matrix, scales, input and
// output; the plan (rows per workgroup, slab, mode) is common, with one
// slab (no last-slab reduction).
constexpr int kMaxSegs = 4;
struct Segs {
  int count;
  int group_end[kMaxSegs];
  int rows[kMaxSegs];
  int wpr[kMaxSegs];
  const uint32_t *M[kMaxSegs];
  const void *in[kMaxSegs];
  const uint16_t *s_in[kMaxSegs];
  const uint16_t *row_scale[kMaxSegs];
  void *out[kMaxSegs];
};

template <bool kInX, bool kOutY, bool kHiLoCols, bool kMulti>
__global__ __launch_bounds__(kThreads) void gemv_segs_kernel(const Segs segs, int slab_words,
                                                             int b, int rt_log2, int mode,
                                                             int in_parts) {
  const int g = (int)blockIdx.x;
  int sg = 0;
#pragma unroll
  for (int i = 0; i + 1 < kMaxSegs; ++i)
    if (i + 1 < segs.count && g >= segs.group_end[i]) sg = i + 1;
  const int g0 = sg > 0 ? segs.group_end[sg - 1] : 0;
  stage_body<kInX, kOutY, kHiLoCols, kMulti>(
      segs.M[sg], segs.in[sg], segs.s_in[sg], segs.row_scale[sg], segs.rows[sg], segs.wpr[sg],
      slab_words, b, rt_log2, 1, mode, in_parts, segs.out[sg], nullptr, nullptr, g - g0,
      (int)blockIdx.y);
}

size_t lds_stage_bytes(int64_t b, int slab_words) {
  // zero slot, staged slots, 16 scratch slots for lanes without a unit
  return (size_t)kSlot * 17 + (size_t)b * row_stride(slab_words);
}

size_t lds_bytes_for(int64_t b, int slab_words) {
  const size_t stage = lds_stage_bytes(b, slab_words);
  return stage > (size_t)kRedBytes ? stage : (size_t)kRedBytes;
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// Static LDS (the kernel's __shared__ variables) of a kernel, looked up once.
int static_lds_bytes(const void *fn) {
  static std::mutex mu;
  static std::vector<std::pair<const void *, int>> known;
  std::lock_guard<std::mutex> lock(mu);
  for (const auto &e : known)
    if (e.first == fn) return e.second;
  hipFuncAttributes a{};
  const int bytes = hipFuncGetAttributes(&a, fn) == hipSuccess ? (int)a.sharedSizeBytes : -1;
  known.emplace_back(fn, bytes);
  return bytes;
}

// A launch requests the kernel's static LDS plus `dynamic`; both must fit
// one compute unit, or no workgroup could ever be placed.
bool launch_fits(const void *fn, size_t dynamic) {
  const int st = static_lds_bytes(fn);
  return st >= 0 && (size_t)st + dynamic <= (size_t)kLdsPerCu;
}

// How one stage is split over workgroups.
//  rt_log2: rows per workgroup = 16 << rt_log2.  More rows per workgroup
//    share one staged copy of the input (its conversion and its reads are
//    paid once per workgroup), which matters as the batch grows; fewer rows
//    per workgroup spread a small stage over more compute units.
//  slab_words: columns (in words) per workgroup; at most what one wave's
//    groups and the LDS budget allow.  Several slabs are added by the last
//    one to finish, or (stage 1, few row tiles, small batch) each writes a
//    partial result that the next stage adds while staging.
struct StagePlan {
  int rt_log2, slab_words, nslabs, mode;
};

int max_slab_words(int64_t b, int rt_log2) {
  int64_t w = ((kLdsBudget - 17 * kSlot) / b - 16) / kSlot;
  const int64_t per_waves = (int64_t)kMaxGroups * kGroupWords * (kWaves >> rt_log2);
  if (w > per_waves) w = per_waves;
  return (int)(w - w % kGroupWords);
}

StagePlan plan_slabs(int64_t rows, int64_t wpr, int64_t b, int rt, bool allow_partial, int cus);

StagePlan plan_stage(int64_t rows, int64_t wpr, int64_t b, bool allow_partial, int cus) {
  const int64_t tiles = (rows + kTileRows - 1) / kTileRows;
  // Preferred tiles per workgroup for this batch (input shared over more
  // rows as b grows), then: no more workgroups than two per compute unit,
  // no fewer than half a workgroup per compute unit, at most
  // kMaxOutPerThread outputs per thread.
  int want = b >= 8 ? 3 : (b >= 4 ? 2 : (b >= 2 ? 1 : 0));
  int rt = 0;
  auto wgs = [&](int r) {
    const int sw = max_slab_words(b, r);
    const int64_t ns = (wpr + sw - 1) / sw;
    return ((tiles + (1 << r) - 1) >> r) * ns;
  };
  while (rt < 3 && (((tiles + (1 << rt) - 1) >> rt) > 2 * cus)) ++rt;
  while (rt < want && wgs(rt + 1) >= cus / 2) ++rt;
  while (((int64_t)kTileRows << rt) * b > (int64_t)kThreads * kMaxOutPerThread) --rt;
  return plan_slabs(rows, wpr, b, rt, allow_partial, cus);
}

// The column split of a stage whose workgroups own 16 << rt rows.
StagePlan plan_slabs(int64_t rows, int64_t wpr, int64_t b, int rt, bool allow_partial, int cus) {
  const int64_t tiles = (rows + kTileRows - 1) / kTileRows;
  StagePlan p{rt, 0, 0, kModeFinal};
  int sw = max_slab_words(b, rt);
  if (rt == 0) {
    // per-wave staging: at most kWaveStageUnits units (groups x b x 16) per wave
    const int groups_per_wave = kWaveStageUnits / (int)(b * kGroupWords * 2);
    const int cap = groups_per_wave * kGroupWords * kWaves;
    if (sw > cap) sw = cap;
  }
  p.slab_words = (int)(sw < wpr ? sw : ((wpr + kGroupWords - 1) / kGroupWords) * kGroupWords);
  p.nslabs = (int)((wpr + p.slab_words - 1) / p.slab_words);
  if (p.nslabs > 1) {
    p.mode = kModeLastSlab;
    return p;
  }
  const int64_t groups = (wpr + kGroupWords - 1) / kGroupWords;
  // Few row tiles: split the columns in two (more workgroups share the
  // latency-bound work).  Long rows split even when the tiles nearly fill
  // the device (per-workgroup sign expansion then dominates).
  if (allow_partial && rt == 0 && (tiles < 192 || (tiles < cus && wpr >= 256)) && groups >= 2 &&
      b <= 8) {
    p.slab_words = (int)(((groups + 1) / 2) * kGroupWords);
    p.nslabs = (int)((wpr + p.slab_words - 1) / p.slab_words);
    p.mode = p.nslabs > 1 ? kModePartial : kModeFinal;
  }
  return p;
}

struct WsLayout {
  StagePlan p1, p2;
  size_t t, part1, cnt1, part2, cnt2, total;
};

// Workspace: a fixed header, then the shape-dependent arrays.  The header
// holds the arrival counters (one per workgroup row group of each stage),
// which must be zero at the start of a call, at offsets that do not depend
// on the shape, so that calls of different shapes can share one workspace
// without their arrays ever overlapping another shape's counters.
constexpr size_t kMaxTiles = ((size_t)1 << 20) / kTileRows;  // rows <= 2^20
constexpr size_t kHeaderBytes = 2 * kMaxTiles * 4;

WsLayout ws_layout(int64_t m, int64_t n, int64_t r, int64_t b, int cus) {
  WsLayout L{};
  L.p1 = plan_stage(r, n / 32, b, true, cus);
  L.p2 = plan_stage(m, r / 32, b, false, cus);
  L.cnt1 = 0;
  L.cnt2 = kMaxTiles * 4;
  const int tparts = L.p1.mode == kModePartial ? L.p1.nslabs : 1;
  size_t off = kHeaderBytes;
  L.t = off;
  off += align256((size_t)tparts * b * r * 4);
  L.part1 = off;
  if (L.p1.mode == kModeLastSlab) off += align256((size_t)L.p1.nslabs * b * r * 4);
  L.part2 = off;
  if (L.p2.mode == kModeLastSlab) off += align256((size_t)L.p2.nslabs * b * m * 4);
  L.total = off;
  return L;
}

struct StageArgs {
  const uint32_t *M;
  const void *in;
  const uint16_t *s_in;
  const uint16_t *row_scale;
  int rows, wpr, b, in_parts;
  void *out;
  float *part;
  uint32_t *cnt;
};

template <bool kInX, bool kOutY>
hipError_t launch_stage(const StageArgs &a, const StagePlan &p, hipStream_t s) {
  const int rows_wg = kTileRows << p.rt_log2;
  if ((int64_t)rows_wg * a.b > (int64_t)kThreads * kMaxOutPerThread) return hipErrorInvalidValue;
  dim3 grid((unsigned)((a.rows + rows_wg - 1) / rows_wg), (unsigned)p.nslabs);
  const bool multi = p.rt_log2 > 0;
  size_t lds = lds_bytes_for(a.b, p.slab_words < a.wpr ? p.slab_words : a.wpr);
  // One row tile per workgroup: the cross-wave sums get their own LDS region
  // past the staged input when it fits (one barrier instead of two).
  int red_off = 0;
  if (!multi) {
    const size_t stage = (lds_stage_bytes(a.b, p.slab_words < a.wpr ? p.slab_words : a.wpr) + 15) &
                         ~(size_t)15;
    if (stage + kRedBytes <= (size_t)kLdsBudget) {
      red_off = (int)stage;
      lds = stage + kRedBytes;
    }
  }
  auto go = [&](auto kernel) -> hipError_t {
    if (!launch_fits(reinterpret_cast<const void *>(kernel), lds)) return hipErrorInvalidValue;
    kernel<<<grid, kThreads, lds, s>>>(a.M, a.in, a.s_in, a.row_scale, a.rows, a.wpr,
                                       p.slab_words, a.b, p.rt_log2, p.nslabs, p.mode,
                                       a.in_parts, a.out, a.part, a.cnt, red_off);
    return hipGetLastError();
  };
  if (a.b <= 8)
    return multi ? go(gemv_stage_kernel<kInX, kOutY, true, true>)
                 : go(gemv_stage_kernel<kInX, kOutY, true, false>);
  return multi ? go(gemv_stage_kernel<kInX, kOutY, false, true>)
               : go(gemv_stage_kernel<kInX, kOutY, false, false>);
}

template <bool kInX, bool kOutY>
hipError_t launch_segs(const Segs &sg, const StagePlan &p, int b, int max_wpr, int in_parts,
                       hipStream_t s) {
  const size_t lds = lds_bytes_for(b, p.slab_words < max_wpr ? p.slab_words : max_wpr);
  dim3 grid((unsigned)sg.group_end[sg.count - 1], (unsigned)p.nslabs);
  auto go = [&](auto kernel) -> hipError_t {
    if (!launch_fits(reinterpret_cast<const void *>(kernel), lds)) return hipErrorInvalidValue;
    kernel<<<grid, kThreads, lds, s>>>(sg, p.slab_words, b, p.rt_log2, p.mode, in_parts);
    return hipGetLastError();
  };
  const bool multi = p.rt_log2 > 0;
  if (b <= 8)
    return multi ? go(gemv_segs_kernel<kInX, kOutY, true, true>)
                 : go(gemv_segs_kernel<kInX, kOutY, true, false>);
  return multi ? go(gemv_segs_kernel<kInX, kOutY, false, true>)
               : go(gemv_segs_kernel<kInX, kOutY, false, false>);
}

// Several layers sharing n in two launches: the stage plans are made for
// the summed rows (stage 2 for the widest rank), and apply when neither
// stage needs a last-slab reduction.
struct MultiLayout {
  StagePlan p1, p2;
  bool fused;
  size_t t[kMaxSegs];
  size_t total;
};

MultiLayout multi_layout(const int64_t *m, const int64_t *r, int count, int64_t n, int64_t b,
                         int cus) {
  MultiLayout L{};
  int64_t rows1 = 0, rows2 = 0, wpr2 = 0;
  for (int i = 0; i < count; ++i) {
    rows1 += r[i];
    rows2 += m[i];
    if (r[i] / 32 > wpr2) wpr2 = r[i] / 32;
  }
  L.p1 = plan_stage(rows1, n / 32, b, true, cus);
  L.p2 = plan_stage(rows2, wpr2, b, false, cus);
  L.fused = L.p1.mode != kModeLastSlab && L.p2.mode == kModeFinal;
  const int tparts = L.p1.mode == kModePartial ? L.p1.nslabs : 1;
  size_t off = kHeaderBytes;
  for (int i = 0; i < count; ++i) {
    L.t[i] = off;
    off += align256((size_t)tparts * b * r[i] * 4);
  }
  L.total = off;
  // the per-layer fallback reuses the workspace one layer at a time
  for (int i = 0; i < count; ++i) {
    const size_t one = ws_layout(m[i], n, r[i], b, cus).total;
    if (one > L.total) L.total = one;
  }
  return L;
}

}  // namespace

// Compute units of the current device, queried once per device.
int device_cus() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
  if (dev < 64) {
    const int c = cache[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    return 256;
  if (dev < 64) cache[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

size_t gemv_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t b) {
  return ws_layout(m, n, r, b, device_cus()).total;
}

size_t gemv_multi_workspace_bytes(const int64_t *m, const int64_t *r, int count, int64_t n,
                                  int64_t b) {
  return multi_layout(m, r, count, n, b, device_cus()).total;
}

hipError_t launch_gemv_multi(int count, const int64_t *m, const int64_t *r, int64_t n,
                             const uint32_t *const *Bu, const uint32_t *const *Bv,
                             const uint16_t *const *s_out, const uint16_t *const *s_mid,
                             const uint16_t *const *s_in, const uint16_t *x, int64_t b,
                             uint16_t *const *y, void *ws, hipStream_t s) {
  if (count < 1 || count > kMaxSegs) return hipErrorInvalidValue;
  const MultiLayout L = multi_layout(m, r, count, n, b, device_cus());
  if (!L.fused) {
    for (int i = 0; i < count; ++i) {
      const hipError_t e =
          launch_gemv(m[i], n, r[i], Bu[i], Bv[i], s_out[i], s_mid[i], s_in[i], x, b, y[i], ws, s);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  uint8_t *base = static_cast<uint8_t *>(ws);
  const int tparts = L.p1.mode == kModePartial ? L.p1.nslabs : 1;
  Segs s1{}, s2{};
  s1.count = s2.count = count;
  const int rw1 = kTileRows << L.p1.rt_log2, rw2 = kTileRows << L.p2.rt_log2;
  int g1 = 0, g2 = 0, wpr2 = 0;
  for (int i = 0; i < count; ++i) {
    float *t = reinterpret_cast<float *>(base + L.t[i]);
    g1 += (int)((r[i] + rw1 - 1) / rw1);
    g2 += (int)((m[i] + rw2 - 1) / rw2);
    s1.group_end[i] = g1;
    s2.group_end[i] = g2;
    s1.rows[i] = (int)r[i];
    s1.wpr[i] = (int)(n / 32);
    s1.M[i] = Bv[i];
    s1.in[i] = x;
    s1.s_in[i] = s_in[i];
    s1.row_scale[i] = s_mid[i];
    s1.out[i] = t;
    s2.rows[i] = (int)m[i];
    s2.wpr[i] = (int)(r[i] / 32);
    s2.M[i] = Bu[i];
    s2.in[i] = t;
    s2.s_in[i] = nullptr;
    s2.row_scale[i] = s_out[i];
    s2.out[i] = y[i];
    if (s2.wpr[i] > wpr2) wpr2 = s2.wpr[i];
  }
  hipError_t e = launch_segs<true, false>(s1, L.p1, (int)b, (int)(n / 32), 1, s);
  if (e != hipSuccess) return e;
  return launch_segs<false, true>(s2, L.p2, (int)b, wpr2, tparts, s);
}

namespace {
__global__ void zero_words_kernel(uint32_t *__restrict__ p, int count) {
  const int i = (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (i < count) p[i] = 0u;
}
}  // namespace

hipError_t launch_gemv_clear_counters(int64_t m, int64_t n, int64_t r, int64_t b, void *ws,
                                      hipStream_t s) {
  const WsLayout L = ws_layout(m, n, r, b, device_cus());
  uint8_t *base = static_cast<uint8_t *>(ws);
  const StagePlan *plans[2] = {&L.p1, &L.p2};
  const size_t offs[2] = {L.cnt1, L.cnt2};
  const int64_t rows[2] = {r, m};
  for (int k = 0; k < 2; ++k) {
    if (plans[k]->mode != kModeLastSlab) continue;
    const int64_t rows_wg = (int64_t)kTileRows << plans[k]->rt_log2;
    const int groups = (int)((rows[k] + rows_wg - 1) / rows_wg);
    zero_words_kernel<<<(unsigned)((groups + 255) / 256), 256, 0, s>>>(
        reinterpret_cast<uint32_t *>(base + offs[k]), groups);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_gemv(int64_t m, int64_t n, int64_t r, const uint32_t *Bu,
                       const uint32_t *Bv, const uint16_t *s_out,
                       const uint16_t *s_mid, const uint16_t *s_in,
                       const uint16_t *x, int64_t b, uint16_t *y, void *ws,
                       hipStream_t s) {
  const WsLayout L = ws_layout(m, n, r, b, device_cus());
  uint8_t *base = static_cast<uint8_t *>(ws);
  float *t = reinterpret_cast<float *>(base + L.t);
  const StageArgs s1{Bv, x, s_in, s_mid, (int)r, (int)(n / 32), (int)b, 1, t,
                     reinterpret_cast<float *>(base + L.part1),
                     reinterpret_cast<uint32_t *>(base + L.cnt1)};
  hipError_t e = launch_stage<true, false>(s1, L.p1, s);
  if (e != hipSuccess) return e;
  const int tparts = L.p1.mode == kModePartial ? L.p1.nslabs : 1;
  const StageArgs s2{Bu, t, nullptr, s_out, (int)m, (int)(r / 32), (int)b, tparts, y,
                     reinterpret_cast<float *>(base + L.part2),
                     reinterpret_cast<uint32_t *>(base + L.cnt2)};
  return launch_stage<false, true>(s2, L.p2, s);
}

// ---------------------------------------------------------------------------
// Layer stream: the decode forward of a sequence of layers in one persistent
// launch.  A decoder step at batch 1 runs dozens of small, dependent
// products; as separate launches each pays a kernel boundary (about 1.6 us
// in a replayed graph) and a cold start.  Here one grid of workgroups (one
// 512-thread workgroup per compute unit, all resident) walks a precomputed
// plan of phases.  A phase is a set of stage segments (the first or second product
// of one layer) whose row groups are spread over the workgroups; phases are
// separated by a grid barrier: every workgroup writes its arrival word and
// polls all of them, with device-scope stores and loads and no atomic
// read-modify-write, so no arrival waits for another (an uncontended
// hand-off between compute units measured about 0.3 us within an XCD and
// 0.4 us across XCDs).  Outputs that later phases read are written and read
// at device scope.  Layers marked `wait` start after every earlier layer of
// the call has finished (they may read those layers' outputs); the first
// product of a layer that does not wait shares a phase with the second
// product of the layer group before it.
// ---------------------------------------------------------------------------
namespace {

constexpr uint32_t kStreamMagic = 0xAF15EA01u;
constexpr int kStreamThreads = kThreads;
constexpr int kStreamMaxGroupItems = 8;  // layers per group (a phase holds up to two groups)
constexpr int kStreamMaxGrid = 512;     // workgroups (one per compute unit)
constexpr int kSpinLimit = 1 << 20;      // polls per barrier before giving up
// workspace header (uint32 words): epoch, error, arrival words
constexpr int kSyncEpoch = 0, kSyncError = 1, kSyncFlags = 64;
constexpr size_t kStreamHeaderBytes = (size_t)(kSyncFlags + 8 * kStreamMaxGrid) * 4;

struct StreamSeg {
  const uint32_t *M;
  const void *in;
  const uint16_t *s_in;
  const uint16_t *row_scale;
  void *out;
  float *part;
  uint32_t *cnt;
  int32_t kind;  // 0: first product (x in, t out); 1: second (t in, y out)
  int32_t rows, wpr, slab_words, rt_log2, nslabs, mode, in_parts, red_off;
  int32_t groups;                // row groups (workgroup tasks per slab)
  int32_t task_begin, task_end;  // this segment's tasks within its phase
};

struct StreamPhase {
  int32_t seg_begin, seg_end, tasks, pad;
};

struct StreamHeader {
  uint32_t magic, version;
  int32_t nphases, nsegs, b, lds_bytes;
  int32_t max_tasks, pad;
  uint64_t plan_bytes, ws_bytes;
  void *ws;  // the workspace the plan's pointers lie in
};

size_t stream_plan_size(int nphases, int nsegs) {
  return sizeof(StreamHeader) + (size_t)nphases * sizeof(StreamPhase) +
         (size_t)nsegs * sizeof(StreamSeg);
}

__device__ __forceinline__ uint32_t load_device_u32(const uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_device_u32(uint32_t *p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Grid barrier number `target`, in two halves so that a workgroup can issue
// the next phase's weight loads while it waits.  Arrival words only grow, so
// a word at or past the target has arrived.  Each workgroup writes its word
// into kFlagReplicas copies and polls one copy (workgroup w polls copy w mod
// kFlagReplicas), so the pollers spread over several memory lines instead
// of all reading the same ones; two polls are kept in flight.
constexpr int kFlagReplicas = 8;
static_assert(kStreamHeaderBytes >= (size_t)(kSyncFlags + kFlagReplicas * kStreamMaxGrid) * 4,
              "arrival words fit the header");

// Every wave first waits for its own memory operations, so the phase's
// stores are complete before the arrival word is written.
__device__ __forceinline__ void barrier_arrive(uint32_t *sync, uint32_t target) {
  wait_memory();
  __syncthreads();
  if (threadIdx.x < kFlagReplicas)
    store_device_u32(sync + kSyncFlags + threadIdx.x * kStreamMaxGrid + blockIdx.x, target);
}

// Returns false when the error word is set (a wait timed out here or
// elsewhere); every wave then leaves the phase loop.
__device__ bool barrier_wait(uint32_t *sync, uint32_t target) {
  __shared__ uint32_t s_ok;
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    const int G = (int)gridDim.x;
    const __amdgpu_buffer_rsrc_t fres = buffer_rsrc(
        sync + kSyncFlags + (blockIdx.x % kFlagReplicas) * kStreamMaxGrid, (int64_t)G * 4);
    auto poll = [&](uint32_t (&f)[kStreamMaxGrid / 64]) {
#pragma unroll
      for (int k = 0; k < kStreamMaxGrid / 64; ++k) {
        const int w = 64 * k + lane;
        f[k] = target;
        if (64 * k < G)  // uniform
          f[k] = __builtin_amdgcn_raw_buffer_load_b32(fres, w < G ? w * 4 : kOob, 0, kDeviceScope);
      }
    };
    auto arrived = [&](const uint32_t (&f)[kStreamMaxGrid / 64]) {
      bool mine = true;
#pragma unroll
      for (int k = 0; k < kStreamMaxGrid / 64; ++k)
        mine = mine && (64 * k + lane >= G || (int)(f[k] - target) >= 0);
      return __all(mine);
    };
    bool ok = true;
    uint32_t fa[kStreamMaxGrid / 64], fb[kStreamMaxGrid / 64];
    poll(fa);
    for (int it = 0;; it += 2) {
      poll(fb);
      if (arrived(fa)) break;
      poll(fa);
      if (arrived(fb)) break;
      if (load_device_u32(sync + kSyncError) != 0u) {
        ok = false;
        break;
      }
      if (it >= kSpinLimit) {
        if (lane == 0) store_device_u32(sync + kSyncError, 1u);
        ok = false;
        break;
      }
    }
    if (lane == 0) s_ok = ok ? 1u : 0u;
  }
  __syncthreads();
  return s_ok != 0u;
}

template <bool kHiLo>
__device__ __forceinline__ void stream_task(const StreamSeg &g, int b, int task,
                                            const SignRegs &pre) {
  const int local = task - g.task_begin;
  const int group = local % g.groups;
  const int slab = local / g.groups;
  if (g.kind == 0) {
    if (g.rt_log2 > 0)
      stage_body<true, false, kHiLo, true, true, true>(g.M, g.in, g.s_in, g.row_scale, g.rows, g.wpr,
                                                 g.slab_words, b, g.rt_log2, g.nslabs, g.mode,
                                                 g.in_parts, g.out, g.part, g.cnt, group, slab,
                                                 g.red_off, &pre);
    else
      stage_body<true, false, kHiLo, false, true, true>(g.M, g.in, g.s_in, g.row_scale, g.rows, g.wpr,
                                                  g.slab_words, b, 0, g.nslabs, g.mode,
                                                  g.in_parts, g.out, g.part, g.cnt, group, slab,
                                                  g.red_off, &pre);
  } else {
    if (g.rt_log2 > 0)
      stage_body<false, true, kHiLo, true, true, true>(g.M, g.in, g.s_in, g.row_scale, g.rows, g.wpr,
                                                 g.slab_words, b, g.rt_log2, g.nslabs, g.mode,
                                                 g.in_parts, g.out, g.part, g.cnt, group, slab,
                                                 g.red_off, &pre);
    else
      stage_body<false, true, kHiLo, false, true, true>(g.M, g.in, g.s_in, g.row_scale, g.rows, g.wpr,
                                                  g.slab_words, b, 0, g.nslabs, g.mode,
                                                  g.in_parts, g.out, g.part, g.cnt, group, slab,
                                                  g.red_off, &pre);
  }
}

// The persistent walk over the plan's phases.  Task t of a phase runs on
// workgroup t mod grid; a workgroup with no task in a phase goes straight to
// the barrier.  A workgroup reads the plan entry of its next task and loads
// that task's sign words as soon as it has arrived at the barrier before it
// (weights do not depend on the phase's outputs), so the HBM latency of the
// signs overlaps the wait.  The epoch (the arrival value of the call's first
// barrier minus one) is read by every workgroup before its first arrival,
// and advanced by workgroup 0 once every workgroup has passed the first
// barrier.
template <bool kHiLo>
__global__ __launch_bounds__(kStreamThreads, 2) void stream_kernel(const uint8_t *__restrict__ plan,
                                                                   uint32_t *__restrict__ sync) {
  const StreamHeader *h = reinterpret_cast<const StreamHeader *>(plan);
  const StreamPhase *phases = reinterpret_cast<const StreamPhase *>(plan + sizeof(StreamHeader));
  const StreamSeg *segs =
      reinterpret_cast<const StreamSeg *>(plan + sizeof(StreamHeader) +
                                          (size_t)h->nphases * sizeof(StreamPhase));
  const int nphases = h->nphases, b = h->b;
  const int G = (int)gridDim.x;
  const uint32_t epoch = load_device_u32(sync + kSyncEpoch);
  if (load_device_u32(sync + kSyncError) != 0u) return;
  // next task of this workgroup: phase np, task nt (np == nphases: none)
  int np = 0, nt = (int)blockIdx.x;
  auto advance = [&]() {
    while (np < nphases && nt >= phases[np].tasks) {
      ++np;
      nt = (int)blockIdx.x;
    }
  };
  StreamSeg nseg;
  SignRegs nsig;
  auto prefetch = [&]() {
    advance();
    if (np >= nphases) return;
    const StreamPhase ph = phases[np];
    int sg = ph.seg_begin;
    while (sg + 1 < ph.seg_end && nt >= segs[sg].task_end) ++sg;
    nseg = segs[sg];
    const int local = nt - nseg.task_begin;
    stage_signs(nsig, nseg.M, nseg.rows, nseg.wpr, nseg.slab_words, nseg.rt_log2,
                local % nseg.groups, local / nseg.groups, nseg.row_scale, b);
  };
  prefetch();
  for (int p = 0; p < nphases; ++p) {
    while (np == p) {
      const StreamSeg seg = nseg;
      const SignRegs sig = nsig;
      const int task = nt;
      nt += G;
      stream_task<kHiLo>(seg, b, task, sig);
      __syncthreads();  // LDS is reused by the next task
      if (np == p && nt < phases[p].tasks) prefetch();  // another task in this phase
      else break;
    }
    if (p + 1 < nphases) {
      barrier_arrive(sync, epoch + (uint32_t)p + 1u);
      if (np == p) prefetch();  // the next task lies in a later phase
      if (!barrier_wait(sync, epoch + (uint32_t)p + 1u)) return;
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0 && nphases > 1)
    store_device_u32(sync + kSyncEpoch, epoch + (uint32_t)nphases);
}

size_t seg_lds_bytes(const StagePlan &p, int64_t b, int wpr, int *red_off) {
  const int sw = p.slab_words < wpr ? p.slab_words : wpr;
  size_t lds = lds_bytes_for(b, sw);
  *red_off = 0;
  if (p.rt_log2 == 0) {
    const size_t stage = (lds_stage_bytes(b, sw) + 15) & ~(size_t)15;
    if (stage + kRedBytes <= (size_t)kLdsBudget) {
      *red_off = (int)stage;
      lds = stage + kRedBytes;
    }
  }
  return lds;
}

struct PendingSeg {
  int item, kind;
  StagePlan p;
};

// A stage plan for the stream kernel: workgroups of 16 << rt rows, whole
// rows of signs (a wave takes as many groups as it needs, in chunks), the
// columns split only when the staged input would not fit the LDS; with
// `halves`, a first product's columns are split in two partial results.
StagePlan stream_stage_plan(int64_t wpr, int64_t b, int rt, bool halves) {
  int64_t sw = ((kLdsBudget - 17 * kSlot) / b - 16) / kSlot;
  sw -= sw % kGroupWords;
  StagePlan p{rt, 0, 0, kModeFinal};
  const int64_t full = ((wpr + kGroupWords - 1) / kGroupWords) * kGroupWords;
  p.slab_words = (int)(sw < full ? sw : full);
  p.nslabs = (int)((wpr + p.slab_words - 1) / p.slab_words);
  if (p.nslabs > 1) {
    p.mode = kModeLastSlab;
    return p;
  }
  const int64_t groups = full / kGroupWords;
  if (halves && rt == 0 && groups >= 2 && b <= 8) {
    p.slab_words = (int)(((groups + 1) / 2) * kGroupWords);
    p.nslabs = (int)((wpr + p.slab_words - 1) / p.slab_words);
    p.mode = p.nslabs > 1 ? kModePartial : kModeFinal;
  }
  return p;
}

}  // namespace


// The plan of a layer stream.  With plan_out == nullptr only the sizes are
// computed (*plan_need, *ws_need); otherwise the plan is written with
// pointers into the workspace at `ws` (plan_bytes must hold *plan_need).
void stream_plan_impl(const af1_stream_item *items, int count, int64_t b, void *ws,
                      void *plan_out, size_t *plan_need, size_t *ws_need) {
  const int cus = device_cus();
  const int grid = cus < kStreamMaxGrid ? cus : kStreamMaxGrid;  // one workgroup per CU
  std::vector<StagePlan> p1(count), p2(count);
  for (int i = 0; i < count; ++i) {
    const af1_factorized_linear &L = items[i].L;
    p1[i] = stream_stage_plan(L.n / 32, b, 0, false);
    p2[i] = stream_stage_plan(L.r / 32, b, 0, false);
  }
  // layer groups: a new group at a layer that waits, or when the group is full
  std::vector<int> gstart;
  for (int i = 0; i < count; ++i)
    if (i == 0 || items[i].wait != 0 || i - gstart.back() >= kStreamMaxGroupItems)
      gstart.push_back(i);
  gstart.push_back(count);
  const int ngroups = (int)gstart.size() - 1;
  // phases as lists of (item, kind)
  std::vector<std::vector<PendingSeg>> ph;
  auto add_stage = [&](std::vector<PendingSeg> &dst, int g, int kind) {
    for (int i = gstart[g]; i < gstart[g + 1]; ++i)
      dst.push_back(PendingSeg{i, kind, kind == 0 ? p1[i] : p2[i]});
  };
  ph.emplace_back();
  add_stage(ph.back(), 0, 0);
  for (int g = 0; g < ngroups; ++g) {
    ph.emplace_back();
    add_stage(ph.back(), g, 1);
    if (g + 1 < ngroups) {
      if (items[gstart[g + 1]].wait == 0) {
        add_stage(ph.back(), g + 1, 0);
      } else {
        ph.emplace_back();
        add_stage(ph.back(), g + 1, 0);
      }
    }
  }
  // Per phase: more rows per workgroup while the phase has more tasks than
  // workgroups (each task beyond the grid is another round of latency),
  // starting with the segment that has the most tasks; then, while the grid
  // has room, first products split their columns in two (more workgroups
  // share a latency-bound product), the segment with the fewest tasks
  // first.
  auto tasks_of = [&](const PendingSeg &sgm) {
    const af1_factorized_linear &L = items[sgm.item].L;
    const int64_t rows = sgm.kind == 0 ? L.r : L.m;
    const int64_t rw = (int64_t)kTileRows << sgm.p.rt_log2;
    return ((rows + rw - 1) / rw) * sgm.p.nslabs;
  };
  auto wpr_of = [&](const PendingSeg &sgm) {
    const af1_factorized_linear &L = items[sgm.item].L;
    return sgm.kind == 0 ? L.n / 32 : L.r / 32;
  };
  for (auto &phase : ph) {
    auto total = [&]() {
      int64_t t = 0;
      for (const auto &sgm : phase) t += tasks_of(sgm);
      return t;
    };
    for (int guard = 0; guard < 64 && total() > grid; ++guard) {
      int best = -1;
      int64_t best_tasks = 0;
      for (int k = 0; k < (int)phase.size(); ++k) {
        const PendingSeg &sgm = phase[k];
        if (sgm.p.rt_log2 >= 3 || ((int64_t)kTileRows << (sgm.p.rt_log2 + 1)) * b >
                                      (int64_t)kThreads * kMaxOutPerThread)
          continue;
        const int64_t t = tasks_of(sgm);
        if (t > best_tasks) {
          best_tasks = t;
          best = k;
        }
      }
      if (best < 0) break;
      PendingSeg &sgm = phase[best];
      sgm.p = stream_stage_plan(wpr_of(sgm), b, sgm.p.rt_log2 + 1, false);
    }
    for (int guard = 0; guard < 64; ++guard) {
      int best = -1;
      int64_t best_tasks = 0;
      for (int k = 0; k < (int)phase.size(); ++k) {
        const PendingSeg &sgm = phase[k];
        if (sgm.kind != 0 || sgm.p.rt_log2 != 0 || sgm.p.mode != kModeFinal) continue;
        const int64_t t = tasks_of(sgm);
        if (best < 0 || t < best_tasks) {
          best_tasks = t;
          best = k;
        }
      }
      if (best < 0) break;
      PendingSeg trial = phase[best];
      trial.p = stream_stage_plan(wpr_of(trial), b, 0, true);
      if (trial.p.mode != kModePartial || total() - best_tasks + tasks_of(trial) > grid) break;
      phase[best] = trial;
    }
    for (const auto &sgm : phase)
      if (sgm.kind == 0) p1[sgm.item] = sgm.p;
  }
  // the second product's input parts follow the first product's final plan
  int nsegs = 0;
  for (const auto &phase : ph) nsegs += (int)phase.size();
  const int nphases = (int)ph.size();
  const size_t need = stream_plan_size(nphases, nsegs);
  // workspace: header, then per item t (parts x b x r fp32), then per
  // last-slab segment its counters and partial sums
  size_t off = align256(kStreamHeaderBytes);
  std::vector<size_t> t_off(count);
  for (int i = 0; i < count; ++i) {
    const int parts = p1[i].mode == kModePartial ? p1[i].nslabs : 1;
    t_off[i] = off;
    off += align256((size_t)parts * b * items[i].L.r * 4);
  }
  // without an output the segments go to a scratch copy (sizes only)
  std::vector<uint8_t> scratch_plan;
  uint8_t *out = static_cast<uint8_t *>(plan_out);
  if (!out) {
    scratch_plan.resize(need);
    out = scratch_plan.data();
  }
  uint8_t *wsb = static_cast<uint8_t *>(ws);
  StreamHeader *hd = reinterpret_cast<StreamHeader *>(out);
  StreamPhase *phs = reinterpret_cast<StreamPhase *>(out + sizeof(StreamHeader));
  StreamSeg *sg = reinterpret_cast<StreamSeg *>(out + sizeof(StreamHeader) +
                                                (size_t)nphases * sizeof(StreamPhase));
  std::memset(out, 0, need);
  size_t lds_max = 0;
  int max_tasks = 0, si = 0;
  for (int pi = 0; pi < nphases; ++pi) {
    phs[pi].seg_begin = si;
    int task = 0;
    for (const auto &sgm : ph[pi]) {
      const af1_stream_item &it = items[sgm.item];
      const af1_factorized_linear &L = it.L;
      StreamSeg &g = sg[si];
      const bool first = sgm.kind == 0;
      g.kind = sgm.kind;
      g.M = first ? L.Bv : L.Bu;
      g.in = first ? static_cast<const void *>(it.x) : nullptr;  // t set below (base-relative)
      g.s_in = first ? L.s_in : nullptr;
      g.row_scale = first ? L.s_mid : L.s_out;
      g.out = first ? nullptr : static_cast<void *>(it.y);
      g.rows = (int)(first ? L.r : L.m);
      g.wpr = (int)(first ? L.n / 32 : L.r / 32);
      g.slab_words = sgm.p.slab_words;
      g.rt_log2 = sgm.p.rt_log2;
      g.nslabs = sgm.p.nslabs;
      g.mode = sgm.p.mode;
      g.in_parts = first ? 1 : (p1[sgm.item].mode == kModePartial ? p1[sgm.item].nslabs : 1);
      const int64_t rw = (int64_t)kTileRows << g.rt_log2;
      g.groups = (int)((g.rows + rw - 1) / rw);
      g.task_begin = task;
      task += g.groups * g.nslabs;
      g.task_end = task;
      int red_off = 0;
      const size_t lds = seg_lds_bytes(sgm.p, b, g.wpr, &red_off);
      g.red_off = red_off;
      if (lds > lds_max) lds_max = lds;
      // the item's t in the workspace
      if (first)
        g.out = wsb + t_off[sgm.item];
      else
        g.in = wsb + t_off[sgm.item];
      if (g.mode == kModeLastSlab) {
        g.cnt = reinterpret_cast<uint32_t *>(wsb + off);
        off += align256((size_t)g.groups * 4);
        g.part = reinterpret_cast<float *>(wsb + off);
        off += align256((size_t)g.nslabs * b * g.rows * 4);
      }
      ++si;
    }
    phs[pi].seg_end = si;
    phs[pi].tasks = task;
    if (task > max_tasks) max_tasks = task;
  }
  hd->magic = kStreamMagic;
  hd->version = 1;
  hd->nphases = nphases;
  hd->nsegs = nsegs;
  hd->b = (int)b;
  hd->lds_bytes = (int)lds_max;
  hd->max_tasks = max_tasks;
  hd->plan_bytes = need;
  hd->ws_bytes = off;
  hd->ws = ws;
  *plan_need = need;
  *ws_need = off;
}

int stream_plan_check(const void *plan, size_t plan_bytes) {
  const StreamHeader *h = static_cast<const StreamHeader *>(plan);
  if (!h || plan_bytes < sizeof(StreamHeader) || h->magic != kStreamMagic || h->version != 1 ||
      h->nphases < 2 || h->nsegs < 2 || h->b < 1 || h->b > 16 || h->plan_bytes > plan_bytes ||
      stream_plan_size(h->nphases, h->nsegs) != h->plan_bytes || !h->ws)
    return -1;
  return 0;
}

void *stream_plan_workspace(const void *plan) {
  return static_cast<const StreamHeader *>(plan)->ws;
}

hipError_t launch_stream(const void *plan_dev, const void *plan_host, hipStream_t s) {
  const StreamHeader *h = static_cast<const StreamHeader *>(plan_host);
  void *ws = h->ws;
  const int cus = device_cus();
  const size_t lds = (size_t)h->lds_bytes;
  auto go = [&](auto kernel) -> hipError_t {
    if (!launch_fits(reinterpret_cast<const void *>(kernel), lds)) return hipErrorInvalidValue;
    int per_cu = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kStreamThreads,
                                                                lds);
    if (e != hipSuccess) return e;
    if (per_cu < 1) return hipErrorInvalidConfiguration;
    // every workgroup must be resident at once (they wait for each other):
    // one per compute unit (the kernel takes up to 256 registers a lane)
    int grid = cus;
    if (grid > kStreamMaxGrid) grid = kStreamMaxGrid;
    kernel<<<grid, kStreamThreads, lds, s>>>(static_cast<const uint8_t *>(plan_dev),
                                             static_cast<uint32_t *>(ws));
    return hipGetLastError();
  };
  return h->b <= 8 ? go(stream_kernel<true>) : go(stream_kernel<false>);
}

}  // namespace af1
