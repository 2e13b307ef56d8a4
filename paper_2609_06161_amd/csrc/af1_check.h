// Host-side argument checks shared by the C entry points (include/af1.h).
// Every entry point validates its arguments with these before it enqueues
// anything, so an argument error returns a status with no side effect.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "af1.h"

namespace af1 {
namespace check {

inline bool dim_ok(int64_t d) { return d >= 32 && d <= AF1_MAX_DIM && d % 32 == 0; }

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Span {
  uintptr_t lo, hi;  // [lo, hi)
};

inline Span span(const void *p, uint64_t bytes) {
  const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
  return Span{lo, lo + (uintptr_t)bytes};
}

inline bool overlap(Span a, Span b) {
  if (a.lo == a.hi || b.lo == b.hi) return false;
  return a.lo < b.hi && b.lo < a.hi;
}

inline hipStream_t as_stream(void *s) { return static_cast<hipStream_t>(s); }

// Checks shared by the forward entry points.  `rows_in` is the batch /
// token count, `ws_need` the workspace the chosen kernels require.
inline af1_status check_forward(const af1_factorized_linear *L, const uint16_t *x,
                                int64_t rows_in, int64_t max_rows, uint16_t *y,
                                const void *ws, size_t ws_bytes, size_t ws_need) {
  if (!L) return AF1_ERR_NULL;
  if (!dim_ok(L->m) || !dim_ok(L->n) || !dim_ok(L->r)) return AF1_ERR_SHAPE;
  if (!L->Bu || !L->Bv || !L->s_out || !L->s_mid || !L->s_in || !x || !y) return AF1_ERR_NULL;
  if (rows_in < 1 || rows_in > max_rows) return AF1_ERR_BATCH;
  if (!aligned16(L->Bu) || !aligned16(L->Bv) || !aligned16(L->s_out) ||
      !aligned16(L->s_mid) || !aligned16(L->s_in) || !aligned16(x) || !aligned16(y) ||
      (ws && !aligned16(ws)))
    return AF1_ERR_ALIGN;
  if (ws_need > 0 && (!ws || ws_bytes < ws_need)) return AF1_ERR_WORKSPACE;

  const int64_t m = L->m, n = L->n, r = L->r;
  const Span sy = span(y, (uint64_t)rows_in * m * 2);
  const Span sws = span(ws, ws ? ws_need : 0);
  const Span inputs[] = {span(x, (uint64_t)rows_in * n * 2), span(L->Bu, (uint64_t)m * r / 8),
                         span(L->Bv, (uint64_t)r * n / 8), span(L->s_out, (uint64_t)m * 2),
                         span(L->s_mid, (uint64_t)r * 2), span(L->s_in, (uint64_t)n * 2)};
  for (const Span &in : inputs)
    if (overlap(sy, in) || overlap(sws, in)) return AF1_ERR_ALIAS;
  if (overlap(sy, sws)) return AF1_ERR_ALIAS;
  return AF1_OK;
}

inline af1_status hip_status(hipError_t e) { return e == hipSuccess ? AF1_OK : AF1_ERR_HIP; }

}  // namespace check
}  // namespace af1
