// af1_linear_gemv_noalloc: the decode forward for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid hipMalloc).  It runs the kernels of
// af1_linear_gemv on a workspace that the library owns: a module-global
// device array, one copy per GPU, held until the process ends.
#include <stdint.h>

#include <mutex>

#include "af1.h"
#include "af1_check.h"
#include "af1_internal.h"

using namespace af1::check;

namespace {

// The workspace.  On the host this name only stands in for the device
// symbol: host code never passes it to a kernel or a copy.  Each device's
// address comes from hipGetSymbolAddress, looked up on the first call on
// that device with the device current.
__device__ __attribute__((aligned(256))) uint8_t scratch[AF1_GEMV_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices];

af1_status scratch_address(void **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return AF1_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return AF1_ERR_HIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return AF1_OK;
}

}  // namespace

extern "C" {

af1_status af1_linear_gemv_noalloc(const af1_factorized_linear *L, const uint16_t *x, int64_t b,
                                   uint16_t *y, void *stream) {
  // validated like af1_linear_gemv with no caller workspace (the scratch
  // cannot overlap a caller buffer); the size check precedes any HIP call
  const af1_status st = check_forward(L, x, b, AF1_GEMV_MAX_BATCH, y, nullptr, 0, 0);
  if (st != AF1_OK) return st;
  if (af1::gemv_workspace_bytes(L->m, L->n, L->r, b) > (size_t)AF1_GEMV_SCRATCH_BYTES)
    return AF1_ERR_WORKSPACE;
  void *ws = nullptr;
  const af1_status sa = scratch_address(&ws);
  if (sa != AF1_OK) return sa;
  const hipStream_t s = as_stream(stream);
  // the arrival counters this call uses start at zero whatever an earlier
  // call left there (a fill kernel, so the call may be graph-captured)
  if (af1::launch_gemv_clear_counters(L->m, L->n, L->r, b, ws, s) != hipSuccess)
    return AF1_ERR_HIP;
  return hip_status(af1::launch_gemv(L->m, L->n, L->r, L->Bu, L->Bv, L->s_out, L->s_mid,
                                     L->s_in, x, b, y, ws, s));
}

}  // extern "C"
