// Host-side launchers behind the C ABI.  Arguments are already validated by
// af1_api.cpp; each launcher only enqueues kernels and reports whether the
// HIP runtime accepted them.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "af1.h"

namespace af1 {

// Compute units of the current device (queried once per device; 256 if the
// query fails).
int device_cus();

hipError_t launch_pack(const void *src, int dtype, int64_t rows, int64_t cols,
                       uint32_t *dst, hipStream_t s);
hipError_t launch_unpack(const uint32_t *words, int64_t rows, int64_t cols,
                         int8_t *dst, hipStream_t s);

// dst (cols x rows signs) = transpose of src (rows x cols signs); rows and
// cols are multiples of 32.
hipError_t launch_transpose(const uint32_t *src, int64_t rows, int64_t cols, uint32_t *dst,
                            hipStream_t s);

size_t gemv_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t b);
hipError_t launch_gemv(int64_t m, int64_t n, int64_t r, const uint32_t *Bu,
                       const uint32_t *Bv, const uint16_t *s_out,
                       const uint16_t *s_mid, const uint16_t *s_in,
                       const uint16_t *x, int64_t b, uint16_t *y, void *ws,
                       hipStream_t s);

// Zero the arrival counters that launch_gemv uses for this shape and batch
// (none when no stage splits its columns); a fill kernel, no memset node.
hipError_t launch_gemv_clear_counters(int64_t m, int64_t n, int64_t r, int64_t b, void *ws,
                                      hipStream_t s);

// Layer stream (one persistent launch for a sequence of layers).  The plan
// is built on the host (sizes only when plan_out is null) with pointers into
// the workspace `ws`; stream_plan_check validates a plan's header;
// launch_stream runs the plan's device copy.
void stream_plan_impl(const af1_stream_item *items, int count, int64_t b, void *ws,
                      void *plan_out, size_t *plan_need, size_t *ws_need);
int stream_plan_check(const void *plan, size_t plan_bytes);
void *stream_plan_workspace(const void *plan);
hipError_t launch_stream(const void *plan_dev, const void *plan_host, hipStream_t s);

// Several layers that share n (count <= 4): two launches for all of them
// when the plan allows, else one call per layer on the same workspace.
size_t gemv_multi_workspace_bytes(const int64_t *m, const int64_t *r, int count, int64_t n,
                                  int64_t b);
hipError_t launch_gemv_multi(int count, const int64_t *m, const int64_t *r, int64_t n,
                             const uint32_t *const *Bu, const uint32_t *const *Bv,
                             const uint16_t *const *s_out, const uint16_t *const *s_mid,
                             const uint16_t *const *s_in, const uint16_t *x, int64_t b,
                             uint16_t *const *y, void *ws, hipStream_t s);

size_t gemm_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t T);
hipError_t launch_gemm(int64_t m, int64_t n, int64_t r, const uint32_t *Bu,
                       const uint32_t *Bv, const uint16_t *s_out,
                       const uint16_t *s_mid, const uint16_t *s_in,
                       const uint16_t *x, int64_t T, uint16_t *y, void *ws,
                       hipStream_t s);

// Scale-only reconstruction (sign matrices frozen): a forward that keeps
// the two pre-scale intermediates, and the gradients with respect to the
// scales and x from the transposed factors.
size_t train_saved_bytes(int64_t m, int64_t n, int64_t r, int64_t T);
size_t train_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t T);
hipError_t launch_forward_train(int64_t m, int64_t n, int64_t r, const uint32_t *Bu,
                                const uint32_t *Bv, const uint16_t *s_out,
                                const uint16_t *s_mid, const uint16_t *s_in,
                                const uint16_t *x, int64_t T, uint16_t *y, void *saved,
                                void *ws, hipStream_t s);
hipError_t launch_backward(int64_t m, int64_t n, int64_t r, const uint32_t *BuT,
                           const uint32_t *BvT, const uint16_t *s_out, const uint16_t *s_mid,
                           const uint16_t *s_in, const uint16_t *x, const uint16_t *dy,
                           int64_t T, const void *saved, uint16_t *dx, float *ds_out,
                           float *ds_mid, float *ds_in, int accumulate, void *ws,
                           hipStream_t s);

}  // namespace af1
