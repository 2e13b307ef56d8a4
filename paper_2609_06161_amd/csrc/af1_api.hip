// C ABI of the AF1 factorized binary linear (declared in include/af1.h).
//
// Every entry point validates its arguments on the host before it enqueues
// anything: an argument error returns a status with no launch and no side
// effect.  The launchers in af1_internal.h then only enqueue kernels on the
// caller's stream.
#include <math.h>
#include <stdint.h>

#include <vector>

#include "af1.h"
#include "af1_check.h"
#include "af1_internal.h"

using namespace af1::check;

namespace {

constexpr const char *kVersion = "af1-mi355x 0.4.0 (gfx950)";

}  // namespace

extern "C" {

af1_status af1_pack(const void *src, int32_t src_dtype, int64_t rows, int64_t cols,
                    uint32_t *dst, void *stream) {
  if (!src || !dst) return AF1_ERR_NULL;
  if (src_dtype < AF1_SRC_F32 || src_dtype > AF1_SRC_I8) return AF1_ERR_DTYPE;
  if (rows < 0 || cols < 32 || cols % 32 != 0 || cols > ((int64_t)1 << 40) ||
      (rows > 0 && rows > (((int64_t)1 << 40) / cols)))
    return AF1_ERR_SHAPE;
  if (!aligned16(src) || !aligned16(dst)) return AF1_ERR_ALIGN;
  static const int kElemBytes[] = {4, 2, 2, 1};
  const uint64_t n = (uint64_t)rows * (uint64_t)cols;
  if (overlap(span(src, n * kElemBytes[src_dtype]), span(dst, n / 8))) return AF1_ERR_ALIAS;
  return hip_status(af1::launch_pack(src, src_dtype, rows, cols, dst, as_stream(stream)));
}

af1_status af1_unpack(const uint32_t *words, int64_t rows, int64_t cols, int8_t *dst,
                      void *stream) {
  if (!words || !dst) return AF1_ERR_NULL;
  if (rows < 0 || cols < 32 || cols % 32 != 0 || cols > ((int64_t)1 << 40) ||
      (rows > 0 && rows > (((int64_t)1 << 40) / cols)))
    return AF1_ERR_SHAPE;
  if (!aligned16(words) || !aligned16(dst)) return AF1_ERR_ALIGN;
  const uint64_t n = (uint64_t)rows * (uint64_t)cols;
  if (overlap(span(words, n / 8), span(dst, n))) return AF1_ERR_ALIAS;
  return hip_status(af1::launch_unpack(words, rows, cols, dst, as_stream(stream)));
}

size_t af1_gemv_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t b) {
  if (!dim_ok(m) || !dim_ok(n) || !dim_ok(r) || b < 1 || b > AF1_GEMV_MAX_BATCH) return 0;
  return af1::gemv_workspace_bytes(m, n, r, b);
}

af1_status af1_linear_gemv(const af1_factorized_linear *L, const uint16_t *x, int64_t b,
                           uint16_t *y, void *ws, size_t ws_bytes, void *stream) {
  const size_t need = (L && dim_ok(L->m) && dim_ok(L->n) && dim_ok(L->r) && b >= 1 &&
                       b <= AF1_GEMV_MAX_BATCH)
                          ? af1::gemv_workspace_bytes(L->m, L->n, L->r, b)
                          : 0;
  const af1_status st = check_forward(L, x, b, AF1_GEMV_MAX_BATCH, y, ws, ws_bytes, need);
  if (st != AF1_OK) return st;
  return hip_status(af1::launch_gemv(L->m, L->n, L->r, L->Bu, L->Bv, L->s_out, L->s_mid,
                                     L->s_in, x, b, y, ws, as_stream(stream)));
}

size_t af1_gemv_multi_workspace_bytes(const af1_factorized_linear *Ls, int32_t count,
                                      int64_t b) {
  if (!Ls || count < 1 || count > AF1_GEMV_MULTI_MAX || b < 1 || b > AF1_GEMV_MAX_BATCH) return 0;
  int64_t m[AF1_GEMV_MULTI_MAX], r[AF1_GEMV_MULTI_MAX];
  for (int i = 0; i < count; ++i) {
    if (!dim_ok(Ls[i].m) || !dim_ok(Ls[i].n) || !dim_ok(Ls[i].r) || Ls[i].n != Ls[0].n) return 0;
    m[i] = Ls[i].m;
    r[i] = Ls[i].r;
  }
  return af1::gemv_multi_workspace_bytes(m, r, count, Ls[0].n, b);
}

af1_status af1_linear_gemv_multi(const af1_factorized_linear *Ls, int32_t count,
                                 const uint16_t *x, int64_t b, uint16_t *const *ys, void *ws,
                                 size_t ws_bytes, void *stream) {
  if (!Ls || !ys) return AF1_ERR_NULL;
  if (count < 1 || count > AF1_GEMV_MULTI_MAX) return AF1_ERR_SHAPE;
  for (int i = 0; i < count; ++i)
    if (dim_ok(Ls[i].n) && dim_ok(Ls[0].n) && Ls[i].n != Ls[0].n) return AF1_ERR_SHAPE;
  const size_t need = af1_gemv_multi_workspace_bytes(Ls, count, b);
  for (int i = 0; i < count; ++i) {
    if (!ys[i]) return AF1_ERR_NULL;
    const af1_status st = check_forward(&Ls[i], x, b, AF1_GEMV_MAX_BATCH, ys[i], ws, ws_bytes, need);
    if (st != AF1_OK) return st;
  }
  // outputs against every other layer's arrays and against each other
  for (int i = 0; i < count; ++i) {
    const Span yi = span(ys[i], (uint64_t)b * Ls[i].m * 2);
    for (int j = 0; j < count; ++j) {
      const af1_factorized_linear &Lj = Ls[j];
      const Span arrays[] = {span(Lj.Bu, (uint64_t)Lj.m * Lj.r / 8),
                             span(Lj.Bv, (uint64_t)Lj.r * Lj.n / 8),
                             span(Lj.s_out, (uint64_t)Lj.m * 2), span(Lj.s_mid, (uint64_t)Lj.r * 2),
                             span(Lj.s_in, (uint64_t)Lj.n * 2)};
      for (const Span &a : arrays)
        if (overlap(yi, a)) return AF1_ERR_ALIAS;
      if (j != i && overlap(yi, span(ys[j], (uint64_t)b * Lj.m * 2))) return AF1_ERR_ALIAS;
    }
  }
  int64_t m[AF1_GEMV_MULTI_MAX], r[AF1_GEMV_MULTI_MAX];
  const uint32_t *Bu[AF1_GEMV_MULTI_MAX], *Bv[AF1_GEMV_MULTI_MAX];
  const uint16_t *so[AF1_GEMV_MULTI_MAX], *sm[AF1_GEMV_MULTI_MAX], *si[AF1_GEMV_MULTI_MAX];
  for (int i = 0; i < count; ++i) {
    m[i] = Ls[i].m;
    r[i] = Ls[i].r;
    Bu[i] = Ls[i].Bu;
    Bv[i] = Ls[i].Bv;
    so[i] = Ls[i].s_out;
    sm[i] = Ls[i].s_mid;
    si[i] = Ls[i].s_in;
  }
  return hip_status(af1::launch_gemv_multi(count, m, r, Ls[0].n, Bu, Bv, so, sm, si, x, b, ys, ws,
                                           as_stream(stream)));
}

}  // extern "C"

namespace {

// Arguments of a layer stream, checked before any plan is made.
af1_status check_stream(const af1_stream_item *items, int32_t count, int64_t b) {
  if (!items) return AF1_ERR_NULL;
  if (count < 1 || count > AF1_STREAM_MAX_ITEMS) return AF1_ERR_SHAPE;
  if (b < 1 || b > AF1_GEMV_MAX_BATCH) return AF1_ERR_BATCH;
  for (int i = 0; i < count; ++i) {
    const af1_status st =
        check_forward(&items[i].L, items[i].x, b, AF1_GEMV_MAX_BATCH, items[i].y, nullptr, 0, 0);
    if (st != AF1_OK) return st;
  }
  // outputs against every layer's arrays, each other, and the inputs of
  // items that run before them or in their group
  std::vector<int> group_start(count);
  for (int i = 0; i < count; ++i)
    group_start[i] = (i == 0 || items[i].wait) ? i : group_start[i - 1];
  for (int i = 0; i < count; ++i) {
    const af1_factorized_linear &Li = items[i].L;
    const Span yi = span(items[i].y, (uint64_t)b * Li.m * 2);
    for (int j = 0; j < count; ++j) {
      const af1_factorized_linear &Lj = items[j].L;
      const Span arrays[] = {span(Lj.Bu, (uint64_t)Lj.m * Lj.r / 8),
                             span(Lj.Bv, (uint64_t)Lj.r * Lj.n / 8),
                             span(Lj.s_out, (uint64_t)Lj.m * 2), span(Lj.s_mid, (uint64_t)Lj.r * 2),
                             span(Lj.s_in, (uint64_t)Lj.n * 2)};
      for (const Span &a : arrays)
        if (overlap(yi, a)) return AF1_ERR_ALIAS;
      if (j != i && overlap(yi, span(items[j].y, (uint64_t)b * Lj.m * 2))) return AF1_ERR_ALIAS;
      // item j may read y_i only from a later group that waits (a group
      // that does not wait shares a phase with the group before it)
      const bool ordered = j > i && group_start[j] > i && items[group_start[j]].wait &&
                           group_start[group_start[j]] == group_start[j];
      if (!ordered && overlap(yi, span(items[j].x, (uint64_t)b * Lj.n * 2))) return AF1_ERR_ALIAS;
    }
  }
  return AF1_OK;
}

}  // namespace

extern "C" {

size_t af1_stream_workspace_bytes(const af1_stream_item *items, int32_t count, int64_t b) {
  if (check_stream(items, count, b) != AF1_OK) return 0;
  size_t plan = 0, ws = 0;
  af1::stream_plan_impl(items, count, b, nullptr, nullptr, &plan, &ws);
  return ws;
}

size_t af1_stream_plan_bytes(const af1_stream_item *items, int32_t count, int64_t b) {
  if (check_stream(items, count, b) != AF1_OK) return 0;
  size_t plan = 0, ws = 0;
  af1::stream_plan_impl(items, count, b, nullptr, nullptr, &plan, &ws);
  return plan;
}

af1_status af1_stream_plan(const af1_stream_item *items, int32_t count, int64_t b, void *ws,
                           size_t ws_bytes, void *plan, size_t plan_bytes) {
  const af1_status st = check_stream(items, count, b);
  if (st != AF1_OK) return st;
  if (!ws || !plan) return AF1_ERR_NULL;
  if (!aligned16(ws) || !aligned16(plan)) return AF1_ERR_ALIGN;
  size_t need_plan = 0, need_ws = 0;
  af1::stream_plan_impl(items, count, b, nullptr, nullptr, &need_plan, &need_ws);
  if (ws_bytes < need_ws || plan_bytes < need_plan) return AF1_ERR_WORKSPACE;
  const Span sws = span(ws, need_ws);
  for (int i = 0; i < count; ++i) {
    const af1_factorized_linear &L = items[i].L;
    const Span arrays[] = {span(items[i].x, (uint64_t)b * L.n * 2),
                           span(items[i].y, (uint64_t)b * L.m * 2),
                           span(L.Bu, (uint64_t)L.m * L.r / 8), span(L.Bv, (uint64_t)L.r * L.n / 8),
                           span(L.s_out, (uint64_t)L.m * 2), span(L.s_mid, (uint64_t)L.r * 2),
                           span(L.s_in, (uint64_t)L.n * 2)};
    for (const Span &a : arrays)
      if (overlap(sws, a)) return AF1_ERR_ALIAS;
  }
  af1::stream_plan_impl(items, count, b, ws, plan, &need_plan, &need_ws);
  return AF1_OK;
}

af1_status af1_linear_stream(const void *plan, const void *plan_dev, void *stream) {
  if (!plan || !plan_dev) return AF1_ERR_NULL;
  if (!aligned16(plan_dev)) return AF1_ERR_ALIGN;
  if (af1::stream_plan_check(plan, (size_t)1 << 40) != 0) return AF1_ERR_PLAN;
  return hip_status(af1::launch_stream(plan_dev, plan, as_stream(stream)));
}

}  // extern "C"

extern "C" {

size_t af1_gemm_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t T) {
  if (!dim_ok(m) || !dim_ok(n) || !dim_ok(r) || T < 1 || T > AF1_GEMM_MAX_TOKENS) return 0;
  return af1::gemm_workspace_bytes(m, n, r, T);
}

af1_status af1_linear_gemm(const af1_factorized_linear *L, const uint16_t *x, int64_t T,
                           uint16_t *y, void *ws, size_t ws_bytes, void *stream) {
  // The kernels address each operand with 32-bit byte offsets: a sign
  // matrix must stay below 2 GiB (else a shape error), and so must the
  // [T, n] and [T, r] activations, which bounds T (else a batch error).
  int64_t max_tokens = AF1_GEMM_MAX_TOKENS;
  if (L && dim_ok(L->m) && dim_ok(L->n) && dim_ok(L->r)) {
    if (L->m * (L->r / 32) * 4 > INT32_MAX || L->r * (L->n / 32) * 4 > INT32_MAX)
      return AF1_ERR_SHAPE;
    const int64_t widest = L->n > L->r ? L->n : L->r;
    const int64_t limit = INT32_MAX / (2 * widest);
    if (limit < max_tokens) max_tokens = limit;
  }
  const size_t need = (L && dim_ok(L->m) && dim_ok(L->n) && dim_ok(L->r) && T >= 1 &&
                       T <= max_tokens)
                          ? af1::gemm_workspace_bytes(L->m, L->n, L->r, T)
                          : 0;
  const af1_status st = check_forward(L, x, T, max_tokens, y, ws, ws_bytes, need);
  if (st != AF1_OK) return st;
  return hip_status(af1::launch_gemm(L->m, L->n, L->r, L->Bu, L->Bv, L->s_out, L->s_mid,
                                     L->s_in, x, T, y, ws, as_stream(stream)));
}

af1_status af1_pack_transpose(const uint32_t *src, int64_t rows, int64_t cols, uint32_t *dst,
                              void *stream) {
  if (!src || !dst) return AF1_ERR_NULL;
  if (rows < 0 || cols < 0 || rows % 32 != 0 || cols % 32 != 0 || rows > AF1_TRANSPOSE_MAX_DIM ||
      cols > AF1_TRANSPOSE_MAX_DIM || (rows > 0 && cols > (((int64_t)1 << 40) / rows)))
    return AF1_ERR_SHAPE;
  if (!aligned16(src) || !aligned16(dst)) return AF1_ERR_ALIGN;
  const uint64_t bytes = (uint64_t)rows * (uint64_t)cols / 8;
  if (overlap(span(src, bytes), span(dst, bytes))) return AF1_ERR_ALIAS;
  return hip_status(af1::launch_transpose(src, rows, cols, dst, as_stream(stream)));
}

namespace {

// Token limit of the training entry points: every [T, m], [T, n] and
// [T, r] bf16/fp16 operand is addressed with 32-bit byte offsets.
int64_t train_max_tokens(const af1_factorized_linear *L) {
  int64_t widest = L->m > L->n ? L->m : L->n;
  if (L->r > widest) widest = L->r;
  const int64_t limit = INT32_MAX / (2 * widest);
  return limit < AF1_GEMM_MAX_TOKENS ? limit : AF1_GEMM_MAX_TOKENS;
}

bool dims_ok(const af1_factorized_linear *L) {
  return L && dim_ok(L->m) && dim_ok(L->n) && dim_ok(L->r);
}

// Sign matrices of the layer (forward) or of its transpose (backward) below
// 2 GiB: m*r/8 and r*n/8 bytes either way.
bool signs_fit(const af1_factorized_linear *L) {
  return L->m * (L->r / 32) * 4 <= INT32_MAX && L->r * (L->n / 32) * 4 <= INT32_MAX &&
         L->r * (L->m / 32) * 4 <= INT32_MAX && L->n * (L->r / 32) * 4 <= INT32_MAX;
}

}  // namespace

size_t af1_train_saved_bytes(int64_t m, int64_t n, int64_t r, int64_t T) {
  if (!dim_ok(m) || !dim_ok(n) || !dim_ok(r) || T < 1 || T > AF1_GEMM_MAX_TOKENS) return 0;
  return af1::train_saved_bytes(m, n, r, T);
}

size_t af1_train_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t T) {
  if (!dim_ok(m) || !dim_ok(n) || !dim_ok(r) || T < 1 || T > AF1_GEMM_MAX_TOKENS) return 0;
  return af1::train_workspace_bytes(m, n, r, T);
}

af1_status af1_linear_forward_train(const af1_factorized_linear *L, const uint16_t *x, int64_t T,
                                    uint16_t *y, void *saved, size_t saved_bytes, void *ws,
                                    size_t ws_bytes, void *stream) {
  int64_t max_tokens = AF1_GEMM_MAX_TOKENS;
  if (dims_ok(L)) {
    if (!signs_fit(L)) return AF1_ERR_SHAPE;
    max_tokens = train_max_tokens(L);
  }
  const bool sized = dims_ok(L) && T >= 1 && T <= max_tokens;
  const size_t need = sized ? af1::train_workspace_bytes(L->m, L->n, L->r, T) : 0;
  af1_status st = check_forward(L, x, T, max_tokens, y, ws, ws_bytes, need);
  if (st != AF1_OK) return st;
  if (!saved) return AF1_ERR_NULL;
  if (!aligned16(saved)) return AF1_ERR_ALIGN;
  const size_t saved_need = af1::train_saved_bytes(L->m, L->n, L->r, T);
  if (saved_bytes < saved_need) return AF1_ERR_WORKSPACE;
  const int64_t m = L->m, n = L->n, r = L->r;
  const Span ss = span(saved, saved_need);
  const Span others[] = {span(x, (uint64_t)T * n * 2), span(L->Bu, (uint64_t)m * r / 8),
                         span(L->Bv, (uint64_t)r * n / 8), span(L->s_out, (uint64_t)m * 2),
                         span(L->s_mid, (uint64_t)r * 2), span(L->s_in, (uint64_t)n * 2),
                         span(y, (uint64_t)T * m * 2), span(ws, need)};
  for (const Span &o : others)
    if (overlap(ss, o)) return AF1_ERR_ALIAS;
  return hip_status(af1::launch_forward_train(m, n, r, L->Bu, L->Bv, L->s_out, L->s_mid,
                                              L->s_in, x, T, y, saved, ws, as_stream(stream)));
}

af1_status af1_linear_backward(const af1_factorized_linear *L, const uint32_t *BuT,
                               const uint32_t *BvT, const uint16_t *x, const uint16_t *dy,
                               int64_t T, const void *saved, size_t saved_bytes, uint16_t *dx,
                               float *ds_out, float *ds_mid, float *ds_in, int32_t accumulate,
                               void *ws, size_t ws_bytes, void *stream) {
  if (!L) return AF1_ERR_NULL;
  if (!dims_ok(L) || !signs_fit(L)) return AF1_ERR_SHAPE;
  if (!BuT || !BvT || !L->s_out || !L->s_mid || !L->s_in || !x || !dy || !saved || !ds_out ||
      !ds_mid || !ds_in)
    return AF1_ERR_NULL;
  if (T < 1 || T > train_max_tokens(L)) return AF1_ERR_BATCH;
  if (!aligned16(BuT) || !aligned16(BvT) || !aligned16(L->s_out) || !aligned16(L->s_mid) ||
      !aligned16(L->s_in) || !aligned16(x) || !aligned16(dy) || !aligned16(saved) ||
      (dx && !aligned16(dx)) || !aligned16(ds_out) || !aligned16(ds_mid) || !aligned16(ds_in) ||
      (ws && !aligned16(ws)))
    return AF1_ERR_ALIGN;
  const int64_t m = L->m, n = L->n, r = L->r;
  const size_t saved_need = af1::train_saved_bytes(m, n, r, T);
  const size_t need = af1::train_workspace_bytes(m, n, r, T);
  if (saved_bytes < saved_need || !ws || ws_bytes < need) return AF1_ERR_WORKSPACE;
  const Span outs[] = {span(dx, dx ? (uint64_t)T * n * 2 : 0), span(ds_out, (uint64_t)m * 4),
                       span(ds_mid, (uint64_t)r * 4), span(ds_in, (uint64_t)n * 4),
                       span(ws, need)};
  const Span ins[] = {span(BuT, (uint64_t)r * m / 8), span(BvT, (uint64_t)n * r / 8),
                      span(L->s_out, (uint64_t)m * 2), span(L->s_mid, (uint64_t)r * 2),
                      span(L->s_in, (uint64_t)n * 2), span(x, (uint64_t)T * n * 2),
                      span(dy, (uint64_t)T * m * 2), span(saved, saved_need)};
  for (size_t i = 0; i < sizeof(outs) / sizeof(outs[0]); ++i) {
    for (const Span &in : ins)
      if (overlap(outs[i], in)) return AF1_ERR_ALIAS;
    for (size_t j = i + 1; j < sizeof(outs) / sizeof(outs[0]); ++j)
      if (overlap(outs[i], outs[j])) return AF1_ERR_ALIAS;
  }
  return hip_status(af1::launch_backward(m, n, r, BuT, BvT, L->s_out, L->s_mid, L->s_in, x, dy,
                                         T, saved, dx, ds_out, ds_mid, ds_in, accumulate ? 1 : 0,
                                         ws, as_stream(stream)));
}

int64_t af1_storage_bits(int64_t m, int64_t n, int64_t r) {
  if (m < 0 || n < 0 || r < 0) return -1;
  return r * (m + n) + 16 * (m + n + r);
}

int64_t af1_budget_rank(int64_t m, int64_t n, double bpw, int64_t multiple) {
  // r*(m+n) + 16*(m+n+r) <= B  <=>  r <= (B - 16*(m+n)) / (m+n+16), with the
  // budget B = floor(bpw * m * n) bits
  if (m <= 0 || n <= 0 || multiple <= 0 || !(bpw > 0.0) || m > AF1_MAX_DIM ||
      n > AF1_MAX_DIM || bpw > 64.0)
    return 0;
  const int64_t budget = (int64_t)floor(bpw * (double)m * (double)n);
  const int64_t num = budget - 16 * (m + n);
  if (num <= 0) return 0;
  const int64_t rmax = num / (m + n + 16);
  return rmax - rmax % multiple;
}

int64_t af1_paper_rank(int64_t m, int64_t n, double bpw) {
  if (m <= 0 || n <= 0 || !(bpw > 0.0) || m > AF1_MAX_DIM || n > AF1_MAX_DIM || bpw > 64.0)
    return 0;
  return (int64_t)llround(bpw * (double)m * (double)n / (double)(m + n));
}

const char *af1_status_string(int32_t status) {
  switch (status) {
    case AF1_OK: return "ok";
    case AF1_ERR_NULL: return "a required pointer is NULL";
    case AF1_ERR_SHAPE: return "dimension <= 0, not a multiple of 32, or too large";
    case AF1_ERR_BATCH: return "batch or token count outside the accepted range";
    case AF1_ERR_ALIGN: return "a device pointer is not 16-byte aligned";
    case AF1_ERR_WORKSPACE: return "workspace missing or too small";
    case AF1_ERR_ALIAS: return "an output overlaps an input or the workspace";
    case AF1_ERR_HIP: return "the HIP runtime rejected a launch";
    case AF1_ERR_DTYPE: return "unknown source element type";
    case AF1_ERR_PLAN: return "not a layer-stream plan of this library";
    default: return "unknown status";
  }
}

const char *af1_version(void) { return kVersion; }

}  // extern "C"
