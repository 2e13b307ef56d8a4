/*
 * af1.h -- C ABI of the AF1 binary-factorized linear layer on AMD MI355X
 * (gfx950).
 *
 * The layer (paper "All for 1-Bit", Sec. 4.1, the deployable reconstruction
 * with merged middle scale, label eq:final_reconstruction; App. A.2.1, the
 * equivalent Diag form, label eq:double_factor_equiv) is
 *
 *     W_hat = Diag(s_out) * Bu * Diag(s_mid) * Bv * Diag(s_in)
 *     y     = s_out .* ( Bu * ( s_mid .* ( Bv * ( s_in .* x ) ) ) )
 *
 * with sign factors Bu in {-1,+1}^{m x r} (the paper's A_pm1) and Bv in
 * {-1,+1}^{r x n} (B_pm1), and 16-bit scale vectors s_out (a, length m),
 * s_mid (m = m1 .* m2, length r) and s_in (b, length n).  m is d_out, n is
 * d_in.  Storage per layer is r*(m+n) sign bits plus 16*(m+n+r) scale bits
 * (App. A.3, label eq:app_af1_memory).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Sign storage: a rows x cols sign matrix is rows * (cols/32) uint32 words,
 *   row-major; column j of a row is bit (j mod 32) of word (j div 32); bit 1
 *   encodes -1 and bit 0 encodes +1.  cols must be a multiple of 32 (the
 *   format has no padding bits).
 * Scales: IEEE binary16 bit patterns (uint16_t).
 * Activations and outputs: bfloat16 bit patterns (uint16_t), row-major
 *   [batch, features], token-major, contiguous.
 * Pointers: all array arguments are DEVICE pointers (hipMalloc / torch CUDA
 *   tensors) and must be 16-byte aligned.  The caller owns every buffer; the
 *   library allocates nothing, keeps no pointer after a call returns and
 *   reads the descriptor struct only during the call.
 * Streams: `stream` is a hipStream_t passed as void*; NULL means the null
 *   stream.  Calls only enqueue work and return without synchronising.
 * Errors: argument errors are detected on the host and returned before any
 *   work is enqueued, with no side effect.  AF1_ERR_HIP means a launch was
 *   rejected by the HIP runtime.  No C++ exception crosses this boundary.
 *   Every entry point is reentrant; the library holds no mutable state.
 * Shapes: m, n, r are multiples of 32 in [32, AF1_MAX_DIM].
 */
#ifndef AF1_H
#define AF1_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Only the entry points below are exported from libaf1.so. */
#define AF1_API __attribute__((visibility("default")))

#define AF1_MAX_DIM (1 << 20)   /* largest m, n or r accepted */
#define AF1_GEMV_MAX_BATCH 16   /* decode batch limit of af1_linear_gemv */
#define AF1_GEMM_MAX_TOKENS (1 << 20)

typedef enum af1_status {
    AF1_OK = 0,
    AF1_ERR_NULL = 1,        /* a required pointer is NULL */
    AF1_ERR_SHAPE = 2,       /* dimension <= 0, not a multiple of 32, or too large */
    AF1_ERR_BATCH = 3,       /* batch / token count outside the accepted range */
    AF1_ERR_ALIGN = 4,       /* a device pointer is not 16-byte aligned */
    AF1_ERR_WORKSPACE = 5,   /* workspace missing or smaller than the query returns */
    AF1_ERR_ALIAS = 6,       /* an output buffer overlaps an input or the workspace */
    AF1_ERR_HIP = 7,         /* the HIP runtime rejected a launch */
    AF1_ERR_DTYPE = 8,       /* unknown source element type */
    AF1_ERR_PLAN = 9         /* a stream plan that this library did not build */
} af1_status;

/* Element type of the dense matrix handed to af1_pack. */
typedef enum af1_src_dtype {
    AF1_SRC_F32 = 0,   /* IEEE binary32 */
    AF1_SRC_BF16 = 1,  /* bfloat16 patterns */
    AF1_SRC_F16 = 2,   /* IEEE binary16 patterns */
    AF1_SRC_I8 = 3     /* int8 */
} af1_src_dtype;

/*
 * One factorized linear layer (Sec. 4.1 / App. A.2.1; storage of App. A.3).
 *   Bu    : m x r signs,  m * (r/32) words   (paper: A_pm1)
 *   Bv    : r x n signs,  r * (n/32) words   (paper: B_pm1)
 *   s_out : m binary16   (paper: a)
 *   s_mid : r binary16   (paper: m = m1 .* m2, merged after optimisation)
 *   s_in  : n binary16   (paper: b)
 */
typedef struct af1_factorized_linear {
    int64_t m;
    int64_t n;
    int64_t r;
    const uint32_t *Bu;
    const uint32_t *Bv;
    const uint16_t *s_out;
    const uint16_t *s_mid;
    const uint16_t *s_in;
} af1_factorized_linear;

/*
 * af1_pack -- sign -> bit packing of a dense rows x cols matrix (the binary
 * factors of App. A.3 are stored one bit per sign).
 *   src      : device, rows*cols elements of `src_dtype`, row-major.
 *   dst      : device, rows*(cols/32) uint32 words (written).
 * The bit of an element is its IEEE sign bit for the floating types (so +0
 * packs as +1, -0 as -1, NaN by its sign bit) and (v < 0) for int8.  The
 * result is bit-exact and deterministic.  rows may be 0 (nothing enqueued);
 * cols must be a positive multiple of 32; rows*cols < 2^40.
 */
AF1_API af1_status af1_pack(const void *src, int32_t src_dtype, int64_t rows,
                    int64_t cols, uint32_t *dst, void *stream);

/*
 * af1_unpack -- inverse of af1_pack into dense int8 +-1 (a debugging and
 * testing aid, not part of the forward path).
 *   words : device, rows*(cols/32) uint32;  dst : device, rows*cols int8.
 */
AF1_API af1_status af1_unpack(const uint32_t *words, int64_t rows, int64_t cols,
                      int8_t *dst, void *stream);

/*
 * af1_linear_gemv -- decode-regime forward of one factorized layer
 * (App. A.2.1, Diag form, evaluated right to left).
 *   x  : device, [b, n] bfloat16.       y : device, [b, m] bfloat16 (written).
 *   b  : 1 .. AF1_GEMV_MAX_BATCH.
 *   ws : device workspace of at least af1_gemv_workspace_bytes(m, n, r, b)
 *        bytes.  Its first 512 KiB are a header of arrival counters at
 *        fixed offsets; the header must be zero-filled before the
 *        workspace's first use, and every call that
 *        completes leaves the counters at zero again, so one workspace
 *        serves any sequence of calls, of any shapes, on one stream.  Calls
 *        that may overlap in time need distinct workspaces.  Recovery: a
 *        call that did not run to completion (a launch error reported by
 *        a later call, a killed stream) may leave counters non-zero, after
 *        which results are wrong; zero-fill the header again before reusing
 *        such a workspace.
 * Arithmetic: s_in .* x in fp32 (exact), both sign products accumulated in
 * fp32, the rank-r intermediate kept in fp32, scales applied in fp32, y
 * rounded to bfloat16 (round to nearest even).  y must not overlap x, the
 * layer's arrays or ws.
 */
AF1_API size_t af1_gemv_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t b);
AF1_API af1_status af1_linear_gemv(const af1_factorized_linear *L, const uint16_t *x,
                           int64_t b, uint16_t *y, void *ws, size_t ws_bytes,
                           void *stream);
/*
 * af1_linear_gemv_noalloc -- af1_linear_gemv for callers that cannot
 * allocate device memory or hand over a workspace: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * kernels, arithmetic and results as af1_linear_gemv (bit for bit); the
 * workspace is a library-owned device array of AF1_GEMV_SCRATCH_BYTES bytes
 * that each GPU the library runs on holds from load until the process
 * ends.  The call allocates nothing and calls no allocating routine.
 *   x, b, y : as af1_linear_gemv (the caller still owns x and y).
 * Errors: as af1_linear_gemv; AF1_ERR_WORKSPACE when the shape and batch
 * need more than AF1_GEMV_SCRATCH_BYTES (af1_gemv_workspace_bytes tells);
 * AF1_ERR_HIP when the device array's address cannot be obtained.
 * Concurrency: every call on one GPU uses that GPU's one array, so calls
 * that overlap in time on one GPU (other streams, other threads) race and
 * give wrong results; serialise them.  The array keeps the last call's
 * contents; each call first clears the arrival counters it uses (with a
 * kernel, no memset), so a previous call cannot corrupt it.
 */
#define AF1_GEMV_SCRATCH_BYTES (4 << 20)
AF1_API af1_status af1_linear_gemv_noalloc(const af1_factorized_linear *L, const uint16_t *x,
                                           int64_t b, uint16_t *y, void *stream);


/*
 * af1_linear_gemv_multi -- decode forward of several layers that read the
 * same input x (all with the same n): the q, k and v projections of an
 * attention block, or the gate and up projections of an MLP.  Each output
 * is what af1_linear_gemv computes for its layer (same arithmetic; the
 * grouping of an output's partial sums may differ).  All layers run in two
 * launches when no layer needs a last-slab reduction at this batch (every
 * configuration up to b = 8 at n, r <= 4096 does); otherwise the layers
 * run one after the other on the same workspace.  A decode step at batch 1
 * is bound by launch and memory latency, so fewer launches are the gain.
 *   Ls    : host array of count layers, 1 <= count <= AF1_GEMV_MULTI_MAX.
 *   x     : device, [b, n] bfloat16.
 *   ys    : host array of count device pointers; ys[i] is [b, Ls[i].m]
 *           bfloat16 (written).
 *   ws    : device workspace of at least
 *           af1_gemv_multi_workspace_bytes(Ls, count, b) bytes, header
 *           zero-filled before first use as for af1_linear_gemv.
 * Errors: as af1_linear_gemv for every layer; AF1_ERR_NULL for a NULL Ls,
 * ys or ys[i]; AF1_ERR_SHAPE for a count outside 1..AF1_GEMV_MULTI_MAX or
 * layers whose n differ; AF1_ERR_ALIAS when an output overlaps another
 * output, x, any layer's arrays or ws.
 */
#define AF1_GEMV_MULTI_MAX 4
AF1_API size_t af1_gemv_multi_workspace_bytes(const af1_factorized_linear *Ls, int32_t count,
                                              int64_t b);
AF1_API af1_status af1_linear_gemv_multi(const af1_factorized_linear *Ls, int32_t count,
                                         const uint16_t *x, int64_t b, uint16_t *const *ys,
                                         void *ws, size_t ws_bytes, void *stream);

/*
 * Layer stream -- the decode forward of a sequence of factorized layers in
 * one persistent launch (the decode setting of Sec. 5.4: batch 1, one
 * decoder step through every linear of the model; heterogeneous ranks as in
 * App. A.3, label eq:app_af1_bpw).  Each item computes what
 * af1_linear_gemv computes for its layer (same arithmetic); items run in
 * order, and an item with `wait` set starts only after every earlier item
 * of the call has written its output, so it may read those outputs (x of a
 * later item may be y of an earlier one).  Items without `wait` may run
 * concurrently with the item group before them: q, k and v, or gate and
 * up, are one group.  The launch replaces a kernel boundary per product by
 * a grid-wide barrier between phases.
 *
 * Use: af1_stream_workspace_bytes for the workspace size (zero-fill it
 * before its first use, like the GEMV workspace: it holds arrival words
 * and counters that every completed call leaves consistent);
 * af1_stream_plan_bytes and af1_stream_plan to build the plan on the host,
 * bound to the items' buffers and to that workspace; copy the plan's bytes
 * to device memory; then af1_linear_stream once per decode step.  Rebuild
 * the plan when any buffer changes.
 *
 * af1_stream_item fields:
 *   L    : the layer (device arrays as for af1_linear_gemv).
 *   x    : device, [b, L.n] bfloat16.       y : device, [b, L.m] bfloat16.
 *   wait : non-zero to start after all earlier items have finished.
 *
 * af1_stream_plan errors: AF1_ERR_NULL (items, plan, ws or an item's
 * pointer), AF1_ERR_SHAPE (count outside 1..AF1_STREAM_MAX_ITEMS or a bad
 * layer), AF1_ERR_BATCH (b outside 1..AF1_GEMV_MAX_BATCH), AF1_ERR_ALIGN,
 * AF1_ERR_WORKSPACE (ws or plan too small), AF1_ERR_ALIAS (an output
 * overlaps any layer's arrays, another output, the workspace, or the input
 * of an item that does not wait for it).
 * af1_linear_stream: `plan` is the host plan, `plan_dev` a device copy of
 * its bytes (16-byte aligned).  AF1_ERR_PLAN when the host plan is not a
 * plan of this library, AF1_ERR_HIP when the launch fails or the device
 * cannot hold every workgroup at once.  If a barrier ever timed out (a
 * workgroup that never arrived; only a device fault causes it) the kernel
 * ends early and leaves word 1 of the workspace non-zero; outputs are then
 * invalid and the workspace header must be zero-filled again.  Calls on
 * one workspace must not overlap in time.
 */
#define AF1_STREAM_MAX_ITEMS 4096
typedef struct af1_stream_item {
    af1_factorized_linear L;
    const uint16_t *x;
    uint16_t *y;
    int32_t wait;
    int32_t reserved;   /* set to 0 */
} af1_stream_item;

AF1_API size_t af1_stream_workspace_bytes(const af1_stream_item *items, int32_t count, int64_t b);
AF1_API size_t af1_stream_plan_bytes(const af1_stream_item *items, int32_t count, int64_t b);
AF1_API af1_status af1_stream_plan(const af1_stream_item *items, int32_t count, int64_t b,
                                   void *ws, size_t ws_bytes, void *plan, size_t plan_bytes);
AF1_API af1_status af1_linear_stream(const void *plan, const void *plan_dev, void *stream);

/*
 * af1_linear_gemm -- prefill-regime forward for T tokens on the matrix cores.
 *   x  : device, [T, n] bfloat16.       y : device, [T, m] bfloat16 (written).
 *   T  : 1 .. AF1_GEMM_MAX_TOKENS, and T * max(n, r) * 2 < 2^31 (the
 *        kernels address operands with 32-bit byte offsets); otherwise
 *        AF1_ERR_BATCH.  A sign matrix of 2 GiB or more is AF1_ERR_SHAPE.
 *   ws : device workspace of at least af1_gemm_workspace_bytes(m, n, r, T)
 *        bytes; holds the fp16 operand s_in .* x, the [T, r] intermediate,
 *        a per-token record and the intermediate's per-tile row sums, and,
 *        for token counts whose tile grid would leave compute units idle,
 *        the fp32 partial sums of a contraction split along K (added in a
 *        fixed order, so results repeat bit for bit).  The size depends on
 *        the current device's compute-unit count.
 * Arithmetic: both products run on fp16 MFMA with fp32 accumulation and
 * exact products; each scale vector is applied outside them.  The sign
 * operand holds, per sign, zero (+1) or a single fp16 exponent bit (-1),
 * the activation operand the matching power of two, and the signed sum is
 * formed in fp32 as R - 2 acc with R the token's row sum of the operand,
 * so each product equals the sum of the fp16 operand times exact +-1 signs
 * up to fp32 rounding.  s_in .* x is rounded once to fp16 (the bf16 x fp16
 * product is exact in fp32), the intermediate s_mid .* (Bv (s_in .* x)) is
 * rounded once to fp16 before the second product, s_out is applied in fp32
 * and y is rounded to bfloat16.  Range: each token's two fp16 operands
 * carry a power of two chosen from that token alone (its largest
 * |s_in .* x| for the first, the bound sum_j |s_in_j x_j| * max|s_mid| on
 * the intermediate for the second), undone in fp32 before s_out, so no
 * fp16 operand overflows for any finite bf16 x: the GEMM is defined on the
 * same inputs as the GEMV.  Entries below about 2^-20 of their token's
 * largest one keep fewer digits, as in any fp16 rounding.
 * Defining passage: App. A.2.1 (Diag form, label eq:double_factor_equiv)
 * and Sec. 4.1 (label eq:final_reconstruction), as for af1_linear_gemv.
 */
AF1_API size_t af1_gemm_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t T);
AF1_API af1_status af1_linear_gemm(const af1_factorized_linear *L, const uint16_t *x,
                           int64_t T, uint16_t *y, void *ws, size_t ws_bytes,
                           void *stream);

/*
 * af1_pack_transpose -- the packed storage of the transpose of a packed sign
 * matrix: dst (cols x rows signs, cols * (rows/32) words) gets at row j,
 * column i the sign of src row i, column j.  The scale-only reconstruction
 * (Sec. 4.1) freezes the sign matrices, so the products with Bu^T and Bv^T
 * that its gradients need read factors transposed once with this call.
 *   src  : device, rows * (cols/32) uint32 words.
 *   dst  : device, cols * (rows/32) uint32 words (written).
 * rows and cols are multiples of 32 in [0, AF1_TRANSPOSE_MAX_DIM] with
 * rows * cols < 2^40 (AF1_ERR_SHAPE otherwise); a zero dimension enqueues
 * nothing.  Bit-exact.  dst must not overlap src (AF1_ERR_ALIAS).
 */
#define AF1_TRANSPOSE_MAX_DIM ((int64_t)1 << 24)
AF1_API af1_status af1_pack_transpose(const uint32_t *src, int64_t rows, int64_t cols,
                                      uint32_t *dst, void *stream);

/*
 * Scale-only reconstruction (Sec. 4.1, paragraph on scale-only global
 * reconstruction, labels eq:final_reconstruction and eq:scale_only_kl):
 * after factorisation the paper freezes Bu and Bv and trains only s_out,
 * s_mid and s_in through the unchanged factorised graph.  These two calls
 * are that graph's forward and backward for T tokens of one layer; the
 * loss (a KL divergence to a full-precision teacher in the paper) and the
 * optimiser stay with the caller.
 *
 * af1_linear_forward_train -- y as af1_linear_gemm computes it (same
 * kernels and rounding, bit-identical y), and in `saved` the two pre-scale
 * intermediates the gradients need: v = Bv (s_in .* x) ([T, r], rounded to
 * fp16 at a per-token power-of-two scale, in a layout private to the
 * library), z = Bu (s_mid .* v) ([T, m], fp32, the second product's
 * accumulator, unscaled) and the per-token scale record.
 *   saved : device, at least af1_train_saved_bytes(m, n, r, T) bytes,
 *           written; hand it unchanged to af1_linear_backward with the same
 *           layer, x and T.
 *   ws    : device, at least af1_train_workspace_bytes(m, n, r, T) bytes
 *           (scratch; one buffer serves both calls).
 *   T     : 1 .. AF1_GEMM_MAX_TOKENS and T * max(m, n, r) * 2 < 2^31, else
 *           AF1_ERR_BATCH.
 * Errors: as af1_linear_gemm; AF1_ERR_NULL / AF1_ERR_ALIGN for saved;
 * AF1_ERR_WORKSPACE when saved_bytes or ws_bytes is too small;
 * AF1_ERR_ALIAS when saved overlaps x, y, ws or the layer's arrays.
 *
 * af1_linear_backward -- for the upstream gradient dy of y:
 *     dz = s_out .* dy,   dt = Bu^T dz,   du = Bv^T (s_mid .* dt)
 *     dx = s_in .* du                                 ([T, n] bfloat16)
 *     ds_out = sum_t dy .* z,  ds_mid = sum_t dt .* v,  ds_in = sum_t du .* x
 * (sums over the T tokens, fp32).
 *   L     : the layer (dims and scales; L->Bu and L->Bv are not read and
 *           may be NULL).
 *   BuT   : device, Bu^T (r x m signs, r * (m/32) words), from
 *           af1_pack_transpose(L->Bu, m, r, BuT).
 *   BvT   : device, Bv^T (n x r signs, n * (r/32) words), from
 *           af1_pack_transpose(L->Bv, r, n, BvT).
 *   x     : device, [T, n] bfloat16, the forward input.
 *   dy    : device, [T, m] bfloat16.
 *   saved : what af1_linear_forward_train wrote for this layer, x and T.
 *   dx    : device, [T, n] bfloat16 (written), or NULL to skip it.
 *   ds_out, ds_mid, ds_in : device fp32 arrays of m, r and n entries.
 *           accumulate = 0 overwrites them; accumulate != 0 adds this
 *           call's sums to their contents (gradient accumulation over
 *           micro-batches).
 *   ws    : device, at least af1_train_workspace_bytes(m, n, r, T) bytes.
 * Arithmetic: both products run on fp16 MFMA with fp32 accumulation against
 * exact +-1 operands.  Their A operands, s_out .* dy and s_mid .* dt, carry
 * a power-of-two scale per group of 64 tokens, chosen from the group's
 * largest entry and a bound on the first product's outputs.  So each
 * operand is rounded once to fp16 (2^-12 relative) with no overflow, and
 * the fp16 range limits nothing: gradients far below 2^-24 keep their
 * digits.  The scales are exact powers of two and are undone in fp32.  dx
 * is rounded to bfloat16.  The token sums are taken in fp32 from the
 * accumulators, per tile and then over tiles in a fixed order, so results
 * are bit-identical from run to run.
 * Errors: AF1_ERR_NULL for a NULL L, BuT, BvT, scale, x, dy, saved or ds_*;
 * AF1_ERR_SHAPE / AF1_ERR_BATCH / AF1_ERR_ALIGN as for the forward;
 * AF1_ERR_WORKSPACE for a short saved or ws; AF1_ERR_ALIAS when an output
 * (dx, ds_*, ws) overlaps another output or any input.
 */
AF1_API size_t af1_train_saved_bytes(int64_t m, int64_t n, int64_t r, int64_t T);
AF1_API size_t af1_train_workspace_bytes(int64_t m, int64_t n, int64_t r, int64_t T);
AF1_API af1_status af1_linear_forward_train(const af1_factorized_linear *L, const uint16_t *x,
                                            int64_t T, uint16_t *y, void *saved,
                                            size_t saved_bytes, void *ws, size_t ws_bytes,
                                            void *stream);
AF1_API af1_status af1_linear_backward(const af1_factorized_linear *L, const uint32_t *BuT,
                                       const uint32_t *BvT, const uint16_t *x,
                                       const uint16_t *dy, int64_t T, const void *saved,
                                       size_t saved_bytes, uint16_t *dx, float *ds_out,
                                       float *ds_mid, float *ds_in, int32_t accumulate,
                                       void *ws, size_t ws_bytes, void *stream);

/* Deployable storage bits of one layer: r*(m+n) + 16*(m+n+r) (App. A.3,
 * label eq:app_af1_memory).  Returns -1 for negative arguments. */
AF1_API int64_t af1_storage_bits(int64_t m, int64_t n, int64_t r);

/* Largest rank r, a multiple of `multiple`, whose storage bits
 * r*(m+n) + 16*(m+n+r) do not exceed floor(bpw * m * n): the layer at an
 * effective budget of bpw bits per weight with its scales counted (App. A.3,
 * labels eq:app_af1_memory and eq:app_af1_bpw); bpw = 1, multiple = 32 is
 * the strict 1.0-BPW rank.  Returns 0 when no positive rank fits or an
 * argument is out of range (m, n in 1..AF1_MAX_DIM, 0 < bpw <= 64,
 * multiple >= 1). */
AF1_API int64_t af1_budget_rank(int64_t m, int64_t n, double bpw, int64_t multiple);

/* The paper's own budget-to-rank rule (App. A.1.3): round(bpw * m * n /
 * (m + n)), counting the sign bits only (so a layer at this rank exceeds
 * bpw once its scales are counted); 2.5 BPW at 4096 x 4096 gives 5120.
 * Rounding half away from zero; 0 for arguments out of the range above. */
AF1_API int64_t af1_paper_rank(int64_t m, int64_t n, double bpw);

/* Static, NUL-terminated description of a status code. */
AF1_API const char *af1_status_string(int32_t status);

/* Library version string. */
AF1_API const char *af1_version(void);

#ifdef __cplusplus
}
#endif

#endif /* AF1_H */
