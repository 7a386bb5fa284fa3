/*
 * liboptimus -- grouped execution of many independent, same-type small
 * operators on one MI355X (gfx950): one kernel launch per operator type
 * instead of one launch per operator instance.
 *
 * The operation is the runtime effect of the horizontal and vertical graph
 * rewrites of "Optimus: A Generic Operator-Level PyTorch Model
 * Transformation Framework" (KDD '26):
 *   - horizontal group fusion (Sec. 3.2, item 1): independent operator
 *     instances, without data dependency between them (Sec. 4.1), executed
 *     in a single launch with their tensor layouts unchanged and their sizes
 *     free to differ;
 *   - vertical split-concat elimination (Sec. 3.2, item 2; appendix Sec. 8.1)
 *     chained with per-piece LayerNorm and activation (Sec. 3.2, chained
 *     example): no split copy and no concat kernel;
 *   - the patterns of Table 1 that these entry points cover: batch_linear /
 *     batch_linear_post_grad (grouped Linear), batch_layernorm (grouped
 *     LayerNorm), batch_relu / sigmoid / tanh and their ATen forms, with
 *     x*sigmoid(x) as the activation product of batch_aten_mul (grouped
 *     pointwise), and split_cat / merge_splits / split_cat_to_slices
 *     (split-op-cat);
 *   - the activation-quantization rewrite (Sec. 5; appendix Sec. 8.2):
 *     saved activations stored as one-byte FP8 codes and restored before
 *     use, grouped over many tensors (fp8 codec below);
 *   - inputs and outputs map one-to-one (Sec. 3.3, item 2): every member
 *     reads its own input tensors and writes its own caller-owned output.
 *
 * Conventions for every entry point
 *   Ownership   The caller owns every tensor (device memory, e.g. from
 *               PyTorch). The library never frees a caller pointer.
 *               Descriptor arrays and the host arrays inside descriptors
 *               (widths, gamma/beta pointer arrays) are read during the call
 *               only and may be freed when it returns.
 *   Layout      2-D row-major tensors with unit inner stride; `ld*` is the
 *               row stride in ELEMENTS (>= the row length). All members of
 *               one call share one dtype (the group key: operator, dtype,
 *               activation); their shapes may differ.
 *   Streams     Work is enqueued on `stream` (a hipStream_t; NULL = the
 *               default stream) and the call returns before it completes.
 *               Device buffers must stay valid until the stream has run it.
 *   Errors      No exception crosses the ABI. On any non-OK status nothing
 *               is launched and optimus_last_error() (thread-local) says why.
 *               G == 0 is a valid no-op (the rewrite's no-op fallback,
 *               Sec. 3.3).
 *               OPTIMUS_ERR_INVALID_ARG  null required pointer, a size < 1,
 *                                        ld < row length, widths not summing
 *                                        to D, G < 0, size above 2^31-1 rows
 *               OPTIMUS_ERR_UNSUPPORTED  unknown dtype or activation
 *               OPTIMUS_ERR_ALIASING     an output overlaps an input or
 *                                        another output (members must be
 *                                        independent, Sec. 4.1); exact
 *                                        in-place (y == x with equal strides)
 *                                        is allowed for LayerNorm, pointwise
 *                                        and split-op-cat (never for the fp8
 *                                        codec)
 *               OPTIMUS_ERR_HIP          a HIP runtime call failed
 *               OPTIMUS_ERR_OOM          device allocation failed
 *   Alignment   Pointers or strides that are not 16-byte aligned, or row
 *               lengths that are not a multiple of 16 bytes, take a
 *               per-element path. This is not an error.
 *   Arithmetic  bf16 members: bf16 storage, fp32 accumulation and
 *               statistics, outputs rounded to nearest-even bf16. fp32
 *               members: fp32 throughout (no reduced-precision products).
 */
#ifndef OPTIMUS_H
#define OPTIMUS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* optimus_stream_t; /* the same type as hipStream_t */

/* The enumerations are int-sized in C; in C++ they take int as their fixed
 * underlying type (the same size), so that any value a caller passes -- an
 * unknown dtype or activation included, which the library rejects -- is a
 * valid value of the type. */
#ifdef __cplusplus
#define OPTIMUS_ENUM(tag) enum tag : int
#else
#define OPTIMUS_ENUM(tag) enum tag
#endif

typedef OPTIMUS_ENUM(optimus_dtype_e) { OPTIMUS_F32 = 0, OPTIMUS_BF16 = 1 } optimus_dtype;

/* Activations of Table 1: relu, sigmoid, tanh, and silu = x * sigmoid(x). */
typedef OPTIMUS_ENUM(optimus_act_e) {
  OPTIMUS_ACT_NONE = 0,
  OPTIMUS_ACT_RELU = 1,
  OPTIMUS_ACT_SIGMOID = 2,
  OPTIMUS_ACT_TANH = 3,
  OPTIMUS_ACT_SILU = 4
} optimus_act;

typedef OPTIMUS_ENUM(optimus_status_e) {
  OPTIMUS_OK = 0,
  OPTIMUS_ERR_INVALID_ARG = -1,
  OPTIMUS_ERR_UNSUPPORTED = -2,
  OPTIMUS_ERR_ALIASING = -3,
  OPTIMUS_ERR_HIP = -4,
  OPTIMUS_ERR_OOM = -5
} optimus_status;

/* One Linear member (torch nn.Linear convention):
 *   y[M][N] = act( x[M][K] . w[N][K]^T + bias[N] )
 * x, w, y: device pointers of the group's dtype; bias may be NULL (no bias). */
typedef struct {
  const void* x;
  int64_t ldx;
  const void* w;
  int64_t ldw;
  const void* bias;
  void* y;
  int64_t ldy;
  int64_t M, N, K;
} optimus_linear_desc;

/* One LayerNorm member over the last dim of x[rows][cols]:
 *   y = act( (x - mean) / sqrt(var + eps) * gamma + beta ),
 * mean and biased variance per row. gamma/beta: device [cols] of the group's
 * dtype, or NULL for 1 / 0. */
typedef struct {
  const void* x;
  int64_t ldx;
  void* y;
  int64_t ldy;
  const void* gamma;
  const void* beta;
  int64_t rows, cols;
  float eps;
} optimus_layernorm_desc;

/* One pointwise member: y[rows][cols] = act(x[rows][cols]). */
typedef struct {
  const void* x;
  int64_t ldx;
  void* y;
  int64_t ldy;
  int64_t rows, cols;
} optimus_pointwise_desc;

/* split along dim 1 of in[rows][D] into n_slices pieces of widths[j]
 * (sum == D, piece j starts at column o_j = sum_{i<j} widths[i]); per piece
 *   out[:, o_j : o_j+w_j] = act( LayerNorm_j(in[:, o_j : o_j+w_j]) )  if apply_layernorm
 *   out[:, o_j : o_j+w_j] = act( in[:, o_j : o_j+w_j] )               otherwise
 * then concat along dim 1 into out[rows][D] -- performed in place in `out`,
 * no split copy and no concat. widths: host array [n_slices]. gamma, beta:
 * host arrays of n_slices device pointers (each [w_j], or NULL entries for
 * 1 / 0), or NULL arrays. LayerNorm off and ACT_NONE is a plain copy.
 * out == in (same ld) is allowed: each row is read whole before it is written. */
typedef struct {
  const void* in;
  int64_t ldin;
  void* out;
  int64_t ldout;
  int64_t rows, D;
  int32_t n_slices;
  const int64_t* widths;
  const void* const* gamma;
  const void* const* beta;
  int32_t apply_layernorm;
  float eps;
  optimus_act act;
} optimus_split_op_cat_desc;

/* One member of the grouped Linear backward (training; the backward graph's
 * grouped Linear, Table 1 batch_linear_post_grad, and the training column of
 * Table 3). Given the forward's X [M][K], W [N][K] and dY = dL/dY [M][N] of
 * the Linear's output (before any activation; apply the activation's
 * backward first):
 *   dX[M][K] = dY . W,   dW[N][K] = dY^T . X,   db[N] = sum over rows of dY
 * Outputs left NULL are not computed; db needs dw (it is summed while the dW
 * launch streams dY). Sums in fp32, outputs rounded to the group's dtype. */
typedef struct {
  const void* x;
  int64_t ldx;
  const void* w;
  int64_t ldw;
  const void* dy;
  int64_t lddy;
  void* dx;
  int64_t lddx;
  void* dw;
  int64_t lddw;
  void* db;
  int64_t M, N, K;
} optimus_linear_grad_desc;

/* One member of the grouped LayerNorm backward: x [rows][cols] is the
 * forward's input (the statistics are recomputed from it), gamma [cols] or
 * NULL (1), dy = dL/dy [rows][cols] of the LayerNorm's output (apply any
 * activation's backward first). Writes dx [rows][cols] and, if not NULL,
 * dgamma and dbeta [cols] (sums over rows). */
typedef struct {
  const void* x;
  int64_t ldx;
  const void* gamma;
  const void* dy;
  int64_t lddy;
  void* dx;
  int64_t lddx;
  void* dgamma;
  void* dbeta;
  int64_t rows, cols;
  float eps;
} optimus_layernorm_grad_desc;

/* One member of the grouped activation backward: dx = dy * act'(x), x the
 * activation's input [rows][cols] (relu passes no gradient at x = 0). */
typedef struct {
  const void* x;
  int64_t ldx;
  const void* dy;
  int64_t lddy;
  void* dx;
  int64_t lddx;
  int64_t rows, cols;
} optimus_act_grad_desc;

/* One member of the fp8 activation codec (paper Sec. 5, peak memory usage
 * reduction; appendix Sec. 8.2, activation quantization: saved activations
 * are stored in FP8 in the forward pass and restored to their own dtype
 * before use in the backward pass, with or without a per-tensor scale).
 * FP8 is OCP E4M3: one byte per value, bias 7, largest finite 448, no
 * infinities, S.1111.111 = NaN. x: values [rows][ldx] of the group's dtype;
 * q: codes [rows][ldq] (uint8); scale: ONE device fp32 value. */
typedef struct {
  const void* x;
  int64_t ldx;
  void* q;
  int64_t ldq;
  float* scale;  /* written by a scaled quantize; unused (may be NULL) unscaled */
  int64_t rows, cols;
} optimus_fp8_quant_desc;

typedef struct {
  const void* q;
  int64_t ldq;
  const float* scale;  /* read; NULL means 1 */
  void* y;
  int64_t ldy;
  int64_t rows, cols;
} optimus_fp8_dequant_desc;

/* ---------------------------------------------------------------- one-shot
 * Validate, build the launch schedule, upload it (stream-ordered) and launch
 * ONE kernel for the whole group on `stream`. */

/* Grouped Linear (Table 1 batch_linear; Sec. 3.2 group fusion): G members
 * d[0..G-1], optional fused epilogue activation. */
optimus_status optimus_grouped_linear(const optimus_linear_desc* d, int32_t G, optimus_dtype dt,
                                      optimus_act epilogue, optimus_stream_t stream);

/* Grouped Linear with the row-wise LayerNorm that consumes each member's
 * output fused into the same launch (Sec. 3.2: vertical optimization of two
 * consecutive operators, applied to a horizontally fused group):
 *   y[M][N] = act( LN_row( x . w^T + bias ) * gamma + beta )
 * mean and biased variance of each output row over its N values, in fp32 on
 * the unrounded accumulator; x . w^T + bias is never written out. gamma,
 * beta: host arrays of G device pointers ([N_g] each, the group's dtype; a
 * NULL entry means 1 / 0), or NULL arrays. One output tile holds whole rows,
 * so N_g <= 256 for bf16 and N_g <= 128 for fp32; a wider member returns
 * OPTIMUS_ERR_UNSUPPORTED (use optimus_grouped_linear then
 * optimus_grouped_layernorm). eps >= 0 and finite, else INVALID_ARG. */
optimus_status optimus_grouped_linear_layernorm(const optimus_linear_desc* d, const void* const* gamma,
                                                const void* const* beta, int32_t G, optimus_dtype dt, float eps,
                                                optimus_act epilogue, optimus_stream_t stream);

/* Grouped row-wise LayerNorm (Table 1 batch_layernorm), optional fused activation. */
optimus_status optimus_grouped_layernorm(const optimus_layernorm_desc* d, int32_t G, optimus_dtype dt,
                                         optimus_act epilogue, optimus_stream_t stream);

/* Grouped pointwise activation (Table 1 batch_tanh / sigmoid / relu, and x*sigmoid(x)). */
optimus_status optimus_grouped_pointwise(const optimus_pointwise_desc* d, int32_t G, optimus_dtype dt,
                                         optimus_act op, optimus_stream_t stream);

/* Fused split -> per-piece LayerNorm/activation -> concat (Sec. 3.2 chained
 * example; split_cat patterns of Table 1), one launch. */
optimus_status optimus_split_op_cat(const optimus_split_op_cat_desc* d, optimus_dtype dt,
                                    optimus_stream_t stream);

/* Grouped fp8 quantize of G activation tensors, one launch (Sec. 3.2 group
 * fusion applied to the activation-quantization rewrite, Sec. 5).
 *   use_scaling = 1: amax = max |x| over the member (NaN values skipped),
 *     scale = amax / 448 and inv = 448 / amax in fp32 (both 1 if amax is 0),
 *     *scale is written, q = E4M3(fp32(x * inv)) with magnitudes saturated
 *     to 448 (no code is NaN unless x holds NaN, or an infinity, which makes
 *     amax infinite, inv 0 and x * inv NaN for the infinities).
 *   use_scaling = 0: q = E4M3(x); magnitudes above 464 (448 plus half a
 *     step; 464 itself rounds to the even 448) and infinities give the NaN
 *     code -- the overflow the paper warns about when scaling is disabled.
 * Rounding is to nearest, ties to even; a NaN value gives S.1111.111 with
 * the sign of x. use_scaling other than 0/1 -> INVALID_ARG; scaled members
 * need a non-NULL scale. Unscaled is one launch; scaled is two for the whole
 * group: an amax pass that writes one partial per tile into plan-owned
 * memory, then the conversion, which reads its member's partials. */
optimus_status optimus_grouped_quantize_fp8(const optimus_fp8_quant_desc* d, int32_t G, optimus_dtype dt,
                                            int32_t use_scaling, optimus_stream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation):
 * optimus_grouped_quantize_fp8 with the group's descriptor table and amax
 * partials placed in a library-owned static device array of
 * OPTIMUS_NOALLOC_SCRATCH_BYTES per GPU (held until the process ends)
 * instead of stream-ordered allocations; the table goes up with one
 * hipMemcpyAsync from host memory. Arguments, results and errors as
 * optimus_grouped_quantize_fp8, bit for bit; a group whose table and
 * partials exceed OPTIMUS_NOALLOC_SCRATCH_BYTES returns
 * OPTIMUS_ERR_UNSUPPORTED with nothing launched. Every call on one GPU uses
 * that GPU's one array: calls on the same stream are ordered, but calls that
 * may overlap on one GPU (other streams, other threads) race and must be
 * ordered by the caller. The array needs no clearing between calls (every
 * amax partial is written before it is read). */
#define OPTIMUS_NOALLOC_SCRATCH_BYTES (4u << 20)
optimus_status optimus_grouped_quantize_fp8_noalloc(const optimus_fp8_quant_desc* d, int32_t G, optimus_dtype dt,
                                                    int32_t use_scaling, optimus_stream_t stream);

/* Grouped fp8 dequantize: y = fp32(value(q) * scale) rounded to the group's
 * dtype (nearest even for bf16); NaN codes give NaN. */
optimus_status optimus_grouped_dequantize_fp8(const optimus_fp8_dequant_desc* d, int32_t G, optimus_dtype dt,
                                              optimus_stream_t stream);

/* Grouped Linear backward: one grouped GEMM launch for every dX, then one
 * for every dW (with db). dX reads W as it lies when every member's widths
 * are multiples of 8 values and its rows 16-byte aligned; otherwise one more
 * launch first transposes W into plan-owned scratch. When the planner splits
 * dW's reduction over the batch, the splits write fp32 partials into
 * plan-owned scratch and one more launch sums them. */
optimus_status optimus_grouped_linear_backward(const optimus_linear_grad_desc* d, int32_t G, optimus_dtype dt,
                                               optimus_stream_t stream);

/* Grouped LayerNorm backward: one launch for dx and per-tile column
 * partials of dgamma / dbeta, one small launch that sums the partials.
 * Exact in-place (dx == dy, equal strides) is allowed. */
optimus_status optimus_grouped_layernorm_backward(const optimus_layernorm_grad_desc* d, int32_t G, optimus_dtype dt,
                                                  optimus_stream_t stream);

/* Grouped Linear backward with the activation backward of the layer below
 * fused into dX: for a member whose input x = act(a) is an activation's
 * output, dX leaves as dL/da = (dY W) * act'(a) instead of dL/dx, which
 * saves the activation backward's pass over dX (Table 1's backward groups,
 * the Linear's and the activation's, in one launch set). act_x: G device
 * pointers to a [M][K] (the member's dtype; entries of members without dx
 * are ignored), ld_act_x: G row strides (>= K). dW and db are those of
 * optimus_grouped_linear_backward. act_x may be the member's dx itself (in
 * place: every value is read before it is written) and must not overlap any
 * other output (OPTIMUS_ERR_ALIASING). Where the input-gradient GEMM cannot read W
 * directly (widths not multiples of 8 values, unaligned rows) the GEMM
 * writes dY W into plan-owned scratch ([M][K] per member) and one grouped
 * activation-backward launch reads it with act_x and writes dx, so the
 * in-place form holds on that path too. act = NONE is
 * optimus_grouped_linear_backward. Errors as there, plus
 * OPTIMUS_ERR_INVALID_ARG for a NULL act_x / ld_act_x or ld_act_x < K and
 * OPTIMUS_ERR_UNSUPPORTED for an unknown activation. */
optimus_status optimus_grouped_linear_act_backward(const optimus_linear_grad_desc* d, const void* const* act_x,
                                                   const int64_t* ld_act_x, int32_t G, optimus_dtype dt,
                                                   optimus_act act, optimus_stream_t stream);

/* Grouped backward of the fused LayerNorm + activation (the forward's
 * optimus_grouped_layernorm with an epilogue activation: out = act(gamma *
 * xhat + beta)), two launches as optimus_grouped_layernorm_backward. Here
 * d[g].dy is dL/d(out), the activation output's gradient; the activation's
 * input gamma * xhat + beta is recomputed from x, so no forward output is
 * read and no intermediate gradient is stored: dx, dgamma and dbeta are the
 * LayerNorm's, of dL/dz = dy * act'(z). The backward graph's activation and
 * LayerNorm groups of Table 1 in one pass. beta: G device pointers ([cols]
 * each, the member's dtype) or NULL (all 0); a NULL entry means 0. act =
 * NONE is optimus_grouped_layernorm_backward. Errors as there, plus
 * OPTIMUS_ERR_UNSUPPORTED for an unknown activation. */
optimus_status optimus_grouped_layernorm_act_backward(const optimus_layernorm_grad_desc* d, const void* const* beta,
                                                      int32_t G, optimus_dtype dt, optimus_act act,
                                                      optimus_stream_t stream);

/* Grouped activation backward, one launch. Exact in-place (dx == dy) is allowed. */
optimus_status optimus_grouped_act_backward(const optimus_act_grad_desc* d, int32_t G, optimus_dtype dt,
                                            optimus_act act, optimus_stream_t stream);

/* ---------------------------------------------------------------- plans
 * A plan validates once and keeps the group's descriptor table and launch
 * schedule resident in device memory (allocated with hipMalloc on the current
 * device at plan time, freed by optimus_plan_destroy), so that executing it is
 * a single kernel launch with no host work: the compile-once / run-many split
 * of the paper's rewrite-then-recompile flow (Sec. 3.2). The device pointers
 * captured in the plan must stay valid while the plan is executed. */
typedef struct optimus_plan_s* optimus_plan;

optimus_status optimus_plan_linear(const optimus_linear_desc* d, int32_t G, optimus_dtype dt,
                                   optimus_act epilogue, optimus_plan* out);
optimus_status optimus_plan_linear_layernorm(const optimus_linear_desc* d, const void* const* gamma,
                                             const void* const* beta, int32_t G, optimus_dtype dt, float eps,
                                             optimus_act epilogue, optimus_plan* out);
optimus_status optimus_plan_layernorm(const optimus_layernorm_desc* d, int32_t G, optimus_dtype dt,
                                      optimus_act epilogue, optimus_plan* out);
optimus_status optimus_plan_pointwise(const optimus_pointwise_desc* d, int32_t G, optimus_dtype dt,
                                      optimus_act op, optimus_plan* out);
/* A split-op-cat plan keeps the pieces' gamma / beta device pointers and
 * reads the values they point to on every execute (an in-place update of
 * gamma / beta between executes is seen by the next one). */
optimus_status optimus_plan_split_op_cat(const optimus_split_op_cat_desc* d, optimus_dtype dt,
                                         optimus_plan* out);
/* A scaled quantize plan also owns the 4-byte amax partials of its members
 * (about 256 per member at most), written by its first launch and read by
 * its second: executions of one scaled plan must not overlap (use one
 * stream, or order them with events); one-shot calls each get their own. */
optimus_status optimus_plan_linear_backward(const optimus_linear_grad_desc* d, int32_t G, optimus_dtype dt,
                                            optimus_plan* out);
optimus_status optimus_plan_layernorm_backward(const optimus_layernorm_grad_desc* d, int32_t G, optimus_dtype dt,
                                               optimus_plan* out);
optimus_status optimus_plan_linear_act_backward(const optimus_linear_grad_desc* d, const void* const* act_x,
                                                const int64_t* ld_act_x, int32_t G, optimus_dtype dt, optimus_act act,
                                                optimus_plan* out);
optimus_status optimus_plan_layernorm_act_backward(const optimus_layernorm_grad_desc* d, const void* const* beta,
                                                   int32_t G, optimus_dtype dt, optimus_act act, optimus_plan* out);
optimus_status optimus_plan_act_backward(const optimus_act_grad_desc* d, int32_t G, optimus_dtype dt, optimus_act act,
                                         optimus_plan* out);
optimus_status optimus_plan_quantize_fp8(const optimus_fp8_quant_desc* d, int32_t G, optimus_dtype dt,
                                         int32_t use_scaling, optimus_plan* out);
optimus_status optimus_plan_dequantize_fp8(const optimus_fp8_dequant_desc* d, int32_t G, optimus_dtype dt,
                                           optimus_plan* out);

/* ---------------------------------------------------------------- plan options
 * Overrides of the planner's own choices, for tests and tuning sweeps. A
 * zeroed struct, or a NULL pointer, leaves every choice to the planner (the
 * plain optimus_plan_* functions). The results do not depend on these
 * choices beyond floating-point summation order.
 *   gemm_tile          OPTIMUS_TILE_AUTO or one tile kernel for every grouped
 *                      GEMM of the plan (a Linear backward: dX and dW). A tile
 *                      that some GEMM of the plan cannot run -- a dtype
 *                      mismatch, the direct-to-LDS tiles on rows that are not
 *                      16-byte aligned or K % 8 != 0, a fused LayerNorm wider
 *                      than the tile, the streaming kernel for K or N > 8 --
 *                      returns OPTIMUS_ERR_UNSUPPORTED.
 *   wgrad_splits       Linear backward: 0 = the planner's split count of dW's
 *                      reduction over the batch, 1..16 = that count
 *                      (OPTIMUS_ERR_UNSUPPORTED if a split would be empty,
 *                      INVALID_ARG outside 0..16).
 *   soc_waves_per_row  split-op-cat: 0 = the planner's choice, 1, 2 or 4
 *                      waves of the fused kernel per row (a row needing more
 *                      waves for its registers takes more; INVALID_ARG for
 *                      other values).
 *   reserved           must be 0 (INVALID_ARG otherwise). */
typedef OPTIMUS_ENUM(optimus_gemm_tile_e) {
  OPTIMUS_TILE_AUTO = 0,
  OPTIMUS_TILE_BF16_128X64 = 1,      /* register-staged, one LDS stage */
  OPTIMUS_TILE_BF16_128X128 = 2,     /* register-staged, two LDS stages */
  OPTIMUS_TILE_BF16_256X256 = 3,     /* register-staged, two LDS stages, 8 waves */
  OPTIMUS_TILE_F32_64X64 = 4,
  OPTIMUS_TILE_BF16_DMA_256X256 = 5, /* direct-to-LDS loads, 8 waves */
  OPTIMUS_TILE_BF16_DMA_128X128 = 6, /* direct-to-LDS loads, 4 waves */
  OPTIMUS_TILE_F32_64X128 = 7,
  OPTIMUS_TILE_SKINNY = 8,           /* every K and N <= 8: streaming, no MFMA */
  OPTIMUS_TILE_F32_32X128 = 9,       /* 4 waves across the 128 columns */
  OPTIMUS_TILE_BF16_STREAM = 10,     /* every K, N <= 64 (multiples of 8, aligned rows): 512-row streams */
  OPTIMUS_TILE_F32_16X128 = 11       /* operands loaded straight into MFMA registers, no LDS staging */
} optimus_gemm_tile;

typedef struct {
  int32_t gemm_tile;
  int32_t wgrad_splits;
  int32_t soc_waves_per_row;
  int32_t reserved;
} optimus_plan_options;

optimus_status optimus_plan_linear_ex(const optimus_linear_desc* d, int32_t G, optimus_dtype dt, optimus_act epilogue,
                                      const optimus_plan_options* opt, optimus_plan* out);
optimus_status optimus_plan_linear_layernorm_ex(const optimus_linear_desc* d, const void* const* gamma,
                                                const void* const* beta, int32_t G, optimus_dtype dt, float eps,
                                                optimus_act epilogue, const optimus_plan_options* opt,
                                                optimus_plan* out);
optimus_status optimus_plan_linear_backward_ex(const optimus_linear_grad_desc* d, int32_t G, optimus_dtype dt,
                                               const optimus_plan_options* opt, optimus_plan* out);
optimus_status optimus_plan_linear_act_backward_ex(const optimus_linear_grad_desc* d, const void* const* act_x,
                                                   const int64_t* ld_act_x, int32_t G, optimus_dtype dt,
                                                   optimus_act act, const optimus_plan_options* opt,
                                                   optimus_plan* out);
optimus_status optimus_plan_split_op_cat_ex(const optimus_split_op_cat_desc* d, optimus_dtype dt,
                                            const optimus_plan_options* opt, optimus_plan* out);

/* Execution modes of a plan.
 *   GROUPED     one launch for the whole group (the optimized program).
 *   CHAIN       the unfused program: one launch per member and per operator
 *               (the "fragmented" execution of Sec. 2.2 / Sec. 5.2), built
 *               from the same kernels run with a group of one. For a
 *               split-op-cat plan: a LayerNorm launch per piece into its own
 *               temporary, an activation launch per piece, and one concat
 *               launch (2 * n_slices + 1 launches).
 *   HORIZONTAL  split-op-cat plans only: horizontal fusion without the
 *               vertical rewrite -- one grouped LayerNorm launch over the
 *               pieces into temporaries, one grouped activation launch, one
 *               concat launch (3 launches).
 * CHAIN and HORIZONTAL on a split-op-cat plan use plan-owned temporaries of
 * rows*D elements, allocated on their first use. */
typedef OPTIMUS_ENUM(optimus_exec_mode_e) {
  OPTIMUS_EXEC_GROUPED = 0,
  OPTIMUS_EXEC_CHAIN = 1,
  OPTIMUS_EXEC_HORIZONTAL = 2
} optimus_exec_mode;

/* An execution only enqueues kernel launches on `stream`: no host
 * synchronization, copies or fills. It can therefore be recorded into a HIP
 * graph and replayed; a CHAIN or HORIZONTAL split-op-cat plan must have run
 * once in that mode before it is recorded (its temporaries are allocated on
 * first use). The plan and every tensor it names must outlive the graph. */
optimus_status optimus_plan_execute(optimus_plan plan, optimus_stream_t stream);
optimus_status optimus_plan_execute_mode(optimus_plan plan, optimus_exec_mode mode, optimus_stream_t stream);
void optimus_plan_destroy(optimus_plan plan);

/* What a plan launches, for measurement. `flops` and `bytes` are the
 * algorithmic work of the group: GEMM flops 2*sum(M*N*K); HBM bytes counted
 * once per tensor element read or written (inputs, weights, bias, gamma/beta,
 * outputs), never padding, re-reads or temporaries. */
typedef struct {
  int32_t kind;            /* 0 linear, 1 layernorm, 2 pointwise, 3 split_op_cat, 4 linear_layernorm,
                              5 quantize_fp8, 6 dequantize_fp8, 7 linear_backward,
                              8 layernorm_backward, 9 act_backward */
  int32_t group_size;      /* G, or n_slices */
  int32_t launches;        /* kernel launches per GROUPED execute (1; 2 for a scaled quantize, a
                              Linear backward with dX and dW, a LayerNorm backward with dgamma/dbeta) */
  int32_t chain_launches;  /* kernel launches per CHAIN execute */
  int64_t work_items;      /* GEMM tiles / row tiles of the grouped launch */
  int32_t grid;            /* workgroups of the grouped launch */
  int32_t block;           /* threads per workgroup */
  double flops;
  double bytes;
  const char* kernel;      /* name of the grouped kernel variant */
} optimus_plan_info;

optimus_status optimus_plan_get_info(optimus_plan plan, optimus_plan_info* out);

/* ---------------------------------------------------------------- host-only
 * Descriptor validation with no device access (no HIP call is made): the
 * same checks the entry points above run before launching. */
optimus_status optimus_validate_linear(const optimus_linear_desc* d, int32_t G, optimus_dtype dt, optimus_act act);
optimus_status optimus_validate_linear_layernorm(const optimus_linear_desc* d, const void* const* gamma,
                                                 const void* const* beta, int32_t G, optimus_dtype dt, float eps,
                                                 optimus_act act);
optimus_status optimus_validate_layernorm(const optimus_layernorm_desc* d, int32_t G, optimus_dtype dt, optimus_act act);
optimus_status optimus_validate_pointwise(const optimus_pointwise_desc* d, int32_t G, optimus_dtype dt, optimus_act act);
optimus_status optimus_validate_split_op_cat(const optimus_split_op_cat_desc* d, optimus_dtype dt);
optimus_status optimus_validate_linear_backward(const optimus_linear_grad_desc* d, int32_t G, optimus_dtype dt);
optimus_status optimus_validate_layernorm_backward(const optimus_layernorm_grad_desc* d, int32_t G, optimus_dtype dt);
optimus_status optimus_validate_act_backward(const optimus_act_grad_desc* d, int32_t G, optimus_dtype dt, optimus_act act);
optimus_status optimus_validate_quantize_fp8(const optimus_fp8_quant_desc* d, int32_t G, optimus_dtype dt,
                                             int32_t use_scaling);
optimus_status optimus_validate_dequantize_fp8(const optimus_fp8_dequant_desc* d, int32_t G, optimus_dtype dt);

/* Message for the last non-OK status returned on this thread ("" if none). */
const char* optimus_last_error(void);

/* Library version string. */
const char* optimus_version(void);

#ifdef __cplusplus
}
#endif

#endif /* OPTIMUS_H */
