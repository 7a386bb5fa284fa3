/*
 * Optimus grouped-operator ORACLE -- test infrastructure only.
 *
 * This file is the plain, slow, obviously-correct CPU reference that the GPU
 * library is checked against. Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load it; the product path never does.
 * It shares no code, header, table or helper with the HIP library.
 *
 * Everything is fp64 and written one member (one operator instance) at a
 * time, exactly as the unfused program would compute it:
 *
 *  - Horizontal optimization, group fusion (paper Sec. 3.2, item 1): a group
 *    of independent operators run in one launch must give the same outputs as
 *    running each operator on its own (the rewrite is semantics-preserving,
 *    Sec. 2.2; inputs and outputs map one-to-one, Sec. 3.3 item 2). So the
 *    oracle of a group is a loop over members calling the single-operator
 *    definition below.
 *  - Vertical optimization, split-concat elimination (Sec. 3.2, item 2;
 *    appendix Sec. 8.1 listings): the oracle materialises every split piece
 *    in its own array, applies the per-piece operator, then concatenates
 *    along dim 1 into a fresh output -- the unoptimised program, step by step.
 *  - The chained example of Sec. 3.2 (LayerNorm per split piece, then an
 *    activation per piece, then the concat) is split_op_cat() below.
 *
 * The paper names the operators (Table 1: batch_linear, batch_layernorm,
 * batch_tanh / sigmoid / relu, batch_aten_mul) but not their formulas; the
 * formulas here are the standard definitions of those PyTorch operators:
 *   Linear      y[m][n] = sum_k x[m][k] * w[n][k] + b[n]   (w is [N, K])
 *   LayerNorm   over the last dim, biased variance, eps inside the sqrt
 *   relu / sigmoid / tanh / silu(x) = x * sigmoid(x)
 *
 * Parity pins for every function are in the CPU test suite (library
 * routines, closed forms, invariants, brute force, the appendix example).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_ACT_NONE = 0, ORC_ACT_RELU = 1, ORC_ACT_SIGMOID = 2, ORC_ACT_TANH = 3, ORC_ACT_SILU = 4 };

/* ---------------------------------------------------------------- scalars */

/* Logistic function 1 / (1 + e^-x), evaluated on the side where the
 * exponential cannot overflow: for x < 0 it is written as e^x / (1 + e^x). */
static double orc_sigmoid(double x) {
  if (x >= 0.0) return 1.0 / (1.0 + exp(-x));
  double e = exp(x);
  return e / (1.0 + e);
}

/* One activation applied to one value (Table 1 pointwise patterns). */
double oracle_act_scalar(double x, int act) {
  switch (act) {
    case ORC_ACT_NONE: return x;
    case ORC_ACT_RELU: return x > 0.0 ? x : 0.0;
    case ORC_ACT_SIGMOID: return orc_sigmoid(x);
    case ORC_ACT_TANH: return tanh(x);
    case ORC_ACT_SILU: return x * orc_sigmoid(x); /* the x * sigmoid(x) product */
    default: return NAN;
  }
}

/* ---------------------------------------------------------------- Linear */

/* One Linear operator: Y[M][N] = X[M][K] . W[N][K]^T (+ bias[N]), then the
 * optional activation. Row-major, unit inner stride, row strides ldx/ldw/ldy.
 * The sum runs over k in ascending order, in fp64. */
void oracle_linear(const double* x, int64_t ldx, const double* w, int64_t ldw,
                   const double* bias, double* y, int64_t ldy,
                   int64_t M, int64_t N, int64_t K, int act) {
#pragma omp parallel for schedule(static)
  for (int64_t m = 0; m < M; ++m) {
    for (int64_t n = 0; n < N; ++n) {
      double s = 0.0;
      for (int64_t k = 0; k < K; ++k) s += x[m * ldx + k] * w[n * ldw + k];
      if (bias) s += bias[n];
      y[m * ldy + n] = oracle_act_scalar(s, act);
    }
  }
}

/* Only the listed rows of the same Linear (rows[i] for i < nrows), written to
 * y[i][*]. Used to check outputs of groups too large for the full oracle. */
void oracle_linear_rows(const double* x, int64_t ldx, const double* w, int64_t ldw,
                        const double* bias, double* y, int64_t ldy,
                        const int64_t* rows, int64_t nrows, int64_t N, int64_t K, int act) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < nrows; ++i) {
    const double* xr = x + rows[i] * ldx;
    for (int64_t n = 0; n < N; ++n) {
      double s = 0.0;
      for (int64_t k = 0; k < K; ++k) s += xr[k] * w[n * ldw + k];
      if (bias) s += bias[n];
      y[i * ldy + n] = oracle_act_scalar(s, act);
    }
  }
}

/* ------------------------------------------------------------- LayerNorm */

/* One row of LayerNorm over `cols` values:
 *   mu = (1/n) sum x,  var = (1/n) sum (x - mu)^2  (biased, two passes),
 *   y  = (x - mu) / sqrt(var + eps) * gamma + beta, then the activation.
 * gamma == NULL means 1, beta == NULL means 0. */
static void orc_ln_row(const double* x, double* y, int64_t cols, const double* gamma,
                       const double* beta, double eps, int act) {
  double mu = 0.0;
  for (int64_t c = 0; c < cols; ++c) mu += x[c];
  mu /= (double)cols;
  double var = 0.0;
  for (int64_t c = 0; c < cols; ++c) {
    double d = x[c] - mu;
    var += d * d;
  }
  var /= (double)cols;
  double inv = 1.0 / sqrt(var + eps);
  for (int64_t c = 0; c < cols; ++c) {
    double v = (x[c] - mu) * inv;
    if (gamma) v *= gamma[c];
    if (beta) v += beta[c];
    y[c] = oracle_act_scalar(v, act);
  }
}

/* One LayerNorm operator over a [rows, cols] member (normalised dim = last). */
void oracle_layernorm(const double* x, int64_t ldx, double* y, int64_t ldy,
                      int64_t rows, int64_t cols, const double* gamma, const double* beta,
                      double eps, int act) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) orc_ln_row(x + r * ldx, y + r * ldy, cols, gamma, beta, eps, act);
}

/* ------------------------------------------------------------- pointwise */

/* One pointwise operator over a [rows, cols] member. */
void oracle_pointwise(const double* x, int64_t ldx, double* y, int64_t ldy,
                      int64_t rows, int64_t cols, int act) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t c = 0; c < cols; ++c) y[r * ldy + c] = oracle_act_scalar(x[r * ldx + c], act);
}

/* ------------------------------------------------------- split-op-concat */

/* The unoptimised split -> per-piece op -> concat program along dim 1 of a
 * [rows, D] tensor (Sec. 3.2 chained example; appendix Sec. 8.1 listing):
 *   1. split: copy piece j, columns [o_j, o_j + w_j) with o_j = sum_{i<j} w_i,
 *      into its own contiguous [rows, w_j] array;
 *   2. per piece: LayerNorm_j (if apply_ln; gamma[j] / beta[j] may be NULL)
 *      then the activation, into a second array;
 *   3. concat along dim 1: copy each result back at column offset o_j of out.
 * Returns 0 on success, -1 if the widths do not sum to D or allocation fails. */
int oracle_split_op_cat(const double* in, int64_t ldin, double* out, int64_t ldout,
                        int64_t rows, int64_t D, int32_t n_pieces, const int64_t* widths,
                        const double* const* gamma, const double* const* beta,
                        int32_t apply_ln, double eps, int act) {
  int64_t total = 0;
  for (int32_t j = 0; j < n_pieces; ++j) total += widths[j];
  if (total != D) return -1;
  int64_t off = 0;
  for (int32_t j = 0; j < n_pieces; ++j) {
    int64_t w = widths[j];
    double* piece = (double*)malloc(sizeof(double) * (size_t)(rows * w + 1));
    double* res = (double*)malloc(sizeof(double) * (size_t)(rows * w + 1));
    if (!piece || !res) { free(piece); free(res); return -1; }
    for (int64_t r = 0; r < rows; ++r)                      /* 1. split */
      for (int64_t c = 0; c < w; ++c) piece[r * w + c] = in[r * ldin + off + c];
    if (apply_ln)                                           /* 2. per-piece op */
      oracle_layernorm(piece, w, res, w, rows, w, gamma ? gamma[j] : NULL,
                       beta ? beta[j] : NULL, eps, act);
    else
      oracle_pointwise(piece, w, res, w, rows, w, act);
    for (int64_t r = 0; r < rows; ++r)                      /* 3. concat */
      for (int64_t c = 0; c < w; ++c) out[r * ldout + off + c] = res[r * w + c];
    free(piece);
    free(res);
    off += w;
  }
  return 0;
}

/* ---------------------------------------------------------------- backward
 *
 * Training runs the gradients of the grouped operators too (the training
 * column of Table 3; batch_linear_post_grad in Table 1 groups the Linears of
 * the backward graph). They are the derivatives of the forward definitions
 * above, each sum in fp64 in ascending index order. */

/* Linear, given dY = dL/dY of the Linear's output (before any activation):
 *   dX[m][k] = sum_n dY[m][n] W[n][k]
 *   dW[n][k] = sum_m dY[m][n] X[m][k]
 *   db[n]    = sum_m dY[m][n]
 * dx, dw or db may be NULL (not wanted). */
void oracle_linear_backward(const double* x, int64_t ldx, const double* w, int64_t ldw,
                            const double* dy, int64_t lddy, double* dx, int64_t lddx,
                            double* dw, int64_t lddw, double* db, int64_t M, int64_t N, int64_t K) {
  if (dx) {
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m)
      for (int64_t k = 0; k < K; ++k) {
        double s = 0.0;
        for (int64_t n = 0; n < N; ++n) s += dy[m * lddy + n] * w[n * ldw + k];
        dx[m * lddx + k] = s;
      }
  }
  if (dw) {
#pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n)
      for (int64_t k = 0; k < K; ++k) {
        double s = 0.0;
        for (int64_t m = 0; m < M; ++m) s += dy[m * lddy + n] * x[m * ldx + k];
        dw[n * lddw + k] = s;
      }
  }
  if (db) {
    for (int64_t n = 0; n < N; ++n) {
      double s = 0.0;
      for (int64_t m = 0; m < M; ++m) s += dy[m * lddy + n];
      db[n] = s;
    }
  }
}

/* Derivative of one activation at its input x. relu' is 0 at x = 0 (the
 * gradient passes where x > 0, as torch's threshold backward does). */
double oracle_act_grad_scalar(double x, int act) {
  switch (act) {
    case ORC_ACT_NONE: return 1.0;
    case ORC_ACT_RELU: return x > 0.0 ? 1.0 : 0.0;
    case ORC_ACT_SIGMOID: {
      const double s = orc_sigmoid(x);
      return s * (1.0 - s);
    }
    case ORC_ACT_TANH: {
      const double t = tanh(x);
      return 1.0 - t * t;
    }
    case ORC_ACT_SILU: { /* d/dx x s(x) = s + x s (1 - s) */
      const double s = orc_sigmoid(x);
      return s + x * s * (1.0 - s);
    }
    default: return NAN;
  }
}

/* Activation backward over a [rows, cols] member: dX = dY * act'(X). */
void oracle_act_backward(const double* x, int64_t ldx, const double* dy, int64_t lddy, double* dx,
                         int64_t lddx, int64_t rows, int64_t cols, int act) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t c = 0; c < cols; ++c)
      dx[r * lddx + c] = dy[r * lddy + c] * oracle_act_grad_scalar(x[r * ldx + c], act);
}

/* LayerNorm backward over a [rows, cols] member, the statistics recomputed
 * from x as the forward takes them (two-pass biased variance). Per row, with
 * xhat = (x - mu) / sqrt(var + eps) and g = dY * gamma:
 *   dX = (g - mean(g) - xhat * mean(g * xhat)) / sqrt(var + eps)
 * and over all rows dgamma[c] = sum dY * xhat, dbeta[c] = sum dY. gamma
 * NULL means 1; dx, dgamma or dbeta may be NULL. */
void oracle_layernorm_backward(const double* x, int64_t ldx, const double* gamma, const double* dy,
                               int64_t lddy, double* dx, int64_t lddx, double* dgamma, double* dbeta,
                               int64_t rows, int64_t cols, double eps) {
  if (dgamma)
    for (int64_t c = 0; c < cols; ++c) dgamma[c] = 0.0;
  if (dbeta)
    for (int64_t c = 0; c < cols; ++c) dbeta[c] = 0.0;
  for (int64_t r = 0; r < rows; ++r) {
    const double* xr = x + r * ldx;
    const double* gr = dy + r * lddy;
    double mu = 0.0;
    for (int64_t c = 0; c < cols; ++c) mu += xr[c];
    mu /= (double)cols;
    double var = 0.0;
    for (int64_t c = 0; c < cols; ++c) {
      const double d = xr[c] - mu;
      var += d * d;
    }
    var /= (double)cols;
    const double rstd = 1.0 / sqrt(var + eps);
    double mg = 0.0, mgx = 0.0;
    for (int64_t c = 0; c < cols; ++c) {
      const double xhat = (xr[c] - mu) * rstd;
      const double g = gr[c] * (gamma ? gamma[c] : 1.0);
      mg += g;
      mgx += g * xhat;
      if (dgamma) dgamma[c] += gr[c] * xhat;
      if (dbeta) dbeta[c] += gr[c];
    }
    mg /= (double)cols;
    mgx /= (double)cols;
    if (dx)
      for (int64_t c = 0; c < cols; ++c) {
        const double xhat = (xr[c] - mu) * rstd;
        const double g = gr[c] * (gamma ? gamma[c] : 1.0);
        dx[r * lddx + c] = (g - mg - xhat * mgx) * rstd;
      }
  }
}

/* ------------------------------------------------------- fp8 activation codec
 *
 * The activation-quantization rewrite (paper Sec. 5 memory results; appendix
 * Sec. 8.2, peak memory usage reduction) stores saved activations in FP8 in
 * the forward pass and restores them before use in the backward pass, with
 * or without a per-tensor scale; without the scale, values that overflow FP8
 * become NaN. FP8 here is the OCP E4M3 format: sign, 4 exponent bits (bias 7),
 * 3 mantissa bits, no infinities, S.1111.111 = NaN, largest finite 448,
 * smallest normal 2^-6, subnormals m * 2^-9 (m = 1..7). Rounding is to
 * nearest, ties to even.
 *
 * Scaled mode: amax = max |x| over the tensor (NaN ignored), scale = amax/448
 * and inv = 448/amax in fp32 (1 and 1 when amax is 0); code = E4M3(fp32(x *
 * inv)), clamped to +-448. Unscaled mode: code = E4M3(x), magnitudes that
 * round above 448 (|x| > 464; 464 itself is a tie that goes to the even 448)
 * give NaN. A NaN input gives the NaN code with the input's sign in both
 * modes; so does an infinite input in scaled mode (amax is then infinite,
 * inv is 0 and x * inv is NaN). Decode: the code's value times scale in
 * fp32. Every fp32 step is
 * written in fp32 (float) arithmetic, so a quantised code is decided in the
 * same precision on every implementation. */

/* Value of an E4M3 code (NaN for S.1111.111). */
double oracle_fp8e4m3_decode(int code) {
  const int s = (code >> 7) & 1, e = (code >> 3) & 15, m = code & 7;
  if (e == 15 && m == 7) return NAN;
  const double mag = e == 0 ? ldexp((double)m, -9) : ldexp(1.0 + m / 8.0, e - 7);
  return s ? -mag : mag;
}

/* E4M3 code of a finite or non-finite value; saturate: clamp overflow to
 * +-448 instead of NaN. */
int oracle_fp8e4m3_encode(double v, int saturate) {
  const int s = signbit(v) ? 0x80 : 0;
  if (isnan(v)) return s | 0x7F; /* NaN keeps its sign, in both modes */
  double a = fabs(v);
  /* 464 is halfway between 448 (mantissa 110) and the next step 480 (111,
   * the NaN pattern): ties-to-even takes 448, so only larger magnitudes
   * overflow (infinities too). */
  if (a > 464.0) return saturate ? (s | 0x7E) : (s | 0x7F);
  int code;
  if (a < ldexp(1.0, -6)) {
    /* subnormal range: steps of 2^-9; 8 steps is the smallest normal (code 8) */
    code = (int)nearbyint(a / ldexp(1.0, -9));
  } else {
    int e2;
    frexp(a, &e2);                              /* a = f * 2^e2, f in [0.5, 1) */
    const int e = e2 - 1;                       /* a in [2^e, 2^(e+1)) */
    long q = (long)nearbyint(a / ldexp(1.0, e - 3)); /* 8 ..16 mantissa steps */
    int ef = e;
    if (q == 16) { q = 8; ef = e + 1; }
    code = ((ef + 7) << 3) | (int)(q - 8);
  }
  if (code > 0x7E) code = saturate ? 0x7E : 0x7F;
  return s | code;
}

/* One tensor x[rows][cols] (fp32 values given exactly as doubles) to codes
 * q[rows][ldq]; *scale_out receives the fp32 scale (scaled mode only). */
void oracle_quantize_fp8(const double* x, int64_t ldx, uint8_t* q, int64_t ldq, int64_t rows, int64_t cols,
                         int use_scaling, float* scale_out) {
  float inv = 1.0f, scale = 1.0f;
  if (use_scaling) {
    float amax = 0.0f;
    for (int64_t r = 0; r < rows; ++r)
      for (int64_t c = 0; c < cols; ++c) {
        const float a = fabsf((float)x[r * ldx + c]);
        if (a > amax) amax = a; /* NaN compares false: ignored */
      }
    if (amax > 0.0f) {
      scale = amax / 448.0f;
      inv = 448.0f / amax;
    }
    if (scale_out) *scale_out = scale;
  }
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t c = 0; c < cols; ++c) {
      const float xv = (float)x[r * ldx + c];
      const float v = use_scaling ? xv * inv : xv;
      /* A NaN value takes the sign of x itself: the sign of the NaN that
       * +-inf * 0 yields (amax infinite, so inv = 0) differs between
       * platforms. */
      q[r * ldq + c] = isnan(v) ? (uint8_t)(signbit(xv) ? 0xFF : 0x7F)
                                : (uint8_t)oracle_fp8e4m3_encode((double)v, use_scaling);
    }
}

/* Codes q[rows][ldq] back to values y = fp32(decode(code) * scale). */
void oracle_dequantize_fp8(const uint8_t* q, int64_t ldq, double* y, int64_t ldy, int64_t rows, int64_t cols,
                           float scale) {
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t c = 0; c < cols; ++c) {
      const float v = (float)oracle_fp8e4m3_decode(q[r * ldq + c]);
      y[r * ldy + c] = (double)(v * scale);
    }
}

/* Threads for the following parallel loops (n >= 1; no effect without
 * OpenMP). Results do not depend on it: every loop writes disjoint outputs. */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
  extern void omp_set_num_threads(int);
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* Number of OpenMP threads the oracle's parallel loops use (1 without OpenMP). */
int oracle_num_threads(void) {
#ifdef _OPENMP
  extern int omp_get_max_threads(void);
  return omp_get_max_threads();
#else
  return 1;
#endif
}
