/* Drives every entry point of the C oracle on small ragged, strided and
 * edge-case inputs. Built with AddressSanitizer and UndefinedBehaviorSanitizer
 * by tests/test_oracle_sanitized.py: buffers are allocated to the exact
 * extent the layouts address (the last row holds only `cols` values), so any
 * access past a member, a leak or undefined behaviour fails the run. The
 * values themselves are checked by the pins, not here. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

double oracle_act_scalar(double x, int act);
double oracle_act_grad_scalar(double x, int act);
void oracle_linear(const double* x, int64_t ldx, const double* w, int64_t ldw, const double* bias, double* y,
                   int64_t ldy, int64_t M, int64_t N, int64_t K, int act);
void oracle_linear_rows(const double* x, int64_t ldx, const double* w, int64_t ldw, const double* bias, double* y,
                        int64_t ldy, const int64_t* rows, int64_t nrows, int64_t N, int64_t K, int act);
void oracle_layernorm(const double* x, int64_t ldx, double* y, int64_t ldy, int64_t rows, int64_t cols,
                      const double* gamma, const double* beta, double eps, int act);
void oracle_pointwise(const double* x, int64_t ldx, double* y, int64_t ldy, int64_t rows, int64_t cols, int act);
int oracle_split_op_cat(const double* in, int64_t ldin, double* out, int64_t ldout, int64_t rows, int64_t D,
                        int32_t n_pieces, const int64_t* widths, const double* const* gamma,
                        const double* const* beta, int32_t apply_ln, double eps, int act);
void oracle_linear_backward(const double* x, int64_t ldx, const double* w, int64_t ldw, const double* dy,
                            int64_t lddy, double* dx, int64_t lddx, double* dw, int64_t lddw, double* db, int64_t M,
                            int64_t N, int64_t K);
void oracle_act_backward(const double* x, int64_t ldx, const double* dy, int64_t lddy, double* dx, int64_t lddx,
                         int64_t rows, int64_t cols, int act);
void oracle_layernorm_backward(const double* x, int64_t ldx, const double* gamma, const double* dy, int64_t lddy,
                               double* dx, int64_t lddx, double* dgamma, double* dbeta, int64_t rows, int64_t cols,
                               double eps);
double oracle_fp8e4m3_decode(int code);
int oracle_fp8e4m3_encode(double v, int saturate);
void oracle_quantize_fp8(const double* x, int64_t ldx, uint8_t* q, int64_t ldq, int64_t rows, int64_t cols,
                         int use_scaling, float* scale_out);
void oracle_dequantize_fp8(const uint8_t* q, int64_t ldq, double* y, int64_t ldy, int64_t rows, int64_t cols,
                           float scale);
void oracle_set_num_threads(int n);
int oracle_num_threads(void);

static uint64_t state = 88172645463325252ull;
static double draw(void) { /* xorshift64, values in [-2, 2) */
  state ^= state << 13;
  state ^= state >> 7;
  state ^= state << 17;
  return (double)(state >> 11) / 9007199254740992.0 * 4.0 - 2.0;
}

/* rows x cols at row stride ld, allocated to the last addressed element */
static size_t extent(int64_t rows, int64_t ld, int64_t cols) {
  return rows > 0 && cols > 0 ? (size_t)((rows - 1) * ld + cols) : 1;
}
static double* mat(int64_t rows, int64_t ld, int64_t cols) {
  const size_t n = extent(rows, ld, cols);
  double* p = (double*)malloc(n * sizeof(double));
  for (size_t i = 0; i < n; ++i) p[i] = draw();
  return p;
}
static void need(int ok, const char* what) {
  if (!ok) {
    fprintf(stderr, "FAILED: %s\n", what);
    exit(1);
  }
}

int main(void) {
  oracle_set_num_threads(2);
  need(oracle_num_threads() >= 1, "threads");
  const double specials[] = {0.0, -0.0, 1e-300, -3.5, 40.0, -800.0, INFINITY, -INFINITY, NAN};
  for (int a = 0; a < 5; ++a)
    for (size_t i = 0; i < sizeof specials / sizeof specials[0]; ++i) {
      (void)oracle_act_scalar(specials[i], a);
      (void)oracle_act_grad_scalar(specials[i], a);
    }

  /* Linear and its backward: (M, N, K) with padded and unpadded strides */
  const int64_t shapes[][3] = {{1, 1, 1}, {3, 5, 7}, {17, 9, 33}, {2, 64, 1}};
  for (size_t s = 0; s < sizeof shapes / sizeof shapes[0]; ++s)
    for (int pad = 0; pad <= 3; pad += 3) {
      const int64_t M = shapes[s][0], N = shapes[s][1], K = shapes[s][2];
      const int64_t ldx = K + pad, ldw = K + pad, ldy = N + pad;
      double *x = mat(M, ldx, K), *w = mat(N, ldw, K), *b = mat(1, N, N), *y = mat(M, ldy, N);
      for (int a = 0; a < 5; ++a) {
        oracle_linear(x, ldx, w, ldw, a & 1 ? NULL : b, y, ldy, M, N, K, a);
        need(isfinite(y[0]), "linear output");
      }
      const int64_t rows[2] = {M - 1, 0};
      double* yr = mat(2, N, N);
      oracle_linear_rows(x, ldx, w, ldw, b, yr, N, rows, 2, N, K, 3);
      double *dy = mat(M, ldy, N), *dx = mat(M, ldx, K), *dw = mat(N, ldw, K), *db = mat(1, N, N);
      oracle_linear_backward(x, ldx, w, ldw, dy, ldy, dx, ldx, dw, ldw, db, M, N, K);
      oracle_linear_backward(x, ldx, w, ldw, dy, ldy, NULL, ldx, dw, ldw, NULL, M, N, K);
      oracle_linear_backward(x, ldx, w, ldw, dy, ldy, dx, ldx, NULL, ldw, NULL, M, N, K);
      free(x), free(w), free(b), free(y), free(yr), free(dy), free(dx), free(dw), free(db);
    }

  /* LayerNorm, pointwise and their backward: (rows, cols), strided */
  const int64_t rc[][2] = {{1, 1}, {4, 13}, {5, 64}, {3, 2}};
  for (size_t s = 0; s < sizeof rc / sizeof rc[0]; ++s)
    for (int pad = 0; pad <= 5; pad += 5) {
      const int64_t R = rc[s][0], C = rc[s][1], ld = C + pad;
      double *x = mat(R, ld, C), *y = mat(R, ld, C), *g = mat(1, C, C), *be = mat(1, C, C);
      double *dy = mat(R, ld, C), *dx = mat(R, ld, C), *dg = mat(1, C, C), *db = mat(1, C, C);
      for (int a = 0; a < 5; ++a) {
        oracle_layernorm(x, ld, y, ld, R, C, a & 1 ? NULL : g, a & 2 ? NULL : be, 1e-5, a);
        oracle_pointwise(x, ld, y, ld, R, C, a);
        oracle_act_backward(x, ld, dy, ld, dx, ld, R, C, a);
      }
      oracle_layernorm_backward(x, ld, g, dy, ld, dx, ld, dg, db, R, C, 1e-5);
      oracle_layernorm_backward(x, ld, NULL, dy, ld, dx, ld, NULL, db, R, C, 0.0);
      oracle_layernorm_backward(x, ld, g, dy, ld, NULL, ld, dg, NULL, R, C, 1e-5);
      /* a constant row: zero variance */
      for (int64_t c = 0; c < C; ++c) x[c] = 0.75;
      oracle_layernorm(x, ld, y, ld, 1, C, g, be, 1e-5, 0);
      need(isfinite(y[0]), "constant row");
      free(x), free(y), free(g), free(be), free(dy), free(dx), free(dg), free(db);
    }

  /* split-op-cat: ragged widths, strided buffers, a NULL gamma entry, widths
   * that do not sum to D */
  {
    const int64_t R = 3, D = 8, ld = 11, widths[3] = {3, 1, 4}, bad[3] = {3, 1, 3};
    double *in = mat(R, ld, D), *out = mat(R, ld, D);
    double *g0 = mat(1, 3, 3), *g2 = mat(1, 4, 4), *b1 = mat(1, 1, 1);
    const double* gam[3] = {g0, NULL, g2};
    const double* bet[3] = {NULL, b1, NULL};
    for (int a = 0; a < 5; ++a) {
      need(oracle_split_op_cat(in, ld, out, ld, R, D, 3, widths, gam, bet, 1, 1e-5, a) == 0, "split-op-cat");
      need(oracle_split_op_cat(in, ld, out, ld, R, D, 3, widths, NULL, NULL, a & 1, 1e-5, a) == 0, "split-op-cat");
    }
    need(oracle_split_op_cat(in, ld, out, ld, R, D, 3, bad, NULL, NULL, 1, 1e-5, 0) == -1, "widths off D");
    free(in), free(out), free(g0), free(g2), free(b1);
  }

  /* fp8: every code, special values, and a strided tensor with NaN / inf */
  for (int c = 0; c < 256; ++c) {
    const double v = oracle_fp8e4m3_decode(c);
    if (!isnan(v)) need(oracle_fp8e4m3_encode(v, 0) == c || v == 0.0, "fp8 round trip");
  }
  const double enc[] = {0.0, -0.0, 448.0, 464.0, 464.0000001, 1e9, -1e9, 1e-12, INFINITY, -INFINITY, NAN};
  for (size_t i = 0; i < sizeof enc / sizeof enc[0]; ++i) {
    need(oracle_fp8e4m3_encode(enc[i], 0) >= 0, "encode");
    need(oracle_fp8e4m3_encode(enc[i], 1) >= 0, "encode saturated");
  }
  {
    const int64_t R = 3, C = 5, ld = 7, ldq = 6;
    double* x = mat(R, ld, C);
    uint8_t* q = (uint8_t*)malloc(extent(R, ldq, C));
    double* y = mat(R, ld, C);
    float scale = 0.f;
    oracle_quantize_fp8(x, ld, q, ldq, R, C, 1, &scale);
    oracle_dequantize_fp8(q, ldq, y, ld, R, C, scale);
    x[1] = NAN, x[ld + 2] = INFINITY, x[2 * ld] = -INFINITY;
    oracle_quantize_fp8(x, ld, q, ldq, R, C, 1, &scale);
    oracle_quantize_fp8(x, ld, q, ldq, R, C, 0, NULL);
    oracle_dequantize_fp8(q, ldq, y, ld, R, C, 1.0f);
    memset(x, 0, extent(R, ld, C) * sizeof(double));
    oracle_quantize_fp8(x, ld, q, ldq, R, C, 1, &scale);
    need(scale == 1.0f, "zero amax");
    free(x), free(q), free(y);
  }
  printf("oracle under sanitizers: ok\n");
  return 0;
}
