// liboptimus C ABI: descriptor validation, the host planner (device descriptor
// tables and tile schedules), plans, and the one-shot entry points.
//
// A group is a set of independent operator instances of one type, dtype and
// activation (paper Sec. 3.2 group fusion; Sec. 4.1: instances are independent
// when no data dependency exists between them; the grouping key of Alg. 1
// encodes such metadata). The planner turns the caller's per-member
// descriptors into one device table plus a list of work items, so that the
// whole group runs as ONE kernel launch; the same tables also drive the
// unfused per-member launch chain used as the baseline.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <cstddef>
#include <string>
#include <vector>

#include "optimus.h"
#include "optimus_internal.h"

using namespace optimus;

// ===================================================================== errors
static thread_local std::string g_last_error;

static optimus_status fail(optimus_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

static optimus_status hip_fail(hipError_t e, const char* what) {
  if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation)
    return fail(OPTIMUS_ERR_OOM, "%s: %s", what, hipGetErrorString(e));
  return fail(OPTIMUS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(call, what)                 \
  do {                                      \
    hipError_t e_ = (call);                 \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

extern "C" const char* optimus_last_error(void) { return g_last_error.c_str(); }
extern "C" const char* optimus_version(void) { return "liboptimus 0.1 (gfx950)"; }

namespace optimus {
int device_cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}
}  // namespace optimus

// ===================================================================== validation
static size_t dtype_size(optimus_dtype dt) { return dt == OPTIMUS_F32 ? 4 : 2; }
static bool dtype_ok(optimus_dtype dt) { return dt == OPTIMUS_F32 || dt == OPTIMUS_BF16; }
static bool act_ok(optimus_act a) { return (int)a >= OPTIMUS_ACT_NONE && (int)a <= OPTIMUS_ACT_SILU; }
static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
static const int64_t kMaxDim = 0x7fffffff;

// A 2-D memory region: `rows` runs of `row_bytes` bytes, `ld_bytes` apart.
struct Region {
  uintptr_t base;
  int64_t ld_bytes, rows, row_bytes;
  int member;
  bool output;
  uintptr_t lo() const { return base; }
  uintptr_t hi() const { return base + (uintptr_t)((rows - 1) * ld_bytes + row_bytes); }
  bool same(const Region& o) const {
    return base == o.base && ld_bytes == o.ld_bytes && rows == o.rows && row_bytes == o.row_bytes;
  }
};

// Exact test for two regions with a common row stride whose runs fit inside
// one stride (slices of one buffer); bounding-range test otherwise.
static bool regions_overlap(const Region& a, const Region& b) {
  if (a.hi() <= b.lo() || b.hi() <= a.lo()) return false;
  if (a.ld_bytes != b.ld_bytes || a.row_bytes > a.ld_bytes || b.row_bytes > b.ld_bytes || a.ld_bytes <= 0) return true;
  const int64_t l = a.ld_bytes;
  const int64_t delta = (int64_t)(b.base - a.base);  // may be negative (two's complement)
  // runs a_i = [i l, i l + ra) and b_j = [delta + j l, delta + j l + rb) meet iff for k = j - i:
  // -rb < delta + k l < ra; k ranges over [-(a.rows-1), b.rows-1]
  const int64_t ra = a.row_bytes, rb = b.row_bytes;
  auto floor_div = [](int64_t p, int64_t q) { return p >= 0 ? p / q : -((-p + q - 1) / q); };
  int64_t k_lo = floor_div(-rb - delta, l) + 1;  // smallest k with k l > -rb - delta
  int64_t k_hi = floor_div(ra - delta - 1, l);   // largest k with k l < ra - delta
  k_lo = std::max(k_lo, -(a.rows - 1));
  k_hi = std::min(k_hi, b.rows - 1);
  return k_lo <= k_hi;
}

// Members must be independent: no output may overlap any input or any other
// output. Exact in-place (an output identical to the same member's input) is
// permitted when `allow_inplace`.
static optimus_status check_aliasing(std::vector<Region>& regs, bool allow_inplace, const char* what) {
  std::sort(regs.begin(), regs.end(), [](const Region& a, const Region& b) { return a.lo() < b.lo(); });
  for (size_t i = 0; i < regs.size(); ++i) {
    for (size_t j = i + 1; j < regs.size() && regs[j].lo() < regs[i].hi(); ++j) {
      const Region& a = regs[i];
      const Region& b = regs[j];
      if (!a.output && !b.output) continue;
      if (allow_inplace && a.member == b.member && a.output != b.output && a.same(b)) continue;
      if (regions_overlap(a, b))
        return fail(OPTIMUS_ERR_ALIASING, "%s: member %d %s overlaps member %d %s (members must be independent)", what,
                    a.member, a.output ? "output" : "input", b.member, b.output ? "output" : "input");
    }
  }
  return OPTIMUS_OK;
}

static Region region(const void* p, int64_t ld, int64_t rows, int64_t cols, size_t s, int member, bool out) {
  return Region{(uintptr_t)p, ld * (int64_t)s, rows, cols * (int64_t)s, member, out};
}

// Linear members, and with `ln` the LayerNorm fused over their output rows
// (gamma / beta: host arrays of G device pointers, or NULL).
static optimus_status validate_linear_impl(const optimus_linear_desc* d, int32_t G, optimus_dtype dt, optimus_act act,
                                           bool ln, const void* const* gamma, const void* const* beta, float eps) {
  const char* what = ln ? "grouped_linear_layernorm" : "grouped_linear";
  if (G < 0) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: G = %d < 0", what, G);
  if (!dtype_ok(dt)) return fail(OPTIMUS_ERR_UNSUPPORTED, "%s: unknown dtype %d", what, (int)dt);
  if (!act_ok(act)) return fail(OPTIMUS_ERR_UNSUPPORTED, "%s: unknown activation %d", what, (int)act);
  if (ln && (!(eps >= 0.f) || !std::isfinite(eps))) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: eps=%g", what, (double)eps);
  if (G == 0) return OPTIMUS_OK;
  if (!d) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: descriptor array is NULL", what);
  const size_t s = dtype_size(dt);
  std::vector<Region> regs;
  regs.reserve((size_t)G * 6);
  for (int g = 0; g < G; ++g) {
    const optimus_linear_desc& m = d[g];
    if (!m.x || !m.w || !m.y) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has a NULL x/w/y", what, g);
    if (m.M < 1 || m.N < 1 || m.K < 1 || m.M > kMaxDim || m.N > kMaxDim || m.K > kMaxDim)
      return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has M=%lld N=%lld K=%lld (need 1..2^31-1)", what, g,
                  (long long)m.M, (long long)m.N, (long long)m.K);
    if (m.ldx < m.K || m.ldw < m.K || m.ldy < m.N)
      return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has a row stride below its row length", what, g);
    if (ln && m.N > gemm_ln_max_n(dt))
      return fail(OPTIMUS_ERR_UNSUPPORTED, "%s: member %d has N=%lld; a fused LayerNorm takes rows of at most %d",
                  what, g, (long long)m.N, gemm_ln_max_n(dt));
    regs.push_back(region(m.x, m.ldx, m.M, m.K, s, g, false));
    regs.push_back(region(m.w, m.ldw, m.N, m.K, s, g, false));
    if (m.bias) regs.push_back(region(m.bias, m.N, 1, m.N, s, g, false));
    if (ln && gamma && gamma[g]) regs.push_back(region(gamma[g], m.N, 1, m.N, s, g, false));
    if (ln && beta && beta[g]) regs.push_back(region(beta[g], m.N, 1, m.N, s, g, false));
    regs.push_back(region(m.y, m.ldy, m.M, m.N, s, g, true));
  }
  return check_aliasing(regs, false, what);
}

extern "C" optimus_status optimus_validate_linear(const optimus_linear_desc* d, int32_t G, optimus_dtype dt,
                                                  optimus_act act) {
  return validate_linear_impl(d, G, dt, act, false, nullptr, nullptr, 0.f);
}

extern "C" optimus_status optimus_validate_linear_layernorm(const optimus_linear_desc* d, const void* const* gamma,
                                                            const void* const* beta, int32_t G, optimus_dtype dt,
                                                            float eps, optimus_act act) {
  return validate_linear_impl(d, G, dt, act, true, gamma, beta, eps);
}

extern "C" optimus_status optimus_validate_layernorm(const optimus_layernorm_desc* d, int32_t G, optimus_dtype dt,
                                                     optimus_act act) {
  if (G < 0) return fail(OPTIMUS_ERR_INVALID_ARG, "grouped_layernorm: G = %d < 0", G);
  if (!dtype_ok(dt)) return fail(OPTIMUS_ERR_UNSUPPORTED, "grouped_layernorm: unknown dtype %d", (int)dt);
  if (!act_ok(act)) return fail(OPTIMUS_ERR_UNSUPPORTED, "grouped_layernorm: unknown activation %d", (int)act);
  if (G == 0) return OPTIMUS_OK;
  if (!d) return fail(OPTIMUS_ERR_INVALID_ARG, "grouped_layernorm: descriptor array is NULL");
  const size_t s = dtype_size(dt);
  std::vector<Region> regs;
  regs.reserve((size_t)G * 4);
  for (int g = 0; g < G; ++g) {
    const optimus_layernorm_desc& m = d[g];
    if (!m.x || !m.y) return fail(OPTIMUS_ERR_INVALID_ARG, "grouped_layernorm: member %d has a NULL x/y", g);
    if (m.rows < 1 || m.cols < 1 || m.rows > kMaxDim || m.cols > kMaxDim)
      return fail(OPTIMUS_ERR_INVALID_ARG, "grouped_layernorm: member %d has rows=%lld cols=%lld", g,
                  (long long)m.rows, (long long)m.cols);
    if (m.ldx < m.cols || m.ldy < m.cols)
      return fail(OPTIMUS_ERR_INVALID_ARG, "grouped_layernorm: member %d has a row stride below cols", g);
    if (!(m.eps >= 0.f) || !std::isfinite(m.eps))
      return fail(OPTIMUS_ERR_INVALID_ARG, "grouped_layernorm: member %d has eps=%g", g, (double)m.eps);
    regs.push_back(region(m.x, m.ldx, m.rows, m.cols, s, g, false));
    if (m.gamma) regs.push_back(region(m.gamma, m.cols, 1, m.cols, s, g, false));
    if (m.beta) regs.push_back(region(m.beta, m.cols, 1, m.cols, s, g, false));
    regs.push_back(region(m.y, m.ldy, m.rows, m.cols, s, g, true));
  }
  return check_aliasing(regs, true, "grouped_layernorm");
}

extern "C" optimus_status optimus_validate_pointwise(const optimus_pointwise_desc* d, int32_t G, optimus_dtype dt,
                                                     optimus_act act) {
  if (G < 0) return fail(OPTIMUS_ERR_INVALID_ARG, "grouped_pointwise: G = %d < 0", G);
  if (!dtype_ok(dt)) return fail(OPTIMUS_ERR_UNSUPPORTED, "grouped_pointwise: unknown dtype %d", (int)dt);
  if (!act_ok(act)) return fail(OPTIMUS_ERR_UNSUPPORTED, "grouped_pointwise: unknown activation %d", (int)act);
  if (G == 0) return OPTIMUS_OK;
  if (!d) return fail(OPTIMUS_ERR_INVALID_ARG, "grouped_pointwise: descriptor array is NULL");
  const size_t s = dtype_size(dt);
  std::vector<Region> regs;
  regs.reserve((size_t)G * 2);
  for (int g = 0; g < G; ++g) {
    const optimus_pointwise_desc& m = d[g];
    if (!m.x || !m.y) return fail(OPTIMUS_ERR_INVALID_ARG, "grouped_pointwise: member %d has a NULL x/y", g);
    if (m.rows < 1 || m.cols < 1 || m.rows > kMaxDim || m.cols > kMaxDim)
      return fail(OPTIMUS_ERR_INVALID_ARG, "grouped_pointwise: member %d has rows=%lld cols=%lld", g,
                  (long long)m.rows, (long long)m.cols);
    if (m.ldx < m.cols || m.ldy < m.cols)
      return fail(OPTIMUS_ERR_INVALID_ARG, "grouped_pointwise: member %d has a row stride below cols", g);
    regs.push_back(region(m.x, m.ldx, m.rows, m.cols, s, g, false));
    regs.push_back(region(m.y, m.ldy, m.rows, m.cols, s, g, true));
  }
  return check_aliasing(regs, true, "grouped_pointwise");
}

extern "C" optimus_status optimus_validate_split_op_cat(const optimus_split_op_cat_desc* d, optimus_dtype dt) {
  if (!d) return fail(OPTIMUS_ERR_INVALID_ARG, "split_op_cat: descriptor is NULL");
  if (!dtype_ok(dt)) return fail(OPTIMUS_ERR_UNSUPPORTED, "split_op_cat: unknown dtype %d", (int)dt);
  if (!act_ok(d->act)) return fail(OPTIMUS_ERR_UNSUPPORTED, "split_op_cat: unknown activation %d", (int)d->act);
  if (!d->in || !d->out) return fail(OPTIMUS_ERR_INVALID_ARG, "split_op_cat: NULL in/out");
  if (d->rows < 1 || d->D < 1 || d->rows > kMaxDim || d->D > kMaxDim)
    return fail(OPTIMUS_ERR_INVALID_ARG, "split_op_cat: rows=%lld D=%lld", (long long)d->rows, (long long)d->D);
  if (d->ldin < d->D || d->ldout < d->D) return fail(OPTIMUS_ERR_INVALID_ARG, "split_op_cat: row stride below D");
  if (d->n_slices < 1 || !d->widths) return fail(OPTIMUS_ERR_INVALID_ARG, "split_op_cat: need n_slices >= 1 and widths");
  int64_t total = 0;
  for (int j = 0; j < d->n_slices; ++j) {
    if (d->widths[j] < 1) return fail(OPTIMUS_ERR_INVALID_ARG, "split_op_cat: width[%d] = %lld < 1", j, (long long)d->widths[j]);
    total += d->widths[j];
  }
  if (total != d->D)
    return fail(OPTIMUS_ERR_INVALID_ARG, "split_op_cat: widths sum to %lld, not D = %lld", (long long)total, (long long)d->D);
  if (d->apply_layernorm && (!(d->eps >= 0.f) || !std::isfinite(d->eps)))
    return fail(OPTIMUS_ERR_INVALID_ARG, "split_op_cat: eps=%g", (double)d->eps);
  const size_t s = dtype_size(dt);
  std::vector<Region> regs;
  regs.push_back(region(d->in, d->ldin, d->rows, d->D, s, 0, false));
  regs.push_back(region(d->out, d->ldout, d->rows, d->D, s, 0, true));
  if (d->apply_layernorm) {
    for (int j = 0; j < d->n_slices; ++j) {
      if (d->gamma && d->gamma[j]) regs.push_back(region(d->gamma[j], d->widths[j], 1, d->widths[j], s, 0, false));
      if (d->beta && d->beta[j]) regs.push_back(region(d->beta[j], d->widths[j], 1, d->widths[j], s, 0, false));
    }
  }
  return check_aliasing(regs, true, "split_op_cat");
}

extern "C" optimus_status optimus_validate_linear_backward(const optimus_linear_grad_desc* d, int32_t G,
                                                          optimus_dtype dt) {
  const char* what = "grouped_linear_backward";
  if (G < 0) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: G = %d < 0", what, G);
  if (!dtype_ok(dt)) return fail(OPTIMUS_ERR_UNSUPPORTED, "%s: unknown dtype %d", what, (int)dt);
  if (G == 0) return OPTIMUS_OK;
  if (!d) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: descriptor array is NULL", what);
  const size_t s = dtype_size(dt);
  std::vector<Region> regs;
  regs.reserve((size_t)G * 6);
  for (int g = 0; g < G; ++g) {
    const optimus_linear_grad_desc& m = d[g];
    if (!m.dy) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has a NULL dy", what, g);
    if (m.dx && !m.w) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d wants dx but has a NULL w", what, g);
    if (m.dw && !m.x) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d wants dw but has a NULL x", what, g);
    if (m.db && !m.dw)
      return fail(OPTIMUS_ERR_UNSUPPORTED, "%s: member %d wants db without dw (db is summed by the dW launch)", what, g);
    if (m.M < 1 || m.N < 1 || m.K < 1 || m.M > kMaxDim || m.N > kMaxDim || m.K > kMaxDim)
      return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has M=%lld N=%lld K=%lld (need 1..2^31-1)", what, g,
                  (long long)m.M, (long long)m.N, (long long)m.K);
    if (m.lddy < m.N || (m.dw && m.ldx < m.K) || (m.dx && m.ldw < m.K) || (m.dx && m.lddx < m.K) ||
        (m.dw && m.lddw < m.K))
      return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has a row stride below its row length", what, g);
    regs.push_back(region(m.dy, m.lddy, m.M, m.N, s, g, false));
    if (m.dw) regs.push_back(region(m.x, m.ldx, m.M, m.K, s, g, false));
    if (m.dx) regs.push_back(region(m.w, m.ldw, m.N, m.K, s, g, false));
    if (m.dx) regs.push_back(region(m.dx, m.lddx, m.M, m.K, s, g, true));
    if (m.dw) regs.push_back(region(m.dw, m.lddw, m.N, m.K, s, g, true));
    if (m.db) regs.push_back(region(m.db, m.N, 1, m.N, s, g, true));
  }
  return check_aliasing(regs, false, what);
}

extern "C" optimus_status optimus_validate_layernorm_backward(const optimus_layernorm_grad_desc* d, int32_t G,
                                                             optimus_dtype dt) {
  const char* what = "grouped_layernorm_backward";
  if (G < 0) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: G = %d < 0", what, G);
  if (!dtype_ok(dt)) return fail(OPTIMUS_ERR_UNSUPPORTED, "%s: unknown dtype %d", what, (int)dt);
  if (G == 0) return OPTIMUS_OK;
  if (!d) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: descriptor array is NULL", what);
  const size_t s = dtype_size(dt);
  std::vector<Region> regs;
  regs.reserve((size_t)G * 6);
  for (int g = 0; g < G; ++g) {
    const optimus_layernorm_grad_desc& m = d[g];
    if (!m.x || !m.dy || !m.dx) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has a NULL x/dy/dx", what, g);
    if (m.rows < 1 || m.cols < 1 || m.rows > kMaxDim || m.cols > kMaxDim)
      return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has rows=%lld cols=%lld", what, g, (long long)m.rows,
                  (long long)m.cols);
    if (m.ldx < m.cols || m.lddy < m.cols || m.lddx < m.cols)
      return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has a row stride below cols", what, g);
    if (!(m.eps >= 0.f) || !std::isfinite(m.eps))
      return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has eps=%g", what, g, (double)m.eps);
    regs.push_back(region(m.x, m.ldx, m.rows, m.cols, s, g, false));
    regs.push_back(region(m.dy, m.lddy, m.rows, m.cols, s, g, false));
    if (m.gamma) regs.push_back(region(m.gamma, m.cols, 1, m.cols, s, g, false));
    regs.push_back(region(m.dx, m.lddx, m.rows, m.cols, s, g, true));
    if (m.dgamma) regs.push_back(region(m.dgamma, m.cols, 1, m.cols, s, g, true));
    if (m.dbeta) regs.push_back(region(m.dbeta, m.cols, 1, m.cols, s, g, true));
  }
  return check_aliasing(regs, true, what);
}

extern "C" optimus_status optimus_validate_act_backward(const optimus_act_grad_desc* d, int32_t G, optimus_dtype dt,
                                                        optimus_act act) {
  const char* what = "grouped_act_backward";
  if (G < 0) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: G = %d < 0", what, G);
  if (!dtype_ok(dt)) return fail(OPTIMUS_ERR_UNSUPPORTED, "%s: unknown dtype %d", what, (int)dt);
  if (!act_ok(act)) return fail(OPTIMUS_ERR_UNSUPPORTED, "%s: unknown activation %d", what, (int)act);
  if (G == 0) return OPTIMUS_OK;
  if (!d) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: descriptor array is NULL", what);
  const size_t s = dtype_size(dt);
  std::vector<Region> regs;
  regs.reserve((size_t)G * 3);
  for (int g = 0; g < G; ++g) {
    const optimus_act_grad_desc& m = d[g];
    if (!m.x || !m.dy || !m.dx) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has a NULL x/dy/dx", what, g);
    if (m.rows < 1 || m.cols < 1 || m.rows > kMaxDim || m.cols > kMaxDim)
      return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has rows=%lld cols=%lld", what, g, (long long)m.rows,
                  (long long)m.cols);
    if (m.ldx < m.cols || m.lddy < m.cols || m.lddx < m.cols)
      return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has a row stride below cols", what, g);
    regs.push_back(region(m.x, m.ldx, m.rows, m.cols, s, g, false));
    regs.push_back(region(m.dy, m.lddy, m.rows, m.cols, s, g, false));
    regs.push_back(region(m.dx, m.lddx, m.rows, m.cols, s, g, true));
  }
  return check_aliasing(regs, true, what);
}

static optimus_status validate_fp8_member(const char* what, int g, const void* a, int64_t lda, size_t sa,
                                          const void* b, int64_t ldb, size_t sb, int64_t rows, int64_t cols) {
  if (!a || !b) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has a NULL tensor", what, g);
  if (rows < 1 || cols < 1 || rows > kMaxDim || cols > kMaxDim)
    return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has rows=%lld cols=%lld", what, g, (long long)rows,
                (long long)cols);
  if (lda < cols || ldb < cols) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d has a row stride below cols", what, g);
  (void)sa;
  (void)sb;
  return OPTIMUS_OK;
}

extern "C" optimus_status optimus_validate_quantize_fp8(const optimus_fp8_quant_desc* d, int32_t G, optimus_dtype dt,
                                                        int32_t use_scaling) {
  const char* what = "grouped_quantize_fp8";
  if (G < 0) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: G = %d < 0", what, G);
  if (!dtype_ok(dt)) return fail(OPTIMUS_ERR_UNSUPPORTED, "%s: unknown dtype %d", what, (int)dt);
  if (use_scaling != 0 && use_scaling != 1)
    return fail(OPTIMUS_ERR_INVALID_ARG, "%s: use_scaling = %d (0 or 1)", what, (int)use_scaling);
  if (G == 0) return OPTIMUS_OK;
  if (!d) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: descriptor array is NULL", what);
  const size_t s = dtype_size(dt);
  std::vector<Region> regs;
  regs.reserve((size_t)G * 3);
  for (int g = 0; g < G; ++g) {
    const optimus_fp8_quant_desc& m = d[g];
    optimus_status st = validate_fp8_member(what, g, m.x, m.ldx, s, m.q, m.ldq, 1, m.rows, m.cols);
    if (st != OPTIMUS_OK) return st;
    if (use_scaling && !m.scale) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d needs a scale pointer", what, g);
    regs.push_back(region(m.x, m.ldx, m.rows, m.cols, s, g, false));
    regs.push_back(region(m.q, m.ldq, m.rows, m.cols, 1, g, true));
    if (use_scaling) regs.push_back(region(m.scale, 1, 1, 1, sizeof(float), g, true));
  }
  return check_aliasing(regs, false, what);
}

extern "C" optimus_status optimus_validate_dequantize_fp8(const optimus_fp8_dequant_desc* d, int32_t G,
                                                          optimus_dtype dt) {
  const char* what = "grouped_dequantize_fp8";
  if (G < 0) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: G = %d < 0", what, G);
  if (!dtype_ok(dt)) return fail(OPTIMUS_ERR_UNSUPPORTED, "%s: unknown dtype %d", what, (int)dt);
  if (G == 0) return OPTIMUS_OK;
  if (!d) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: descriptor array is NULL", what);
  const size_t s = dtype_size(dt);
  std::vector<Region> regs;
  regs.reserve((size_t)G * 3);
  for (int g = 0; g < G; ++g) {
    const optimus_fp8_dequant_desc& m = d[g];
    optimus_status st = validate_fp8_member(what, g, m.q, m.ldq, 1, m.y, m.ldy, s, m.rows, m.cols);
    if (st != OPTIMUS_OK) return st;
    regs.push_back(region(m.q, m.ldq, m.rows, m.cols, 1, g, false));
    if (m.scale) regs.push_back(region(m.scale, 1, 1, 1, sizeof(float), g, false));
    regs.push_back(region(m.y, m.ldy, m.rows, m.cols, s, g, true));
  }
  return check_aliasing(regs, false, what);
}

// ===================================================================== plan options
// The planner's choices a caller may pin (tests, tuning): the GEMM tile
// variant (-1: the planner's), dW's split count (0: the planner's) and the
// fused split-op-cat kernel's waves per row (0: the planner's).
struct PlanOpts {
  int pin = -1;
  int splits = 0;
  int wpr = 0;
};

static optimus_status parse_options(const optimus_plan_options* o, PlanOpts& po) {
  po = PlanOpts{};
  if (!o) return OPTIMUS_OK;
  if (o->reserved != 0) return fail(OPTIMUS_ERR_INVALID_ARG, "plan options: reserved must be 0");
  if (o->gemm_tile < OPTIMUS_TILE_AUTO || o->gemm_tile > OPTIMUS_TILE_F32_16X128)
    return fail(OPTIMUS_ERR_INVALID_ARG, "plan options: unknown gemm_tile %d", (int)o->gemm_tile);
  if (o->wgrad_splits < 0 || o->wgrad_splits > 16)
    return fail(OPTIMUS_ERR_INVALID_ARG, "plan options: wgrad_splits %d outside 0..16", (int)o->wgrad_splits);
  const int w = o->soc_waves_per_row;
  if (w != 0 && w != 1 && w != 2 && w != 4)
    return fail(OPTIMUS_ERR_INVALID_ARG, "plan options: soc_waves_per_row %d is not 0, 1, 2 or 4", w);
  po.pin = o->gemm_tile - 1;  // OPTIMUS_TILE_* = kernel-table index + 1
  po.splits = o->wgrad_splits;
  po.wpr = w;
  return OPTIMUS_OK;
}

static optimus_status tile_unsupported(const PlanOpts& po, const char* what) {
  return fail(OPTIMUS_ERR_UNSUPPORTED, "%s: gemm_tile %d cannot run every member of this group", what, po.pin + 1);
}

// ===================================================================== host plans
// A HostPlan is everything a launch needs, built on the host: a byte blob that
// becomes the device table, offsets into it, and launch parameters.
enum Kind {
  KIND_LINEAR = 0, KIND_LN = 1, KIND_PW = 2, KIND_SOC = 3, KIND_Q8 = 5, KIND_DQ8 = 6, KIND_LINBWD = 7,
  KIND_LNBWD = 8, KIND_ACTBWD = 9
};

struct Blob {
  std::vector<char> bytes;
  size_t add(const void* p, size_t n) {
    size_t off = (bytes.size() + 255) & ~(size_t)255;
    bytes.resize(off + n);
    if (p && n) memcpy(bytes.data() + off, p, n);
    return off;
  }
};

// One kernel launch over a row-wise table (grouped or one member of a chain).
struct RowLaunch {
  size_t descs_off, tiles_off;
  int32_t first_tile, num_tiles, grid;
};

// One grouped GEMM launch: tile shape, operand layout (tr: 0 forward, 2 / 3
// the backward GEMMs), member table, tile list, grid, and per member of the
// plan's group its tile range for a CHAIN launch (empty if it has none here).
struct GemmSet {
  GemmConfig cfg{};
  int tr = 0;
  optimus_act act = OPTIMUS_ACT_NONE;  // the instance's epilogue activation (TR = 2: its backward)
  size_t descs_off = 0, tiles_off = 0;
  int32_t num_tiles = 0, grid = 0;
  int64_t real_tiles = 0;
  std::vector<RowLaunch> chain;
};

struct HostPlan {
  Kind kind;
  optimus_dtype dt;
  optimus_act act;
  int32_t G = 0;
  Blob blob;
  // GEMM
  GemmSet gs[2];       // forward: gs[0]; backward: dX in gs[0], dW (+ db) in gs[1]
  int n_gs = 0;
  bool g_ln = false;  // the row LayerNorm is fused into the GEMM epilogue
  // row-wise (LN / PW, or the split-op-cat fallbacks)
  int row_kernel = KIND_LN;  // which row kernel the grouped launch uses
  optimus_act row_act = OPTIMUS_ACT_NONE;
  RowLaunch rows{};
  std::vector<RowLaunch> rows_chain;
  // fused split-op-cat
  bool soc_fused = false;
  size_t soc_off = 0;
  int32_t soc_rows = 0, soc_nchunks = 0, soc_pieces = 0, soc_grid = 0, soc_wpr = 1;
  // split-op-cat unfused programs (CHAIN / HORIZONTAL) over plan-owned temporaries
  bool soc_has_unfused = false;
  bool soc_apply_ln = false;
  int64_t soc_temp_elems = 0;
  size_t soc_ln_descs = 0, soc_act_descs = 0, soc_cat_descs = 0, soc_tiles = 0;
  std::vector<int32_t> soc_piece_first, soc_piece_count;  // per piece: tile range in soc_tiles
  int32_t soc_piece_tiles_total = 0;
  std::vector<size_t> soc_temp_fixups;  // blob offsets of DevRows pointers relative to the temp base
  // pointer fields of the blob that hold a blob offset, rebased to the device table
  std::vector<size_t> table_fixups;
  // plan-owned device scratch (split-reduction partials), not part of the
  // uploaded table: pointer fields holding an offset into it
  size_t scratch_bytes = 0;
  std::vector<size_t> scratch_fixups;
  RowLaunch red{};                  // split reduction of the dW set
  std::vector<RowLaunch> red_chain;
  RowLaunch tp{};                   // transpose of W before the dX set
  std::vector<RowLaunch> tp_chain;
  // row-wise backward: the main launch (rows / rows_chain) and the dgamma /
  // dbeta finalize of a LayerNorm backward
  RowLaunch fin{};
  std::vector<RowLaunch> fin_chain;
  // fp8 codec: member table, item lists (grouped launches, then per member
  // the items of its CHAIN launches), and for scaled quantize the amax slots
  bool q_scaled = false;
  size_t q_descs_off = 0, q_items_off = 0, q_slots_off = 0;
  RowLaunch q_grouped{}, q_amax{};                    // q_amax: scaled quantize only
  std::vector<RowLaunch> q_chain, q_chain_amax;
  // measurement
  int32_t launches = 1, chain_launches = 0, grid = 0, block = 0;
  int64_t work_items = 0;
  double flops = 0, bytes = 0;
  std::string kernel;
};

static int pow2ceil(int v) {
  int p = 1;
  while (p < v) p <<= 1;
  return p;
}

// Row-wise member: lanes per row and the 16-byte path.
static DevRows make_rows(const void* x, int64_t ldx, void* y, int64_t ldy, const void* gamma, const void* beta,
                         int64_t rows, int64_t cols, float eps, optimus_dtype dt, bool layernorm) {
  const int VEC = dt == OPTIMUS_F32 ? 4 : 8;
  DevRows r{};
  r.x = x; r.y = y; r.gamma = gamma; r.beta = beta;
  r.ldx = ldx; r.ldy = ldy;
  r.rows = (int32_t)rows; r.cols = (int32_t)cols;
  r.eps = eps;
  r.inv_cols = (float)(1.0 / (double)cols);
  const bool vec = cols % VEC == 0 && ldx % VEC == 0 && ldy % VEC == 0 && aligned16(x) && aligned16(y) &&
                   (!gamma || aligned16(gamma)) && (!beta || aligned16(beta));
  const int cpr = (int)(cols / VEC);
  r.vec = 0;
  r.lanes = 0;
  if (vec) {
    if (layernorm) {
      const int maxc = kLnChunksPerLane;  // chunks per lane held in registers by the LayerNorm kernel
      if (cpr <= 64 * maxc) {
        r.vec = 1;
        r.lanes = pow2ceil((cpr + maxc - 1) / maxc);
      }
    } else {
      r.vec = 1;
      r.lanes = std::min(64, pow2ceil(cpr));
    }
  }
  return r;
}

// Row tiles of one member: about kRowTileBytes of input per tile, a whole
// number of the block's row slots.
static constexpr int64_t kRowTileBytes = 32768;
static void add_row_tiles(std::vector<RowTile>& tiles, int member, const DevRows& r, size_t s) {
  const int rpb = r.vec ? 4 * (64 / r.lanes) : 4;
  const int64_t row_bytes = std::max<int64_t>(1, (int64_t)r.cols * (int64_t)s);
  int64_t per = std::max<int64_t>(1, kRowTileBytes / row_bytes);
  per = std::max<int64_t>(rpb, (per / rpb) * rpb);
  for (int64_t r0 = 0; r0 < r.rows; r0 += per)
    tiles.push_back(RowTile{member, (int32_t)r0, (int32_t)std::min<int64_t>(per, r.rows - r0), 0});
}

// Row-wise grids: one workgroup per tile. The hardware dispatcher refills a
// CU as soon as one of its workgroups ends, so short-lived workgroups keep
// every CU streaming to the end of the launch; a persistent grid of the
// resident workgroups, each walking its share of tiles, left the CUs that
// finished early idle (large_group's LayerNorm + tanh: 229 us persistent,
// 237 us with more workgroups than fit, 209 us with one per 32 KB tile; the
// fp8 codec's dequantize 171 -> 163 us).
static int32_t row_grid(int64_t tiles) {
  return (int32_t)std::max<int64_t>(1, std::min<int64_t>(tiles, (int64_t)1 << 30));
}

// Balanced row segments for a grouped row launch of `resident` workgroups:
// every workgroup gets one contiguous, equal share of all members' row bytes
// (rows[g] rows of row_bytes[g] each, members in order), cut at member
// boundaries into segments (pad = the segment's index within its member,
// nseg[g] of them). Segment r of workgroup b sits at index r * B + b (the
// kernels walk t = b, b + B, ...), padded with member -1; shares below 64 KB
// take fewer workgroups. Returns B, the launch's grid.
static int64_t balanced_row_segments(const std::vector<int64_t>& rows, const std::vector<double>& row_bytes,
                                     int64_t resident, std::vector<RowTile>& tiles, std::vector<int>& nseg) {
  const size_t G = rows.size();
  double total = 0.0;
  for (size_t g = 0; g < G; ++g) total += (double)rows[g] * row_bytes[g];
  constexpr double kMinSegmentBytes = 64.0 * 1024.0;
  const int64_t B = std::max<int64_t>(1, std::min<int64_t>(resident, (int64_t)(total / kMinSegmentBytes)));
  std::vector<std::vector<RowTile>> per_block((size_t)B);
  nseg.assign(G, 0);
  double cum = 0.0;
  int64_t blk = 0;
  for (size_t g = 0; g < G; ++g) {
    const double rb = row_bytes[g];
    int64_t r = 0;
    while (r < rows[g]) {
      const double end = total * (double)(blk + 1) / (double)B;
      int64_t k = rows[g] - r;
      if (blk + 1 < B) k = std::min<int64_t>(k, std::max<int64_t>(1, (int64_t)std::ceil((end - cum) / rb)));
      per_block[(size_t)blk].push_back(RowTile{(int)g, (int32_t)r, (int32_t)k, nseg[g]++});
      r += k;
      cum += (double)k * rb;
      while (blk + 1 < B && cum >= total * (double)(blk + 1) / (double)B) ++blk;
    }
  }
  size_t rounds = 0;
  for (const auto& v : per_block) rounds = std::max(rounds, v.size());
  tiles.assign(rounds * (size_t)B, RowTile{-1, 0, 0, 0});
  for (int64_t bb = 0; bb < B; ++bb)
    for (size_t r = 0; r < per_block[(size_t)bb].size(); ++r) tiles[r * (size_t)B + (size_t)bb] = per_block[(size_t)bb][r];
  return B;
}

// Row-wise plan over `members` (LayerNorm or pointwise), member-major tiles
// of about kRowTileBytes. (Balanced per-workgroup segments, as the LayerNorm
// backward uses, measured slower here: 268 against 253 us for large_group's
// LayerNorm + tanh. The hardware spreads the small tiles better.)
static void build_rows(HostPlan& hp, const std::vector<DevRows>& members, bool layernorm, size_t s,
                       optimus_act act) {
  std::vector<RowTile> tiles;
  hp.rows_chain.clear();
  for (size_t g = 0; g < members.size(); ++g) {
    const int first = (int)tiles.size();
    add_row_tiles(tiles, (int)g, members[g], s);
    hp.rows_chain.push_back(RowLaunch{0, 0, first, (int)tiles.size() - first, 0});
  }
  const size_t doff = hp.blob.add(members.data(), members.size() * sizeof(DevRows));
  const size_t toff = hp.blob.add(tiles.data(), tiles.size() * sizeof(RowTile));
  for (auto& c : hp.rows_chain) {
    c.descs_off = doff;
    c.tiles_off = toff;
    c.grid = row_grid(c.num_tiles);
  }
  hp.rows = RowLaunch{doff, toff, 0, (int32_t)tiles.size(), row_grid((int64_t)tiles.size())};
  hp.row_kernel = layernorm ? KIND_LN : KIND_PW;
  hp.work_items = (int64_t)tiles.size();
  hp.grid = hp.rows.grid;
  hp.block = kRowThreads;
  hp.chain_launches = (int32_t)members.size();
}

// Tile list of one grouped GEMM over `descs` (ids[i]: the plan-group member
// descs[i] belongs to): heavy members first (tile cost grows with K),
// member-major, M-blocks then N-blocks, padded to a multiple of 8; the
// persistent grid is no larger than what is resident at once (a workgroup
// that had to wait for a free slot would start its whole share late).
// Forward members that read one input (the same x, ldx, M and K: Table 1's
// batch_linear_lhs) are walked M-block by M-block across all of them, so the
// tiles that read one x panel sit side by side in the list (the kernel deals
// contiguous slices of it to each L2); the per-member CHAIN launches then
// read a member-major copy of the list.
static void build_gemm_set(HostPlan& hp, GemmSet& gs, const GemmConfig& cfg, int tr, const std::vector<DevLinear>& descs,
                           const std::vector<int>& ids, int group_size, optimus_act act, bool ln, int splits = 1) {
  const int n = (int)descs.size();
  gs.cfg = cfg;
  gs.tr = tr;
  gs.act = act;
  std::vector<int> order(n);
  for (int i = 0; i < n; ++i) order[i] = i;
  // the streaming kernel's item cost is its rows' bytes, x row plus y row
  // (K + N values); the tiled kernels' tile cost grows with K
  if (cfg.variant == 9)
    std::stable_sort(order.begin(), order.end(),
                     [&](int a, int b) { return descs[a].K + descs[a].N > descs[b].K + descs[b].N; });
  else
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return descs[a].K > descs[b].K; });
  const int bm = cfg.bm, bn = cfg.bn;
  auto member_tiles = [&](std::vector<GemmTile>& tl, int i, int64_t mb) {
    const int64_t nbs = (descs[i].N + bn - 1) / bn;
    // split index fastest: measured on the weight gradient, this beats the
    // split-major order (all tiles of one reduction range side by side on
    // one L2) by 3.5 % despite 16 % more HBM reads
    for (int64_t nb = 0; nb < nbs; ++nb)
      for (int ks = 0; ks < splits; ++ks) tl.push_back(GemmTile{i, (int32_t)mb, (int32_t)nb, ks});
  };
  // member-major list (and the CHAIN ranges)
  std::vector<GemmTile> chain_tiles;
  gs.chain.assign(group_size, RowLaunch{});
  for (int i : order) {
    const int first = (int)chain_tiles.size();
    for (int64_t mb = 0; mb < (descs[i].M + bm - 1) / bm; ++mb) member_tiles(chain_tiles, i, mb);
    gs.chain[ids[i]].first_tile = first;
    gs.chain[ids[i]].num_tiles = (int)chain_tiles.size() - first;
  }
  // grouped list: a run of consecutive members (in `order`) that share x is
  // walked in groups of kSharedMBlocks M-blocks: for each group, every
  // member's N-blocks in turn, each over the group's M-blocks. Consecutive
  // items then share a weight block, and a group's x rows serve every member
  // while they are in L2 (walking all members' N-blocks per M-block instead
  // kept x resident but fetched each weight block once per M-block).
  constexpr int64_t kSharedMBlocks = 8;
  std::vector<GemmTile> tiles;
  bool shared = false;
  for (int a = 0; a < n;) {
    int b = a + 1;
    const DevLinear& da = descs[order[a]];
    while (tr == 0 && b < n) {
      const DevLinear& db = descs[order[b]];
      if (db.x != da.x || db.ldx != da.ldx || db.M != da.M || db.K != da.K) break;
      ++b;
    }
    const int64_t mbs = (da.M + bm - 1) / bm;
    if (b - a == 1) {
      for (int64_t mb = 0; mb < mbs; ++mb) member_tiles(tiles, order[a], mb);
    } else {
      shared = true;
      for (int64_t g0 = 0; g0 < mbs; g0 += kSharedMBlocks)
        for (int r = a; r < b; ++r) {
          const int i = order[r];
          for (int64_t nb = 0; nb < (descs[i].N + bn - 1) / bn; ++nb)
            for (int64_t mb = g0; mb < std::min(mbs, g0 + kSharedMBlocks); ++mb)
              tiles.push_back(GemmTile{i, (int32_t)mb, (int32_t)nb, 0});
        }
    }
    a = b;
  }
  gs.real_tiles = (int64_t)tiles.size();
  const int64_t cap = (int64_t)device_cu_count() * gemm_resident_per_cu(cfg, hp.dt, act, ln, tr);
  // The kernels hand XCD x (the hardware deals workgroups round-robin to the
  // 8 XCDs) the items at positions r * grid + x * grid / 8 + [0, grid / 8) of
  // round r. Over more than one round, each XCD gets one contiguous eighth of
  // the list instead of a slice of every round, so the items that share a
  // weight block (a member's M-blocks) or an x panel stay on one L2, and the
  // last round's items spread over all XCDs; empty positions are padding.
  // Only for members of one K: with K unequal the heavy-first list relies on
  // every round mixing all XCDs (dealt, one XCD would take all the long items).
  bool reordered = false;  // the grouped list is no longer member-major
  {
    const int64_t T = (int64_t)tiles.size();
    int64_t g = std::min<int64_t>((T + 7) / 8 * 8, cap);
    if (g >= 8) g -= g % 8;
    bool one_k = true;
    for (const DevLinear& dd : descs) one_k = one_k && dd.K == descs[0].K;
    // (the tiled kernels; the skinny kernel walks items in plain order, the streaming kernel below)
    if (tr == 0 && one_k && g >= 8 && T > g && cfg.variant != 7 && cfg.variant != 9) {
      const int64_t per = g / 8, chunk = (T + 7) / 8, rounds = (chunk + per - 1) / per;
      std::vector<GemmTile> dealt_tiles((size_t)(rounds * g), GemmTile{-1, 0, 0, 0});
      for (int64_t x = 0; x < 8; ++x)
        for (int64_t j = 0; j < chunk && x * chunk + j < T; ++j)
          dealt_tiles[(size_t)((j / per) * g + x * per + j % per)] = tiles[(size_t)(x * chunk + j)];
      tiles.swap(dealt_tiles);
      reordered = true;
    }
    // Streaming items, costliest first, run as one round of resident
    // workgroups dispatched across the CUs in list order, so the workgroups
    // that share a CU sit about a device-width apart in the list. Every other
    // device-width is reversed: a CU that takes one of the costliest items of
    // one stretch takes one of the cheapest of the next (launch_bound:
    // 22.1 -> 21.6 us; sorting alone gave 21.5 against 22.1 on another box).
    if (cfg.variant == 9 && T > device_cu_count()) {
      const int64_t C = device_cu_count();
      for (int64_t s0 = C; s0 < T; s0 += 2 * C) std::reverse(tiles.begin() + s0, tiles.begin() + std::min(T, s0 + C));
      reordered = true;
    }
  }
  while (tiles.size() % 8) tiles.push_back(GemmTile{-1, 0, 0, 0});
  gs.descs_off = hp.blob.add(descs.data(), descs.size() * sizeof(DevLinear));
  gs.tiles_off = hp.blob.add(tiles.data(), tiles.size() * sizeof(GemmTile));
  gs.num_tiles = (int32_t)tiles.size();
  // the CHAIN launches walk each member's tiles in member order: their own list unless it equals the grouped one
  const size_t chain_off =
      shared || reordered ? hp.blob.add(chain_tiles.data(), chain_tiles.size() * sizeof(GemmTile)) : gs.tiles_off;
  int64_t grid = std::min<int64_t>((int64_t)tiles.size(), cap);
  if (grid >= 8) grid -= grid % 8;
  gs.grid = (int32_t)std::max<int64_t>(1, grid);
  for (auto& c : gs.chain) {
    c.descs_off = gs.descs_off;
    c.tiles_off = chain_off;
    c.grid = (int32_t)std::max<int64_t>(1, std::min<int64_t>(c.num_tiles, cap));
  }
}

static optimus_status build_linear(const optimus_linear_desc* d, int32_t G, optimus_dtype dt, optimus_act act,
                                   HostPlan& hp, bool ln = false, const void* const* gamma = nullptr,
                                   const void* const* beta = nullptr, float eps = 0.f, const PlanOpts& po = PlanOpts{}) {
  optimus_status st = validate_linear_impl(d, G, dt, act, ln, gamma, beta, eps);
  if (st != OPTIMUS_OK) return st;
  hp.kind = KIND_LINEAR; hp.dt = dt; hp.act = act; hp.G = G; hp.g_ln = ln;
  const size_t s = dtype_size(dt);
  const int VEC = dt == OPTIMUS_F32 ? 4 : 8;
  std::vector<DevLinear> descs(G);
  for (int g = 0; g < G; ++g) {
    const optimus_linear_desc& m = d[g];
    DevLinear& o = descs[g];
    o.x = m.x; o.w = m.w; o.bias = m.bias; o.y = m.y;
    o.ldx = m.ldx; o.ldw = m.ldw; o.ldy = m.ldy;
    o.M = (int32_t)m.M; o.N = (int32_t)m.N; o.K = (int32_t)m.K;
    const bool vin = m.K % VEC == 0 && m.ldx % VEC == 0 && m.ldw % VEC == 0 && aligned16(m.x) && aligned16(m.w);
    const bool vout = m.ldy % VEC == 0 && aligned16(m.y);
    o.vec = (vin ? 1 : 0) | (vout ? 2 : 0);
    o.gamma = ln && gamma ? gamma[g] : nullptr;
    o.beta = ln && beta ? beta[g] : nullptr;
    o.eps = eps;
    o.inv_n = 1.0f / (float)m.N;
    hp.flops += 2.0 * (double)m.M * (double)m.N * (double)m.K;
    // an input shared with an earlier member is read once
    bool seen = false;
    for (int e = 0; e < g && !seen; ++e)
      seen = d[e].x == m.x && d[e].ldx == m.ldx && d[e].M == m.M && d[e].K == m.K;
    hp.bytes += (double)s * ((seen ? 0.0 : (double)m.M * m.K) + (double)m.N * m.K + (m.bias ? (double)m.N : 0.0) +
                             (double)m.M * m.N);
    if (ln) hp.bytes += (double)s * ((o.gamma ? (double)m.N : 0.0) + (o.beta ? (double)m.N : 0.0));
  }
  std::vector<int> ids(G);
  for (int g = 0; g < G; ++g) ids[g] = g;
  const GemmConfig cfg = gemm_pick_config(dt, d, G, ln, G > 0 ? po.pin : -1);
  if (cfg.variant < 0) return tile_unsupported(po, ln ? "plan_linear_layernorm" : "plan_linear");
  build_gemm_set(hp, hp.gs[0], cfg, 0, descs, ids, G, act, ln);
  hp.n_gs = 1;
  hp.work_items = hp.gs[0].real_tiles;
  hp.grid = hp.gs[0].grid;
  hp.block = hp.gs[0].cfg.threads;
  hp.chain_launches = G;
  hp.kernel = std::string(hp.gs[0].cfg.name) + (ln ? "_layernorm" : "");
  return OPTIMUS_OK;
}

// Linear backward as two grouped GEMMs in the forward kernel's terms
// (y[m][n] = sum_k x[m][k] w[n][k]):
//   dX: x = dY (as stored), w[n'][k'] = W[k'][n'] (reduction-major), y = dX,
//       M' = M, N' = K, K' = N
//   dW: x[m'][k'] = dY[k'][m'] and w[n'][k'] = X[k'][n'] (both
//       reduction-major), y = dW, M' = N, N' = K, K' = M; the row sums of x
//       over k' are db.
static DevRowsGrad make_rows_grad(const void* x, int64_t ldx, const void* dy, int64_t lddy, void* dx, int64_t lddx,
                                  const void* gamma, int64_t rows, int64_t cols, float eps, optimus_dtype dt,
                                  bool layernorm);
static std::vector<RowTile> grad_row_tiles(HostPlan& hp, const std::vector<DevRowsGrad>& members, size_t s,
                                           std::vector<int>& ntiles, int64_t max_tiles);

// act != NONE: dX leaves with the activation backward of the layer below
// applied, dX * act'(act_x[g]) (act_x [M][K], row stride ld_act_x[g]).
static optimus_status build_linear_backward(const optimus_linear_grad_desc* d, int32_t G, optimus_dtype dt,
                                            HostPlan& hp, optimus_act act = OPTIMUS_ACT_NONE,
                                            const void* const* act_x = nullptr, const int64_t* ld_act_x = nullptr,
                                            const PlanOpts& po = PlanOpts{}) {
  optimus_status st = optimus_validate_linear_backward(d, G, dt);
  if (st != OPTIMUS_OK) return st;
  const char* what = "grouped_linear_act_backward";
  if (!act_ok(act)) return fail(OPTIMUS_ERR_UNSUPPORTED, "%s: unknown activation %d", what, (int)act);
  if (act != OPTIMUS_ACT_NONE) {
    if (!act_x || !ld_act_x) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: act_x or ld_act_x is NULL", what);
    for (int g = 0; g < G; ++g) {
      if (!d[g].dx) continue;
      if (!act_x[g] && d[g].M > 0 && d[g].K > 0)
        return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d: act_x is NULL", what, g);
      if (ld_act_x[g] < d[g].K) return fail(OPTIMUS_ERR_INVALID_ARG, "%s: member %d: ld_act_x < K", what, g);
    }
    // act_x is read while dX, dW and db are written: it may be a member's dX
    // itself (each value is read before it is written), no other output
    std::vector<Region> regs;
    const size_t es = dtype_size(dt);
    for (int g = 0; g < G; ++g) {
      if (!d[g].dx || d[g].M <= 0 || d[g].K <= 0) continue;
      regs.push_back(region(act_x[g], ld_act_x[g], d[g].M, d[g].K, es, g, false));
      regs.push_back(region(d[g].dx, d[g].lddx, d[g].M, d[g].K, es, g, true));
      if (d[g].dw) regs.push_back(region(d[g].dw, d[g].lddw, d[g].N, d[g].K, es, g, true));
      if (d[g].db) regs.push_back(region(d[g].db, d[g].N, 1, d[g].N, es, g, true));
    }
    st = check_aliasing(regs, true, what);
    if (st != OPTIMUS_OK) return st;
  }
  hp.kind = KIND_LINBWD; hp.dt = dt; hp.act = act; hp.G = G;
  const size_t s = dtype_size(dt);
  const int VEC = dt == OPTIMUS_F32 ? 4 : 8;
  std::vector<DevLinear> dxs, dws;
  std::vector<int> dx_ids, dw_ids;
  std::vector<optimus_linear_desc> dx_shape, dw_shape;  // (M', N', K') for the tile picker
  std::vector<TransposeItem> tps;  // W -> W^T tiles, member by member
  std::vector<int> tp_end;  // per dX member: end of its transpose tiles
  // dX straight from W (no transpose, no scratch copy) when every dX member
  // allows the direct-to-LDS tiles to read W as it lies, reduction-major
  bool direct = false;
  GemmConfig dx_cfg{};
  if (dt == OPTIMUS_BF16) {
    std::vector<optimus_linear_desc> sh;
    for (int g = 0; g < G; ++g)
      if (d[g].dx) {
        optimus_linear_desc e{};
        e.M = d[g].M; e.N = d[g].K; e.K = d[g].N;
        e.x = d[g].dy; e.ldx = d[g].lddy; e.w = d[g].w; e.ldw = d[g].ldw;
        sh.push_back(e);
      }
    if (!sh.empty() && gemm_dma_wt_ok(sh.data(), (int32_t)sh.size())) {
      dx_cfg = gemm_pick_config(dt, sh.data(), (int32_t)sh.size(), false, po.pin);
      direct = dx_cfg.variant == 4 || dx_cfg.variant == 5;
    }
  }
  // without the direct tiles and with an activation backward, dY W goes to
  // plan scratch (offset, row stride per member) and the activation backward
  // reads it beside act_x and writes dx: act_x may then be dx itself
  std::vector<int64_t> g_off(G, -1), g_ld(G, 0);
  for (int g = 0; g < G; ++g) {
    const optimus_linear_grad_desc& m = d[g];
    if (m.dx && direct) {
      DevLinear o{};
      o.x = m.dy; o.ldx = m.lddy; o.w = m.w; o.ldw = m.ldw; o.y = m.dx; o.ldy = m.lddx;
      o.M = (int32_t)m.M; o.N = (int32_t)m.K; o.K = (int32_t)m.N;
      const bool vout = m.lddx % VEC == 0 && aligned16(m.dx);
      o.vec = 1 | 4 | (vout ? 2 : 0);
      if (act != OPTIMUS_ACT_NONE) {  // fused into the epilogue
        o.ax = act_x[g];
        o.ldax = ld_act_x[g];
        o.vec |= (o.ldax % VEC == 0 && aligned16(o.ax)) ? 8 : 0;
      }
      o.inv_n = 1.0f / (float)m.K;
      dxs.push_back(o);
      dx_ids.push_back(g);
      hp.flops += 2.0 * (double)m.M * (double)m.N * (double)m.K;
      // dY, W and dX, plus the activation input the fused epilogue reads
      hp.bytes += (double)s * ((double)m.M * m.N + (double)m.N * m.K + (double)m.M * m.K *
                               (act != OPTIMUS_ACT_NONE ? 2.0 : 1.0));
    } else if (m.dx) {
      // dX = dY . W as a forward GEMM on W^T [K][N'] (N' = N rounded up to 8
      // values), transposed into plan scratch by the first launch
      DevLinear o{};
      const int64_t ldt = (m.N + 7) / 8 * 8;
      const size_t off = (hp.scratch_bytes + 255) & ~(size_t)255;
      hp.scratch_bytes = off + (size_t)(m.K * ldt) * s;
      o.x = m.dy; o.ldx = m.lddy; o.w = (const void*)(uintptr_t)off; o.ldw = ldt; o.y = m.dx; o.ldy = m.lddx;
      o.M = (int32_t)m.M; o.N = (int32_t)m.K; o.K = (int32_t)m.N;
      if (act != OPTIMUS_ACT_NONE) {
        g_ld[g] = (m.K + VEC - 1) / VEC * VEC;
        g_off[g] = (int64_t)((hp.scratch_bytes + 255) & ~(size_t)255);
        hp.scratch_bytes = (size_t)g_off[g] + (size_t)(m.M * g_ld[g]) * s;
        o.y = (void*)(uintptr_t)g_off[g];
        o.ldy = g_ld[g];
      }
      const bool vin = m.N % VEC == 0 && m.lddy % VEC == 0 && aligned16(m.dy);
      const bool vout = o.ldy % VEC == 0 && aligned16(o.y);
      o.vec = (vin ? 1 : 0) | (vout ? 2 : 0);
      for (int64_t r0 = 0; r0 < m.N; r0 += 64)
        for (int64_t c0 = 0; c0 < m.K; c0 += 64)
          tps.push_back(TransposeItem{m.w, (void*)(uintptr_t)off, m.ldw, ldt, (int32_t)m.N, (int32_t)m.K,
                                      (int32_t)r0, (int32_t)c0});
      tp_end.push_back((int)tps.size());
      o.inv_n = 1.0f / (float)m.K;
      dxs.push_back(o);
      dx_ids.push_back(g);
      optimus_linear_desc sh{};
      sh.M = m.M; sh.N = m.K; sh.K = m.N;
      sh.x = m.dy; sh.ldx = m.lddy; sh.w = (const void*)(uintptr_t)256; sh.ldw = ldt;  // W^T: 256-byte aligned
      dx_shape.push_back(sh);
      hp.flops += 2.0 * (double)m.M * (double)m.N * (double)m.K;
      // dY, W and dX; with an activation backward the GEMM writes dY W to
      // scratch and the activation backward reads it and a, and writes dX
      hp.bytes += (double)s * ((double)m.M * m.N + (double)m.N * m.K + (double)m.M * m.K *
                               (act != OPTIMUS_ACT_NONE ? 4.0 : 1.0));
    }
    if (m.dw) {
      DevLinear o{};
      o.x = m.dy; o.ldx = m.lddy; o.w = m.x; o.ldw = m.ldx; o.y = m.dw; o.ldy = m.lddw; o.xsum = m.db;
      o.M = (int32_t)m.N; o.N = (int32_t)m.K; o.K = (int32_t)m.M;
      const bool vx = m.lddy % VEC == 0 && aligned16(m.dy);
      const bool vout = m.lddw % VEC == 0 && aligned16(m.dw);
      const bool vw = m.ldx % VEC == 0 && aligned16(m.x);
      o.vec = (vx ? 1 : 0) | (vout ? 2 : 0) | (vw ? 4 : 0);
      o.inv_n = 1.0f / (float)m.K;
      dws.push_back(o);
      dw_ids.push_back(g);
      optimus_linear_desc sh{};
      sh.M = m.N; sh.N = m.K; sh.K = m.M;
      sh.x = m.dy; sh.ldx = m.lddy; sh.w = m.x; sh.ldw = m.ldx;  // both reduction-major
      dw_shape.push_back(sh);
      hp.flops += 2.0 * (double)m.M * (double)m.N * (double)m.K;
      hp.bytes += (double)s * ((double)m.M * m.N + (double)m.M * m.K + (double)m.N * m.K + (m.db ? (double)m.N : 0.0));
    }
  }
  hp.n_gs = 0;
  hp.work_items = 0;
  hp.chain_launches = 0;
  std::string name;
  hp.tp_chain.assign(G, RowLaunch{});
  static const char* const act_names[] = {"", "_relu", "_sigmoid", "_tanh", "_silu"};
  if (!dxs.empty() && direct) {
    GemmSet& gs = hp.gs[hp.n_gs++];
    build_gemm_set(hp, gs, dx_cfg, 2, dxs, dx_ids, G, act, false);
    name = std::string(gs.cfg.name) + "_dgrad_direct" + act_names[(int)act];
  } else if (!dxs.empty()) {
    // the transposes of W, then dX on the forward kernels (direct-to-LDS when
    // dY rows and N are 16-byte multiples)
    const size_t toff = hp.blob.add(tps.data(), tps.size() * sizeof(TransposeItem));
    for (size_t i = 0; i < tps.size(); ++i)
      hp.scratch_fixups.push_back(toff + i * sizeof(TransposeItem) + offsetof(TransposeItem, dst));
    const int32_t cap = device_cu_count() * 4;
    hp.tp = RowLaunch{toff, toff, 0, (int32_t)tps.size(), std::max(1, std::min((int32_t)tps.size(), cap))};
    int prev = 0;
    for (size_t i = 0; i < dx_ids.size(); ++i) {
      hp.tp_chain[dx_ids[i]] = RowLaunch{toff, toff, prev, tp_end[i] - prev, std::max(1, std::min(tp_end[i] - prev, cap))};
      prev = tp_end[i];
    }
    const GemmConfig fcfg = gemm_pick_config(dt, dx_shape.data(), (int32_t)dx_shape.size(), false, po.pin);
    if (fcfg.variant < 0) return tile_unsupported(po, "plan_linear_backward (dX)");
    GemmSet& gs = hp.gs[hp.n_gs++];
    build_gemm_set(hp, gs, fcfg, 0, dxs, dx_ids, G, OPTIMUS_ACT_NONE, false);
    for (size_t i = 0; i < dxs.size(); ++i) {
      hp.scratch_fixups.push_back(gs.descs_off + i * sizeof(DevLinear) + offsetof(DevLinear, w));
      if (g_off[dx_ids[i]] >= 0) hp.scratch_fixups.push_back(gs.descs_off + i * sizeof(DevLinear) + offsetof(DevLinear, y));
    }
    name = std::string(gs.cfg.name) + "_dgrad" + act_names[(int)act];
    if (act != OPTIMUS_ACT_NONE) {
      // no fused epilogue on these tiles: one grouped activation-backward
      // launch, x = act_x, dy = dY W in scratch, dx (members without dX get
      // no rows)
      std::vector<DevRowsGrad> rm;
      for (int g = 0; g < G; ++g) {
        const bool has = d[g].dx != nullptr;
        rm.push_back(make_rows_grad(has ? act_x[g] : nullptr, has ? ld_act_x[g] : 1,
                                    has ? (const void*)(uintptr_t)g_off[g] : nullptr, has ? g_ld[g] : 1, d[g].dx,
                                    d[g].lddx, nullptr, has ? d[g].M : 0, d[g].K, 0.f, dt, false));
      }
      std::vector<int> nt;
      std::vector<RowTile> rt = grad_row_tiles(hp, rm, s, nt, 0);
      const size_t roff = hp.blob.add(rm.data(), rm.size() * sizeof(DevRowsGrad));
      for (int g = 0; g < G; ++g)
        if (d[g].dx) hp.scratch_fixups.push_back(roff + g * sizeof(DevRowsGrad) + offsetof(DevRowsGrad, dy));
      const size_t rtoff = hp.blob.add(rt.data(), rt.size() * sizeof(RowTile));
      for (auto& c : hp.rows_chain) {
        c.descs_off = roff;
        c.tiles_off = rtoff;
      }
      hp.rows = RowLaunch{roff, rtoff, 0, (int32_t)rt.size(), row_grid((int64_t)rt.size())};
    }
  }
  hp.red_chain.assign(G, RowLaunch{});
  if (!dws.empty()) {
    GemmSet& gs = hp.gs[hp.n_gs++];
    // dW reduces over the batch: few output tiles, a long K. Splitting K into
    // `splits` ranges multiplies the work items (split index fastest, as
    // build_gemm_set lays them out); their fp32 partials cost one write by
    // the GEMM and one read by the reduce launch, 8 bytes per output element
    // and split. The tile edge (bf16: 256 or 128) and the split count are the
    // pair with the least estimated time: the launch's makespan under its
    // static schedule (item i on workgroup i mod grid), each item its K steps
    // of one tile on one workgroup slot plus its output tile's write (fp32
    // when split), then the reduce launch's reads and writes. Rates measured
    // on MI355X: a direct-to-LDS K step at 4.6 TFLOP/s per CU (256x256) and
    // 3.6 (128x128), HBM at 4.7 TB/s shared by the slots. A larger split count
    // must gain 3 %: the estimate is that close to the measured times.
    double out_elems = 0.0;
    for (const auto& o : dws) out_elems += (double)o.M * o.N;
    auto est_of = [&](const GemmConfig& c, int sp) {
      const int bkc = c.variant == 3 ? 32 : 64;
      const int occ = gemm_resident_per_cu(c, dt, OPTIMUS_ACT_NONE, false, 3);
      const int64_t slots = (int64_t)device_cu_count() * occ;
      const double cu_rate = c.variant == 4 ? 4.6e12 : c.variant == 5 ? 3.6e12
                           : (c.variant == 3 || c.variant == 6) ? 0.4e12 : 3.0e12;
      const double t_step = 2.0 * c.bm * c.bn * bkc / (cu_rate / occ);
      const double t_out = (double)c.bm * c.bn * (sp > 1 ? 4.0 : (double)s) / (4.7e12 / (double)slots);
      std::vector<int64_t> steps;  // per work item, in list order
      for (const auto& o : dws) {
        const int64_t kc = ((o.K + sp - 1) / sp + bkc - 1) / bkc * bkc;
        if ((int64_t)(sp - 1) * kc >= o.K) return -1.0;  // an empty split
        const int64_t tiles = ((o.M + c.bm - 1) / c.bm) * ((o.N + c.bn - 1) / c.bn);
        for (int64_t t = 0; t < tiles; ++t)
          for (int k = 0; k < sp; ++k) steps.push_back((std::min<int64_t>(o.K, (k + 1) * kc) - k * kc + bkc - 1) / bkc);
      }
      const int64_t n8 = ((int64_t)steps.size() + 7) / 8 * 8;
      int64_t grid = std::min<int64_t>(n8, slots);
      if (grid >= 8) grid -= grid % 8;
      grid = std::max<int64_t>(grid, 1);
      std::vector<double> load((size_t)grid, 0.0);
      for (size_t i = 0; i < steps.size(); ++i) load[i % grid] += (double)steps[i] * t_step + t_out;
      const double makespan = *std::max_element(load.begin(), load.end());
      // the reduce reads every split's partials and writes the output once
      // (plus about 6 us of launch gap and ramp)
      return makespan + (sp > 1 ? out_elems * (4.0 * sp + (double)s) / 4.7e12 + 6e-6 : 0.0);
    };
    const int n_dw = (int32_t)dw_shape.size();
    GemmConfig cfg = gemm_pick_config_trans(dt, dw_shape.data(), n_dw, true, 0, po.pin);
    if (cfg.variant < 0) return tile_unsupported(po, "plan_linear_backward (dW)");
    int splits = 1;
    {
      std::vector<GemmConfig> cands{cfg};
      if (dt == OPTIMUS_BF16 && po.pin < 0)
        for (int edge : {256, 128}) {
          const GemmConfig c = gemm_pick_config_trans(dt, dw_shape.data(), n_dw, true, edge);
          if (c.variant != cfg.variant) cands.push_back(c);
        }
      double best = -1.0;
      for (const GemmConfig& c : cands) {
        int sp_best = 1;
        double e_best = est_of(c, 1);
        for (int sp = 2; sp <= 16; ++sp) {
          const double e = est_of(c, sp);
          if (e >= 0.0 && e < e_best * 0.97) {
            e_best = e;
            sp_best = sp;
          }
        }
        if (best < 0.0 || e_best < best * 0.99) {
          best = e_best;
          cfg = c;
          splits = sp_best;
        }
      }
    }
    const int bk = cfg.variant == 3 ? 32 : 64;  // every split but the last a whole number of K steps
    // a pinned split count (plan options), where no split comes out empty
    if (po.splits > 0) {
      if (est_of(cfg, po.splits) < 0.0)
        return fail(OPTIMUS_ERR_UNSUPPORTED, "plan_linear_backward: wgrad_splits %d leaves a split empty", po.splits);
      splits = po.splits;
    }
    if (splits > 1) {
      std::vector<SplitReduceItem> red;
      for (size_t i = 0; i < dws.size(); ++i) {
        DevLinear& o = dws[i];
        const int64_t kc = ((o.K + splits - 1) / splits + bk - 1) / bk * bk;
        o.kchunk = (int32_t)kc;
        o.splits = splits;
        const int64_t floats = (int64_t)splits * o.M * o.N + (int64_t)splits * o.M;
        const size_t off = (hp.scratch_bytes + 255) & ~(size_t)255;
        o.ws = (float*)(uintptr_t)off;
        hp.scratch_bytes = off + (size_t)floats * sizeof(float);
        // about 1024 groups of 4 columns per item
        const int rows_per = std::max<int32_t>(1, 4096 / std::max<int32_t>(o.N, 1));
        const int first = (int)red.size();
        for (int32_t r0 = 0; r0 < o.M; r0 += rows_per)
          red.push_back(SplitReduceItem{(const float*)(uintptr_t)off, o.y, o.xsum, o.ldy, o.M, o.N, splits, r0,
                                        std::min<int32_t>(rows_per, o.M - r0), 0});
        hp.red_chain[dw_ids[i]] = RowLaunch{0, 0, first, (int)red.size() - first, 0};
      }
      const size_t roff = hp.blob.add(red.data(), red.size() * sizeof(SplitReduceItem));
      for (size_t i = 0; i < red.size(); ++i)
        hp.scratch_fixups.push_back(roff + i * sizeof(SplitReduceItem) + offsetof(SplitReduceItem, ws));
      const int32_t cap = device_cu_count() * 4;
      hp.red = RowLaunch{roff, roff, 0, (int32_t)red.size(), std::max(1, std::min((int32_t)red.size(), cap))};
      for (auto& c : hp.red_chain) {
        c.descs_off = c.tiles_off = roff;
        c.grid = std::max(1, std::min(c.num_tiles, cap));
      }
    }
    build_gemm_set(hp, gs, cfg, 3, dws, dw_ids, G, OPTIMUS_ACT_NONE, false, splits);
    for (size_t i = 0; i < dws.size() && splits > 1; ++i)
      hp.scratch_fixups.push_back(gs.descs_off + i * sizeof(DevLinear) + offsetof(DevLinear, ws));
    name += std::string(name.empty() ? "" : "+") + gs.cfg.name + "_wgrad" +
            (splits > 1 ? "_split" + std::to_string(splits) : "");
  }
  for (int i = 0; i < hp.n_gs; ++i) {
    hp.work_items += hp.gs[i].real_tiles;
    for (const RowLaunch& c : hp.gs[i].chain) hp.chain_launches += c.num_tiles > 0 ? 1 : 0;
  }
  for (const RowLaunch& c : hp.red_chain) hp.chain_launches += c.num_tiles > 0 ? 1 : 0;
  for (const RowLaunch& c : hp.tp_chain) hp.chain_launches += c.num_tiles > 0 ? 1 : 0;
  for (const RowLaunch& c : hp.rows_chain) hp.chain_launches += c.num_tiles > 0 ? 1 : 0;
  hp.launches = std::max(hp.n_gs, 1) + (hp.red.num_tiles > 0 ? 1 : 0) + (hp.tp.num_tiles > 0 ? 1 : 0) +
                (hp.rows.num_tiles > 0 ? 1 : 0);
  hp.grid = hp.n_gs ? hp.gs[0].grid : 0;
  hp.block = hp.n_gs ? hp.gs[0].cfg.threads : 0;
  hp.kernel = name.empty() ? "grouped_linear_backward_empty" : name;
  return OPTIMUS_OK;
}

// Row-wise backward member: the forward's geometry (lanes per row, the
// 16-byte path when x, dy, dx (and gamma) rows are 16-byte chunks).
static DevRowsGrad make_rows_grad(const void* x, int64_t ldx, const void* dy, int64_t lddy, void* dx, int64_t lddx,
                                  const void* gamma, int64_t rows, int64_t cols, float eps, optimus_dtype dt,
                                  bool layernorm) {
  DevRows geo = make_rows(x, ldx, dx, lddx, gamma, nullptr, rows, cols, eps, dt, layernorm);
  const int VEC = dt == OPTIMUS_F32 ? 4 : 8;
  const bool dy_ok = lddy % VEC == 0 && aligned16(dy);
  DevRowsGrad r{};
  r.x = x; r.dy = dy; r.dx = dx; r.gamma = gamma;
  r.ldx = ldx; r.lddy = lddy; r.lddx = lddx;
  r.rows = (int32_t)rows; r.cols = (int32_t)cols;
  r.vec = geo.vec && dy_ok ? 1 : 0;
  r.lanes = r.vec ? geo.lanes : 0;
  r.eps = eps;
  r.inv_cols = geo.inv_cols;
  return r;
}

// Row tiles of every member (pad = the tile's index within its member), the
// grouped launch and the per-member CHAIN ranges. With `max_tiles` a member
// gets at most that many tiles (each LayerNorm-backward tile writes a
// partial row of dgamma / dbeta that the finalize reads back).
static constexpr int64_t kGradMaxTilesPerMember = 64;
static std::vector<RowTile> grad_row_tiles(HostPlan& hp, const std::vector<DevRowsGrad>& members, size_t s,
                                           std::vector<int>& ntiles, int64_t max_tiles) {
  std::vector<RowTile> tiles;
  hp.rows_chain.clear();
  ntiles.assign(members.size(), 0);
  for (size_t g = 0; g < members.size(); ++g) {
    const DevRowsGrad& m = members[g];
    const int rpb = m.vec ? 4 * (64 / m.lanes) : 4;
    const int64_t row_bytes = std::max<int64_t>(1, (int64_t)m.cols * (int64_t)s);
    int64_t per = std::max<int64_t>(1, kRowTileBytes / row_bytes);
    if (max_tiles > 0) per = std::max<int64_t>(per, (m.rows + max_tiles - 1) / max_tiles);
    per = (per + rpb - 1) / rpb * rpb;
    const int first = (int)tiles.size();
    for (int64_t r0 = 0; r0 < m.rows; r0 += per)
      tiles.push_back(RowTile{(int)g, (int32_t)r0, (int32_t)std::min<int64_t>(per, m.rows - r0), 0});
    for (int t = first; t < (int)tiles.size(); ++t) tiles[t].pad = t - first;
    ntiles[g] = (int)tiles.size() - first;
    hp.rows_chain.push_back(RowLaunch{0, 0, first, ntiles[g], row_grid(ntiles[g])});
  }
  return tiles;
}

// act != NONE: the backward of the fused LayerNorm + activation (beta: G
// pointers or NULL).
static optimus_status build_layernorm_backward(const optimus_layernorm_grad_desc* d, int32_t G, optimus_dtype dt,
                                               HostPlan& hp, const void* const* beta = nullptr,
                                               optimus_act act = OPTIMUS_ACT_NONE) {
  optimus_status st = optimus_validate_layernorm_backward(d, G, dt);
  if (st != OPTIMUS_OK) return st;
  if (!act_ok(act)) return fail(OPTIMUS_ERR_UNSUPPORTED, "grouped_layernorm_act_backward: unknown activation %d", (int)act);
  hp.kind = KIND_LNBWD; hp.dt = dt; hp.act = act; hp.G = G;
  const size_t s = dtype_size(dt);
  std::vector<DevRowsGrad> members;
  for (int g = 0; g < G; ++g) {
    const optimus_layernorm_grad_desc& m = d[g];
    members.push_back(make_rows_grad(m.x, m.ldx, m.dy, m.lddy, m.dx, m.lddx, m.gamma, m.rows, m.cols, m.eps, dt, true));
    members.back().want_params = (m.dgamma || m.dbeta) ? 1 : 0;
    members.back().beta = act != OPTIMUS_ACT_NONE && beta ? beta[g] : nullptr;
    hp.bytes += (double)s * (3.0 * m.rows * m.cols + (m.gamma ? m.cols : 0) + (m.dgamma ? m.cols : 0) +
                             (m.dbeta ? m.cols : 0));
  }
  // The per-op chain launches each member over at most kGradMaxTilesPerMember
  // row tiles (hp.rows_chain). The grouped launch takes balanced row
  // segments (balanced_row_segments): the work is balanced to a row, and a
  // member has one dgamma / dbeta partial row per segment (about one per
  // workgroup that touches it), not per tile.
  std::vector<int> ntiles;
  std::vector<RowTile> chain_tiles = grad_row_tiles(hp, members, s, ntiles, kGradMaxTilesPerMember);
  std::vector<int> nseg;
  std::vector<RowTile> tiles;
  int64_t B;
  {
    std::vector<int64_t> rows;
    std::vector<double> rb;
    for (const auto& m : members) {
      rows.push_back(m.rows);
      rb.push_back((double)m.cols * (double)s);
    }
    B = balanced_row_segments(rows, rb, (int64_t)device_cu_count() * layernorm_backward_resident_per_cu(dt, act),
                              tiles, nseg);
  }
  // partial rows: one per segment or chain tile (16-byte path), per wave of
  // one (per-value path); room for the larger of the two layouts
  std::vector<int> nparts(G, 0), nparts_chain(G, 0);
  std::vector<int64_t> part_rows(G, 0);
  for (int g = 0; g < G; ++g) {
    if (!members[g].want_params) continue;
    const int k = members[g].vec ? 1 : kGradWavesPerBlock;
    nparts[g] = nseg[g] * k;
    nparts_chain[g] = ntiles[g] * k;
    part_rows[g] = std::max(nparts[g], nparts_chain[g]);
  }
  int64_t part_floats = 0;  // offsets in floats of each member's first partial row
  std::vector<int64_t> part_off(G, 0);
  for (int g = 0; g < G; ++g) {
    part_off[g] = part_floats;
    if (members[g].want_params) part_floats += part_rows[g] * 2 * members[g].cols;
  }
  // the kernel addresses partial row p of a member at part + p * 2 * cols: give
  // each member its own base so rows of different widths do not overlap
  const size_t part_off_blob = hp.blob.add(nullptr, (size_t)std::max<int64_t>(part_floats, 1) * sizeof(float));
  for (int g = 0; g < G; ++g) {
    members[g].part = (float*)(uintptr_t)(part_off_blob + (size_t)part_off[g] * sizeof(float));
    members[g].part0 = 0;
  }
  const size_t doff = hp.blob.add(members.data(), members.size() * sizeof(DevRowsGrad));
  for (int g = 0; g < G; ++g) hp.table_fixups.push_back(doff + g * sizeof(DevRowsGrad) + offsetof(DevRowsGrad, part));
  const size_t toff = hp.blob.add(tiles.data(), tiles.size() * sizeof(RowTile));
  const size_t ctoff = hp.blob.add(chain_tiles.data(), chain_tiles.size() * sizeof(RowTile));
  for (auto& c : hp.rows_chain) {
    c.descs_off = doff;
    c.tiles_off = ctoff;
  }
  hp.rows = RowLaunch{doff, toff, 0, (int32_t)tiles.size(), (int32_t)B};
  // finalize items: kFinCols columns each, for the grouped layout, then for the chain's
  std::vector<GradFinItem> fin;
  auto add_fin = [&](int g, int np) {
    if (members[g].want_params)
      for (int c0 = 0; c0 < members[g].cols; c0 += kFinCols)
        fin.push_back(GradFinItem{(const float*)(uintptr_t)(part_off_blob + (size_t)part_off[g] * sizeof(float)),
                                  d[g].dgamma, d[g].dbeta, members[g].cols, np, c0, 0});
  };
  for (int g = 0; g < G; ++g) add_fin(g, nparts[g]);
  const int32_t n_fin_grouped = (int32_t)fin.size();
  hp.fin_chain.assign(G, RowLaunch{});
  for (int g = 0; g < G; ++g) {
    const int first = (int)fin.size();
    add_fin(g, nparts_chain[g]);
    hp.fin_chain[g] = RowLaunch{0, 0, first, (int)fin.size() - first, 0};
  }
  const size_t foff = hp.blob.add(fin.data(), fin.size() * sizeof(GradFinItem));
  for (size_t i = 0; i < fin.size(); ++i) hp.table_fixups.push_back(foff + i * sizeof(GradFinItem) + offsetof(GradFinItem, part));
  const int32_t fin_cap = device_cu_count() * 4;
  hp.fin = RowLaunch{foff, foff, 0, n_fin_grouped, std::max<int32_t>(1, std::min<int32_t>(n_fin_grouped, fin_cap))};
  for (auto& c : hp.fin_chain) {
    c.descs_off = c.tiles_off = foff;
    c.grid = std::max(1, std::min(c.num_tiles, fin_cap));
  }
  int64_t segs = 0;
  for (int g = 0; g < G; ++g) segs += nseg[g];
  hp.work_items = segs;
  hp.grid = hp.rows.grid;
  hp.block = kRowThreads;
  hp.launches = n_fin_grouped == 0 ? 1 : 2;
  hp.chain_launches = 0;
  for (int g = 0; g < G; ++g) hp.chain_launches += 1 + (hp.fin_chain[g].num_tiles > 0 ? 1 : 0);
  static const char* const act_names[] = {"", "_relu", "_sigmoid", "_tanh", "_silu"};
  hp.kernel = std::string("grouped_layernorm_backward") + act_names[(int)act] + (dt == OPTIMUS_F32 ? "_f32" : "_bf16");
  return OPTIMUS_OK;
}

static optimus_status build_act_backward(const optimus_act_grad_desc* d, int32_t G, optimus_dtype dt, optimus_act act,
                                         HostPlan& hp) {
  optimus_status st = optimus_validate_act_backward(d, G, dt, act);
  if (st != OPTIMUS_OK) return st;
  hp.kind = KIND_ACTBWD; hp.dt = dt; hp.act = act; hp.G = G;
  const size_t s = dtype_size(dt);
  std::vector<DevRowsGrad> members;
  for (int g = 0; g < G; ++g) {
    const optimus_act_grad_desc& m = d[g];
    members.push_back(make_rows_grad(m.x, m.ldx, m.dy, m.lddy, m.dx, m.lddx, nullptr, m.rows, m.cols, 0.f, dt, false));
    hp.bytes += (double)s * 3.0 * m.rows * m.cols;
  }
  std::vector<int> ntiles;
  std::vector<RowTile> tiles = grad_row_tiles(hp, members, s, ntiles, 0);
  const size_t doff = hp.blob.add(members.data(), members.size() * sizeof(DevRowsGrad));
  const size_t toff = hp.blob.add(tiles.data(), tiles.size() * sizeof(RowTile));
  for (auto& c : hp.rows_chain) {
    c.descs_off = doff;
    c.tiles_off = toff;
  }
  hp.rows = RowLaunch{doff, toff, 0, (int32_t)tiles.size(), row_grid((int64_t)tiles.size())};
  hp.work_items = (int64_t)tiles.size();
  hp.grid = hp.rows.grid;
  hp.block = kRowThreads;
  hp.chain_launches = G;
  hp.kernel = dt == OPTIMUS_F32 ? "grouped_act_backward_f32" : "grouped_act_backward_bf16";
  return OPTIMUS_OK;
}

static optimus_status build_layernorm(const optimus_layernorm_desc* d, int32_t G, optimus_dtype dt, optimus_act act,
                                      HostPlan& hp) {
  optimus_status st = optimus_validate_layernorm(d, G, dt, act);
  if (st != OPTIMUS_OK) return st;
  hp.kind = KIND_LN; hp.dt = dt; hp.act = act; hp.G = G; hp.row_act = act;
  const size_t s = dtype_size(dt);
  std::vector<DevRows> members;
  for (int g = 0; g < G; ++g) {
    const optimus_layernorm_desc& m = d[g];
    members.push_back(make_rows(m.x, m.ldx, m.y, m.ldy, m.gamma, m.beta, m.rows, m.cols, m.eps, dt, true));
    hp.bytes += (double)s * (2.0 * m.rows * m.cols + (m.gamma ? m.cols : 0) + (m.beta ? m.cols : 0));
  }
  build_rows(hp, members, true, s, act);
  hp.kernel = dt == OPTIMUS_F32 ? "grouped_layernorm_f32" : "grouped_layernorm_bf16";
  return OPTIMUS_OK;
}

static constexpr int64_t kPwWideRow = 4096;  // elements per re-viewed row of a contiguous pointwise member
static optimus_status build_pointwise(const optimus_pointwise_desc* d, int32_t G, optimus_dtype dt, optimus_act act,
                                      HostPlan& hp) {
  optimus_status st = optimus_validate_pointwise(d, G, dt, act);
  if (st != OPTIMUS_OK) return st;
  hp.kind = KIND_PW; hp.dt = dt; hp.act = act; hp.G = G; hp.row_act = act;
  const size_t s = dtype_size(dt);
  std::vector<DevRows> members;
  for (int g = 0; g < G; ++g) {
    const optimus_pointwise_desc& m = d[g];
    // an elementwise map ignores the row structure: a member whose rows are
    // contiguous (ld == cols) and shorter than the wide row is re-viewed as
    // rows of kPwWideRow elements, so that every lane keeps several 16-byte
    // loads in flight instead of one per narrow row
    int64_t rows = m.rows, cols = m.cols;
    const int64_t total = m.rows * m.cols;
    if (m.ldx == m.cols && m.ldy == m.cols && m.cols < kPwWideRow && total % kPwWideRow == 0) {
      rows = total / kPwWideRow;
      cols = kPwWideRow;
    }
    members.push_back(make_rows(m.x, cols, m.y, cols, nullptr, nullptr, rows, cols, 0.f, dt, false));
    hp.bytes += (double)s * 2.0 * m.rows * m.cols;
  }
  build_rows(hp, members, false, s, act);
  hp.kernel = dt == OPTIMUS_F32 ? "grouped_pointwise_f32" : "grouped_pointwise_bf16";
  return OPTIMUS_OK;
}

static optimus_status build_split_op_cat(const optimus_split_op_cat_desc* d, optimus_dtype dt, HostPlan& hp,
                                         int32_t wpr = 0) {
  optimus_status st = optimus_validate_split_op_cat(d, dt);
  if (st != OPTIMUS_OK) return st;
  hp.kind = KIND_SOC; hp.dt = dt; hp.act = d->act; hp.G = d->n_slices;
  const size_t s = dtype_size(dt);
  const int VEC = dt == OPTIMUS_F32 ? 4 : 8;
  const int n = d->n_slices;
  const int64_t rows = d->rows, D = d->D;
  std::vector<int64_t> off(n + 1, 0);
  for (int j = 0; j < n; ++j) off[j + 1] = off[j] + d->widths[j];
  hp.bytes = (double)s * 2.0 * rows * D;
  if (d->apply_layernorm)
    for (int j = 0; j < n; ++j)
      hp.bytes += (double)s * ((d->gamma && d->gamma[j] ? d->widths[j] : 0) + (d->beta && d->beta[j] ? d->widths[j] : 0));

  // ---- the optimized program
  bool widths_vec = true;
  for (int j = 0; j < n; ++j) widths_vec = widths_vec && d->widths[j] % VEC == 0;
  const bool vec = widths_vec && d->ldin % VEC == 0 && d->ldout % VEC == 0 && aligned16(d->in) && aligned16(d->out);
  const int64_t nchunks = D / VEC;
  if (!d->apply_layernorm) {
    // same activation on every piece: split and concat vanish into one pointwise pass over [rows, D]
    std::vector<DevRows> m{make_rows(d->in, d->ldin, d->out, d->ldout, nullptr, nullptr, rows, D, 0.f, dt, false)};
    build_rows(hp, m, false, s, d->act);
    hp.row_act = d->act;
    hp.kernel = "split_op_cat_as_pointwise";
  } else if (vec && nchunks <= kSocMaxChunks && n <= kSocMaxPieces) {
    std::vector<uint8_t> cp((size_t)nchunks);
    std::vector<SocPiece> pieces(n);
    for (int j = 0; j < n; ++j) {
      const int c0 = (int)(off[j] / VEC), c1 = (int)(off[j + 1] / VEC);
      pieces[j] = SocPiece{c0, c1, (float)(1.0 / (double)d->widths[j]), 0, nullptr, nullptr};
      for (int c = c0; c < c1; ++c) cp[c] = (uint8_t)j;
    }
    DevSoc soc{};
    soc.in = d->in; soc.out = d->out;
    soc.ldin = d->ldin; soc.ldout = d->ldout;
    soc.rows = (int32_t)rows; soc.D = (int32_t)D; soc.nchunks = (int32_t)nchunks;
    soc.n_pieces = n;
    soc.apply_ln = 1; soc.eps = d->eps;
    // the pieces keep the caller's gamma / beta pointers (read by every launch)
    for (int j = 0; j < n; ++j) {
      pieces[j].gamma = d->gamma ? d->gamma[j] : nullptr;
      pieces[j].beta = d->beta ? d->beta[j] : nullptr;
      pieces[j].vec = (pieces[j].gamma && aligned16(pieces[j].gamma) ? 1 : 0) |
                      (pieces[j].beta && aligned16(pieces[j].beta) ? 2 : 0);
    }
    const size_t cp_off = hp.blob.add(cp.data(), cp.size());
    const size_t pc_off = hp.blob.add(pieces.data(), pieces.size() * sizeof(SocPiece));
    // device pointers inside DevSoc are filled in at upload (relative offsets kept here)
    soc.chunk_piece = (const uint8_t*)(uintptr_t)cp_off;
    soc.pieces = (const SocPiece*)(uintptr_t)pc_off;
    hp.soc_off = hp.blob.add(&soc, sizeof soc);
    hp.soc_fused = true;
    hp.soc_rows = (int32_t)rows;
    hp.soc_nchunks = (int32_t)nchunks;
    hp.soc_pieces = n;
    // the planner's waves per row: at most four of a row's chunks per lane
    // (bf16 rows of 4096: 26.7 -> 26.1 us on two waves per row; of 8192:
    // 40.6 -> 37.3 us on four; rows of 1024 and 2048 gain nothing from two)
    if (wpr == 0) {
      wpr = 1;
      while (wpr < 4 && (nchunks + 64 * wpr - 1) / (64 * wpr) > 4) wpr *= 2;
    }
    // persistent grid: exactly the workgroups that fit at once, each wave walking rows
    hp.soc_wpr = wpr;
    const int64_t resident = (int64_t)device_cu_count() * soc_blocks_per_cu(dt, d->act, (int32_t)nchunks, n, wpr);
    const int rpb = soc_rows_per_block(dt, (int32_t)nchunks, n, wpr);
    hp.soc_grid = (int32_t)std::max<int64_t>(1, std::min<int64_t>((rows + rpb - 1) / rpb, resident));
    hp.work_items = rows;
    hp.grid = hp.soc_grid;
    hp.block = kSocThreads;
    hp.kernel = dt == OPTIMUS_F32 ? "split_op_cat_fused_f32" : "split_op_cat_fused_bf16";
  } else {
    // any other shape: the pieces become the members of one grouped LayerNorm
    // launch that reads and writes them in place (still no split copy, no concat)
    std::vector<DevRows> m;
    for (int j = 0; j < n; ++j)
      m.push_back(make_rows((const char*)d->in + off[j] * s, d->ldin, (char*)d->out + off[j] * s, d->ldout,
                            d->gamma ? d->gamma[j] : nullptr, d->beta ? d->beta[j] : nullptr, rows, d->widths[j],
                            d->eps, dt, true));
    build_rows(hp, m, true, s, d->act);
    hp.row_act = d->act;
    hp.kernel = "split_op_cat_as_grouped_layernorm";
  }
  hp.launches = 1;

  // ---- the unfused programs, for measurement (CHAIN and HORIZONTAL modes):
  // piece j lives in the temporaries at element offset rows * off[j] as a
  // contiguous [rows, w_j] array. Pointers into the temporaries are stored as
  // offsets and rebased when the temporaries exist.
  hp.soc_has_unfused = true;
  hp.soc_apply_ln = d->apply_layernorm != 0;
  hp.soc_temp_elems = rows * D;
  std::vector<DevRows> ln(n), act(n), cat(n);
  for (int j = 0; j < n; ++j) {
    const int64_t w = d->widths[j];
    const uintptr_t t1 = (uintptr_t)(rows * off[j]) * s;                 // offset in temp 1
    const uintptr_t t2 = (uintptr_t)(rows * D + rows * off[j]) * s;      // offset in temp 2
    if (d->apply_layernorm)
      ln[j] = make_rows((const char*)d->in + off[j] * s, d->ldin, (void*)t1, w, d->gamma ? d->gamma[j] : nullptr,
                        d->beta ? d->beta[j] : nullptr, rows, w, d->eps, dt, true);
    else
      ln[j] = make_rows((const char*)d->in + off[j] * s, d->ldin, (void*)t1, w, nullptr, nullptr, rows, w, 0.f, dt,
                        false);
    act[j] = make_rows((const void*)t1, w, (void*)t2, w, nullptr, nullptr, rows, w, 0.f, dt, false);
    cat[j] = make_rows((const void*)t2, w, (char*)d->out + off[j] * s, d->ldout, nullptr, nullptr, rows, w, 0.f, dt, false);
  }
  // make_rows sees temporary offsets in place of pointers; the temporaries are
  // 256-byte aligned, so an offset's alignment is the pointer's alignment.
  std::vector<RowTile> tl;
  hp.soc_piece_first.assign(n, 0);
  hp.soc_piece_count.assign(n, 0);
  for (int j = 0; j < n; ++j) {
    hp.soc_piece_first[j] = (int32_t)tl.size();
    add_row_tiles(tl, j, ln[j], s);  // same row count for every piece: one tile list serves all three
    hp.soc_piece_count[j] = (int32_t)tl.size() - hp.soc_piece_first[j];
  }
  hp.soc_ln_descs = hp.blob.add(ln.data(), n * sizeof(DevRows));
  hp.soc_act_descs = hp.blob.add(act.data(), n * sizeof(DevRows));
  hp.soc_cat_descs = hp.blob.add(cat.data(), n * sizeof(DevRows));
  hp.soc_tiles = hp.blob.add(tl.data(), tl.size() * sizeof(RowTile));
  hp.soc_piece_tiles_total = (int32_t)tl.size();
  for (int j = 0; j < n; ++j) {
    hp.soc_temp_fixups.push_back(hp.soc_ln_descs + j * sizeof(DevRows) + offsetof(DevRows, y));
    hp.soc_temp_fixups.push_back(hp.soc_act_descs + j * sizeof(DevRows) + offsetof(DevRows, x));
    hp.soc_temp_fixups.push_back(hp.soc_act_descs + j * sizeof(DevRows) + offsetof(DevRows, y));
    hp.soc_temp_fixups.push_back(hp.soc_cat_descs + j * sizeof(DevRows) + offsetof(DevRows, x));
  }
  hp.chain_launches = 2 * n + 1;
  return OPTIMUS_OK;
}

// ===================================================================== fp8 codec plans
// Value-side bytes of a convert / dequantize item; an amax item covers
// OPTIMUS_FP8_AMAX_TILES of them, or 1/kFp8MaxSlots of its member if that is
// more, so a convert item reduces at most about kFp8MaxSlots slots.
#ifndef OPTIMUS_FP8_TILE_BYTES
#define OPTIMUS_FP8_TILE_BYTES 32768
#endif
#ifndef OPTIMUS_FP8_AMAX_TILES
#define OPTIMUS_FP8_AMAX_TILES 4
#endif
static constexpr int64_t kFp8MaxSlots = 256;

// Item geometry of one member: the 16-byte path needs value rows made of
// 16-byte chunks (16-byte aligned) and code rows of as many bytes (aligned
// to that many); a unit is then one chunk, else one value.
struct Fp8Geom {
  bool vec;
  int64_t units;       // units per row
  int64_t unit_bytes;  // value-side bytes of a unit
  int lanes;           // threads per row
};

// Widest row segment of an item of about `budget` value bytes, in units (a
// multiple of the 256 threads of a block).
static int64_t fp8_seg(const Fp8Geom& g, int64_t budget) {
  return std::max<int64_t>(256, (budget / g.unit_bytes) / 256 * 256);
}

static Fp8Geom fp8_geom(const void* vals, int64_t ldv, const void* codes, int64_t ldc, int64_t cols, optimus_dtype dt) {
  const int64_t s = (int64_t)dtype_size(dt), VEC = 16 / s;
  Fp8Geom g{};
  g.vec = cols % VEC == 0 && ldv % VEC == 0 && ldc % VEC == 0 && aligned16(vals) && ((uintptr_t)codes % VEC) == 0;
  g.units = g.vec ? cols / VEC : cols;
  g.unit_bytes = g.vec ? 16 : s;
  g.lanes = std::min(256, pow2ceil((int)std::min<int64_t>(g.units, fp8_seg(g, OPTIMUS_FP8_TILE_BYTES))));
  return g;
}

// Items covering one member with tiles of about `budget` value bytes: whole
// rows (a multiple of the block's row slots) when a row fits, else
// single-row segments. slot >= 0: amax items, slots numbered from `slot`.
// Every item is at least as wide as the member's lanes cover or is a whole
// row, so the block walk of the kernels fits any of them.
static void fp8_items(const Fp8Geom& g, int member, int64_t rows, int64_t budget, int32_t slot,
                      std::vector<Fp8Item>& out) {
  const int64_t row_bytes = g.units * g.unit_bytes;
  const int64_t seg = fp8_seg(g, budget);
  if (g.units <= seg) {
    const int64_t rpb = 256 / g.lanes;
    int64_t per = std::max<int64_t>(1, budget / row_bytes);
    per = std::max<int64_t>(rpb, per / rpb * rpb);
    for (int64_t r0 = 0; r0 < rows; r0 += per)
      out.push_back(Fp8Item{member, (int32_t)r0, (int32_t)std::min<int64_t>(per, rows - r0), 0, (int32_t)g.units,
                            slot < 0 ? -1 : slot++});
  } else {
    for (int64_t r = 0; r < rows; ++r)
      for (int64_t c0 = 0; c0 < g.units; c0 += seg)
        out.push_back(Fp8Item{member, (int32_t)r, 1, (int32_t)c0, (int32_t)std::min<int64_t>(c0 + seg, g.units),
                              slot < 0 ? -1 : slot++});
  }
}


// Shared by quantize and dequantize: the member table and item lists.
// Grouped: (scaled: the amax items, then) the convert items, member order.
// CHAIN: per member, its own items.
static void build_fp8(HostPlan& hp, std::vector<DevFp8>& members, const std::vector<Fp8Geom>& geo, bool scaled) {
  const int G = (int)members.size();
  std::vector<std::vector<Fp8Item>> conv(G), amax(G);
  int32_t nslots = 0;
  for (int g = 0; g < G; ++g) {
    DevFp8& m = members[g];
    m.lanes = geo[g].vec ? geo[g].lanes : 0;
    m.lanes_scalar = geo[g].vec ? 0 : geo[g].lanes;
    fp8_items(geo[g], g, m.rows, OPTIMUS_FP8_TILE_BYTES, -1, conv[g]);
    if (scaled) {
      const int64_t bytes = (int64_t)m.rows * geo[g].units * geo[g].unit_bytes;
      const int64_t budget = std::max<int64_t>((int64_t)OPTIMUS_FP8_TILE_BYTES * OPTIMUS_FP8_AMAX_TILES,
                                               (bytes + kFp8MaxSlots - 1) / kFp8MaxSlots);
      m.slot0 = nslots;
      fp8_items(geo[g], g, m.rows, budget, nslots, amax[g]);
      m.nslots = (int32_t)amax[g].size();
      nslots += m.nslots;
    }
  }
  std::vector<Fp8Item> items;
  // one workgroup per item, as for the row-wise grids
  auto add = [&](const std::vector<Fp8Item>& v) {
    const int32_t first = (int32_t)items.size();
    items.insert(items.end(), v.begin(), v.end());
    return RowLaunch{0, 0, first, (int32_t)v.size(), row_grid((int64_t)v.size())};
  };
  std::vector<Fp8Item> all_a, all_c;
  for (int g = 0; g < G; ++g) all_a.insert(all_a.end(), amax[g].begin(), amax[g].end());
  for (int g = 0; g < G; ++g) all_c.insert(all_c.end(), conv[g].begin(), conv[g].end());
  hp.q_amax = scaled ? add(all_a) : RowLaunch{};
  hp.q_grouped = add(all_c);
  hp.q_chain.clear();
  hp.q_chain_amax.clear();
  for (int g = 0; g < G; ++g) {
    if (scaled) hp.q_chain_amax.push_back(add(amax[g]));
    hp.q_chain.push_back(add(conv[g]));
  }
  hp.q_scaled = scaled;
  hp.q_descs_off = hp.blob.add(members.data(), members.size() * sizeof(DevFp8));
  hp.q_items_off = hp.blob.add(items.data(), items.size() * sizeof(Fp8Item));
  if (scaled) hp.q_slots_off = hp.blob.add(nullptr, (size_t)std::max(nslots, 1) * sizeof(uint32_t));
  hp.work_items = (int64_t)all_a.size() + (int64_t)all_c.size();
  hp.grid = hp.q_grouped.grid;
  hp.block = 256;
  hp.launches = scaled ? 2 : 1;
  hp.chain_launches = scaled ? 2 * G : G;
}

static optimus_status build_quantize_fp8(const optimus_fp8_quant_desc* d, int32_t G, optimus_dtype dt,
                                         int32_t use_scaling, HostPlan& hp) {
  optimus_status st = optimus_validate_quantize_fp8(d, G, dt, use_scaling);
  if (st != OPTIMUS_OK) return st;
  hp.kind = KIND_Q8; hp.dt = dt; hp.G = G;
  const size_t s = dtype_size(dt);
  std::vector<DevFp8> members;
  std::vector<Fp8Geom> geo;
  for (int g = 0; g < G; ++g) {
    const optimus_fp8_quant_desc& m = d[g];
    DevFp8 r{};
    r.x = m.x; r.y = m.q; r.scale = use_scaling ? m.scale : nullptr;
    r.ldx = m.ldx; r.ldy = m.ldq; r.rows = (int32_t)m.rows; r.cols = (int32_t)m.cols;
    members.push_back(r);
    geo.push_back(fp8_geom(m.x, m.ldx, m.q, m.ldq, m.cols, dt));
    hp.bytes += (double)m.rows * m.cols * (double)(s + 1) + (use_scaling ? 4.0 : 0.0);
  }
  build_fp8(hp, members, geo, use_scaling != 0);
  hp.kernel = std::string(use_scaling ? "grouped_quantize_fp8_scaled_" : "grouped_quantize_fp8_") +
              (dt == OPTIMUS_F32 ? "f32" : "bf16");
  return OPTIMUS_OK;
}

static optimus_status build_dequantize_fp8(const optimus_fp8_dequant_desc* d, int32_t G, optimus_dtype dt,
                                           HostPlan& hp) {
  optimus_status st = optimus_validate_dequantize_fp8(d, G, dt);
  if (st != OPTIMUS_OK) return st;
  hp.kind = KIND_DQ8; hp.dt = dt; hp.G = G;
  const size_t s = dtype_size(dt);
  std::vector<DevFp8> members;
  std::vector<Fp8Geom> geo;
  for (int g = 0; g < G; ++g) {
    const optimus_fp8_dequant_desc& m = d[g];
    DevFp8 r{};
    r.x = m.q; r.y = m.y; r.scale = const_cast<float*>(m.scale);
    r.ldx = m.ldq; r.ldy = m.ldy; r.rows = (int32_t)m.rows; r.cols = (int32_t)m.cols;
    members.push_back(r);
    geo.push_back(fp8_geom(m.y, m.ldy, m.q, m.ldq, m.cols, dt));
    hp.bytes += (double)m.rows * m.cols * (double)(s + 1) + (m.scale ? 4.0 : 0.0);
  }
  build_fp8(hp, members, geo, false);
  hp.kernel = std::string("grouped_dequantize_fp8_") + (dt == OPTIMUS_F32 ? "f32" : "bf16");
  return OPTIMUS_OK;
}

// ===================================================================== device side of a plan
struct optimus_plan_s {
  HostPlan hp;
  int device = 0;
  char* table = nullptr;       // device copy of hp.blob
  char* temps = nullptr;       // split-op-cat unfused temporaries (lazy)
  char* scratch = nullptr;     // hp.scratch_bytes of plan-owned scratch
  bool temps_ready = false;
};

// Rebase the pointer fields that hold blob offsets (split-op-cat tables).
static void rebase_soc(HostPlan& hp, char* table) {
  if (!hp.soc_fused) return;
  DevSoc* s = (DevSoc*)(hp.blob.bytes.data() + hp.soc_off);
  s->chunk_piece = (const uint8_t*)(table + (uintptr_t)s->chunk_piece);
  s->pieces = (const SocPiece*)(table + (uintptr_t)s->pieces);
}

// Every pointer the planner stored as a blob (or scratch) offset, made a device address.
static void rebase_fixups(HostPlan& hp, char* table, char* scratch = nullptr) {
  for (int pass = 0; pass < 2; ++pass) {
    const std::vector<size_t>& list = pass ? hp.scratch_fixups : hp.table_fixups;
    char* base = pass ? scratch : table;
    for (size_t off : list) {
      uintptr_t v;
      memcpy(&v, hp.blob.bytes.data() + off, sizeof v);
      v += (uintptr_t)base;
      memcpy(hp.blob.bytes.data() + off, &v, sizeof v);
    }
  }
}

template <typename P>
static const P* at(char* table, size_t off) {
  return (const P*)(table + off);
}

// One execution of a codec plan over the given item ranges: for scaled
// quantize the amax launch, then the convert launch.
static hipError_t launch_fp8(const HostPlan& hp, char* table, const RowLaunch* amax, const RowLaunch& conv,
                             hipStream_t stream) {
  const DevFp8* descs = at<DevFp8>(table, hp.q_descs_off);
  const Fp8Item* items = at<Fp8Item>(table, hp.q_items_off);
  if (hp.kind == KIND_DQ8)
    return fp8_dequantize_launch(hp.dt, descs, items + conv.first_tile, conv.num_tiles, conv.grid, stream);
  uint32_t* slots = nullptr;
  if (hp.q_scaled) {
    slots = (uint32_t*)(table + hp.q_slots_off);
    hipError_t e = fp8_amax_launch(hp.dt, descs, items + amax->first_tile, amax->num_tiles, amax->grid, slots, stream);
    if (e != hipSuccess) return e;
  }
  return fp8_quantize_launch(hp.dt, descs, items + conv.first_tile, conv.num_tiles, conv.grid, slots, stream);
}

static hipError_t launch_grouped(const HostPlan& hp, char* table, hipStream_t stream) {
  switch (hp.kind) {
    case KIND_Q8:
    case KIND_DQ8:
      return launch_fp8(hp, table, &hp.q_amax, hp.q_grouped, stream);
    case KIND_ACTBWD:
      return act_backward_launch(hp.dt, hp.act, at<DevRowsGrad>(table, hp.rows.descs_off),
                                 at<RowTile>(table, hp.rows.tiles_off), hp.rows.num_tiles, hp.rows.grid, stream);
    case KIND_LNBWD: {
      hipError_t e = layernorm_backward_launch(hp.dt, hp.act, at<DevRowsGrad>(table, hp.rows.descs_off),
                                               at<RowTile>(table, hp.rows.tiles_off), hp.rows.num_tiles,
                                               hp.rows.grid, stream);
      if (e != hipSuccess) return e;
      return grad_finalize_launch(hp.dt, at<GradFinItem>(table, hp.fin.descs_off), hp.fin.num_tiles, hp.fin.grid,
                                  stream);
    }
    case KIND_LINEAR:
    case KIND_LINBWD:
      if (hp.tp.num_tiles > 0) {
        hipError_t e = transpose_launch(hp.dt, at<TransposeItem>(table, hp.tp.descs_off), hp.tp.num_tiles, hp.tp.grid,
                                        stream);
        if (e != hipSuccess) return e;
      }
      for (int i = 0; i < hp.n_gs; ++i) {
        const GemmSet& g = hp.gs[i];
        hipError_t e = gemm_launch(g.cfg, hp.dt, g.act, hp.g_ln, at<DevLinear>(table, g.descs_off),
                                   at<GemmTile>(table, g.tiles_off), g.num_tiles, g.grid, stream, g.tr);
        if (e != hipSuccess) return e;
      }
      if (hp.kind == KIND_LINBWD && hp.rows.num_tiles > 0) {
        // the activation backward of the layer below, over dX in place
        hipError_t e = act_backward_launch(hp.dt, hp.act, at<DevRowsGrad>(table, hp.rows.descs_off),
                                           at<RowTile>(table, hp.rows.tiles_off), hp.rows.num_tiles, hp.rows.grid,
                                           stream);
        if (e != hipSuccess) return e;
      }
      return splitk_reduce_launch(hp.dt, at<SplitReduceItem>(table, hp.red.descs_off), hp.red.num_tiles, hp.red.grid,
                                  stream);
    case KIND_LN:
    case KIND_PW:
    case KIND_SOC:
      if (hp.kind == KIND_SOC && hp.soc_fused)
        return soc_launch(hp.dt, hp.act, at<DevSoc>(table, hp.soc_off), hp.soc_nchunks, hp.soc_pieces, hp.soc_wpr,
                          hp.soc_grid, stream);
      if (hp.row_kernel == KIND_LN)
        return layernorm_launch(hp.dt, hp.row_act, at<DevRows>(table, hp.rows.descs_off),
                                at<RowTile>(table, hp.rows.tiles_off), hp.rows.num_tiles, hp.rows.grid, stream);
      return pointwise_launch(hp.dt, hp.row_act, at<DevRows>(table, hp.rows.descs_off),
                              at<RowTile>(table, hp.rows.tiles_off), hp.rows.num_tiles, hp.rows.grid, stream);
  }
  return hipErrorInvalidValue;
}

static optimus_status make_plan(HostPlan&& hp, optimus_plan* out) {
  if (!out) return fail(OPTIMUS_ERR_INVALID_ARG, "plan: output pointer is NULL");
  *out = nullptr;
  optimus_plan p = new (std::nothrow) optimus_plan_s();
  if (!p) return fail(OPTIMUS_ERR_OOM, "plan: host allocation failed");
  p->hp = std::move(hp);
  if (hipGetDevice(&p->device) != hipSuccess) p->device = 0;
  const size_t n = std::max<size_t>(p->hp.blob.bytes.size(), 256);
  hipError_t e = hipMalloc((void**)&p->table, n);
  if (e != hipSuccess) {
    delete p;
    return hip_fail(e, "plan: device table allocation");
  }
  if (p->hp.scratch_bytes) {
    e = hipMalloc((void**)&p->scratch, p->hp.scratch_bytes);
    if (e != hipSuccess) {
      (void)hipFree(p->table);
      delete p;
      return hip_fail(e, "plan: scratch allocation");
    }
  }
  rebase_soc(p->hp, p->table);
  rebase_fixups(p->hp, p->table, p->scratch);
  e = hipMemcpy(p->table, p->hp.blob.bytes.data(), p->hp.blob.bytes.size(), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(p->table);
    if (p->scratch) (void)hipFree(p->scratch);
    delete p;
    return hip_fail(e, "plan: device table upload");
  }
  *out = p;
  return OPTIMUS_OK;
}

extern "C" optimus_status optimus_plan_linear_ex(const optimus_linear_desc* d, int32_t G, optimus_dtype dt,
                                                 optimus_act epilogue, const optimus_plan_options* opt,
                                                 optimus_plan* out) {
  PlanOpts po;
  optimus_status st = parse_options(opt, po);
  if (st != OPTIMUS_OK) return st;
  HostPlan hp;
  st = build_linear(d, G, dt, epilogue, hp, false, nullptr, nullptr, 0.f, po);
  if (st != OPTIMUS_OK) return st;
  return make_plan(std::move(hp), out);
}
extern "C" optimus_status optimus_plan_linear(const optimus_linear_desc* d, int32_t G, optimus_dtype dt,
                                              optimus_act epilogue, optimus_plan* out) {
  return optimus_plan_linear_ex(d, G, dt, epilogue, nullptr, out);
}
extern "C" optimus_status optimus_plan_linear_layernorm_ex(const optimus_linear_desc* d, const void* const* gamma,
                                                           const void* const* beta, int32_t G, optimus_dtype dt,
                                                           float eps, optimus_act epilogue,
                                                           const optimus_plan_options* opt, optimus_plan* out) {
  PlanOpts po;
  optimus_status st = parse_options(opt, po);
  if (st != OPTIMUS_OK) return st;
  HostPlan hp;
  st = build_linear(d, G, dt, epilogue, hp, true, gamma, beta, eps, po);
  if (st != OPTIMUS_OK) return st;
  return make_plan(std::move(hp), out);
}
extern "C" optimus_status optimus_plan_linear_layernorm(const optimus_linear_desc* d, const void* const* gamma,
                                                        const void* const* beta, int32_t G, optimus_dtype dt,
                                                        float eps, optimus_act epilogue, optimus_plan* out) {
  return optimus_plan_linear_layernorm_ex(d, gamma, beta, G, dt, eps, epilogue, nullptr, out);
}
extern "C" optimus_status optimus_plan_layernorm(const optimus_layernorm_desc* d, int32_t G, optimus_dtype dt,
                                                 optimus_act epilogue, optimus_plan* out) {
  HostPlan hp;
  optimus_status st = build_layernorm(d, G, dt, epilogue, hp);
  if (st != OPTIMUS_OK) return st;
  return make_plan(std::move(hp), out);
}
extern "C" optimus_status optimus_plan_pointwise(const optimus_pointwise_desc* d, int32_t G, optimus_dtype dt,
                                                 optimus_act op, optimus_plan* out) {
  HostPlan hp;
  optimus_status st = build_pointwise(d, G, dt, op, hp);
  if (st != OPTIMUS_OK) return st;
  return make_plan(std::move(hp), out);
}
extern "C" optimus_status optimus_plan_split_op_cat_ex(const optimus_split_op_cat_desc* d, optimus_dtype dt,
                                                       const optimus_plan_options* opt, optimus_plan* out) {
  PlanOpts po;
  optimus_status st = parse_options(opt, po);
  if (st != OPTIMUS_OK) return st;
  HostPlan hp;
  st = build_split_op_cat(d, dt, hp, po.wpr);
  if (st != OPTIMUS_OK) return st;
  return make_plan(std::move(hp), out);
}
extern "C" optimus_status optimus_plan_split_op_cat(const optimus_split_op_cat_desc* d, optimus_dtype dt,
                                                    optimus_plan* out) {
  return optimus_plan_split_op_cat_ex(d, dt, nullptr, out);
}
extern "C" optimus_status optimus_plan_linear_backward_ex(const optimus_linear_grad_desc* d, int32_t G,
                                                          optimus_dtype dt, const optimus_plan_options* opt,
                                                          optimus_plan* out) {
  PlanOpts po;
  optimus_status st = parse_options(opt, po);
  if (st != OPTIMUS_OK) return st;
  HostPlan hp;
  st = build_linear_backward(d, G, dt, hp, OPTIMUS_ACT_NONE, nullptr, nullptr, po);
  if (st != OPTIMUS_OK) return st;
  return make_plan(std::move(hp), out);
}
extern "C" optimus_status optimus_plan_linear_backward(const optimus_linear_grad_desc* d, int32_t G, optimus_dtype dt,
                                                       optimus_plan* out) {
  return optimus_plan_linear_backward_ex(d, G, dt, nullptr, out);
}
extern "C" optimus_status optimus_plan_layernorm_backward(const optimus_layernorm_grad_desc* d, int32_t G,
                                                          optimus_dtype dt, optimus_plan* out) {
  HostPlan hp;
  optimus_status st = build_layernorm_backward(d, G, dt, hp);
  if (st != OPTIMUS_OK) return st;
  return make_plan(std::move(hp), out);
}
extern "C" optimus_status optimus_plan_linear_act_backward_ex(const optimus_linear_grad_desc* d,
                                                              const void* const* act_x, const int64_t* ld_act_x,
                                                              int32_t G, optimus_dtype dt, optimus_act act,
                                                              const optimus_plan_options* opt, optimus_plan* out) {
  PlanOpts po;
  optimus_status st = parse_options(opt, po);
  if (st != OPTIMUS_OK) return st;
  HostPlan hp;
  st = build_linear_backward(d, G, dt, hp, act, act_x, ld_act_x, po);
  if (st != OPTIMUS_OK) return st;
  return make_plan(std::move(hp), out);
}
extern "C" optimus_status optimus_plan_linear_act_backward(const optimus_linear_grad_desc* d, const void* const* act_x,
                                                           const int64_t* ld_act_x, int32_t G, optimus_dtype dt,
                                                           optimus_act act, optimus_plan* out) {
  return optimus_plan_linear_act_backward_ex(d, act_x, ld_act_x, G, dt, act, nullptr, out);
}
extern "C" optimus_status optimus_plan_layernorm_act_backward(const optimus_layernorm_grad_desc* d,
                                                              const void* const* beta, int32_t G, optimus_dtype dt,
                                                              optimus_act act, optimus_plan* out) {
  HostPlan hp;
  optimus_status st = build_layernorm_backward(d, G, dt, hp, beta, act);
  if (st != OPTIMUS_OK) return st;
  return make_plan(std::move(hp), out);
}
extern "C" optimus_status optimus_plan_act_backward(const optimus_act_grad_desc* d, int32_t G, optimus_dtype dt,
                                                    optimus_act act, optimus_plan* out) {
  HostPlan hp;
  optimus_status st = build_act_backward(d, G, dt, act, hp);
  if (st != OPTIMUS_OK) return st;
  return make_plan(std::move(hp), out);
}
extern "C" optimus_status optimus_plan_quantize_fp8(const optimus_fp8_quant_desc* d, int32_t G, optimus_dtype dt,
                                                    int32_t use_scaling, optimus_plan* out) {
  HostPlan hp;
  optimus_status st = build_quantize_fp8(d, G, dt, use_scaling, hp);
  if (st != OPTIMUS_OK) return st;
  return make_plan(std::move(hp), out);
}
extern "C" optimus_status optimus_plan_dequantize_fp8(const optimus_fp8_dequant_desc* d, int32_t G, optimus_dtype dt,
                                                      optimus_plan* out) {
  HostPlan hp;
  optimus_status st = build_dequantize_fp8(d, G, dt, hp);
  if (st != OPTIMUS_OK) return st;
  return make_plan(std::move(hp), out);
}

extern "C" void optimus_plan_destroy(optimus_plan p) {
  if (!p) return;
  int cur = 0;
  const bool switched = hipGetDevice(&cur) == hipSuccess && cur != p->device && hipSetDevice(p->device) == hipSuccess;
  (void)hipFree(p->table);
  if (p->temps) (void)hipFree(p->temps);
  if (p->scratch) (void)hipFree(p->scratch);
  if (switched) (void)hipSetDevice(cur);
  delete p;
}

// Temporaries of the unfused split-op-cat programs, with the descriptor
// pointers that refer to them rebased and re-uploaded.
static optimus_status soc_prepare_temps(optimus_plan p) {
  if (p->temps_ready) return OPTIMUS_OK;
  HostPlan& hp = p->hp;
  const size_t bytes = (size_t)hp.soc_temp_elems * 2 * dtype_size(hp.dt);
  HIP_TRY(hipMalloc((void**)&p->temps, std::max<size_t>(bytes, 256)), "split_op_cat: temporaries");
  for (size_t off : hp.soc_temp_fixups) {
    uintptr_t v;
    memcpy(&v, hp.blob.bytes.data() + off, sizeof v);
    v += (uintptr_t)p->temps;
    HIP_TRY(hipMemcpy(p->table + off, &v, sizeof v, hipMemcpyHostToDevice), "split_op_cat: temporaries table");
  }
  p->temps_ready = true;
  return OPTIMUS_OK;
}

extern "C" optimus_status optimus_plan_execute_mode(optimus_plan p, optimus_exec_mode mode, optimus_stream_t stream) {
  if (!p) return fail(OPTIMUS_ERR_INVALID_ARG, "execute: plan is NULL");
  HostPlan& hp = p->hp;
  hipStream_t st = (hipStream_t)stream;
  if (hp.G == 0) return OPTIMUS_OK;
  if (mode == OPTIMUS_EXEC_GROUPED) {
    hipError_t e = launch_grouped(hp, p->table, st);
    return e == hipSuccess ? OPTIMUS_OK : hip_fail(e, "execute: grouped launch");
  }
  if (mode == OPTIMUS_EXEC_CHAIN && hp.kind != KIND_SOC) {
    for (int g = 0; g < hp.G; ++g) {
      hipError_t e;
      if (hp.kind == KIND_ACTBWD || hp.kind == KIND_LNBWD) {
        const RowLaunch& c = hp.rows_chain[g];
        const DevRowsGrad* ds = at<DevRowsGrad>(p->table, c.descs_off);
        const RowTile* ts = at<RowTile>(p->table, c.tiles_off) + c.first_tile;
        if (hp.kind == KIND_ACTBWD) {
          e = act_backward_launch(hp.dt, hp.act, ds, ts, c.num_tiles, c.grid, st);
        } else {
          e = layernorm_backward_launch(hp.dt, hp.act, ds, ts, c.num_tiles, c.grid, st);
          const RowLaunch& f = hp.fin_chain[g];
          if (e == hipSuccess && f.num_tiles > 0)
            e = grad_finalize_launch(hp.dt, at<GradFinItem>(p->table, f.descs_off) + f.first_tile, f.num_tiles, f.grid,
                                     st);
        }
      } else if (hp.kind == KIND_Q8 || hp.kind == KIND_DQ8) {
        e = launch_fp8(hp, p->table, hp.q_scaled ? &hp.q_chain_amax[g] : nullptr, hp.q_chain[g], st);
      } else if (hp.kind == KIND_LINEAR || hp.kind == KIND_LINBWD) {
        e = hipSuccess;
        if (!hp.tp_chain.empty() && hp.tp_chain[g].num_tiles > 0) {
          const RowLaunch& c = hp.tp_chain[g];
          e = transpose_launch(hp.dt, at<TransposeItem>(p->table, c.descs_off) + c.first_tile, c.num_tiles, c.grid, st);
        }
        for (int i = 0; i < hp.n_gs && e == hipSuccess; ++i) {
          const GemmSet& gs = hp.gs[i];
          const RowLaunch& c = gs.chain[g];
          if (c.num_tiles > 0)
            e = gemm_launch(gs.cfg, hp.dt, gs.act, hp.g_ln, at<DevLinear>(p->table, gs.descs_off),
                            at<GemmTile>(p->table, c.tiles_off) + c.first_tile, c.num_tiles, c.grid, st, gs.tr);
        }
        if (e == hipSuccess && hp.kind == KIND_LINBWD && hp.rows.num_tiles > 0 && hp.rows_chain[g].num_tiles > 0) {
          const RowLaunch& c = hp.rows_chain[g];
          e = act_backward_launch(hp.dt, hp.act, at<DevRowsGrad>(p->table, c.descs_off),
                                  at<RowTile>(p->table, c.tiles_off) + c.first_tile, c.num_tiles, c.grid, st);
        }
        if (e == hipSuccess && !hp.red_chain.empty() && hp.red_chain[g].num_tiles > 0) {
          const RowLaunch& r = hp.red_chain[g];
          e = splitk_reduce_launch(hp.dt, at<SplitReduceItem>(p->table, r.descs_off) + r.first_tile, r.num_tiles,
                                   r.grid, st);
        }
      } else {
        const RowLaunch& c = hp.rows_chain[g];
        const DevRows* ds = at<DevRows>(p->table, c.descs_off);
        const RowTile* ts = at<RowTile>(p->table, c.tiles_off) + c.first_tile;
        e = hp.row_kernel == KIND_LN ? layernorm_launch(hp.dt, hp.row_act, ds, ts, c.num_tiles, c.grid, st)
                                     : pointwise_launch(hp.dt, hp.row_act, ds, ts, c.num_tiles, c.grid, st);
      }
      if (e != hipSuccess) return hip_fail(e, "execute: chain launch");
    }
    return OPTIMUS_OK;
  }
  if (hp.kind != KIND_SOC || (mode != OPTIMUS_EXEC_CHAIN && mode != OPTIMUS_EXEC_HORIZONTAL))
    return fail(OPTIMUS_ERR_INVALID_ARG, "execute: mode %d does not apply to this plan", (int)mode);
  optimus_status s = soc_prepare_temps(p);
  if (s != OPTIMUS_OK) return s;
  const DevRows* ln = at<DevRows>(p->table, hp.soc_ln_descs);
  const DevRows* act = at<DevRows>(p->table, hp.soc_act_descs);
  const DevRows* cat = at<DevRows>(p->table, hp.soc_cat_descs);
  const RowTile* tl = at<RowTile>(p->table, hp.soc_tiles);
  const bool ln_on = hp.soc_apply_ln;
  const int n = hp.G;
  hipError_t e = hipSuccess;
  if (mode == OPTIMUS_EXEC_HORIZONTAL) {
    const int32_t T = hp.soc_piece_tiles_total, grid = row_grid(T);
    e = ln_on ? layernorm_launch(hp.dt, OPTIMUS_ACT_NONE, ln, tl, T, grid, st)
              : pointwise_launch(hp.dt, OPTIMUS_ACT_NONE, ln, tl, T, grid, st);
    if (e == hipSuccess) e = pointwise_launch(hp.dt, hp.act, act, tl, T, grid, st);
    if (e == hipSuccess) e = pointwise_launch(hp.dt, OPTIMUS_ACT_NONE, cat, tl, T, grid, st);
  } else {
    for (int j = 0; j < n && e == hipSuccess; ++j) {
      const RowTile* tj = tl + hp.soc_piece_first[j];
      const int32_t cnt = hp.soc_piece_count[j];
      e = ln_on ? layernorm_launch(hp.dt, OPTIMUS_ACT_NONE, ln, tj, cnt, row_grid(cnt), st)
                : pointwise_launch(hp.dt, OPTIMUS_ACT_NONE, ln, tj, cnt, row_grid(cnt), st);
    }
    for (int j = 0; j < n && e == hipSuccess; ++j) {
      const RowTile* tj = tl + hp.soc_piece_first[j];
      const int32_t cnt = hp.soc_piece_count[j];
      e = pointwise_launch(hp.dt, hp.act, act, tj, cnt, row_grid(cnt), st);
    }
    if (e == hipSuccess) {
      const int32_t T = hp.soc_piece_tiles_total;
      e = pointwise_launch(hp.dt, OPTIMUS_ACT_NONE, cat, tl, T, row_grid(T), st);
    }
  }
  return e == hipSuccess ? OPTIMUS_OK : hip_fail(e, "execute: split-op-cat unfused launch");
}

extern "C" optimus_status optimus_plan_execute(optimus_plan p, optimus_stream_t stream) {
  return optimus_plan_execute_mode(p, OPTIMUS_EXEC_GROUPED, stream);
}

extern "C" optimus_status optimus_plan_get_info(optimus_plan p, optimus_plan_info* out) {
  if (!p || !out) return fail(OPTIMUS_ERR_INVALID_ARG, "plan_get_info: NULL argument");
  const HostPlan& hp = p->hp;
  out->kind = hp.kind == KIND_LINEAR && hp.g_ln ? 4 : (int32_t)hp.kind;
  out->group_size = hp.G;
  out->launches = hp.G ? hp.launches : 0;
  out->chain_launches = hp.chain_launches;
  out->work_items = hp.work_items;
  out->grid = hp.grid;
  out->block = hp.block;
  out->flops = hp.flops;
  out->bytes = hp.bytes;
  out->kernel = hp.kernel.c_str();
  return OPTIMUS_OK;
}

// ===================================================================== one-shot entry points
// The table goes up through a pinned staging buffer (per thread, grow-only)
// into stream-ordered device memory, the group is launched, and the device
// memory is released in stream order; the call does not wait for the GPU.
namespace {
struct Staging {
  void* host = nullptr;
  size_t cap = 0;
  hipEvent_t ev = nullptr;
  bool pending = false;
};
thread_local Staging* tl_stage = nullptr;  // intentionally never freed (process lifetime)
}  // namespace

static optimus_status run_oneshot(HostPlan& hp, hipStream_t stream) {
  if (hp.G == 0) return OPTIMUS_OK;
  if (!tl_stage) tl_stage = new Staging();
  Staging& sg = *tl_stage;
  const size_t n = std::max<size_t>(hp.blob.bytes.size(), 256);
  // host-side steps first: nothing on the device exists yet if one fails
  if (!sg.ev) HIP_TRY(hipEventCreateWithFlags(&sg.ev, hipEventDisableTiming), "one-shot: event");
  if (sg.pending) HIP_TRY(hipEventSynchronize(sg.ev), "one-shot: staging reuse");
  sg.pending = false;
  if (sg.cap < n) {
    if (sg.host) (void)hipHostFree(sg.host);
    sg.host = nullptr;
    sg.cap = 0;
    HIP_TRY(hipHostMalloc(&sg.host, n, hipHostMallocDefault), "one-shot: pinned staging");
    sg.cap = n;
  }
  // then the stream-ordered device memory, released in stream order on every path
  char* table = nullptr;
  char* scratch = nullptr;
  auto release = [&]() {
    if (table) (void)hipFreeAsync(table, stream);
    if (scratch) (void)hipFreeAsync(scratch, stream);
  };
  hipError_t e = hipMallocAsync((void**)&table, n, stream);
  if (e != hipSuccess) return hip_fail(e, "one-shot: device table");
  if (hp.scratch_bytes) {
    e = hipMallocAsync((void**)&scratch, hp.scratch_bytes, stream);
    if (e != hipSuccess) {
      scratch = nullptr;
      release();
      return hip_fail(e, "one-shot: scratch");
    }
  }
  rebase_soc(hp, table);
  rebase_fixups(hp, table, scratch);
  memcpy(sg.host, hp.blob.bytes.data(), hp.blob.bytes.size());
  e = hipMemcpyAsync(table, sg.host, hp.blob.bytes.size(), hipMemcpyHostToDevice, stream);
  if (e == hipSuccess) {
    e = hipEventRecord(sg.ev, stream);
    // the staging buffer may be in use until the event has passed
    sg.pending = true;
  }
  if (e != hipSuccess) {
    release();
    return hip_fail(e, "one-shot: upload");
  }
  e = launch_grouped(hp, table, stream);
  release();
  return e == hipSuccess ? OPTIMUS_OK : hip_fail(e, "one-shot: launch");
}

extern "C" optimus_status optimus_grouped_linear(const optimus_linear_desc* d, int32_t G, optimus_dtype dt,
                                                 optimus_act epilogue, optimus_stream_t stream) {
  HostPlan hp;
  optimus_status st = build_linear(d, G, dt, epilogue, hp);
  return st != OPTIMUS_OK ? st : run_oneshot(hp, (hipStream_t)stream);
}
extern "C" optimus_status optimus_grouped_linear_layernorm(const optimus_linear_desc* d, const void* const* gamma,
                                                           const void* const* beta, int32_t G, optimus_dtype dt,
                                                           float eps, optimus_act epilogue, optimus_stream_t stream) {
  HostPlan hp;
  optimus_status st = build_linear(d, G, dt, epilogue, hp, true, gamma, beta, eps);
  return st != OPTIMUS_OK ? st : run_oneshot(hp, (hipStream_t)stream);
}
extern "C" optimus_status optimus_grouped_layernorm(const optimus_layernorm_desc* d, int32_t G, optimus_dtype dt,
                                                    optimus_act epilogue, optimus_stream_t stream) {
  HostPlan hp;
  optimus_status st = build_layernorm(d, G, dt, epilogue, hp);
  return st != OPTIMUS_OK ? st : run_oneshot(hp, (hipStream_t)stream);
}
extern "C" optimus_status optimus_grouped_pointwise(const optimus_pointwise_desc* d, int32_t G, optimus_dtype dt,
                                                    optimus_act op, optimus_stream_t stream) {
  HostPlan hp;
  optimus_status st = build_pointwise(d, G, dt, op, hp);
  return st != OPTIMUS_OK ? st : run_oneshot(hp, (hipStream_t)stream);
}
extern "C" optimus_status optimus_split_op_cat(const optimus_split_op_cat_desc* d, optimus_dtype dt,
                                               optimus_stream_t stream) {
  HostPlan hp;
  optimus_status st = build_split_op_cat(d, dt, hp);
  return st != OPTIMUS_OK ? st : run_oneshot(hp, (hipStream_t)stream);
}
extern "C" optimus_status optimus_grouped_linear_backward(const optimus_linear_grad_desc* d, int32_t G,
                                                          optimus_dtype dt, optimus_stream_t stream) {
  HostPlan hp;
  optimus_status st = build_linear_backward(d, G, dt, hp);
  return st != OPTIMUS_OK ? st : run_oneshot(hp, (hipStream_t)stream);
}
extern "C" optimus_status optimus_grouped_layernorm_backward(const optimus_layernorm_grad_desc* d, int32_t G,
                                                             optimus_dtype dt, optimus_stream_t stream) {
  HostPlan hp;
  optimus_status st = build_layernorm_backward(d, G, dt, hp);
  return st != OPTIMUS_OK ? st : run_oneshot(hp, (hipStream_t)stream);
}
extern "C" optimus_status optimus_grouped_linear_act_backward(const optimus_linear_grad_desc* d,
                                                              const void* const* act_x, const int64_t* ld_act_x,
                                                              int32_t G, optimus_dtype dt, optimus_act act,
                                                              optimus_stream_t stream) {
  HostPlan hp;
  optimus_status st = build_linear_backward(d, G, dt, hp, act, act_x, ld_act_x);
  return st != OPTIMUS_OK ? st : run_oneshot(hp, (hipStream_t)stream);
}
extern "C" optimus_status optimus_grouped_layernorm_act_backward(const optimus_layernorm_grad_desc* d,
                                                                 const void* const* beta, int32_t G, optimus_dtype dt,
                                                                 optimus_act act, optimus_stream_t stream) {
  HostPlan hp;
  optimus_status st = build_layernorm_backward(d, G, dt, hp, beta, act);
  return st != OPTIMUS_OK ? st : run_oneshot(hp, (hipStream_t)stream);
}
extern "C" optimus_status optimus_grouped_act_backward(const optimus_act_grad_desc* d, int32_t G, optimus_dtype dt,
                                                       optimus_act act, optimus_stream_t stream) {
  HostPlan hp;
  optimus_status st = build_act_backward(d, G, dt, act, hp);
  return st != OPTIMUS_OK ? st : run_oneshot(hp, (hipStream_t)stream);
}
extern "C" optimus_status optimus_grouped_quantize_fp8(const optimus_fp8_quant_desc* d, int32_t G, optimus_dtype dt,
                                                       int32_t use_scaling, optimus_stream_t stream) {
  HostPlan hp;
  optimus_status st = build_quantize_fp8(d, G, dt, use_scaling, hp);
  return st != OPTIMUS_OK ? st : run_oneshot(hp, (hipStream_t)stream);
}
// ===================================================================== no-allocation entry point
// The table (and any plan scratch after it) of a call that may not allocate
// lives in this array: one copy per GPU, for the life of the process. Host
// code never passes the array's name to a kernel; it uses the device address
// hipGetSymbolAddress returns, looked up once per device with that device
// current.
static __device__ __align__(256) char scratch[OPTIMUS_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

static optimus_status noalloc_scratch(char** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev), "noalloc: current device");
  if (dev < 0 || dev >= kMaxDevices) return fail(OPTIMUS_ERR_UNSUPPORTED, "noalloc: device %d out of range", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "noalloc: scratch address");
    if (!p) return fail(OPTIMUS_ERR_HIP, "noalloc: scratch address is NULL");
    g_scratch_ptr[dev] = (char*)p;
  }
  *out = g_scratch_ptr[dev];
  return OPTIMUS_OK;
}

// One grouped execution with the table, then the plan scratch, in the
// static array: no device or pinned allocation. The blob is host memory the
// copy reads before the enqueue returns (pageable source).
static optimus_status run_noalloc(HostPlan& hp, hipStream_t stream, const char* what) {
  if (hp.G == 0) return OPTIMUS_OK;
  const size_t table = (std::max<size_t>(hp.blob.bytes.size(), 256) + 255) & ~(size_t)255;
  const size_t need = table + hp.scratch_bytes;
  if (need > (size_t)OPTIMUS_NOALLOC_SCRATCH_BYTES)
    return fail(OPTIMUS_ERR_UNSUPPORTED, "%s: the group needs %zu bytes of scratch, above the %u-byte limit", what,
                need, (unsigned)OPTIMUS_NOALLOC_SCRATCH_BYTES);
  char* base = nullptr;
  optimus_status st = noalloc_scratch(&base);
  if (st != OPTIMUS_OK) return st;
  rebase_soc(hp, base);
  rebase_fixups(hp, base, hp.scratch_bytes ? base + table : nullptr);
  HIP_TRY(hipMemcpyAsync(base, hp.blob.bytes.data(), hp.blob.bytes.size(), hipMemcpyHostToDevice, stream),
          "noalloc: table upload");
  hipError_t e = launch_grouped(hp, base, stream);
  return e == hipSuccess ? OPTIMUS_OK : hip_fail(e, "noalloc: launch");
}

extern "C" optimus_status optimus_grouped_quantize_fp8_noalloc(const optimus_fp8_quant_desc* d, int32_t G,
                                                               optimus_dtype dt, int32_t use_scaling,
                                                               optimus_stream_t stream) {
  HostPlan hp;
  optimus_status st = build_quantize_fp8(d, G, dt, use_scaling, hp);
  return st != OPTIMUS_OK ? st : run_noalloc(hp, (hipStream_t)stream, "grouped_quantize_fp8_noalloc");
}

extern "C" optimus_status optimus_grouped_dequantize_fp8(const optimus_fp8_dequant_desc* d, int32_t G,
                                                         optimus_dtype dt, optimus_stream_t stream) {
  HostPlan hp;
  optimus_status st = build_dequantize_fp8(d, G, dt, hp);
  return st != OPTIMUS_OK ? st : run_oneshot(hp, (hipStream_t)stream);
}
