// Drives the library's host-only descriptor validation (the checks every
// entry point runs before it launches) through valid groups, every class of
// invalid descriptor, aliasing and exact in-place members, G = 0 and a large
// group. Built with AddressSanitizer and UndefinedBehaviorSanitizer on the
// host side by tests/test_validate_sanitized.py. The pointers are host
// addresses standing in for device ones: validation compares addresses and
// extents only and never dereferences a member pointer.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "optimus.h"

static int failures = 0;
static void expect(optimus_status got, optimus_status want, const char* what) {
  if (got != want) {
    std::fprintf(stderr, "FAILED %s: status %d, expected %d (%s)\n", what, (int)got, (int)want, optimus_last_error());
    ++failures;
  } else if (got != OPTIMUS_OK && std::strlen(optimus_last_error()) == 0) {
    std::fprintf(stderr, "FAILED %s: no message for status %d\n", what, (int)got);
    ++failures;
  }
}

int main() {
  static char arena[1 << 24];  // 16 MiB of distinct addresses
  auto at = [&](size_t off) { return (void*)(arena + off); };
  const optimus_dtype BF = OPTIMUS_BF16, F32 = OPTIMUS_F32;
  const optimus_act NONE = OPTIMUS_ACT_NONE, TANH = OPTIMUS_ACT_TANH;

  // ---- Linear (and the fused Linear + LayerNorm)
  optimus_linear_desc L[3] = {
      {at(0), 64, at(1 << 16), 64, at(2 << 16), at(3 << 16), 32, 100, 32, 64},
      {at(4 << 16), 40, at(5 << 16), 40, nullptr, at(6 << 16), 24, 7, 24, 40},
      {at(7 << 16), 16, at(8 << 16), 16, at(9 << 16), at(10 << 16), 8, 1, 8, 16}};
  expect(optimus_validate_linear(L, 3, BF, TANH), OPTIMUS_OK, "linear ok");
  expect(optimus_validate_linear(L, 0, BF, TANH), OPTIMUS_OK, "linear G = 0");
  expect(optimus_validate_linear(L, -1, BF, TANH), OPTIMUS_ERR_INVALID_ARG, "linear G < 0");
  expect(optimus_validate_linear(nullptr, 2, BF, TANH), OPTIMUS_ERR_INVALID_ARG, "linear null descriptors");
  expect(optimus_validate_linear(L, 3, (optimus_dtype)7, TANH), OPTIMUS_ERR_UNSUPPORTED, "linear dtype");
  expect(optimus_validate_linear(L, 3, BF, (optimus_act)9), OPTIMUS_ERR_UNSUPPORTED, "linear activation");
  {
    optimus_linear_desc b[3];
    std::memcpy(b, L, sizeof b);
    b[1].x = nullptr;
    expect(optimus_validate_linear(b, 3, BF, NONE), OPTIMUS_ERR_INVALID_ARG, "linear null x");
    std::memcpy(b, L, sizeof b);
    b[0].ldx = 63;
    expect(optimus_validate_linear(b, 3, BF, NONE), OPTIMUS_ERR_INVALID_ARG, "linear ldx < K");
    std::memcpy(b, L, sizeof b);
    b[2].M = 0;
    expect(optimus_validate_linear(b, 3, BF, NONE), OPTIMUS_ERR_INVALID_ARG, "linear M = 0");
    std::memcpy(b, L, sizeof b);
    b[2].M = (int64_t)1 << 40;
    expect(optimus_validate_linear(b, 3, BF, NONE), OPTIMUS_ERR_INVALID_ARG, "linear M too large");
    std::memcpy(b, L, sizeof b);
    b[1].y = const_cast<void*>(b[0].x);  // an output over another member's input
    expect(optimus_validate_linear(b, 3, BF, NONE), OPTIMUS_ERR_ALIASING, "linear output over input");
    std::memcpy(b, L, sizeof b);
    b[2].y = (char*)b[0].y + 100;  // two outputs overlapping
    expect(optimus_validate_linear(b, 3, F32, NONE), OPTIMUS_ERR_ALIASING, "linear outputs overlap");
  }
  const void* gam[3] = {at(11 << 16), nullptr, at(12 << 16)};
  const void* bet[3] = {nullptr, at(13 << 16), at(14 << 16)};
  expect(optimus_validate_linear_layernorm(L, gam, bet, 3, BF, 1e-5f, TANH), OPTIMUS_OK, "linear+ln ok");
  expect(optimus_validate_linear_layernorm(L, nullptr, nullptr, 3, F32, 1e-5f, NONE), OPTIMUS_OK, "linear+ln no affine");
  expect(optimus_validate_linear_layernorm(L, gam, bet, 3, BF, -1.f, TANH), OPTIMUS_ERR_INVALID_ARG, "linear+ln eps");

  // ---- LayerNorm, pointwise, activation backward
  optimus_layernorm_desc N[2] = {{at(0), 256, at(1 << 20), 256, at(2 << 20), nullptr, 10, 200, 1e-5f},
                                 {at(3 << 20), 64, at(3 << 20), 64, nullptr, nullptr, 33, 64, 1e-5f}};
  expect(optimus_validate_layernorm(N, 2, BF, NONE), OPTIMUS_OK, "layernorm ok (one in place)");
  {
    optimus_layernorm_desc b[2];
    std::memcpy(b, N, sizeof b);
    b[1].ldy = 65;  // in place with a different stride
    expect(optimus_validate_layernorm(b, 2, BF, NONE), OPTIMUS_ERR_ALIASING, "layernorm shifted in place");
    std::memcpy(b, N, sizeof b);
    b[0].cols = 0;
    expect(optimus_validate_layernorm(b, 2, BF, NONE), OPTIMUS_ERR_INVALID_ARG, "layernorm cols = 0");
  }
  optimus_pointwise_desc P[2] = {{at(0), 8, at(1 << 12), 8, 3, 5}, {at(2 << 12), 5, at(2 << 12), 5, 2, 5}};
  expect(optimus_validate_pointwise(P, 2, F32, TANH), OPTIMUS_OK, "pointwise ok");
  P[1].ldx = 4;
  expect(optimus_validate_pointwise(P, 2, F32, TANH), OPTIMUS_ERR_INVALID_ARG, "pointwise ldx < cols");
  optimus_act_grad_desc A[1] = {{at(0), 16, at(1 << 12), 16, at(2 << 12), 16, 4, 16}};
  expect(optimus_validate_act_backward(A, 1, BF, OPTIMUS_ACT_SILU), OPTIMUS_OK, "act backward ok");
  A[0].dx = (void*)A[0].x;  // exact in place
  expect(optimus_validate_act_backward(A, 1, BF, OPTIMUS_ACT_SILU), OPTIMUS_OK, "act backward in place");
  A[0].lddx = 20;
  expect(optimus_validate_act_backward(A, 1, BF, OPTIMUS_ACT_SILU), OPTIMUS_ERR_ALIASING, "act backward shifted");

  // ---- split-op-cat
  const int64_t widths[4] = {16, 8, 24, 16}, bad[4] = {16, 8, 24, 15};
  const void* sg[4] = {at(5 << 20), nullptr, at(6 << 20), nullptr};
  optimus_split_op_cat_desc S = {at(0), 64, at(1 << 20), 64, 100, 64, 4, widths, sg, nullptr, 1, 1e-5f, TANH};
  expect(optimus_validate_split_op_cat(&S, BF), OPTIMUS_OK, "split-op-cat ok");
  S.out = (void*)S.in;
  expect(optimus_validate_split_op_cat(&S, BF), OPTIMUS_OK, "split-op-cat in place");
  S.ldout = 72;
  expect(optimus_validate_split_op_cat(&S, BF), OPTIMUS_ERR_ALIASING, "split-op-cat shifted in place");
  S.out = at(1 << 20), S.ldout = 64, S.widths = bad;
  expect(optimus_validate_split_op_cat(&S, BF), OPTIMUS_ERR_INVALID_ARG, "split-op-cat widths");
  S.widths = nullptr;
  expect(optimus_validate_split_op_cat(&S, BF), OPTIMUS_ERR_INVALID_ARG, "split-op-cat null widths");
  expect(optimus_validate_split_op_cat(nullptr, BF), OPTIMUS_ERR_INVALID_ARG, "split-op-cat null descriptor");

  // ---- backward
  optimus_linear_grad_desc G[1] = {{at(0), 32, at(1 << 16), 32, at(2 << 16), 16, at(3 << 16), 32, at(4 << 16), 32,
                                    at(5 << 16), 50, 16, 32}};
  expect(optimus_validate_linear_backward(G, 1, BF), OPTIMUS_OK, "linear backward ok");
  G[0].dw = nullptr;  // db needs dw
  expect(optimus_validate_linear_backward(G, 1, BF), OPTIMUS_ERR_UNSUPPORTED, "linear backward db without dw");
  optimus_layernorm_grad_desc NG[1] = {{at(0), 40, nullptr, at(1 << 16), 40, at(2 << 16), 40, at(3 << 16),
                                        at(4 << 16), 9, 40, 1e-5f}};
  expect(optimus_validate_layernorm_backward(NG, 1, F32), OPTIMUS_OK, "layernorm backward ok");
  NG[0].dgamma = NG[0].dx;
  expect(optimus_validate_layernorm_backward(NG, 1, F32), OPTIMUS_ERR_ALIASING, "layernorm backward dgamma over dx");

  // ---- fp8 codec
  optimus_fp8_quant_desc Q[2] = {{at(0), 24, at(1 << 16), 24, (float*)at(2 << 16), 5, 24},
                                 {at(3 << 16), 8, at(4 << 16), 8, (float*)at((2 << 16) + 64), 3, 8}};
  expect(optimus_validate_quantize_fp8(Q, 2, BF, 1), OPTIMUS_OK, "quantize ok");
  Q[1].q = (void*)Q[1].x;  // never in place
  expect(optimus_validate_quantize_fp8(Q, 2, BF, 1), OPTIMUS_ERR_ALIASING, "quantize in place");
  Q[1].q = at(4 << 16);
  Q[0].scale = nullptr;
  expect(optimus_validate_quantize_fp8(Q, 2, BF, 1), OPTIMUS_ERR_INVALID_ARG, "scaled quantize without scale");
  expect(optimus_validate_quantize_fp8(Q, 2, BF, 0), OPTIMUS_OK, "unscaled quantize without scale");
  optimus_fp8_dequant_desc DQ[1] = {{at(0), 24, nullptr, at(1 << 16), 24, 5, 24}};
  expect(optimus_validate_dequantize_fp8(DQ, 1, F32), OPTIMUS_OK, "dequantize ok");

  // ---- a large group: many small disjoint members, then one overlap at the end
  {
    const int n = 20000;
    std::vector<optimus_pointwise_desc> big(n);
    for (int i = 0; i < n; ++i)
      big[i] = optimus_pointwise_desc{at((size_t)i * 256), 8, at((size_t)(n + i) * 256), 8, 4, 8};
    expect(optimus_validate_pointwise(big.data(), n, BF, NONE), OPTIMUS_OK, "large group ok");
    big[n - 1].y = at(256);
    expect(optimus_validate_pointwise(big.data(), n, BF, NONE), OPTIMUS_ERR_ALIASING, "large group overlap");
  }
  if (std::strlen(optimus_version()) == 0) ++failures;
  if (failures) return 1;
  std::printf("validation under sanitizers: ok\n");
  return 0;
}
