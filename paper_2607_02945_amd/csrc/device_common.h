// Device helpers shared by the liboptimus kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "optimus_internal.h"

namespace optimus {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

struct bf16_t {
  uint16_t bits;
};

#define OPTIMUS_GLOBAL __attribute__((address_space(1)))

// ------------------------------------------------------------------ conversions
__device__ __forceinline__ float bf16_lo(uint32_t u) { return __builtin_bit_cast(float, u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __builtin_bit_cast(float, u & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __builtin_bit_cast(float, (uint32_t)b << 16); }

// Two fp32 values to a packed pair of bf16, round to nearest even (gfx950 has
// a native packed conversion for this).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float a) { return __builtin_bit_cast(uint16_t, (__bf16)a); }

// Storage-type traits: a 16-byte chunk holds VEC elements.
template <typename T>
struct Elem;
template <>
struct Elem<float> {
  static constexpr int VEC = 4;
  // Whole-vector bit casts only: hipcc (clang 22) miscompiles a bit cast
  // applied to a single element of an ext_vector_type value (it reads
  // element 0 whatever the index).
  __device__ static __forceinline__ void unpack(const u32x4& c, float* v) {
    const f32x4 f = __builtin_bit_cast(f32x4, c);
    v[0] = f[0];
    v[1] = f[1];
    v[2] = f[2];
    v[3] = f[3];
  }
  __device__ static __forceinline__ u32x4 pack(const float* v) {
    const f32x4 f = {v[0], v[1], v[2], v[3]};
    return __builtin_bit_cast(u32x4, f);
  }
  __device__ static __forceinline__ float load1(const void* p, int64_t i) { return ((const OPTIMUS_GLOBAL float*)p)[i]; }
  __device__ static __forceinline__ void store1(void* p, int64_t i, float v) { ((OPTIMUS_GLOBAL float*)p)[i] = v; }
};
template <>
struct Elem<bf16_t> {
  static constexpr int VEC = 8;
  __device__ static __forceinline__ void unpack(const u32x4& c, float* v) {
    v[0] = bf16_lo(c.x); v[1] = bf16_hi(c.x);
    v[2] = bf16_lo(c.y); v[3] = bf16_hi(c.y);
    v[4] = bf16_lo(c.z); v[5] = bf16_hi(c.z);
    v[6] = bf16_lo(c.w); v[7] = bf16_hi(c.w);
  }
  __device__ static __forceinline__ u32x4 pack(const float* v) {
    u32x4 c;
    c.x = pack_bf16x2(v[0], v[1]);
    c.y = pack_bf16x2(v[2], v[3]);
    c.z = pack_bf16x2(v[4], v[5]);
    c.w = pack_bf16x2(v[6], v[7]);
    return c;
  }
  __device__ static __forceinline__ float load1(const void* p, int64_t i) {
    return bf16_to_f32(((const OPTIMUS_GLOBAL uint16_t*)p)[i]);
  }
  __device__ static __forceinline__ void store1(void* p, int64_t i, float v) {
    ((OPTIMUS_GLOBAL uint16_t*)p)[i] = f32_to_bf16(v);
  }
};

// Sum of the values of one 16-byte chunk in fp32. bf16: four v_dot2 with
// (1, 1) on the packed pairs (products by 1 are exact), no unpacking.
template <typename T>
__device__ __forceinline__ float chunk_sum(const u32x4& c);
template <>
__device__ __forceinline__ float chunk_sum<bf16_t>(const u32x4& c) {
  const bf16x8 v = __builtin_bit_cast(bf16x8, c);
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
  float a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 0, 1), one, 0.f, false);
  a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 2, 3), one, a, false);
  a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 4, 5), one, a, false);
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 6, 7), one, a, false);
}
template <>
__device__ __forceinline__ float chunk_sum<float>(const u32x4& c) {
  const f32x4 f = __builtin_bit_cast(f32x4, c);
  return (f[0] + f[1]) + (f[2] + f[3]);
}

// Sum of the squares of one chunk's values in fp32 (bf16: v_dot2 of each
// packed pair with itself; the products of two bf16 values are exact in fp32).
template <typename T>
__device__ __forceinline__ float chunk_sumsq(const u32x4& c);
template <>
__device__ __forceinline__ float chunk_sumsq<bf16_t>(const u32x4& c) {
  const bf16x8 v = __builtin_bit_cast(bf16x8, c);
  const bf16x2 p0 = __builtin_shufflevector(v, v, 0, 1), p1 = __builtin_shufflevector(v, v, 2, 3);
  const bf16x2 p2 = __builtin_shufflevector(v, v, 4, 5), p3 = __builtin_shufflevector(v, v, 6, 7);
  float a = __builtin_amdgcn_fdot2_f32_bf16(p0, p0, 0.f, false);
  a = __builtin_amdgcn_fdot2_f32_bf16(p1, p1, a, false);
  a = __builtin_amdgcn_fdot2_f32_bf16(p2, p2, a, false);
  return __builtin_amdgcn_fdot2_f32_bf16(p3, p3, a, false);
}
template <>
__device__ __forceinline__ float chunk_sumsq<float>(const u32x4& c) {
  const f32x4 f = __builtin_bit_cast(f32x4, c);
  return __builtin_fmaf(f[0], f[0], f[1] * f[1]) + __builtin_fmaf(f[2], f[2], f[3] * f[3]);
}

// ------------------------------------------------------------------ activations
// exp via the hardware base-2 exponential; reciprocal via the hardware
// approximate reciprocal (1 ulp). Large |x| saturates correctly: e^x -> inf
// gives 1/inf = 0.
__device__ __forceinline__ float fast_exp(float x) { return __builtin_amdgcn_exp2f(x * 1.4426950408889634f); }
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

template <int ACT>
__device__ __forceinline__ float act_apply(float x) {
  if constexpr (ACT == OPTIMUS_ACT_RELU) {
    return x > 0.f ? x : 0.f;
  } else if constexpr (ACT == OPTIMUS_ACT_SIGMOID) {
    return fast_rcp(1.f + fast_exp(-x));
  } else if constexpr (ACT == OPTIMUS_ACT_TANH) {
    // tanh x = 1 - 2 / (e^{2x} + 1)
    return 1.f - 2.f * fast_rcp(fast_exp(2.f * x) + 1.f);
  } else if constexpr (ACT == OPTIMUS_ACT_SILU) {
    return x * fast_rcp(1.f + fast_exp(-x));
  } else {
    return x;
  }
}

// The activations whose exponent argument is a fixed multiple of the input
// (sigmoid and silu: 2^(-x log2 e); tanh: 2^(2 x log2 e)) can take that
// product directly: act_in_scale is the multiple (1 for the others) and
// act_scaled_in(u) = act_apply(u / act_in_scale). For silu,
// x / (1 + e^-x) = u / ((1 + 2^u) * (-log2 e)) with u = -x log2 e, so the
// scale goes into the denominator's fma.
template <int ACT>
__device__ __forceinline__ constexpr float act_in_scale() {
  return ACT == OPTIMUS_ACT_SIGMOID || ACT == OPTIMUS_ACT_SILU ? -1.4426950408889634f
         : ACT == OPTIMUS_ACT_TANH                            ? 2.8853900817779268f
                                                              : 1.f;
}
template <int ACT>
__device__ __forceinline__ float act_scaled_in(float u) {
  if constexpr (ACT == OPTIMUS_ACT_SIGMOID) {
    return fast_rcp(1.f + __builtin_amdgcn_exp2f(u));
  } else if constexpr (ACT == OPTIMUS_ACT_TANH) {
    return 1.f - 2.f * fast_rcp(__builtin_amdgcn_exp2f(u) + 1.f);
  } else if constexpr (ACT == OPTIMUS_ACT_SILU) {
    return u * fast_rcp(__builtin_fmaf(__builtin_amdgcn_exp2f(u), -1.4426950408889634f, -1.4426950408889634f));
  } else {
    return act_apply<ACT>(u);
  }
}

// d[e] = x[e] - m for the values of one chunk, in fp32.
template <typename T>
__device__ __forceinline__ void centred(const u32x4& c, float m, float* d);
template <>
__device__ __forceinline__ void centred<bf16_t>(const u32x4& c, float m, float* d) {
  Elem<bf16_t>::unpack(c, d);
#pragma unroll
  for (int e = 0; e < 8; ++e) d[e] -= m;
}
template <>
__device__ __forceinline__ void centred<float>(const u32x4& c, float m, float* d) {
  const f32x4 f = __builtin_bit_cast(f32x4, c);
  d[0] = f[0] - m;
  d[1] = f[1] - m;
  d[2] = f[2] - m;
  d[3] = f[3] - m;
}

// Derivative of one activation at its input, in the same hardware
// exponential / reciprocal forms as the forward activations.
template <int ACT>
__device__ __forceinline__ float act_grad(float x) {
  if constexpr (ACT == OPTIMUS_ACT_RELU) {
    return x > 0.f ? 1.f : 0.f;
  } else if constexpr (ACT == OPTIMUS_ACT_SIGMOID) {
    const float s = fast_rcp(1.f + fast_exp(-x));
    return s * (1.f - s);
  } else if constexpr (ACT == OPTIMUS_ACT_TANH) {
    const float t = 1.f - 2.f * fast_rcp(fast_exp(2.f * x) + 1.f);
    return 1.f - t * t;
  } else if constexpr (ACT == OPTIMUS_ACT_SILU) {
    const float s = fast_rcp(1.f + fast_exp(-x));
    return s + x * s * (1.f - s);
  } else {
    return 1.f;
  }
}

// ------------------------------------------------------------------ memory
// Every tensor access goes through these helpers, which name the global
// address space: pointers read from a descriptor table are otherwise generic,
// and generic (flat) accesses also count against the LDS wait counter, which
// would make every LDS wait drain the in-flight global loads too.
__device__ __forceinline__ u32x4 ld16(const void* p) { return *(const OPTIMUS_GLOBAL u32x4*)p; }
__device__ __forceinline__ void st16(void* p, const u32x4& v) { *(OPTIMUS_GLOBAL u32x4*)p = v; }
// Streaming variants: data touched once (nontemporal hint).
__device__ __forceinline__ u32x4 ld16_nt(const void* p) {
  return __builtin_nontemporal_load((const OPTIMUS_GLOBAL u32x4*)p);
}
__device__ __forceinline__ void st16_nt(void* p, const u32x4& v) {
  __builtin_nontemporal_store(v, (OPTIMUS_GLOBAL u32x4*)p);
}

// ------------------------------------------------------------------ lane reductions
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float swz_xor16(float v) {
  // ds_swizzle bit mode: and_mask 0x1f, or_mask 0, xor_mask 0x10 (within 32 lanes)
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x401F));
}

// Sum over aligned groups of L consecutive lanes (L a power of two <= 64,
// wave-uniform); every lane of a group receives the group's sum.
__device__ __forceinline__ float group_sum(float v, int L) {
  if (L > 1) v += dpp_f<0xB1>(v);    // quad_perm [1,0,3,2]: lane ^ 1
  if (L > 2) v += dpp_f<0x4E>(v);    // quad_perm [2,3,0,1]: lane ^ 2
  if (L > 4) v += dpp_f<0x141>(v);   // row_half_mirror: pairs the two quads of 8
  if (L > 8) v += dpp_f<0x140>(v);   // row_mirror: pairs the two halves of 16
  if (L > 16) v += swz_xor16(v);     // lane ^ 16
  if (L > 32) {
    float a = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
    float b = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
    v = a + b;
  }
  return v;
}

__device__ __forceinline__ void lds_wave_sync() {
  // Complete this wave's LDS operations and keep the compiler from moving
  // memory accesses across this point.
  __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_wave_barrier();
}

}  // namespace optimus
