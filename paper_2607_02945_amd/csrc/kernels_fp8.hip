// FP8 activation codec of liboptimus for gfx950: grouped quantize of saved
// activations to OCP E4M3 codes (one byte each), with or without a
// per-tensor scale, and grouped dequantize back to the storage dtype (paper
// Sec. 5, peak memory usage reduction; appendix Sec. 8.2, activation
// quantization: forward saves in FP8, backward restores before use).
//
// Arithmetic, per member:
//   scaled    amax = max |x| (NaN skipped), scale = amax / 448, inv = 448 / amax
//             (both 1 when amax is 0), code = E4M3(fp32(x * inv)) saturated to +-448
//   unscaled  code = E4M3(x); magnitudes above 464 give the NaN code
//   NaN       a NaN value gives the NaN code S.1111.111 with the sign of x
//   decode    y = fp32(value(code) * scale), rounded to the storage dtype
// The conversions are gfx950's v_cvt_pk_fp8_f32 (round to nearest even; the
// overflow tie 464 goes to 448, larger magnitudes and infinities to the NaN
// code) and v_cvt_pk_f32_fp8 (exact).
//
// Scaled quantize is two launches per group, whatever G is:
//   amax     every member in tiles of at most 1/256 of it (and at least
//            128 KB): each tile's max |x| (and whether it holds a NaN) goes to
//            the tile's own slot -- one writer per slot, no atomics
//   convert  tiles of 32 KB: a tile reduces its member's slots (a few hundred
//            bytes, cached), derives scale and inv, converts and stores
// x is read twice. A single launch would need workgroups to wait for other
// workgroups' amax tiles; handing work out through a global counter, the one
// schedule whose waits provably end, costs a same-address device atomic per
// tile, and those serialize at about 12 ns each on this GPU -- more than the
// second pass. Both passes stream (nontemporal loads): the memory-side cache
// gives too little on a re-read for the amax pass to leave x in it.
#include <type_traits>

#include "device_common.h"

namespace optimus {

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Block barrier that orders LDS only: global loads in flight stay in flight.
__device__ __forceinline__ void lds_barrier() {
  __asm__ volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Max over the 64 lanes of a wave (unsigned).
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false));   // lane ^ 1
  v = max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false));   // lane ^ 2
  v = max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x141, 0xF, 0xF, false));  // half-row mirror
  v = max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x140, 0xF, 0xF, false));  // row mirror
  v = max(v, (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x401F));              // lane ^ 16
  const uint32_t a = (uint32_t)__builtin_amdgcn_readlane((int)v, 0);
  const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)v, 32);
  return max(a, b);
}

// ------------------------------------------------------------------ E4M3 conversion
// Four fp32 values to four codes (value i in byte i), hardware rounding.
__device__ __forceinline__ uint32_t cvt4(float a, float b, float c, float d) {
  const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(c, d, lo, true);
}

// One value, exact rules for NaN and saturation: v is the (scaled) value,
// xbits the fp32 bits of the input element (for the sign of a NaN code).
template <bool SAT>
__device__ __forceinline__ uint32_t encode1(float v, uint32_t xbits) {
  if (v != v) return (xbits >> 31) ? 0xFFu : 0x7Fu;
  if (SAT) v = __builtin_amdgcn_fmed3f(v, -448.0f, 448.0f);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(v, 0.0f, 0, false) & 0xFFu;
}

// ------------------------------------------------------------------ tile walk
// A work item covers rows [row0, row0 + nrows) and chunk columns [c0, c1) of
// one member. L lanes (a power of two up to the 256 of the block) share a row:
// thread t takes row slot t / L and chunk column li = t % L; with L = 256 a
// row's chunks are strided by 256. Chunks are visited U at a time so that U
// loads per lane are in flight; `body(r, c, ok)` gets U (row, chunk) pairs.
constexpr int kFp8Threads = 256;
#ifndef OPTIMUS_FP8_U
#define OPTIMUS_FP8_U 4
#endif
constexpr int kFp8U = OPTIMUS_FP8_U;
// Load policy of the two passes over x (1: nontemporal, streaming).
#ifndef OPTIMUS_FP8_AMAX_NT
#define OPTIMUS_FP8_AMAX_NT 1
#endif
#ifndef OPTIMUS_FP8_CONVERT_NT
#define OPTIMUS_FP8_CONVERT_NT 1
#endif

template <int U, class Body>
__device__ __forceinline__ void walk_tile(const Fp8Item& it, int L, int tid, Body&& body) {
  const int rpb = kFp8Threads / L;
  const int slot = tid / L, li = tid & (L - 1);
  const int end = it.row0 + it.nrows;
  const int cw = it.c1 - it.c0;
  int r[U], c[U];
  bool ok[U];
  if (cw <= L) {
    const int cc = it.c0 + li;
    const bool cok = li < cw;
    for (int rb = it.row0 + slot; rb < end; rb += U * rpb) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        r[u] = rb + u * rpb;
        c[u] = cc;
        ok[u] = cok && r[u] < end;
      }
      body(r, c, ok);
    }
  } else {
    for (int rr = it.row0 + slot; rr < end; rr += rpb) {
      for (int cb = it.c0 + li; cb < it.c1; cb += U * L) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          r[u] = rr;
          c[u] = cb + u * L;
          ok[u] = c[u] < it.c1;
        }
        body(r, c, ok);
      }
    }
  }
}

// Storage element traits for the codec. A vector chunk is 16 bytes of the
// wide side (VEC values), i.e. VEC codes.
template <typename T>
struct Fp8Side;
template <>
struct Fp8Side<bf16_t> {
  static constexpr int VEC = 8;
  typedef u32x2 Codes;
  __device__ static __forceinline__ uint32_t bits(const void* p, int64_t i) {
    return (uint32_t)((const OPTIMUS_GLOBAL uint16_t*)p)[i] << 16;
  }
};
template <>
struct Fp8Side<float> {
  static constexpr int VEC = 4;
  typedef uint32_t Codes;
  __device__ static __forceinline__ uint32_t bits(const void* p, int64_t i) {
    return ((const OPTIMUS_GLOBAL uint32_t*)p)[i];
  }
};

// max |x| bits of one vector chunk folded into the accumulator. bf16: the
// absolute values stay packed two to a register (packed 16-bit integer max);
// fp32: one integer max per value. A NaN shows as bits above the infinity's.
__device__ __forceinline__ void amax_chunk(u16x2& acc, const u32x4& v) {
  const uint32_t m = 0x7FFF7FFFu;
  u16x2 a = __builtin_bit_cast(u16x2, v.x & m), b = __builtin_bit_cast(u16x2, v.y & m);
  u16x2 c = __builtin_bit_cast(u16x2, v.z & m), d = __builtin_bit_cast(u16x2, v.w & m);
  acc = __builtin_elementwise_max(acc, __builtin_elementwise_max(__builtin_elementwise_max(a, b),
                                                                 __builtin_elementwise_max(c, d)));
}
__device__ __forceinline__ void amax_chunk(uint32_t& acc, const u32x4& v) {
  const uint32_t m = 0x7FFFFFFFu;
  acc = max(acc, max(max(v.x & m, v.y & m), max(v.z & m, v.w & m)));
}
__device__ __forceinline__ uint32_t amax_bits(const u16x2& acc) { return (uint32_t)max(acc.x, acc.y) << 16; }
__device__ __forceinline__ uint32_t amax_bits(uint32_t acc) { return acc; }

// Codes of one vector chunk, fast path (no NaN in the chunk, no saturation needed).
__device__ __forceinline__ u32x2 codes_fast(const u32x4& v, float inv, bf16_t*) {
  u32x2 o;
  o.x = cvt4(bf16_lo(v.x) * inv, bf16_hi(v.x) * inv, bf16_lo(v.y) * inv, bf16_hi(v.y) * inv);
  o.y = cvt4(bf16_lo(v.z) * inv, bf16_hi(v.z) * inv, bf16_lo(v.w) * inv, bf16_hi(v.w) * inv);
  return o;
}
__device__ __forceinline__ uint32_t codes_fast(const u32x4& v, float inv, float*) {
  const f32x4 f = __builtin_bit_cast(f32x4, v);
  return cvt4(f[0] * inv, f[1] * inv, f[2] * inv, f[3] * inv);
}
// Exact per-value rules (NaN sign, saturation).
template <bool SAT>
__device__ __forceinline__ u32x2 codes_exact(const u32x4& v, float inv, bf16_t*) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  uint32_t o[2] = {0u, 0u};
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t xb = (e & 1) ? (w[e >> 1] & 0xFFFF0000u) : (w[e >> 1] << 16);
    o[e >> 2] |= encode1<SAT>(__builtin_bit_cast(float, xb) * inv, xb) << (8 * (e & 3));
  }
  return u32x2{o[0], o[1]};
}
template <bool SAT>
__device__ __forceinline__ uint32_t codes_exact(const u32x4& v, float inv, float*) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  uint32_t o = 0u;
#pragma unroll
  for (int e = 0; e < 4; ++e) o |= encode1<SAT>(__builtin_bit_cast(float, w[e]) * inv, w[e]) << (8 * e);
  return o;
}
// Does a chunk hold a NaN?
__device__ __forceinline__ bool chunk_has_nan(const u32x4& v, bf16_t*) {
  u16x2 m = {0, 0};
  amax_chunk(m, v);
  return max(m.x, m.y) > 0x7F80;
}
__device__ __forceinline__ bool chunk_has_nan(const u32x4& v, float*) {
  uint32_t m = 0;
  amax_chunk(m, v);
  return m > 0x7F800000u;
}

__device__ __forceinline__ void st_codes(void* p, const u32x2& c) { __builtin_nontemporal_store(c, (OPTIMUS_GLOBAL u32x2*)p); }
__device__ __forceinline__ void st_codes(void* p, uint32_t c) { __builtin_nontemporal_store(c, (OPTIMUS_GLOBAL uint32_t*)p); }

// ------------------------------------------------------------------ amax of one tile
// Per-thread max |x| bits over the thread's share of the tile, NaN skipped;
// *nan is set when the share holds a NaN.
template <typename T>
__device__ __forceinline__ uint32_t tile_amax(const DevFp8& d, const Fp8Item& it, int tid, bool* nan) {
  constexpr int VEC = Fp8Side<T>::VEC;
  constexpr int U = kFp8U;
  const size_t s = sizeof(T);
  uint32_t m;
  if (d.lanes > 0) {
    typename std::conditional<sizeof(T) == 2, u16x2, uint32_t>::type acc{};
    walk_tile<U>(it, d.lanes, tid, [&](const int* r, const int* c, const bool* ok) {
      u32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u)
        v[u] = ok[u] ? (OPTIMUS_FP8_AMAX_NT ? ld16_nt : ld16)((const char*)d.x + ((int64_t)r[u] * d.ldx + (int64_t)c[u] * VEC) * s)
                     : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int u = 0; u < U; ++u) amax_chunk(acc, v[u]);
    });
    m = amax_bits(acc);
  } else {
    m = 0;
    walk_tile<U>(it, d.lanes_scalar, tid, [&](const int* r, const int* c, const bool* ok) {
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (ok[u]) m = max(m, Fp8Side<T>::bits(d.x, (int64_t)r[u] * d.ldx + c[u]) & 0x7FFFFFFFu);
    });
  }
  *nan = m > 0x7F800000u;
  if (*nan) {
    // Rare: walk the share again, one value at a time, skipping NaN.
    m = 0;
    const int64_t vec = d.lanes > 0 ? VEC : 1;
    const int L = d.lanes > 0 ? d.lanes : d.lanes_scalar;
    walk_tile<1>(it, L, tid, [&](const int* r, const int* c, const bool* ok) {
      if (!ok[0]) return;
      for (int e = 0; e < vec; ++e) {
        const uint32_t a = Fp8Side<T>::bits(d.x, (int64_t)r[0] * d.ldx + (int64_t)c[0] * vec + e) & 0x7FFFFFFFu;
        if (a <= 0x7F800000u) m = max(m, a);
      }
    });
  }
  return m;
}

// ------------------------------------------------------------------ convert one tile
// MODE 0: unscaled (per-chunk NaN check); 1: scaled, fast; 2: scaled, exact
// (the member holds a NaN or its amax is infinite).
template <typename T, int MODE>
__device__ __forceinline__ void tile_convert(const DevFp8& d, const Fp8Item& it, int tid, float inv) {
  constexpr int VEC = Fp8Side<T>::VEC;
  constexpr int U = kFp8U;
  constexpr bool SAT = MODE != 0;
  const size_t s = sizeof(T);
  if (d.lanes > 0) {
    walk_tile<U>(it, d.lanes, tid, [&](const int* r, const int* c, const bool* ok) {
      u32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u)
        v[u] = ok[u] ? (OPTIMUS_FP8_CONVERT_NT ? ld16_nt : ld16)((const char*)d.x + ((int64_t)r[u] * d.ldx + (int64_t)c[u] * VEC) * s)
                     : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (!ok[u]) continue;
        typename Fp8Side<T>::Codes q;
        if (MODE == 1)
          q = codes_fast(v[u], inv, (T*)nullptr);
        else if (MODE == 2)
          q = codes_exact<true>(v[u], inv, (T*)nullptr);
        else
          q = chunk_has_nan(v[u], (T*)nullptr) ? codes_exact<false>(v[u], 1.0f, (T*)nullptr)
                                                : codes_fast(v[u], 1.0f, (T*)nullptr);
        st_codes((char*)d.y + (int64_t)r[u] * d.ldy + (int64_t)c[u] * VEC, q);
      }
    });
  } else {
    walk_tile<U>(it, d.lanes_scalar, tid, [&](const int* r, const int* c, const bool* ok) {
      uint32_t xb[U];
#pragma unroll
      for (int u = 0; u < U; ++u) xb[u] = ok[u] ? Fp8Side<T>::bits(d.x, (int64_t)r[u] * d.ldx + c[u]) : 0u;
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (ok[u])
          ((OPTIMUS_GLOBAL uint8_t*)d.y)[(int64_t)r[u] * d.ldy + c[u]] =
              (uint8_t)encode1<SAT>(__builtin_bit_cast(float, xb[u]) * inv, xb[u]);
    });
  }
}

// ------------------------------------------------------------------ quantize kernels
// Unscaled: every item converts.
template <typename T>
__global__ __launch_bounds__(kFp8Threads) void grouped_quantize_fp8_kernel(const DevFp8* __restrict__ descs,
                                                                           const Fp8Item* __restrict__ items,
                                                                           int32_t num_items) {
  const int tid = threadIdx.x;
  for (int t = blockIdx.x; t < num_items; t += gridDim.x) {
    const Fp8Item it = items[t];
    tile_convert<T, 0>(descs[it.member], it, tid, 1.0f);
  }
}

// Scaled, first launch: per amax tile, (nan flag << 31 | max |x| bits) into
// slots[it.slot].
template <typename T>
__global__ __launch_bounds__(kFp8Threads) void grouped_fp8_amax_kernel(const DevFp8* __restrict__ descs,
                                                                       const Fp8Item* __restrict__ items,
                                                                       int32_t num_items, uint32_t* __restrict__ slots) {
  __shared__ uint32_t s_red[kFp8Threads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int t = blockIdx.x; t < num_items; t += gridDim.x) {
    const Fp8Item it = items[t];
    bool nan;
    const uint32_t m = tile_amax<T>(descs[it.member], it, tid, &nan);
    const uint32_t wm = wave_max_u32(m) | (wave_max_u32(nan ? 1u : 0u) << 31);
    if (lane == 0) s_red[wave] = wm;
    lds_barrier();
    if (tid == 0) {
      uint32_t a = 0, n = 0;
#pragma unroll
      for (int w = 0; w < kFp8Threads / 64; ++w) {
        a = max(a, s_red[w] & 0x7FFFFFFFu);
        n |= s_red[w] & 0x80000000u;
      }
      slots[it.slot] = n | a;
    }
    lds_barrier();  // s_red is reused by the next item
  }
}

// Scaled, second launch: every wave reduces the member's slots itself (no
// block barrier), then the tile is converted; the member's first tile also
// writes the scale.
template <typename T>
__global__ __launch_bounds__(kFp8Threads) void grouped_quantize_fp8_scaled_kernel(
    const DevFp8* __restrict__ descs, const Fp8Item* __restrict__ items, int32_t num_items,
    const uint32_t* __restrict__ slots) {
  const int tid = threadIdx.x, lane = tid & 63;
  for (int t = blockIdx.x; t < num_items; t += gridDim.x) {
    const Fp8Item it = items[t];
    const DevFp8 d = descs[it.member];
    uint32_t m = 0, nan = 0;
    for (int i = lane; i < d.nslots; i += 64) {
      const uint32_t v = slots[d.slot0 + i];
      m = max(m, v & 0x7FFFFFFFu);
      nan |= v & 0x80000000u;
    }
    m = wave_max_u32(m);
    nan = wave_max_u32(nan);
    const float amax = __builtin_bit_cast(float, m);
    float scale = 1.0f, inv = 1.0f;
    if (amax > 0.0f) {
      scale = amax / 448.0f;
      inv = 448.0f / amax;
    }
    if (tid == 0 && it.row0 == 0 && it.c0 == 0) ((OPTIMUS_GLOBAL float*)d.scale)[0] = scale;
    // The fast path needs every x * inv finite and within 464: no NaN in the
    // member, amax finite, and inv finite (a tiny amax overflows it).
    if (nan || !(amax < __builtin_inff()) || !(inv < __builtin_inff()))
      tile_convert<T, 2>(d, it, tid, inv);
    else
      tile_convert<T, 1>(d, it, tid, inv);
  }
}

// ------------------------------------------------------------------ dequantize
template <typename T>
__global__ __launch_bounds__(kFp8Threads) void grouped_dequantize_fp8_kernel(const DevFp8* __restrict__ descs,
                                                                             const Fp8Item* __restrict__ items,
                                                                             int32_t num_items) {
  constexpr int VEC = Fp8Side<T>::VEC;
  constexpr int U = kFp8U;
  const int tid = threadIdx.x;
  for (int t = blockIdx.x; t < num_items; t += gridDim.x) {
    const Fp8Item it = items[t];
    const DevFp8 d = descs[it.member];
    const float scale = d.scale ? ((const OPTIMUS_GLOBAL float*)d.scale)[0] : 1.0f;
    if (d.lanes > 0) {
      walk_tile<U>(it, d.lanes, tid, [&](const int* r, const int* c, const bool* ok) {
        typename Fp8Side<T>::Codes q[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const char* p = (const char*)d.x + (int64_t)r[u] * d.ldx + (int64_t)c[u] * VEC;
          q[u] = ok[u] ? __builtin_nontemporal_load((const OPTIMUS_GLOBAL typename Fp8Side<T>::Codes*)p)
                       : typename Fp8Side<T>::Codes{};
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (!ok[u]) continue;
          float v[VEC];
          if constexpr (VEC == 8) {
            const u32x2 w = q[u];
            f32x2 a = __builtin_amdgcn_cvt_pk_f32_fp8((int)w.x, false), b = __builtin_amdgcn_cvt_pk_f32_fp8((int)w.x, true);
            f32x2 e = __builtin_amdgcn_cvt_pk_f32_fp8((int)w.y, false), f = __builtin_amdgcn_cvt_pk_f32_fp8((int)w.y, true);
            v[0] = a.x; v[1] = a.y; v[2] = b.x; v[3] = b.y;
            v[4] = e.x; v[5] = e.y; v[6] = f.x; v[7] = f.y;
          } else {
            const uint32_t w = q[u];
            f32x2 a = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, false), b = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, true);
            v[0] = a.x; v[1] = a.y; v[2] = b.x; v[3] = b.y;
          }
#pragma unroll
          for (int e = 0; e < VEC; ++e) v[e] *= scale;
          st16_nt((char*)d.y + ((int64_t)r[u] * d.ldy + (int64_t)c[u] * VEC) * sizeof(T), Elem<T>::pack(v));
        }
      });
    } else {
      walk_tile<U>(it, d.lanes_scalar, tid, [&](const int* r, const int* c, const bool* ok) {
        uint32_t q[U];
#pragma unroll
        for (int u = 0; u < U; ++u) q[u] = ok[u] ? ((const OPTIMUS_GLOBAL uint8_t*)d.x)[(int64_t)r[u] * d.ldx + c[u]] : 0u;
#pragma unroll
        for (int u = 0; u < U; ++u)
          if (ok[u]) Elem<T>::store1(d.y, (int64_t)r[u] * d.ldy + c[u], __builtin_amdgcn_cvt_f32_fp8((int)q[u], 0) * scale);
      });
    }
  }
}

// ------------------------------------------------------------------ launchers
hipError_t fp8_amax_launch(optimus_dtype dt, const DevFp8* descs, const Fp8Item* items, int32_t num_items,
                           int32_t grid, uint32_t* slots, hipStream_t stream) {
  if (num_items <= 0) return hipSuccess;
  if (dt == OPTIMUS_BF16)
    hipLaunchKernelGGL(grouped_fp8_amax_kernel<bf16_t>, dim3(grid), dim3(kFp8Threads), 0, stream, descs, items,
                       num_items, slots);
  else
    hipLaunchKernelGGL(grouped_fp8_amax_kernel<float>, dim3(grid), dim3(kFp8Threads), 0, stream, descs, items,
                       num_items, slots);
  return hipGetLastError();
}

hipError_t fp8_quantize_launch(optimus_dtype dt, const DevFp8* descs, const Fp8Item* items, int32_t num_items,
                               int32_t grid, const uint32_t* slots, hipStream_t stream) {
  if (num_items <= 0) return hipSuccess;
  if (slots) {
    if (dt == OPTIMUS_BF16)
      hipLaunchKernelGGL(grouped_quantize_fp8_scaled_kernel<bf16_t>, dim3(grid), dim3(kFp8Threads), 0, stream, descs,
                         items, num_items, slots);
    else
      hipLaunchKernelGGL(grouped_quantize_fp8_scaled_kernel<float>, dim3(grid), dim3(kFp8Threads), 0, stream, descs,
                         items, num_items, slots);
  } else {
    if (dt == OPTIMUS_BF16)
      hipLaunchKernelGGL(grouped_quantize_fp8_kernel<bf16_t>, dim3(grid), dim3(kFp8Threads), 0, stream, descs, items,
                         num_items);
    else
      hipLaunchKernelGGL(grouped_quantize_fp8_kernel<float>, dim3(grid), dim3(kFp8Threads), 0, stream, descs, items,
                         num_items);
  }
  return hipGetLastError();
}

hipError_t fp8_dequantize_launch(optimus_dtype dt, const DevFp8* descs, const Fp8Item* items, int32_t num_items,
                                 int32_t grid, hipStream_t stream) {
  if (num_items <= 0) return hipSuccess;
  if (dt == OPTIMUS_BF16)
    hipLaunchKernelGGL(grouped_dequantize_fp8_kernel<bf16_t>, dim3(grid), dim3(kFp8Threads), 0, stream, descs, items,
                       num_items);
  else
    hipLaunchKernelGGL(grouped_dequantize_fp8_kernel<float>, dim3(grid), dim3(kFp8Threads), 0, stream, descs, items,
                       num_items);
  return hipGetLastError();
}

}  // namespace optimus
