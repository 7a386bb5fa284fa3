// Persistent grouped GEMM of liboptimus for gfx950 (Table 1 batch_linear /
// batch_linear_post_grad; Sec. 3.2 group fusion: heterogeneous members in one
// launch with their own layouts).
//
//   y_g[M_g][N_g] = act( x_g[M_g][K_g] . w_g[N_g][K_g]^T + bias_g[N_g] )
//
// One launch walks a device table of output tiles of all members. A tile is
// BM x BN of one member; its K loop stages x and w sub-tiles (BK wide, both
// K-contiguous) through LDS with a register prefetch of the next sub-tile, and
// feeds MFMA instructions: v_mfma_f32_32x32x16_bf16 for bf16 (fp32
// accumulate), v_mfma_f32_32x32x2f32 for fp32. The MFMA A operand is the
// weight tile and B the input tile, so each lane ends with four consecutive
// output columns of one output row: the epilogue adds the bias, applies the
// activation, rounds, and writes 8- or 16-byte pieces to an LDS staging tile
// from which whole rows leave in 16-byte coalesced stores. Rows past M, columns
// past N and K past K_g are zero-filled on load and masked on store (the
// in-kernel form of the pad -> matmul -> slice steps of the paper's pad_mm
// case study, appendix Sec. 8.2, without materialising any padding).
#include <stdlib.h>

#include "device_common.h"

namespace optimus {

template <typename T>
struct Mfma;

// bf16: one 16-byte chunk per lane half = 8 consecutive k; one instruction covers k = 16.
template <>
struct Mfma<bf16_t> {
  static constexpr int KPC = 16;  // k covered per 16-byte chunk pair
  __device__ static __forceinline__ void run(const u32x4& a, const u32x4& b, f32x16& c) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                0, 0);
  }
};

// fp32: a 16-byte chunk holds 4 k values per lane half. Instruction e pairs
// element e of the lower lane half with element e of the upper half, so the
// four instructions together cover the 8 k values of the chunk pair (the sum
// over k is taken in a fixed permuted order, identical for both operands).
template <>
struct Mfma<float> {
  static constexpr int KPC = 8;
  __device__ static __forceinline__ void run(const u32x4& a, const u32x4& b, f32x16& c) {
    // whole-vector casts (an element-wise bit cast of a vector is miscompiled)
    const f32x4 af = __builtin_bit_cast(f32x4, a), bf = __builtin_bit_cast(f32x4, b);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(af[0], bf[0], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(af[1], bf[1], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(af[2], bf[2], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(af[3], bf[3], c, 0, 0, 0);
  }
};

template <typename T, int BM, int BN, int BK, int WM, int WN, int STAGES>
struct GemmShape {
  static constexpr int VEC = Elem<T>::VEC;
  static constexpr int NT = WM * WN * 64;
  static constexpr int TM = BM / WM, TN = BN / WN;  // wave tile (rows of y, columns of y)
  static constexpr int FM = TM / 32, FN = TN / 32;  // 32x32 MFMA blocks per wave
  static constexpr int CPR = BK / VEC;              // 16-byte chunks per staged row
  static constexpr int LDK = BK + VEC;              // padded LDS row (elements): +16 bytes
  static constexpr int LX = BM * CPR / NT;          // x chunks per thread per K step
  static constexpr int LW = BN * CPR / NT;          // w chunks per thread per K step
  static constexpr int LDC = BN + (sizeof(T) == 2 ? 8 : 4);  // staging row (elements), 16-byte multiple
  static constexpr int STAGE_ELEMS = (BM + BN) * LDK;
  static constexpr size_t LDS_BYTES_AB = (size_t)STAGES * STAGE_ELEMS * sizeof(T);
  static constexpr size_t LDS_BYTES_C = (size_t)BM * LDC * sizeof(T);
  static constexpr size_t LDS_BYTES = (LDS_BYTES_AB > LDS_BYTES_C ? LDS_BYTES_AB : LDS_BYTES_C) + BN * sizeof(float);
  static_assert(TM % 32 == 0 && TN % 32 == 0, "wave tile must be a multiple of 32");
  static_assert((BM * CPR) % NT == 0 && (BN * CPR) % NT == 0, "staging must divide evenly");
  static_assert(BK % (2 * VEC) == 0, "BK must hold whole chunk pairs");
  static_assert((BM * BN / VEC) % NT == 0, "store phase must divide evenly");
};

// Load one 16-byte chunk of a K-contiguous operand row with zero fill past
// the row count or past K. `vec` = rows are 16-byte aligned and K % VEC == 0.
template <typename T>
__device__ __forceinline__ u32x4 load_chunk(const void* base, int64_t ld, int row, int nrows, int k, int K, bool vec) {
  constexpr int VEC = Elem<T>::VEC;
  u32x4 v = {0u, 0u, 0u, 0u};
  if (row < nrows && k < K) {
    const T* p = (const T*)base + (int64_t)row * ld + k;
    if (vec) {
      v = ld16(p);
    } else {
      float f[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) f[e] = (k + e < K) ? Elem<T>::load1(p, e) : 0.f;
      v = Elem<T>::pack(f);  // exact: the values are already representable in T
    }
  }
  return v;
}

template <typename T, int BM, int BN, int BK, int WM, int WN, int STAGES, int ACT>
__global__ __launch_bounds__(WM* WN * 64) void grouped_gemm_kernel(const DevLinear* __restrict__ descs,
                                                                   const GemmTile* __restrict__ tiles,
                                                                   int32_t num_tiles) {
  using S = GemmShape<T, BM, BN, BK, WM, WN, STAGES>;
  constexpr int VEC = S::VEC, NT = S::NT, CPR = S::CPR, LDK = S::LDK;
  extern __shared__ __align__(16) char smem[];
  T* sAB = (T*)smem;                                       // [STAGES][(BM + BN) * LDK]: x rows then w rows
  T* sC = (T*)smem;                                        // [BM][LDC] staging, reuses the A/B area
  float* sBias = (float*)(smem + (S::LDS_BYTES - BN * sizeof(float)));

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int l32 = lane & 31, lh = lane >> 5;

  // XCD-aware order: hardware deals workgroups round-robin to the 8 XCDs;
  // give each XCD a contiguous range of the (member-major) tile list so tiles
  // that share an x panel or a weight run on the same L2.
  int vb = blockIdx.x;
  if ((gridDim.x & 7) == 0) vb = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);

  for (int t = vb; t < num_tiles; t += gridDim.x) {
    const GemmTile tile = tiles[t];
    if (tile.member < 0) continue;
    const DevLinear d = descs[tile.member];
    const int m0 = tile.mb * BM, n0 = tile.nb * BN;
    const int Mr = d.M - m0, Nr = d.N - n0;  // rows / columns left in this tile (may exceed BM / BN)
    const bool vin = d.vec & 1;
    const T* xb = (const T*)d.x + (int64_t)m0 * d.ldx;
    const T* wb = (const T*)d.w + (int64_t)n0 * d.ldw;

    if (tid < BN) sBias[tid] = (d.bias && tid < Nr) ? Elem<T>::load1(d.bias, n0 + tid) : 0.f;

    f32x16 acc[S::FM][S::FN];
#pragma unroll
    for (int i = 0; i < S::FM; ++i)
#pragma unroll
      for (int j = 0; j < S::FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    u32x4 rx[S::LX], rw[S::LW];
    auto gload = [&](int k0) {
#pragma unroll
      for (int i = 0; i < S::LX; ++i) {
        const int idx = tid + i * NT, row = idx / CPR, c = idx % CPR;
        rx[i] = load_chunk<T>(xb, d.ldx, row, Mr, k0 + c * VEC, d.K, vin);
      }
#pragma unroll
      for (int i = 0; i < S::LW; ++i) {
        const int idx = tid + i * NT, row = idx / CPR, c = idx % CPR;
        rw[i] = load_chunk<T>(wb, d.ldw, row, Nr, k0 + c * VEC, d.K, vin);
      }
    };
    auto lstore = [&](int stage) {
      T* sx = sAB + stage * S::STAGE_ELEMS;
      T* sw = sx + BM * LDK;
#pragma unroll
      for (int i = 0; i < S::LX; ++i) {
        const int idx = tid + i * NT, row = idx / CPR, c = idx % CPR;
        *(u32x4*)(sx + row * LDK + c * VEC) = rx[i];
      }
#pragma unroll
      for (int i = 0; i < S::LW; ++i) {
        const int idx = tid + i * NT, row = idx / CPR, c = idx % CPR;
        *(u32x4*)(sw + row * LDK + c * VEC) = rw[i];
      }
    };
    auto compute = [&](int stage) {
      const T* sx = sAB + stage * S::STAGE_ELEMS;
      const T* sw = sx + BM * LDK;
#pragma unroll
      for (int kc = 0; kc < BK / (2 * VEC); ++kc) {
        const int ko = kc * 2 * VEC + lh * VEC;
        u32x4 a[S::FN], b[S::FM];
#pragma unroll
        for (int j = 0; j < S::FN; ++j) a[j] = *(const u32x4*)(sw + (wn * S::TN + j * 32 + l32) * LDK + ko);
#pragma unroll
        for (int i = 0; i < S::FM; ++i) b[i] = *(const u32x4*)(sx + (wm * S::TM + i * 32 + l32) * LDK + ko);
#pragma unroll
        for (int i = 0; i < S::FM; ++i)
#pragma unroll
          for (int j = 0; j < S::FN; ++j) Mfma<T>::run(a[j], b[i], acc[i][j]);
      }
    };

    const int nk = (d.K + BK - 1) / BK;
    if constexpr (STAGES == 2) {
      gload(0);
      lstore(0);
      __syncthreads();
      for (int kb = 0; kb < nk; ++kb) {
        if (kb + 1 < nk) gload((kb + 1) * BK);
        compute(kb & 1);
        if (kb + 1 < nk) lstore((kb + 1) & 1);
        __syncthreads();
      }
    } else {
      for (int kb = 0; kb < nk; ++kb) {
        gload(kb * BK);
        lstore(0);
        __syncthreads();
        compute(0);
        __syncthreads();
      }
    }

    // ---- epilogue: bias + activation + rounding into the LDS staging tile.
    // acc[i][j][r] is y row m = wm*TM + 32 i + l32, column
    // n = wn*TN + 32 j + 8 (r / 4) + 4 lh + (r % 4).
#pragma unroll
    for (int i = 0; i < S::FM; ++i) {
      const int m = wm * S::TM + i * 32 + l32;
#pragma unroll
      for (int j = 0; j < S::FN; ++j) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int n = wn * S::TN + j * 32 + q * 8 + lh * 4;
          const f32x4 bv = *(const f32x4*)(sBias + n);
          float o[4];
          o[0] = act_apply<ACT>(acc[i][j][q * 4 + 0] + bv.x);
          o[1] = act_apply<ACT>(acc[i][j][q * 4 + 1] + bv.y);
          o[2] = act_apply<ACT>(acc[i][j][q * 4 + 2] + bv.z);
          o[3] = act_apply<ACT>(acc[i][j][q * 4 + 3] + bv.w);
          if constexpr (sizeof(T) == 2) {
            u32x2 pk = {pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
            *(u32x2*)(sC + m * S::LDC + n) = pk;
          } else {
            *(f32x4*)(sC + m * S::LDC + n) = f32x4{o[0], o[1], o[2], o[3]};
          }
        }
      }
    }
    __syncthreads();
    // ---- store: whole 16-byte pieces of y rows
    const bool vout = (d.vec & 2) != 0;
    constexpr int SCPR = BN / VEC;
#pragma unroll
    for (int i = 0; i < BM * SCPR / NT; ++i) {
      const int idx = tid + i * NT, row = idx / SCPR, c = idx % SCPR;
      const int n = c * VEC;
      if (row < Mr && n < Nr) {
        T* yp = (T*)d.y + (int64_t)(m0 + row) * d.ldy + n0 + n;
        const T* sp = sC + row * S::LDC + n;
        if (vout && n + VEC <= Nr) {
          st16(yp, *(const u32x4*)sp);
        } else {
          for (int e = 0; e < VEC && n + e < Nr; ++e) {
            if constexpr (sizeof(T) == 2)
              ((OPTIMUS_GLOBAL uint16_t*)yp)[e] = ((const uint16_t*)sp)[e];
            else
              ((OPTIMUS_GLOBAL float*)yp)[e] = ((const float*)sp)[e];
          }
        }
      }
    }
    __syncthreads();  // staging and bias reads done before the next tile overwrites them
  }
}

// ===================================================================== configurations
struct GemmVariant {
  int bm, bn, threads, occ;  // occ: workgroups resident per CU (LDS / register bound)
  const char* name;
};

// 0: members with N, K <= 64 (one K step); 1: 128x128; 2: 256x256 (8 waves);
// 3: fp32; 4: 256x256 (4 waves); 5: 256x128 (4 waves).
static const GemmVariant kVariants[] = {
    {128, 64, 256, 4, "grouped_gemm_bf16_128x64x64_w4x1_s1"},
    {128, 128, 256, 2, "grouped_gemm_bf16_128x128x64_w2x2_s2"},
    {256, 256, 512, 1, "grouped_gemm_bf16_256x256x64_w2x4_s2"},
    {64, 64, 256, 4, "grouped_gemm_f32_64x64x32_w2x2_s2"},
    {256, 256, 256, 1, "grouped_gemm_bf16_256x256x64_w2x2_s2"},
    {256, 128, 256, 1, "grouped_gemm_bf16_256x128x64_w2x2_s2"},
};
static const int kNumVariants = (int)(sizeof(kVariants) / sizeof(kVariants[0]));

GemmConfig gemm_pick_config(optimus_dtype dt, const optimus_linear_desc* d, int32_t G) {
  int v;
  if (dt == OPTIMUS_F32) {
    v = 3;
  } else {
    int64_t maxN = 0, maxK = 0;
    double tiles256 = 0.0;
    for (int g = 0; g < G; ++g) {
      maxN = d[g].N > maxN ? d[g].N : maxN;
      maxK = d[g].K > maxK ? d[g].K : maxK;
      tiles256 += (double)((d[g].M + 255) / 256) * (double)((d[g].N + 255) / 256);
    }
    if (maxN <= 64 && maxK <= 64)
      v = 0;
    else if (tiles256 >= 2.0 * device_cu_count())
      v = 2;
    else
      v = 1;
  }
  // OPTIMUS_GEMM_VARIANT=<n> pins the bf16 tile shape (tests and tuning).
  if (dt == OPTIMUS_BF16) {
    const char* f = getenv("OPTIMUS_GEMM_VARIANT");
    if (f && f[0] >= '0' && f[0] <= '9' && f[1] == 0 && f[0] - '0' < kNumVariants && f[0] != '3') v = f[0] - '0';
  }
  const GemmVariant& k = kVariants[v];
  return GemmConfig{k.bm, k.bn, v, k.threads, k.occ, k.name};
}

template <typename T, int BM, int BN, int BK, int WM, int WN, int STAGES>
static hipError_t launch_shape(optimus_act act, const DevLinear* descs, const GemmTile* tiles, int32_t n, int32_t grid,
                               hipStream_t stream) {
  using S = GemmShape<T, BM, BN, BK, WM, WN, STAGES>;
  const size_t smem = S::LDS_BYTES;
#define OPTIMUS_GEMM_LAUNCH(A)                                                                                      \
  {                                                                                                                \
    auto kfn = grouped_gemm_kernel<T, BM, BN, BK, WM, WN, STAGES, A>;                                              \
    static bool attr_set = false; /* per device-independent kernel; setting it twice is harmless */               \
    if (smem > 65536 && !attr_set) {                                                                               \
      hipError_t e = hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem); \
      if (e != hipSuccess) return e;                                                                               \
      attr_set = true;                                                                                             \
    }                                                                                                              \
    hipLaunchKernelGGL(kfn, dim3(grid), dim3(S::NT), smem, stream, descs, tiles, n);                              \
  }
  switch (act) {
    case OPTIMUS_ACT_NONE: OPTIMUS_GEMM_LAUNCH(0); break;
    case OPTIMUS_ACT_RELU: OPTIMUS_GEMM_LAUNCH(1); break;
    case OPTIMUS_ACT_SIGMOID: OPTIMUS_GEMM_LAUNCH(2); break;
    case OPTIMUS_ACT_TANH: OPTIMUS_GEMM_LAUNCH(3); break;
    case OPTIMUS_ACT_SILU: OPTIMUS_GEMM_LAUNCH(4); break;
    default: return hipErrorInvalidValue;
  }
#undef OPTIMUS_GEMM_LAUNCH
  return hipGetLastError();
}

hipError_t gemm_launch(const GemmConfig& cfg, optimus_dtype dt, optimus_act act, const DevLinear* descs,
                       const GemmTile* tiles, int32_t num_tiles, int32_t grid, hipStream_t stream) {
  if (num_tiles <= 0) return hipSuccess;
  switch (cfg.variant) {
    case 0: return launch_shape<bf16_t, 128, 64, 64, 4, 1, 1>(act, descs, tiles, num_tiles, grid, stream);
    case 1: return launch_shape<bf16_t, 128, 128, 64, 2, 2, 2>(act, descs, tiles, num_tiles, grid, stream);
    case 2: return launch_shape<bf16_t, 256, 256, 64, 2, 4, 2>(act, descs, tiles, num_tiles, grid, stream);
    case 3: return launch_shape<float, 64, 64, 32, 2, 2, 2>(act, descs, tiles, num_tiles, grid, stream);
    case 4: return launch_shape<bf16_t, 256, 256, 64, 2, 2, 2>(act, descs, tiles, num_tiles, grid, stream);
    case 5: return launch_shape<bf16_t, 256, 128, 64, 2, 2, 2>(act, descs, tiles, num_tiles, grid, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace optimus
