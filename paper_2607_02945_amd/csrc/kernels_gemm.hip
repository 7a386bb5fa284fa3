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
#include "device_common.h"

namespace optimus {

typedef float f32x2 __attribute__((ext_vector_type(2)));

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
  static constexpr size_t LDS_MAIN = LDS_BYTES_AB > LDS_BYTES_C ? LDS_BYTES_AB : LDS_BYTES_C;
  // then fp32 [BN] bias; with a fused LayerNorm also [BN] gamma, [BN] beta and
  // two [BM][WN] row-partial buffers
  static constexpr size_t LDS_BYTES = LDS_MAIN + BN * sizeof(float);
  static constexpr size_t LDS_BYTES_LN = LDS_MAIN + 3 * BN * sizeof(float) + 2 * BM * WN * sizeof(float);
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

// ----------------------------------------------------------------- transposed operands
// An operand stored reduction-major (element (row, k) at base[k * ld + row]):
// the gradients dX = dY . W and dW = dY^T . X read W and X, dY across their
// rows. A thread loads KB reduction rows of one 16-byte chunk (VEC tile rows)
// and writes VEC pieces of KB reduction-consecutive values into the same
// [row][k] LDS layout the MFMA fragment reads use: for bf16 four rows, and the
// 4 x 8 block is transposed with two byte permutes per output word. Lanes
// take consecutive reduction blocks first: the 8-byte LDS writes of a wave
// then fall on distinct bank pairs (consecutive row groups sit 8 rows apart,
// a multiple of the bank period at the padded row pitch), while each global
// load still reads 64 contiguous bytes per reduction row.
template <typename T>
struct Trans;
template <>
struct Trans<bf16_t> {
  static constexpr int KB = 4;
};
template <>
struct Trans<float> {
  static constexpr int KB = 2;
};

// One 16-byte chunk of tile rows row..row+VEC-1 at reduction index k, zero
// past nrows or K. `vec`: the chunk is 16-byte aligned (ld % VEC == 0 and an
// aligned base).
template <typename T>
__device__ __forceinline__ u32x4 load_chunk_t(const void* base, int64_t ld, int row, int nrows, int k, int K,
                                              bool vec) {
  constexpr int VEC = Elem<T>::VEC;
  u32x4 v = {0u, 0u, 0u, 0u};
  if (k < K && row < nrows) {
    const T* p = (const T*)base + (int64_t)k * ld + row;
    if (vec && row + VEC <= nrows) {
      v = ld16(p);
    } else {
      float f[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) f[e] = (row + e < nrows) ? Elem<T>::load1(p, e) : 0.f;
      v = Elem<T>::pack(f);
    }
  }
  return v;
}

// v[j]: reduction row k0 + j of the chunk; dst: LDS element (row0, k0) of the
// [row][k] layout with row pitch LDK. Also adds each tile row's KB values to
// rs[] when `sum` (the row sums of the x operand: db for dW = dY^T X).
__device__ __forceinline__ void store_trans(const u32x4 (&v)[4], bf16_t* dst, int LDK, bool sum, float (&rs)[8]) {
  const uint32_t r0[4] = {v[0].x, v[0].y, v[0].z, v[0].w}, r1[4] = {v[1].x, v[1].y, v[1].z, v[1].w};
  const uint32_t r2[4] = {v[2].x, v[2].y, v[2].z, v[2].w}, r3[4] = {v[3].x, v[3].y, v[3].z, v[3].w};
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const u32x2 lo = {__builtin_amdgcn_perm(r1[p], r0[p], 0x05040100u), __builtin_amdgcn_perm(r3[p], r2[p], 0x05040100u)};
    const u32x2 hi = {__builtin_amdgcn_perm(r1[p], r0[p], 0x07060302u), __builtin_amdgcn_perm(r3[p], r2[p], 0x07060302u)};
    *(u32x2*)(dst + (2 * p) * LDK) = lo;
    *(u32x2*)(dst + (2 * p + 1) * LDK) = hi;
    if (sum) {
      rs[2 * p] += (bf16_lo(r0[p]) + bf16_lo(r1[p])) + (bf16_lo(r2[p]) + bf16_lo(r3[p]));
      rs[2 * p + 1] += (bf16_hi(r0[p]) + bf16_hi(r1[p])) + (bf16_hi(r2[p]) + bf16_hi(r3[p]));
    }
  }
}
__device__ __forceinline__ void store_trans(const u32x4 (&v)[2], float* dst, int LDK, bool sum, float (&rs)[4]) {
  const f32x4 a = __builtin_bit_cast(f32x4, v[0]), b = __builtin_bit_cast(f32x4, v[1]);
  const float fa[4] = {a[0], a[1], a[2], a[3]}, fb[4] = {b[0], b[1], b[2], b[3]};
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    *(f32x2*)(dst + c * LDK) = f32x2{fa[c], fb[c]};
    if (sum) rs[c] += fa[c] + fb[c];
  }
}

// Fused LayerNorm over each output row of a tile that holds whole rows
// (BN >= N, so n0 = 0): adds the bias to the accumulators, takes every row's
// mean and biased variance in two passes -- lane pair, then the WN waves that
// share the row, through `red` ([2][BM][WN]) -- and leaves
// (v - mean) / sqrt(var + eps) * gamma + beta in acc, in fp32 on the unrounded
// accumulator. Columns past N hold exact zeros (zero weights and bias), so
// they add nothing to the sum and are masked out of the centred squares.
// acc[i][j][r] holds row wm*TM + 32 i + (lane % 32), column
// wn*TN + 32 j + 8 (r / 4) + 4 (lane / 32) + (r % 4).
template <int BM, int BN, int WM, int WN>
__device__ __forceinline__ void ln_rows(f32x16 (&acc)[BM / WM / 32][BN / WN / 32], const float* sBias,
                                        const float* sGamma, const float* sBeta, float* red, const DevLinear& d) {
  constexpr int TM = BM / WM, TN = BN / WN, FM = TM / 32, FN = TN / 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN, l32 = lane & 31, lh = lane >> 5;
  const int c0 = wn * TN + lh * 4;  // this lane's first column
#pragma unroll
  for (int j = 0; j < FN; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 bv = *(const f32x4*)(sBias + c0 + j * 32 + q * 8);
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        acc[i][j][q * 4 + 0] += bv.x;
        acc[i][j][q * 4 + 1] += bv.y;
        acc[i][j][q * 4 + 2] += bv.z;
        acc[i][j][q * 4 + 3] += bv.w;
      }
    }
  float* red1 = red;
  float* red2 = red + BM * WN;
  float part[FM], mu[FM], rs[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    float t = 0.f;
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) t += acc[i][j][r];
    part[i] = t + __shfl_xor(t, 32);
  }
  if (lh == 0)
#pragma unroll
    for (int i = 0; i < FM; ++i) red1[(wm * TM + i * 32 + l32) * WN + wn] = part[i];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < WN; ++w) t += red1[(wm * TM + i * 32 + l32) * WN + w];
    mu[i] = t * d.inv_n;
  }
  if (d.N >= BN) {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      float t = 0.f;
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float c = acc[i][j][r] - mu[i];
          t += c * c;
        }
      part[i] = t;
    }
  } else {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      float t = 0.f;
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float c = c0 + j * 32 + (r >> 2) * 8 + (r & 3) < d.N ? acc[i][j][r] - mu[i] : 0.f;
          t += c * c;
        }
      part[i] = t;
    }
  }
#pragma unroll
  for (int i = 0; i < FM; ++i) part[i] += __shfl_xor(part[i], 32);
  if (lh == 0)
#pragma unroll
    for (int i = 0; i < FM; ++i) red2[(wm * TM + i * 32 + l32) * WN + wn] = part[i];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < WN; ++w) t += red2[(wm * TM + i * 32 + l32) * WN + w];
    rs[i] = __builtin_amdgcn_rsqf(t * d.inv_n + d.eps);
  }
#pragma unroll
  for (int j = 0; j < FN; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 gv = *(const f32x4*)(sGamma + c0 + j * 32 + q * 8);
      const f32x4 bv = *(const f32x4*)(sBeta + c0 + j * 32 + q * 8);
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        acc[i][j][q * 4 + 0] = (acc[i][j][q * 4 + 0] - mu[i]) * rs[i] * gv.x + bv.x;
        acc[i][j][q * 4 + 1] = (acc[i][j][q * 4 + 1] - mu[i]) * rs[i] * gv.y + bv.y;
        acc[i][j][q * 4 + 2] = (acc[i][j][q * 4 + 2] - mu[i]) * rs[i] * gv.z + bv.z;
        acc[i][j][q * 4 + 3] = (acc[i][j][q * 4 + 3] - mu[i]) * rs[i] * gv.w + bv.w;
      }
    }
}

// The fp32 per-column parameters of a tile: bias and, for a fused LayerNorm,
// gamma (1 when absent) and beta (0), zero past the member's last column.
template <typename T, int BN, bool LN>
__device__ __forceinline__ void load_col_params(float* sBias, float* sGamma, float* sBeta, const DevLinear& d, int n0,
                                                int Nr) {
  const int tid = threadIdx.x;
  if (tid < BN) {
    sBias[tid] = (d.bias && tid < Nr) ? Elem<T>::load1(d.bias, n0 + tid) : 0.f;
    if constexpr (LN) {
      sGamma[tid] = tid < Nr ? (d.gamma ? Elem<T>::load1(d.gamma, tid) : 1.f) : 0.f;
      sBeta[tid] = (d.beta && tid < Nr) ? Elem<T>::load1(d.beta, tid) : 0.f;
    }
  }
}

// Epilogue shared by the GEMM kernels: bias + activation + rounding into the
// LDS staging tile sC ([BM][LDC], reusing the operand area), then whole
// 16-byte pieces of y rows leave in coalesced stores, masked at the M/N tails.
// ACT bit 3 set: the bias was added and the row LayerNorm applied in acc.
// acc[i][j][r] holds y row m = wm*TM + 32 i + (lane % 32) and column
// n = wn*TN + 32 j + 8 (r / 4) + 4 (lane / 32) + (r % 4) (A operand = weights).
template <typename T, int BM, int BN, int WM, int WN, int LDC, int ACTX>
__device__ __forceinline__ void gemm_epilogue(const f32x16 (&acc)[BM / WM / 32][BN / WN / 32], T* sC,
                                              const float* sBias, const DevLinear& d, int m0, int n0, int Mr,
                                              int Nr) {
  constexpr int ACT = ACTX & 7;
  constexpr bool LN = (ACTX & 8) != 0;
  constexpr int VEC = Elem<T>::VEC, NT = WM * WN * 64, TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN, l32 = lane & 31, lh = lane >> 5;
  // One base address per lane and compile-time offsets: per-(i, j, q)
  // addresses would otherwise be kept live across the whole tile loop.
  T* const cbase = sC + (wm * TM + l32) * LDC + wn * TN + lh * 4;
  const float* const bbase = sBias + wn * TN + lh * 4;
  // this lane's bias values, read before any staging write (the compiler
  // cannot tell that those writes miss the bias, so reads placed after them
  // would each wait for their own LDS round trip)
  f32x4 bias[FN][4];
  if constexpr (!LN) {
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) bias[j][q] = *(const f32x4*)(bbase + j * 32 + q * 8);
  }
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int j = 0; j < FN; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float o[4];
        if constexpr (LN) {
          o[0] = act_apply<ACT>(acc[i][j][q * 4 + 0]);
          o[1] = act_apply<ACT>(acc[i][j][q * 4 + 1]);
          o[2] = act_apply<ACT>(acc[i][j][q * 4 + 2]);
          o[3] = act_apply<ACT>(acc[i][j][q * 4 + 3]);
        } else {
          const f32x4 bv = bias[j][q];
          o[0] = act_apply<ACT>(acc[i][j][q * 4 + 0] + bv.x);
          o[1] = act_apply<ACT>(acc[i][j][q * 4 + 1] + bv.y);
          o[2] = act_apply<ACT>(acc[i][j][q * 4 + 2] + bv.z);
          o[3] = act_apply<ACT>(acc[i][j][q * 4 + 3] + bv.w);
        }
        T* const cp = cbase + i * 32 * LDC + j * 32 + q * 8;
        if constexpr (sizeof(T) == 2) {
          u32x2 pk = {pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
          *(u32x2*)cp = pk;
        } else {
          *(f32x4*)cp = f32x4{o[0], o[1], o[2], o[3]};
        }
      }
    }
  }
  __syncthreads();
  const bool vout = (d.vec & 2) != 0;
  constexpr int SCPR = BN / VEC;  // 16-byte pieces per staged row
  static_assert(NT % SCPR == 0 && (BM * SCPR) % NT == 0, "store phase must divide evenly");
  constexpr int RSTEP = NT / SCPR;  // rows covered per pass of the workgroup
  const int r0 = tid / SCPR, n = (tid % SCPR) * VEC;
  const T* sp = sC + r0 * LDC + n;
  T* yp = (T*)d.y + (int64_t)(m0 + r0) * d.ldy + n0 + n;
  const int64_t ystep = (int64_t)RSTEP * d.ldy;
  if (n < Nr) {
    for (int row = r0; row < BM && row < Mr; row += RSTEP, sp += RSTEP * LDC, yp += ystep) {
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
}

// TR bit 0: x stored reduction-major; bit 1: w stored reduction-major (the
// transposed operands of the backward GEMMs). With bit 0 set and d.xsum
// given, the tiles of the first column block also write the row sums of x
// over the whole reduction (db beside dW = dY^T X).
// PRE > 0 (forward, two stages): a tile of at most PRE K steps issues the
// global loads of all its steps at once into registers, so the steps wait
// for one load latency instead of one each; with one row of four waves
// (WM = 1, WN = 4) and a member no wider than half the tile, the two wave
// pairs then take alternate K steps over the same columns and add their
// partial sums through LDS before the epilogue (the tile's MFMA time halves).
template <typename T, int BM, int BN, int BK, int WM, int WN, int STAGES, int ACT, int TR = 0, int PRE = 0>
__global__ __launch_bounds__(WM* WN * 64) void grouped_gemm_kernel(const DevLinear* __restrict__ descs,
                                                                   const GemmTile* __restrict__ tiles,
                                                                   int32_t num_tiles) {
  using S = GemmShape<T, BM, BN, BK, WM, WN, STAGES>;
  constexpr int VEC = S::VEC, NT = S::NT, CPR = S::CPR, LDK = S::LDK;
  constexpr bool TX = (TR & 1) != 0, TW = (TR & 2) != 0;
  constexpr int KB = Trans<T>::KB;
  // transposed operands: (rows / VEC) x (BK / KB) blocks, whole blocks per thread
  constexpr int LXT = (BM / VEC) * (BK / KB) / NT, LWT = (BN / VEC) * (BK / KB) / NT;
  static_assert(!TX || (LXT >= 1 && LXT * NT == (BM / VEC) * (BK / KB)), "transposed x staging must divide evenly");
  static_assert(!TW || (LWT >= 1 && LWT * NT == (BN / VEC) * (BK / KB)), "transposed w staging must divide evenly");
  static_assert(!TX || (size_t)(BK / KB) * BM * sizeof(float) <= S::LDS_MAIN, "row-sum partials must fit");
  constexpr int NRX = TX ? LXT * KB : S::LX, NRW = TW ? LWT * KB : S::LW;
  extern __shared__ __align__(16) char smem[];
  T* sAB = (T*)smem;                                       // [STAGES][(BM + BN) * LDK]: x rows then w rows
  T* sC = (T*)smem;                                        // [BM][LDC] staging, reuses the A/B area
  float* sBias = (float*)(smem + S::LDS_MAIN);             // [BN], then (fused LayerNorm) gamma, beta, partials
  float* sGamma = sBias + BN;
  float* sBeta = sGamma + BN;
  float* red = sBeta + BN;
  constexpr bool LN = (ACT & 8) != 0;

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
    const bool vw = TW ? (d.vec & 4) != 0 : vin;
    const T* xb = TX ? (const T*)d.x + m0 : (const T*)d.x + (int64_t)m0 * d.ldx;
    const T* wb = TW ? (const T*)d.w + n0 : (const T*)d.w + (int64_t)n0 * d.ldw;
    const bool want_sum = TX && d.xsum && tile.nb == 0;
    // the reduction range: all of K, or one split of it
    int kbeg = 0, kend = d.K;
    if constexpr (TR != 0) {
      if (d.ws) {
        kbeg = tile.pad * d.kchunk;
        kend = min(d.K, kbeg + d.kchunk);
      }
    }
    float xs[TX ? LXT : 1][VEC];
#pragma unroll
    for (int i = 0; i < (TX ? LXT : 1); ++i)
#pragma unroll
      for (int e = 0; e < VEC; ++e) xs[i][e] = 0.f;

    f32x16 acc[S::FM][S::FN];
#pragma unroll
    for (int i = 0; i < S::FM; ++i)
#pragma unroll
      for (int j = 0; j < S::FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    u32x4 rx[NRX], rw[NRW];
    auto gload_to = [&](u32x4 (&ox)[NRX], u32x4 (&ow)[NRW], int k0) {
      if constexpr (TX) {
#pragma unroll
        for (int i = 0; i < LXT; ++i) {
          const int idx = tid + i * NT, kq = idx % (BK / KB), rg = idx / (BK / KB);
#pragma unroll
          for (int j = 0; j < KB; ++j) ox[i * KB + j] = load_chunk_t<T>(xb, d.ldx, rg * VEC, Mr, k0 + kq * KB + j, kend, vin);
        }
      } else {
#pragma unroll
        for (int i = 0; i < S::LX; ++i) {
          const int idx = tid + i * NT, row = idx / CPR, c = idx % CPR;
          ox[i] = load_chunk<T>(xb, d.ldx, row, Mr, k0 + c * VEC, kend, vin);
        }
      }
      if constexpr (TW) {
#pragma unroll
        for (int i = 0; i < LWT; ++i) {
          const int idx = tid + i * NT, kq = idx % (BK / KB), rg = idx / (BK / KB);
#pragma unroll
          for (int j = 0; j < KB; ++j) ow[i * KB + j] = load_chunk_t<T>(wb, d.ldw, rg * VEC, Nr, k0 + kq * KB + j, kend, vw);
        }
      } else {
#pragma unroll
        for (int i = 0; i < S::LW; ++i) {
          const int idx = tid + i * NT, row = idx / CPR, c = idx % CPR;
          ow[i] = load_chunk<T>(wb, d.ldw, row, Nr, k0 + c * VEC, kend, vin);
        }
      }
    };
    auto gload = [&](int k0) { gload_to(rx, rw, k0); };
    auto lstore_from = [&](const u32x4 (&rx)[NRX], const u32x4 (&rw)[NRW], int stage) {
      T* sx = sAB + stage * S::STAGE_ELEMS;
      T* sw = sx + BM * LDK;
      if constexpr (TX) {
#pragma unroll
        for (int i = 0; i < LXT; ++i) {
          const int idx = tid + i * NT, kq = idx % (BK / KB), rg = idx / (BK / KB);
          u32x4 blk[KB];
#pragma unroll
          for (int j = 0; j < KB; ++j) blk[j] = rx[i * KB + j];
          store_trans(blk, sx + rg * VEC * LDK + kq * KB, LDK, want_sum, xs[i]);
        }
      } else {
#pragma unroll
        for (int i = 0; i < S::LX; ++i) {
          const int idx = tid + i * NT, row = idx / CPR, c = idx % CPR;
          *(u32x4*)(sx + row * LDK + c * VEC) = rx[i];
        }
      }
      if constexpr (TW) {
        float unused[VEC];
#pragma unroll
        for (int i = 0; i < LWT; ++i) {
          const int idx = tid + i * NT, kq = idx % (BK / KB), rg = idx / (BK / KB);
          u32x4 blk[KB];
#pragma unroll
          for (int j = 0; j < KB; ++j) blk[j] = rw[i * KB + j];
          store_trans(blk, sw + rg * VEC * LDK + kq * KB, LDK, false, unused);
        }
      } else {
#pragma unroll
        for (int i = 0; i < S::LW; ++i) {
          const int idx = tid + i * NT, row = idx / CPR, c = idx % CPR;
          *(u32x4*)(sw + row * LDK + c * VEC) = rw[i];
        }
      }
    };
    auto lstore = [&](int stage) { lstore_from(rx, rw, stage); };
    // MFMA over one staged step; wcol: the wave's column block (wn, or the
    // block it shares under the K split)
    auto compute = [&](int stage, int wcol) {
      const T* sx = sAB + stage * S::STAGE_ELEMS;
      const T* sw = sx + BM * LDK;
#pragma unroll
      for (int kc = 0; kc < BK / (2 * VEC); ++kc) {
        const int ko = kc * 2 * VEC + lh * VEC;
        u32x4 a[S::FN], b[S::FM];
#pragma unroll
        for (int j = 0; j < S::FN; ++j) a[j] = *(const u32x4*)(sw + (wcol * S::TN + j * 32 + l32) * LDK + ko);
#pragma unroll
        for (int i = 0; i < S::FM; ++i) b[i] = *(const u32x4*)(sx + (wm * S::TM + i * 32 + l32) * LDK + ko);
#pragma unroll
        for (int i = 0; i < S::FM; ++i)
#pragma unroll
          for (int j = 0; j < S::FN; ++j) Mfma<T>::run(a[j], b[i], acc[i][j]);
      }
    };

    // the first K step's operand loads go out before the tile's bias (and
    // LayerNorm parameter) loads, whose values are written to LDS: that
    // write waits for them, and the operand loads then fly meanwhile
    const int nk = (kend - kbeg + BK - 1) / BK;
    bool staged = false;  // K loop done by the all-steps-in-flight path
    if constexpr (PRE > 0 && STAGES == 2 && TR == 0) {
      if (nk <= PRE) {
        staged = true;
        u32x4 px[PRE][NRX], pw[PRE][NRW];
#pragma unroll
        for (int s = 0; s < PRE; ++s)
          if (s < nk) gload_to(px[s], pw[s], kbeg + s * BK);
        load_col_params<T, BN, LN>(sBias, sGamma, sBeta, d, n0, Nr);
        if (WM == 1 && WN == 4 && 2 * d.N <= BN && nk > 1) {
          // K split: wave pair p = wn / 2 takes steps s + p of each staged pair
          const int pair = wn >> 1;
#pragma unroll
          for (int s = 0; s < PRE; s += 2) {
            if (s < nk) {
              lstore_from(px[s], pw[s], 0);
              if (s + 1 < nk) lstore_from(px[s + 1], pw[s + 1], 1);
              __syncthreads();
              if (s + pair < nk) compute(pair, wn & 1);
              __syncthreads();
            }
          }
          // pair 1 hands its sums to pair 0 (same columns) through the operand
          // area; its own columns, past N, must read as zeros afterwards
          float* hand = (float*)smem + (wn & 1) * (S::FM * S::FN * 16 * 64);
          if (pair == 1) {
#pragma unroll
            for (int i = 0; i < S::FM; ++i)
#pragma unroll
              for (int j = 0; j < S::FN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                  hand[((i * S::FN + j) * 16 + r) * 64 + lane] = acc[i][j][r];
                  acc[i][j][r] = 0.f;
                }
          }
          __syncthreads();
          if (pair == 0) {
#pragma unroll
            for (int i = 0; i < S::FM; ++i)
#pragma unroll
              for (int j = 0; j < S::FN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[i][j][r] += hand[((i * S::FN + j) * 16 + r) * 64 + lane];
          }
          __syncthreads();  // hand-over read before the epilogue stages into the same area
        } else {
          lstore_from(px[0], pw[0], 0);
          __syncthreads();
#pragma unroll
          for (int s = 0; s < PRE; ++s) {
            if (s < nk) {
              compute(s & 1, wn);
              if (s + 1 < nk) lstore_from(px[s + 1], pw[s + 1], (s + 1) & 1);
              __syncthreads();
            }
          }
        }
      }
    }
    if (staged) {
    } else if constexpr (STAGES == 2) {
      gload(kbeg);
      load_col_params<T, BN, LN>(sBias, sGamma, sBeta, d, n0, Nr);
      lstore(0);
      __syncthreads();
      for (int kb = 0; kb < nk; ++kb) {
        if (kb + 1 < nk) gload(kbeg + (kb + 1) * BK);
        compute(kb & 1, wn);
        if (kb + 1 < nk) lstore((kb + 1) & 1);
        __syncthreads();
      }
    } else {
      for (int kb = 0; kb < nk; ++kb) {
        gload(kbeg + kb * BK);
        if (kb == 0) load_col_params<T, BN, LN>(sBias, sGamma, sBeta, d, n0, Nr);
        lstore(0);
        __syncthreads();
        compute(0, wn);
        __syncthreads();
      }
      if (nk == 0) load_col_params<T, BN, LN>(sBias, sGamma, sBeta, d, n0, Nr);
    }

    if constexpr (TX) {
      if (want_sum) {
        // row sums of x: per-thread partials over (kq, rows) -> LDS -> one sum per tile row
        float* part = (float*)smem;  // [BK / KB][BM], the operand area is free after the K loop
#pragma unroll
        for (int i = 0; i < LXT; ++i) {
          const int idx = tid + i * NT, kq = idx % (BK / KB), rg = idx / (BK / KB);
#pragma unroll
          for (int e = 0; e < VEC; ++e) part[kq * BM + rg * VEC + e] = xs[i][e];
        }
        __syncthreads();
        for (int r = tid; r < BM && r < Mr; r += NT) {
          float sum = 0.f;
          for (int q = 0; q < BK / KB; ++q) sum += part[q * BM + r];
          if (d.ws)  // this split's share of the row sums
            d.ws[(int64_t)d.splits * d.M * d.N + (int64_t)tile.pad * d.M + m0 + r] = sum;
          else
            Elem<T>::store1(d.xsum, m0 + r, sum);
        }
        __syncthreads();
      }
    }
    if constexpr (TR != 0) {
      if (d.ws) {
        // fp32 partial tile straight from the accumulators: each lane holds
        // four consecutive columns of one row per (i, j, quad)
        float* wb = d.ws + ((int64_t)tile.pad * d.M + m0) * d.N + n0;
        const bool v4 = (d.N & 3) == 0;
#pragma unroll
        for (int i = 0; i < S::FM; ++i) {
          const int row = wm * S::TM + i * 32 + l32;
          if (row >= Mr) continue;
#pragma unroll
          for (int j = 0; j < S::FN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int col = wn * S::TN + j * 32 + 8 * q + 4 * lh;
              float* p = wb + (int64_t)row * d.N + col;
              if (v4 && col + 3 < Nr) {
                *(OPTIMUS_GLOBAL f32x4*)p = f32x4{acc[i][j][q * 4 + 0], acc[i][j][q * 4 + 1], acc[i][j][q * 4 + 2],
                                                 acc[i][j][q * 4 + 3]};
              } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                  if (col + e < Nr) ((OPTIMUS_GLOBAL float*)p)[e] = acc[i][j][q * 4 + e];
              }
            }
        }
        continue;
      }
    }
    if constexpr (LN) ln_rows<BM, BN, WM, WN>(acc, sBias, sGamma, sBeta, red, d);
    gemm_epilogue<T, BM, BN, WM, WN, S::LDC, ACT>(acc, sC, sBias, d, m0, n0, Mr, Nr);
    __syncthreads();  // staging and bias reads done before the next tile overwrites them
  }
}

// ===================================================================== 16-row fp32 tiles
// Small fp32 groups (fewer 32-row tiles than CUs, at most 128 outputs per row)
// are latency bound: a workgroup's time is its descriptor and operand load
// latency plus its serial MFMA work. This kernel halves that work per
// workgroup with 16-row tiles on v_mfma_f32_16x16x4f32, and stages no operand
// through LDS: each lane loads its MFMA operands straight from global memory
// as 16-byte chunks of four consecutive k (w row n = lane % 16, x row
// m = lane % 16, k offset 4 (lane / 16) in a group of 16 k), so the waves of a
// tile never wait for one another inside the K loop. Instruction e of a group
// pairs element e of every lane's chunks, i.e. it sums k = 4 q + e over the
// lane quarters q; the four instructions cover the group's 16 k (a fixed
// permuted order, the same for both operands). The A operand is the weight
// tile, so output register r of lane l holds row l % 16 and column
// 4 (l / 16) + r of its 16-column block: four consecutive columns of a row.
//
// The four waves take the tile's 32-column blocks (two MFMA blocks each).
// When the tile holds fewer columns (N <= 64, or the last block of a wider
// member), the spare waves split the K range with the waves of the same
// columns and hand their partial sums over through LDS, added in a fixed
// order. A wave loads batches of kR16Batch k-groups, the next batch in flight
// while the current one is multiplied; even and odd k-groups go to separate
// accumulators, so four independent MFMA chains run per wave. Bias, gamma and
// beta are read once per column, by the first kR16Cols threads after the
// first operand batch is on its way, and reach the lanes through LDS after
// the K loop (one 4-byte load per value and lane had doubled the memory
// instructions ahead of the first MFMA).
constexpr int kR16Rows = 16, kR16Cols = 128, kR16Batch = 8;

template <int ACTX>
__global__ __launch_bounds__(256) void grouped_gemm_rows16_kernel(const DevLinear* __restrict__ descs,
                                                                 const GemmTile* __restrict__ tiles,
                                                                 int32_t num_tiles) {
  constexpr int ACT = ACTX & 7;
  constexpr bool LN = (ACTX & 8) != 0;
  constexpr int KB = kR16Batch;
  __shared__ float hand[3][4][8][64];    // K-split partials: [split - 1][column block][value][lane]
  __shared__ float red[2][kR16Rows][4];  // fused LayerNorm row partials: [pass][row][column block]
  __shared__ __align__(16) float par[3][kR16Cols];  // the tile's bias, gamma, beta per column; 0 past N
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, lq = lane >> 4;

  int vb = blockIdx.x;
  if ((gridDim.x & 7) == 0) vb = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);

  for (int t = vb; t < num_tiles; t += gridDim.x) {
    const GemmTile tile = tiles[t];
    if (tile.member < 0) continue;
    const DevLinear d = descs[tile.member];
    const int m0 = tile.mb * kR16Rows, n0 = tile.nb * kR16Cols;
    const int Mr = d.M - m0;                     // rows left from the tile's first (may exceed 16)
    const int Nr = min(d.N - n0, kR16Cols);      // columns in this tile
    const int ncb = Nr > 64 ? 4 : Nr > 32 ? 2 : 1;  // 32-column blocks in use
    const int ks = 4 / ncb;                      // waves per column block (K-split ways)
    const int cb = wave & (ncb - 1), sk = wave / ncb;
    const int c0 = cb * 32;                      // the wave's first column in the tile
    const int nkg = (d.K + 15) >> 4;             // k-groups of 16
    const int per = (nkg + ks - 1) / ks;
    const int g_beg = min(nkg, sk * per), g_end = min(nkg, g_beg + per);
    const bool vin = d.vec & 1;
    const float* xb = (const float*)d.x + (int64_t)m0 * d.ldx;
    const float* wb = (const float*)d.w + (int64_t)(n0 + c0) * d.ldw;
    const int wrows = Nr - c0;                   // w rows left from the wave's first column

    u32x4 bufA[KB][3], bufB[KB][3];              // per k-group: w block 0, w block 1, x
    auto load = [&](u32x4 (&b)[KB][3], int g0) {
#pragma unroll
      for (int i = 0; i < KB; ++i) {
        if (g0 + i < g_end) {
          const int k = (g0 + i) * 16 + lq * 4;
          b[i][0] = load_chunk<float>(wb, d.ldw, l16, wrows, k, d.K, vin);
          b[i][1] = load_chunk<float>(wb, d.ldw, 16 + l16, wrows, k, d.K, vin);
          b[i][2] = load_chunk<float>(xb, d.ldx, l16, Mr, k, d.K, vin);
        }
      }
    };
    f32x4 acc[2][2];  // [column block][k-group parity]
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int p = 0; p < 2; ++p) acc[j][p] = f32x4{0.f, 0.f, 0.f, 0.f};
    auto compute = [&](const u32x4 (&b)[KB][3], int g0) {
#pragma unroll
      for (int i = 0; i < KB; ++i) {
        if (g0 + i < g_end) {
          const f32x4 w0 = __builtin_bit_cast(f32x4, b[i][0]), w1 = __builtin_bit_cast(f32x4, b[i][1]);
          const f32x4 xv = __builtin_bit_cast(f32x4, b[i][2]);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[0][i & 1] = __builtin_amdgcn_mfma_f32_16x16x4f32(w0[e], xv[e], acc[0][i & 1], 0, 0, 0);
            acc[1][i & 1] = __builtin_amdgcn_mfma_f32_16x16x4f32(w1[e], xv[e], acc[1][i & 1], 0, 0, 0);
          }
        }
      }
    };

    // this lane's columns: c0 + 16 j + 4 lq + r of the tile
    const int cl = c0 + lq * 4;

    if (g_beg < g_end) load(bufA, g_beg);
    // thread tid < kR16Cols: column tid's parameters (zero past the member's columns)
    float qb = 0.f, qg = 0.f, qe = 0.f;
    if (tid < kR16Cols && tid < Nr) {
      qb = d.bias ? Elem<float>::load1(d.bias, n0 + tid) : 0.f;
      if constexpr (LN) {
        qg = d.gamma ? Elem<float>::load1(d.gamma, tid) : 1.f;
        qe = d.beta ? Elem<float>::load1(d.beta, tid) : 0.f;
      }
    }
    for (int g = g_beg; g < g_end; g += 2 * KB) {
      if (g + KB < g_end) load(bufB, g + KB);
      compute(bufA, g);
      if (g + 2 * KB < g_end) load(bufA, g + 2 * KB);
      if (g + KB < g_end) compute(bufB, g + KB);
    }
    f32x4 s[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) s[j] = acc[j][0] + acc[j][1];

    if (tid < kR16Cols) {
      par[0][tid] = qb;
      if constexpr (LN) {
        par[1][tid] = qg;
        par[2][tid] = qe;
      }
    }
    // the K-split waves hand their sums to the first wave of their columns
    if (ks > 1 && sk > 0)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) hand[sk - 1][cb][j * 4 + r][lane] = s[j][r];
    __syncthreads();
    if (ks > 1 && sk == 0)
      for (int q = 1; q < ks; ++q)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) s[j][r] += hand[q - 1][cb][j * 4 + r][lane];
    f32x4 pb[2], pg[2], pe[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      pb[j] = *(const f32x4*)&par[0][cl + 16 * j];
      if constexpr (LN) {
        pg[j] = *(const f32x4*)&par[1][cl + 16 * j];
        pe[j] = *(const f32x4*)&par[2][cl + 16 * j];
      }
    }

    float o[2][4];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) o[j][r] = s[j][r] + pb[j][r];
    if constexpr (LN) {
      // the tile holds whole rows (n0 = 0); columns past N are exact zeros
      // (zero weights and bias), so they add nothing to the sum
      float tsum = 0.f;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) tsum += o[j][r];
      tsum += __shfl_xor(tsum, 16);
      tsum += __shfl_xor(tsum, 32);
      if (sk == 0 && lq == 0) red[0][l16][cb] = tsum;
      __syncthreads();
      float mu = 0.f;
      for (int c = 0; c < ncb; ++c) mu += red[0][l16][c];
      mu *= d.inv_n;
      float tsq = 0.f;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float c = cl + 16 * j + r < Nr ? o[j][r] - mu : 0.f;
          tsq += c * c;
        }
      tsq += __shfl_xor(tsq, 16);
      tsq += __shfl_xor(tsq, 32);
      if (sk == 0 && lq == 0) red[1][l16][cb] = tsq;
      __syncthreads();
      float var = 0.f;
      for (int c = 0; c < ncb; ++c) var += red[1][l16][c];
      const float rs = __builtin_amdgcn_rsqf(var * d.inv_n + d.eps);
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) o[j][r] = (o[j][r] - mu) * rs * pg[j][r] + pe[j][r];
    }
    if (sk == 0 && l16 < Mr) {
      float* yr = (float*)d.y + (int64_t)(m0 + l16) * d.ldy + n0;
      const bool vout = (d.vec & 2) != 0;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int c = cl + 16 * j;
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = act_apply<ACT>(o[j][r]);
        if (vout && c + 3 < Nr) {
          st16(yr + c, __builtin_bit_cast(u32x4, f32x4{v[0], v[1], v[2], v[3]}));
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (c + r < Nr) Elem<float>::store1(yr, c + r, v[r]);
        }
      }
    }
    __syncthreads();  // hand-over and row partials read before the next tile writes them
  }
}

// ===================================================================== direct-to-LDS variant
// bf16 members whose x and w rows are 16-byte aligned with K % 8 == 0. The K
// loop stages BK = 64 columns of the x and w tiles straight from global memory
// into LDS with buffer_load_dwordx4 ... lds (no register staging, no LDS write
// instructions), two stages deep. Each such instruction of a wave fills 1 KB
// of LDS = 8 staged rows of 128 bytes; lane l brings the chunk that belongs at
// byte 16 l of it. A row keeps its 8 chunks, XOR-swizzled by (row / 2) mod 8 so
// that the 16 lanes of an MFMA operand read (16 consecutive rows, one chunk)
// hit distinct LDS banks.
//
// Addressing goes through one buffer resource per operand and tile whose
// record count ends at the tile's last valid row: rows past M (N) read as zero
// in hardware, and chunks past K are sent to an offset beyond any record count.
// The loads of step k+1 are issued in small groups between the first MFMA
// groups of step k, so the address unit works while the matrix cores do; one
// workgroup barrier per step then makes step k+1's stage visible and frees
// step k's. The last step of a tile fetches the next tile's first step.
// The K loop starts at a step that depends on the tile's coordinates, so the
// tiles that share an x panel or a weight block (which run side by side on one
// L2) do not request the same lines at the same moment.
typedef int i32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ i32x4 make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = (uint64_t)(uintptr_t)base;
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)b);
  r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(b >> 32) & 0xffffu));  // stride 0
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);                              // record count in bytes
  r[3] = 0x00020000;                                                               // 32-bit data format
  return r;
}

// One 16-byte chunk per lane into LDS at M0 + 16 * lane; an offset at or past
// the record count returns zeros. The compiler is not told that this writes
// LDS, so the K loop's waits are placed by hand.
__device__ __forceinline__ void lds_dma16(const i32x4& rsrc, uint32_t voff, uint32_t lds_addr) {
  // the address is wave-uniform; readfirstlane only tells the compiler so
  // where its analysis cannot see it
  const uint32_t a = (uint32_t)__builtin_amdgcn_readfirstlane((int)lds_addr);
  __asm__ volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
                   :
                   : "v"(voff), "s"(rsrc), "s"(a)
                   : "memory", "m0");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  __asm__ volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }

constexpr uint32_t kOutOfRange = 0x80000000u;  // larger than any tile's record count

template <int BM, int BN, int WM, int WN>
struct DmaShape {
  static constexpr int BK = 64, KC = BK / 16, NW = WM * WN, NT = NW * 64;
  static constexpr int TM = BM / WM, TN = BN / WN, FM = TM / 32, FN = TN / 32;
  static constexpr int XBYTES = BM * 128, WBYTES = BN * 128, STAGE = XBYTES + WBYTES;
  static constexpr int XI = BM / (8 * NW), WI = BN / (8 * NW);  // DMA instructions per wave per stage
  // ... issued over the first two MFMA groups of the step before (later ones
  // would leave too little of the step to cover their latency)
  static constexpr int NQ = XI + WI, PER = (NQ + 1) / 2;
  // epilogue: each wave stages HR rows of its TM x TN result at a time in its
  // own slice of the stage buffer the last K step read
  static constexpr int HR = 32, NH = TM / HR;  // one 32-row fragment row per pass
  // staged rows are padded by 16 bytes (8 rows at one chunk fall in 8 distinct
  // bank groups) so that every staging address is a lane base plus a constant
  static constexpr int PITCH = TN * 2 + 16, CPRW = TN / 8;  // staged row bytes, 16-byte chunks per row
  static constexpr size_t BIAS = 2 * (size_t)STAGE;        // fp32 bias of the current tile
  static constexpr size_t LDS_BYTES = BIAS + BN * sizeof(float);
  // a fused LayerNorm adds [BN] gamma, [BN] beta and two [BM][WN] row-partial buffers
  static constexpr size_t LDS_BYTES_LN = BIAS + 3 * BN * sizeof(float) + 2 * BM * WN * sizeof(float);
  static_assert(BM % (8 * NW) == 0 && BN % (8 * NW) == 0, "whole DMA instructions per wave");
  static_assert((8 * NW) % 16 == 0, "the swizzle of a lane's rows must not change between instructions");
  static_assert(TM % 32 == 0 && TN % 32 == 0, "wave tile must be a multiple of 32");
  static_assert(NW * HR * PITCH <= STAGE, "epilogue staging must fit in one stage buffer");
  static_assert((HR * CPRW) % 64 == 0 && CPRW >= 8, "staged rows leave in whole 64-lane passes");
  // Reduction-major operands (both stored [k][row]): a stage holds BK rows of
  // BM (BN) values, RB bytes each; one DMA instruction fills RPI of them, CPR
  // chunks per row. Chunk c of staged row r sits at position c ^ 4 (r mod 4),
  // so the four rows one transposing fragment read touches fall in four
  // distinct 64-byte bank windows; a wave's rows stay 0 mod 4 apart between
  // its instructions, so the swizzle of a lane's chunk is fixed.
  static constexpr int RB = BM * 2, RPI = 1024 / RB, CPR = RB / 16;
  static_assert(RPI * RB == 1024 && (NW * RPI) % 4 == 0 && CPR >= 16, "reduction-major staging layout");
};

// Transposing LDS read (gfx950): in each group of 16 lanes, element r of lane
// 4a + b is element b of the 8 bytes that lane a + 4r addressed. Lanes that
// address four consecutive values of four consecutive reduction rows thus
// receive four reduction values of one output row each.
typedef short s16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x2 lds_read_tr16(const char* p) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(
      (__attribute__((address_space(3))) char*)p));
  return __builtin_bit_cast(u32x2, v);
}

// What one K step's DMA instructions of a member tile need: the buffer
// resources of its x and w rows, this lane's byte offsets (already sent out of
// range for chunks past K), the bytes between a wave's consecutive
// instructions, and the step's first column. k0 < 0: no loads.
struct DmaLoads {
  const void* xp;          // first x / w row of the tile
  const void* wp;
  uint32_t xbytes, wbytes; // record counts: bytes up to the end of the tile's last valid row
  uint32_t sx, sw, xrow, wrow;
  int k0;
};

// First K step of a tile: tiles that share an x panel (same mb, run side by
// side on one L2) walk K in step so that the panel is fetched once; tiles
// that share a weight block (same nb, a block that stays in L2) start apart.
// With both operands reduction-major (the weight gradient) both panels are
// long streams through the batch: every tile starts at step 0, so the tiles
// of one member that run side by side share both.
template <int TR>
__device__ __forceinline__ int dma_rot(const GemmTile& tile, int nk) { return TR == 3 ? 0 : tile.mb % nk; }

// This lane's first staged row and (swizzled) element offset of its chunk,
// per operand: row-major operands stage 8 rows of 128 bytes per DMA
// instruction, reduction-major ones RPI rows of RB bytes.
struct DmaLanes {
  int lrx, kchx, lrw, kchw;
};

template <int BM, int BN, int NW, int TR>
__device__ __forceinline__ DmaLoads dma_loads(const DevLinear& d, int m0, int n0, int kbeg, int kend, int k0,
                                              const DmaLanes& ln) {
  constexpr bool TX = (TR & 1) != 0, TW = (TR & 2) != 0;
  DmaLoads L;
  // reduction-major: rows are reduction steps [kbeg, kend) starting at the
  // tile's first column; the record count ends at the last valid column of
  // the last row, so rows past kend and chunks past the last column read as
  // zero. Row-major: the record count ends at the tile's last valid row and
  // chunks past K are sent out of range.
  if constexpr (TX) {
    constexpr int RPI = 1024 / (BM * 2);
    L.xp = (const bf16_t*)d.x + (int64_t)kbeg * d.ldx + m0;
    L.xbytes = (uint32_t)(((int64_t)(kend - kbeg - 1) * d.ldx + (d.M - m0)) * 2);
    L.sx = (uint32_t)(((int64_t)(k0 + ln.lrx) * d.ldx + ln.kchx) * 2);
    L.xrow = (uint32_t)(NW * RPI * d.ldx * 2);
  } else {
    const int Mr = d.M - m0;
    L.xp = (const bf16_t*)d.x + (int64_t)m0 * d.ldx;
    L.xbytes = (uint32_t)((Mr < BM ? Mr : BM) * d.ldx * 2);
    L.sx = k0 + ln.kchx < d.K ? (uint32_t)((ln.lrx * d.ldx + ln.kchx) * 2) : kOutOfRange;
    L.xrow = (uint32_t)(NW * 8 * d.ldx * 2);
  }
  if constexpr (TW) {
    constexpr int RPI = 1024 / (BN * 2);
    L.wp = (const bf16_t*)d.w + (int64_t)kbeg * d.ldw + n0;
    L.wbytes = (uint32_t)(((int64_t)(kend - kbeg - 1) * d.ldw + (d.N - n0)) * 2);
    L.sw = (uint32_t)(((int64_t)(k0 + ln.lrw) * d.ldw + ln.kchw) * 2);
    L.wrow = (uint32_t)(NW * RPI * d.ldw * 2);
  } else {
    const int Nr = d.N - n0;
    L.wp = (const bf16_t*)d.w + (int64_t)n0 * d.ldw;
    L.wbytes = (uint32_t)((Nr < BN ? Nr : BN) * d.ldw * 2);
    L.sw = k0 + ln.kchw < d.K ? (uint32_t)((ln.lrw * d.ldw + ln.kchw) * 2) : kOutOfRange;
    L.wrow = (uint32_t)(NW * 8 * d.ldw * 2);
  }
  L.k0 = k0;
  return L;
}

// The reduction range of a work item: all of K, or (both operands
// reduction-major, a split reduction) split tile.pad of it.
template <int TR>
__device__ __forceinline__ void dma_krange(const DevLinear& d, const GemmTile& tile, int& kbeg, int& kend) {
  kbeg = 0;
  kend = d.K;
  if constexpr (TR == 3) {
    if (d.ws) {
      kbeg = tile.pad * d.kchunk;
      kend = min(d.K, kbeg + d.kchunk);
    }
  }
}

// The first K step's loads of work item t (k0 < 0 past the end or for a padding entry).
template <int BM, int BN, int NW, int TR>
__device__ __forceinline__ DmaLoads dma_first(const DevLinear* __restrict__ descs, const GemmTile* __restrict__ tiles,
                                              int t, int num_tiles, const DmaLanes& ln) {
  DmaLoads L;
  L.k0 = -1;
  if (t >= num_tiles) return L;
  const GemmTile tile = tiles[t];
  if (tile.member < 0) return L;
  const DevLinear& d = descs[tile.member];
  int kbeg, kend;
  dma_krange<TR>(d, tile, kbeg, kend);
  const int nk = (kend - kbeg + 63) / 64;
  return dma_loads<BM, BN, NW, TR>(d, tile.mb * BM, tile.nb * BN, kbeg, kend, dma_rot<TR>(tile, nk) * 64, ln);
}

template <int BM, int BN, int WM, int WN, int ACT, int TR = 0>
__global__ __launch_bounds__(WM* WN * 64) void grouped_gemm_dma_kernel(const DevLinear* __restrict__ descs,
                                                                       const GemmTile* __restrict__ tiles,
                                                                       int32_t num_tiles) {
  using S = DmaShape<BM, BN, WM, WN>;
  constexpr int NW = S::NW, A = ACT & 7;
  constexpr bool LN = (ACT & 8) != 0;  // the row LayerNorm is fused into the epilogue
  // TR bit 0: x stored reduction-major, bit 1: w. TR = 3 is the weight
  // gradient dW = dY^T X (x = dY, w = X), TR = 2 the input gradient
  // dX = dY W read straight from W; no bias, activation or LayerNorm
  constexpr bool TX = (TR & 1) != 0, TW = (TR & 2) != 0;
  static_assert(TR == 0 || ((TR == 3 && ACT == 0) || (TR == 2 && ACT < 8)) && BM == BN,
                "transposed instances: no bias or LayerNorm; TR = 2 may fuse an activation backward");
  // the epilogue's forward activation (TR = 0), or the activation whose
  // backward multiplies the stored input gradient (TR = 2, by act'(d.ax))
  constexpr int AF = TR == 0 ? A : 0, AG = TR == 2 ? A : 0;
  extern __shared__ __align__(16) char smem[];
  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)smem;
  float* sBias = (float*)(smem + S::BIAS);
  float* sGamma = sBias + BN;
  float* sBeta = sGamma + BN;
  float* red = sBeta + BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN, l32 = lane & 31, lh = lane >> 5;
  // this lane's first staged row and its (swizzled) chunk per operand; each
  // further DMA instruction of the wave is NW * 8 rows (reduction-major:
  // NW * RPI rows) further down, with the same swizzle
  DmaLanes ln;
  {
    const int lrn = wave * 8 + (lane >> 3), kchn = ((lane & 7) ^ swz(lrn)) << 3;
    const int lrt = wave * S::RPI + lane / S::CPR, kcht = ((lane % S::CPR) ^ (4 * (lrt & 3))) << 3;
    ln.lrx = TX ? lrt : lrn;
    ln.kchx = TX ? kcht : kchn;
    ln.lrw = TW ? lrt : lrn;
    ln.kchw = TW ? kcht : kchn;
  }

  int t = blockIdx.x;
  if ((gridDim.x & 7) == 0) t = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);

  // Load q of one K step (q < XI: x rows, then w rows) lands at byte lds_off(q)
  // of the stage plus 16 * lane.
  auto lds_off = [&](int q) {
    return q < S::XI ? wave * 8 * 128 + q * NW * 8 * 128 : S::XBYTES + wave * 8 * 128 + (q - S::XI) * NW * 8 * 128;
  };
  auto gofs = [&](const DmaLoads& L, int q) {
    // reduction-major offsets already hold the step's first row
    return q < S::XI ? L.sx + q * L.xrow + (TX ? 0 : L.k0 * 2) : L.sw + (q - S::XI) * L.wrow + (TW ? 0 : L.k0 * 2);
  };
  // every load of one K step into `stage`
  auto issue_all = [&](const DmaLoads& L, int stage) {
    const i32x4 rx = make_rsrc(L.xp, L.xbytes), rw = make_rsrc(L.wp, L.wbytes);
#pragma unroll
    for (int q = 0; q < S::NQ; ++q) lds_dma16(q < S::XI ? rx : rw, gofs(L, q), lds_base + stage * S::STAGE + lds_off(q));
  };

  int sbase = 0;  // stage holding the current tile's first K step
  {
    const DmaLoads L = dma_first<BM, BN, NW, TR>(descs, tiles, t, num_tiles, ln);
    if (L.k0 >= 0) issue_all(L, 0);
  }

  for (; t < num_tiles; t += gridDim.x) {
    const GemmTile tile = tiles[t];
    if (tile.member < 0) {
      // padding (only at the end of the list): nothing was loaded for it
      const DmaLoads L = dma_first<BM, BN, NW, TR>(descs, tiles, t + gridDim.x, num_tiles, ln);
      if (L.k0 >= 0) issue_all(L, sbase);
      continue;
    }
    const DevLinear& d = descs[tile.member];
    const int m0 = tile.mb * BM, n0 = tile.nb * BN;
    const int Mr = d.M - m0, Nr = d.N - n0;
    int kbeg, kend;
    dma_krange<TR>(d, tile, kbeg, kend);
    const int nk = (kend - kbeg + S::BK - 1) / S::BK, rot = dma_rot<TR>(tile, nk);
    // reduction-major x: the tiles of the first column block also sum each x
    // row over the reduction (db beside dW), from the fragments that the
    // waves of the first wave column read anyway
    const bool rsum = TX && d.xsum && tile.nb == 0 && wn == 0;
    float rs[S::FM];
#pragma unroll
    for (int i = 0; i < S::FM; ++i) rs[i] = 0.f;

    f32x16 acc[S::FM][S::FN];
#pragma unroll
    for (int i = 0; i < S::FM; ++i)
#pragma unroll
      for (int j = 0; j < S::FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // one K step on `stage`; the fragments of k-chunk kc + 1 are read from LDS
    // while the MFMAs of kc run, and the DMA instructions of the following
    // step (of this tile, or the next tile's first; none when nk0 < 0) are
    // spread over the first MFMA groups
    auto step = [&](int stage, const DmaLoads& L, int nstage) {
      const char* sxp = smem + stage * S::STAGE;
      const char* swp = sxp + S::XBYTES;
      u32x4 a[2][S::FN], b[2][S::FM];
      auto frag = [&](int kc, int set) {
        // reduction-major: lane 16 g + s reads reduction rows 16 kc +
        // 8 (g / 2) + s / 4 (+ 4 for the second read), values 4 (s mod 4) ..
        // + 3 of the fragment's 16 columns [16 (g mod 2), + 16); the reads
        // hand lane l the eight reduction values 8 (l / 32) .. + 7 of
        // fragment row l mod 32, the row-major read's layout
        const int s16 = lane & 15, t4 = s16 >> 2;
        const int kr = kc * 16 + 8 * lh + t4;
        const int cl = 2 * ((lane >> 4) & 1) + ((s16 & 3) >> 1);  // chunk within the 32-column fragment
        const int lo = kr * S::RB + cl * 16 + 8 * (s16 & 1);
        auto tr = [&](const char* base, int rowbase) {
          const char* p = base + lo + (((rowbase >> 5) ^ t4) << 6);
          const u32x2 v0 = lds_read_tr16(p), v1 = lds_read_tr16(p + 4 * S::RB);
          return u32x4{v0.x, v0.y, v1.x, v1.y};
        };
        const int lc = kc * 2 + lh;
#pragma unroll
        for (int j = 0; j < S::FN; ++j) {
          const int row = wn * S::TN + j * 32 + l32;
          if constexpr (TW)
            a[set][j] = tr(swp, wn * S::TN + j * 32);
          else
            a[set][j] = *(const u32x4*)(swp + row * 128 + ((lc ^ swz(row)) << 4));
        }
#pragma unroll
        for (int i = 0; i < S::FM; ++i) {
          const int row = wm * S::TM + i * 32 + l32;
          if constexpr (TX)
            b[set][i] = tr(sxp, wm * S::TM + i * 32);
          else
            b[set][i] = *(const u32x4*)(sxp + row * 128 + ((lc ^ swz(row)) << 4));
        }
      };
      const bool go = L.k0 >= 0;
      const i32x4 rx = make_rsrc(L.xp, L.xbytes), rw = make_rsrc(L.wp, L.wbytes);
      frag(0, 0);
#pragma unroll
      for (int kc = 0; kc < S::KC; ++kc) {
        if (kc + 1 < S::KC) frag(kc + 1, (kc + 1) & 1);
        if (go) {
#pragma unroll
          for (int q = kc * S::PER; q < (kc + 1) * S::PER && q < S::NQ; ++q)
            lds_dma16(q < S::XI ? rx : rw, gofs(L, q), lds_base + nstage * S::STAGE + lds_off(q));
        }
#pragma unroll
        for (int i = 0; i < S::FM; ++i)
#pragma unroll
          for (int j = 0; j < S::FN; ++j) Mfma<bf16_t>::run(a[kc & 1][j], b[kc & 1][i], acc[i][j]);
        if constexpr (TX) {
          if (rsum) {
#pragma unroll
            for (int i = 0; i < S::FM; ++i)
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const uint32_t v = b[kc & 1][i][e];
                rs[i] += __uint_as_float(v << 16) + __uint_as_float(v & 0xffff0000u);
              }
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    };

    for (int kb = 0; kb < nk; ++kb) {
      // this wave's loads of step kb (and its earlier stores) have landed;
      // the barrier extends that to every wave and frees step kb - 1's stage
      wait_vmcnt<0>();
      __syncthreads();
      const int stage = (sbase + kb) & 1;
      // the bias of this tile: the previous tile's epilogue read sBias before this barrier
      float bv = 0.f, gv = 0.f, ev = 0.f;
      if (kb == 0 && tid < BN) {
        bv = (d.bias && tid < Nr) ? Elem<bf16_t>::load1(d.bias, n0 + tid) : 0.f;
        if constexpr (LN) {
          gv = tid < Nr ? (d.gamma ? Elem<bf16_t>::load1(d.gamma, tid) : 1.f) : 0.f;
          ev = (d.beta && tid < Nr) ? Elem<bf16_t>::load1(d.beta, tid) : 0.f;
        }
      }
      // the following step of this tile, or at the last step the next tile's first
      DmaLoads L;
      if (kb + 1 < nk) {
        const int q = kb + 1 + rot;
        L = dma_loads<BM, BN, NW, TR>(d, m0, n0, kbeg, kend, (q >= nk ? q - nk : q) * S::BK, ln);
      } else {
        L = dma_first<BM, BN, NW, TR>(descs, tiles, t + gridDim.x, num_tiles, ln);
      }
      step(stage, L, stage ^ 1);
      if (kb == 0 && tid < BN) {
        sBias[tid] = bv;
        if constexpr (LN) {
          sGamma[tid] = gv;
          sBeta[tid] = ev;
        }
      }
    }
    __syncthreads();  // every wave is done with the last stage (staging) and the bias is written
    if constexpr (LN) ln_rows<BM, BN, WM, WN>(acc, sBias, sGamma, sBeta, red, d);
    if constexpr (TR == 3) {
      if (rsum) {
        // lanes l and l + 32 hold the two halves of row l mod 32's sum
#pragma unroll
        for (int i = 0; i < S::FM; ++i) {
          const float v = rs[i] + __shfl_xor(rs[i], 32);
          const int row = wm * S::TM + i * 32 + l32;
          if (lh == 0 && row < Mr) {
            if (d.ws)  // this split's share of the row sums
              d.ws[(int64_t)d.splits * d.M * d.N + (int64_t)tile.pad * d.M + m0 + row] = v;
            else
              Elem<bf16_t>::store1(d.xsum, m0 + row, v);
          }
        }
      }
      if (d.ws) {
        // fp32 partial tile straight from the accumulators: each lane holds
        // four consecutive columns of one row per (i, j, quad)
        float* wb = d.ws + ((int64_t)tile.pad * d.M + m0) * d.N + n0;
        const bool v4 = (d.N & 3) == 0;
#pragma unroll
        for (int i = 0; i < S::FM; ++i) {
          const int row = wm * S::TM + i * 32 + l32;
          if (row >= Mr) continue;
#pragma unroll
          for (int j = 0; j < S::FN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int col = wn * S::TN + j * 32 + 8 * q + 4 * lh;
              float* p = wb + (int64_t)row * d.N + col;
              if (v4 && col + 3 < Nr) {
                *(OPTIMUS_GLOBAL f32x4*)p = f32x4{acc[i][j][q * 4 + 0], acc[i][j][q * 4 + 1], acc[i][j][q * 4 + 2],
                                                 acc[i][j][q * 4 + 3]};
              } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                  if (col + e < Nr) ((OPTIMUS_GLOBAL float*)p)[e] = acc[i][j][q * 4 + e];
              }
            }
        }
      }
    }

    // epilogue: bias + activation + rounding into this wave's staging slice,
    // then whole 16-byte pieces of y rows leave in coalesced stores. Every
    // address is one lane base plus constants and every bound a per-tile
    // scalar, so nothing lane-dependent stays live across the tile loop.
    // (A split reduction has written its partial tile instead.)
    if (!(TR == 3 && d.ws)) {
      constexpr int RPP = 64 / S::CPRW;  // staged rows per store pass
      // opaque copies: computed here, per tile, instead of being hoisted out
      // of the tile loop and kept live across the K loop
      int lane_o = lane, wrow0 = wm * S::TM, wcol0 = wn * S::TN;
      __asm__ volatile("" : "+v"(lane_o));
      __asm__ volatile("" : "+s"(wrow0), "+s"(wcol0));
      const int lstage = (sbase + nk - 1) & 1;
      char* wst = smem + lstage * S::STAGE + wave * S::HR * S::PITCH;
      char* wput = wst + (lane_o & 31) * S::PITCH + (lane_o >> 5) * 8;
      const int lrow = lane_o / S::CPRW, lc = lane_o % S::CPRW;
      const char* wget = wst + lrow * S::PITCH + lc * 16;
      const float* bput = sBias + wcol0 + (lane_o >> 5) * 4;
      const int tc = wcol0 + lc * 8;  // tile column of this lane's stores
      const bool col_in = tc < Nr, col_vec = (d.vec & 2) != 0 && tc + 8 <= Nr;
      bf16_t* ybase = (bf16_t*)d.y + (int64_t)(m0 + wrow0) * d.ldy + n0 + tc + (int64_t)lrow * d.ldy;
      const bf16_t* abase = nullptr;
      if constexpr (AG != 0) abase = (const bf16_t*)d.ax + (int64_t)(m0 + wrow0 + lrow) * d.ldax + n0 + tc;
      // this lane's bias values, all read before the first staging write
      // (a fused LayerNorm has already added them)
      f32x4 bias[S::FN][4];
      if constexpr (!LN) {
#pragma unroll
        for (int j = 0; j < S::FN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) bias[j][q] = *(const f32x4*)(bput + j * 32 + q * 8);
      }
#pragma unroll
      for (int h = 0; h < S::NH; ++h) {
        // AG: this pass's activation-input chunks go out before the staging,
        // so their latency overlaps it and the wave barrier
        u32x4 av[S::HR / RPP];
        if constexpr (AG != 0) {
#pragma unroll
          for (int r = 0; r < S::HR / RPP; ++r) {
            const int lim = Mr - (wrow0 + h * S::HR + r * RPP);
            av[r] = (lrow < lim && col_vec && (d.vec & 8))
                        ? ld16_nt(abase + (int64_t)(h * S::HR + r * RPP) * d.ldax)
                        : u32x4{0u, 0u, 0u, 0u};
          }
        }
#pragma unroll
        for (int j = 0; j < S::FN; ++j) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x4 bv = LN ? f32x4{0.f, 0.f, 0.f, 0.f} : bias[j][q];
            float o0 = acc[h][j][q * 4 + 0], o1 = acc[h][j][q * 4 + 1];
            float o2 = acc[h][j][q * 4 + 2], o3 = acc[h][j][q * 4 + 3];
            if constexpr (!LN) {
              o0 += bv.x;
              o1 += bv.y;
              o2 += bv.z;
              o3 += bv.w;
            }
            o0 = act_apply<AF>(o0);
            o1 = act_apply<AF>(o1);
            o2 = act_apply<AF>(o2);
            o3 = act_apply<AF>(o3);
            *(u32x2*)(wput + (4 * j + q) * 16) = u32x2{pack_bf16x2(o0, o1), pack_bf16x2(o2, o3)};
          }
        }
        lds_wave_sync();
#pragma unroll
        for (int r = 0; r < S::HR / RPP; ++r) {
          const u32x4 v = *(const u32x4*)(wget + r * RPP * S::PITCH);
          const int lim = Mr - (wrow0 + h * S::HR + r * RPP);  // rows of this pass inside the tile
          if (lrow < lim && col_in) {
            bf16_t* yp = ybase + (int64_t)(h * S::HR + r * RPP) * d.ldy;
            if constexpr (AG != 0) {
              // dX * act'(ax): the stored value times the derivative at the
              // activation's input, rounded once more to bf16
              const bf16_t* ap = abase + (int64_t)(h * S::HR + r * RPP) * d.ldax;
              if (col_vec && (d.vec & 8)) {
                float g[8], a[8];
                Elem<bf16_t>::unpack(v, g);
                Elem<bf16_t>::unpack(av[r], a);
#pragma unroll
                for (int e = 0; e < 8; ++e) g[e] *= act_grad<AG>(a[e]);
                st16_nt(yp, Elem<bf16_t>::pack(g));
              } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                  if (tc + e < Nr) {
                    const float g = bf16_to_f32((uint16_t)(v[e >> 1] >> (16 * (e & 1))));
                    ((OPTIMUS_GLOBAL uint16_t*)yp)[e] =
                        f32_to_bf16(g * act_grad<AG>(bf16_to_f32(((const OPTIMUS_GLOBAL uint16_t*)ap)[e])));
                  }
              }
            } else if (col_vec) {
              st16_nt(yp, v);  // y is not read again by this launch
            } else {
#pragma unroll
              for (int e = 0; e < 8; ++e)
                if (tc + e < Nr) ((OPTIMUS_GLOBAL uint16_t*)yp)[e] = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
            }
          }
        }
        lds_wave_sync();  // staging read before the next pass overwrites it
      }
    }
    sbase = (sbase + nk) & 1;
  }
}

// ===================================================================== streaming members
// Every member has K <= 64 and N <= 64 values (bf16, N and K multiples of 8,
// 16-byte aligned rows): a member's whole weight is one K step of at most
// 64 x 64, so a tile's work is its x rows in and its y rows out -- a
// streaming pass over the batch rather than a tiled contraction. A work item
// is kStreamRows rows of one member. The block stages the member's weight
// and bias in LDS once per item (the MFMA A operand is w,
// v_mfma_f32_32x32x16_bf16, so a lane ends with four consecutive columns of
// one row); each wave then walks 32-row slabs of the item: a slab's x rows
// are loaded whole (coalesced 16-byte pieces: loading them straight into
// the MFMA B layout, 32 rows x 32 bytes per instruction, was 30 % slower)
// and turned into B operands through the wave's own LDS slice, the loads of
// the next two slabs are in flight while the current slab is multiplied and
// stored, and the result leaves through the same slice in whole 16-byte
// pieces of rows. Within an item the waves never wait for each other.
constexpr int kStreamRows = 512;  // 4 waves x 4 slabs of 32 rows (256: +1 %, 1024: +10 %)
constexpr int kStreamPitch = 144; // staged row bytes: 64 bf16 + 16 (distinct bank groups for the 8-row passes)
constexpr int kStreamWave = 32 * kStreamPitch;             // a wave's staging slice
constexpr int kStreamW = 4 * kStreamWave;                  // then the weight [64][kStreamPitch] and fp32 bias [64]
constexpr size_t kStreamLds = kStreamW + 64 * kStreamPitch + 64 * sizeof(float);

template <int ACT>
__global__ __launch_bounds__(256, 4) void grouped_gemm_stream_kernel(const DevLinear* __restrict__ descs,
                                                                     const GemmTile* __restrict__ tiles,
                                                                     int32_t num_tiles) {
  extern __shared__ __align__(16) char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, lh = lane >> 5;
  char* stg = smem + wave * kStreamWave;
  char* sw = smem + kStreamW;                           // w rows n, 64 k values each (zero past N, K)
  float* sbias = (float*)(sw + 64 * kStreamPitch);
  for (int t = blockIdx.x; t < num_tiles; t += gridDim.x) {
    const GemmTile tile = tiles[t];
    if (tile.member < 0) continue;
    const DevLinear& d = descs[tile.member];
    const int KC = (d.K + 15) >> 4, NB = (d.N + 31) >> 5;
    const int row0 = tile.mb * kStreamRows;
    const int rows = min(kStreamRows, d.M - row0);
    const int nslab = (rows + 31) >> 5;
    const bf16_t* xb = (const bf16_t*)d.x + (int64_t)row0 * d.ldx;
    // a slab's x rows in whole-row order: load i of lane l is 16-byte chunk
    // (l + 64 i) % 8 of slab row (l + 64 i) / 8
    auto xload = [&](int sl, u32x4 (&b)[4]) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int idx = lane + 64 * i, r = sl * 32 + (idx >> 3), c = idx & 7;
        b[i] = (r < rows && 8 * c < d.K) ? ld16_nt(xb + (int64_t)r * d.ldx + 8 * c) : u32x4{0u, 0u, 0u, 0u};
      }
    };
    // the first slab's x loads go out first, then the block's weight and bias
    // two slabs ahead in flight (2.5 % faster than one)
    u32x4 bx[4], bn[4], bn2[4];
    if (wave + 4 < nslab) xload(wave + 4, bn);
    if (wave < nslab) xload(wave, bx);
    __syncthreads();  // every wave is done with the previous item's weight and bias
    {
      // 64 rows x 8 chunks of 16 bytes, two per thread
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int idx = tid + 256 * i, n = idx >> 3, c = idx & 7;
        const u32x4 v = (n < d.N && 8 * c < d.K) ? ld16((const bf16_t*)d.w + (int64_t)n * d.ldw + 8 * c)
                                                 : u32x4{0u, 0u, 0u, 0u};
        *(u32x4*)(sw + n * kStreamPitch + 16 * c) = v;
      }
      if (tid < 64) sbias[tid] = (d.bias && tid < d.N) ? Elem<bf16_t>::load1(d.bias, tid) : 0.f;
    }
    __syncthreads();
    for (int sl = wave; sl < nslab; sl += 4) {
      if (sl + 8 < nslab) xload(sl + 8, bn2);
      // the slab through this wave's LDS slice into the MFMA B layout
      // (lane l: row l % 32, k values 16 kc + 8 (l / 32), + 8)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int idx = lane + 64 * i;
        *(u32x4*)(stg + (idx >> 3) * kStreamPitch + 16 * (idx & 7)) = bx[i];
      }
      lds_wave_sync();
      u32x4 xf[4];
#pragma unroll
      for (int kc = 0; kc < 4; ++kc) xf[kc] = *(const u32x4*)(stg + l32 * kStreamPitch + 32 * kc + 16 * lh);
      f32x16 acc[2];
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
#pragma unroll
      for (int kc = 0; kc < 4; ++kc) {
        if (kc < KC) {
#pragma unroll
          for (int j = 0; j < 2; ++j)
            if (j < NB) {
              // A operand: w[32 j + l32][16 kc + 8 lh, + 8)
              const u32x4 a = *(const u32x4*)(sw + (32 * j + l32) * kStreamPitch + 32 * kc + 16 * lh);
              Mfma<bf16_t>::run(a, xf[kc], acc[j]);
            }
        }
      }
      // bias + activation + rounding into this wave's staging slice: lane
      // (l32, lh) holds row l32, columns 32 j + 8 q + 4 lh + (0..3). Column
      // groups of 8 at or past N (N is a multiple of 8) are skipped whole, a
      // uniform branch: their values are never stored, and the activation's
      // transcendentals are most of the epilogue (launch_bound 21.1 ->
      // 20.3 us)
      char* put = stg + l32 * kStreamPitch + lh * 8;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (32 * j + 8 * q >= d.N) continue;
          const f32x4 bv = *(const f32x4*)(sbias + 32 * j + 8 * q + 4 * lh);
          const float o0 = act_apply<ACT>(acc[j][q * 4 + 0] + bv.x), o1 = act_apply<ACT>(acc[j][q * 4 + 1] + bv.y);
          const float o2 = act_apply<ACT>(acc[j][q * 4 + 2] + bv.z), o3 = act_apply<ACT>(acc[j][q * 4 + 3] + bv.w);
          *(u32x2*)(put + (32 * j + 8 * q) * 2) = u32x2{pack_bf16x2(o0, o1), pack_bf16x2(o2, o3)};
        }
      lds_wave_sync();
      // whole 16-byte pieces of rows: lane -> row (lane / 8) + 8 p, piece lane % 8
      const int pr = lane >> 3, pc = lane & 7;
      bf16_t* yb = (bf16_t*)d.y + (int64_t)(row0 + sl * 32 + pr) * d.ldy + pc * 8;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const int r = sl * 32 + p * 8 + pr;
        const u32x4 v = *(const u32x4*)(stg + (p * 8 + pr) * kStreamPitch + pc * 16);
        if (r < rows && pc * 8 < d.N) st16_nt(yb + (int64_t)(p * 8) * d.ldy, v);
      }
      lds_wave_sync();  // staging read before the next slab overwrites it
#pragma unroll
      for (int kc = 0; kc < 4; ++kc) {
        bx[kc] = bn[kc];
        bn[kc] = bn2[kc];
      }
    }
  }
}

// ===================================================================== skinny members
// Every member has K <= 8 and N <= 8: a tall-skinny matrix product such as
// [2e7, 8] x [8, 8], which the paper's decompose_mm rewrite (appendix Sec. 8.2)
// turns into pointwise products and a reduction over K because a tiled GEMM
// wastes nearly all of its work on such shapes. Here it is one streaming
// kernel with no MFMA: each lane owns whole rows, multiplies a row's K values
// by the member's weights (fp32 FMAs, ascending k) and writes the row's N
// outputs. A work item is kSkinnyRows rows of one member, walked in passes
// of RPL rows per lane (8 for the small classes, 4 for 8 x 8), and a lane
// loads all of a pass's rows before it uses any. A member's weights and bias are staged in LDS as fp32 when a
// workgroup's items reach it (while its first rows are in flight) and read
// back as broadcasts. A uniform branch per item picks the smallest shape class
// (KV, NV) that holds the member, so the paper's [*, 4] x [4, 2] and
// [*, 8] x [8, 8] members pay no padded FMAs.
constexpr int kSkinnyMax = 8;      // largest K and N of the path
constexpr int kSkinnyRows = 2048;  // rows per work item (4 waves)

template <typename T, int KV>
__device__ __forceinline__ void skinny_load(const T* p, int K, bool vec, float (&v)[KV]) {
  if constexpr (sizeof(T) == 4) {
    if (vec && KV % 4 == 0) {  // K == KV, 16-byte aligned rows
#pragma unroll
      for (int c = 0; c < KV / 4; ++c) {
        const f32x4 q = __builtin_bit_cast(f32x4, ld16_nt(p + 4 * c));
        v[4 * c + 0] = q.x;
        v[4 * c + 1] = q.y;
        v[4 * c + 2] = q.z;
        v[4 * c + 3] = q.w;
      }
      return;
    }
  } else {
    if (vec && KV % 8 == 0) {
      float f[8];
      Elem<bf16_t>::unpack(ld16_nt(p), f);
#pragma unroll
      for (int e = 0; e < KV; ++e) v[e] = f[e];
      return;
    }
  }
#pragma unroll
  for (int k = 0; k < KV; ++k) v[k] = k < K ? Elem<T>::load1(p, k) : 0.f;
}

template <typename T, int NV>
__device__ __forceinline__ void skinny_store(T* p, int N, bool vec, const float (&o)[NV]) {
  // vec: N == NV and rows aligned to their size (16 bytes, or 8 / 4 for narrower rows)
  if constexpr (sizeof(T) == 4) {
    if (vec && NV % 4 == 0) {
#pragma unroll
      for (int c = 0; c < NV / 4; ++c)
        st16_nt(p + 4 * c, __builtin_bit_cast(u32x4, f32x4{o[4 * c], o[4 * c + 1], o[4 * c + 2], o[4 * c + 3]}));
      return;
    }
    if (vec && NV == 2) {
      __builtin_nontemporal_store(u32x2{__builtin_bit_cast(uint32_t, o[0]), __builtin_bit_cast(uint32_t, o[1])},
                                  (OPTIMUS_GLOBAL u32x2*)p);
      return;
    }
  } else {
    if (vec && NV % 8 == 0) {
      st16_nt(p, u32x4{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]), pack_bf16x2(o[4], o[5]),
                       pack_bf16x2(o[6], o[7])});
      return;
    }
    if (vec && NV == 4) {
      __builtin_nontemporal_store(u32x2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])}, (OPTIMUS_GLOBAL u32x2*)p);
      return;
    }
    if (vec && NV == 2) {
      __builtin_nontemporal_store(pack_bf16x2(o[0], o[1]), (OPTIMUS_GLOBAL uint32_t*)p);
      return;
    }
  }
#pragma unroll
  for (int n = 0; n < NV; ++n)
    if (n < N) Elem<T>::store1(p, n, o[n]);
}

// The lane's rows of one pass: rows base + 64 i of [r0, r0 + count).
template <typename T, int KV, int RPL>
__device__ __forceinline__ void skinny_rows_load(const DevLinear& d, int r0, int count, float (&x)[RPL][KV]) {
  const bool vin = (d.vec & 1) && d.K == KV;
  const int base = (threadIdx.x >> 6) * 64 * RPL + (threadIdx.x & 63);
#pragma unroll
  for (int i = 0; i < RPL; ++i) {
    const int r = base + 64 * i;
    if (r < count) skinny_load<T, KV>((const T*)d.x + (int64_t)(r0 + r) * d.ldx, d.K, vin, x[i]);
  }
}

// Products, bias, activation and stores of the loaded rows; weights sW[n][k]
// (kSkinnyMax x kSkinnyMax, zero outside N x K) and bias sB in LDS.
template <typename T, int KV, int NV, int ACT, int RPL>
__device__ __forceinline__ void skinny_rows_out(const DevLinear& d, int r0, int count, const float (&x)[RPL][KV],
                                                const float* sW, const float* sB) {
  // rows of NV elements aligned to their size: 16-byte pieces, or one 8- / 4-byte piece
  constexpr int ROWB = NV * (int)sizeof(T);
  const bool vout = d.N == NV && ((ROWB >= 16) ? (d.vec & 2) != 0
                                               : ((uintptr_t)d.y % ROWB == 0 && (d.ldy * sizeof(T)) % ROWB == 0));
  const int base = (threadIdx.x >> 6) * 64 * RPL + (threadIdx.x & 63);
  float o[RPL][NV];
#pragma unroll
  for (int n = 0; n < NV; ++n) {
    float w[KV];
#pragma unroll
    for (int k = 0; k < KV; ++k) w[k] = sW[n * kSkinnyMax + k];
    const float b = sB[n];
#pragma unroll
    for (int i = 0; i < RPL; ++i) {
      float s = 0.f;
#pragma unroll
      for (int k = 0; k < KV; ++k) s = fmaf(x[i][k], w[k], s);
      o[i][n] = act_apply<ACT>(s + b);
    }
  }
#pragma unroll
  for (int i = 0; i < RPL; ++i) {
    const int r = base + 64 * i;
    if (r < count) skinny_store<T, NV>((T*)d.y + (int64_t)(r0 + r) * d.ldy, d.N, vout, o[i]);
  }
}

// One work item in shape class (KV, NV), in passes of 256 * RPL rows: the
// first pass's loads go out first, then (only when the member changed) the
// weights are staged while they fly.
template <typename T, int KV, int NV, int ACT, int RPL>
__device__ __forceinline__ void skinny_item(const DevLinear& d, int r0, int count, bool restage, float* sW, float* sB) {
  constexpr int PASS = 256 * RPL;
  static_assert(kSkinnyRows % PASS == 0, "whole passes per item");
  float x[RPL][KV];
  skinny_rows_load<T, KV, RPL>(d, r0, count, x);
  if (restage) {
    __syncthreads();  // every wave is done with the previous member's weights
    const int tid = threadIdx.x;
    if (tid < kSkinnyMax * kSkinnyMax) {
      const int n = tid / kSkinnyMax, k = tid % kSkinnyMax;
      sW[tid] = (n < d.N && k < d.K) ? Elem<T>::load1(d.w, (int64_t)n * d.ldw + k) : 0.f;
    }
    if (tid < kSkinnyMax) sB[tid] = (d.bias && tid < d.N) ? Elem<T>::load1(d.bias, tid) : 0.f;
    __syncthreads();
  }
  skinny_rows_out<T, KV, NV, ACT, RPL>(d, r0, count, x, sW, sB);
#pragma unroll 1
  for (int p = PASS; p < kSkinnyRows && p < count; p += PASS) {
    skinny_rows_load<T, KV, RPL>(d, r0 + p, count - p, x);
    skinny_rows_out<T, KV, NV, ACT, RPL>(d, r0 + p, count - p, x, sW, sB);
  }
}

// fp32 members with K = N = 8 and contiguous rows (32 bytes each): a lane pair
// per row, so that every load and store instruction moves consecutive 16-byte
// chunks. Thread t takes chunks t + 256 j of the item (chunk c is half c % 2
// of row c / 2; the two halves of a row sit in adjacent lanes), forms the
// partial products of its four k for all eight outputs, adds its partner's
// partials (DPP lane ^ 1 swap), and stores its half of the row's outputs,
// which is the same chunk index of y.
constexpr int kSkinnyChunks = 8;  // chunks per thread per pass (a pass is 1024 rows)
template <int ACT>
__device__ __forceinline__ void skinny_pairs_pass(const float* xb, float* yb, int nchunks, const f32x4 (&w)[8],
                                                  const f32x4& b, f32x4 (&x)[kSkinnyChunks], bool loaded) {
  const int tid = threadIdx.x, half = tid & 1;
  if (!loaded) {
#pragma unroll
    for (int j = 0; j < kSkinnyChunks; ++j) {
      const int c = tid + 256 * j;
      x[j] = c < nchunks ? __builtin_bit_cast(f32x4, ld16_nt(xb + 4 * c)) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
#pragma unroll
  for (int j = 0; j < kSkinnyChunks; ++j) {
    float p[8];
#pragma unroll
    for (int n = 0; n < 8; ++n) {
      float t = x[j].x * w[n].x;
      t = fmaf(x[j].y, w[n].y, t);
      t = fmaf(x[j].z, w[n].z, t);
      t = fmaf(x[j].w, w[n].w, t);
      p[n] = t;
    }
    float o[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      // outputs q and 4 + q: this lane keeps one, its partner the other
      const float mine = half ? p[4 + q] : p[q], theirs = half ? p[q] : p[4 + q];
      o[q] = mine + dpp_f<0xB1>(theirs);  // partner's partial of the same output
    }
    const int c = tid + 256 * j;
    if (c < nchunks)
      st16_nt(yb + 4 * c, __builtin_bit_cast(u32x4, f32x4{act_apply<ACT>(o[0] + b.x), act_apply<ACT>(o[1] + b.y),
                                                           act_apply<ACT>(o[2] + b.z), act_apply<ACT>(o[3] + b.w)}));
  }
}

template <int ACT>
__device__ __forceinline__ void skinny_item_pairs(const DevLinear& d, int r0, int count, bool restage, float* sW,
                                                  float* sB) {
  constexpr int PASS = 256 * kSkinnyChunks / 2;  // rows per pass
  static_assert(kSkinnyRows % PASS == 0, "whole passes per item");
  const int tid = threadIdx.x, half = tid & 1;
  const float* xb = (const float*)d.x + (int64_t)r0 * 8;
  float* yb = (float*)d.y + (int64_t)r0 * 8;
  f32x4 x[kSkinnyChunks];
#pragma unroll
  for (int j = 0; j < kSkinnyChunks; ++j) {
    const int c = tid + 256 * j;
    x[j] = c < 2 * count ? __builtin_bit_cast(f32x4, ld16_nt(xb + 4 * c)) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  if (restage) {
    __syncthreads();
    if (tid < kSkinnyMax * kSkinnyMax) sW[tid] = Elem<float>::load1(d.w, (int64_t)(tid / 8) * d.ldw + tid % 8);
    if (tid < kSkinnyMax) sB[tid] = d.bias ? Elem<float>::load1(d.bias, tid) : 0.f;
    __syncthreads();
  }
  // this lane's four k of every output row, and the bias of its four outputs
  f32x4 w[8];
#pragma unroll
  for (int n = 0; n < 8; ++n) w[n] = *(const f32x4*)(sW + n * 8 + half * 4);
  const f32x4 b = *(const f32x4*)(sB + half * 4);
  skinny_pairs_pass<ACT>(xb, yb, 2 * count, w, b, x, true);
#pragma unroll 1
  for (int p = PASS; p < kSkinnyRows && p < count; p += PASS)
    skinny_pairs_pass<ACT>(xb + (int64_t)p * 8, yb + (int64_t)p * 8, 2 * (count - p), w, b, x, false);
}

template <typename T, int ACT>
__global__ __launch_bounds__(256) void grouped_gemm_skinny_kernel(const DevLinear* __restrict__ descs,
                                                                  const GemmTile* __restrict__ tiles,
                                                                  int32_t num_tiles) {
  __shared__ __align__(16) float sW[kSkinnyMax * kSkinnyMax];
  __shared__ __align__(16) float sB[kSkinnyMax];
  int staged = -1;  // member whose weights sW / sB hold
  for (int t = blockIdx.x; t < num_tiles; t += gridDim.x) {
    const GemmTile tile = tiles[t];
    if (tile.member < 0) continue;
    const DevLinear& d = descs[tile.member];
    const bool restage = tile.member != staged;
    staged = tile.member;
    const int r0 = tile.mb * kSkinnyRows;
    const int count = min(kSkinnyRows, d.M - r0);
    bool pairs = false;
    if constexpr (sizeof(T) == 4) pairs = d.K == 8 && d.N == 8 && d.ldx == 8 && d.ldy == 8 && (d.vec & 3) == 3;
    if (pairs)
      skinny_item_pairs<ACT>(d, r0, count, restage, sW, sB);
    else if (d.K <= 4 && d.N <= 2)
      skinny_item<T, 4, 2, ACT, 8>(d, r0, count, restage, sW, sB);
    else if (d.K <= 4 && d.N <= 4)
      skinny_item<T, 4, 4, ACT, 8>(d, r0, count, restage, sW, sB);
    else
      skinny_item<T, 8, 8, ACT, 4>(d, r0, count, restage, sW, sB);
  }
}

// ===================================================================== split reduction
// y[m][n] = sum over the splits of the fp32 partials, rounded once; the row
// sums likewise. An item is a run of rows; its (row, 4-column group) pairs
// are spread over the workgroup's threads, so every thread has a few
// independent loads per split in flight whatever the width.
template <typename T>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const SplitReduceItem* __restrict__ items,
                                                            int32_t num_items) {
  const int tid = threadIdx.x;
  for (int t = blockIdx.x; t < num_items; t += gridDim.x) {
    const SplitReduceItem it = items[t];
    const int64_t plane = (int64_t)it.M * it.N;
    const int nc4 = (it.N + 3) >> 2;
    const int total = it.nrows * nc4;
    const bool v4 = (it.N & 3) == 0;
    for (int e = tid; e < total; e += 256) {
      const int r = it.row0 + e / nc4;
      const int c = (e % nc4) * 4;
      const float* src = it.ws + (int64_t)r * it.N + c;
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
      if (v4) {
        for (int s = 0; s < it.splits; ++s) {
          const f32x4 v = *(const OPTIMUS_GLOBAL f32x4*)(src + s * plane);
          acc[0] += v[0];
          acc[1] += v[1];
          acc[2] += v[2];
          acc[3] += v[3];
        }
      } else {
        for (int s = 0; s < it.splits; ++s)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (c + q < it.N) acc[q] += ((const OPTIMUS_GLOBAL float*)(src + s * plane))[q];
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (c + q < it.N) Elem<T>::store1(it.y, (int64_t)r * it.ldy + c + q, acc[q]);
    }
    if (it.xsum) {
      const float* sums = it.ws + (int64_t)it.splits * plane;
      for (int r = it.row0 + tid; r < it.row0 + it.nrows; r += 256) {
        float a = 0.f;
        for (int s = 0; s < it.splits; ++s) a += sums[(int64_t)s * it.M + r];
        Elem<T>::store1(it.xsum, r, a);
      }
    }
  }
}

hipError_t splitk_reduce_launch(optimus_dtype dt, const SplitReduceItem* items, int32_t num_items, int32_t grid,
                                hipStream_t stream) {
  if (num_items <= 0) return hipSuccess;
  if (dt == OPTIMUS_BF16)
    hipLaunchKernelGGL(splitk_reduce_kernel<bf16_t>, dim3(grid), dim3(256), 0, stream, items, num_items);
  else
    hipLaunchKernelGGL(splitk_reduce_kernel<float>, dim3(grid), dim3(256), 0, stream, items, num_items);
  return hipGetLastError();
}

// ===================================================================== grouped transpose
// W [N][K] -> W^T [K][N] for the dX GEMM of the Linear backward (W is small
// next to the activations, so the copy costs little and dX then runs on the
// forward's direct-to-LDS kernel). 64 x 64 tiles through LDS, rows padded by
// one element; values moved as raw bits.
template <typename U>
__global__ __launch_bounds__(256) void grouped_transpose_kernel(const TransposeItem* __restrict__ items,
                                                                int32_t num_items) {
  __shared__ U tile[64][65];
  const int tid = threadIdx.x, tc = tid & 63, tr = tid >> 6;
  for (int t = blockIdx.x; t < num_items; t += gridDim.x) {
    const TransposeItem it = items[t];
    const OPTIMUS_GLOBAL U* src = (const OPTIMUS_GLOBAL U*)it.src;
    OPTIMUS_GLOBAL U* dst = (OPTIMUS_GLOBAL U*)it.dst;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int r = it.r0 + tr + 4 * i, c = it.c0 + tc;
      if (r < it.rows && c < it.cols) tile[tr + 4 * i][tc] = src[(int64_t)r * it.lds + c];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int c = it.c0 + tr + 4 * i, r = it.r0 + tc;  // dst row c, column r
      if (r < it.rows && c < it.cols) dst[(int64_t)c * it.ldd + r] = tile[tc][tr + 4 * i];
    }
    __syncthreads();
  }
}

hipError_t transpose_launch(optimus_dtype dt, const TransposeItem* items, int32_t num_items, int32_t grid,
                            hipStream_t stream) {
  if (num_items <= 0) return hipSuccess;
  if (dt == OPTIMUS_BF16)
    hipLaunchKernelGGL(grouped_transpose_kernel<uint16_t>, dim3(grid), dim3(256), 0, stream, items, num_items);
  else
    hipLaunchKernelGGL(grouped_transpose_kernel<float>, dim3(grid), dim3(256), 0, stream, items, num_items);
  return hipGetLastError();
}

// ===================================================================== configurations
struct GemmVariant {
  int bm, bn, threads, occ;  // occ: workgroups resident per CU (LDS / register bound)
  const char* name;
};

// 0: members with N, K <= 64 (one K step); 1: 128x128; 2: 256x256 (8 waves);
// 3: fp32 64x64; 4-5: direct-to-LDS (bf16, aligned rows, K % 8 == 0):
// 256x256 8 waves, 128x128 4 waves; 6: fp32 64x128 (a fused LayerNorm over
// fp32 rows of 65 to 128 columns); 7: skinny members (every K, N <= 8), fp32 or
// bf16, streamed with no MFMA; 8: fp32 32x128, 4 waves across the columns
// (groups with fewer 64-row tiles than CUs); 9: streaming bf16 members
// (every K, N <= 64, multiples of 8, aligned rows; no fused LayerNorm); 10:
// fp32 16x128, operands loaded straight into MFMA registers (small groups).
static const GemmVariant kVariants[] = {
    {128, 64, 256, 4, "grouped_gemm_bf16_128x64x64_w4x1_s1"},
    {128, 128, 256, 2, "grouped_gemm_bf16_128x128x64_w2x2_s2"},
    {256, 256, 512, 1, "grouped_gemm_bf16_256x256x64_w2x4_s2"},
    {64, 64, 256, 4, "grouped_gemm_f32_64x64x32_w2x2_s2"},
    {256, 256, 512, 1, "grouped_gemm_dma_bf16_256x256x64_w2x4"},
    {128, 128, 256, 2, "grouped_gemm_dma_bf16_128x128x64_w2x2"},
    {64, 128, 256, 1, "grouped_gemm_f32_64x128x64_w2x2_s2"},
    {kSkinnyRows, kSkinnyMax, 256, 4, "grouped_gemm_skinny"},
    {32, 128, 256, 2, "grouped_gemm_f32_32x128x64_w1x4_s2"},
    {kStreamRows, 64, 256, 8, "grouped_gemm_stream_bf16"},
    {kR16Rows, kR16Cols, 256, 2, "grouped_gemm_rows16_f32_16x128_w4"},
};
static const int kNumVariants = (int)(sizeof(kVariants) / sizeof(kVariants[0]));

// The streaming kernel: bf16 members with K, N <= 64 values, both multiples
// of 8, and 16-byte aligned x, w, y rows.
static bool gemm_stream_ok(const optimus_linear_desc* d, int32_t G) {
  for (int g = 0; g < G; ++g) {
    if (d[g].K > 64 || d[g].N > 64 || d[g].K % 8 || d[g].N % 8 || d[g].ldx % 8 || d[g].ldw % 8 || d[g].ldy % 8 ||
        ((uintptr_t)d[g].x & 15) || ((uintptr_t)d[g].w & 15) || ((uintptr_t)d[g].y & 15))
      return false;
  }
  return true;
}

// The direct-to-LDS kernels address a tile of at most 256 rows through 32-bit
// buffer offsets below 2^31 (larger offsets mark out-of-range chunks).
static bool gemm_dma_ok(const optimus_linear_desc* d, int32_t G) {
  for (int g = 0; g < G; ++g) {
    if (d[g].K % 8 || d[g].ldx % 8 || d[g].ldw % 8 || ((uintptr_t)d[g].x & 15) || ((uintptr_t)d[g].w & 15)) return false;
    if (256 * d[g].ldx * 2 >= (int64_t)1 << 31 || 256 * d[g].ldw * 2 >= (int64_t)1 << 31) return false;
  }
  return true;
}

// Transposed operands on the direct-to-LDS tiles: bf16 x and w stored
// reduction-major ([K][M] and [K][N]) with 16-byte aligned rows, M and N
// multiples of 8 (no chunk straddles a row's end), and the offsets of a
// whole reduction range below 2^31.
static bool gemm_dma_trans_ok(const optimus_linear_desc* d, int32_t G) {
  for (int g = 0; g < G; ++g) {
    if (d[g].M % 8 || d[g].N % 8 || d[g].ldx % 8 || d[g].ldw % 8 || ((uintptr_t)d[g].x & 15) ||
        ((uintptr_t)d[g].w & 15))
      return false;
    if ((d[g].K + 128) * d[g].ldx * 2 >= (int64_t)1 << 31 || (d[g].K + 128) * d[g].ldw * 2 >= (int64_t)1 << 31)
      return false;
  }
  return true;
}

// dX read straight from W on the direct-to-LDS tiles (template argument 2):
// x = dY row-major as in the forward, w = W [K_red][N] reduction-major; both
// widths multiples of 8 values, rows 16-byte aligned, offsets below 2^31.
bool gemm_dma_wt_ok(const optimus_linear_desc* d, int32_t G) {
  for (int g = 0; g < G; ++g) {
    if (d[g].N % 8 || d[g].K % 8 || d[g].ldx % 8 || d[g].ldw % 8 || ((uintptr_t)d[g].x & 15) || ((uintptr_t)d[g].w & 15))
      return false;
    if (256 * d[g].ldx * 2 >= (int64_t)1 << 31 || (d[g].K + 128) * d[g].ldw * 2 >= (int64_t)1 << 31) return false;
  }
  return true;
}

int gemm_ln_max_n(optimus_dtype dt) { return dt == OPTIMUS_F32 ? 128 : 256; }

GemmConfig gemm_pick_config(optimus_dtype dt, const optimus_linear_desc* d, int32_t G, bool ln, int pin) {
  int64_t maxN = 0, maxK = 0;
  double tiles256 = 0.0;
  for (int g = 0; g < G; ++g) {
    maxN = d[g].N > maxN ? d[g].N : maxN;
    maxK = d[g].K > maxK ? d[g].K : maxK;
    tiles256 += (double)((d[g].M + 255) / 256) * (double)((d[g].N + 255) / 256);
  }
  int v;
  const bool dma = dt == OPTIMUS_BF16 && gemm_dma_ok(d, G);
  const bool skinny = !ln && maxN <= kSkinnyMax && maxK <= kSkinnyMax;
  if (pin >= 0) {
    // a pinned tile (plan options): the direct-to-LDS variants need every
    // member's x / w rows 16-byte aligned and K % 8 == 0, a fused LayerNorm
    // a tile as wide as the widest row, the streaming kernel K, N <= 8
    bool ok;
    if (pin >= kNumVariants)
      ok = false;
    else if (pin == 7)
      ok = skinny;
    else if (pin == 9)
      ok = dt == OPTIMUS_BF16 && !ln && gemm_stream_ok(d, G);
    else if ((dt == OPTIMUS_F32) != (pin == 3 || pin == 6 || pin == 8 || pin == 10))
      ok = false;
    else
      ok = (dt == OPTIMUS_F32 || pin < 4 || dma) && (!ln || kVariants[pin].bn >= maxN);
    if (!ok) return GemmConfig{0, 0, -1, 0, 0, "unsupported"};
    v = pin;
  } else if (skinny) {
    v = 7;
  } else if (dt == OPTIMUS_F32) {
    v = (ln && maxN > 64) ? 6 : 3;
    // a group of fewer 32-row tiles than CUs is latency bound: 16-row tiles
    // with register-direct operands halve each workgroup's serial MFMA work
    // and spread it over twice the CUs (tiny_group's eight members of 512
    // rows: 15.7 us on 64-row tiles, 9.2 on 32-row tiles)
    double tiles32 = 0.0;
    for (int g = 0; g < G; ++g) tiles32 += (double)((d[g].M + 31) / 32) * (double)((d[g].N + 127) / 128);
    if (tiles32 < device_cu_count() && maxK <= 1024) v = 10;
  } else if (maxN <= 64 && maxK <= 64) {
    v = (!ln && gemm_stream_ok(d, G)) ? 9 : 0;
  } else if (tiles256 >= 0.5 * device_cu_count() || (ln && maxN > 128)) {
    // measured over groups of 64 to 4096 256x256 tiles: the 256x256 tile wins
    // from half a tile per CU on (and is the one that holds rows past 128)
    v = dma ? 4 : 2;
  } else {
    // smaller groups need the 128x128 tile to spread over the CUs
    v = dma ? 5 : 1;
  }
  const GemmVariant& k = kVariants[v];
  return GemmConfig{k.bm, k.bn, v, k.threads, k.occ, k.name};
}

// Workgroups of one kernel instance that fit on a CU at once (registers, LDS).
static hipError_t resident_of(const void* kfn, int threads, size_t smem, int* out) {
  int b = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, kfn, threads, smem);
  if (e != hipSuccess) return e;
  *out = b;
  return hipSuccess;
}

// One kernel instance: the dynamic LDS limit is raised once per instance; with
// `occ` set the instance is not launched and its resident workgroups per CU
// are reported instead.
#define OPTIMUS_LAUNCH_ONE(KFN, SMEM, NT)                                                                          \
  {                                                                                                                \
    auto kfn = KFN;                                                                                                \
    static bool attr_set = false; /* the attribute is device-independent; setting it twice is harmless */         \
    if ((SMEM) > 65536 && !attr_set) {                                                                             \
      hipError_t e = hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)(SMEM)); \
      if (e != hipSuccess) return e;                                                                               \
      attr_set = true;                                                                                             \
    }                                                                                                              \
    if (occ) return resident_of((const void*)kfn, (NT), (SMEM), occ);                                              \
    hipLaunchKernelGGL(kfn, dim3(grid), dim3(NT), (SMEM), stream, descs, tiles, n);                                \
  }

static hipError_t launch_stream(optimus_act act, const DevLinear* descs, const GemmTile* tiles, int32_t n,
                                int32_t grid, hipStream_t stream, int* occ) {
  constexpr size_t smem = kStreamLds;
  switch (act) {
    case OPTIMUS_ACT_NONE: OPTIMUS_LAUNCH_ONE((grouped_gemm_stream_kernel<0>), smem, 256); break;
    case OPTIMUS_ACT_RELU: OPTIMUS_LAUNCH_ONE((grouped_gemm_stream_kernel<1>), smem, 256); break;
    case OPTIMUS_ACT_SIGMOID: OPTIMUS_LAUNCH_ONE((grouped_gemm_stream_kernel<2>), smem, 256); break;
    case OPTIMUS_ACT_TANH: OPTIMUS_LAUNCH_ONE((grouped_gemm_stream_kernel<3>), smem, 256); break;
    case OPTIMUS_ACT_SILU: OPTIMUS_LAUNCH_ONE((grouped_gemm_stream_kernel<4>), smem, 256); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T>
static hipError_t launch_skinny(optimus_act act, const DevLinear* descs, const GemmTile* tiles, int32_t n,
                                int32_t grid, hipStream_t stream, int* occ) {
  switch (act) {
    case OPTIMUS_ACT_NONE: OPTIMUS_LAUNCH_ONE((grouped_gemm_skinny_kernel<T, 0>), 0, 256); break;
    case OPTIMUS_ACT_RELU: OPTIMUS_LAUNCH_ONE((grouped_gemm_skinny_kernel<T, 1>), 0, 256); break;
    case OPTIMUS_ACT_SIGMOID: OPTIMUS_LAUNCH_ONE((grouped_gemm_skinny_kernel<T, 2>), 0, 256); break;
    case OPTIMUS_ACT_TANH: OPTIMUS_LAUNCH_ONE((grouped_gemm_skinny_kernel<T, 3>), 0, 256); break;
    case OPTIMUS_ACT_SILU: OPTIMUS_LAUNCH_ONE((grouped_gemm_skinny_kernel<T, 4>), 0, 256); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T, int BM, int BN, int BK, int WM, int WN, int STAGES, int PRE = 0>
static hipError_t launch_shape(optimus_act act, bool ln, const DevLinear* descs, const GemmTile* tiles, int32_t n,
                               int32_t grid, hipStream_t stream, int* occ) {
  using S = GemmShape<T, BM, BN, BK, WM, WN, STAGES>;
#define OPTIMUS_GEMM_LAUNCH(A)                                                                                   \
  if (ln)                                                                                                        \
    OPTIMUS_LAUNCH_ONE((grouped_gemm_kernel<T, BM, BN, BK, WM, WN, STAGES, (A) | 8, 0, PRE>), S::LDS_BYTES_LN, S::NT) \
  else                                                                                                           \
    OPTIMUS_LAUNCH_ONE((grouped_gemm_kernel<T, BM, BN, BK, WM, WN, STAGES, (A), 0, PRE>), S::LDS_BYTES, S::NT)
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

static hipError_t launch_rows16(optimus_act act, bool ln, const DevLinear* descs, const GemmTile* tiles, int32_t n,
                               int32_t grid, hipStream_t stream, int* occ) {
#define OPTIMUS_R16_LAUNCH(A)                                                 \
  if (ln)                                                                     \
    OPTIMUS_LAUNCH_ONE((grouped_gemm_rows16_kernel<(A) | 8>), 0, 256) \
  else                                                                        \
    OPTIMUS_LAUNCH_ONE((grouped_gemm_rows16_kernel<(A)>), 0, 256)
  switch (act) {
    case OPTIMUS_ACT_NONE: OPTIMUS_R16_LAUNCH(0); break;
    case OPTIMUS_ACT_RELU: OPTIMUS_R16_LAUNCH(1); break;
    case OPTIMUS_ACT_SIGMOID: OPTIMUS_R16_LAUNCH(2); break;
    case OPTIMUS_ACT_TANH: OPTIMUS_R16_LAUNCH(3); break;
    case OPTIMUS_ACT_SILU: OPTIMUS_R16_LAUNCH(4); break;
    default: return hipErrorInvalidValue;
  }
#undef OPTIMUS_R16_LAUNCH
  return hipGetLastError();
}

// Backward GEMM instances: no bias, no activation, no LayerNorm.
template <typename T, int BM, int BN, int BK, int WM, int WN, int STAGES>
static hipError_t launch_trans(int tr, const DevLinear* descs, const GemmTile* tiles, int32_t n, int32_t grid,
                               hipStream_t stream, int* occ) {
  using S = GemmShape<T, BM, BN, BK, WM, WN, STAGES>;
  if (tr == 3)
    OPTIMUS_LAUNCH_ONE((grouped_gemm_kernel<T, BM, BN, BK, WM, WN, STAGES, 0, 3>), S::LDS_BYTES, S::NT)
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN>
static hipError_t launch_dma_trans(int tr, optimus_act act, const DevLinear* descs, const GemmTile* tiles, int32_t n,
                                   int32_t grid, hipStream_t stream, int* occ) {
  using S = DmaShape<BM, BN, WM, WN>;
  if (tr == 3)
    OPTIMUS_LAUNCH_ONE((grouped_gemm_dma_kernel<BM, BN, WM, WN, 0, 3>), S::LDS_BYTES, S::NT)
  else if (tr == 2) {
    switch (act) {
      case OPTIMUS_ACT_NONE: OPTIMUS_LAUNCH_ONE((grouped_gemm_dma_kernel<BM, BN, WM, WN, 0, 2>), S::LDS_BYTES, S::NT); break;
      case OPTIMUS_ACT_RELU: OPTIMUS_LAUNCH_ONE((grouped_gemm_dma_kernel<BM, BN, WM, WN, 1, 2>), S::LDS_BYTES, S::NT); break;
      case OPTIMUS_ACT_SIGMOID: OPTIMUS_LAUNCH_ONE((grouped_gemm_dma_kernel<BM, BN, WM, WN, 2, 2>), S::LDS_BYTES, S::NT); break;
      case OPTIMUS_ACT_TANH: OPTIMUS_LAUNCH_ONE((grouped_gemm_dma_kernel<BM, BN, WM, WN, 3, 2>), S::LDS_BYTES, S::NT); break;
      case OPTIMUS_ACT_SILU: OPTIMUS_LAUNCH_ONE((grouped_gemm_dma_kernel<BM, BN, WM, WN, 4, 2>), S::LDS_BYTES, S::NT); break;
      default: return hipErrorInvalidValue;
    }
  } else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN>
static hipError_t launch_dma(optimus_act act, bool ln, const DevLinear* descs, const GemmTile* tiles, int32_t n,
                             int32_t grid, hipStream_t stream, int* occ) {
  using S = DmaShape<BM, BN, WM, WN>;
#define OPTIMUS_DMA_LAUNCH(A)                                                                      \
  if (ln)                                                                                          \
    OPTIMUS_LAUNCH_ONE((grouped_gemm_dma_kernel<BM, BN, WM, WN, (A) | 8>), S::LDS_BYTES_LN, S::NT) \
  else                                                                                             \
    OPTIMUS_LAUNCH_ONE((grouped_gemm_dma_kernel<BM, BN, WM, WN, (A)>), S::LDS_BYTES, S::NT)
  switch (act) {
    case OPTIMUS_ACT_NONE: OPTIMUS_DMA_LAUNCH(0); break;
    case OPTIMUS_ACT_RELU: OPTIMUS_DMA_LAUNCH(1); break;
    case OPTIMUS_ACT_SIGMOID: OPTIMUS_DMA_LAUNCH(2); break;
    case OPTIMUS_ACT_TANH: OPTIMUS_DMA_LAUNCH(3); break;
    case OPTIMUS_ACT_SILU: OPTIMUS_DMA_LAUNCH(4); break;
    default: return hipErrorInvalidValue;
  }
#undef OPTIMUS_DMA_LAUNCH
  return hipGetLastError();
}
#undef OPTIMUS_LAUNCH_ONE

static hipError_t gemm_dispatch(const GemmConfig& cfg, optimus_dtype dt, optimus_act act, bool ln, int tr,
                                const DevLinear* descs, const GemmTile* tiles, int32_t n, int32_t grid,
                                hipStream_t stream, int* occ) {
  if (tr) {
    if (ln || (act != OPTIMUS_ACT_NONE && tr != 2)) return hipErrorInvalidValue;
    switch (cfg.variant) {
      case 1: return launch_trans<bf16_t, 128, 128, 64, 2, 2, 2>(tr, descs, tiles, n, grid, stream, occ);
      case 2: return launch_trans<bf16_t, 256, 256, 64, 2, 4, 2>(tr, descs, tiles, n, grid, stream, occ);
      case 3: return launch_trans<float, 64, 64, 32, 2, 2, 2>(tr, descs, tiles, n, grid, stream, occ);
      case 4: return launch_dma_trans<256, 256, 2, 4>(tr, act, descs, tiles, n, grid, stream, occ);
      case 5: return launch_dma_trans<128, 128, 2, 2>(tr, act, descs, tiles, n, grid, stream, occ);
      case 6: return launch_trans<float, 64, 128, 64, 2, 2, 2>(tr, descs, tiles, n, grid, stream, occ);
      default: return hipErrorInvalidValue;
    }
  }
  switch (cfg.variant) {
    case 0: return launch_shape<bf16_t, 128, 64, 64, 4, 1, 1>(act, ln, descs, tiles, n, grid, stream, occ);
    case 1: return launch_shape<bf16_t, 128, 128, 64, 2, 2, 2>(act, ln, descs, tiles, n, grid, stream, occ);
    case 2: return launch_shape<bf16_t, 256, 256, 64, 2, 4, 2>(act, ln, descs, tiles, n, grid, stream, occ);
    case 3: return launch_shape<float, 64, 64, 32, 2, 2, 2>(act, ln, descs, tiles, n, grid, stream, occ);
    case 4: return launch_dma<256, 256, 2, 4>(act, ln, descs, tiles, n, grid, stream, occ);
    case 5: return launch_dma<128, 128, 2, 2>(act, ln, descs, tiles, n, grid, stream, occ);
    case 6: return launch_shape<float, 64, 128, 64, 2, 2, 2>(act, ln, descs, tiles, n, grid, stream, occ);
    case 8: return launch_shape<float, 32, 128, 64, 1, 4, 2, 4>(act, ln, descs, tiles, n, grid, stream, occ);
    case 10:
      if (dt != OPTIMUS_F32) return hipErrorInvalidValue;
      return launch_rows16(act, ln, descs, tiles, n, grid, stream, occ);
    case 9:
      if (ln || dt != OPTIMUS_BF16) return hipErrorInvalidValue;
      return launch_stream(act, descs, tiles, n, grid, stream, occ);
    case 7:
      if (ln) return hipErrorInvalidValue;
      return dt == OPTIMUS_F32 ? launch_skinny<float>(act, descs, tiles, n, grid, stream, occ)
                               : launch_skinny<bf16_t>(act, descs, tiles, n, grid, stream, occ);
    default: return hipErrorInvalidValue;
  }
}

hipError_t gemm_launch(const GemmConfig& cfg, optimus_dtype dt, optimus_act act, bool ln, const DevLinear* descs,
                       const GemmTile* tiles, int32_t num_tiles, int32_t grid, hipStream_t stream, int tr) {
  if (num_tiles <= 0) return hipSuccess;
  return gemm_dispatch(cfg, dt, act, ln, tr, descs, tiles, num_tiles, grid, stream, nullptr);
}

// Backward GEMMs (transposed operands): 256x256 from half a tile per CU on,
// else 128x128, direct-to-LDS when every member allows it, else register-
// staged; fp32 64x64.
GemmConfig gemm_pick_config_trans(optimus_dtype dt, const optimus_linear_desc* d, int32_t G, bool split_k, int tile,
                                  int pin) {
  double tiles256 = 0.0, area = 0.0;
  for (int g = 0; g < G; ++g) {
    tiles256 += (double)((d[g].M + 255) / 256) * (double)((d[g].N + 255) / 256);
    area += (double)d[g].M * (double)d[g].N;
  }
  // the share of the 256x256 tiles' area that holds output: narrow members
  // (N of 64 or 128) leave most of a large tile idle
  const double fill256 = area / (tiles256 * 65536.0);
  // a split reduction fills the machine with the large tile's better per-tile rate
  const bool dma = dt == OPTIMUS_BF16 && gemm_dma_trans_ok(d, G);
  int v;
  if (pin >= 0) {
    // a pinned tile (plan options): 1, 2 register-staged, 4, 5 direct-to-LDS
    // where every member allows it; fp32 3, 6
    const bool ok = dt == OPTIMUS_F32 ? (pin == 3 || pin == 6)
                                      : (pin == 1 || pin == 2 || ((pin == 4 || pin == 5) && dma));
    if (!ok) return GemmConfig{0, 0, -1, 0, 0, "unsupported"};
    v = pin;
  } else {
    // tile = 256 or 128 asks for that bf16 tile edge; 0 chooses by the fill rule
    const bool big = tile ? tile == 256 : fill256 >= 0.75 && (split_k || tiles256 >= 0.5 * device_cu_count());
    v = dt == OPTIMUS_F32 ? 3 : big ? (dma ? 4 : 2) : (dma ? 5 : 1);
  }
  const GemmVariant& k = kVariants[v];
  return GemmConfig{k.bm, k.bn, v, k.threads, k.occ, k.name};
}

int gemm_resident_per_cu(const GemmConfig& cfg, optimus_dtype dt, optimus_act act, bool ln, int tr) {
  int occ = 0;
  if (gemm_dispatch(cfg, dt, act, ln, tr, nullptr, nullptr, 0, 0, nullptr, &occ) != hipSuccess || occ < 1) {
    (void)hipGetLastError();
    return cfg.occ;
  }
  return occ;
}

}  // namespace optimus
