// Memory-bound grouped kernels of liboptimus for gfx950:
//   - grouped row-wise LayerNorm (+ fused activation)  -- Table 1 batch_layernorm
//   - grouped pointwise activation                      -- Table 1 batch_relu/sigmoid/tanh, x*sigmoid(x)
//   - fused split -> per-piece LayerNorm/activation -> concat, one launch for the
//     whole row (paper Sec. 3.2 chained example; appendix Sec. 8.1 split-concat)
//
// Grouped kernels walk a device table of (member, row range) tiles written by
// the planner, so one launch serves members of different shapes (Sec. 3.2
// group fusion: instances keep their own layouts and sizes).
#include "device_common.h"

namespace optimus {

// ===================================================================== LayerNorm
// A row of one member is handled by a group of L lanes (L = power of two set
// per member by the planner, so that L * MAXC chunks of 16 bytes cover the
// row); a wave handles 64 / L rows at a time and the four waves of a block
// take consecutive row slots, so the lanes of a wave read consecutive 16-byte
// chunks of consecutive rows. Statistics are in fp32: mean first, then the
// centred sum of squares over the row held in registers (two passes, no
// cancellation), reduced across the L lanes with DPP / swizzle moves.
template <typename T, int ACT, int MAXC>
__device__ __forceinline__ void ln_rows_vec(const DevRows& d, const RowTile& rt, int lane, int wave) {
  constexpr int VEC = Elem<T>::VEC;
  const int L = d.lanes;
  const int rpw = 64 / L;
  const int sub = lane / L;
  const int li = lane & (L - 1);
  const int cpr = d.cols / VEC;

  float g[MAXC][VEC], b[MAXC][VEC];
#pragma unroll
  for (int j = 0; j < MAXC; ++j) {
    const int c = j * L + li;
#pragma unroll
    for (int e = 0; e < VEC; ++e) { g[j][e] = 1.f; b[j][e] = 0.f; }
    if (c < cpr) {
      if (d.gamma) Elem<T>::unpack(ld16((const char*)d.gamma + (int64_t)c * 16), g[j]);
      if (d.beta) Elem<T>::unpack(ld16((const char*)d.beta + (int64_t)c * 16), b[j]);
    }
  }
  const int rpb = 4 * rpw;
  const int end = rt.row0 + rt.nrows;
  for (int base = rt.row0; base < end; base += rpb) {
    const int r = base + wave * rpw + sub;
    const bool valid = r < end;
    float x[MAXC][VEC];
    const char* xr = (const char*)d.x + (int64_t)r * d.ldx * sizeof(T);
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = j * L + li;
      if (valid && c < cpr) {
        Elem<T>::unpack(ld16_nt(xr + (int64_t)c * 16), x[j]);
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) x[j][e] = 0.f;
      }
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < MAXC; ++j)
#pragma unroll
      for (int e = 0; e < VEC; ++e) s += x[j][e];
    const float mean = group_sum(s, L) * d.inv_cols;
    float q = 0.f;
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const bool in = valid && (j * L + li) < cpr;
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float t = x[j][e] - mean;
        q += in ? t * t : 0.f;
      }
    }
    const float rstd = __builtin_amdgcn_rsqf(group_sum(q, L) * d.inv_cols + d.eps);
    char* yr = (char*)d.y + (int64_t)r * d.ldy * sizeof(T);
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = j * L + li;
      if (valid && c < cpr) {
        float o[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) o[e] = act_apply<ACT>((x[j][e] - mean) * rstd * g[j][e] + b[j][e]);
        st16_nt(yr + (int64_t)c * 16, Elem<T>::pack(o));
      }
    }
  }
}

// Any shape, any alignment: one wave per row, three passes over global memory.
template <typename T, int ACT>
__device__ __forceinline__ void ln_rows_scalar(const DevRows& d, const RowTile& rt, int lane, int wave) {
  const int end = rt.row0 + rt.nrows;
  for (int r = rt.row0 + wave; r < end; r += 4) {
    const int64_t xo = (int64_t)r * d.ldx, yo = (int64_t)r * d.ldy;
    float s = 0.f;
    for (int c = lane; c < d.cols; c += 64) s += Elem<T>::load1(d.x, xo + c);
    const float mean = group_sum(s, 64) * d.inv_cols;
    float q = 0.f;
    for (int c = lane; c < d.cols; c += 64) {
      const float t = Elem<T>::load1(d.x, xo + c) - mean;
      q += t * t;
    }
    const float rstd = __builtin_amdgcn_rsqf(group_sum(q, 64) * d.inv_cols + d.eps);
    // All reads of this row are complete (the reductions above depend on
    // them), so writing in place is safe.
    for (int c = lane; c < d.cols; c += 64) {
      const float gm = d.gamma ? Elem<T>::load1(d.gamma, c) : 1.f;
      const float bt = d.beta ? Elem<T>::load1(d.beta, c) : 0.f;
      Elem<T>::store1(d.y, yo + c, act_apply<ACT>((Elem<T>::load1(d.x, xo + c) - mean) * rstd * gm + bt));
    }
  }
}

template <typename T>
constexpr int ln_maxc() { return 4; }

template <typename T, int ACT>
__global__ __launch_bounds__(kRowThreads) void grouped_layernorm_kernel(const DevRows* __restrict__ descs,
                                                                        const RowTile* __restrict__ tiles,
                                                                        int32_t num_tiles) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int t = blockIdx.x; t < num_tiles; t += gridDim.x) {
    const RowTile rt = tiles[t];
    const DevRows d = descs[rt.member];
    if (d.vec && d.lanes > 0)
      ln_rows_vec<T, ACT, ln_maxc<T>()>(d, rt, lane, wave);
    else
      ln_rows_scalar<T, ACT>(d, rt, lane, wave);
  }
}

// ===================================================================== pointwise
// Same row/lane mapping as the LayerNorm kernel, without the reductions; a
// lane group loops over the row's chunks (any row length).
template <typename T, int ACT>
__global__ __launch_bounds__(kRowThreads) void grouped_pointwise_kernel(const DevRows* __restrict__ descs,
                                                                        const RowTile* __restrict__ tiles,
                                                                        int32_t num_tiles) {
  constexpr int VEC = Elem<T>::VEC;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int t = blockIdx.x; t < num_tiles; t += gridDim.x) {
    const RowTile rt = tiles[t];
    const DevRows d = descs[rt.member];
    const int end = rt.row0 + rt.nrows;
    if (d.vec) {
      const int L = d.lanes, rpw = 64 / L, sub = lane / L, li = lane & (L - 1);
      const int cpr = d.cols / VEC;
      for (int r = rt.row0 + wave * rpw + sub; r < end; r += 4 * rpw) {
        const char* xr = (const char*)d.x + (int64_t)r * d.ldx * sizeof(T);
        char* yr = (char*)d.y + (int64_t)r * d.ldy * sizeof(T);
        for (int c = li; c < cpr; c += L) {
          float v[VEC];
          Elem<T>::unpack(ld16_nt(xr + (int64_t)c * 16), v);
#pragma unroll
          for (int e = 0; e < VEC; ++e) v[e] = act_apply<ACT>(v[e]);
          st16_nt(yr + (int64_t)c * 16, Elem<T>::pack(v));
        }
      }
    } else {
      for (int r = rt.row0 + wave; r < end; r += 4) {
        const int64_t xo = (int64_t)r * d.ldx, yo = (int64_t)r * d.ldy;
        for (int c = lane; c < d.cols; c += 64) Elem<T>::store1(d.y, yo + c, act_apply<ACT>(Elem<T>::load1(d.x, xo + c)));
      }
    }
  }
}

// ===================================================================== split-op-cat
// One wave owns one whole row of the [rows, D] tensor: step j, lane l holds
// 16-byte chunk c = 64 j + l, so every step reads 1 KB of the row contiguously
// and writes it back at the same columns of `out` -- the split and the concat
// are index arithmetic only. Piece statistics: chunk partial sums go to a
// per-wave LDS array; each lane then sums one or two planner-built runs of
// chunks that lie in a single piece and adds the run total into that piece's
// LDS accumulator; every chunk then reads its piece's statistic back. Two
// passes (mean, then centred squares) as in the row kernel above. Piece gamma
// and beta are staged once per block in LDS.
template <typename T, int ACT, int STEPS>
__global__ __launch_bounds__(kSocThreads) void split_op_cat_kernel(const DevSoc* __restrict__ sp) {
  constexpr int VEC = Elem<T>::VEC;
  extern __shared__ __align__(16) char smem[];
  const DevSoc s = *sp;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nch = s.nchunks, npc = s.n_pieces;
  // LDS layout: gamma [nch * 16 B] | beta [nch * 16 B] | part [4][nch] f32 | stat [4][2][npc] f32
  char* lg = smem;
  char* lb = lg + (size_t)nch * 16;
  float* part = (float*)(lb + (size_t)nch * 16) + wave * nch;
  float* stat = (float*)(lb + (size_t)nch * 16) + 4 * nch + wave * 2 * npc;
  for (int c = threadIdx.x; c < nch; c += kSocThreads) {
    u32x4 gv, bv;
    if (s.gamma) gv = ld16((const char*)s.gamma + (int64_t)c * 16);
    if (s.beta) bv = ld16((const char*)s.beta + (int64_t)c * 16);
    if (!s.gamma) { float one[VEC]; for (int e = 0; e < VEC; ++e) one[e] = 1.f; gv = Elem<T>::pack(one); }
    if (!s.beta) { float z[VEC]; for (int e = 0; e < VEC; ++e) z[e] = 0.f; bv = Elem<T>::pack(z); }
    *(u32x4*)(lg + (size_t)c * 16) = gv;
    *(u32x4*)(lb + (size_t)c * 16) = bv;
  }
  __syncthreads();

  // per-lane static data: piece of each owned chunk, its 1/width, the lane's runs
  int pc[STEPS];
  float invw[STEPS];
#pragma unroll
  for (int j = 0; j < STEPS; ++j) {
    const int c = j * 64 + lane;
    pc[j] = c < nch ? s.chunk_piece[c] : 0;
    invw[j] = c < nch ? s.pieces[pc[j]].inv_width : 0.f;
  }
  SocTask tk0 = {0, 0, 0, 0}, tk1 = {0, 0, 0, 0};
  if (lane < s.n_tasks) tk0 = s.tasks[lane];
  if (lane + 64 < s.n_tasks) tk1 = s.tasks[lane + 64];

  for (int row = blockIdx.x * 4 + wave; row < s.rows; row += gridDim.x * 4) {
    const char* xr = (const char*)s.in + (int64_t)row * s.ldin * sizeof(T);
    char* yr = (char*)s.out + (int64_t)row * s.ldout * sizeof(T);
    float x[STEPS][VEC];
#pragma unroll
    for (int j = 0; j < STEPS; ++j) {
      const int c = j * 64 + lane;
      if (c < nch) {
        Elem<T>::unpack(ld16_nt(xr + (int64_t)c * 16), x[j]);
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) x[j][e] = 0.f;
      }
    }
    float mean[STEPS], rstd[STEPS];
    if (s.apply_ln) {
      for (int p = lane; p < 2 * npc; p += 64) stat[p] = 0.f;
      // pass 1: sums
#pragma unroll
      for (int j = 0; j < STEPS; ++j) {
        const int c = j * 64 + lane;
        float t = 0.f;
#pragma unroll
        for (int e = 0; e < VEC; ++e) t += x[j][e];
        if (c < nch) part[c] = t;
      }
      lds_wave_sync();
      {
        float a = 0.f, b2 = 0.f;
        for (int c = tk0.c0; c < tk0.c1; ++c) a += part[c];
        for (int c = tk1.c0; c < tk1.c1; ++c) b2 += part[c];
        if (tk0.c1 > tk0.c0) atomicAdd(&stat[tk0.piece], a);
        if (tk1.c1 > tk1.c0) atomicAdd(&stat[tk1.piece], b2);
      }
      lds_wave_sync();
#pragma unroll
      for (int j = 0; j < STEPS; ++j) mean[j] = stat[pc[j]] * invw[j];
      // pass 2: centred squares
#pragma unroll
      for (int j = 0; j < STEPS; ++j) {
        const int c = j * 64 + lane;
        float t = 0.f;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const float u = x[j][e] - mean[j];
          t += u * u;
        }
        if (c < nch) part[c] = t;
      }
      lds_wave_sync();
      {
        float a = 0.f, b2 = 0.f;
        for (int c = tk0.c0; c < tk0.c1; ++c) a += part[c];
        for (int c = tk1.c0; c < tk1.c1; ++c) b2 += part[c];
        if (tk0.c1 > tk0.c0) atomicAdd(&stat[npc + tk0.piece], a);
        if (tk1.c1 > tk1.c0) atomicAdd(&stat[npc + tk1.piece], b2);
      }
      lds_wave_sync();
#pragma unroll
      for (int j = 0; j < STEPS; ++j) rstd[j] = __builtin_amdgcn_rsqf(stat[npc + pc[j]] * invw[j] + s.eps);
      lds_wave_sync();  // statistics read before the next row clears them
    }
#pragma unroll
    for (int j = 0; j < STEPS; ++j) {
      const int c = j * 64 + lane;
      if (c < nch) {
        float o[VEC];
        if (s.apply_ln) {
          float g[VEC], b[VEC];
          Elem<T>::unpack(*(const u32x4*)(lg + (size_t)c * 16), g);
          Elem<T>::unpack(*(const u32x4*)(lb + (size_t)c * 16), b);
#pragma unroll
          for (int e = 0; e < VEC; ++e) o[e] = act_apply<ACT>((x[j][e] - mean[j]) * rstd[j] * g[e] + b[e]);
        } else {
#pragma unroll
          for (int e = 0; e < VEC; ++e) o[e] = act_apply<ACT>(x[j][e]);
        }
        st16_nt(yr + (int64_t)c * 16, Elem<T>::pack(o));
      }
    }
  }
}

// ===================================================================== launchers
#define OPTIMUS_ACT_SWITCH(ACTV, ...)                                  \
  switch (ACTV) {                                                      \
    case OPTIMUS_ACT_NONE: { constexpr int A = 0; __VA_ARGS__; } break;    \
    case OPTIMUS_ACT_RELU: { constexpr int A = 1; __VA_ARGS__; } break;    \
    case OPTIMUS_ACT_SIGMOID: { constexpr int A = 2; __VA_ARGS__; } break; \
    case OPTIMUS_ACT_TANH: { constexpr int A = 3; __VA_ARGS__; } break;    \
    case OPTIMUS_ACT_SILU: { constexpr int A = 4; __VA_ARGS__; } break;    \
    default: return hipErrorInvalidValue;                              \
  }

hipError_t layernorm_launch(optimus_dtype dt, optimus_act act, const DevRows* descs, const RowTile* tiles,
                            int32_t num_tiles, int32_t grid, hipStream_t stream) {
  if (num_tiles <= 0) return hipSuccess;
  if (dt == OPTIMUS_BF16) {
    OPTIMUS_ACT_SWITCH(act, hipLaunchKernelGGL((grouped_layernorm_kernel<bf16_t, A>), dim3(grid), dim3(kRowThreads), 0,
                                               stream, descs, tiles, num_tiles));
  } else {
    OPTIMUS_ACT_SWITCH(act, hipLaunchKernelGGL((grouped_layernorm_kernel<float, A>), dim3(grid), dim3(kRowThreads), 0,
                                               stream, descs, tiles, num_tiles));
  }
  return hipGetLastError();
}

hipError_t pointwise_launch(optimus_dtype dt, optimus_act act, const DevRows* descs, const RowTile* tiles,
                            int32_t num_tiles, int32_t grid, hipStream_t stream) {
  if (num_tiles <= 0) return hipSuccess;
  if (dt == OPTIMUS_BF16) {
    OPTIMUS_ACT_SWITCH(act, hipLaunchKernelGGL((grouped_pointwise_kernel<bf16_t, A>), dim3(grid), dim3(kRowThreads), 0,
                                               stream, descs, tiles, num_tiles));
  } else {
    OPTIMUS_ACT_SWITCH(act, hipLaunchKernelGGL((grouped_pointwise_kernel<float, A>), dim3(grid), dim3(kRowThreads), 0,
                                               stream, descs, tiles, num_tiles));
  }
  return hipGetLastError();
}

template <typename T, int ACT>
static hipError_t soc_launch_t(const DevSoc* soc, int32_t nchunks, int32_t n_pieces, int32_t grid, hipStream_t stream) {
  const size_t smem = (size_t)nchunks * 32 + (size_t)4 * nchunks * 4 + (size_t)4 * 2 * n_pieces * 4;
  const int steps = (nchunks + 63) / 64;
  if (steps <= 4)
    hipLaunchKernelGGL((split_op_cat_kernel<T, ACT, 4>), dim3(grid), dim3(kSocThreads), smem, stream, soc);
  else if (steps <= 8)
    hipLaunchKernelGGL((split_op_cat_kernel<T, ACT, 8>), dim3(grid), dim3(kSocThreads), smem, stream, soc);
  else
    hipLaunchKernelGGL((split_op_cat_kernel<T, ACT, 16>), dim3(grid), dim3(kSocThreads), smem, stream, soc);
  return hipGetLastError();
}

hipError_t soc_launch(optimus_dtype dt, optimus_act act, const DevSoc* soc, int32_t rows, int32_t nchunks,
                      int32_t n_pieces, int32_t n_tasks, int32_t grid, hipStream_t stream) {
  (void)rows;
  (void)n_tasks;
  if (nchunks <= 0 || nchunks > kSocMaxChunks || n_pieces > kSocMaxPieces) return hipErrorInvalidValue;
  if (dt == OPTIMUS_BF16) {
    OPTIMUS_ACT_SWITCH(act, return soc_launch_t<bf16_t, A>(soc, nchunks, n_pieces, grid, stream));
  } else {
    OPTIMUS_ACT_SWITCH(act, return soc_launch_t<float, A>(soc, nchunks, n_pieces, grid, stream));
  }
  return hipSuccess;
}

}  // namespace optimus
