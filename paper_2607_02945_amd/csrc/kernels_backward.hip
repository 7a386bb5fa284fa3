// Row-wise backward kernels of liboptimus for gfx950 (training: the
// gradients of the grouped operators, the training column of Table 3):
//   - grouped activation backward   dx = dy * act'(x)
//   - grouped LayerNorm backward    dx = rstd (g - mean(g) - xhat mean(g xhat)),
//                                   g = dy * gamma, xhat = (x - mean) rstd,
//                                   dgamma = sum_rows dy xhat, dbeta = sum_rows dy
//   - the finalize of dgamma / dbeta over the per-tile column partials
// The row mapping is the forward's: L lanes per row, a wave 64 / L rows, a
// block of four waves consecutive row slots, 16-byte chunks; the statistics
// are recomputed from x in fp32 (two passes) as the forward takes them.
#include "device_common.h"

namespace optimus {

// ===================================================================== activation
template <typename T, int ACT>
__global__ __launch_bounds__(kRowThreads) void grouped_act_backward_kernel(const DevRowsGrad* __restrict__ descs,
                                                                           const RowTile* __restrict__ tiles,
                                                                           int32_t num_tiles) {
  constexpr int VEC = Elem<T>::VEC;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  for (int t = blockIdx.x; t < num_tiles; t += gridDim.x) {
    const RowTile rt = tiles[t];
    const DevRowsGrad d = descs[rt.member];
    const int end = rt.row0 + rt.nrows;
    if (d.vec) {
      const int L = d.lanes, rpw = 64 / L, sub = lane / L, li = lane & (L - 1);
      const int cpr = d.cols / VEC;
      for (int r = rt.row0 + wave * rpw + sub; r < end; r += 4 * rpw) {
        const char* xr = (const char*)d.x + (int64_t)r * d.ldx * sizeof(T);
        const char* gr = (const char*)d.dy + (int64_t)r * d.lddy * sizeof(T);
        char* orow = (char*)d.dx + (int64_t)r * d.lddx * sizeof(T);
        int c = li;
        for (; c + L < cpr; c += 2 * L) {
          u32x4 xv[2], gv[2];
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            xv[u] = ld16_nt(xr + (int64_t)(c + u * L) * 16);
            gv[u] = ld16_nt(gr + (int64_t)(c + u * L) * 16);
          }
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            float a[VEC], g[VEC];
            Elem<T>::unpack(xv[u], a);
            Elem<T>::unpack(gv[u], g);
#pragma unroll
            for (int e = 0; e < VEC; ++e) a[e] = g[e] * act_grad<ACT>(a[e]);
            st16_nt(orow + (int64_t)(c + u * L) * 16, Elem<T>::pack(a));
          }
        }
        for (; c < cpr; c += L) {
          float a[VEC], g[VEC];
          Elem<T>::unpack(ld16_nt(xr + (int64_t)c * 16), a);
          Elem<T>::unpack(ld16_nt(gr + (int64_t)c * 16), g);
#pragma unroll
          for (int e = 0; e < VEC; ++e) a[e] = g[e] * act_grad<ACT>(a[e]);
          st16_nt(orow + (int64_t)c * 16, Elem<T>::pack(a));
        }
      }
    } else {
      for (int r = rt.row0 + wave; r < end; r += 4) {
        const int64_t xo = (int64_t)r * d.ldx, go = (int64_t)r * d.lddy, oo = (int64_t)r * d.lddx;
        for (int c = lane; c < d.cols; c += 64)
          Elem<T>::store1(d.dx, oo + c, Elem<T>::load1(d.dy, go + c) * act_grad<ACT>(Elem<T>::load1(d.x, xo + c)));
      }
    }
  }
}

// ===================================================================== LayerNorm
// 16-byte path: the row's chunks in registers (MAXC per lane), as the forward.
// Each lane keeps its columns' dgamma / dbeta sums over the rows it handles;
// at the end of the tile each wave writes its sums to its own slot sPart
// ([2][cols] in LDS, one per wave) and the block adds the four slots in a
// fixed order as the tile's partial row leaves in one coalesced pass, so the
// sums do not depend on timing.
// gamma (and beta) are staged in LDS as fp32 (sGamma, sBeta: [cols], filled
// by the caller) and read where they are used. ACT != 0: the backward of the
// fused LayerNorm + activation -- the incoming gradient is the activation
// output's, and is multiplied by act'(gamma * xhat + beta), recomputed here
// once per value: the pass that forms the row sums leaves the products in
// the wave's slot sPart (free until the tile's sums are written there) and
// the output pass reads them back (the derivative is two transcendentals per
// value; large_group's LayerNorm + tanh backward 454 -> 413 us). Keeping
// xhat there too saved nothing.
template <typename T, int MAXC, int ACT>
__device__ __forceinline__ void lnb_rows_vec(const DevRowsGrad& d, const RowTile& rt, int lane, int wave,
                                             float* sPart, const float* sGamma, const float* sBeta) {
  constexpr int VEC = Elem<T>::VEC;
  const int L = d.lanes;
  const int rpw = 64 / L;
  const int sub = lane / L;
  const int li = lane & (L - 1);
  const int cpr = d.cols / VEC;
  const bool params = d.want_params != 0;
  auto param_of = [&](const float* src, int j, float (&gm)[VEC]) {
    const int c = j * L + li;
    const f32x4* p = (const f32x4*)(src + (c < cpr ? c : 0) * VEC);
#pragma unroll
    for (int h = 0; h < VEC / 4; ++h) {
      const f32x4 v = p[h];
      gm[4 * h] = v.x;
      gm[4 * h + 1] = v.y;
      gm[4 * h + 2] = v.z;
      gm[4 * h + 3] = v.w;
    }
  };
  auto gamma_of = [&](int j, float (&gm)[VEC]) { param_of(sGamma, j, gm); };
  // the gradient entering the LayerNorm: dy, or dy * act'(gamma xhat + beta)
  auto grad_in = [&](int j, const float (&gm)[VEC], const float (&xh)[VEC], float (&g)[VEC]) {
    if constexpr (ACT != 0) {
      float be[VEC];
      param_of(sBeta, j, be);
#pragma unroll
      for (int e = 0; e < VEC; ++e) g[e] *= act_grad<ACT>(gm[e] * xh[e] + be[e]);
    }
  };
  float accG[MAXC][VEC], accB[MAXC][VEC];
#pragma unroll
  for (int j = 0; j < MAXC; ++j)
#pragma unroll
    for (int e = 0; e < VEC; ++e) accG[j][e] = accB[j][e] = 0.f;
  const int end = rt.row0 + rt.nrows;
  const int rpb = 4 * rpw;
  // The next row slot's x and dy chunks are loaded while the current one is
  // computed (as the forward kernel does).
  u32x4 rx[MAXC], rg[MAXC];
  auto fetch = [&](int r) {
    const char* xr = (const char*)d.x + (int64_t)r * d.ldx * sizeof(T);
    const char* gr = (const char*)d.dy + (int64_t)r * d.lddy * sizeof(T);
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = j * L + li;
      const bool in = r < end && c < cpr;
      rx[j] = in ? ld16_nt(xr + (int64_t)c * 16) : u32x4{0u, 0u, 0u, 0u};
      rg[j] = in ? ld16_nt(gr + (int64_t)c * 16) : u32x4{0u, 0u, 0u, 0u};
    }
  };
  fetch(rt.row0 + wave * rpw + sub);
  // every lane of the wave runs the loop the same number of times (the
  // lane-group sums need all 64); rows past the tile contribute nothing.
  // The current row stays packed (cx, cg) and is unpacked in each pass, so
  // that it and the prefetched next row fit in registers together.
  for (int base = rt.row0; base < end; base += rpb) {
    const int r = base + wave * rpw + sub;
    const bool valid = r < end;
    u32x4 cx[MAXC], cg[MAXC];
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      cx[j] = rx[j];
      cg[j] = rg[j];
    }
    if (base + rpb < end) fetch(r + rpb);
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      float x[VEC];
      Elem<T>::unpack(cx[j], x);
#pragma unroll
      for (int e = 0; e < VEC; ++e) s += x[e];
    }
    const float mean = group_sum(s, L) * d.inv_cols;
    float q = 0.f;
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const bool in = valid && (j * L + li) < cpr;
      float x[VEC];
      Elem<T>::unpack(cx[j], x);
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float t = x[e] - mean;
        q += in ? t * t : 0.f;
      }
    }
    const float rstd = __builtin_amdgcn_rsqf(group_sum(q, L) * d.inv_cols + d.eps);
    // this lane's products g * act' of chunk j, element group h (ACT != 0)
    auto gslot = [&](int j, int h) { return (f32x4*)sPart + (j * (VEC / 4) + h) * 64 + lane; };
    float sg = 0.f, sgx = 0.f;
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const bool in = valid && (j * L + li) < cpr;
      float x[VEC], g[VEC], gm[VEC], xh[VEC];
      Elem<T>::unpack(cx[j], x);
      Elem<T>::unpack(cg[j], g);
      gamma_of(j, gm);
#pragma unroll
      for (int e = 0; e < VEC; ++e) xh[e] = (x[e] - mean) * rstd;
      grad_in(j, gm, xh, g);
      if constexpr (ACT != 0) {
#pragma unroll
        for (int h = 0; h < VEC / 4; ++h) *gslot(j, h) = f32x4{g[4 * h], g[4 * h + 1], g[4 * h + 2], g[4 * h + 3]};
      }
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float gg = g[e] * gm[e];
        sg += in ? gg : 0.f;
        sgx += in ? gg * xh[e] : 0.f;
      }
    }
    const float mg = group_sum(sg, L) * d.inv_cols;
    const float mgx = group_sum(sgx, L) * d.inv_cols;
    char* orow = (char*)d.dx + (int64_t)r * d.lddx * sizeof(T);
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = j * L + li;
      if (valid && c < cpr) {
        float x[VEC], g[VEC], gm[VEC], o[VEC], xh[VEC];
        Elem<T>::unpack(cx[j], x);
        gamma_of(j, gm);
#pragma unroll
        for (int e = 0; e < VEC; ++e) xh[e] = (x[e] - mean) * rstd;
        if constexpr (ACT != 0) {
#pragma unroll
          for (int h = 0; h < VEC / 4; ++h) {
            const f32x4 v = *gslot(j, h);
            g[4 * h] = v.x;
            g[4 * h + 1] = v.y;
            g[4 * h + 2] = v.z;
            g[4 * h + 3] = v.w;
          }
        } else {
          Elem<T>::unpack(cg[j], g);
        }
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          o[e] = rstd * (g[e] * gm[e] - mg - xh[e] * mgx);
          accG[j][e] += g[e] * xh[e];
          accB[j][e] += g[e];
        }
        st16_nt(orow + (int64_t)c * 16, Elem<T>::pack(o));
      }
    }
  }
  if (params) {
    // the rpw row slots of a wave hold the same columns (lanes li + k * L):
    // add them up across the wave first, then one slot per wave goes to LDS
    for (int off = L; off < 64; off <<= 1) {
#pragma unroll
      for (int j = 0; j < MAXC; ++j)
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          accG[j][e] += __shfl_xor(accG[j][e], off);
          accB[j][e] += __shfl_xor(accB[j][e], off);
        }
    }
    // the wave's lanes of slot 0 own every column of the row exactly once
    if (sub == 0) {
#pragma unroll
      for (int j = 0; j < MAXC; ++j) {
        const int c = j * L + li;
        if (c < cpr) {
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            sPart[c * VEC + e] = accG[j][e];
            sPart[d.cols + c * VEC + e] = accB[j][e];
          }
        }
      }
    }
  }
}

// Any shape, any alignment: one wave per row, four passes over global memory;
// the wave's dgamma / dbeta sums go to its own partial row (written by its
// first row, added to by the next ones: only this wave touches it).
template <typename T, int ACT>
__device__ __forceinline__ void lnb_rows_scalar(const DevRowsGrad& d, const RowTile& rt, int lane, int wave) {
  const int end = rt.row0 + rt.nrows;
  const bool params = d.want_params != 0;
  float* pg = d.part + (int64_t)(d.part0 + rt.pad * kGradWavesPerBlock + wave) * 2 * d.cols;
  float* pb = pg + d.cols;
  bool first = true;
  for (int r = rt.row0 + wave; r < end; r += 4) {
    const int64_t xo = (int64_t)r * d.ldx, go = (int64_t)r * d.lddy, oo = (int64_t)r * d.lddx;
    float s = 0.f;
    for (int c = lane; c < d.cols; c += 64) s += Elem<T>::load1(d.x, xo + c);
    const float mean = group_sum(s, 64) * d.inv_cols;
    float q = 0.f;
    for (int c = lane; c < d.cols; c += 64) {
      const float t = Elem<T>::load1(d.x, xo + c) - mean;
      q += t * t;
    }
    const float rstd = __builtin_amdgcn_rsqf(group_sum(q, 64) * d.inv_cols + d.eps);
    // the gradient entering the LayerNorm at column c (ACT: times act' of
    // the recomputed activation input)
    auto grad_in = [&](int c, float xh) {
      float g = Elem<T>::load1(d.dy, go + c);
      if constexpr (ACT != 0) {
        const float gm = d.gamma ? Elem<T>::load1(d.gamma, c) : 1.f;
        const float be = d.beta ? Elem<T>::load1(d.beta, c) : 0.f;
        g *= act_grad<ACT>(gm * xh + be);
      }
      return g;
    };
    float sg = 0.f, sgx = 0.f;
    for (int c = lane; c < d.cols; c += 64) {
      const float xh = (Elem<T>::load1(d.x, xo + c) - mean) * rstd;
      const float gg = grad_in(c, xh) * (d.gamma ? Elem<T>::load1(d.gamma, c) : 1.f);
      sg += gg;
      sgx += gg * xh;
    }
    const float mg = group_sum(sg, 64) * d.inv_cols;
    const float mgx = group_sum(sgx, 64) * d.inv_cols;
    // every read of the row's dy is done (the sums above depend on them), so
    // dx may overwrite dy in place
    for (int c = lane; c < d.cols; c += 64) {
      const float xh = (Elem<T>::load1(d.x, xo + c) - mean) * rstd;
      const float gy = grad_in(c, xh);
      const float gg = gy * (d.gamma ? Elem<T>::load1(d.gamma, c) : 1.f);
      Elem<T>::store1(d.dx, oo + c, rstd * (gg - mg - xh * mgx));
      if (params) {
        pg[c] = first ? gy * xh : pg[c] + gy * xh;
        pb[c] = first ? gy : pb[c] + gy;
      }
    }
    first = false;
  }
  if (params && first) {  // no row for this wave: its partial row is zero
    for (int c = lane; c < d.cols; c += 64) {
      pg[c] = 0.f;
      pb[c] = 0.f;
    }
  }
}

template <typename T, int ACT>
__global__ __launch_bounds__(kRowThreads, 3) void grouped_layernorm_backward_kernel(
    const DevRowsGrad* __restrict__ descs, const RowTile* __restrict__ tiles, int32_t num_tiles) {
  // [2][cols] partials and [cols] gamma for the widest row the 16-byte path
  // holds: 64 lanes x the chunks per lane x the values per chunk
  constexpr int MAXCOLS = 64 * kLnChunksPerLane * Elem<T>::VEC;
  __shared__ __align__(16) float sPart[4][2 * MAXCOLS];  // one [2][cols] slot per wave
  __shared__ __align__(16) float sGamma[MAXCOLS];
  __shared__ __align__(16) float sBeta[ACT != 0 ? MAXCOLS : 4];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  for (int t = blockIdx.x; t < num_tiles; t += gridDim.x) {
    const RowTile rt = tiles[t];
    if (rt.member < 0) continue;  // padding of a block with fewer segments
    const DevRowsGrad d = descs[rt.member];
    if (d.vec && d.lanes > 0) {
      const bool params = d.want_params != 0;
      for (int i = tid; i < d.cols; i += kRowThreads) sGamma[i] = d.gamma ? Elem<T>::load1(d.gamma, i) : 1.f;
      if constexpr (ACT != 0)
        for (int i = tid; i < d.cols; i += kRowThreads) sBeta[i] = d.beta ? Elem<T>::load1(d.beta, i) : 0.f;
      __syncthreads();
      lnb_rows_vec<T, kLnChunksPerLane, ACT>(d, rt, lane, wave, sPart[wave], sGamma, sBeta);
      __syncthreads();  // every wave is done with sGamma and has written its slot
      if (params) {
        float* out = d.part + (int64_t)(d.part0 + rt.pad) * 2 * d.cols;
        for (int i = tid; i < 2 * d.cols; i += kRowThreads) out[i] = ((sPart[0][i] + sPart[1][i]) + sPart[2][i]) + sPart[3][i];
        __syncthreads();  // the slots are written again by the next tile
      }
    } else {
      lnb_rows_scalar<T, ACT>(d, rt, lane, wave);
    }
  }
}

// ===================================================================== finalize
// One item is kFinCols columns of one member: the four waves of a block take
// every fourth partial row each (four loads in flight per lane), then the
// four sums meet in LDS.
template <typename T>
__global__ __launch_bounds__(256) void grad_finalize_kernel(const GradFinItem* __restrict__ items, int32_t num_items) {
  __shared__ float red[2][4][kFinCols];
  const int cl = threadIdx.x % kFinCols, pg = threadIdx.x / kFinCols;
  for (int t = blockIdx.x; t < num_items; t += gridDim.x) {
    const GradFinItem it = items[t];
    const int c = it.c0 + cl;
    float sg = 0.f, sb = 0.f;
    if (c < it.cols) {
      const int64_t stride = 2 * (int64_t)it.cols;
      const float* base = it.part + c;
      int p = pg;
      for (; p + 12 < it.nparts; p += 16) {
        float g[4], b[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          g[u] = base[(int64_t)(p + 4 * u) * stride];
          b[u] = base[(int64_t)(p + 4 * u) * stride + it.cols];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          sg += g[u];
          sb += b[u];
        }
      }
      for (; p < it.nparts; p += 4) {
        sg += base[(int64_t)p * stride];
        sb += base[(int64_t)p * stride + it.cols];
      }
    }
    red[0][pg][cl] = sg;
    red[1][pg][cl] = sb;
    __syncthreads();
    if (pg == 0 && c < it.cols) {
      const float g = (red[0][0][cl] + red[0][1][cl]) + (red[0][2][cl] + red[0][3][cl]);
      const float b = (red[1][0][cl] + red[1][1][cl]) + (red[1][2][cl] + red[1][3][cl]);
      if (it.dgamma) Elem<T>::store1(it.dgamma, c, g);
      if (it.dbeta) Elem<T>::store1(it.dbeta, c, b);
    }
    __syncthreads();  // red is rewritten by the next item
  }
}

// ===================================================================== launchers
#define OPTIMUS_BWD_ACT_SWITCH(act, ...)                           \
  switch (act) {                                                   \
    case OPTIMUS_ACT_NONE: { constexpr int A = 0; __VA_ARGS__; } break;    \
    case OPTIMUS_ACT_RELU: { constexpr int A = 1; __VA_ARGS__; } break;    \
    case OPTIMUS_ACT_SIGMOID: { constexpr int A = 2; __VA_ARGS__; } break; \
    case OPTIMUS_ACT_TANH: { constexpr int A = 3; __VA_ARGS__; } break;    \
    case OPTIMUS_ACT_SILU: { constexpr int A = 4; __VA_ARGS__; } break;    \
    default: return hipErrorInvalidValue;                          \
  }

hipError_t act_backward_launch(optimus_dtype dt, optimus_act act, const DevRowsGrad* descs, const RowTile* tiles,
                               int32_t num_tiles, int32_t grid, hipStream_t stream) {
  if (num_tiles <= 0) return hipSuccess;
  if (dt == OPTIMUS_BF16) {
    OPTIMUS_BWD_ACT_SWITCH(act, hipLaunchKernelGGL((grouped_act_backward_kernel<bf16_t, A>), dim3(grid),
                                                   dim3(kRowThreads), 0, stream, descs, tiles, num_tiles));
  } else {
    OPTIMUS_BWD_ACT_SWITCH(act, hipLaunchKernelGGL((grouped_act_backward_kernel<float, A>), dim3(grid),
                                                   dim3(kRowThreads), 0, stream, descs, tiles, num_tiles));
  }
  return hipGetLastError();
}

hipError_t layernorm_backward_launch(optimus_dtype dt, optimus_act act, const DevRowsGrad* descs,
                                     const RowTile* tiles, int32_t num_tiles, int32_t grid, hipStream_t stream) {
  if (num_tiles <= 0) return hipSuccess;
  if (dt == OPTIMUS_BF16) {
    OPTIMUS_BWD_ACT_SWITCH(act, hipLaunchKernelGGL((grouped_layernorm_backward_kernel<bf16_t, A>), dim3(grid),
                                                   dim3(kRowThreads), 0, stream, descs, tiles, num_tiles));
  } else {
    OPTIMUS_BWD_ACT_SWITCH(act, hipLaunchKernelGGL((grouped_layernorm_backward_kernel<float, A>), dim3(grid),
                                                   dim3(kRowThreads), 0, stream, descs, tiles, num_tiles));
  }
  return hipGetLastError();
}

int layernorm_backward_resident_per_cu(optimus_dtype dt, optimus_act act) {
  const void* k = nullptr;
  if (dt == OPTIMUS_BF16) {
    OPTIMUS_BWD_ACT_SWITCH(act, k = (const void*)grouped_layernorm_backward_kernel<bf16_t, A>);
  } else {
    OPTIMUS_BWD_ACT_SWITCH(act, k = (const void*)grouped_layernorm_backward_kernel<float, A>);
  }
  int b = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, k, kRowThreads, 0) != hipSuccess || b < 1) {
    (void)hipGetLastError();
    return 2;
  }
  return b;
}

hipError_t grad_finalize_launch(optimus_dtype dt, const GradFinItem* items, int32_t num_items, int32_t grid,
                                hipStream_t stream) {
  if (num_items <= 0) return hipSuccess;
  if (dt == OPTIMUS_BF16)
    hipLaunchKernelGGL(grad_finalize_kernel<bf16_t>, dim3(grid), dim3(256), 0, stream, items, num_items);
  else
    hipLaunchKernelGGL(grad_finalize_kernel<float>, dim3(grid), dim3(256), 0, stream, items, num_items);
  return hipGetLastError();
}

}  // namespace optimus
