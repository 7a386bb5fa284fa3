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
constexpr int kLnDepth = 2;  // row slots loaded ahead of the one being computed

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
  // gamma / beta unpacked once per tile into fp32 registers; for sigmoid,
  // silu and tanh they also carry the activation's input scale
  // (act_scaled_in), so that the affine step yields the exponent's argument
  // directly
  constexpr float ks = act_in_scale<ACT>();
  float gf[MAXC][VEC], bf[MAXC][VEC];
#pragma unroll
  for (int j = 0; j < MAXC; ++j) {
    const int c = j * L + li;
    if (d.gamma && c < cpr) {
      Elem<T>::unpack(ld16((const char*)d.gamma + (int64_t)c * 16), gf[j]);
    } else {
#pragma unroll
      for (int e = 0; e < VEC; ++e) gf[j][e] = 1.f;
    }
    if (d.beta && c < cpr) {
      Elem<T>::unpack(ld16((const char*)d.beta + (int64_t)c * 16), bf[j]);
    } else {
#pragma unroll
      for (int e = 0; e < VEC; ++e) bf[j][e] = 0.f;
    }
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      gf[j][e] *= ks;
      bf[j][e] *= ks;
    }
  }
  const int rpb = 4 * rpw;
  const int end = rt.row0 + rt.nrows;
  // The next kLnDepth row slots' chunks are loaded while the current one is
  // computed (a ring of row registers, rotated by register moves).
  constexpr int PF = kLnDepth;
  u32x4 ring[PF][MAXC];
  auto fetch = [&](u32x4 (&dst)[MAXC], int r) {
    const char* xr = (const char*)d.x + (int64_t)r * d.ldx * sizeof(T);
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = j * L + li;
      dst[j] = (r < end && c < cpr) ? ld16_nt(xr + (int64_t)c * 16) : u32x4{0u, 0u, 0u, 0u};
    }
  };
#pragma unroll
  for (int p = 0; p < PF; ++p) fetch(ring[p], rt.row0 + wave * rpw + sub + p * rpb);
  for (int base = rt.row0; base < end; base += rpb) {
    const int r = base + wave * rpw + sub;
    const bool valid = r < end;
    float x[MAXC][VEC];
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      Elem<T>::unpack(ring[0][j], x[j]);  // zero where out of range
#pragma unroll
      for (int p = 0; p + 1 < PF; ++p) ring[p][j] = ring[p + 1][j];
    }
    if (base + PF * rpb < end) fetch(ring[PF - 1], r + PF * rpb);
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
        x[j][e] -= mean;
        q += in ? x[j][e] * x[j][e] : 0.f;
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
        for (int e = 0; e < VEC; ++e) o[e] = act_scaled_in<ACT>(x[j][e] * (rstd * gf[j][e]) + bf[j][e]);
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

template <typename T, int ACT>
__global__ __launch_bounds__(kRowThreads) void grouped_layernorm_kernel(const DevRows* __restrict__ descs,
                                                                        const RowTile* __restrict__ tiles,
                                                                        int32_t num_tiles) {
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  for (int t = blockIdx.x; t < num_tiles; t += gridDim.x) {
    const RowTile rt = tiles[t];
    const DevRows d = descs[rt.member];
    if (d.vec && d.lanes > 0)
      ln_rows_vec<T, ACT, kLnChunksPerLane>(d, rt, lane, wave);
    else
      ln_rows_scalar<T, ACT>(d, rt, lane, wave);
  }
}

// ===================================================================== pointwise
// Same row/lane mapping as the LayerNorm kernel, without the reductions; a
// lane group loops over the row's chunks (any row length), kPwInflight loads
// in flight per lane.
constexpr int kPwInflight = 4;  // eight was faster on 1.25 GB but slower on 134 MB
template <typename T, int ACT>
__global__ __launch_bounds__(kRowThreads) void grouped_pointwise_kernel(const DevRows* __restrict__ descs,
                                                                        const RowTile* __restrict__ tiles,
                                                                        int32_t num_tiles) {
  constexpr int VEC = Elem<T>::VEC;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
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
        // kPwInflight chunks per lane in flight, then the rest one at a time
        int c = li;
        for (; c + (kPwInflight - 1) * L < cpr; c += kPwInflight * L) {
          u32x4 rv[kPwInflight];
#pragma unroll
          for (int u = 0; u < kPwInflight; ++u) rv[u] = ld16_nt(xr + (int64_t)(c + u * L) * 16);
#pragma unroll
          for (int u = 0; u < kPwInflight; ++u) {
            float v[VEC];
            Elem<T>::unpack(rv[u], v);
#pragma unroll
            for (int e = 0; e < VEC; ++e) v[e] = act_apply<ACT>(v[e]);
            st16_nt(yr + (int64_t)(c + u * L) * 16, Elem<T>::pack(v));
          }
        }
        for (; c < cpr; c += L) {
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
// WPR waves share one row (a block of four waves works on 4 / WPR rows at a
// time); in step j, lane l of the row's w-th wave holds the 16-byte chunk
// c = 64 S w + 64 j + l, so every step of a wave reads 1 KB of the row
// contiguously and writes it back at the same columns of `out` -- the split
// and the concat are index arithmetic only. The next row is loaded while the
// current one is computed.
//
// Piece statistics take one pass: every chunk contributes its sum and its sum
// of squares (fp32), written to LDS in row order. Each of the row's 64 WPR
// lanes then adds up the run of S consecutive chunks starting at chunk
// (its index in the row) * S, piece by piece: a piece that starts and ends
// inside the run gets its total written to the piece's slot, and the run's
// first and last segments are written back over the run's first two entries.
// The lane that owns a piece then adds, in a fixed order, the segments of
// the runs the piece spans, so the statistics do not depend on timing. The
// variance is E[x^2] - mean^2; where that would lose accuracy (a piece whose
// squared mean exceeds 16 times its variance) the row recomputes the
// variance from the centred values in a second pass. With one wave per row
// the row's LDS traffic is private to the wave and needs no workgroup
// barrier. Piece gamma and beta are gathered from each piece's own arrays
// and staged once per block in LDS as fp32, times the activation's input
// scale (act_scaled_in).
template <typename T, int ACT, int S, int WPR, bool FULL>
__global__ __launch_bounds__(kSocThreads) void split_op_cat_kernel(const DevSoc* __restrict__ sp) {
  constexpr int VEC = Elem<T>::VEC;
  constexpr int PACKS = (S + 3) / 4;    // piece ids packed four per register
  constexpr int SLOTS = 4 / WPR;        // rows in flight per block
  constexpr int RL = 64 * WPR;          // lanes per row
  constexpr int PL = S > 1 ? 1 : 0;     // where a run keeps its last segment
  extern __shared__ __align__(16) char smem[];
  const DevSoc s = *sp;
  // wave, slot and part are uniform across a wave: keep them (and row addresses) scalar
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int slot = wave / WPR, wr = wave % WPR;
  // FULL: the row is exactly RL * S chunks, so no chunk needs a range check
  const int nch = FULL ? RL * S : s.nchunks, npc = s.n_pieces;
  // LDS: gamma [nch * VEC] f32 | beta [nch * VEC] f32 | per slot: part [RL * S] (sum, sum of squares),
  // acc [2][npc] f32 (piece sums -> mean, squares -> 1/sqrt(var + eps)), flag
  const int slot_floats = 2 * RL * S + ((2 * npc + 4) & ~3);
  float* lg = (float*)smem;
  float* lb = lg + (size_t)nch * VEC;
  float2* part = (float2*)(lb + (size_t)nch * VEC + slot * slot_floats);
  float* acc = (float*)(part + RL * S);
  // one flag per row with one wave per row; one per block otherwise, so every
  // wave of the block takes the same branch (its barriers are block-wide)
  int* flag = (int*)(lb + (size_t)nch * VEC + (WPR == 1 ? slot : 0) * slot_floats + 2 * RL * S + 2 * npc);
  // each chunk's gamma / beta values from its piece's own arrays (read on
  // every launch, so the caller may update them between launches)
  for (int c = threadIdx.x; c < nch; c += kSocThreads) {
    const SocPiece pc = s.pieces[s.chunk_piece[c]];
    const int64_t e0 = (int64_t)(c - pc.c0) * VEC;  // first element of the chunk within the piece
    float g[VEC], b[VEC];
    if (pc.gamma && (pc.vec & 1)) {
      Elem<T>::unpack(ld16((const T*)pc.gamma + e0), g);
    } else {
#pragma unroll
      for (int e = 0; e < VEC; ++e) g[e] = pc.gamma ? Elem<T>::load1(pc.gamma, e0 + e) : 1.f;
    }
    if (pc.beta && (pc.vec & 2)) {
      Elem<T>::unpack(ld16((const T*)pc.beta + e0), b);
    } else {
#pragma unroll
      for (int e = 0; e < VEC; ++e) b[e] = pc.beta ? Elem<T>::load1(pc.beta, e0 + e) : 0.f;
    }
    constexpr float ks = act_in_scale<ACT>();
#pragma unroll
    for (int e = 0; e < VEC; e += 4) {
      *(f32x4*)(lg + (size_t)c * VEC + e) = f32x4{g[e] * ks, g[e + 1] * ks, g[e + 2] * ks, g[e + 3] * ks};
      *(f32x4*)(lb + (size_t)c * VEC + e) = f32x4{b[e] * ks, b[e + 1] * ks, b[e + 2] * ks, b[e + 3] * ks};
    }
  }
  __syncthreads();
  // row-local LDS ordering: a wave-local wait with one wave per row, else a workgroup barrier
  auto row_sync = [&]() {
    if constexpr (WPR == 1)
      lds_wave_sync();
    else
      __syncthreads();
  };

  const int cbase = wr * 64 * S;  // first chunk of this wave's part of the row
  const int ls = wr * 64 + lane;  // lane index within the row
  const int run0 = ls * S;        // this lane's reduction run
  // Per-lane static data: the piece of each chunk this lane holds and of each
  // chunk of its reduction run, a byte each.
  uint32_t pc[PACKS], rp[PACKS];
#pragma unroll
  for (int k = 0; k < PACKS; ++k) { pc[k] = 0u; rp[k] = 0u; }
#pragma unroll
  for (int j = 0; j < S; ++j) {
    const int c = cbase + j * 64 + lane, cr = run0 + j;
    pc[j >> 2] |= (uint32_t)(c < nch ? s.chunk_piece[c] : 0) << (8 * (j & 3));
    rp[j >> 2] |= (uint32_t)(cr < nch ? s.chunk_piece[cr] : 0) << (8 * (j & 3));
  }
  auto piece_of = [](const uint32_t* pk, int j) { return (int)((pk[j >> 2] >> (8 * (j & 3))) & 0xffu); };

  // The pieces this lane owns (ls, ls + RL; n_pieces <= 2 RL) and where their
  // totals come from: kind 1 = the first segment of run l0, 2 = its last
  // segment, 3 = a piece inside run l0 (its own slot), 0 = the last segment
  // of run l0 plus the first segments of runs l0 + 1 .. l1.
  struct Owned {
    int p, l0, l1, kind;
    float w, iw;  // width in values, and its reciprocal
  };
  auto owned = [&](int p) {
    Owned o{p, 0, -1, 0, 1.f, 0.f};
    if (p < npc) {
      const SocPiece q = s.pieces[p];
      o.w = (float)((q.c1 - q.c0) * VEC);
      o.iw = q.inv_width;
      o.l0 = q.c0 / S;
      o.l1 = (q.c1 - 1) / S;
      if (o.l0 == o.l1) {
        const int rs = o.l0 * S, re = min(rs + S, nch);
        o.kind = q.c0 == rs ? 1 : q.c1 == re ? 2 : 3;
      }
    }
    return o;
  };
  const Owned own0 = owned(ls), own1 = owned(ls + RL);
  auto total = [&](const Owned& o, const float* ix, const float* iy) -> float2 {
    if (o.kind == 1) return part[o.l0 * S];
    if (o.kind == 2) return part[o.l0 * S + PL];
    if (o.kind == 3) return float2{ix[o.p], iy ? iy[o.p] : 0.f};
    float2 v = part[o.l0 * S + PL];
    for (int l = o.l0 + 1; l <= o.l1; ++l) {
      const float2 f = part[l * S];
      v.x += f.x;
      v.y += f.y;
    }
    return v;
  };

  // Per-piece totals of the row's chunk pairs in part[] (see above): pieces
  // inside a run go to ix[p] (and iy[p] unless iy is null).
  auto run_reduce = [&](float* ix, float* iy) {
    if (run0 < nch) {
      float2 run[S];
#pragma unroll
      for (int i = 0; i < S; i += 2) {
        if constexpr (S > 1) {
          const f32x4 v = *(const f32x4*)(part + run0 + i);
          run[i] = float2{v[0], v[1]};
          run[i + 1] = float2{v[2], v[3]};
        } else {
          run[i] = part[run0 + i];
        }
      }
      int cur = piece_of(rp, 0);
      float2 a{0.f, 0.f}, first{0.f, 0.f};
      bool in_first = true;
#pragma unroll
      for (int i = 0; i < S; ++i) {
        if (FULL || run0 + i < nch) {
          const int p = piece_of(rp, i);
          if (p != cur) {
            if (in_first) {
              first = a;
              in_first = false;
            } else {
              ix[cur] = a.x;
              if (iy) iy[cur] = a.y;
            }
            a = float2{0.f, 0.f};
            cur = p;
          }
          a.x += run[i].x;
          a.y += run[i].y;
        }
      }
      if (in_first) first = a;
      if constexpr (PL) {
        *(f32x4*)(part + run0) = f32x4{first.x, first.y, a.x, a.y};
      } else {
        part[run0] = a;
      }
    }
  };

  u32x4 raw[S];
  auto fetch = [&](int row) {
    const char* xr = (const char*)s.in + (int64_t)row * s.ldin * sizeof(T);
#pragma unroll
    for (int j = 0; j < S; ++j) {
      const int c = cbase + j * 64 + lane;
      raw[j] = (FULL || c < nch) ? ld16_nt(xr + c * 16) : u32x4{0u, 0u, 0u, 0u};
    }
  };
  const int row_step = gridDim.x * SLOTS;
  int r0 = blockIdx.x * SLOTS;
  if (r0 + slot < s.rows) fetch(r0 + slot);
  // every wave of the block runs the same number of iterations (barriers inside when WPR > 1)
  for (; r0 < s.rows; r0 += row_step) {
    const int row = r0 + slot;
    const bool valid = row < s.rows;
    if (WPR == 1 && !valid) break;
    u32x4 cur[S];
#pragma unroll
    for (int j = 0; j < S; ++j) cur[j] = raw[j];
    if (row + row_step < s.rows) fetch(row + row_step);
    char* yr = (char*)s.out + (int64_t)row * s.ldout * sizeof(T);
    if (s.apply_ln) {
      // one pass: chunk sums and sums of squares
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int c = cbase + j * 64 + lane;
        if (FULL || c < nch) part[c] = float2{chunk_sum<T>(cur[j]), chunk_sumsq<T>(cur[j])};
      }
      if ((WPR == 1 ? lane : threadIdx.x) == 0) *flag = 0;
      row_sync();
      run_reduce(acc, acc + npc);
      row_sync();
      // owners: mean, E[x^2] - mean^2, and whether that lost accuracy
      auto finish = [&](const Owned& o) {
        if (o.p < npc) {
          const float2 t = total(o, acc, acc + npc);
          // a correctly rounded division: a constant piece gets its value back exactly
          const float m = __fdiv_rn(t.x, o.w), m2 = m * m;
          const float var = t.y * o.iw - m2;
          if (m2 > 16.f * var) *flag = 1;
          acc[o.p] = m;
          acc[npc + o.p] = __builtin_amdgcn_rsqf(fmaxf(var, 0.f) + s.eps);
        }
      };
      finish(own0);
      finish(own1);
      row_sync();
      if (__builtin_amdgcn_readfirstlane(*flag)) {  // the same word for every wave that shares it
        // second pass for the variance: sums of centred squares (the squared
        // means are large next to the variance, so E[x^2] - mean^2 cancels)
#pragma unroll
        for (int j = 0; j < S; ++j) {
          const int c = cbase + j * 64 + lane;
          const float m = acc[piece_of(pc, j)];
          float dx[VEC];
          u32x4 cj = cur[j];
          __asm__ volatile("" : "+v"(cj));  // unpacked here and again below, never held across
          centred<T>(cj, m, dx);
          float a = 0.f;
#pragma unroll
          for (int e = 0; e < VEC; ++e) a += dx[e] * dx[e];
          if (FULL || c < nch) part[c] = float2{a, 0.f};
        }
        row_sync();
        run_reduce(acc + npc, nullptr);  // inside-run pieces' totals go to the (recomputed) second slot
        row_sync();
        auto refinish = [&](const Owned& o) {
          if (o.p < npc) {
            const float q = total(o, acc + npc, nullptr).x;
            acc[npc + o.p] = __builtin_amdgcn_rsqf(q * o.iw + s.eps);
          }
        };
        refinish(own0);
        refinish(own1);
        row_sync();
      }
      // normalise: y = (x - mean) * (rstd * gamma) + beta, then the activation
      // (gamma and beta carry its input scale)
      if (valid) {
#pragma unroll
        for (int j = 0; j < S; ++j) {
          const int c = cbase + j * 64 + lane;
          if (FULL || c < nch) {
            const int pj = piece_of(pc, j);
            const float m = acc[pj], rs = acc[npc + pj];
            float dx[VEC], o[VEC];
            u32x4 cj = cur[j];
            __asm__ volatile("" : "+v"(cj));  // unpack at the use instead of keeping floats live
            centred<T>(cj, m, dx);
#pragma unroll
            for (int e = 0; e < VEC; e += 4) {
              const f32x4 g = *(const f32x4*)(lg + (size_t)c * VEC + e);
              const f32x4 b = *(const f32x4*)(lb + (size_t)c * VEC + e);
              o[e + 0] = act_scaled_in<ACT>(dx[e + 0] * (rs * g[0]) + b[0]);
              o[e + 1] = act_scaled_in<ACT>(dx[e + 1] * (rs * g[1]) + b[1]);
              o[e + 2] = act_scaled_in<ACT>(dx[e + 2] * (rs * g[2]) + b[2]);
              o[e + 3] = act_scaled_in<ACT>(dx[e + 3] * (rs * g[3]) + b[3]);
            }
            st16_nt(yr + c * 16, Elem<T>::pack(o));
          }
        }
      }
      row_sync();  // statistics read before the next row overwrites them
    } else if (valid) {
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int c = cbase + j * 64 + lane;
        if (FULL || c < nch) {
          float x[VEC], o[VEC];
          Elem<T>::unpack(cur[j], x);
#pragma unroll
          for (int e = 0; e < VEC; ++e) o[e] = act_apply<ACT>(x[e]);
          st16_nt(yr + c * 16, Elem<T>::pack(o));
        }
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

template <typename T, int ACT, int S, int WPR, bool FULL>
static const void* soc_kernel_ptr() {
  return (const void*)split_op_cat_kernel<T, ACT, S, WPR, FULL>;
}

struct SocShape {
  int steps, wpr;
  bool full;
  size_t smem;
};

// wpr waves per row (1: no workgroup barriers), more where a row would need
// over 8 chunks per lane in registers.
static SocShape soc_shape(int32_t nchunks, int32_t n_pieces, optimus_dtype dt, int32_t wpr) {
  if (wpr != 2 && wpr != 4) wpr = 1;
  // at most 8 chunks per lane in registers
  while (wpr < 4 && (nchunks + 64 * wpr - 1) / (64 * wpr) > 8) wpr *= 2;
  const int per = (nchunks + 64 * wpr - 1) / (64 * wpr);
  const int st = per <= 1 ? 1 : per <= 2 ? 2 : per <= 4 ? 4 : 8;
  const int vec = dt == OPTIMUS_F32 ? 4 : 8;
  const int slots = 4 / wpr;
  return SocShape{st, wpr, nchunks == 64 * wpr * st,
                  (size_t)nchunks * vec * 4 * 2 +
                      (size_t)slots * (2 * 64 * wpr * st + ((2 * n_pieces + 4) & ~3)) * 4};
}

template <typename T, int ACT, int WPR>
static const void* soc_kernel_w(const SocShape& sh) {
  switch (sh.steps) {
    case 1: return sh.full ? soc_kernel_ptr<T, ACT, 1, WPR, true>() : soc_kernel_ptr<T, ACT, 1, WPR, false>();
    case 2: return sh.full ? soc_kernel_ptr<T, ACT, 2, WPR, true>() : soc_kernel_ptr<T, ACT, 2, WPR, false>();
    case 4: return sh.full ? soc_kernel_ptr<T, ACT, 4, WPR, true>() : soc_kernel_ptr<T, ACT, 4, WPR, false>();
    default: return sh.full ? soc_kernel_ptr<T, ACT, 8, WPR, true>() : soc_kernel_ptr<T, ACT, 8, WPR, false>();
  }
}

template <typename T, int ACT>
static const void* soc_kernel_for(const SocShape& sh) {
  if (sh.wpr == 1) return soc_kernel_w<T, ACT, 1>(sh);
  if (sh.wpr == 2) return soc_kernel_w<T, ACT, 2>(sh);
  return soc_kernel_w<T, ACT, 4>(sh);
}

static const void* soc_kernel(optimus_dtype dt, optimus_act act, const SocShape& sh) {
  if (dt == OPTIMUS_BF16) {
    switch (act) {
      case OPTIMUS_ACT_NONE: return soc_kernel_for<bf16_t, 0>(sh);
      case OPTIMUS_ACT_RELU: return soc_kernel_for<bf16_t, 1>(sh);
      case OPTIMUS_ACT_SIGMOID: return soc_kernel_for<bf16_t, 2>(sh);
      case OPTIMUS_ACT_TANH: return soc_kernel_for<bf16_t, 3>(sh);
      case OPTIMUS_ACT_SILU: return soc_kernel_for<bf16_t, 4>(sh);
      default: return nullptr;
    }
  }
  switch (act) {
    case OPTIMUS_ACT_NONE: return soc_kernel_for<float, 0>(sh);
    case OPTIMUS_ACT_RELU: return soc_kernel_for<float, 1>(sh);
    case OPTIMUS_ACT_SIGMOID: return soc_kernel_for<float, 2>(sh);
    case OPTIMUS_ACT_TANH: return soc_kernel_for<float, 3>(sh);
    case OPTIMUS_ACT_SILU: return soc_kernel_for<float, 4>(sh);
    default: return nullptr;
  }
}

// Kernels whose dynamic LDS exceeds the 64 KB default need the limit raised once.
static hipError_t soc_allow_lds(const void* k, size_t smem) {
  if (smem <= 65536) return hipSuccess;
  return hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
}

int soc_blocks_per_cu(optimus_dtype dt, optimus_act act, int32_t nchunks, int32_t n_pieces, int32_t wpr) {
  const SocShape sh = soc_shape(nchunks, n_pieces, dt, wpr);
  const void* k = soc_kernel(dt, act, sh);
  int n = 0;
  if (k && soc_allow_lds(k, sh.smem) != hipSuccess) return 1;
  if (!k || hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k, kSocThreads, sh.smem) != hipSuccess || n < 1) n = 1;
  return n;
}

int soc_rows_per_block(optimus_dtype dt, int32_t nchunks, int32_t n_pieces, int32_t wpr) {
  return 4 / soc_shape(nchunks, n_pieces, dt, wpr).wpr;
}

hipError_t soc_launch(optimus_dtype dt, optimus_act act, const DevSoc* soc, int32_t nchunks, int32_t n_pieces,
                      int32_t wpr, int32_t grid, hipStream_t stream) {
  if (nchunks <= 0 || nchunks > kSocMaxChunks || n_pieces > kSocMaxPieces) return hipErrorInvalidValue;
  const SocShape sh = soc_shape(nchunks, n_pieces, dt, wpr);
  const void* k = soc_kernel(dt, act, sh);
  if (!k) return hipErrorInvalidValue;
  hipError_t e = soc_allow_lds(k, sh.smem);
  if (e != hipSuccess) return e;
  void* args[] = {(void*)&soc};
  return hipLaunchKernel(k, dim3(grid), dim3(kSocThreads), args, sh.smem, stream);
}

}  // namespace optimus
