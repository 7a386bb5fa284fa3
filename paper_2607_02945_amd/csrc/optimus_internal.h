// Internal types shared by the host planner and the gfx950 kernels of liboptimus.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "optimus.h"

namespace optimus {

// ------------------------------------------------------------------ device tables
// Every grouped launch reads a device-resident table written once by the planner.

// One Linear member as the GEMM kernel reads it (operand pointers, strides,
// sizes, and a flag telling whether 16-byte vector access is legal).
struct DevLinear {
  const void* x;
  const void* w;
  const void* bias;
  void* y;
  int64_t ldx, ldw, ldy;
  int32_t M, N, K;
  int32_t vec;  // bit0: x/w rows 16-B loadable (K, ldx, ldw, pointers); bit1: y rows 16-B storable
  // fused LayerNorm over each output row (used by the LN kernel instances only)
  const void* gamma;  // [N] or NULL (1)
  const void* beta;   // [N] or NULL (0)
  float eps, inv_n;   // inv_n = 1 / N
  // backward GEMMs: vec bit 2 = w 16-B loadable in its reduction-major layout;
  // xsum [M] receives the row sums of x over K (db beside dW), or NULL
  void* xsum;
  // split reduction (dW over a long batch): tile.pad is the split index, the
  // split covers k in [pad * kchunk, pad * kchunk + kchunk) and writes fp32
  // partials to ws ([splits][M][N], then the row sums [splits][M]); 0 / NULL
  // when not split
  float* ws;
  int32_t kchunk, splits;
  // input gradient with the activation backward of the layer below fused in
  // (dX = (dY W) * act'(ax), the instance's activation): ax [M][N] is that
  // activation's input, row stride ldax; vec bit 3 = ax rows 16-B loadable
  const void* ax;
  int64_t ldax;
};

// Sum of the split partials of one member over rows [row0, row0 + nrows):
// y = sum_s ws[s] (rounded to the dtype), and the row sums into xsum.
struct SplitReduceItem {
  const float* ws;
  void* y;
  void* xsum;
  int64_t ldy;
  int32_t M, N, splits, row0, nrows, pad;
};
hipError_t splitk_reduce_launch(optimus_dtype dt, const SplitReduceItem* items, int32_t num_items, int32_t grid,
                                hipStream_t stream);

// One 64 x 64 tile of a grouped transpose: dst[c][r] = src[r][c] for src rows
// [r0, r0 + 64) and columns [c0, c0 + 64), clipped to rows x cols.
struct TransposeItem {
  const void* src;
  void* dst;
  int64_t lds, ldd;
  int32_t rows, cols, r0, c0;
};
hipError_t transpose_launch(optimus_dtype dt, const TransposeItem* items, int32_t num_items, int32_t grid,
                            hipStream_t stream);

// One GEMM work item: the BM x BN output tile (mb, nb) of member `member`;
// member < 0 marks a padding entry that does no work.
struct GemmTile {
  int32_t member, mb, nb, pad;
};

// One row-wise member (LayerNorm or pointwise; a split-op-cat piece is a
// member that points into the shared input/output at its column offset).
struct DevRows {
  const void* x;
  void* y;
  const void* gamma;
  const void* beta;
  int64_t ldx, ldy;
  int32_t rows, cols;
  int32_t lanes;   // lanes per row (power of two, 1..64) for the LayerNorm kernel
  int32_t vec;     // 1 when rows are 16-B loadable/storable
  float eps;
  float inv_cols;
};

// One row-wise work item: rows [row0, row0 + nrows) of member `member`.
struct RowTile {
  int32_t member, row0, nrows, pad;
};

// Fused split-op-cat: per 16-byte chunk of a row, the piece it belongs to;
// per reduction task, a run of chunks of one piece. Each piece keeps the
// caller's gamma / beta pointers, which the kernel reads on every launch.
struct SocPiece {
  int32_t c0, c1;      // chunk range [c0, c1) of the piece
  float inv_width;
  int32_t vec;         // bit 0: gamma rows 16-B loadable; bit 1: beta
  const void* gamma;   // [width] of the group's dtype, or null (1)
  const void* beta;    // [width], or null (0)
};

struct DevSoc {
  const void* in;
  void* out;
  const uint8_t* chunk_piece;   // [nchunks]
  const SocPiece* pieces;       // [n_pieces]
  int64_t ldin, ldout;
  int32_t rows, D, nchunks, n_pieces;
  int32_t apply_ln;
  float eps;
};

// ------------------------------------------------------------------ launchers
// Implemented in the kernel translation units; each enqueues exactly one
// kernel launch on `stream` and returns the launch status.
struct GemmConfig {
  int bm, bn;          // tile
  int variant;         // index into the kernel table
  int threads;
  int occ;             // workgroups resident per CU
  const char* name;
};

// ln: the group's LayerNorm is fused into the epilogue, so one tile must hold
// a whole output row (the picked variant has bn >= every member's N).
// pin >= 0: that variant (index into the kernel table) if every member can
// run on it, else a config with variant -1.
GemmConfig gemm_pick_config(optimus_dtype dt, const optimus_linear_desc* d, int32_t G, bool ln, int pin = -1);
// Widest output row a fused LayerNorm can take for the dtype.
int gemm_ln_max_n(optimus_dtype dt);
// tr: 0 forward; 2 = w reduction-major (dX = dY . W); 3 = x and w
// reduction-major (dW = dY^T . X, with db from d.xsum).
hipError_t gemm_launch(const GemmConfig& cfg, optimus_dtype dt, optimus_act act, bool ln, const DevLinear* descs,
                       const GemmTile* tiles, int32_t num_tiles, int32_t grid, hipStream_t stream, int tr = 0);
// Whether every member of a dX group (x = dY [M][K_red], w = W [K_red][N])
// can run on the direct-to-LDS tiles reading W as it lies (no transpose).
bool gemm_dma_wt_ok(const optimus_linear_desc* d, int32_t G);
// Tile shape for the backward GEMMs with both operands reduction-major
// (direct-to-LDS where every member allows it, else register-staged).
// split_k: the set's K will be split (dW over the batch), so prefer the large
// tile; tile = 256 or 128 asks for that bf16 tile edge instead of the rule.
GemmConfig gemm_pick_config_trans(optimus_dtype dt, const optimus_linear_desc* d, int32_t G, bool split_k = false,
                                  int tile = 0, int pin = -1);
// Workgroups of the instance gemm_launch would run that fit on one CU at once
// (the HIP runtime's occupancy of its registers and LDS; cfg.occ if the query fails).
int gemm_resident_per_cu(const GemmConfig& cfg, optimus_dtype dt, optimus_act act, bool ln, int tr = 0);

constexpr int kRowThreads = 256;
// 16-byte chunks of a row each lane of the LayerNorm kernel holds in registers
// (rows up to 64 * this many chunks take the register path).
constexpr int kLnChunksPerLane = 2;
hipError_t layernorm_launch(optimus_dtype dt, optimus_act act, const DevRows* descs, const RowTile* tiles,
                            int32_t num_tiles, int32_t grid, hipStream_t stream);
hipError_t pointwise_launch(optimus_dtype dt, optimus_act act, const DevRows* descs, const RowTile* tiles,
                            int32_t num_tiles, int32_t grid, hipStream_t stream);

constexpr int kSocThreads = 256;
constexpr int kSocMaxChunks = 1024;  // 16-byte chunks per row held in registers by two waves (8 per lane)
constexpr int kSocMaxPieces = 128;   // two owned by each lane of a one-wave row
// wpr: waves per row asked for (1, 2 or 4; a row that needs more waves for
// its registers takes more).
hipError_t soc_launch(optimus_dtype dt, optimus_act act, const DevSoc* soc, int32_t nchunks, int32_t n_pieces,
                      int32_t wpr, int32_t grid, hipStream_t stream);
// Workgroups of the fused split-op-cat kernel resident per CU (occupancy query)
// and rows one workgroup works on at a time.
int soc_blocks_per_cu(optimus_dtype dt, optimus_act act, int32_t nchunks, int32_t n_pieces, int32_t wpr);
int soc_rows_per_block(optimus_dtype dt, int32_t nchunks, int32_t n_pieces, int32_t wpr);

// ------------------------------------------------------------------ backward
// One member of the LayerNorm / activation backward. Row mapping as for the
// forward row kernels (lanes, vec). LayerNorm: every row tile writes column
// partials of dgamma and dbeta (fp32, [2][cols] per partial row) into the
// plan's partial buffer from row part0 + RowTile.pad (one partial row per
// tile on the 16-byte path, one per wave on the per-value path).
struct DevRowsGrad {
  const void* x;
  const void* dy;
  void* dx;
  const void* gamma;
  float* part;      // the plan's partial buffer
  int64_t ldx, lddy, lddx;
  int32_t rows, cols;
  int32_t lanes, vec;
  float eps, inv_cols;
  int32_t part0;    // this member's first partial row
  int32_t want_params;  // dgamma / dbeta wanted
  // fused activation backward (LayerNorm + activation): the activation's
  // input gamma * xhat + beta is recomputed from x; beta [cols] or NULL (0)
  const void* beta;
};

// Finalize: columns [c0, c0 + kFinCols) of one member, the sum of its partial rows.
constexpr int kFinCols = 64;
struct GradFinItem {
  const float* part;  // first partial row of the member ([2][cols] each)
  void* dgamma;
  void* dbeta;
  int32_t cols, nparts, c0, pad;
};

constexpr int kGradWavesPerBlock = 4;  // partial rows per tile on the per-value path
// Workgroups of the LayerNorm-backward kernel resident on one CU.
int layernorm_backward_resident_per_cu(optimus_dtype dt, optimus_act act);
hipError_t act_backward_launch(optimus_dtype dt, optimus_act act, const DevRowsGrad* descs, const RowTile* tiles,
                               int32_t num_tiles, int32_t grid, hipStream_t stream);
hipError_t layernorm_backward_launch(optimus_dtype dt, optimus_act act, const DevRowsGrad* descs, const RowTile* tiles,
                                     int32_t num_tiles, int32_t grid, hipStream_t stream);
hipError_t grad_finalize_launch(optimus_dtype dt, const GradFinItem* items, int32_t num_items, int32_t grid,
                                hipStream_t stream);

// ------------------------------------------------------------------ fp8 codec
// One member of the fp8 activation codec. Quantize: x = values of the group's
// dtype, y = codes (one byte each); dequantize: x = codes, y = values.
// Strides in elements of each side. With lanes > 0 the member takes the
// 16-byte path: its item columns count chunks of 16 bytes of the wide (value)
// side, i.e. 16 / sizeof(value) values and as many codes; otherwise
// (lanes_scalar > 0) they count single values.
struct DevFp8 {
  const void* x;
  void* y;
  float* scale;        // quantize, scaled: written; dequantize: read, or null (1)
  int64_t ldx, ldy;
  int32_t rows, cols;
  int32_t lanes;         // threads per row of the 16-byte path (power of two, 1..256), or 0
  int32_t lanes_scalar;  // threads per row of the per-value path
  int32_t slot0, nslots; // the member's amax slots (scaled quantize)
};

// One work item: rows [row0, row0 + nrows) x item columns [c0, c1) of
// `member`; slot: the amax slot an amax item writes (-1 for other items).
struct Fp8Item {
  int32_t member, row0, nrows, c0, c1, slot;
};

// Scaled quantize: amax launch (one slot per amax item: nan flag << 31 |
// max |x| bits), then the convert launch, which reads the member's slots.
hipError_t fp8_amax_launch(optimus_dtype dt, const DevFp8* descs, const Fp8Item* items, int32_t num_items,
                           int32_t grid, uint32_t* slots, hipStream_t stream);
// slots == nullptr: unscaled quantize; else the scaled convert launch.
hipError_t fp8_quantize_launch(optimus_dtype dt, const DevFp8* descs, const Fp8Item* items, int32_t num_items,
                               int32_t grid, const uint32_t* slots, hipStream_t stream);
hipError_t fp8_dequantize_launch(optimus_dtype dt, const DevFp8* descs, const Fp8Item* items, int32_t num_items,
                                 int32_t grid, hipStream_t stream);

int device_cu_count();

}  // namespace optimus
