// Internal interface between the host dispatcher (api.hip) and the kernels.
// Not installed; the public interface is include/maddness.h.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mdn {

constexpr int kK = 16;       // prototypes per codebook
constexpr int kLevels = 4;   // tree depth
constexpr int kNodes = 15;   // thresholds per codebook (heap order)
constexpr int kMaxC = 512;   // codebooks supported by one launch
constexpr int kMaxFitC = 256; // codebooks of the table fit (16 C <= 4096 unknowns per column)
constexpr int kLdsBytes = 160 * 1024;  // LDS per workgroup on gfx950

enum Mode : int { kEncode = 0, kAccum = 1, kFused = 2 };
enum Elem : int { kI8 = 0, kF32 = 1 };

// Byte offsets of the LDS regions of one workgroup (all 16-byte aligned).
struct LdsLayout {
  int lut;     // LUT tile: [C*16 rows][lut_rs bytes]
  int thr;     // [C][16] fp32 thresholds (heap order, slot 15 unused)
  int split;   // [C][4] int32 split columns (clamped to [0, D))
  int misc;    // int32[4]: e_min, max shift, bias32 bits, step bits
  int sh;      // [C] int32 per-codebook shift e_c - e_min
  int shp;     // [ceil(C/8)] uint32: the shifts as nibbles, 8 codebooks per word
  int a;       // per wave: [RW][Dp] fp32 staged rows of A, then a 16-byte dummy slot
  int a_wave;  //   bytes per wave of the region above
  int idx;     // per wave: [RW][Cp] uint8 indices, then a 16-byte dummy slot
  int idx_wave;
  int total;
};

struct KArgs {
  const float* A;         // [N][lda]
  const uint8_t* idx_in;  // [N][C] (accumulate mode)
  const int32_t* split;   // [C][4]
  const float* thr;       // [C][15]
  const void* lut;        // [C][16][M] int8 or fp32
  const float* scale;     // [C]
  const float* offset;    // [C]
  float* y;               // [N][M]
  int32_t* acc;           // [N][M] or null
  uint8_t* idx_out;       // [N][C] or null
  int64_t N;
  int64_t lda;
  int D, C, M;
  int Mt;        // columns per LUT tile (blockIdx.y selects the tile)
  int lut_rs;    // LDS bytes per (c,k) row of the LUT tile
  int Dp;        // LDS row stride of staged A rows, floats
  int Cp;        // LDS row stride of staged indices, bytes (multiple of 4)
  int RW;        // rows per wave chunk (power of two, 1..64)
  int rw_log2;
  int64_t nchunks;       // ceil(N / RW)
  uint32_t c_magic;      // p / C == umulhi(p, c_magic) >> c_shift for p < 2^16
  int c_shift;
  int vec_rows;          // 1: staged rows move in 16-byte units
  int vec_out;           // 1: outputs / LUT rows allow 16-byte (4-column) stores
  int enc_reg;           // tree walk: 1 registers, lanes = (row, codebook) (C divides 64, RW*C % 64 == 0);
                         // 2 registers, lanes = codebooks (C % 64 == 0); 0 thresholds read from LDS
  int c_log2;            // log2(C) when enc_reg
  LdsLayout L;
};

// Arguments of the gather-fused kernel (fused_gather.hip): C divides 64 and the
// whole table fits in LDS.
struct GArgs {
  const float* A;         // [N][lda]
  const int32_t* split;   // [C][4]
  const float* thr;       // [C][15]
  const void* lut;        // [C][16][M] int8 or fp32
  const float* scale;     // [C]
  const float* offset;    // [C]
  float* y;               // [N][M] (null: accumulate-only calls with acc only)
  int32_t* acc;           // [N][M] or null
  uint8_t* idx_out;       // [N][C] or null
  const uint8_t* idx_in;  // [N][C]: accumulate only (no encode) when not null
  int64_t N;
  int64_t lda;
  int D, C, M;
  int c_log2;
  int rs8, rs16, rs32;    // LDS bytes per (c,k) row: int8, int16 and fp32 staging
  int R;                  // rows per wavefront step (NG * 64 / C)
  int NSP;                // offset slots per row (C rounded up to 4)
  int lpr_log2;           // accumulate: 2^lpr_log2 lanes per row, 8 columns each
  int vec_out;            // outputs allow 16-byte stores
  int vec16;              // table rows are whole 16-byte units (int8: M % 16 == 0; fp32: M % 4 == 0)
  const float* col_bias;  // [M] or null (layer output sigma)
  int act;                // 0 none, 1 bias, 2 bias + ReLU, 3 bias + row softmax
  int off_shc, off_misc, off_wave, off_bias, lds_total;  // LDS byte offsets
};

hipError_t launch_gfused(int elem, int ng, int uq, const GArgs& g, int nw, int cus, hipStream_t stream);

// Arguments of the column-tiled accumulate kernel (tiled_accum.hip): one work
// item is RB rows x Mt output columns; the table is staged CT codebooks at a
// time.
struct TArgs {
  const uint8_t* idx;     // [N][C]
  const void* lut;        // [C][16][M] int8 or fp32
  const float* scale;     // [C] (int8 tables)
  const float* offset;    // [C] (int8 tables)
  float* y;               // [N][M] or null (int8 tables with acc)
  int32_t* acc;           // [N][M] or null
  int64_t N;
  int C, M;
  int lpr_log2;           // lanes per output row: 8 or 16
  int Mt;                 // columns per tile: 8 (int8) or 4 (fp32) per lane
  int CT;                 // codebooks per LDS tile (multiple of 4)
  int RB;                 // rows per work item: waves * (64 / lanes per row) * NJ
  int ntm;                // column tiles
  int64_t nwork;          // ntm * ceil(N / RB)
  int vec_lut;            // table rows move in 16-byte units
  int vec_idx;            // index rows move in 4-byte units (C % 4 == 0)
  int vec_out;            // outputs allow 16-byte stores
  const float* col_bias;  // [M] or null (layer output sigma)
  int act;                // 0 none, 1 bias, 2 bias + ReLU, 3 bias + row softmax (one column tile only)
  int off_tab, off_idx, off_sh, off_misc, lds_total;  // LDS byte offsets
  int bias_lds, off_bias; // row-uniform kernels: column biases staged in LDS at off_bias (else read from memory)
  int64_t idx_stride;     // row-uniform kernels: bytes between index rows (C, or another layout's row pitch)
  int only_wide;          // row-uniform int8 kernel: do nothing when the 16-bit field sums fit (the
                          // fused row-streaming kernel has already written every output then)
};

// Row softmax in place over y [N][M] (layer outputs whose rows span several
// column tiles of the accumulate).
hipError_t launch_softmax_rows(float* y, int64_t N, int M, int cus, hipStream_t stream);

hipError_t launch_tacc(int elem, int nj, const TArgs& t, int nw, int cus, hipStream_t stream);

// Row-uniform accumulate (tiled_accum.hip): one 1024-thread workgroup per CU,
// work items of 256 rows x 512 columns (int8 tables) or 256 columns (fp32);
// idx must not overlap the outputs.
constexpr int kRowTileCols = 512;
constexpr int kRowTileColsF32 = 256;
hipError_t launch_trow(int elem, const TArgs& t, int cus, hipStream_t stream);

// Accumulate with one output row per lane (row_lanes.hip), fp32 tables with C
// % 16 == 0 and M % 4 == 0: one 1024-thread workgroup per CU, work items of
// 1024 rows x kRowLaneCols columns, the table staged kRowLaneCT codebooks at a
// time; idx rows (idx_stride bytes apart, a multiple of 16) must not overlap
// the outputs.
constexpr int kRowLaneCols = 64;
constexpr int kRowLaneCT = 16;
constexpr int kRowLaneLds = 2 * kRowLaneCT * 16 * (kRowLaneCols * 4 + 16);   // two tile buffers
hipError_t launch_rlane_f32(const TArgs& t, int cus, hipStream_t stream);
// int8 tables with C % 16 == 0, C >= 32, M % 16 == 0: work items of 1024 rows x
// kRowLaneColsI8 columns; the launch does nothing unless the 16-bit field sums
// fit (the row-uniform kernel with only_wide set then does the other case).
constexpr int kRowLaneColsI8 = 128;
hipError_t launch_rlane_i8(const TArgs& t, int cus, hipStream_t stream);

// Fused encode + accumulate streaming rows (fused_rows.hip): int8 tables of
// exactly 64 codebooks and M <= 512 columns (M % 16 == 0), one 1024-thread
// workgroup per CU over a contiguous block of rows_per_block rows.
constexpr int kFRing = 20;   // steps of index rows the row-streaming kernel keeps in LDS
struct FArgs {
  const float* A;         // [N][lda]
  const int32_t* split;   // [64][4]
  const float* thr;       // [64][15]
  const int8_t* lut;      // [64][16][M]
  const float* scale;     // [64]
  const float* offset;    // [64]
  float* y;               // [N][M]
  int32_t* acc;           // [N][M] or null
  uint8_t* idx_out;       // [N][64] or null
  const float* col_bias;  // [M] or null
  int64_t N, lda, rows_per_block;
  int D, M, act;
  int bias_lds;           // column biases staged in LDS (act != 0 and col_bias given)
  int off_ring, off_bias, lds_total;   // LDS byte offsets (the two table tile buffers at 0)
};
hipError_t launch_fenc(const FArgs& f, int blocks, hipStream_t stream);

// Lookup-accumulate as a one-hot int8 product on the matrix cores
// (onehot_mfma.hip): int8 tables with C % 16 == 0 and C <= 128, M % 4 == 0.
// Workgroups of 8 wavefronts each own one column slice (macc_width(C)
// columns) of one row group; with xcd_map (a grid of whole multiples of 8)
// block b takes pair gi = (b % 8) (grid / 8) + b / 8 of the (group, slice)
// pairs in group-major order, else slice b % nslices of group b / nslices.
struct MArgs {
  const uint8_t* idx;     // [N][C], 8-byte aligned
  const int8_t* lut;      // [C][16][M], 4-byte aligned
  const float* scale;     // [C]
  const float* offset;    // [C]
  float* y;               // [N][M] or null, 16-byte aligned
  int32_t* acc;           // [N][M] or null, 16-byte aligned
  const float* col_bias;  // [M] or null
  int64_t N, rows_per_group;   // rows_per_group: a multiple of 64
  int C, M, act;          // act: 0 none, 1 bias, 2 bias + ReLU (a softmax runs as a second pass)
  int bias_lds;           // column biases staged in LDS (act != 0 and col_bias given)
  int nslices, xcd_map;
  int off_val, off_sh, off_misc, off_bias, lds_total;   // LDS byte offsets (the table slice at 0)
};
constexpr int kMaccGroups = 5;   // one-hot shift groups of 7 for shifts up to 30
int macc_width(int C);
hipError_t launch_macc(const MArgs& m, int blocks, hipStream_t stream);

// Rounded 8-bit summation over codebooks: the whole [C][16][Mt] column slice
// (one byte per entry) staged once per workgroup, Mt = 16 * lanes per row.
hipError_t launch_tavg(const TArgs& t, int nw, int cus, hipStream_t stream);

// Compute units of the current device (queried once per device).
int device_cus();

// Per (device, kernel, block size, dynamic LDS bytes): raises the kernel's
// dynamic-LDS limit when it needs more than 64 KB and returns how many such
// workgroups one CU holds (at least 1); *err receives a failed attribute call.
int launch_prepare(const void* fn, int block, int lds, hipError_t* err);

// Launch one kernel of the family; returns hipSuccess or the launch error.
hipError_t launch_path(int mode, int elem, int pf, int uq, const KArgs& a,
                       dim3 grid, dim3 block, hipStream_t stream);

// Offline table build (T = P B, quantization); see lut_build.hip.
hipError_t launch_build_lut(const float* P, const float* B, int C, int D, int M,
                            int8_t* lut, float* scale, float* offset, int cap,
                            hipStream_t stream);
hipError_t launch_build_lut_f32(const float* P, const float* B, int C, int D, int M,
                                float* lut, hipStream_t stream);
hipError_t launch_quantize_lut(const double* T, int C, int M, int8_t* lut, float* scale, float* offset,
                               int cap, hipStream_t stream);

// Model-aware table fit (Eq. 3, affine output); see lut_fit.hip.
hipError_t launch_gram(const uint8_t* idx, int64_t N, int C, int32_t* H, int cus, hipStream_t stream);
hipError_t launch_scatter(const uint8_t* idx, int64_t N, int C, const float* Y, int M, double* R,
                          int32_t* perm, int32_t* start, hipStream_t stream);
hipError_t launch_fit_gd(const uint8_t* idx, int64_t N, int C, const float* Y, int M, const float* bias, int act,
                         const float* T0, double lam, double eta, int iters, double* T, double* P, double* D,
                         double* R, int32_t* perm, int32_t* start, hipStream_t stream);
hipError_t launch_fit_ridge(const uint8_t* idx, int64_t N, int C, const float* Y, int M, const float* T0,
                            double lam, double* T, int32_t* H, double* A, int32_t* perm, int32_t* start,
                            int cus, hipStream_t stream);

}  // namespace mdn
