// C ABI of libmaddness: argument validation, launch planning and dispatch.
// Declarations and the meaning of every argument: include/maddness.h.
#include "maddness.h"
#include "internal.hpp"

#include <stdint.h>
#include <cmath>
#include <mutex>

// Index array of maddness_matmul_noalloc's two-phase path, for callers that
// cannot allocate device memory: kScratchBytes on each device the library
// runs on, held until the process ends.  Host code never uses this name as
// an address: scratch_base() resolves it per device.
constexpr int64_t kScratchBytes = int64_t(32) << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace mdn {
namespace {

constexpr int kPFs[] = {1, 2, 4, 8, 9, 16};  // instantiated prefetch depths

bool aligned(const void* p, uintptr_t n) { return (reinterpret_cast<uintptr_t>(p) & (n - 1)) == 0; }
int round_up(int v, int m) { return (v + m - 1) / m * m; }
int64_t round_up64(int64_t v, int64_t m) { return (v + m - 1) / m * m; }
int ilog2(int v) { int r = 0; while ((1 << r) < v) ++r; return r; }

int pick_pf(int units) {  // smallest instantiated depth holding `units` 16-byte units per wavefront
  for (int pf : kPFs)
    if (units <= 64 * pf) return pf;
  return -1;
}

int status_from(hipError_t e) { return e == hipSuccess ? MADDNESS_OK : MADDNESS_EHIP; }

struct Shape {
  int mode, elem;
  const float* A; int64_t N; int D; int64_t lda;
  const int32_t* split; const float* thr; int C;
  const void* lut; const float* scale; const float* offset; int M;
  const uint8_t* idx_in;
  float* y; int32_t* acc; uint8_t* idx_out;
  const float* col_bias; int act;   // layer output sigma (fused entry points only)
};

// LDS layout for one workgroup of `nw` wavefronts.
LdsLayout layout(const Shape& s, int nw, int rw, int Dp, int Cp, int lut_bytes) {
  LdsLayout L{};
  int off = 0;
  auto take = [&](int bytes) { const int o = off; off += round_up(bytes, 16); return o; };
  const bool enc = s.mode != kAccum;
  L.lut = take(s.mode != kEncode ? lut_bytes : 0);
  L.thr = take(enc ? s.C * 16 * 4 : 0);
  L.split = take(enc ? s.C * kLevels * 4 : 0);
  L.misc = take(16);
  const bool q8 = s.mode != kEncode && s.elem == kI8;
  L.sh = take(q8 ? s.C * 4 : 0);
  L.shp = take(q8 ? (s.C + 7) / 8 * 4 : 0);
  L.a_wave = enc ? round_up(rw * Dp * 4 + 16, 16) : 0;
  L.a = take(nw * L.a_wave);
  L.idx_wave = round_up(rw * Cp + 16, 16);
  L.idx = take(nw * L.idx_wave);
  L.total = off;
  return L;
}

struct Plan {
  KArgs a;
  int pf, uq, nw;
  dim3 grid, block;
};

// LDS bytes of one (c, k) row of a LUT tile of `cols` columns.
int lut_row_stride(int elem, int cols) {
  if (elem == kI8) {
    int b = round_up(cols, 4);
    if (((b >> 2) & 1) == 0) b += 4;  // odd dword stride spreads the 16 rows of a codebook over banks
    return b;
  }
  return round_up(cols, 4) * 4;
}

// Widest column tile (<= max_cols, multiple of 4 unless it is all of M) whose
// C*16 rows fit in LDS next to `reserve` bytes, then narrowed to split M into
// equal tiles.  Returns false when not even 4 columns fit.
bool lut_tile(int elem, int C, int M, int reserve, int max_cols, int* Mt, int* rs) {
  const int64_t rows = (int64_t)C * kK;
  int cols = M < max_cols ? M : (max_cols & ~3);
  while (cols > 0 && rows * lut_row_stride(elem, cols) + reserve > kLdsBytes)
    cols = (cols > 4) ? ((cols - 1) & ~3) : 0;
  if (cols <= 0) return false;
  if (cols < M) {
    const int ntiles = (M + cols - 1) / cols;
    cols = round_up((M + ntiles - 1) / ntiles, 4);
  }
  *Mt = cols;
  *rs = lut_row_stride(elem, cols);
  return true;
}

// Builds the launch plan; returns a status (EUNSUPPORTED when the shape cannot run).
// Chunk size RW (rows per wavefront iteration) is chosen by, in order:
// fewest column tiles, fewest column quads per lane, largest RW.
int plan(const Shape& s, Plan* out, bool single_tile_only) {
  KArgs a{};
  a.A = s.A; a.idx_in = s.idx_in; a.split = s.split; a.thr = s.thr;
  a.lut = s.lut; a.scale = s.scale; a.offset = s.offset;
  a.y = s.y; a.acc = s.acc; a.idx_out = s.idx_out;
  a.N = s.N; a.lda = s.lda; a.D = s.D; a.C = s.C; a.M = s.M;
  a.Cp = round_up(s.C, 4);
  a.c_magic = s.C > 1 ? (uint32_t)((1ull << 32) / (uint64_t)s.C + 1) : 0u;

  const bool enc = s.mode != kAccum;
  const bool acc = s.mode != kEncode;
  const int nw = 4;

  bool vec_rows;
  int upr;  // 16-byte units per staged source row
  if (enc) {
    vec_rows = (s.D % 4 == 0) && (s.lda % 4 == 0) && aligned(s.A, 16);
    upr = s.D / 4;
  } else {
    vec_rows = (s.C % 16 == 0) && aligned(s.idx_in, 16);
    upr = s.C / 16;
  }
  if (enc) {
    a.Dp = round_up(s.D, 4);
    if (a.Dp % 32 == 0) a.Dp += 4;  // rows of one chunk start on different banks
  }
  a.vec_out = acc && (s.M % 4 == 0) && aligned(s.lut, 4) && (s.y == nullptr || aligned(s.y, 16)) &&
              (s.acc == nullptr || aligned(s.acc, 16));

  // Accumulate cost model: lane-quad slots per row = tiles * LPR * UQ (idle
  // lanes included); ties go to fewer quads per lane, then to larger chunks.
  bool found = false;
  int best_rw = 0, best_pf = 0, best_uq = 0, best_Mt = 1, best_rs = 0, best_tiles = 1;
  int64_t best_cost = 0;
  for (int rw_log2 = 6; rw_log2 >= 0; --rw_log2) {
    const int rw = 1 << rw_log2;
    const int lpr = 64 / rw;
    int pf = 0;
    if (vec_rows) {
      pf = pick_pf(rw * upr);
      if (pf < 0 || (pf > 9 && rw > 1)) continue;  // bound the prefetch registers
      if (enc && (int64_t)rw * s.lda * 4 >= (1ll << 31)) continue;
    } else if (rw > 8) {
      continue;  // synchronous staging: small chunks
    }
    const int reserve = layout(s, nw, rw, a.Dp, a.Cp, 0).total;
    if (reserve > kLdsBytes) continue;
    for (int uq_cap = 1; uq_cap <= (acc ? 4 : 1); uq_cap *= 2) {
      int uq = 1, Mt = 1, rs = 0, tiles = 1;
      if (acc) {
        if (!lut_tile(s.elem, s.C, s.M, reserve, 4 * lpr * uq_cap, &Mt, &rs)) continue;
        tiles = (s.M + Mt - 1) / Mt;
        if (single_tile_only && tiles > 1) continue;
        if (tiles > 65535) continue;
        uq = ((Mt + 3) / 4 + lpr - 1) / lpr;
        if (uq == 3) uq = 4;
        if (uq > 4) continue;
      }
      const int64_t cost = (int64_t)tiles * lpr * uq;
      const bool better = !found || cost < best_cost || (cost == best_cost && uq < best_uq);
      if (better) {
        found = true;
        best_cost = cost;
        best_rw = rw; best_pf = pf; best_uq = uq; best_Mt = Mt; best_rs = rs; best_tiles = tiles;
      }
    }
  }
  if (!found) return MADDNESS_EUNSUPPORTED;

  a.RW = best_rw;
  a.rw_log2 = ilog2(best_rw);
  a.Mt = best_Mt;
  a.lut_rs = best_rs;
  a.vec_rows = vec_rows;
  a.enc_reg = !enc ? 0
              : ((64 % s.C == 0) && ((best_rw * s.C) % 64 == 0)) ? 1   // lanes = (row, codebook)
              : (s.C % 64 == 0) ? 2                                   // lanes = codebooks, rows looped
              : 0;                                                    // threshold walk in LDS
  a.c_log2 = ilog2(s.C);
  a.nchunks = (s.N + best_rw - 1) / best_rw;
  a.L = layout(s, nw, best_rw, a.Dp, a.Cp, acc ? s.C * kK * best_rs : 0);
  if (a.L.total > kLdsBytes) return MADDNESS_EUNSUPPORTED;

  int per_cu = kLdsBytes / (a.L.total > 0 ? a.L.total : 1);
  const int by_threads = 2048 / (nw * 64);
  if (per_cu > by_threads) per_cu = by_threads;
  if (per_cu < 1) per_cu = 1;
  int64_t gx = (int64_t)256 * per_cu / best_tiles;
  if (gx < 8) gx = 8;
  const int64_t need = (a.nchunks + nw - 1) / nw;
  if (gx > need) gx = need;
  if (gx < 1) gx = 1;

  out->a = a;
  out->pf = vec_rows ? best_pf : 0;
  out->uq = best_uq;
  out->nw = nw;
  out->grid = dim3((unsigned)gx, (unsigned)best_tiles, 1);
  out->block = dim3(nw * 64, 1, 1);
  return MADDNESS_OK;
}

// Gather-fused plan: C divides 64 and the whole table (plus one zero row,
// staged as int16 for int8 tables) fits in LDS.  Returns false when the
// shape does not qualify.
bool plan_gfused(const Shape& s, GArgs* g, int* ng_out, int* uq_out, int* nw_out) {
  if (s.C > 64 || (64 % s.C) != 0) return false;
  int nw = 16;   // one 1024-thread workgroup per CU stages the table once
  const int G = 64 / s.C;
  const int no = (s.M + 7) / 8;   // column octets
  int best_ng = 0, best_uq = 0, best_lpr = 0;
  int64_t best_cost = 0;
  for (int ng = 1; ng <= 4; ng *= 2) {
    const int R = ng * G;
    if (R > 64) break;
    for (int uq = 1; uq <= 4; uq *= 2) {
      int lpr = 1;
      while (lpr < 64 && lpr * uq < no) lpr *= 2;
      if (lpr < 64 / R) lpr = 64 / R;   // one accumulate pass covers at most R rows
      int uq_eff = (no + lpr - 1) / lpr;
      if (uq_eff == 3) uq_eff = 4;
      if (uq_eff > uq) continue;
      const int64_t cost = (int64_t)lpr * uq_eff;   // lane-slots per row
      if (best_ng == 0 || cost < best_cost) {
        best_ng = ng; best_uq = uq_eff; best_lpr = lpr; best_cost = cost;
      }
    }
  }
  if (best_ng == 0) return false;
  GArgs a{};
  a.A = s.A; a.split = s.split; a.thr = s.thr; a.lut = s.lut; a.scale = s.scale; a.offset = s.offset;
  a.y = s.y; a.acc = s.acc; a.idx_out = s.idx_out;
  a.N = s.N; a.lda = s.lda; a.D = s.D; a.C = s.C; a.M = s.M;
  a.c_log2 = ilog2(s.C);
  a.rs8 = round_up(s.M, 8);
  a.rs16 = 2 * round_up(s.M, 8);
  a.rs32 = 4 * round_up(s.M, 8);
  a.R = best_ng * G;
  a.NSP = round_up(s.C, 4);
  a.lpr_log2 = ilog2(best_lpr);
  a.vec_out = (s.M % 4 == 0) && aligned(s.y, 16) && (s.acc == nullptr || aligned(s.acc, 16));
  a.vec16 = aligned(s.lut, 16) && (s.elem == kF32 ? (s.M % 4 == 0) : (s.M % 16 == 0));
  a.col_bias = s.col_bias;
  a.act = s.act;
  if ((int64_t)a.R * s.lda * 4 >= (1ll << 31)) return false;   // 32-bit per-lane gather offsets
  const int64_t tab = (int64_t)(s.C * kK + 1) * (s.elem == kF32 ? a.rs32 : a.rs16);
  if (tab > kLdsBytes) return false;
  int off = 0;
  for (;; nw /= 2) {   // widest workgroup whose offsets fit next to the table
    off = 0;
    auto take = [&](int64_t bytes) { const int o = off; off += round_up((int)bytes, 16); return o; };
    take(tab);
    a.off_shc = take(s.C * 4);
    a.off_misc = take(32);
    a.off_wave = take((int64_t)nw * a.R * a.NSP * 4);
    a.off_bias = take(s.act ? 8 * ((s.M + 7) / 8) * 4 : 0);   // bias row, whole octets of columns
    if (off <= kLdsBytes || nw == 1) break;
  }
  a.lds_total = off;
  if (off > kLdsBytes) return false;
  *g = a;
  *ng_out = best_ng;
  *uq_out = best_uq;
  *nw_out = nw;
  return true;
}

// Column-tiled accumulate (tiled_accum.hip): 8 wavefronts, 4 row passes per
// wavefront per work item, table tiles of CT codebooks sized for two
// workgroups per CU.
bool plan_tacc(const Shape& s, TArgs* t, int* nj_out, int* nw_out) {
  const bool f32 = s.elem == kF32;
  const int eg = f32 ? 4 : 1;                 // global bytes per table entry
  if ((int64_t)s.C * kK * s.M * eg >= (1ll << 31)) return false;   // 32-bit buffer offsets
  const int nw = 8, nj = 4;
  const int cpl = f32 ? 4 : 8;                // columns per lane
  const int lpr = s.M > 8 * cpl ? 16 : 8;     // lanes per output row
  TArgs a{};
  a.idx = s.idx_in; a.lut = s.lut; a.scale = s.scale; a.offset = s.offset; a.y = s.y; a.acc = s.acc;
  a.N = s.N; a.C = s.C; a.M = s.M;
  a.lpr_log2 = ilog2(lpr);
  a.Mt = cpl * lpr;
  a.RB = nw * (64 / lpr) * nj;
  const int upc = 16 / eg;                    // columns per 16-byte global unit
  const int units_per_cb = kK * (a.Mt / upc);
  int ct = 4;   // largest multiple of 4 whose units and index words fit the staging registers
  while (ct * 2 <= round_up(s.C, 4) && (ct * 2) * units_per_cb <= 4 * nw * 64 && a.RB * (ct * 2) / 4 <= 2 * nw * 64)
    ct *= 2;
  a.CT = ct;
  a.ntm = (s.M + a.Mt - 1) / a.Mt;
  a.nwork = (int64_t)a.ntm * ((s.N + a.RB - 1) / a.RB);
  a.vec_lut = aligned(s.lut, 16) && (s.M % upc == 0);
  a.vec_idx = (s.C % 4 == 0) && aligned(s.idx_in, 4);
  a.vec_out = (s.M % 4 == 0) && (s.y == nullptr || aligned(s.y, 16)) && (s.acc == nullptr || aligned(s.acc, 16));
  a.col_bias = s.col_bias;
  a.act = (s.act == 3 && a.ntm > 1) ? 1 : s.act;   // rows over several tiles: softmax as a second pass
  int off = 0;
  auto take = [&](int bytes) { const int o = off; off += round_up(bytes, 16); return o; };
  a.off_tab = take(a.CT * kK * a.Mt * (f32 ? 4 : 2));   // 0: the kernel relies on it
  a.off_idx = take(a.RB * a.CT * 4);
  a.off_sh = take(s.C * 4);
  a.off_misc = take(16);
  a.lds_total = off;
  if (off > kLdsBytes) return false;
  *t = a;
  *nj_out = nj;
  *nw_out = nw;
  return true;
}

// Row-uniform accumulate (tiled_accum.hip) for tables at least one column
// tile wide (512 int8 or 256 fp32 columns): scalar loads of 4-byte index words
// (C % 4 == 0), table rows in whole 16-byte units (int8: M % 16 == 0, fp32:
// M % 4 == 0 and a 16-byte aligned table), 16-byte output stores, and enough
// 256-row work items to occupy a quarter of the CUs.  `companion`: the launch
// after the row-streaming fused kernel (int8, any M % 16 == 0 up to one tile,
// index rows `idx_stride` bytes apart), which sums only when that kernel could
// not.
bool plan_trow(const Shape& s, TArgs* t, bool companion = false, int64_t idx_stride = 0) {
  const bool f32 = s.elem == kF32;
  const int cols = f32 ? kRowTileColsF32 : kRowTileCols;
  if ((!companion && s.M < cols) || s.M % (f32 ? 4 : 16) != 0 || s.C % 4 != 0) return false;
  if (!aligned(s.idx_in, 4) || !aligned(s.lut, f32 ? 16 : 4)) return false;
  if ((s.y && !aligned(s.y, 16)) || (s.acc && !aligned(s.acc, 16))) return false;
  if ((int64_t)s.C * kK * s.M * (f32 ? 4 : 1) >= (1ll << 31)) return false;   // 32-bit buffer offsets
  TArgs a{};
  a.idx = s.idx_in; a.lut = s.lut; a.scale = s.scale; a.offset = s.offset; a.y = s.y; a.acc = s.acc;
  a.N = s.N; a.C = s.C; a.M = s.M;
  a.Mt = cols;
  a.RB = 256;
  a.ntm = (s.M + cols - 1) / cols;
  a.nwork = (int64_t)a.ntm * ((s.N + a.RB - 1) / a.RB);
  if (!companion && a.nwork * 4 < device_cus()) return false;
  a.idx_stride = companion ? idx_stride : s.C;
  a.only_wide = companion ? 1 : 0;
  a.col_bias = s.col_bias;
  a.act = (s.act == 3 && a.ntm > 1) ? 1 : s.act;   // rows over several tiles: softmax as a second pass
  int off = 0;
  auto take = [&](int bytes) { const int o = off; off += round_up(bytes, 16); return o; };
  a.off_tab = take(8 * kK * 2 * kRowTileCols);   // 0: the kernel relies on it
  a.off_sh = take(s.C * 4);
  a.off_misc = take(16);
  if (a.act != 0 && a.col_bias && (int64_t)off + round_up(s.M * 4, 16) <= kLdsBytes) {
    a.bias_lds = 1;   // the whole bias row, staged once per workgroup
    a.off_bias = take(s.M * 4);
  }
  a.lds_total = off;
  if (off > kLdsBytes) return false;
  *t = a;
  return true;
}

// One output row per lane (row_lanes.hip): fp32 tables of at least 256
// columns (M % 4 == 0) and C % 16 == 0, 16-byte aligned table, outputs and
// index rows, the column biases in LDS when there are any, enough work items
// for the CUs.  A row softmax takes the row-uniform kernel when the row is one
// of its column tiles (fused there), else it is a second pass here too.
bool plan_rlane(const Shape& s, TArgs* t) {
  if (s.elem != kF32 || s.M < kRowTileColsF32 || s.M % 4 != 0 || s.C % kRowLaneCT != 0) return false;
  if (s.act == 3 && s.M <= kRowTileColsF32) return false;
  if (!aligned(s.idx_in, 16) || !aligned(s.lut, 16) || (s.y && !aligned(s.y, 16))) return false;
  if (!s.y || s.acc) return false;
  if ((int64_t)s.C * kK * s.M * 4 + 1024 >= (1ll << 31)) return false;   // 32-bit buffer offsets
  TArgs a{};
  a.idx = s.idx_in; a.lut = s.lut; a.y = s.y;
  a.N = s.N; a.C = s.C; a.M = s.M;
  a.Mt = kRowLaneCols;
  a.RB = 1024;
  a.ntm = (s.M + kRowLaneCols - 1) / kRowLaneCols;
  a.nwork = (int64_t)a.ntm * ((s.N + a.RB - 1) / a.RB);
  if (a.nwork * 4 < device_cus()) return false;
  a.idx_stride = s.C;
  a.col_bias = s.col_bias;
  a.act = s.act == 3 ? 1 : s.act;   // (rows over several tiles) softmax as a second pass
  int off = kRowLaneLds;
  if (a.act != 0 && a.col_bias) {
    a.bias_lds = 1;
    a.off_bias = off;
    off += a.ntm * kRowLaneCols * 4;   // zero-padded to whole column tiles
  }
  a.lds_total = off;
  if (off > kLdsBytes) return false;
  *t = a;
  return true;
}

// One output row per lane for int8 tables (row_lanes.hip): y only (no int32
// sums), the row-uniform kernel's shapes (it is the companion launch, for
// 32-bit sums) with C % 16 == 0, C >= 32 and 16-byte aligned index rows and
// table; a row softmax the row-uniform kernel would fuse (M <= 512) stays
// with that kernel alone.
bool plan_rlane_i8(const Shape& s, TArgs* t, TArgs* companion) {
  if (s.elem != kI8 || s.C % kRowLaneCT != 0 || s.C < 2 * kRowLaneCT) return false;
  if (!s.y || s.acc) return false;   // y only: with the int32 sums too, the row-uniform kernel's stores win
  if (s.act == 3 && s.M <= kRowTileCols) return false;
  if (!aligned(s.idx_in, 16) || !aligned(s.lut, 16)) return false;
  TArgs r;
  if (!plan_trow(s, &r)) return false;
  TArgs a{};
  a.idx = s.idx_in; a.lut = s.lut; a.scale = s.scale; a.offset = s.offset; a.y = s.y; a.acc = s.acc;
  a.N = s.N; a.C = s.C; a.M = s.M;
  a.Mt = kRowLaneColsI8;
  a.RB = 1024;
  a.ntm = (s.M + kRowLaneColsI8 - 1) / kRowLaneColsI8;
  a.nwork = (int64_t)a.ntm * ((s.N + a.RB - 1) / a.RB);
  if (a.nwork * 4 < device_cus()) return false;
  a.idx_stride = s.C;
  a.col_bias = s.col_bias;
  a.act = r.act;   // 1 for a softmax over rows of several tiles (then a second pass), as there
  int off = kRowLaneLds;
  auto take = [&](int bytes) { const int o = off; off += round_up(bytes, 16); return o; };
  a.off_sh = take(s.C * 4);
  a.off_misc = take(16);
  if (a.act != 0 && a.col_bias) {
    a.bias_lds = 1;
    a.off_bias = take(a.ntm * kRowLaneColsI8 * 4);   // zero-padded to whole column tiles
  }
  a.lds_total = off;
  if (off > kLdsBytes) return false;
  r.only_wide = 1;   // does the call only when the 16-bit field sums do not fit
  *t = a;
  *companion = r;
  return true;
}

int run(const Shape& s, bool single_tile_only, hipStream_t stream) {
  Plan p;
  const int rc = plan(s, &p, single_tile_only);
  if (rc != MADDNESS_OK) return rc;
  return status_from(launch_path(s.mode, s.elem, p.pf, p.uq, p.a, p.grid, p.block, stream));
}

// Row-streaming fused kernel (fused_rows.hip): int8 tables of 64 codebooks,
// 16 <= M <= 512 with M % 16 == 0, at least kFencMinRows rows (each of the at
// least 64 workgroups gets a few hundred), 16-byte aligned table and outputs,
// row blocks whose byte offsets fit 32 bits.  With `cus` = 0 (the index-bytes
// query, which makes no HIP call) only the shape is checked.  The companion
// launch (row-uniform accumulate, 32-bit sums when the 16-bit fields do not
// fit) reads the indices from idx_out, else from the first 64 bytes of each
// output row.
constexpr int64_t kFencMinRows = 98304;
bool plan_fenc(const Shape& s, FArgs* f, int* blocks_out, TArgs* companion, int cus) {
  if (s.mode != kFused || s.elem != kI8 || s.C != 64) return false;
  if (s.M < 16 || s.M > kRowTileCols || s.M % 16 != 0 || s.N < kFencMinRows) return false;
  if (!aligned(s.lut, 16) || !aligned(s.y, 16) || (s.acc && !aligned(s.acc, 16))) return false;
  // rows per workgroup with at least 64 workgroups; the kernel's gathers run
  // up to 12 x 36 rows past its block (those offsets must stay below 2^31)
  const int64_t max_block = (s.N + 63) / 64;
  if ((max_block + 512) * s.lda * 4 >= (1ll << 31)) return false;
  if (cus <= 0) return true;
  const int blocks = cus > 64 ? cus : 64;
  FArgs a{};
  a.A = s.A; a.split = s.split; a.thr = s.thr; a.lut = static_cast<const int8_t*>(s.lut);
  a.scale = s.scale; a.offset = s.offset; a.y = s.y; a.acc = s.acc; a.idx_out = s.idx_out;
  a.col_bias = s.col_bias; a.act = s.act;
  a.N = s.N; a.lda = s.lda; a.D = s.D; a.M = s.M;
  a.rows_per_block = (s.N + blocks - 1) / blocks;
  a.bias_lds = (s.act != 0 && s.col_bias) ? 1 : 0;
  int off = 2 * 4 * kK * 2 * kRowTileCols;   // two tile buffers of 4 codebooks x 16 rows x 1 KB
  a.off_ring = off;
  off += kFRing * (12 * 64 + 4);
  a.off_bias = off;
  off += a.bias_lds ? round_up(s.M * 4, 16) : 0;
  a.lds_total = off;
  if (off > kLdsBytes) return false;
  Shape q = s;
  q.mode = kAccum;
  q.idx_in = s.idx_out ? s.idx_out : reinterpret_cast<const uint8_t*>(s.y);
  q.idx_out = nullptr;
  if (!plan_trow(q, companion, true, s.idx_out ? (int64_t)s.C : (int64_t)s.M * 4)) return false;
  *f = a;
  *blocks_out = blocks;
  return true;
}

// Rounded 8-bit averaging accumulate (tiled_accum.hip): 8 wavefronts, the
// whole column slice of the table (C x 16 x Mt bytes, at most 128 KB) in LDS,
// 16 columns per lane.
bool plan_tavg(const Shape& s, TArgs* t, int* nw_out) {
  if ((int64_t)s.C * kK * s.M >= (1ll << 31)) return false;   // 32-bit buffer offsets
  if (s.C > 128) return false;   // the index batch must fit next to the table slice
  const int nw = 8;
  const int C8 = round_up(s.C, 8);   // staged codebooks: whole groups of 8
  int Mt = 256;
  while (Mt > 16 && (int64_t)(C8 + 1) * kK * Mt > 136 * 1024) Mt /= 2;   // + a padding block
  // no wider than the outputs, while a batch of the narrower tile's minimum
  // rows (8 wavefronts x 64 / lanes-per-row rows) still fits the staging
  while (Mt > 16 && Mt / 2 >= s.M && nw * (64 / (Mt / 32)) * s.C <= 16 * 1024) Mt /= 2;
  if ((int64_t)(C8 + 1) * kK * Mt > 136 * 1024) return false;
  TArgs a{};
  a.idx = s.idx_in; a.lut = s.lut; a.scale = s.scale; a.offset = s.offset; a.y = s.y; a.acc = s.acc;
  a.N = s.N; a.C = s.C; a.M = s.M;
  a.Mt = Mt;
  a.lpr_log2 = ilog2(Mt / 16);
  a.CT = 8;
  a.ntm = (s.M + Mt - 1) / Mt;
  a.vec_lut = aligned(s.lut, 16) && (s.M % 16 == 0);
  a.vec_idx = (s.C % 4 == 0) && aligned(s.idx_in, 4);
  a.vec_out = (s.M % 4 == 0) && (s.y == nullptr || aligned(s.y, 16)) && (s.acc == nullptr || aligned(s.acc, 16));
  int off = 0;
  auto take = [&](int bytes) { const int o = off; off += round_up(bytes, 16); return o; };
  // index batches: B rows of C bytes, at most 16 KB and two 16-byte units per thread
  const int RS = 64 / (Mt / 16);
  int nwb = nw;   // 512-thread workgroups
  while (nwb > 8 && nwb * RS * s.C > 16 * 1024) nwb /= 2;
  if (nwb * RS * s.C > 16 * 1024) return false;
  int J = 1;
  while (2 * J * nwb * RS * s.C <= 16 * 1024) J *= 2;
  a.RB = nwb * RS * J;
  if ((a.RB * s.C) % 16 != 0 || (a.RB * s.C) / 16 > 2 * nwb * 64) return false;
  a.off_tab = take((C8 + 1) * kK * Mt);   // 0: the kernel relies on it
  a.off_idx = take(a.RB * s.C + 16);   // + the (at most 7) bytes a last row's partial group reads past its end
  a.off_misc = take(16);
  a.lds_total = off;
  if (off > kLdsBytes) return false;
  *t = a;
  *nw_out = nwb;
  return true;
}

// One-hot product on the matrix cores (onehot_mfma.hip): int8 tables with
// C % 16 == 0 and 48 <= C <= 128, M % 4 == 0 and M >= 128, a 4-byte aligned
// table, 8-byte aligned index rows and 16-byte aligned outputs, at row counts
// where each of the workgroups (one per CU) gets whole tiles of rows to
// stream.  (Fewer codebooks or columns would leave half of the products on
// padding; such tables fit the gather-fused kernel, which takes them: the
// 131072 x 64 output of a 32-codebook layer in 19 against 31 us.)
constexpr int64_t kMaccMinRows = 16384;
bool macc_shape(const Shape& s) {   // (everything but the index rows' alignment)
  if (s.elem != kI8 || s.C % 16 != 0 || s.C < 48 || s.C > 128 || s.M % 4 != 0 || s.M < 128) return false;
  if (s.N < kMaccMinRows) return false;
  if (!aligned(s.lut, 4)) return false;
  if ((s.y && !aligned(s.y, 16)) || (s.acc && !aligned(s.acc, 16))) return false;
  return (int64_t)s.C * kK * s.M < (1ll << 31);
}
bool plan_macc(const Shape& s, MArgs* m, int* blocks_out) {
  if (!macc_shape(s) || !aligned(s.idx_in, 8)) return false;
  const int W = macc_width(s.C);
  MArgs a{};
  a.idx = s.idx_in; a.lut = static_cast<const int8_t*>(s.lut); a.scale = s.scale; a.offset = s.offset;
  a.y = s.y; a.acc = s.acc; a.col_bias = s.col_bias;
  a.N = s.N; a.C = s.C; a.M = s.M;
  a.act = s.act == 3 ? 1 : s.act;   // the softmax as a second pass
  a.bias_lds = (a.act != 0 && s.col_bias) ? 1 : 0;
  a.nslices = (s.M + W - 1) / W;
  int groups = device_cus() / a.nslices;
  if (groups < 1) groups = 1;
  a.xcd_map = (groups * a.nslices) % 8 == 0;
  a.rows_per_group = round_up64((s.N + groups - 1) / groups, 64);
  if (a.rows_per_group * s.M * 4 >= (1ll << 31)) return false;   // a group's outputs: 32-bit store offsets
  int off = (s.C <= 64 ? 64 : 128) * W * 16;   // the transposed table slice
  auto take = [&](int bytes) { const int o = off; off += round_up(bytes, 16); return o; };
  const int cp = s.C <= 64 ? 64 : 128;
  a.off_val = take(kMaccGroups * cp);
  a.off_sh = take(4 * cp);
  a.off_misc = take(16);
  a.off_bias = take(4 * W);
  a.lds_total = off;
  if (off > kLdsBytes) return false;
  *m = a;
  *blocks_out = groups * a.nslices;
  return true;
}

// Accumulate-only work: the column-tiled kernel, else the general path.
int accumulate(const Shape& s, hipStream_t stream) {
  TArgs t;
  int nj, nw;
  MArgs m;
  int mb;
  if (plan_macc(s, &m, &mb)) {
    const int rc = status_from(launch_macc(m, mb, stream));
    if (rc != MADDNESS_OK || m.act == s.act) return rc;
    return status_from(launch_softmax_rows(s.y, s.N, s.M, device_cus(), stream));
  }
  if (plan_rlane(s, &t)) {
    const int rc = status_from(launch_rlane_f32(t, device_cus(), stream));
    if (rc != MADDNESS_OK || t.act == s.act) return rc;
    return status_from(launch_softmax_rows(s.y, s.N, s.M, device_cus(), stream));
  }
  TArgs wide;
  if (plan_rlane_i8(s, &t, &wide)) {
    int rc = status_from(launch_rlane_i8(t, device_cus(), stream));
    if (rc == MADDNESS_OK) rc = status_from(launch_trow(kI8, wide, device_cus(), stream));
    if (rc != MADDNESS_OK || t.act == s.act) return rc;
    return status_from(launch_softmax_rows(s.y, s.N, s.M, device_cus(), stream));
  }
  if (plan_trow(s, &t)) {
    const int rc = status_from(launch_trow(s.elem, t, device_cus(), stream));
    if (rc != MADDNESS_OK || t.act == s.act) return rc;
    return status_from(launch_softmax_rows(s.y, s.N, s.M, device_cus(), stream));
  }
  {
    // C divides 64 and the table fits in LDS: the gather-fused kernel with
    // index loads in place of the encode
    GArgs g;
    int ng, uq, gnw;
    if (plan_gfused(s, &g, &ng, &uq, &gnw)) {
      g.idx_in = s.idx_in;
      return status_from(launch_gfused(s.elem, ng, uq, g, gnw, device_cus(), stream));
    }
  }
  if (plan_tacc(s, &t, &nj, &nw)) {
    const int rc = status_from(launch_tacc(s.elem, nj, t, nw, device_cus(), stream));
    if (rc != MADDNESS_OK || t.act == s.act) return rc;
    return status_from(launch_softmax_rows(s.y, s.N, s.M, device_cus(), stream));
  }
  if (s.act != 0) return MADDNESS_EUNSUPPORTED;   // the general path has no sigma epilogue
  return run(s, false, stream);
}


// ----------------------------------------------------------------- checks
int check_encode_args(const float* A, int64_t N, int32_t D, int64_t lda, const int32_t* split,
                      const float* thr, int32_t C) {
  if (N < 0 || D <= 0 || C <= 0 || lda < D) return MADDNESS_EINVAL;
  if (N == 0) return C > kMaxC ? MADDNESS_EUNSUPPORTED : MADDNESS_OK;
  if (!A || !split || !thr) return MADDNESS_EINVAL;
  if (!aligned(A, 4) || !aligned(split, 4) || !aligned(thr, 4)) return MADDNESS_EINVAL;
  if (C > kMaxC) return MADDNESS_EUNSUPPORTED;
  return MADDNESS_OK;
}

int check_accum_args(int64_t N, int32_t C, const void* lut, int32_t M) {
  if (N < 0 || C <= 0 || M <= 0) return MADDNESS_EINVAL;
  if (N == 0) return C > kMaxC ? MADDNESS_EUNSUPPORTED : MADDNESS_OK;
  if (!lut) return MADDNESS_EINVAL;
  if (C > kMaxC) return MADDNESS_EUNSUPPORTED;
  return MADDNESS_OK;
}

Shape shape(int mode, int elem) {
  Shape s{};
  s.mode = mode;
  s.elem = elem;
  return s;
}

// Two-phase path for tables larger than the single-launch kernels take:
// encode into the caller's index array, then accumulate from it.
int two_phase(const Shape& s, uint8_t* idx, hipStream_t stream) {
  Shape e = s;
  e.mode = kEncode;
  e.idx_out = idx;
  int rc = run(e, false, stream);
  if (rc != MADDNESS_OK) return rc;
  Shape q = s;
  q.mode = kAccum;
  q.idx_in = idx;
  q.idx_out = nullptr;
  return accumulate(q, stream);
}

// Whether a fused call that the row-streaming kernel could take runs faster
// as encode + the one-hot product, through an index array: measured on 1M
// rows of 512 columns of A with 64 codebooks, 0.84 against 1.05 ms at 512
// output columns, 0.62 against 0.94 at 256, 0.51 against 0.89 at 128 (the
// encode alone is 0.37 ms).  Not for a row softmax, which the row-streaming
// kernel fuses and the two-phase path runs as a pass of its own.
constexpr int kTwoPhaseMinCols = 128;
bool two_phase_faster(const Shape& s) {
  FArgs f;
  int blocks;
  return s.act != 3 && s.M >= kTwoPhaseMinCols && macc_shape(s) && plan_fenc(s, &f, &blocks, nullptr, 0);
}

// Whether a fused call runs as one launch (the gather-fused kernel, or the
// general kernel with the whole table in one column tile; the latter has no
// layer-output epilogue).
bool single_launch(const Shape& s) {
  GArgs g;
  int ng, uq, nw;
  if (plan_gfused(s, &g, &ng, &uq, &nw)) return true;
  FArgs f;
  int blocks;
  if (plan_fenc(s, &f, &blocks, nullptr, 0)) return true;   // (needs no index array)
  Plan p;
  return s.act == 0 && plan(s, &p, true) == MADDNESS_OK;
}

// Every fused entry point: one launch when the shape allows it, else the
// two-phase path through the caller's index array (required there).  When
// the table's rows are not whole 16-byte units the gather-fused kernel stages
// them element by element, and the general kernel (rows of A staged with
// 16-byte loads, no dependent gather) is faster on such layers (the tiny
// classifier, M = 10: 6.9 against 10.5 us per call, at 256 to 16384 rows);
// it has no layer-output epilogue, so it takes act == 0 only.
int fused(const Shape& s, hipStream_t st) {
  GArgs g;
  int ng, uq, nw;
  Plan p;
  const bool gf = plan_gfused(s, &g, &ng, &uq, &nw);
  if (gf && !g.vec16 && s.act == 0 && plan(s, &p, true) == MADDNESS_OK)
    return status_from(launch_path(s.mode, s.elem, p.pf, p.uq, p.a, p.grid, p.block, st));
  if (gf) return status_from(launch_gfused(s.elem, ng, uq, g, nw, device_cus(), st));
  FArgs f;
  TArgs t;
  int blocks;
  // (given an index array the row-streaming kernel's shapes may go faster
  // in two phases; without one they take that kernel, as one launch)
  const bool two = s.idx_out && aligned(s.idx_out, 8) && two_phase_faster(s);
  if (!two && plan_fenc(s, &f, &blocks, &t, device_cus())) {
    const int rc = status_from(launch_fenc(f, blocks, st));
    if (rc != MADDNESS_OK) return rc;
    return status_from(launch_trow(kI8, t, device_cus(), st));
  }
  if (s.act == 0 && plan(s, &p, true) == MADDNESS_OK)
    return status_from(launch_path(s.mode, s.elem, p.pf, p.uq, p.a, p.grid, p.block, st));
  if (!s.idx_out) return MADDNESS_EINVAL;
  return two_phase(s, s.idx_out, st);
}

// Device address of `scratch` on the current device, resolved once per device
// (hipGetSymbolAddress with that device current) and cached; nullptr with
// *rc = EHIP when the device or the symbol cannot be queried.
uint8_t* scratch_base(int* rc) {
  constexpr int kDevs = 64;
  static std::mutex mu;
  static uint8_t* base[kDevs] = {};
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kDevs) {
    *rc = MADDNESS_EHIP;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!base[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      *rc = MADDNESS_EHIP;
      return nullptr;
    }
    base[dev] = static_cast<uint8_t*>(p);
  }
  return base[dev];
}

}  // namespace
}  // namespace mdn

using namespace mdn;

extern "C" {

int maddness_version(void) { return 100; }

const char* maddness_status_string(int status) {
  switch (status) {
    case MADDNESS_OK: return "ok";
    case MADDNESS_EINVAL: return "invalid argument";
    case MADDNESS_EHIP: return "HIP runtime error";
    case MADDNESS_EUNSUPPORTED: return "unsupported shape";
    case MADDNESS_ENOMEM: return "out of device memory (reserved)";
    default: return "unknown status";
  }
}

int maddness_encode(const float* A, int64_t N, int32_t D, int64_t lda, const int32_t* split_dims,
                    const float* thresholds, int32_t C, uint8_t* idx_out, void* stream) {
  int rc = check_encode_args(A, N, D, lda, split_dims, thresholds, C);
  if (rc != MADDNESS_OK || N == 0) return rc;
  if (!idx_out) return MADDNESS_EINVAL;
  Shape s = shape(kEncode, kI8);
  s.A = A; s.N = N; s.D = D; s.lda = lda; s.split = split_dims; s.thr = thresholds; s.C = C;
  s.M = 1; s.idx_out = idx_out;
  return run(s, false, static_cast<hipStream_t>(stream));
}

int maddness_lut_accumulate(const uint8_t* idx, int64_t N, int32_t C, const int8_t* lut,
                            const float* scale, const float* offset, int32_t M, int32_t* acc_out,
                            float* y_out, void* stream) {
  int rc = check_accum_args(N, C, lut, M);
  if (rc != MADDNESS_OK || N == 0) return rc;
  if (!idx || !scale || !offset || (!acc_out && !y_out)) return MADDNESS_EINVAL;
  if (!aligned(scale, 4) || !aligned(offset, 4) || (acc_out && !aligned(acc_out, 4)) ||
      (y_out && !aligned(y_out, 4)))
    return MADDNESS_EINVAL;
  Shape s = shape(kAccum, kI8);
  s.idx_in = idx; s.N = N; s.C = C; s.lut = lut; s.scale = scale; s.offset = offset; s.M = M;
  s.acc = acc_out; s.y = y_out;
  return accumulate(s, static_cast<hipStream_t>(stream));
}

int maddness_lut_accumulate_avg(const uint8_t* idx, int64_t N, int32_t C, const int8_t* lut,
                                const float* scale, const float* offset, int32_t M, int32_t* acc_out,
                                float* y_out, void* stream) {
  int rc = check_accum_args(N, C, lut, M);
  if (rc != MADDNESS_OK || N == 0) return rc;
  if (!idx || !scale || !offset || (!acc_out && !y_out)) return MADDNESS_EINVAL;
  if (!aligned(scale, 4) || !aligned(offset, 4) || (acc_out && !aligned(acc_out, 4)) ||
      (y_out && !aligned(y_out, 4)) || !aligned(idx, 16))
    return MADDNESS_EINVAL;
  Shape s = shape(kAccum, kI8);
  s.idx_in = idx; s.N = N; s.C = C; s.lut = lut; s.scale = scale; s.offset = offset; s.M = M;
  s.acc = acc_out; s.y = y_out;
  TArgs t;
  int nw;
  if (!plan_tavg(s, &t, &nw)) return MADDNESS_EUNSUPPORTED;
  return status_from(launch_tavg(t, nw, device_cus(), static_cast<hipStream_t>(stream)));
}

int maddness_lut_accumulate_f32(const uint8_t* idx, int64_t N, int32_t C, const float* lut, int32_t M,
                                float* y_out, void* stream) {
  int rc = check_accum_args(N, C, lut, M);
  if (rc != MADDNESS_OK || N == 0) return rc;
  if (!idx || !y_out || !aligned(lut, 4) || !aligned(y_out, 4)) return MADDNESS_EINVAL;
  Shape s = shape(kAccum, kF32);
  s.idx_in = idx; s.N = N; s.C = C; s.lut = lut; s.M = M; s.y = y_out;
  return accumulate(s, static_cast<hipStream_t>(stream));
}

int maddness_matmul(const float* A, int64_t N, int32_t D, int64_t lda, const int32_t* split_dims,
                    const float* thresholds, int32_t C, const int8_t* lut, const float* scale,
                    const float* offset, int32_t M, float* y_out, int32_t* acc_out, uint8_t* idx_out,
                    void* stream) {
  int rc = check_encode_args(A, N, D, lda, split_dims, thresholds, C);
  if (rc != MADDNESS_OK) return rc;
  rc = check_accum_args(N, C, lut, M);
  if (rc != MADDNESS_OK || N == 0) return rc;
  if (!scale || !offset || !y_out || !aligned(scale, 4) || !aligned(offset, 4) || !aligned(y_out, 4) ||
      (acc_out && !aligned(acc_out, 4)))
    return MADDNESS_EINVAL;
  Shape s = shape(kFused, kI8);
  s.A = A; s.N = N; s.D = D; s.lda = lda; s.split = split_dims; s.thr = thresholds; s.C = C;
  s.lut = lut; s.scale = scale; s.offset = offset; s.M = M; s.y = y_out; s.acc = acc_out;
  s.idx_out = idx_out;
  return fused(s, static_cast<hipStream_t>(stream));
}

int maddness_matmul_f32(const float* A, int64_t N, int32_t D, int64_t lda, const int32_t* split_dims,
                        const float* thresholds, int32_t C, const float* lut, int32_t M, float* y_out,
                        uint8_t* idx_out, void* stream) {
  int rc = check_encode_args(A, N, D, lda, split_dims, thresholds, C);
  if (rc != MADDNESS_OK) return rc;
  rc = check_accum_args(N, C, lut, M);
  if (rc != MADDNESS_OK || N == 0) return rc;
  if (!y_out || !aligned(lut, 4) || !aligned(y_out, 4)) return MADDNESS_EINVAL;
  Shape s = shape(kFused, kF32);
  s.A = A; s.N = N; s.D = D; s.lda = lda; s.split = split_dims; s.thr = thresholds; s.C = C;
  s.lut = lut; s.M = M; s.y = y_out; s.idx_out = idx_out;
  return fused(s, static_cast<hipStream_t>(stream));
}

int maddness_matmul_act(const float* A, int64_t N, int32_t D, int64_t lda, const int32_t* split_dims,
                        const float* thresholds, int32_t C, const int8_t* lut, const float* scale,
                        const float* offset, int32_t M, const float* col_bias, int32_t act, float* y_out,
                        uint8_t* idx_out, void* stream) {
  if (act < MADDNESS_ACT_NONE || act > MADDNESS_ACT_SOFTMAX) return MADDNESS_EINVAL;
  int rc = check_encode_args(A, N, D, lda, split_dims, thresholds, C);
  if (rc != MADDNESS_OK) return rc;
  rc = check_accum_args(N, C, lut, M);
  if (rc != MADDNESS_OK || N == 0) return rc;
  if (!scale || !offset || !y_out || !aligned(scale, 4) || !aligned(offset, 4) || !aligned(y_out, 4) ||
      (col_bias && !aligned(col_bias, 4)))
    return MADDNESS_EINVAL;
  Shape s = shape(kFused, kI8);
  s.A = A; s.N = N; s.D = D; s.lda = lda; s.split = split_dims; s.thr = thresholds; s.C = C;
  s.lut = lut; s.scale = scale; s.offset = offset; s.M = M; s.y = y_out;
  s.col_bias = col_bias; s.act = act; s.idx_out = idx_out;
  return fused(s, static_cast<hipStream_t>(stream));
}

int maddness_matmul_act_f32(const float* A, int64_t N, int32_t D, int64_t lda, const int32_t* split_dims,
                            const float* thresholds, int32_t C, const float* lut, int32_t M,
                            const float* col_bias, int32_t act, float* y_out, uint8_t* idx_out, void* stream) {
  if (act < MADDNESS_ACT_NONE || act > MADDNESS_ACT_SOFTMAX) return MADDNESS_EINVAL;
  int rc = check_encode_args(A, N, D, lda, split_dims, thresholds, C);
  if (rc != MADDNESS_OK) return rc;
  rc = check_accum_args(N, C, lut, M);
  if (rc != MADDNESS_OK || N == 0) return rc;
  if (!y_out || !aligned(lut, 4) || !aligned(y_out, 4) || (col_bias && !aligned(col_bias, 4)))
    return MADDNESS_EINVAL;
  Shape s = shape(kFused, kF32);
  s.A = A; s.N = N; s.D = D; s.lda = lda; s.split = split_dims; s.thr = thresholds; s.C = C;
  s.lut = lut; s.M = M; s.y = y_out;
  s.col_bias = col_bias; s.act = act; s.idx_out = idx_out;
  return fused(s, static_cast<hipStream_t>(stream));
}

int maddness_matmul_noalloc(const float* A, int64_t N, int32_t D, int64_t lda, const int32_t* split_dims,
                            const float* thresholds, int32_t C, const int8_t* lut, const float* scale,
                            const float* offset, int32_t M, float* y_out, int32_t* acc_out, uint8_t* idx_out,
                            void* stream) {
  int rc = check_encode_args(A, N, D, lda, split_dims, thresholds, C);
  if (rc != MADDNESS_OK) return rc;
  rc = check_accum_args(N, C, lut, M);
  if (rc != MADDNESS_OK || N == 0) return rc;
  if (!scale || !offset || !y_out || !aligned(scale, 4) || !aligned(offset, 4) || !aligned(y_out, 4) ||
      (acc_out && !aligned(acc_out, 4)))
    return MADDNESS_EINVAL;
  Shape s = shape(kFused, kI8);
  s.A = A; s.N = N; s.D = D; s.lda = lda; s.split = split_dims; s.thr = thresholds; s.C = C;
  s.lut = lut; s.scale = scale; s.offset = offset; s.M = M; s.y = y_out; s.acc = acc_out;
  s.idx_out = idx_out;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (idx_out || single_launch(s)) return fused(s, st);
  uint8_t* idx = scratch_base(&rc);
  if (!idx) return rc;
  // rows per chunk: as many whole 256-row groups as the scratch holds (C <=
  // 512, so at least 65536 rows); each chunk is encoded into the scratch and
  // accumulated from it before the next chunk's encode, in stream order
  const int64_t chunk = (kScratchBytes / C) / 256 * 256;
  for (int64_t r0 = 0; r0 < N; r0 += chunk) {
    Shape c = s;
    c.N = (N - r0 < chunk) ? N - r0 : chunk;
    c.A = A + r0 * lda;
    c.y = y_out + r0 * M;
    c.acc = acc_out ? acc_out + r0 * M : nullptr;
    rc = two_phase(c, idx, st);
    if (rc != MADDNESS_OK) return rc;
  }
  return MADDNESS_OK;
}

int64_t maddness_matmul_index_bytes(const float* A, int64_t N, int32_t D, int64_t lda, int32_t C, int32_t M,
                                    int32_t f32, int32_t act) {
  if (N < 0 || D <= 0 || C <= 0 || M <= 0 || lda < D) return -1;
  if (act < MADDNESS_ACT_NONE || act > MADDNESS_ACT_SOFTMAX) return -1;
  if (C > kMaxC) return -3;
  if (N == 0) return 0;
  if (!A || !aligned(A, 4)) return -1;
  Shape s = shape(kFused, f32 ? kF32 : kI8);
  s.A = A; s.N = N; s.D = D; s.lda = lda; s.C = C; s.M = M; s.act = act;
  return (two_phase_faster(s) || !single_launch(s)) ? N * (int64_t)C : 0;
}

int maddness_build_lut(const float* P, const float* B, int32_t C, int32_t D, int32_t M, int8_t* lut_out,
                       float* scale_out, float* offset_out, void* stream) {
  if (C <= 0 || D <= 0 || M <= 0 || !P || !B || !lut_out || !scale_out || !offset_out)
    return MADDNESS_EINVAL;
  if (!aligned(P, 4) || !aligned(B, 4) || !aligned(scale_out, 4) || !aligned(offset_out, 4))
    return MADDNESS_EINVAL;
  if (127.0 * C >= 16777216.0) return MADDNESS_EINVAL;
  if (C > kMaxC) return MADDNESS_EUNSUPPORTED;
  int cap = 0;
  while (127.0 * C * (double)(1ll << (cap + 1)) < 16777216.0) ++cap;
  return status_from(launch_build_lut(P, B, C, D, M, lut_out, scale_out, offset_out, cap,
                                      static_cast<hipStream_t>(stream)));
}

int maddness_build_lut_shared(const float* P, const float* B, int32_t C, int32_t D, int32_t M, int8_t* lut_out,
                              float* scale_out, float* offset_out, void* stream) {
  if (C <= 0 || D <= 0 || M <= 0 || !P || !B || !lut_out || !scale_out || !offset_out)
    return MADDNESS_EINVAL;
  if (!aligned(P, 4) || !aligned(B, 4) || !aligned(scale_out, 4) || !aligned(offset_out, 4))
    return MADDNESS_EINVAL;
  if (C > kMaxC) return MADDNESS_EUNSUPPORTED;
  return status_from(launch_build_lut(P, B, C, D, M, lut_out, scale_out, offset_out, 0,
                                      static_cast<hipStream_t>(stream)));
}

int maddness_quantize_lut(const double* T, int32_t C, int32_t M, int32_t shared, int8_t* lut_out,
                          float* scale_out, float* offset_out, void* stream) {
  if (C <= 0 || M <= 0 || !T || !lut_out || !scale_out || !offset_out) return MADDNESS_EINVAL;
  if (!aligned(T, 8) || !aligned(scale_out, 4) || !aligned(offset_out, 4)) return MADDNESS_EINVAL;
  if (127.0 * C >= 16777216.0) return MADDNESS_EINVAL;
  if (C > kMaxC) return MADDNESS_EUNSUPPORTED;
  int cap = 0;
  if (!shared)
    while (127.0 * C * (double)(1ll << (cap + 1)) < 16777216.0) ++cap;
  return status_from(launch_quantize_lut(T, C, M, lut_out, scale_out, offset_out, cap,
                                         static_cast<hipStream_t>(stream)));
}

int maddness_encoder_gram(const uint8_t* idx, int64_t N, int32_t C, int32_t* gram_out, void* stream) {
  if (N < 0 || C <= 0 || !gram_out || (N > 0 && !idx)) return MADDNESS_EINVAL;
  if (!aligned(gram_out, 4)) return MADDNESS_EINVAL;
  if (C > kMaxFitC || N >= (1ll << 31)) return MADDNESS_EUNSUPPORTED;   // int32 counts
  return status_from(launch_gram(idx, N, C, gram_out, device_cus(), static_cast<hipStream_t>(stream)));
}

int64_t maddness_encoder_scatter_workspace_bytes(int64_t N, int32_t C) {
  if (N < 0 || N >= (1ll << 31) || C <= 0 || C > kMaxFitC) return -1;
  return round_up64((int64_t)C * (N + 128) * 4, 256) + (int64_t)C * (kK + 1) * 4;   // row lists + 128 padding each
}

int maddness_encoder_scatter(const uint8_t* idx, int64_t N, int32_t C, const float* Y, int32_t M, double* out,
                             void* workspace, int64_t workspace_bytes, void* stream) {
  if (N < 0 || C <= 0 || M <= 0 || !out || !workspace || (N > 0 && (!idx || !Y))) return MADDNESS_EINVAL;
  if (!aligned(out, 8) || !aligned(workspace, 256) || (N > 0 && !aligned(Y, 4))) return MADDNESS_EINVAL;
  if (C > kMaxFitC || N >= (1ll << 31)) return MADDNESS_EUNSUPPORTED;
  if (workspace_bytes < maddness_encoder_scatter_workspace_bytes(N, C)) return MADDNESS_EINVAL;
  int32_t* perm = static_cast<int32_t*>(workspace);
  int32_t* start = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + round_up64((int64_t)C * (N + 128) * 4, 256));
  return status_from(launch_scatter(idx, N, C, Y, M, out, perm, start, static_cast<hipStream_t>(stream)));
}

int64_t maddness_fit_lut_workspace_bytes(int64_t N, int32_t C) {
  const int64_t ws = maddness_encoder_scatter_workspace_bytes(N, C);
  if (ws < 0) return -1;
  const int64_t n = (int64_t)C * kK;
  return round_up64(n * n * 4, 256) + round_up64(n * n * 8, 256) + ws;
}

int maddness_fit_lut_ridge(const uint8_t* idx, int64_t N, int32_t C, const float* Y, int32_t M, const float* T0,
                           double lambda, double* T_out, void* workspace, int64_t workspace_bytes, void* stream) {
  if (N < 0 || C <= 0 || M <= 0 || !T0 || !T_out || !workspace || (N > 0 && (!idx || !Y)))
    return MADDNESS_EINVAL;
  if (!(lambda > 0.0) || !std::isfinite(lambda)) return MADDNESS_EINVAL;
  if (!aligned(T_out, 8) || !aligned(T0, 4) || !aligned(workspace, 256) || (N > 0 && !aligned(Y, 4)))
    return MADDNESS_EINVAL;
  if (C > kMaxFitC || N >= (1ll << 31)) return MADDNESS_EUNSUPPORTED;
  const int64_t need = maddness_fit_lut_workspace_bytes(N, C);
  if (workspace_bytes < need) return MADDNESS_EINVAL;
  const int64_t n = (int64_t)C * kK;
  char* w = static_cast<char*>(workspace);
  int32_t* H = reinterpret_cast<int32_t*>(w);
  w += round_up64(n * n * 4, 256);
  double* A = reinterpret_cast<double*>(w);
  w += round_up64(n * n * 8, 256);
  int32_t* perm = reinterpret_cast<int32_t*>(w);
  int32_t* start = reinterpret_cast<int32_t*>(w + round_up64((int64_t)C * (N + 128) * 4, 256));
  return status_from(launch_fit_ridge(idx, N, C, Y, M, T0, lambda, T_out, H, A, perm, start, device_cus(),
                                      static_cast<hipStream_t>(stream)));
}

int64_t maddness_fit_lut_gd_workspace_bytes(int64_t N, int32_t C, int32_t M) {
  const int64_t ws = maddness_encoder_scatter_workspace_bytes(N, C);
  if (ws < 0 || M <= 0) return -1;
  return 2 * round_up64(N * M * 8, 256) + round_up64((int64_t)C * kK * M * 8, 256) + ws;
}

int maddness_fit_lut_gd(const uint8_t* idx, int64_t N, int32_t C, const float* Y, int32_t M, const float* col_bias,
                        int32_t act, const float* T0, double lambda, double eta, int32_t iters, double* T_out,
                        void* workspace, int64_t workspace_bytes, void* stream) {
  if (N < 0 || C <= 0 || M <= 0 || !T0 || !T_out || !workspace || (N > 0 && (!idx || !Y)))
    return MADDNESS_EINVAL;
  if (act != MADDNESS_FIT_RELU_SQERR && act != MADDNESS_FIT_SOFTMAX_KLD && act != MADDNESS_FIT_SOFTMAX_SQERR)
    return MADDNESS_EINVAL;
  if (!(lambda >= 0.0) || !std::isfinite(lambda) || !(eta > 0.0) || !std::isfinite(eta) || iters < 0)
    return MADDNESS_EINVAL;
  if (!aligned(T_out, 8) || !aligned(T0, 4) || !aligned(workspace, 256) || (N > 0 && !aligned(Y, 4)) ||
      (col_bias && !aligned(col_bias, 4)))
    return MADDNESS_EINVAL;
  if (C > kMaxFitC || N >= (1ll << 31)) return MADDNESS_EUNSUPPORTED;
  if (workspace_bytes < maddness_fit_lut_gd_workspace_bytes(N, C, M)) return MADDNESS_EINVAL;
  char* w = static_cast<char*>(workspace);
  double* P = reinterpret_cast<double*>(w);
  w += round_up64(N * M * 8, 256);
  double* D = reinterpret_cast<double*>(w);
  w += round_up64(N * M * 8, 256);
  double* R = reinterpret_cast<double*>(w);
  w += round_up64((int64_t)C * kK * M * 8, 256);
  int32_t* perm = reinterpret_cast<int32_t*>(w);
  int32_t* start = reinterpret_cast<int32_t*>(w + round_up64((int64_t)C * (N + 128) * 4, 256));
  return status_from(launch_fit_gd(idx, N, C, Y, M, col_bias, act, T0, lambda, eta, iters, T_out, P, D, R, perm,
                                   start, static_cast<hipStream_t>(stream)));
}

int maddness_build_lut_f32(const float* P, const float* B, int32_t C, int32_t D, int32_t M, float* lut_out,
                           void* stream) {
  if (C <= 0 || D <= 0 || M <= 0 || !P || !B || !lut_out) return MADDNESS_EINVAL;
  if (!aligned(P, 4) || !aligned(B, 4) || !aligned(lut_out, 4)) return MADDNESS_EINVAL;
  if (C > kMaxC) return MADDNESS_EUNSUPPORTED;
  return status_from(launch_build_lut_f32(P, B, C, D, M, lut_out, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
