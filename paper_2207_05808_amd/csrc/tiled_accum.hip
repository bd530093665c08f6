// Lookup-accumulate kernels for tables larger than LDS and for the
// accumulate-only entry points (§1 of McCarter & Dronen: the product is the
// sum over codebooks of the table rows the encoder selected):
//  * trow_kernel / trow_f32_kernel, the row-uniform kernels, for tables at
//    least 512 int8 or 256 fp32 columns wide (below);
//  * tacc_kernel, the column-tiled kernel, for every other shape (first);
//  * tavg_kernel, the rounded 8-bit summation (last);
//  * softmax_rows_kernel, the row softmax for rows spanning several tiles.
//
// Column-tiled kernel.
//
// A work item is RB rows x Mt output columns.  The lanes of a wavefront form
// groups of LPR lanes, one group per output row; lane g of a group covers Mt /
// LPR consecutive columns (8 for int8 tables, 4 for fp32), so the group reads
// one contiguous LPR x 16-byte segment of a table row (with LPR = 16: 256
// bytes, every LDS bank once).  The table is staged CT codebooks at a time,
// [CT * 16 rows][Mt columns], with the matching [RB][CT] tile of indices; the
// next tile's table units and indices are loaded into registers while the
// current tile is summed.  Accumulators stay in registers across codebook
// tiles, so fp32 sums keep the ascending codebook order.
//  * int8 tables whose shifted codes cannot overflow 16 bits in total
//    (128 * sum_c 2^(e_c - e_min) <= 32768) are staged as int16 q << (e_c -
//    e_min) and summed with packed 16-bit adds: modular arithmetic whose exact
//    total fits, so the sum equals the int32 sum;
//  * other int8 tables are staged as int16 q and summed in int32 with shifts;
//  * fp32 tables are summed with ordered fp32 adds.
// The last codebook tile is padded to a multiple of 4 codebooks with all-zero
// table rows.
#include "internal.hpp"

#include <climits>
#include <type_traits>

namespace mdn {

namespace {

typedef uint32_t tu32x4 __attribute__((ext_vector_type(4)));
typedef float tf32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char tlds_t;
typedef __attribute__((address_space(3))) uint32_t tlds_u32;
typedef __attribute__((address_space(3))) int32_t tlds_i32;
typedef __attribute__((address_space(3))) tu32x4 tlds_u32x4;
typedef __attribute__((address_space(3))) tf32x4 tlds_f32x4;
typedef __attribute__((address_space(3))) float tlds_f32;

constexpr int kBufDword3 = 0x00020000;   // raw, unswizzled buffer descriptor (gfx9 family)
constexpr int kTU = 4;                   // 16-byte table units per thread per tile (vector staging)
constexpr int kIU = 2;                   // 4-byte index words per thread per tile (vector staging)
constexpr int kOob = INT_MAX;            // buffer offset past any descriptor range: reads zero

__device__ __forceinline__ int tuni(int v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ uint32_t tpk_add16(uint32_t a, uint32_t b) {
  typedef short s2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, (s2)(__builtin_bit_cast(s2, a) + __builtin_bit_cast(s2, b)));
}

// max / sum over the 64 lanes of a wavefront, the same value in every lane:
// DPP within each row of 16 lanes (pairs, quads, mirrored halves, mirrored
// rows), then the four row results through readlane.  No LDS round trips.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}

template <bool MAX>
__device__ __forceinline__ float wave_reduce64(float x) {
  auto op = [](float a, float b) { return MAX ? __builtin_fmaxf(a, b) : a + b; };
  x = op(x, dpp_f32<0xB1>(x));    // quad_perm [1,0,3,2]
  x = op(x, dpp_f32<0x4E>(x));    // quad_perm [2,3,0,1]
  x = op(x, dpp_f32<0x141>(x));   // row_half_mirror
  x = op(x, dpp_f32<0x140>(x));   // row_mirror
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return op(op(r0, r1), op(r2, r3));
}

// four int8 codes -> two dwords of int16 q << sh (0 <= sh <= 8), column order
// kept: v_perm puts each code in the high byte of its 16-bit half, then a
// packed arithmetic shift right by 8 - sh sign-extends and scales it
__device__ __forceinline__ void widen4(uint32_t v, int sh, uint32_t& lo, uint32_t& hi) {
  typedef short s2 __attribute__((ext_vector_type(2)));
  const s2 r = {(short)(8 - sh), (short)(8 - sh)};
  lo = __builtin_bit_cast(uint32_t, __builtin_bit_cast(s2, __builtin_amdgcn_perm(0u, v, 0x010c000cu)) >> r);
  hi = __builtin_bit_cast(uint32_t, __builtin_bit_cast(s2, __builtin_amdgcn_perm(0u, v, 0x030c020cu)) >> r);
}

}  // namespace

// LDS layout (bytes): [table tile: CT*16 rows of Mt entries (int16 or fp32)]
// [index tile: RB x CT int32, each the LDS byte offset of the selected table
// row, (c_local * 16 + k) * row bytes][shift per codebook][misc]
template <int ELEM, int NJ>
__global__ void __launch_bounds__(512, 4) tacc_kernel(const TArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  tlds_t* smem = (tlds_t*)smem_raw;

  const int tid = threadIdx.x;
  const int nt = blockDim.x;
  const int lane = tid & 63;
  const int wave = tuni(tid >> 6);
  const int nw = nt >> 6;
  const int C = a.C, M = a.M, CT = a.CT, Mt = a.Mt, RB = a.RB;
  const int64_t N = a.N;
  const int lpr_log2 = a.lpr_log2;
  const int RS = 64 >> lpr_log2;          // output rows per wavefront pass
  const int r4 = lane >> lpr_log2;        // row within the pass
  const int cg = lane & ((1 << lpr_log2) - 1);
  constexpr int EB = (ELEM == kF32) ? 4 : 2;     // LDS bytes per staged entry
  constexpr int EG = (ELEM == kF32) ? 4 : 1;     // global bytes per entry
  constexpr int CPL = 16 / EB;                   // columns per lane (one 16-byte LDS read)
  const int rby = Mt * EB;                       // LDS bytes per table row (a power of two)
  const int rby_log2 = 31 - __builtin_clz(rby);

  tlds_t* s_tab = smem;   // the table tile starts the LDS block (off_tab == 0)
  tlds_t* s_idx = smem + a.off_idx;
  tlds_i32* s_sh = reinterpret_cast<tlds_i32*>(smem + a.off_sh);
  tlds_i32* s_misc = reinterpret_cast<tlds_i32*>(smem + a.off_misc);   // bias32, e_min, sum of 2^sh

  // ---------------- block exponents, shifts and bias32 (int8 tables)
  bool narrow = false;
  float step = 1.0f, bias = 0.0f;
  if (ELEM == kI8) {
    if (tid == 0) { s_misc[1] = INT_MAX; s_misc[2] = 0; }
    __syncthreads();
    const uint32_t* sb = reinterpret_cast<const uint32_t*>(a.scale);
    for (int c = tid; c < C; c += nt) atomicMin((int*)&s_misc[1], (int)((sb[c] >> 23) & 0xffu) - 127);
    __syncthreads();
    const int emin = tuni(s_misc[1]);
    for (int c = tid; c < C; c += nt) {
      const int sh = min((int)((sb[c] >> 23) & 0xffu) - 127 - emin, 30);
      s_sh[c] = sh;
      atomicAdd((int*)&s_misc[2], sh <= 14 ? (1 << sh) : (1 << 15));
    }
    if (wave == 0) {
      // bias32: double sum over codebooks in ascending order
      double sum = 0.0;
      for (int c0 = 0; c0 < C; c0 += 64) {
        const float ov = a.offset[min(c0 + lane, C - 1)];
        const int n = min(64, C - c0);
        for (int j = 0; j < n; ++j) sum += (double)__int_as_float(__builtin_amdgcn_readlane(__float_as_int(ov), j));
      }
      if (lane == 0) s_misc[0] = __float_as_int((float)sum);
    }
    __syncthreads();
    narrow = 128 * tuni(s_misc[2]) <= 32768;   // every int8 code, -128 included
    step = __builtin_ldexpf(1.0f, emin);
    bias = __int_as_float(tuni(s_misc[0]));
  }

  // ---------------- staging helpers
  const int upc = 16 / EG;              // columns per 16-byte global unit
  const int upr = Mt / upc;             // units per table row of the tile (a power of two)
  const int upr_log2 = __builtin_ctz(upr);
  const int units = CT * 16 * upr;      // units per tile
  const int iw = CT >> 2;               // index words per row of the index tile (a power of two)
  const int iw_log2 = __builtin_ctz(iw);
  const int iwords = RB * iw;
  const bool vec = a.vec_lut && a.vec_idx;
  const __amdgpu_buffer_rsrc_t trs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.lut), 0, (int)((int64_t)C * 16 * M * EG), kBufDword3);
  tu32x4 tv[kTU];
  uint32_t iv[kIU];

  // registers <- tile (c0) of work item (r0, m0); invalid units and words read zero
  auto load_tile = [&](int c0, int64_t r0, int m0) {
#pragma unroll
    for (int j = 0; j < kTU; ++j) {
      const int u = tid + j * nt;
      const int row = u >> upr_log2, part = u & (upr - 1);
      const int c = c0 + (row >> 4), m = m0 + part * upc;
      const bool ok = u < units && c < C && m < M;
      const int off = ok ? ((c * 16 + (row & 15)) * M + m) * EG : kOob;
      tv[j] = __builtin_amdgcn_raw_buffer_load_b128(trs, off, 0, 0);
    }
    const int64_t rows = min((int64_t)RB, N - r0);
    const __amdgpu_buffer_rsrc_t irs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(a.idx + r0 * C), 0, (int)min(rows * C, (int64_t)INT_MAX), kBufDword3);
#pragma unroll
    for (int j = 0; j < kIU; ++j) {
      const int d = tid + j * nt;
      const int i = d >> iw_log2, q = d & (iw - 1);
      const bool ok = d < iwords && c0 + 4 * q < C;
      iv[j] = __builtin_amdgcn_raw_buffer_load_b32(irs, ok ? i * C + c0 + 4 * q : kOob, 0, 0);
    }
  };
  // registers -> LDS
  auto store_tile = [&](int c0) {
#pragma unroll
    for (int j = 0; j < kTU; ++j) {
      const int u = tid + j * nt;
      if (u < units) {
        const int row = u >> upr_log2, part = u & (upr - 1);
        if (ELEM == kF32) {
          *reinterpret_cast<tlds_u32x4*>(s_tab + (row << rby_log2) + part * 16) = tv[j];
        } else {
          const int c = min(c0 + (row >> 4), C - 1);
          const int sh = narrow ? s_sh[c] : 0;
          uint32_t w[8];
          widen4(tv[j].x, sh, w[0], w[1]);
          widen4(tv[j].y, sh, w[2], w[3]);
          widen4(tv[j].z, sh, w[4], w[5]);
          widen4(tv[j].w, sh, w[6], w[7]);
          const tu32x4 lo = {w[0], w[1], w[2], w[3]}, hi = {w[4], w[5], w[6], w[7]};
          *reinterpret_cast<tlds_u32x4*>(s_tab + (row << rby_log2) + part * 32) = lo;
          *reinterpret_cast<tlds_u32x4*>(s_tab + (row << rby_log2) + part * 32 + 16) = hi;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < kIU; ++j) {
      const int d = tid + j * nt;   // index word d: row d / iw, codebooks 4 (d % iw) .. + 3 of the tile
      if (d < iwords) {
        const uint32_t cb = (uint32_t)(4 * (d & (iw - 1))) * 16u;
        tu32x4 o;
#pragma unroll
        for (int b = 0; b < 4; ++b) o[b] = (cb + 16u * b + ((iv[j] >> (8 * b)) & 15u)) << rby_log2;
        *reinterpret_cast<tlds_u32x4*>(s_idx + 16 * d) = o;
      }
    }
  };
  // general staging, straight from global memory (rows not in whole 16-byte
  // units, or index rows not in whole words)
  auto stage_direct = [&](int c0, int64_t r0, int m0) {
    const int8_t* q8 = reinterpret_cast<const int8_t*>(a.lut);
    const float* qf = reinterpret_cast<const float*>(a.lut);
    const int ent = CT * 16 * Mt;
    for (int e = tid; e < ent; e += nt) {
      const int row = e / Mt, col = e - row * Mt;
      const int c = c0 + (row >> 4), m = m0 + col;
      const bool ok = c < C && m < M;
      const int64_t g = ((int64_t)c * 16 + (row & 15)) * M + m;
      if (ELEM == kF32) {
        *reinterpret_cast<__attribute__((address_space(3))) float*>(s_tab + (row << rby_log2) + 4 * col) =
            ok ? qf[g] : 0.0f;
      } else {
        const int sh = narrow ? s_sh[min(c, C - 1)] : 0;
        *reinterpret_cast<__attribute__((address_space(3))) int16_t*>(s_tab + (row << rby_log2) + 2 * col) =
            ok ? (int16_t)((int)q8[g] << sh) : (int16_t)0;
      }
    }
    for (int e = tid; e < RB * CT; e += nt) {
      const int i = e / CT, cc = e - i * CT;
      const bool ok = r0 + i < N && c0 + cc < C;
      const uint32_t k = ok ? (uint32_t)(a.idx[(r0 + i) * C + c0 + cc] & 15u) : 0u;
      *reinterpret_cast<tlds_u32*>(s_idx + 4 * e) = ((uint32_t)cc * 16u + k) << rby_log2;
    }
  };

  // ---------------- work items: (column tile, row block), column tile fastest
  // this lane's 16 bytes of any table row, and its rows' index-tile entries:
  // a read address is then one add of an index-tile entry
  const tlds_t* s_tab_lane = s_tab + cg * 16;
  int ib[NJ];
  const tlds_t* s_idx_row[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    ib[j] = (j * nw + wave) * RS + r4;
    s_idx_row[j] = s_idx + ib[j] * CT * 4;
  }

  // MODE 0: fp32 tables; 1: int16 packed sums; 2: int32 sums with shifts
  auto run = [&](auto mode_tag) {
    constexpr int MODE = decltype(mode_tag)::value;
    for (int64_t w = blockIdx.x; w < a.nwork; w += gridDim.x) {
      const int mt = (int)(w % a.ntm);
      const int64_t r0 = (w / a.ntm) * RB;
      const int m0 = mt * Mt;

      constexpr int NACC = (MODE == 2) ? 8 : 4;
      uint32_t acc[NJ][NACC];   // fp32 bits, packed int16 pairs, or int32
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int e = 0; e < NACC; ++e) acc[j][e] = 0u;

      if (vec) load_tile(0, r0, m0);
      for (int c0 = 0; c0 < C; c0 += CT) {
        __syncthreads();   // every reader of the previous tile is done
        if (vec) store_tile(c0); else stage_direct(c0, r0, m0);
        __syncthreads();
        if (vec && c0 + CT < C) load_tile(c0 + CT, r0, m0);   // in flight during the sums below
        const int ncb = (min(CT, C - c0) + 3) & ~3;
        for (int cc = 0; cc < ncb; cc += 4) {
          tu32x4 kk[NJ];   // LDS offsets of the 4 selected table rows
#pragma unroll
          for (int j = 0; j < NJ; ++j) kk[j] = *reinterpret_cast<const tlds_u32x4*>(s_idx_row[j] + cc * 4);
          int shb[4] = {0, 0, 0, 0};
          if (MODE == 2) {
#pragma unroll
            for (int b = 0; b < 4; ++b) shb[b] = tuni(s_sh[min(c0 + cc + b, C - 1)]);   // zero rows: any shift
          }
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            tu32x4 v[4];
#pragma unroll
            for (int b = 0; b < 4; ++b) v[b] = *reinterpret_cast<const tlds_u32x4*>(s_tab_lane + kk[j][b]);
#pragma unroll
            for (int b = 0; b < 4; ++b) {   // codebooks strictly in ascending order
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                if (MODE == 0) {
                  acc[j][e] = __float_as_uint(__uint_as_float(acc[j][e]) + __uint_as_float(v[b][e]));
                } else if (MODE == 1) {
                  acc[j][e] = tpk_add16(acc[j][e], v[b][e]);
                } else {
                  acc[j][2 * e] += (uint32_t)(__builtin_amdgcn_sbfe((int)v[b][e], 0, 16) << shb[b]);
                  acc[j][2 * e + 1] += (uint32_t)(((int)v[b][e] >> 16) << shb[b]);
                }
              }
            }
          }
        }
      }

      // ---------------- epilogue
      const int col0 = m0 + cg * CPL;
      const int LPR = 1 << lpr_log2;
      float cb[CPL];   // this lane's column biases, loaded once (stores to y may alias them)
#pragma unroll
      for (int e = 0; e < CPL; ++e) cb[e] = (a.act != 0 && a.col_bias && col0 + e < M) ? a.col_bias[col0 + e] : 0.0f;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int64_t row = r0 + ib[j];
        int out[8];
        float yv[8];
#pragma unroll
        for (int e = 0; e < CPL; ++e) {
          if (MODE == 0) {
            out[e] = 0;
            yv[e] = __uint_as_float(acc[j][e]);
          } else {
            out[e] = (MODE == 1) ? ((e & 1) ? (int)acc[j][e >> 1] >> 16 : __builtin_amdgcn_sbfe((int)acc[j][e >> 1], 0, 16))
                                 : (int)acc[j][e];
            yv[e] = __builtin_fmaf((float)out[e], step, bias);
          }
        }
        if (a.act != 0) {
          // layer output sigma: z = y + bias, then ReLU, or a softmax over the
          // row's LPR lanes (a row lies in one column tile; every lane takes
          // part in the reductions)
          float vmax = -__builtin_inff();
#pragma unroll
          for (int e = 0; e < CPL; ++e) {
            const bool ok = col0 + e < M;
            float z = yv[e] + cb[e];
            if (a.act == 2) z = (z > 0.0f) ? z : 0.0f;
            yv[e] = z;
            if (ok) vmax = __builtin_fmaxf(vmax, z);
          }
          if (a.act == 3) {
            for (int o = 1; o < LPR; o <<= 1) vmax = __builtin_fmaxf(vmax, __shfl_xor(vmax, o));
            float sum = 0.0f;
#pragma unroll
            for (int e = 0; e < CPL; ++e) {
              yv[e] = (col0 + e < M) ? expf(yv[e] - vmax) : 0.0f;
              sum += yv[e];
            }
            for (int o = 1; o < LPR; o <<= 1) sum += __shfl_xor(sum, o);
#pragma unroll
            for (int e = 0; e < CPL; ++e) yv[e] = yv[e] / sum;
          }
        }
        if (row >= N || col0 >= M) continue;
        float* yr = a.y ? a.y + row * M + col0 : nullptr;
        int32_t* ar = (MODE != 0 && a.acc) ? a.acc + row * M + col0 : nullptr;
        if (a.vec_out && col0 + CPL <= M) {
#pragma unroll
          for (int h = 0; h < CPL / 4; ++h) {
            if (yr)
              __builtin_nontemporal_store((tf32x4){yv[4 * h], yv[4 * h + 1], yv[4 * h + 2], yv[4 * h + 3]},
                                          reinterpret_cast<tf32x4*>(yr + 4 * h));
            if (ar)
              __builtin_nontemporal_store((tu32x4){(uint32_t)out[4 * h], (uint32_t)out[4 * h + 1],
                                                   (uint32_t)out[4 * h + 2], (uint32_t)out[4 * h + 3]},
                                          reinterpret_cast<tu32x4*>(ar + 4 * h));
          }
        } else {
#pragma unroll
          for (int e = 0; e < CPL; ++e)
            if (col0 + e < M) {
              if (yr) yr[e] = yv[e];
              if (ar) ar[e] = out[e];
            }
        }
      }
    }
  };
  if (ELEM == kF32) run(std::integral_constant<int, 0>{});
  else if (narrow) run(std::integral_constant<int, 1>{});
  else run(std::integral_constant<int, 2>{});
}

// Row-uniform accumulate for int8 tables with at least 512 columns (the same
// sum as tacc_kernel).  A wavefront sums one output row at a time over a
// 512-column slice; lane l owns output columns 4l..4l+3 and 256+4l..256+4l+3
// of the slice, held as eight 16-bit entries in a 16-byte slot of each staged
// table row.  The table row that a codebook selects is then the same for the
// whole wavefront: the row's index bytes come from scalar loads, a lookup is
// a uniform row offset added to the lane's slot plus one 16-byte LDS read,
// no index tile goes through LDS, and every output store instruction writes
// 1 KB of one row.
//
// A work item is RB rows x 512 columns.  The table goes through two LDS
// buffers of 4 codebooks each ([4 x 16 rows][512 entries], 64 KB; one
// 1024-thread workgroup per CU): while a tile is summed from one buffer, every
// wavefront first stages its share of the next tile into the other, from
// registers loaded one tile ahead, so each tile costs one barrier and no
// staging-only phase; the last tile's loads fetch the next work item's first.
//  * When 255 * sum_c 2^(e_c - e_min) <= 65535, an entry is staged as the
//    unsigned u = (q + 128) << (e_c - e_min): no 16-bit field can carry into
//    the next while the codebooks are summed, so one 32-bit add sums two
//    columns and v_add3_u32 adds two codebooks; the int32 sum is the field
//    minus 128 * sum_c 2^(e_c - e_min).  16 rows per wavefront.
//  * Otherwise entries are staged as signed q and summed in int32 with the
//    shifts, 8 rows per wavefront.
constexpr int kRowWaves = 16;           // wavefronts per workgroup
constexpr int kRowCT = 4;               // codebooks per staged tile
constexpr int kRowMt = 512;             // columns per work item
constexpr int kRowBytes = 2 * kRowMt;   // LDS bytes per staged table row
constexpr int kRowTileBytes = kRowCT * 16 * kRowBytes;   // one of two tile buffers (64 KB)
constexpr int kRowJG = 2;               // rows summed between scheduling barriers

__global__ void __launch_bounds__(1024) trow_kernel(const TArgs a, const uint8_t* __restrict__ idx) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  tlds_t* smem = (tlds_t*)smem_raw;
  typedef unsigned short us2 __attribute__((ext_vector_type(2)));

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tuni(tid >> 6);
  const int C = a.C, M = a.M, ntm = a.ntm;
  const int64_t N = a.N;
  tlds_t* s_tab = smem;   // off_tab == 0
  tlds_i32* s_sh = reinterpret_cast<tlds_i32*>(smem + a.off_sh);
  tlds_i32* s_misc = reinterpret_cast<tlds_i32*>(smem + a.off_misc);   // bias32, e_min, sum of 2^sh, max shift

  if (a.only_wide) {
    // the launch after the row-streaming kernel: leave at once unless the
    // 16-bit field sums did not fit (every wavefront decides alone, from the
    // scales: the same test as below)
    const uint32_t* sb0 = reinterpret_cast<const uint32_t*>(a.scale);
    int e = INT_MAX;
    for (int c = lane; c < C; c += 64) e = min(e, (int)((sb0[c] >> 23) & 0xffu) - 127);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) e = min(e, __shfl_xor(e, o));
    int S0 = 0;
    for (int c = lane; c < C; c += 64) {
      const int sh = min((int)((sb0[c] >> 23) & 0xffu) - 127 - e, 30);
      S0 += sh <= 14 ? (1 << sh) : (1 << 15);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) S0 += __shfl_xor(S0, o);
    if (tuni(S0) <= 257) return;   // uniform over the workgroup
  }

  // ---------------- block exponents, shifts and bias32
  if (tid == 0) { s_misc[1] = INT_MAX; s_misc[2] = 0; s_misc[3] = 0; }
  __syncthreads();
  const uint32_t* sb = reinterpret_cast<const uint32_t*>(a.scale);
  for (int c = tid; c < C; c += kRowWaves * 64) atomicMin((int*)&s_misc[1], (int)((sb[c] >> 23) & 0xffu) - 127);
  __syncthreads();
  const int emin = tuni(s_misc[1]);
  for (int c = tid; c < C; c += kRowWaves * 64) {
    const int sh = min((int)((sb[c] >> 23) & 0xffu) - 127 - emin, 30);
    s_sh[c] = sh;
    atomicAdd((int*)&s_misc[2], sh <= 14 ? (1 << sh) : (1 << 15));
    atomicMax((int*)&s_misc[3], sh);
  }
  if (wave == 0) {
    // bias32: double sum over codebooks in ascending order
    double sum = 0.0;
    for (int c0 = 0; c0 < C; c0 += 64) {
      const float ov = a.offset[min(c0 + lane, C - 1)];
      const int n = min(64, C - c0);
      for (int j = 0; j < n; ++j) sum += (double)__int_as_float(__builtin_amdgcn_readlane(__float_as_int(ov), j));
    }
    if (lane == 0) s_misc[0] = __float_as_int((float)sum);
  }
  // column biases of the layer output, staged once (the epilogue of every
  // work item then reads them from LDS instead of waiting on global loads)
  tlds_f32x4* s_bias = reinterpret_cast<tlds_f32x4*>(smem + a.off_bias);
  if (a.bias_lds)   // (col_bias is only 4-byte aligned: one float per load)
    for (int m = tid; m < M; m += kRowWaves * 64) reinterpret_cast<tlds_f32*>(s_bias)[m] = a.col_bias[m];
  __syncthreads();
  const int S = tuni(s_misc[2]);        // sum of 2^sh (saturated per codebook at 2^15)
  const bool fields = S <= 257;         // 255 * S <= 65535
  const bool shifted = tuni(s_misc[3]) != 0;
  const float step = __builtin_ldexpf(1.0f, emin);
  const float bias = __int_as_float(tuni(s_misc[0]));

  // ---------------- staging.  Lane l = 16 a + 4 b + c's 16-byte slot
  // (columns 4l..4l+3 and 256+4l..256+4l+3) sits at position 16 a + 4 b +
  // (c + a) % 4 of each staged row: the 16 lanes of a read pass (fixed a)
  // cover one 256-byte span, and so do the 16 threads of a write pass below
  // (fixed c).  Thread t stages staged row t / 16 of a tile (codebook c0 +
  // t / 256, prototype (t / 16) % 16), the 16 columns 16 (t % 16).. of each
  // half of the slice: two 16-byte loads, the four whole slots of lanes
  // 4 (t % 16) + c.
  const int tp = tid & 15;
  const int tr = tid >> 4;
  const __amdgpu_buffer_rsrc_t trs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.lut), 0, (int)((int64_t)C * 16 * M), kBufDword3);
  tu32x4 tv[2];   // the two halves
  // (the lane bases are re-derived per tile through an empty asm, so the
  // compiler does not keep precomputed addresses in registers)
  auto load_tile = [&](int c0, int m0) {
    int base = (c0 * 16 + tr) * M + m0 + 16 * tp;
    asm volatile("" : "+v"(base));
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const bool ok = m0 + 256 * h + 16 * tp < M;   // M % 16 == 0: units are whole
      tv[h] = __builtin_amdgcn_raw_buffer_load_b128(trs, ok ? base + 256 * h : kOob, 0, 0);
    }
  };
  auto store_tile = [&](int c0, int buf) {
    int base = buf * kRowTileBytes + tr * kRowBytes + tp * 64;   // slot 4 tp + i at position 4 tp + (i + tp / 4) % 4
    asm volatile("" : "+v"(base));
    const unsigned short sh = (fields && shifted) ? (unsigned short)s_sh[c0 + (tr >> 4)] : 0;
    const us2 s2 = {sh, sh};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t w[4];   // quad i of each half, 4 entries each
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint32_t x = tv[h][i];
        uint32_t lo, hi;
        if (fields) {
          const uint32_t u = x ^ 0x80808080u;   // q + 128 per byte
          lo = __builtin_amdgcn_perm(0u, u, 0x0c010c00u);
          hi = __builtin_amdgcn_perm(0u, u, 0x0c030c02u);
          if (shifted) {
            lo = __builtin_bit_cast(uint32_t, __builtin_bit_cast(us2, lo) << s2);
            hi = __builtin_bit_cast(uint32_t, __builtin_bit_cast(us2, hi) << s2);
          }
        } else {
          widen4(x, 0, lo, hi);
        }
        w[2 * h] = lo;
        w[2 * h + 1] = hi;
      }
      *reinterpret_cast<tlds_u32x4*>(s_tab + base + 16 * ((i + (tp >> 2)) & 3)) = (tu32x4){w[0], w[1], w[2], w[3]};
    }
  };

  // the lane's slot of staged row cb * 16 + k of buffer b: (k << 10) + base
  // in one v_lshl_add_u32 with the uniform code in a scalar register
  const uint32_t lane_slot =
      (uint32_t)(uintptr_t)(s_tab + 16 * ((lane & ~3) + (((lane & 3) + (lane >> 4)) & 3)));
  auto run = [&](auto nj_tag) {
    constexpr int NJ = decltype(nj_tag)::value;   // 16: 16-bit fields; 8: int32 sums
    constexpr bool F = NJ == 16;
    constexpr int NA = F ? 4 : 8;
    const int RB = kRowWaves * NJ;
    const int64_t nwork = (int64_t)ntm * ((N + RB - 1) / RB);
    const int T = C / kRowCT;   // tiles per work item (C % 4 == 0)
    if (blockIdx.x < nwork) load_tile(0, (int)(blockIdx.x % ntm) * kRowMt);
    for (int64_t w = blockIdx.x; w < nwork; w += gridDim.x) {
      const int mt = (int)(w % ntm);
      const int64_t r0 = (w / ntm) * RB + (int64_t)wave * NJ;   // this wavefront's first row
      const int m0 = mt * kRowMt;
      const int64_t wn = w + gridDim.x;   // this workgroup's next work item
      // after staging tile s: load tile s + 1, or the next work item's first
      auto load_after = [&](int s) {
        if (s + 1 < T) load_tile((s + 1) * kRowCT, m0);
        else if (wn < nwork) load_tile(0, (int)(wn % ntm) * kRowMt);
      };
      uint32_t acc[NJ][NA];
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int e = 0; e < NA; ++e) acc[j][e] = 0u;

      // buffer 0 is free: the previous work item ended with a barrier
      store_tile(0, 0);
      load_after(0);
      __syncthreads();
      for (int t = 0; t < T; ++t) {
        // tile t is in buffer t % 2; stage tile t + 1 into the other one
        // (its readers, tile t - 1, finished before the last barrier)
        if (t + 1 < T) {
          store_tile((t + 1) * kRowCT, (t + 1) & 1);
          load_after(t + 1);   // in flight during the sums below
        }
        const int c0 = t * kRowCT;
        uint32_t d[NJ];   // index bytes of codebooks c0..c0+3 (uniform)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
          d[j] = *reinterpret_cast<const uint32_t*>(idx + min(r0 + j, N - 1) * a.idx_stride + c0);   // rows past N: any valid row
        const uint32_t lane_buf = lane_slot + (t & 1) * kRowTileBytes;
        auto slot_of = [&](int cb, int k) -> const tlds_t* {
          uint32_t adr;
          asm("v_lshl_add_u32 %0, %1, 10, %2" : "=v"(adr) : "s"(k), "v"(lane_buf));
          return (const tlds_t*)(uintptr_t)adr + cb * 16 * kRowBytes;
        };
        if (F) {
          // items i = (codebook pair cp = 2 (i / NJ), row j = i % NJ), software
          // pipelined: the two reads of item i + 1 are issued before item i is
          // summed, so each wavefront keeps reads in flight during its sums
          constexpr int NI = (kRowCT / 2) * NJ;
          tu32x4 v0[2], v1[2];
          auto rd = [&](int i, tu32x4& x0, tu32x4& x1) {
            const int cp = 2 * (i / NJ);
            const uint32_t dw = d[i % NJ];
            x0 = *reinterpret_cast<const tlds_u32x4*>(slot_of(cp, (dw >> (8 * cp)) & 15));
            x1 = *reinterpret_cast<const tlds_u32x4*>(slot_of(cp + 1, (dw >> (8 * cp + 8)) & 15));
          };
          __builtin_amdgcn_sched_barrier(0);   // every index load issued before the first table read
          rd(0, v0[0], v1[0]);
#pragma unroll
          for (int i = 0; i < NI; ++i) {
            __builtin_amdgcn_sched_barrier(0);
            if (i + 1 < NI) rd(i + 1, v0[(i + 1) & 1], v1[(i + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
            const int j = i % NJ;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              acc[j][e] += v0[i & 1][e] + v1[i & 1][e];
              asm("" : "+v"(acc[j][e]));   // opaque: no reassociation across codebook pairs
            }
          }
        } else {
#pragma unroll
          for (int cc = 0; cc < kRowCT; ++cc) {
            const int sh = tuni(s_sh[c0 + cc]);
#pragma unroll
            for (int g = 0; g < NJ; g += kRowJG) {
              tu32x4 v[kRowJG];
              __builtin_amdgcn_sched_barrier(0);
#pragma unroll
              for (int jj = 0; jj < kRowJG; ++jj)
                v[jj] = *reinterpret_cast<const tlds_u32x4*>(slot_of(cc, (d[g + jj] >> (8 * cc)) & 15));
              __builtin_amdgcn_sched_barrier(0);
#pragma unroll
              for (int jj = 0; jj < kRowJG; ++jj)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                  acc[g + jj][2 * e] += (uint32_t)(__builtin_amdgcn_sbfe((int)v[jj][e], 0, 16) << sh);
                  acc[g + jj][2 * e + 1] += (uint32_t)(((int)v[jj][e] >> 16) << sh);
                  asm("" : "+v"(acc[g + jj][2 * e]), "+v"(acc[g + jj][2 * e + 1]));
                }
            }
          }
        }
        __syncthreads();   // tile t + 1 visible; every reader of buffer t % 2 done
      }

      // ---------------- epilogue: outputs i < 4 are columns colA + i, the rest colB + i - 4
      const int colA = m0 + 4 * lane, colB = colA + 256;
      float cb[8];   // this lane's column biases, once per work item (stores to y may alias the global row)
      if (a.bias_lds) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {   // M % 16 == 0: a quad is in range as a whole
          const int col = h ? colB : colA;
          const tf32x4 b4 = col < M ? s_bias[col >> 2] : (tf32x4){0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int e = 0; e < 4; ++e) cb[4 * h + e] = b4[e];
        }
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int col = (i < 4 ? colA : colB - 4) + i;
          cb[i] = (a.act != 0 && a.col_bias && col < M) ? a.col_bias[col] : 0.0f;
        }
      }
      const int off128 = F ? 128 * S : 0;   // S <= 257 in field mode
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int64_t row = r0 + j;
        int out[8];
        float yv[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (F) {
            out[2 * e] = (int)(acc[j][e] & 0xffffu) - off128;
            out[2 * e + 1] = (int)(acc[j][e] >> 16) - off128;
          } else {
            out[2 * e] = (int)acc[j][2 * e];
            out[2 * e + 1] = (int)acc[j][2 * e + 1];
          }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) yv[i] = __builtin_fmaf((float)out[i], step, bias);
        if (a.act != 0) {
          // layer output sigma: z = y + bias, then ReLU, or a softmax over the
          // row (one column tile: the whole row is in this wavefront)
          float vmax = -__builtin_inff();
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const bool ok = (i < 4 ? colA : colB - 4) + i < M;
            float z = yv[i] + cb[i];
            if (a.act == 2) z = (z > 0.0f) ? z : 0.0f;
            yv[i] = z;
            if (ok) vmax = __builtin_fmaxf(vmax, z);
          }
          if (a.act == 3) {
            vmax = wave_reduce64<true>(vmax);
            float sum = 0.0f;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              yv[i] = ((i < 4 ? colA : colB - 4) + i < M) ? expf(yv[i] - vmax) : 0.0f;
              sum += yv[i];
            }
            const float rs = 1.0f / wave_reduce64<false>(sum);   // correctly rounded reciprocal, then products
#pragma unroll
            for (int i = 0; i < 8; ++i) yv[i] = yv[i] * rs;
          }
        }
        if (row >= N) continue;   // uniform: one row per wavefront
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int col = h ? colB : colA;
          if (col >= M) continue;
          if (a.y)
            __builtin_nontemporal_store((tf32x4){yv[4 * h], yv[4 * h + 1], yv[4 * h + 2], yv[4 * h + 3]},
                                        reinterpret_cast<tf32x4*>(a.y + row * M + col));
          if (a.acc)
            __builtin_nontemporal_store((tu32x4){(uint32_t)out[4 * h], (uint32_t)out[4 * h + 1],
                                                 (uint32_t)out[4 * h + 2], (uint32_t)out[4 * h + 3]},
                                        reinterpret_cast<tu32x4*>(a.acc + row * M + col));
        }
      }
    }
  };
  if (fields) run(std::integral_constant<int, 16>{});
  else run(std::integral_constant<int, 8>{});
}

// fp32 tables: the same row-uniform scheme with four fp32 columns per lane.
// A work item is 256 rows x 256 columns; lane l owns columns 4l..4l+3 in their
// own order, so lane slot l of a staged row is the row's 16-byte unit l: each
// staged row arrives by one direct-to-LDS buffer load per wavefront (64 lanes x
// 16 bytes into consecutive LDS), with no registers or LDS writes on the way,
// and each output store instruction writes 1 KB of one row.  Each lane adds
// the selected entries to its sums codebook by codebook, strictly ascending
// from +0.0f, so the sums are the ordered fp32 sums of tacc_kernel.  Tiles of
// 4 codebooks alternate between the two 64 KB buffers over the workgroup's
// whole sequence of tiles: the loads of the next tile (the next work item's
// first after a work item's last) are in flight while a tile is summed, and
// each tile costs one wait and one barrier.
constexpr int kRowMtF = 256;   // columns per work item (fp32 tables)

__global__ void __launch_bounds__(1024) trow_f32_kernel(const TArgs a, const uint8_t* __restrict__ idx) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  tlds_t* s_tab = (tlds_t*)smem_raw;   // two tile buffers of kRowTileBytes
  constexpr int NJ = 16;               // rows per wavefront
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tuni(tid >> 6);
  const int C = a.C, M = a.M, ntm = a.ntm;
  const int64_t N = a.N;

  const __amdgpu_buffer_rsrc_t trs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.lut), 0, (int)((int64_t)C * 16 * M * 4), kBufDword3);
  // stage tile c0 of column tile m0 into buffer buf: wavefront w loads staged
  // rows 4w..4w+3 (codebook c0 + w / 4, prototypes 4 (w % 4)..); columns past
  // M read as zeros
  auto stage = [&](int c0, int m0, int buf) {
    const bool ok = m0 + 4 * lane < M;   // M % 4 == 0: units are whole
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 4 * wave + i;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          trs, (__attribute__((address_space(3))) void*)(s_tab + buf * kRowTileBytes + r * kRowBytes), 16,
          ok ? ((c0 * 16 + r) * M + m0 + 4 * lane) * 4 : kOob, 0, 0, 0);
    }
  };
  auto publish = [&]() {   // this wavefront's staged rows are in LDS, then the barrier
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  };

  const uint32_t lane_slot = (uint32_t)(uintptr_t)(s_tab + lane * 16);
  const int RB = kRowWaves * NJ;
  const int64_t nwork = (int64_t)ntm * ((N + RB - 1) / RB);
  const int T = C / 4;   // tiles per work item (C % 4 == 0)
  int gb = 0;            // buffer of the current tile (alternates over the whole sequence)
  // column biases of the layer output, staged once (visible after the first barrier)
  tlds_f32x4* s_bias = reinterpret_cast<tlds_f32x4*>(s_tab + a.off_bias);
  if (a.bias_lds)   // (col_bias is only 4-byte aligned: one float per load)
    for (int m = tid; m < M; m += kRowWaves * 64) reinterpret_cast<tlds_f32*>(s_bias)[m] = a.col_bias[m];
  if (blockIdx.x < nwork) {
    stage(0, (int)(blockIdx.x % ntm) * kRowMtF, 0);
    publish();
  }
  for (int64_t w = blockIdx.x; w < nwork; w += gridDim.x) {
    const int mt = (int)(w % ntm);
    const int64_t r0 = (w / ntm) * RB + (int64_t)wave * NJ;   // this wavefront's first row
    const int m0 = mt * kRowMtF;
    const int64_t wn = w + gridDim.x;
    float acc[NJ][4];
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[j][e] = 0.0f;

    for (int t = 0; t < T; ++t) {
      // the other buffer's readers (the previous tile) finished before the last barrier
      if (t + 1 < T) stage((t + 1) * 4, m0, gb ^ 1);
      else if (wn < nwork) stage(0, (int)(wn % ntm) * kRowMtF, gb ^ 1);
      const int c0 = t * 4;
      uint32_t d[NJ];   // index bytes of codebooks c0..c0+3 (uniform)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        d[j] = *reinterpret_cast<const uint32_t*>(idx + min(r0 + j, N - 1) * a.idx_stride + c0);   // rows past N: any valid row
      const uint32_t lane_buf = lane_slot + gb * kRowTileBytes;
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
#pragma unroll
        for (int g = 0; g < NJ; g += kRowJG) {
          tu32x4 v[kRowJG];
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int jj = 0; jj < kRowJG; ++jj) {
            uint32_t adr;
            asm("v_lshl_add_u32 %0, %1, 10, %2" : "=v"(adr) : "s"((d[g + jj] >> (8 * cb)) & 15), "v"(lane_buf));
            v[jj] = *reinterpret_cast<const tlds_u32x4*>((const tlds_t*)(uintptr_t)adr + cb * 16 * kRowBytes);
          }
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int jj = 0; jj < kRowJG; ++jj)
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[g + jj][e] += __uint_as_float(v[jj][e]);   // codebooks ascending
        }
      }
      publish();   // the next tile visible; every reader of this buffer done
      gb ^= 1;
    }

    // ---------------- epilogue: this lane's columns col..col+3
    const int col = m0 + 4 * lane;
    float cb[4];   // column biases, once per work item (stores to y may alias the global row)
    if (a.bias_lds) {   // M % 4 == 0: a quad is in range as a whole
      const tf32x4 b4 = col < M ? s_bias[col >> 2] : (tf32x4){0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int e = 0; e < 4; ++e) cb[e] = b4[e];
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) cb[e] = (a.act != 0 && a.col_bias && col + e < M) ? a.col_bias[col + e] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int64_t row = r0 + j;
      float yv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) yv[e] = acc[j][e];
      if (a.act != 0) {
        float vmax = -__builtin_inff();
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float z = yv[e] + cb[e];
          if (a.act == 2) z = (z > 0.0f) ? z : 0.0f;
          yv[e] = z;
          if (col + e < M) vmax = __builtin_fmaxf(vmax, z);
        }
        if (a.act == 3) {   // one column tile: the whole row is in this wavefront
          vmax = wave_reduce64<true>(vmax);
          float sum = 0.0f;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            yv[e] = (col + e < M) ? expf(yv[e] - vmax) : 0.0f;
            sum += yv[e];
          }
          const float rs = 1.0f / wave_reduce64<false>(sum);   // correctly rounded reciprocal, then products
#pragma unroll
          for (int e = 0; e < 4; ++e) yv[e] = yv[e] * rs;
        }
      }
      if (row >= N || col >= M) continue;   // row: uniform; col: whole quads (M % 4 == 0)
      __builtin_nontemporal_store((tf32x4){yv[0], yv[1], yv[2], yv[3]}, reinterpret_cast<tf32x4*>(a.y + row * M + col));
    }
  }
}

// Rounded 8-bit summation over codebooks (§1 names it; reading R20): the
// codes of a row, biased to bytes u = q + 128 and padded with 128 to P = 2^L
// codebooks, are reduced by a balanced tree of rounded byte averages in
// codebook order, four columns per v_lerp_u8; the root r gives
// acc = P (r - 128).
//
// One byte per staged entry lets a workgroup hold the table's whole column
// slice, [C * 16 rows][Mt columns] (at most 128 KB), staged once: a workgroup
// keeps one column tile for its lifetime and its wavefronts then stream row
// sets.  16 columns per lane, LPR = Mt / 16 lanes per output row.  Index rows
// come in batches of B rows staged in LDS, the next batch loaded into
// registers while the current one is summed (one barrier pair per batch).
// Codebooks are taken 8 at a time: one level-3 subtree (or the level-L root
// when P < 8), merged into a binary-counter stack of higher tree levels held
// in registers; subtrees of pure padding (all 128) finish the tree when C is
// not a power of two.
__device__ __forceinline__ uint32_t avg4(uint32_t a, uint32_t b) { return __builtin_amdgcn_lerp(a, b, 0x01010101u); }


// The padded tree has GA = P / 8 subtrees of 8 codebooks (at least 1), taken
// GI at a time (unrolled, their merges resolved at compile time) in GO = GA /
// GI rounds of a runtime loop whose results (subtrees of 8 GI codebooks) merge
// through up to three pending levels.  The unrolled subtrees bound the LDS
// reads in flight, and with them the registers: GI = 4 within the 256 VGPRs
// of a 512-thread workgroup.
// WIDX: C % 4 == 0, index words read as dwords (else byte by byte).
template <int GI, int GO, bool WIDX, int NT>
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(NT / 256, NT / 256)))
tavg_kernel(const TArgs a) {
  static_assert(GI == 1 || GI == 2 || GI == 4, "inner subtrees");
  static_assert(GO == 1 || GO == 2 || GO == 4 || GO == 8, "outer rounds");
  constexpr int kLev = (GI >= 4) ? 2 : (GI >= 2) ? 1 : 0;
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  tlds_t* smem = (tlds_t*)smem_raw;

  const int tid = threadIdx.x;
  const int nt = blockDim.x;
  const int lane = tid & 63;
  const int wave = tuni(tid >> 6);
  const int nw = nt >> 6;
  const int C = a.C, M = a.M, Mt = a.Mt;
  const int C8 = (C + 7) & ~7;            // codebooks staged: whole groups of 8, padding rows all 128
  const int64_t N = a.N;
  const int lpr_log2 = a.lpr_log2;
  const int RS = 64 >> lpr_log2;          // output rows per wavefront pass
  const int r4 = lane >> lpr_log2;
  const int cg = lane & ((1 << lpr_log2) - 1);
  const int rby_log2 = 31 - __builtin_clz(Mt);   // one byte per entry: row bytes = Mt
  tlds_t* s_tab = smem;   // [C8 * 16 + 16][Mt] biased codes, then a 16-row block of 128 (off_tab == 0)
  tlds_i32* s_misc = reinterpret_cast<tlds_i32*>(smem + a.off_misc);

  // block exponent (one shared by every codebook) and bias32
  if (tid == 0) s_misc[1] = INT_MAX;
  __syncthreads();
  const uint32_t* sb = reinterpret_cast<const uint32_t*>(a.scale);
  for (int c = tid; c < C; c += nt) atomicMin((int*)&s_misc[1], (int)((sb[c] >> 23) & 0xffu) - 127);
  if (wave == 0) {
    double sum = 0.0;
    for (int c0 = 0; c0 < C; c0 += 64) {
      const float ov = a.offset[min(c0 + lane, C - 1)];
      const int n = min(64, C - c0);
      for (int j = 0; j < n; ++j) sum += (double)__int_as_float(__builtin_amdgcn_readlane(__float_as_int(ov), j));
    }
    if (lane == 0) s_misc[0] = __float_as_int((float)sum);
  }

  // column tile of this workgroup: stage every codebook's [16][Mt] slice.
  // Columns are permuted within a tile row so that the 16 bytes a lane reads
  // are the 4-column groups d = cg, cg + LPR, cg + 2 LPR, cg + 3 LPR: each
  // output store of the wavefront then writes LPR x 16 contiguous bytes of a
  // row (whole cache lines) instead of 16-byte pieces 64 bytes apart.
  const int lpr = 1 << lpr_log2;
  auto lds_dword = [&](int d) { return ((d & (lpr - 1)) << 2) + (d >> lpr_log2); };
  const int mt = blockIdx.x % a.ntm;
  const int m0 = mt * Mt;
  {
    const int rows = C8 * 16 + 16;   // the last 16 rows: padding subtrees read them (all 128)
    if (a.vec_lut) {
      const __amdgpu_buffer_rsrc_t trs =
          __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.lut), 0, (int)((int64_t)C * 16 * M), kBufDword3);
      const int upr_log2 = rby_log2 - 4;   // 16-byte units per tile row
      const int units = rows << upr_log2;
      for (int u0 = tid; u0 < units; u0 += 4 * nt) {
        tu32x4 v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {   // all loads of the round first; rows past C * 16 read zero
          const int u = u0 + j * nt;
          const int row = u >> upr_log2, part = u & ((1 << upr_log2) - 1);
          const bool ok = u < units && row < C * 16 && m0 + part * 16 < M;
          v[j] = __builtin_amdgcn_raw_buffer_load_b128(trs, ok ? row * M + m0 + part * 16 : kOob, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int u = u0 + j * nt;
          if (u < units) {
            const int row = u >> upr_log2, part = u & ((1 << upr_log2) - 1);
            tlds_u32* dst = reinterpret_cast<tlds_u32*>(s_tab + (row << rby_log2));
#pragma unroll
            for (int i = 0; i < 4; ++i) dst[lds_dword(4 * part + i)] = v[j][i] ^ 0x80808080u;   // q + 128
          }
        }
      }
    } else {
      const uint8_t* q8 = reinterpret_cast<const uint8_t*>(a.lut);
      for (int e = tid; e < (rows << rby_log2); e += nt) {
        const int row = e >> rby_log2, col = e & (Mt - 1);
        const int m = m0 + col;
        s_tab[(row << rby_log2) + 4 * lds_dword(col >> 2) + (col & 3)] =
            (char)((row < C * 16 && m < M) ? (q8[(int64_t)row * M + m] ^ 0x80u) : 0x80u);
      }
    }
  }
  __syncthreads();
  const float step = __builtin_ldexpf(1.0f, tuni(s_misc[1]));
  const float bias = __int_as_float(tuni(s_misc[0]));
  int L = 0;
  while ((1 << L) < C) ++L;
  const int P = 1 << L;
  const int ngroup = C8 >> 3;   // subtrees holding real codes; the rest of the GA are pure padding
  const int col0 = m0 + cg * 4;   // the lane's columns: col0 + 4 lpr h + e, h, e < 4
  const tlds_t* s_tab_lane = s_tab + cg * 16;

  // index batches of B = nw * RS * J rows (C bytes each, contiguous in
  // memory), shared out over the workgroups of this column tile
  tlds_t* s_idx = smem + a.off_idx;
  const int J = a.RB / (nw * RS);
  const int B = a.RB;
  const int64_t nbatch = (N + B - 1) / B;
  const int64_t bstride = gridDim.x / a.ntm;
  const int bunits = (B * C) >> 4;   // 16-byte units per batch (B * C % 16 == 0)
  tu32x4 ipf[2];
  auto load_batch = [&](int64_t bi) {
    const int64_t r0 = bi * B;
    const int64_t bytes = bi < nbatch ? min((int64_t)B, N - r0) * C : 0;
    const __amdgpu_buffer_rsrc_t irs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(a.idx + min(r0, N - 1) * C), 0, (int)min(bytes, (int64_t)INT_MAX), kBufDword3);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int u = tid + j * nt;
      if (u < bunits && 16 * u + 16 > bytes && 16 * u < bytes) {
        // the unit holding the end of the index array: bytes one by one (the
        // range check is per dword, and reading past the array is not allowed)
        tu32x4 w = {0u, 0u, 0u, 0u};
        for (int b = 0; b < 16; ++b)
          w[b >> 2] |= (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(irs, 16 * u + b, 0, 0) << (8 * (b & 3));
        ipf[j] = w;
      } else {
        ipf[j] = __builtin_amdgcn_raw_buffer_load_b128(irs, u < bunits ? 16 * u : kOob, 0, 0);
      }
    }
  };
  int64_t bi = blockIdx.x / a.ntm;
  load_batch(bi);
  for (; bi < nbatch; bi += bstride) {
    __syncthreads();   // every reader of the previous batch is done
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int u = tid + j * nt;
      if (u < bunits) *reinterpret_cast<tlds_u32x4*>(s_idx + 16 * u) = ipf[j];
    }
    __syncthreads();
    load_batch(bi + bstride);   // in flight during the sums below
    for (int jj = 0; jj < J; ++jj) {
    const int ii = (jj * nw + wave) * RS + r4;   // row within the batch
    const int64_t row = bi * B + ii;
    const tlds_t* ir = s_idx + ii * C;
    tu32x4 root, pend0, pend1, pend2;   // pend<l>: a finished round at outer level l
#pragma unroll 1
    for (int h = 0; h < GO; ++h) {
      tu32x4 stk[kLev + 1];   // stk[l]: a pending node 3 + l levels above the leaves
      tu32x4 sub;
#pragma unroll
      for (int gi = 0; gi < GI; ++gi) {
        const int g = h * GI + gi;   // subtree index
        tu32x4 x;
        // indices of codebooks 8g .. 8g + 7 (bytes past the row's C, at most 7,
        // belong to padding codebooks, whose rows are all 128: any k); a
        // subtree of pure padding reads group 0's bytes and masks them
        const tlds_t* ig = ir + 8 * (g < ngroup ? g : 0);
        uint32_t w0, w1;
        if (WIDX) {
          w0 = *reinterpret_cast<const tlds_u32*>(ig);
          w1 = *reinterpret_cast<const tlds_u32*>(ig + 4);
        } else {
          w0 = w1 = 0u;
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            w0 |= (uint32_t)(uint8_t)ig[b] << (8 * b);
            w1 |= (uint32_t)(uint8_t)ig[4 + b] << (8 * b);
          }
        }
        // a subtree of pure padding reads the all-128 block for its 8 leaves
        const uint32_t rbase = g < ngroup ? (uint32_t)(128 * g) : (uint32_t)(C8 * 16);
        const uint32_t kmask = g < ngroup ? 15u : 0u;
        tu32x4 v[8];
#pragma unroll
        for (int b = 0; b < 8; ++b) {
          const uint32_t k = ((b < 4 ? w0 : w1) >> (8 * (b & 3))) & kmask;
          const uint32_t r = g < ngroup ? rbase + 16 * b + k : rbase;
          v[b] = *reinterpret_cast<const tlds_u32x4*>(s_tab_lane + (r << rby_log2));
        }
        tu32x4 a0, a1, a2, a3, b0, b1;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          a0[e] = avg4(v[0][e], v[1][e]);
          a1[e] = avg4(v[2][e], v[3][e]);
          a2[e] = avg4(v[4][e], v[5][e]);
          a3[e] = avg4(v[6][e], v[7][e]);
          b0[e] = avg4(a0[e], a1[e]);
          b1[e] = avg4(a2[e], a3[e]);
          x[e] = avg4(b0[e], b1[e]);
        }
        if (GI == 1 && GO == 1) root = (L == 0) ? v[0] : (L == 1) ? a0 : (L == 2) ? b0 : x;
        if (GI == 1) sub = x;
        else {
          // binary counter over gi (compile-time): merge while the low bits of gi are 1
          int l = 0;
#pragma unroll
          for (; l < kLev && ((gi >> l) & 1); ++l)
#pragma unroll
            for (int e = 0; e < 4; ++e) x[e] = avg4(stk[l][e], x[e]);
          stk[l] = x;
        }
      }
      if (GI > 1) sub = stk[kLev];
      if (GO > 1) {
        // binary counter over h (uniform branches): merge while the low bits
        // of h are 1, then wait at the first level whose bit is 0; the last
        // round (h = GO - 1, all bits 1) finishes the tree
        if (h & 1) {
#pragma unroll
          for (int e = 0; e < 4; ++e) sub[e] = avg4(pend0[e], sub[e]);
          if (h & 2) {
#pragma unroll
            for (int e = 0; e < 4; ++e) sub[e] = avg4(pend1[e], sub[e]);
            if (h & 4) {
#pragma unroll
              for (int e = 0; e < 4; ++e) sub[e] = avg4(pend2[e], sub[e]);
            } else {
              pend2 = sub;
            }
          } else {
            pend1 = sub;
          }
        } else {
          pend0 = sub;
        }
      }
      if (!(GI == 1 && GO == 1)) root = sub;
    }

    // epilogue: acc = P (r - 128) for the lane's 16 columns
    if (row >= N || col0 >= M) continue;
    int out[16];   // out[4 h + e]: column col0 + 4 lpr h + e
#pragma unroll
    for (int e = 0; e < 16; ++e) out[e] = P * ((int)((root[e >> 2] >> (8 * (e & 3))) & 0xffu) - 128);
    float* yr = a.y ? a.y + row * M + col0 : nullptr;
    int32_t* ar = a.acc ? a.acc + row * M + col0 : nullptr;
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const int ch = col0 + 4 * lpr * h;
      if (a.vec_out && ch + 4 <= M) {
        if (yr)
          __builtin_nontemporal_store((tf32x4){__builtin_fmaf((float)out[4 * h], step, bias),
                                               __builtin_fmaf((float)out[4 * h + 1], step, bias),
                                               __builtin_fmaf((float)out[4 * h + 2], step, bias),
                                               __builtin_fmaf((float)out[4 * h + 3], step, bias)},
                                      reinterpret_cast<tf32x4*>(yr + 4 * lpr * h));
        if (ar)
          __builtin_nontemporal_store((tu32x4){(uint32_t)out[4 * h], (uint32_t)out[4 * h + 1],
                                               (uint32_t)out[4 * h + 2], (uint32_t)out[4 * h + 3]},
                                      reinterpret_cast<tu32x4*>(ar + 4 * lpr * h));
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (ch + e < M) {
            if (yr) yr[4 * lpr * h + e] = __builtin_fmaf((float)out[4 * h + e], step, bias);
            if (ar) ar[4 * lpr * h + e] = out[4 * h + e];
          }
      }
    }
    }
  }
}


template <int ELEM, int NJ>
static hipError_t tlaunch(const TArgs& t, int nw, int cus, hipStream_t stream) {
  const void* fn = reinterpret_cast<const void*>(&tacc_kernel<ELEM, NJ>);
  hipError_t err = hipSuccess;
  const int per_cu = launch_prepare(fn, nw * 64, t.lds_total, &err);
  if (err != hipSuccess) return err;
  int64_t blocks = t.nwork;
  const int64_t resident = (int64_t)per_cu * cus;
  if (blocks > resident) blocks = resident;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL((tacc_kernel<ELEM, NJ>), dim3((unsigned)blocks), dim3(nw * 64), t.lds_total, stream, t);
  return hipGetLastError();
}

// Row softmax in place, one wavefront per row (rows whose outputs span several
// column tiles of the accumulate): the row is read once into registers (up to
// 64 values per lane, 4-column chunks when M % 4 == 0), max and sum are
// reduced across the wavefront, and the row is written once.
constexpr int kSoftChunks = 16;   // 4-column chunks per lane: M <= 4096

__global__ void __launch_bounds__(256) softmax_rows_kernel(float* y, int64_t N, int M) {
  const int lane = threadIdx.x & 63;
  const int64_t nw_total = (int64_t)gridDim.x * (blockDim.x >> 6);
  const int nq = M >> 2;   // whole 4-column chunks (M % 4 == 0 and M <= 4096 on this path)
  for (int64_t row = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); row < N; row += nw_total) {
    tf32x4* yr = reinterpret_cast<tf32x4*>(y + row * M);
    tf32x4 v[kSoftChunks];
    float vmax = -__builtin_inff();
#pragma unroll
    for (int i = 0; i < kSoftChunks; ++i) {
      const int q = lane + 64 * i;
      v[i] = q < nq ? __builtin_nontemporal_load(yr + q) : (tf32x4){-__builtin_inff(), -__builtin_inff(), -__builtin_inff(), -__builtin_inff()};
      vmax = __builtin_fmaxf(vmax, __builtin_fmaxf(__builtin_fmaxf(v[i].x, v[i].y), __builtin_fmaxf(v[i].z, v[i].w)));
    }
    vmax = wave_reduce64<true>(vmax);
    float sum = 0.0f;
#pragma unroll
    for (int i = 0; i < kSoftChunks; ++i) {
      if (lane + 64 * i < nq) {
        v[i].x = expf(v[i].x - vmax); v[i].y = expf(v[i].y - vmax);
        v[i].z = expf(v[i].z - vmax); v[i].w = expf(v[i].w - vmax);
        sum += (v[i].x + v[i].y) + (v[i].z + v[i].w);
      }
    }
    const float rs = 1.0f / wave_reduce64<false>(sum);   // correctly rounded reciprocal, then products
#pragma unroll
    for (int i = 0; i < kSoftChunks; ++i) {
      const int q = lane + 64 * i;
      if (q < nq) __builtin_nontemporal_store((tf32x4){v[i].x * rs, v[i].y * rs, v[i].z * rs, v[i].w * rs}, yr + q);
    }
  }
}

// General rows (any M): three strided passes over the row.
__global__ void __launch_bounds__(256) softmax_rows_any_kernel(float* y, int64_t N, int M) {
  const int lane = threadIdx.x & 63;
  const int64_t nw_total = (int64_t)gridDim.x * (blockDim.x >> 6);
  for (int64_t row = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); row < N; row += nw_total) {
    float* yr = y + row * M;
    float vmax = -__builtin_inff();
    for (int m = lane; m < M; m += 64) vmax = __builtin_fmaxf(vmax, yr[m]);
    for (int o = 1; o < 64; o <<= 1) vmax = __builtin_fmaxf(vmax, __shfl_xor(vmax, o));
    float sum = 0.0f;
    for (int m = lane; m < M; m += 64) sum += expf(yr[m] - vmax);
    for (int o = 1; o < 64; o <<= 1) sum += __shfl_xor(sum, o);
    for (int m = lane; m < M; m += 64) yr[m] = expf(yr[m] - vmax) / sum;
  }
}

hipError_t launch_softmax_rows(float* y, int64_t N, int M, int cus, hipStream_t stream) {
  int64_t blocks = (N + 3) / 4;
  if (blocks > (int64_t)cus * 32) blocks = (int64_t)cus * 32;
  if (blocks < 1) blocks = 1;
  const bool vec = (M % 4 == 0) && (M <= 4 * 64 * kSoftChunks) && ((reinterpret_cast<uintptr_t>(y) & 15) == 0);
  if (vec)
    hipLaunchKernelGGL(softmax_rows_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, y, N, M);
  else
    hipLaunchKernelGGL(softmax_rows_any_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, y, N, M);
  return hipGetLastError();
}

template <int GI, int GO, bool WIDX, int NT>
static hipError_t alaunch(const TArgs& t, int cus, hipStream_t stream) {
  const void* fn = reinterpret_cast<const void*>(&tavg_kernel<GI, GO, WIDX, NT>);
  hipError_t err = hipSuccess;
  const int per_cu = launch_prepare(fn, NT, t.lds_total, &err);
  if (err != hipSuccess) return err;
  // every workgroup keeps one column tile: a whole number of workgroups per tile
  int64_t per_tile = ((int64_t)per_cu * cus) / t.ntm;
  const int64_t batches = (t.N + t.RB - 1) / t.RB;
  if (per_tile > batches) per_tile = batches;
  if (per_tile < 1) per_tile = 1;
  hipLaunchKernelGGL((tavg_kernel<GI, GO, WIDX, NT>), dim3((unsigned)(per_tile * t.ntm)), dim3(NT),
                     t.lds_total, stream, t);
  return hipGetLastError();
}

// GA = P / 8 subtrees (at least 1) split into GI unrolled x GO rounds
template <int GA, int NT>
static hipError_t alaunch_g(const TArgs& t, int cus, hipStream_t stream) {
  constexpr int kGI = GA < 4 ? GA : 4;
  constexpr int kGO = GA / kGI;
  if (t.C % 4 == 0) return alaunch<kGI, kGO, true, NT>(t, cus, stream);
  return alaunch<kGI, kGO, false, NT>(t, cus, stream);
}

template <int NT>
static hipError_t launch_tavg_nt(const TArgs& t, int cus, hipStream_t stream) {
  int P = 1;
  while (P < t.C) P *= 2;
  switch (P <= 8 ? 1 : P / 8) {
    case 1: return alaunch_g<1, NT>(t, cus, stream);
    case 2: return alaunch_g<2, NT>(t, cus, stream);
    case 4: return alaunch_g<4, NT>(t, cus, stream);
    case 8: return alaunch_g<8, NT>(t, cus, stream);
    case 16: return alaunch_g<16, NT>(t, cus, stream);
    default: return hipErrorInvalidValue;   // C <= 128 (the planner checks)
  }
}

hipError_t launch_tavg(const TArgs& t, int nw, int cus, hipStream_t stream) {
  if (nw == 8) return launch_tavg_nt<512>(t, cus, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_trow(int elem, const TArgs& t, int cus, hipStream_t stream) {
  const void* fn = elem == kF32 ? reinterpret_cast<const void*>(&trow_f32_kernel)
                                : reinterpret_cast<const void*>(&trow_kernel);
  hipError_t err = hipSuccess;
  const int per_cu = launch_prepare(fn, kRowWaves * 64, t.lds_total, &err);
  if (err != hipSuccess) return err;
  int64_t blocks = t.nwork;   // work items at 16 rows per wavefront (the kernel recounts for 8)
  const int64_t resident = (int64_t)per_cu * cus;
  if (blocks > resident) blocks = resident;
  if (blocks < 1) blocks = 1;
  if (elem == kF32)
    hipLaunchKernelGGL(trow_f32_kernel, dim3((unsigned)blocks), dim3(kRowWaves * 64), t.lds_total, stream, t, t.idx);
  else
    hipLaunchKernelGGL(trow_kernel, dim3((unsigned)blocks), dim3(kRowWaves * 64), t.lds_total, stream, t, t.idx);
  return hipGetLastError();
}

hipError_t launch_tacc(int elem, int nj, const TArgs& t, int nw, int cus, hipStream_t stream) {
  if (elem == kI8 && nj == 4) return tlaunch<kI8, 4>(t, nw, cus, stream);
  if (elem == kF32 && nj == 4) return tlaunch<kF32, 4>(t, nw, cus, stream);
  return hipErrorInvalidValue;
}

}  // namespace mdn
