// Column-tiled lookup-accumulate (§1 of McCarter & Dronen: the product is the
// sum over codebooks of the table rows the encoder selected) for tables larger
// than LDS and for the accumulate-only entry points.
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
//    (127 * sum_c 2^(e_c - e_min) <= 32767) are staged as int16 q << (e_c -
//    e_min) and summed with packed 16-bit adds: modular arithmetic whose exact
//    total fits, so the sum equals the int32 sum;
//  * other int8 tables are staged as int16 q and summed in int32 with shifts;
//  * fp32 tables are summed with ordered fp32 adds.
// The last codebook tile is padded to a multiple of 4 codebooks with all-zero
// table rows.
#include "internal.hpp"

#include <climits>
#include <mutex>
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

constexpr int kBufDword3 = 0x00020000;   // raw, unswizzled buffer descriptor (gfx9 family)
constexpr int kTU = 4;                   // 16-byte table units per thread per tile (vector staging)
constexpr int kIU = 2;                   // 4-byte index words per thread per tile (vector staging)
constexpr int kOob = INT_MAX;            // buffer offset past any descriptor range: reads zero

__device__ __forceinline__ int tuni(int v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ uint32_t tpk_add16(uint32_t a, uint32_t b) {
  typedef short s2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, (s2)(__builtin_bit_cast(s2, a) + __builtin_bit_cast(s2, b)));
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
    narrow = 127 * tuni(s_misc[2]) <= 32767;
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

// Rounded 8-bit summation over codebooks (§1 names it; reading R20): the
// codes of a row, biased to bytes u = q + 128 and padded with 128 to P = 2^L
// codebooks, are reduced by a balanced tree of rounded byte averages in
// codebook order, four columns per v_lerp_u8; the root r gives
// acc = P (r - 128).  Layout as in tacc_kernel with one byte per entry: 16
// columns per lane, LPR lanes per output row, tiles of 8 codebooks.  Each
// tile is one level-3 subtree (or the level-L root when P < 8); tiles merge
// through a binary-counter stack of higher tree levels held in registers;
// pad tiles (all 128) finish the tree when C is not a power of two.
// stack levels above a tile: LV = 4 covers P / 8 <= 8 tiles (C <= 64), 5
// covers C <= 128, 7 covers C <= 512

__device__ __forceinline__ uint32_t avg4(uint32_t a, uint32_t b) { return __builtin_amdgcn_lerp(a, b, 0x01010101u); }

template <int NJ, int LV>
__global__ void __launch_bounds__(512, 4) tavg_kernel(const TArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  tlds_t* smem = (tlds_t*)smem_raw;

  const int tid = threadIdx.x;
  const int nt = blockDim.x;
  const int lane = tid & 63;
  const int wave = tuni(tid >> 6);
  const int nw = nt >> 6;
  const int C = a.C, M = a.M, Mt = a.Mt, RB = a.RB;
  constexpr int CT = 8;
  const int64_t N = a.N;
  const int lpr_log2 = a.lpr_log2;
  const int RS = 64 >> lpr_log2;
  const int r4 = lane >> lpr_log2;
  const int cg = lane & ((1 << lpr_log2) - 1);
  const int rby_log2 = 31 - __builtin_clz(Mt);   // one byte per entry: row bytes = Mt
  tlds_t* s_tab = smem;   // the table tile starts the LDS block (off_tab == 0)
  tlds_t* s_idx = smem + a.off_idx;
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
  __syncthreads();
  const float step = __builtin_ldexpf(1.0f, tuni(s_misc[1]));
  const float bias = __int_as_float(tuni(s_misc[0]));
  int L = 0;
  while ((1 << L) < C) ++L;
  const int P = 1 << L;
  const int ntile = (C + CT - 1) / CT;
  const int ntile_all = max(1, P / CT);

  const int upr = Mt >> 4;              // 16-byte units per table row of the tile
  const int upr_log2 = __builtin_ctz(upr);
  const int units = CT * 16 * upr;
  const int iwords = RB * 2;            // two index words (8 codebooks) per row
  const bool vec = a.vec_lut && a.vec_idx;
  const __amdgpu_buffer_rsrc_t trs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.lut), 0, (int)((int64_t)C * 16 * M), kBufDword3);
  tu32x4 tv[kTU];
  uint32_t iv[kIU];
  auto load_tile = [&](int c0, int64_t r0, int m0) {
#pragma unroll
    for (int j = 0; j < kTU; ++j) {
      const int u = tid + j * nt;
      const int row = u >> upr_log2, part = u & (upr - 1);
      const int c = c0 + (row >> 4), m = m0 + part * 16;
      const bool ok = u < units && c < C && m < M;
      tv[j] = __builtin_amdgcn_raw_buffer_load_b128(trs, ok ? (c * 16 + (row & 15)) * M + m : kOob, 0, 0);
    }
    const int64_t rows = min((int64_t)RB, N - r0);
    const __amdgpu_buffer_rsrc_t irs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(a.idx + r0 * C), 0, (int)min(rows * C, (int64_t)INT_MAX), kBufDword3);
#pragma unroll
    for (int j = 0; j < kIU; ++j) {
      const int d = tid + j * nt;
      const int i = d >> 1, q = d & 1;
      const bool ok = d < iwords && c0 + 4 * q < C;
      iv[j] = __builtin_amdgcn_raw_buffer_load_b32(irs, ok ? i * C + c0 + 4 * q : kOob, 0, 0);
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int j = 0; j < kTU; ++j) {
      const int u = tid + j * nt;
      if (u < units) {
        const int row = u >> upr_log2, part = u & (upr - 1);
        const tu32x4 b = tv[j] ^ (tu32x4){0x80808080u, 0x80808080u, 0x80808080u, 0x80808080u};  // q + 128
        *reinterpret_cast<tlds_u32x4*>(s_tab + (row << rby_log2) + part * 16) = b;
      }
    }
#pragma unroll
    for (int j = 0; j < kIU; ++j) {
      const int d = tid + j * nt;
      if (d < iwords) {
        const uint32_t cb = (uint32_t)(4 * (d & 1)) * 16u;
        tu32x4 o;
#pragma unroll
        for (int b = 0; b < 4; ++b) o[b] = (cb + 16u * b + ((iv[j] >> (8 * b)) & 15u)) << rby_log2;
        *reinterpret_cast<tlds_u32x4*>(s_idx + 16 * d) = o;
      }
    }
  };
  auto stage_direct = [&](int c0, int64_t r0, int m0) {
    const uint8_t* q8 = reinterpret_cast<const uint8_t*>(a.lut);
    for (int e = tid; e < CT * 16 * Mt; e += nt) {
      const int row = e >> rby_log2, col = e & (Mt - 1);
      const int c = c0 + (row >> 4), m = m0 + col;
      const bool ok = c < C && m < M;
      s_tab[(row << rby_log2) + col] = (char)(ok ? (q8[((int64_t)c * 16 + (row & 15)) * M + m] ^ 0x80u) : 0x80u);
    }
    for (int e = tid; e < RB * CT; e += nt) {
      const int i = e >> 3, cc = e & 7;
      const bool ok = r0 + i < N && c0 + cc < C;
      const uint32_t k = ok ? (uint32_t)(a.idx[(r0 + i) * C + c0 + cc] & 15u) : 0u;
      *reinterpret_cast<tlds_u32*>(s_idx + 4 * e) = ((uint32_t)cc * 16u + k) << rby_log2;
    }
  };

  const tlds_t* s_tab_lane = s_tab + cg * 16;
  int ib[NJ];
  const tlds_t* s_idx_row[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    ib[j] = (j * nw + wave) * RS + r4;
    s_idx_row[j] = s_idx + ib[j] * CT * 4;
  }

  for (int64_t w = blockIdx.x; w < a.nwork; w += gridDim.x) {
    const int mt = (int)(w % a.ntm);
    const int64_t r0 = (w / a.ntm) * RB;
    const int m0 = mt * Mt;
    tu32x4 stk[NJ][LV];   // stack[l]: a pending node at tree level 3 + l
    tu32x4 root[NJ];
    // merge a level-3 node x of tile t into the stack (carry chain of t's low bits)
    auto merge = [&](int j, tu32x4 x, int t) {
      bool carry = true;
#pragma unroll
      for (int l = 0; l < LV; ++l) {
        if (carry) {
          if ((t >> l) & 1) {
#pragma unroll
            for (int e = 0; e < 4; ++e) x[e] = avg4(stk[j][l][e], x[e]);
          } else {
            stk[j][l] = x;
            carry = false;
          }
        }
      }
    };

    if (vec) load_tile(0, r0, m0);
    for (int t = 0; t < ntile; ++t) {
      __syncthreads();
      if (vec) store_tile(); else stage_direct(t * CT, r0, m0);
      __syncthreads();
      if (vec && t + 1 < ntile) load_tile((t + 1) * CT, r0, m0);
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const tu32x4 k0 = *reinterpret_cast<const tlds_u32x4*>(s_idx_row[j]);
        const tu32x4 k1 = *reinterpret_cast<const tlds_u32x4*>(s_idx_row[j] + 16);
        tu32x4 v[8];
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          v[b] = *reinterpret_cast<const tlds_u32x4*>(s_tab_lane + k0[b]);
          v[4 + b] = *reinterpret_cast<const tlds_u32x4*>(s_tab_lane + k1[b]);
        }
        tu32x4 a0, a1, a2, a3, b0, b1, x;
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
        if (L >= 3) merge(j, x, t);
        else root[j] = (L == 0) ? v[0] : (L == 1) ? a0 : b0;
      }
    }
    if (L >= 3) {
      const tu32x4 pad = {0x80808080u, 0x80808080u, 0x80808080u, 0x80808080u};
      for (int t = ntile; t < ntile_all; ++t)
#pragma unroll
        for (int j = 0; j < NJ; ++j) merge(j, pad, t);
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
#pragma unroll
        for (int l = 0; l < LV; ++l)
          if (l == L - 3) root[j] = stk[j][l];
      }
    }

    // epilogue: acc = P (r - 128) for the lane's 16 columns
    const int col0 = m0 + cg * 16;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int64_t row = r0 + ib[j];
      if (row >= N || col0 >= M) continue;
      int out[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) out[e] = P * ((int)((root[j][e >> 2] >> (8 * (e & 3))) & 0xffu) - 128);
      float* yr = a.y ? a.y + row * M + col0 : nullptr;
      int32_t* ar = a.acc ? a.acc + row * M + col0 : nullptr;
      if (a.vec_out && col0 + 16 <= M) {
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          if (yr)
            __builtin_nontemporal_store((tf32x4){__builtin_fmaf((float)out[4 * h], step, bias),
                                                 __builtin_fmaf((float)out[4 * h + 1], step, bias),
                                                 __builtin_fmaf((float)out[4 * h + 2], step, bias),
                                                 __builtin_fmaf((float)out[4 * h + 3], step, bias)},
                                        reinterpret_cast<tf32x4*>(yr + 4 * h));
          if (ar)
            __builtin_nontemporal_store((tu32x4){(uint32_t)out[4 * h], (uint32_t)out[4 * h + 1],
                                                 (uint32_t)out[4 * h + 2], (uint32_t)out[4 * h + 3]},
                                        reinterpret_cast<tu32x4*>(ar + 4 * h));
        }
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (col0 + e < M) {
            if (yr) yr[e] = __builtin_fmaf((float)out[e], step, bias);
            if (ar) ar[e] = out[e];
          }
      }
    }
  }
}

// Per (kernel, block, LDS size): the LDS attribute is raised once and the
// number of resident workgroups per CU is queried once.
static int t_prepare(const void* fn, int block, int lds, hipError_t* err) {
  struct Entry { const void* fn; int block, lds, n; };
  static Entry cache[32];
  static int used = 0;
  static std::mutex mu;
  std::lock_guard<std::mutex> lock(mu);
  for (int i = 0; i < used; ++i)
    if (cache[i].fn == fn && cache[i].block == block && cache[i].lds == lds) return cache[i].n;
  if (lds > 64 * 1024) {
    const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) { *err = e; return 0; }
  }
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, block, lds) != hipSuccess || n < 1) n = 1;
  if (used < 32) cache[used++] = Entry{fn, block, lds, n};
  return n;
}

template <int ELEM, int NJ>
static hipError_t tlaunch(const TArgs& t, int nw, int cus, hipStream_t stream) {
  const void* fn = reinterpret_cast<const void*>(&tacc_kernel<ELEM, NJ>);
  hipError_t err = hipSuccess;
  const int per_cu = t_prepare(fn, nw * 64, t.lds_total, &err);
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
    for (int o = 1; o < 64; o <<= 1) vmax = __builtin_fmaxf(vmax, __shfl_xor(vmax, o));
    float sum = 0.0f;
#pragma unroll
    for (int i = 0; i < kSoftChunks; ++i) {
      if (lane + 64 * i < nq) {
        v[i].x = expf(v[i].x - vmax); v[i].y = expf(v[i].y - vmax);
        v[i].z = expf(v[i].z - vmax); v[i].w = expf(v[i].w - vmax);
        sum += (v[i].x + v[i].y) + (v[i].z + v[i].w);
      }
    }
    for (int o = 1; o < 64; o <<= 1) sum += __shfl_xor(sum, o);
#pragma unroll
    for (int i = 0; i < kSoftChunks; ++i) {
      const int q = lane + 64 * i;
      if (q < nq) __builtin_nontemporal_store((tf32x4){v[i].x / sum, v[i].y / sum, v[i].z / sum, v[i].w / sum}, yr + q);
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

template <int NJ, int LV>
static hipError_t alaunch(const TArgs& t, int nw, int cus, hipStream_t stream) {
  const void* fn = reinterpret_cast<const void*>(&tavg_kernel<NJ, LV>);
  hipError_t err = hipSuccess;
  const int per_cu = t_prepare(fn, nw * 64, t.lds_total, &err);
  if (err != hipSuccess) return err;
  int64_t blocks = t.nwork;
  const int64_t resident = (int64_t)per_cu * cus;
  if (blocks > resident) blocks = resident;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL((tavg_kernel<NJ, LV>), dim3((unsigned)blocks), dim3(nw * 64), t.lds_total, stream, t);
  return hipGetLastError();
}

hipError_t launch_tavg(int nj, const TArgs& t, int nw, int cus, hipStream_t stream) {
  if (nj != 1) return hipErrorInvalidValue;
  if (t.C <= 64) return alaunch<1, 4>(t, nw, cus, stream);
  if (t.C <= 128) return alaunch<1, 5>(t, nw, cus, stream);
  return alaunch<1, 7>(t, nw, cus, stream);
}

hipError_t launch_tacc(int elem, int nj, const TArgs& t, int nw, int cus, hipStream_t stream) {
  if (elem == kI8 && nj == 4) return tlaunch<kI8, 4>(t, nw, cus, stream);
  if (elem == kI8 && nj == 8) return tlaunch<kI8, 8>(t, nw, cus, stream);
  if (elem == kF32 && nj == 4) return tlaunch<kF32, 4>(t, nw, cus, stream);
  if (elem == kF32 && nj == 8) return tlaunch<kF32, 8>(t, nw, cus, stream);
  return hipErrorInvalidValue;
}

}  // namespace mdn
