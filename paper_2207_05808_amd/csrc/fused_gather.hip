// Fused encode + lookup-accumulate for tables that fit in LDS and codebook
// counts that divide 64 (§1, §2.1 of McCarter & Dronen: the encoding function
// is 4 comparisons per codebook; the product is the sum over codebooks of the
// selected table rows).
//
// Rows of A never go through LDS.  Lane l owns codebook c = l % C and row
// l / C of every group of G = 64 / C rows; it keeps c's 15 thresholds and 4
// split columns in registers and loads exactly the 4 values its walk compares
// (plain cached loads: a codebook's 4 columns share cache lines, and every
// line of a row is fetched from HBM once).  A wavefront handles R = NG * G
// rows per step through a buffer descriptor per step (uniform base, per-lane
// 32-bit offsets, range = the rows that exist) and keeps two steps of gathers
// in flight: the gathers of step s + 2 reuse step s's registers right after
// its walk.  The prologue issues the table's 16-byte units and the first two
// steps' gathers before it waits for anything, reduces the block exponents
// inside each wavefront, and has a single workgroup barrier.
//
// The walk writes, per (row, codebook), the LDS byte offset of the selected
// table row.  The accumulate gives each lane 8 consecutive columns of one row
// and, 4 codebooks at a time, adds the selected rows:
//  * int8 tables whose shifted codes cannot overflow 16 bits in total
//    (128 * sum_c 2^(e_c - e_min) <= 32768) are staged in LDS as int16
//    values q << (e_c - e_min) and summed with packed 16-bit adds: the
//    arithmetic is modular and the exact total fits, so the sum is exact;
//  * other int8 tables are staged as int8; each code is sign-extended from
//    its byte (v_bfe_i32), shifted by its codebook's e_c - e_min and added
//    in int32 (exact under the accumulator's precondition);
//  * fp32 tables are summed with ordered fp32 adds, codebooks ascending.
// Codebooks are padded to a multiple of 4 with offsets of an all-zero row.
#include "internal.hpp"


namespace mdn {

namespace {

typedef uint32_t u32x4g __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2g __attribute__((ext_vector_type(2)));
typedef float f32x4g __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char glds_t;
typedef __attribute__((address_space(3))) int32_t glds_i32;
typedef __attribute__((address_space(3))) uint32_t glds_u32;
typedef __attribute__((address_space(3))) u32x4g glds_u32x4;
typedef __attribute__((address_space(3))) u32x2g glds_u32x2;
typedef __attribute__((address_space(3))) f32x4g glds_f32x4;
typedef __attribute__((address_space(3))) float glds_f32;

// third descriptor dword for a raw (untyped, unswizzled) buffer on gfx9-family chips
constexpr int kBufferDword3 = 0x00020000;

__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ void wsync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int walk(float x0, float x1, float x2, float x3, float t0, float t1, float t2,
                                    float t3, float t4, float t5, float t6, float t7, float t8, float t9,
                                    float t10, float t11, float t12, float t13, float t14) {
  const bool b0 = x0 > t0;
  const bool b1 = x1 > (b0 ? t2 : t1);
  const float v2 = b0 ? (b1 ? t6 : t5) : (b1 ? t4 : t3);
  const bool b2 = x2 > v2;
  const float lo = b1 ? (b2 ? t10 : t9) : (b2 ? t8 : t7);
  const float hi = b1 ? (b2 ? t14 : t13) : (b2 ? t12 : t11);
  const bool b3 = x3 > (b0 ? hi : lo);
  return ((int)b0 << 3) | ((int)b1 << 2) | ((int)b2 << 1) | (int)b3;
}

// packed 16-bit add, lanes independent (wrap-around)
__device__ __forceinline__ uint32_t pk_add16(uint32_t a, uint32_t b) {
  typedef short s2 __attribute__((ext_vector_type(2)));
  const s2 x = __builtin_bit_cast(s2, a), y = __builtin_bit_cast(s2, b);
  return __builtin_bit_cast(uint32_t, (s2)(x + y));
}

}  // namespace

// LDS layout (bytes): [table: C*16 rows + 1 zero row, rs bytes each (sized for
// the widest staging)][shift per codebook][misc]
// [per wavefront: R rows x NSP int32 table offsets]
// IDX: the accumulate-only entry points.  The same kernel with the encode
// replaced by loads of the given indices: lane (row, codebook) loads one
// index byte per row group instead of 4 values of A, two steps in flight.
template <int ELEM, int NG, int UQ, bool IDX>
__global__ void __launch_bounds__(1024) gfused_kernel(const GArgs g) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  glds_t* smem = (glds_t*)smem_raw;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = uni(tid >> 6);
  const int nw = blockDim.x >> 6;
  const int C = g.C, M = g.M;
  const int no = (M + 7) >> 3;   // column octets
  const int NSP = g.NSP;

  glds_t* s_tab = smem;
  glds_i32* s_shc = reinterpret_cast<glds_i32*>(smem + g.off_shc);    // [C] shifts
  glds_i32* s_misc = reinterpret_cast<glds_i32*>(smem + g.off_misc);  // bias32
  glds_i32* s_off = reinterpret_cast<glds_i32*>(smem + g.off_wave) + (size_t)wave * g.R * NSP;

  const int c = lane & (C - 1);
  const int gsub = lane >> g.c_log2;   // row within a group of G rows
  const int G = 64 >> g.c_log2;
  const int R = g.R;
  const int64_t N = g.N;

  // ---------------- loads issued before any waiting, oldest first: the split
  // columns (the gather offsets need them), the dequantization constants, the
  // table as 16-byte units, then the gathers of this wavefront's first two
  // steps.  The prologue below waits only for what it uses, so HBM streams A
  // while the table is staged.
  int sp[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) sp[t] = IDX ? 0 : g.split[c * 4 + t];
  const uint32_t sbits = (ELEM == kI8) ? __float_as_uint(g.scale[c]) : 0u;
  const float ofs = (ELEM == kI8) ? g.offset[c] : 0.0f;

  constexpr int kTabUnits = 4;   // 16-byte table units per thread loaded up front
  const int upr = g.vec16 ? (ELEM == kF32 ? M >> 2 : M >> 4) : 0;   // units per table row
  const int units = C * 16 * upr;
  const __amdgpu_buffer_rsrc_t trs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(g.lut), 0, units * 16, kBufferDword3);
  u32x4g tv[kTabUnits];   // units past the table read as zeros and are not used
#pragma unroll
  for (int j = 0; j < kTabUnits; ++j)
    tv[j] = __builtin_amdgcn_raw_buffer_load_b128(trs, (tid + j * (int)blockDim.x) * 16, 0, 0);

  const unsigned dmax = IDX ? 0u : (unsigned)(g.D - 1);
  // byte offsets from the step's first row (split columns clamped: memory
  // safety); group q of G rows adds the uniform q * G * lda * 4 as soffset
  int goff[4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
    goff[t] = IDX ? gsub * C + c : (int)(((int64_t)gsub * g.lda + min((unsigned)sp[t], dmax)) * 4);
  // (indices: rows of C bytes)
  const int qstride = IDX ? G * C : (int)((int64_t)G * g.lda * 4);

  const int64_t tw = (int64_t)gridDim.x * nw;
  int64_t st = (int64_t)blockIdx.x * nw + wave;   // step index: rows [st * R, st * R + R)
  const char* A8 = IDX ? reinterpret_cast<const char*>(g.idx_in) : reinterpret_cast<const char*>(g.A);
  const int64_t step_bytes = IDX ? (int64_t)R * C : (int64_t)R * g.lda * 4;

  // Buffer loads against a per-step descriptor (uniform base in SGPRs, the
  // 32-bit lane offsets as voffset).  The descriptor's range is the rows that
  // exist: a partial last step reads zeros past row N - 1 (those rows are
  // encoded but never stored), and a step past the end has an empty range and
  // touches no memory, so every prefetch is issued unconditionally.  The 4
  // loads of a row group (which touch the same cache lines) are issued back to
  // back, a scheduling barrier after each group keeping the compiler from
  // interleaving groups: measured 3% faster than interleaved issue.
  const int64_t last_step = (N - 1) / R;
  auto gather = [&](int64_t s, float (&v)[NG][4]) {
    const int64_t sc = min(s, last_step);
    const int64_t rows = s > last_step ? 0 : min((int64_t)R, N - s * R);
    const int32_t nbytes =
        rows > 0 ? (int32_t)(IDX ? rows * C : min(step_bytes, (rows - 1) * g.lda * 4 + (int64_t)g.D * 4)) : 0;
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(A8 + sc * step_bytes), 0, nbytes, kBufferDword3);
    if (IDX) {
#pragma unroll
      for (int q = 0; q < NG; ++q) {
        v[q][0] = __int_as_float((int)__builtin_amdgcn_raw_buffer_load_b8(rsrc, goff[0], q * qstride, 0));
        v[q][1] = v[q][2] = v[q][3] = 0.0f;
      }
      return;
    }
#pragma unroll
    for (int q = 0; q < NG; ++q) {
#pragma unroll
      for (int t = 0; t < 4; ++t)
        v[q][t] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc, goff[t], q * qstride, 0));
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  float x[NG][4], xn[NG][4];
  gather(st, x);
  gather(st + tw, xn);

  float t0 = 0, t1 = 0, t2 = 0, t3 = 0, t4 = 0, t5 = 0, t6 = 0, t7 = 0, t8 = 0, t9 = 0, t10 = 0, t11 = 0,
        t12 = 0, t13 = 0, t14 = 0;
  if (!IDX) {
    const float* th = g.thr + c * kNodes;
    t0 = th[0]; t1 = th[1]; t2 = th[2]; t3 = th[3]; t4 = th[4]; t5 = th[5]; t6 = th[6]; t7 = th[7];
    t8 = th[8]; t9 = th[9]; t10 = th[10]; t11 = th[11]; t12 = th[12]; t13 = th[13]; t14 = th[14];
  }

  // ---------------- dequantization constants, reduced inside each wavefront
  // (lane l holds codebook l % C; every wavefront reaches the same values)
  const int e_c = (int)((sbits >> 23) & 0xffu) - 127;   // exponent of scale_c, an exact power of two
  int emin = e_c;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) emin = min(emin, __shfl_xor(emin, o));
  const int sh = (ELEM == kI8) ? min(e_c - emin, 30) : 0;
  int pw = (lane < C) ? (sh <= 14 ? (1 << sh) : (1 << 15)) : 0;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) pw += __shfl_xor(pw, o);
  const bool narrow = (ELEM == kI8) && (128 * pw <= 32768);   // every int8 code, -128 included
  const int rs = (ELEM == kF32) ? g.rs32 : (narrow ? g.rs16 : g.rs8);
  const float step = __builtin_ldexpf(1.0f, emin);
  if (wave == 0) {
    if (lane < C) s_shc[lane] = sh;
    if (ELEM == kI8) {
      // bias32: double sum over codebooks in ascending order (every lane computes it)
      double sum = 0.0;
      for (int cc = 0; cc < C; ++cc)
        sum += (double)__int_as_float(__builtin_amdgcn_readlane(__float_as_int(ofs), cc));
      if (lane == 0) s_misc[0] = __float_as_int((float)sum);
    }
  }

  // ---------------- table staging: rows (c, k) plus the all-zero row C * 16
  const int rows = C * 16;
  const bool vec_all = units > 0 && units <= kTabUnits * (int)blockDim.x;
  if (vec_all) {
    // unit u is bytes [16 (u % upr), 16 (u % upr) + 16) of table row u / upr
#pragma unroll
    for (int j = 0; j < kTabUnits; ++j) {
      const int u = tid + j * (int)blockDim.x;
      const int row = min(u, units - 1) / upr;
      const int col = (min(u, units - 1) - row * upr) * 16;   // byte offset in the global row
      const int shr = __shfl(sh, row >> 4);   // lane row / 16 holds that codebook's shift
      if (u < units) {
        if (ELEM == kI8 && narrow) {
          u32x4g lo, hi;
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const int v = (int)tv[j][w];
            const uint32_t p0 = ((uint32_t)(__builtin_amdgcn_sbfe(v, 0, 8) << shr) & 0xffffu) |
                                ((uint32_t)(__builtin_amdgcn_sbfe(v, 8, 8) << shr) << 16);
            const uint32_t p1 = ((uint32_t)(__builtin_amdgcn_sbfe(v, 16, 8) << shr) & 0xffffu) |
                                ((uint32_t)(__builtin_amdgcn_sbfe(v, 24, 8) << shr) << 16);
            if (w < 2) { lo[2 * w] = p0; lo[2 * w + 1] = p1; } else { hi[2 * w - 4] = p0; hi[2 * w - 3] = p1; }
          }
          *reinterpret_cast<glds_u32x4*>(s_tab + row * rs + 2 * col) = lo;
          *reinterpret_cast<glds_u32x4*>(s_tab + row * rs + 2 * col + 16) = hi;
        } else {
          *reinterpret_cast<glds_u32x4*>(s_tab + row * rs + col) = tv[j];
        }
      }
    }
    for (int w = tid; w < (rs >> 2); w += blockDim.x) *reinterpret_cast<glds_u32*>(s_tab + rows * rs + 4 * w) = 0u;
  }
  if (!vec_all) {
    // general staging (tables larger than the up-front units, or rows that are
    // not whole 16-byte units): 8 LDS dwords per thread per round, all global
    // loads of a round issued first; columns padded to octets with zeros
    __syncthreads();   // shifts visible
    const int wpr = (ELEM == kF32) ? 8 * no : (narrow ? 4 * no : 2 * no);  // dwords per LDS row
    int wlog = 0;
    while ((1 << wlog) < wpr) ++wlog;
    const int total = (rows + 1) << wlog;
    const int8_t* q8 = reinterpret_cast<const int8_t*>(g.lut);
    const float* qf = reinterpret_cast<const float*>(g.lut);
    const int64_t last = (int64_t)rows * M - 1;
    for (int base = tid; base < total; base += 8 * blockDim.x) {
      uint32_t v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int u = base + j * blockDim.x;
        const int row = u >> wlog, w = u & ((1 << wlog) - 1);
        const int64_t e0 = (int64_t)row * M;
        if (ELEM == kF32) {
          v[j] = __float_as_uint(qf[min(e0 + w, last)]);
        } else if (narrow) {
          const uint32_t lo = (uint8_t)q8[min(e0 + 2 * w, last)], hi = (uint8_t)q8[min(e0 + 2 * w + 1, last)];
          v[j] = lo | (hi << 8);
        } else {
          uint32_t xx = 0;
#pragma unroll
          for (int e = 0; e < 4; ++e) xx |= (uint32_t)(uint8_t)q8[min(e0 + 4 * w + e, last)] << (8 * e);
          v[j] = xx;
        }
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int u = base + j * blockDim.x;
        const int row = u >> wlog, w = u & ((1 << wlog) - 1);
        if (u >= total || w >= wpr) continue;
        uint32_t xx = 0;
        if (row < rows) {
          if (ELEM == kF32) {
            xx = w < M ? v[j] : 0u;
          } else if (narrow) {
            const int shr = s_shc[row >> 4];
            const int m = 2 * w;
            const int lo = m < M ? ((int)(int8_t)(v[j] & 0xffu) << shr) : 0;
            const int hi = m + 1 < M ? ((int)(int8_t)(v[j] >> 8) << shr) : 0;
            xx = ((uint32_t)lo & 0xffffu) | ((uint32_t)hi << 16);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (4 * w + e < M) xx |= v[j] & (0xffu << (8 * e));
          }
        }
        *reinterpret_cast<glds_u32*>(s_tab + row * rs + 4 * w) = xx;
      }
    }
  }
  {
    // padding codebook slots of every row point at the zero row
    glds_i32* all_off = reinterpret_cast<glds_i32*>(smem + g.off_wave);
    for (int u = tid; u < nw * g.R * NSP; u += blockDim.x) all_off[u] = rows * rs;
  }
  if (g.act != 0) {
    // layer bias row, zero past M (and everywhere without a bias)
    glds_f32* sbias = reinterpret_cast<glds_f32*>(smem + g.off_bias);
    for (int u = tid; u < 8 * no; u += blockDim.x) sbias[u] = (g.col_bias && u < M) ? g.col_bias[u] : 0.0f;
  }
  __syncthreads();

  const float bias = __int_as_float(uni(s_misc[0]));
  const int cbase = c * 16 * rs;
  // ---------------- accumulate lane mapping: LPR lanes per row, 8 columns per lane-slot
  const int lpr_log2 = g.lpr_log2;
  const int LPR = 1 << lpr_log2;
  const int ar = lane >> lpr_log2;
  const int cg = lane & (LPR - 1);
  const int RA = 64 >> lpr_log2;
  // lane-slot u covers column quads qa = cg + 2 LPR u and qb = qa + LPR, so each
  // output store instruction writes LPR consecutive 16-byte chunks of a row
  const int nq4 = (M + 3) >> 2;
  const int qbytes = (ELEM == kF32) ? 16 : (narrow ? 8 : 4);  // LDS bytes of 4 columns
  int lqa[UQ], lqb[UQ];
#pragma unroll
  for (int u = 0; u < UQ; ++u) {
    lqa[u] = min(cg + 2 * LPR * u, nq4 - 1) * qbytes;
    lqb[u] = min(cg + 2 * LPR * u + LPR, nq4 - 1) * qbytes;
  }
  const int nslot = (C + 3) & ~3;

  // One step: walk step st from `cur`, reuse `cur` for the gathers of step
  // st + 2 tw (so two steps of gathers stay in flight with two buffers), then
  // accumulate step st.
  auto step_body = [&](float (&cur)[NG][4]) {
    const int64_t row0 = st * R;
    // walks and the next gathers at raised wavefront priority, so that a
    // wavefront whose data has arrived issues its next loads ahead of the
    // other wavefronts' accumulate work
    __builtin_amdgcn_s_setprio(2);
    // encode: one walk per (row, codebook) of this lane
#pragma unroll
    for (int q = 0; q < NG; ++q) {
      // (indices are preconditions in [0, 16); the mask keeps LDS reads in the table)
      const int k = IDX ? (__float_as_int(cur[q][0]) & 15)
                        : walk(cur[q][0], cur[q][1], cur[q][2], cur[q][3], t0, t1, t2, t3, t4, t5, t6, t7, t8, t9,
                               t10, t11, t12, t13, t14);
      const int r = q * G + gsub;
      s_off[r * NSP + c] = cbase + k * rs;
      if (g.idx_out) {
        const int64_t row = row0 + r;
        if (row < N) g.idx_out[row * C + c] = (uint8_t)k;
      }
    }
    gather(st + 2 * tw, cur);
    __builtin_amdgcn_s_setprio(0);
    wsync();

    for (int rb = 0; rb < R; rb += RA) {
      const int rr = rb + ar;
      const glds_i32* orow = s_off + rr * NSP;
      int iacc[UQ][8];
      float facc[UQ][8];
#pragma unroll
      for (int u = 0; u < UQ; ++u)
#pragma unroll
        for (int e = 0; e < 8; ++e) { iacc[u][e] = 0; facc[u][e] = 0.0f; }
      u32x4g o = *reinterpret_cast<const glds_u32x4*>(orow);
      if (ELEM == kI8 && narrow) {
        uint32_t hacc[UQ][4];     // 8 int16 sums in 4 dwords
#pragma unroll
        for (int u = 0; u < UQ; ++u)
#pragma unroll
          for (int e = 0; e < 4; ++e) hacc[u][e] = 0u;
        for (int j = 0; j < nslot; j += 4) {
          const u32x4g on = *reinterpret_cast<const glds_u32x4*>(orow + min(j + 4, nslot - 4));
          u32x2g va[4][UQ], vb[4][UQ];
#pragma unroll
          for (int u = 0; u < UQ; ++u) {
            va[0][u] = *reinterpret_cast<const glds_u32x2*>(s_tab + o.x + lqa[u]);
            vb[0][u] = *reinterpret_cast<const glds_u32x2*>(s_tab + o.x + lqb[u]);
            va[1][u] = *reinterpret_cast<const glds_u32x2*>(s_tab + o.y + lqa[u]);
            vb[1][u] = *reinterpret_cast<const glds_u32x2*>(s_tab + o.y + lqb[u]);
            va[2][u] = *reinterpret_cast<const glds_u32x2*>(s_tab + o.z + lqa[u]);
            vb[2][u] = *reinterpret_cast<const glds_u32x2*>(s_tab + o.z + lqb[u]);
            va[3][u] = *reinterpret_cast<const glds_u32x2*>(s_tab + o.w + lqa[u]);
            vb[3][u] = *reinterpret_cast<const glds_u32x2*>(s_tab + o.w + lqb[u]);
          }
#pragma unroll
          for (int b = 0; b < 4; ++b)
#pragma unroll
            for (int u = 0; u < UQ; ++u) {
              hacc[u][0] = pk_add16(hacc[u][0], va[b][u].x);
              hacc[u][1] = pk_add16(hacc[u][1], va[b][u].y);
              hacc[u][2] = pk_add16(hacc[u][2], vb[b][u].x);
              hacc[u][3] = pk_add16(hacc[u][3], vb[b][u].y);
            }
          o = on;
        }
#pragma unroll
        for (int u = 0; u < UQ; ++u)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            iacc[u][2 * e] = __builtin_amdgcn_sbfe((int)hacc[u][e], 0, 16);
            iacc[u][2 * e + 1] = (int)hacc[u][e] >> 16;
          }
      } else if (ELEM == kI8) {
        for (int j = 0; j < nslot; j += 4) {
          const u32x4g on = *reinterpret_cast<const glds_u32x4*>(orow + min(j + 4, nslot - 4));
          u32x2g v[4][UQ];
#pragma unroll
          for (int u = 0; u < UQ; ++u) {
            v[0][u].x = *reinterpret_cast<const glds_u32*>(s_tab + o.x + lqa[u]);
            v[0][u].y = *reinterpret_cast<const glds_u32*>(s_tab + o.x + lqb[u]);
            v[1][u].x = *reinterpret_cast<const glds_u32*>(s_tab + o.y + lqa[u]);
            v[1][u].y = *reinterpret_cast<const glds_u32*>(s_tab + o.y + lqb[u]);
            v[2][u].x = *reinterpret_cast<const glds_u32*>(s_tab + o.z + lqa[u]);
            v[2][u].y = *reinterpret_cast<const glds_u32*>(s_tab + o.z + lqb[u]);
            v[3][u].x = *reinterpret_cast<const glds_u32*>(s_tab + o.w + lqa[u]);
            v[3][u].y = *reinterpret_cast<const glds_u32*>(s_tab + o.w + lqb[u]);
          }
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const int cc = min(j + b, C - 1);   // padding slots read the zero row: any weight
            const int sh = uni(s_shc[cc]);
#pragma unroll
            for (int u = 0; u < UQ; ++u)
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                iacc[u][e] += __builtin_amdgcn_sbfe((int)v[b][u].x, 8 * e, 8) << sh;
                iacc[u][4 + e] += __builtin_amdgcn_sbfe((int)v[b][u].y, 8 * e, 8) << sh;
              }
          }
          o = on;
        }
      } else {
        for (int j = 0; j < nslot; j += 4) {
          const u32x4g on = *reinterpret_cast<const glds_u32x4*>(orow + min(j + 4, nslot - 4));
          f32x4g v[4][UQ][2];
#pragma unroll
          for (int u = 0; u < UQ; ++u) {
            v[0][u][0] = *reinterpret_cast<const glds_f32x4*>(s_tab + o.x + lqa[u]);
            v[0][u][1] = *reinterpret_cast<const glds_f32x4*>(s_tab + o.x + lqb[u]);
            v[1][u][0] = *reinterpret_cast<const glds_f32x4*>(s_tab + o.y + lqa[u]);
            v[1][u][1] = *reinterpret_cast<const glds_f32x4*>(s_tab + o.y + lqb[u]);
            v[2][u][0] = *reinterpret_cast<const glds_f32x4*>(s_tab + o.z + lqa[u]);
            v[2][u][1] = *reinterpret_cast<const glds_f32x4*>(s_tab + o.z + lqb[u]);
            v[3][u][0] = *reinterpret_cast<const glds_f32x4*>(s_tab + o.w + lqa[u]);
            v[3][u][1] = *reinterpret_cast<const glds_f32x4*>(s_tab + o.w + lqb[u]);
          }
#pragma unroll
          for (int b = 0; b < 4; ++b)   // codebooks strictly in ascending order
#pragma unroll
            for (int u = 0; u < UQ; ++u) {
              facc[u][0] = facc[u][0] + v[b][u][0].x;
              facc[u][1] = facc[u][1] + v[b][u][0].y;
              facc[u][2] = facc[u][2] + v[b][u][0].z;
              facc[u][3] = facc[u][3] + v[b][u][0].w;
              facc[u][4] = facc[u][4] + v[b][u][1].x;
              facc[u][5] = facc[u][5] + v[b][u][1].y;
              facc[u][6] = facc[u][6] + v[b][u][1].z;
              facc[u][7] = facc[u][7] + v[b][u][1].w;
            }
          o = on;
        }
      }

      // epilogue: 8 columns per lane-slot
      const int64_t row = row0 + rr;
      const bool store = rr < R && row < N;
      auto store_slot = [&](int u, const float (&o)[8]) {
        float* yrow = g.y + row * M;
        int32_t* arow = (ELEM == kI8 && g.acc) ? g.acc + row * M : nullptr;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int qd = cg + 2 * LPR * u + h * LPR;
          if (qd >= nq4) continue;
          const int mh = 4 * qd;
          if (g.vec_out && mh + 4 <= M) {
            if (!IDX || g.y)   // (y is required unless the indices are given)
              __builtin_nontemporal_store((f32x4g){o[4 * h], o[4 * h + 1], o[4 * h + 2], o[4 * h + 3]},
                                          reinterpret_cast<f32x4g*>(yrow + mh));
            if (arow)
              __builtin_nontemporal_store((u32x4g){(uint32_t)iacc[u][4 * h], (uint32_t)iacc[u][4 * h + 1],
                                                   (uint32_t)iacc[u][4 * h + 2], (uint32_t)iacc[u][4 * h + 3]},
                                          reinterpret_cast<u32x4g*>(arow + mh));
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (mh + e < M) {
                if (!IDX || g.y) yrow[mh + e] = o[4 * h + e];
                if (arow) arow[mh + e] = iacc[u][4 * h + e];
              }
          }
        }
      };
      if (g.act == 0) {
        if (store) {
#pragma unroll
          for (int u = 0; u < UQ; ++u) {
            float o[8];
#pragma unroll
            for (int e = 0; e < 8; ++e)
              o[e] = (ELEM == kI8) ? __builtin_fmaf((float)iacc[u][e], step, bias) : facc[u][e];
            store_slot(u, o);
          }
        }
      } else {
        // layer output sigma: z = y + bias, then ReLU, or a softmax over the
        // row's LPR lanes (every lane takes part in the reductions)
        float out[UQ][8];
        const glds_f32* sbias = reinterpret_cast<const glds_f32*>(smem + g.off_bias);
        float vmax = -__builtin_inff();
#pragma unroll
        for (int u = 0; u < UQ; ++u)
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int qd = cg + 2 * LPR * u + h * LPR;
            const f32x4g bv = *reinterpret_cast<const glds_f32x4*>(sbias + 4 * min(qd, nq4 - 1));
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float y0 = (ELEM == kI8) ? __builtin_fmaf((float)iacc[u][4 * h + e], step, bias)
                                             : facc[u][4 * h + e];
              float z = y0 + bv[e];
              if (g.act == 2) z = (z > 0.0f) ? z : 0.0f;
              out[u][4 * h + e] = z;
              if (4 * qd + e < M) vmax = __builtin_fmaxf(vmax, z);
            }
          }
        if (g.act == 3) {
          for (int o = 1; o < LPR; o <<= 1) vmax = __builtin_fmaxf(vmax, __shfl_xor(vmax, o));
          float sum = 0.0f;
#pragma unroll
          for (int u = 0; u < UQ; ++u)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const int qd = cg + 2 * LPR * u + h * LPR;
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const float ex = (4 * qd + e < M) ? expf(out[u][4 * h + e] - vmax) : 0.0f;
                out[u][4 * h + e] = ex;
                sum += ex;
              }
            }
          for (int o = 1; o < LPR; o <<= 1) sum += __shfl_xor(sum, o);
#pragma unroll
          for (int u = 0; u < UQ; ++u)
#pragma unroll
            for (int e = 0; e < 8; ++e) out[u][e] = out[u][e] / sum;
        }
        if (store) {
#pragma unroll
          for (int u = 0; u < UQ; ++u) store_slot(u, out[u]);
        }
      }
    }
    wsync();  // the next step overwrites this wavefront's offsets
  };

  while (st * R < N) {
    step_body(x);
    st += tw;
    if (st * R >= N) break;
    step_body(xn);
    st += tw;
  }
}

template <int ELEM, int NG, int UQ, bool IDX>
static hipError_t glaunch(const GArgs& g, int nw, int cus, hipStream_t stream) {
  const void* fn = reinterpret_cast<const void*>(&gfused_kernel<ELEM, NG, UQ, IDX>);
  hipError_t err = hipSuccess;
  const int per_cu = launch_prepare(fn, nw * 64, g.lds_total, &err);
  if (err != hipSuccess) return err;
  const int64_t steps = (g.N + g.R - 1) / g.R;
  int64_t blocks = (steps + nw - 1) / nw;
  const int64_t resident = (int64_t)per_cu * cus;
  if (blocks > resident) blocks = resident;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL((gfused_kernel<ELEM, NG, UQ, IDX>), dim3((unsigned)blocks), dim3(nw * 64), g.lds_total, stream, g);
  return hipGetLastError();
}

#define MDN_G_CASE(E, NG, UQ) \
  if (elem == E && ng == NG && uq == UQ)                                   \
    return g.idx_in ? glaunch<E, NG, UQ, true>(g, nw, cus, stream) : glaunch<E, NG, UQ, false>(g, nw, cus, stream);

hipError_t launch_gfused(int elem, int ng, int uq, const GArgs& g, int nw, int cus, hipStream_t stream) {
  MDN_G_CASE(kI8, 1, 1) MDN_G_CASE(kI8, 2, 1) MDN_G_CASE(kI8, 4, 1)
  MDN_G_CASE(kI8, 1, 2) MDN_G_CASE(kI8, 2, 2) MDN_G_CASE(kI8, 4, 2)
  MDN_G_CASE(kI8, 1, 4) MDN_G_CASE(kI8, 2, 4) MDN_G_CASE(kI8, 4, 4)
  MDN_G_CASE(kF32, 1, 1) MDN_G_CASE(kF32, 2, 1) MDN_G_CASE(kF32, 4, 1)
  MDN_G_CASE(kF32, 1, 2) MDN_G_CASE(kF32, 2, 2) MDN_G_CASE(kF32, 4, 2)
  MDN_G_CASE(kF32, 1, 4) MDN_G_CASE(kF32, 2, 4) MDN_G_CASE(kF32, 4, 4)
  return hipErrorInvalidValue;
}

}  // namespace mdn
