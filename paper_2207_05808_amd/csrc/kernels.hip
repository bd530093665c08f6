// Hot-path kernels for gfx950: tree encoding (§1, §2.1 of McCarter & Dronen)
// and lookup-accumulate over 8-bit block floating point or fp32 tables (§1).
//
// One templated kernel covers three modes:
//   kEncode : stage rows of A in LDS, walk C 4-level trees per row, write idx.
//   kAccum  : stage idx rows in LDS, gather-accumulate a LUT column tile.
//   kFused  : both, the indices never leaving LDS.
//
// Work split.  A workgroup of NW wavefronts first stages its LUT column tile
// ([C*16 rows][Mt columns], blockIdx.y picks the tile), the thresholds and
// split columns in LDS; then every wavefront loops independently over
// "chunks" of RW consecutive rows (persistent grid-stride loop, no further
// workgroup barriers).  Per chunk a wavefront
//   1. writes the chunk prefetched into VGPRs during the previous iteration
//      into its private LDS row buffer and issues the loads of its next chunk
//      (16-byte non-temporal loads, coalesced across the wavefront),
//   2. encodes: lane p handles (row, codebook) pairs p, p+64, ... reading the
//      4 split columns and the heap-ordered thresholds from LDS,
//   3. accumulates: lane -> (row = lane / LPR, column quad cg = lane % LPR),
//      LPR = 64 / RW; per codebook it reads the 4-byte (int8) or 16-byte
//      (fp32) quad of LUT row (c, idx) and accumulates it.  For int8 tables
//      v_dot4c_i32_i8 with the weight 2^sh << 8b extracts, sign-extends and
//      shifts byte b in one instruction; shifts above 6 take a bfe+shift path.
//   4. applies the epilogue y = fmaf(float(acc), 2^e_min, bias32) and stores
//      with 16-byte non-temporal stores.
#include "internal.hpp"

#include <climits>
#include <type_traits>

#include <atomic>
#include <mutex>

namespace mdn {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32_ua __attribute__((aligned(1)));   // a dword at any byte address
#define MDN_CONST __attribute__((address_space(4)))
typedef __attribute__((address_space(3))) char lds_t;           // 32-bit LDS addresses
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Exponent of a normal fp32 power of two: scale = 2^e.
__device__ __forceinline__ int exp_of_bits(uint32_t bits) { return (int)((bits >> 23) & 0xffu) - 127; }

// Minimum and maximum over the 64 lanes of a wavefront (the same value in
// every lane): DPP exchanges within each row of 16 lanes (quad butterflies,
// then rotations by 4 and 8), then the four row results through readlane.
// (__shfl_xor compiles to ds_bpermute with a wait on each step.)
__device__ __forceinline__ void wave_minmax(int& lo, int& hi) {
#define MDN_MINMAX_STEP(CTRL)                                              \
  lo = min(lo, __builtin_amdgcn_update_dpp(lo, lo, CTRL, 0xf, 0xf, false)); \
  hi = max(hi, __builtin_amdgcn_update_dpp(hi, hi, CTRL, 0xf, 0xf, false));
  MDN_MINMAX_STEP(0xB1)    // quad_perm [1, 0, 3, 2]
  MDN_MINMAX_STEP(0x4E)    // quad_perm [2, 3, 0, 1]
  MDN_MINMAX_STEP(0x124)   // row_ror 4
  MDN_MINMAX_STEP(0x128)   // row_ror 8
#undef MDN_MINMAX_STEP
  lo = min(min(__builtin_amdgcn_readlane(lo, 0), __builtin_amdgcn_readlane(lo, 16)),
           min(__builtin_amdgcn_readlane(lo, 32), __builtin_amdgcn_readlane(lo, 48)));
  hi = max(max(__builtin_amdgcn_readlane(hi, 0), __builtin_amdgcn_readlane(hi, 16)),
           max(__builtin_amdgcn_readlane(hi, 32), __builtin_amdgcn_readlane(hi, 48)));
}

__device__ __forceinline__ uint32_t bfe(uint32_t v, int off, int width) {
  return __builtin_amdgcn_ubfe(v, off, width);
}

// Rows of a strided 2-D byte array, RW rows per chunk, prefetched in 16-byte
// units through VGPRs.  Unit j of lane l is u = l + 64 j; it belongs to row
// u / upr and column unit u % upr.  Loads and LDS stores carry no per-lane
// predicate (a predicate would make the compiler wait for every load in
// turn): idle units re-read unit 0 and land in a per-wavefront dummy slot,
// and in the last, partial chunk the rows past N re-read the last valid row.
template <int PF, bool NT>
struct Prefetch {
  u32x4 buf[PF > 0 ? PF : 1];
  int goff[PF > 0 ? PF : 1];   // byte offset from the chunk's first row in global memory
  int loff[PF > 0 ? PF : 1];   // byte offset in the LDS buffer (dummy slot when idle)
  int rrow[PF > 0 ? PF : 1];   // row within the chunk (0 when idle)

  __device__ __forceinline__ void init(int lane, int rw, int upr, int64_t src_rs, int lds_rs, int dummy) {
    // u / upr as (u + 1/2) * rcp(upr), truncated: with rcp within 1 ulp and
    // one more rounding, the product is within 2^-21 (u + 1/2) / upr of
    // (u + 1/2) / upr, which lies at least 1/(2 upr) from every integer, so
    // the truncation is exact for u < 2^20 (and upr < 2^24, exact in fp32)
    const float rcp = __builtin_amdgcn_rcpf((float)upr);
#pragma unroll
    for (int j = 0; j < PF; ++j) {
      const int u = lane + 64 * j;
      const bool live = u < rw * upr;
      const int r = live ? (int)(((float)u + 0.5f) * rcp) : 0;
      const int col = live ? u - r * upr : 0;
      goff[j] = (int)(r * src_rs) + col * 16;
      loff[j] = live ? r * lds_rs + col * 16 : dummy;
      rrow[j] = r;
    }
  }
  __device__ __forceinline__ u32x4 ld(const char* p) const {
    const u32x4* q = reinterpret_cast<const u32x4*>(p);
    return NT ? __builtin_nontemporal_load(q) : *q;
  }
  // rows_valid is wavefront-uniform, so the tail test is a scalar branch
  __device__ __forceinline__ void load(const char* base, int rows_valid, int rw, int src_rs) {
    if (rows_valid == rw) {
#pragma unroll
      for (int j = 0; j < PF; ++j) buf[j] = ld(base + goff[j]);
    } else {
#pragma unroll
      for (int j = 0; j < PF; ++j) {
        const int over = max(rrow[j] - (rows_valid - 1), 0);
        buf[j] = ld(base + goff[j] - over * src_rs);
      }
    }
  }
  __device__ __forceinline__ void store(lds_t* lds) const {
#pragma unroll
    for (int j = 0; j < PF; ++j) *reinterpret_cast<lds_u32x4*>(lds + loff[j]) = buf[j];
  }
};

typedef __attribute__((address_space(3))) float lds_f32;
typedef __attribute__((address_space(3))) int lds_i32;
typedef __attribute__((address_space(3))) uint32_t lds_u32;
typedef __attribute__((address_space(3))) uint8_t lds_u8;
typedef __attribute__((address_space(3))) f32x4 lds_f32x4;

// One group of G codebooks (G = 8 or 16) of the accumulate: all idx words and
// all G x UQ LUT quads are read first (independent LDS reads), then the
// updates run.  int8 with DOT: v_dot4c_i32_i8 against weight 2^sh << 8e picks
// byte e of the quad, sign-extends it and shifts it; fp32: ordered adds.
template <int ELEM, int UQ, bool DOT, int G>
__device__ __forceinline__ void acc_group(int c0, const lds_t* ir, const lds_t* const* lq, int rs,
                                          const lds_t* s_shp, const lds_i32* s_sh,
                                          int (&iacc)[UQ][4], float (&facc)[UQ][4]) {
  uint32_t kw[G / 4];
#pragma unroll
  for (int q = 0; q < G / 4; ++q) kw[q] = *reinterpret_cast<const lds_u32*>(ir + c0 + 4 * q);
  if (ELEM == kI8) {
    int v[G][UQ];
#pragma unroll
    for (int b = 0; b < G; ++b) {
      const int k = (int)bfe(kw[b >> 2], 8 * (b & 3), 4);
      const int off = (int)__umul24((uint32_t)((c0 + b) * kK + k), (uint32_t)rs);
#pragma unroll
      for (int u = 0; u < UQ; ++u) v[b][u] = *reinterpret_cast<const lds_i32*>(lq[u] + off);
    }
    if (DOT) {
      uint32_t shw[G / 8];
#pragma unroll
      for (int q = 0; q < G / 8; ++q)
        shw[q] = (uint32_t)uniform((int)*reinterpret_cast<const lds_u32*>(s_shp + (c0 >> 1) + 4 * q));
#pragma unroll
      for (int b = 0; b < G; ++b) {
        const int w = 1 << bfe(shw[b >> 3], 4 * (b & 7), 4);
#pragma unroll
        for (int u = 0; u < UQ; ++u) {
          iacc[u][0] = __builtin_amdgcn_sdot4(v[b][u], w, iacc[u][0], false);
          iacc[u][1] = __builtin_amdgcn_sdot4(v[b][u], w << 8, iacc[u][1], false);
          iacc[u][2] = __builtin_amdgcn_sdot4(v[b][u], w << 16, iacc[u][2], false);
          iacc[u][3] = __builtin_amdgcn_sdot4(v[b][u], w << 24, iacc[u][3], false);
        }
      }
    } else {
#pragma unroll
      for (int b = 0; b < G; ++b) {
        const int sh = uniform(s_sh[c0 + b]);
#pragma unroll
        for (int u = 0; u < UQ; ++u)
#pragma unroll
          for (int e = 0; e < 4; ++e) iacc[u][e] += __builtin_amdgcn_sbfe(v[b][u], 8 * e, 8) << sh;
      }
    }
  } else {
    f32x4 v[G][UQ];
#pragma unroll
    for (int b = 0; b < G; ++b) {
      const int k = (int)bfe(kw[b >> 2], 8 * (b & 3), 4);
      const int off = (int)__umul24((uint32_t)((c0 + b) * kK + k), (uint32_t)rs);
#pragma unroll
      for (int u = 0; u < UQ; ++u) v[b][u] = *reinterpret_cast<const lds_f32x4*>(lq[u] + off);
    }
#pragma unroll
    for (int b = 0; b < G; ++b)   // codebooks strictly in ascending order
#pragma unroll
      for (int u = 0; u < UQ; ++u) {
        facc[u][0] = facc[u][0] + v[b][u].x;
        facc[u][1] = facc[u][1] + v[b][u].y;
        facc[u][2] = facc[u][2] + v[b][u].z;
        facc[u][3] = facc[u][3] + v[b][u].w;
      }
  }
}

// Accumulate one chunk of rows over the LUT tile.  Lane (ar, cg) owns column
// quads q = cg + u * LPR of row ar (u < UQ); quads past the tile are clamped
// to the last one (read, never stored), so no load carries a predicate.
template <int ELEM, int UQ, bool DOT>
__device__ __forceinline__ void accumulate(const lds_t* ir, const lds_t* const* lq, int C, int rs,
                                           const lds_t* s_shp, const lds_i32* s_sh,
                                           int (&iacc)[UQ][4], float (&facc)[UQ][4]) {
  int c0 = 0;
  for (; c0 + 16 <= C; c0 += 16) acc_group<ELEM, UQ, DOT, 16>(c0, ir, lq, rs, s_shp, s_sh, iacc, facc);
  if (c0 + 8 <= C) {
    acc_group<ELEM, UQ, DOT, 8>(c0, ir, lq, rs, s_shp, s_sh, iacc, facc);
    c0 += 8;
  }
  for (; c0 < C; ++c0) {
    const int k = (int)(*reinterpret_cast<const lds_u8*>(ir + c0) & 15u);
    const int off = (int)__umul24((uint32_t)(c0 * kK + k), (uint32_t)rs);
    if (ELEM == kI8) {
      const int sh = uniform(s_sh[c0]);
#pragma unroll
      for (int u = 0; u < UQ; ++u) {
        const int v = *reinterpret_cast<const lds_i32*>(lq[u] + off);
#pragma unroll
        for (int e = 0; e < 4; ++e) iacc[u][e] += __builtin_amdgcn_sbfe(v, 8 * e, 8) << sh;
      }
    } else {
#pragma unroll
      for (int u = 0; u < UQ; ++u) {
        const f32x4 v = *reinterpret_cast<const lds_f32x4*>(lq[u] + off);
        facc[u][0] = facc[u][0] + v.x;
        facc[u][1] = facc[u][1] + v.y;
        facc[u][2] = facc[u][2] + v.z;
        facc[u][3] = facc[u][3] + v.w;
      }
    }
  }
}

// One tree walk with the codebook's 15 thresholds in registers, passed as 15
// scalars (an array or struct would let the compiler turn a select between
// two elements into one dynamically indexed load and push it to scratch).
// The four compared values are independent loads; each level's threshold is
// selected by the decisions above it, with no memory access.
#define MDN_TREE_PARAMS float t0, float t1, float t2, float t3, float t4, float t5, float t6, \
  float t7, float t8, float t9, float t10, float t11, float t12, float t13, float t14
#define MDN_TREE_ARGS t0, t1, t2, t3, t4, t5, t6, t7, t8, t9, t10, t11, t12, t13, t14
__device__ __forceinline__ int tree_walk(float x0, float x1, float x2, float x3, MDN_TREE_PARAMS) {
  const bool b0 = x0 > t0;
  const bool b1 = x1 > (b0 ? t2 : t1);
  const float v2 = b0 ? (b1 ? t6 : t5) : (b1 ? t4 : t3);
  const bool b2 = x2 > v2;
  const float lo = b1 ? (b2 ? t10 : t9) : (b2 ? t8 : t7);
  const float hi = b1 ? (b2 ? t14 : t13) : (b2 ? t12 : t11);
  const bool b3 = x3 > (b0 ? hi : lo);
  return ((int)b0 << 3) | ((int)b1 << 2) | ((int)b2 << 1) | (int)b3;
}

template <int MODE, int ELEM, int PF, int UQ>
__global__ void __launch_bounds__(512) path_kernel(const KArgs a) {
  constexpr bool kEnc = MODE != kAccum;
  constexpr bool kAcc = MODE != kEncode;
  constexpr int kQB = ELEM == kI8 ? 4 : 16;  // bytes of one 4-column quad of a LUT row
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  lds_t* smem = (lds_t*)smem_raw;

  // The argument block lives in memory; read where first used, its fields
  // arrive in several dependent scalar-load rounds ahead of the first data
  // load.  Pinning them all here issues every scalar load at once and waits
  // once.
#define MDN_PIN(x) asm volatile("" ::"s"(x))
  MDN_PIN(a.A); MDN_PIN(a.idx_in); MDN_PIN(a.split); MDN_PIN(a.thr); MDN_PIN(a.lut);
  MDN_PIN(a.scale); MDN_PIN(a.offset); MDN_PIN(a.y); MDN_PIN(a.acc); MDN_PIN(a.idx_out);
  MDN_PIN(a.N); MDN_PIN(a.lda); MDN_PIN(a.D); MDN_PIN(a.C); MDN_PIN(a.M); MDN_PIN(a.Mt);
  MDN_PIN(a.lut_rs); MDN_PIN(a.Dp); MDN_PIN(a.Cp); MDN_PIN(a.RW); MDN_PIN(a.rw_log2);
  MDN_PIN(a.nchunks); MDN_PIN(a.c_magic); MDN_PIN(a.vec_out); MDN_PIN(a.enc_reg); MDN_PIN(a.c_log2);
  MDN_PIN(a.L.lut); MDN_PIN(a.L.thr); MDN_PIN(a.L.split); MDN_PIN(a.L.misc); MDN_PIN(a.L.sh);
  MDN_PIN(a.L.shp); MDN_PIN(a.L.a); MDN_PIN(a.L.a_wave); MDN_PIN(a.L.idx); MDN_PIN(a.L.idx_wave);
  MDN_PIN(blockDim.x); MDN_PIN(gridDim.x);
#undef MDN_PIN

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = uniform(tid >> 6);   // wavefront-uniform: loop control stays scalar
  const int nw = blockDim.x >> 6;
  const int C = a.C;
  const int m0 = blockIdx.y * a.Mt;
  const int mt = min(a.Mt, a.M - m0);   // columns of this tile
  const int nq = (mt + 3) >> 2;         // column quads of this tile

  lds_t* s_lut = smem + a.L.lut;
  lds_f32* s_thr = reinterpret_cast<lds_f32*>(smem + a.L.thr);
  lds_i32* s_split = reinterpret_cast<lds_i32*>(smem + a.L.split);
  lds_i32* s_misc = reinterpret_cast<lds_i32*>(smem + a.L.misc);
  lds_i32* s_sh = reinterpret_cast<lds_i32*>(smem + a.L.sh);
  lds_t* s_shp = smem + a.L.shp;

  // ---------------- the first chunk's rows, in flight during the prologue
  const int RW = a.RW;
  lds_t* sA = smem + a.L.a + wave * a.L.a_wave;
  lds_t* sI = smem + a.L.idx + wave * a.L.idx_wave;
  const int64_t tw = (int64_t)gridDim.x * nw;
  int64_t ch = (int64_t)blockIdx.x * nw + wave;

  // source rows of this mode: rows of A (encode) or of idx (accumulate)
  const char* src0 = kEnc ? reinterpret_cast<const char*>(a.A) : reinterpret_cast<const char*>(a.idx_in);
  const int64_t src_rs = kEnc ? a.lda * 4 : (int64_t)C;  // bytes between rows
  Prefetch<PF, kEnc> pf;
  if (PF > 0) {
    if (kEnc) pf.init(lane, RW, a.D >> 2, src_rs, a.Dp * 4, RW * a.Dp * 4);
    else      pf.init(lane, RW, C >> 4, src_rs, a.Cp, RW * a.Cp);
    if (ch < a.nchunks) {
      const int64_t row0 = ch << a.rw_log2;
      pf.load(src0 + row0 * src_rs, (int)min<int64_t>(RW, a.N - row0), RW, (int)src_rs);
    }
  }

  // the first round of the parameter loads below, issued before anything waits
  const uint32_t* sb = reinterpret_cast<const uint32_t*>(a.scale);
  float thr0 = 0.0f, off0 = 0.0f;
  int split0 = 0;
  uint32_t sb0 = 0u;
  if (kEnc) {
    if (tid < C * 16 && (tid & 15) < kNodes) thr0 = a.thr[(tid >> 4) * kNodes + (tid & 15)];
    if (tid < C * kLevels) split0 = a.split[tid];
  }
  if (kAcc && ELEM == kI8) {
    sb0 = sb[min(lane, C - 1)];
    if (wave == 0) off0 = a.offset[min(lane, C - 1)];
  }

  // ---------------- workgroup prologue ----------------
  // Table staging: 8 LDS dwords per thread per round with every global load
  // issued first (clamped addresses, masked afterwards), so a round costs one
  // memory latency instead of eight.
  if (kAcc) {
    const int rows = C * kK;
    const int wpr = (ELEM == kI8) ? nq : 4 * nq;   // LDS dwords per table row
    int wlog = 0;
    while ((1 << wlog) < wpr) ++wlog;
    const int total = rows << wlog;
    const int8_t* q8 = reinterpret_cast<const int8_t*>(a.lut);
    const float* qf = reinterpret_cast<const float*>(a.lut);
    const int64_t last = (int64_t)rows * a.M - 1;
    // one round: NJ LDS dwords per thread, starting at element `base`
    auto stage_round = [&](int base, auto nj_tag) {
      constexpr int NJ = decltype(nj_tag)::value;
      uint32_t v[NJ];
      // (one branch around each whole round, so that its loads are issued back
      // to back: a branch per element made the compiler wait after each one)
      auto e0_of = [&](int j, int& w) {
        const int u = base + j * blockDim.x;
        const int row = u >> wlog;
        w = u & ((1 << wlog) - 1);
        return (int64_t)row * a.M + m0;
      };
      if (ELEM == kF32) {
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          int w;
          const int64_t e0 = e0_of(j, w);
          v[j] = __float_as_uint(qf[min(e0 + w, last)]);
        }
      } else {
        // four columns per load, unaligned when M % 4 != 0 (the memory system
        // serves unaligned dwords); a dword that would run past the table is
        // read from its last four bytes and shifted down
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          int w;
          const int64_t e = e0_of(j, w) + 4 * w;
          const int64_t p = min(e, last - 3);
          const int sh = (int)min<int64_t>(e - p, 3);
          v[j] = *reinterpret_cast<const u32_ua*>(q8 + p) >> (8 * sh);
        }
      }
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int u = base + j * blockDim.x;
        const int row = u >> wlog, w = u & ((1 << wlog) - 1);
        if (u >= total || w >= wpr) continue;
        uint32_t x;
        if (ELEM == kF32) {
          x = w < mt ? v[j] : 0u;
        } else {
          const int live = min(mt - 4 * w, 4);   // columns of this dword inside the tile
          x = live >= 4 ? v[j] : v[j] & ((1u << (8 * live)) - 1u);
        }
        *reinterpret_cast<lds_u32*>(s_lut + row * a.lut_rs + 4 * w) = x;
      }
    };
    // (the first round outside the loop, as straight-line code: at a loop
    // header the compiler's wait analysis waited for every load in flight,
    // the first chunk's rows included, before the table's loads were issued;
    // a table of at most one dword per thread takes a one-load round)
    if (total <= (int)blockDim.x) {
      if (tid < total) stage_round(tid, std::integral_constant<int, 1>());
    } else {
      if (tid < total) stage_round(tid, std::integral_constant<int, 8>());
      for (int base = tid + 8 * blockDim.x; base < total; base += 8 * blockDim.x)
        stage_round(base, std::integral_constant<int, 8>());
    }
  }
  if (kEnc) {
    // node-major [16][C] thresholds and level-major [4][C] split columns:
    // lanes walking consecutive codebooks read consecutive banks at any node
    // (the first round from the registers loaded at entry, the rest from memory)
    if (tid < C * 16) s_thr[(tid & 15) * C + (tid >> 4)] = thr0;
    for (int u = tid + blockDim.x; u < C * 16; u += blockDim.x) {
      const int c = u >> 4, j = u & 15;
      s_thr[j * C + c] = (j < kNodes) ? a.thr[c * kNodes + j] : 0.0f;
    }
    if (tid < C * kLevels) s_split[(tid & 3) * C + (tid >> 2)] = (int)min((unsigned)split0, (unsigned)(a.D - 1));
    for (int u = tid + blockDim.x; u < C * kLevels; u += blockDim.x) {
      const unsigned sp = (unsigned)a.split[u];
      s_split[(u & 3) * C + (u >> 2)] = (int)min(sp, (unsigned)(a.D - 1));  // memory safety only
    }
  }
  // block exponents: every wavefront reduces e_min and the largest shift over
  // the scales itself (no barrier); wave 0 also sums the offsets
  int emin = 0, maxsh = 0;
  if (kAcc && ELEM == kI8) {
    int lo = INT_MAX, hi = INT_MIN;
    if (lane < C) lo = hi = exp_of_bits(sb0);
    for (int c = lane + 64; c < C; c += 64) {
      const int e = exp_of_bits(sb[c]);
      lo = min(lo, e);
      hi = max(hi, e);
    }
    wave_minmax(lo, hi);
    emin = lo;
    maxsh = hi - emin;
    if (wave == 0 && lane < C) s_sh[lane] = exp_of_bits(sb0) - emin;
    for (int c = tid + 64; c < C; c += blockDim.x) s_sh[c] = exp_of_bits(sb[c]) - emin;
    // shifts packed as nibbles, 8 codebooks per dword (used while every shift
    // <= 6): up to 64 codebooks from wave 0's registers (an OR over each 8
    // lanes, every lane taking part), more from memory
    if (C <= 64) {
      if (wave == 0) {
        // (DPP: quad butterflies, then lane 8k + 4 takes lane 8k's quad by a
        // row shift, so it holds the OR of lanes 8k .. 8k + 7)
        uint32_t w = lane < C ? (uint32_t)min(exp_of_bits(sb0) - emin, 15) << (4 * (lane & 7)) : 0u;
        w |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)w, 0xB1, 0xf, 0xf, true);
        w |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)w, 0x4E, 0xf, 0xf, true);
        w |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)w, 0x114, 0xf, 0xf, true);   // row_shr 4
        if ((lane & 7) == 4 && lane - 4 < C) *reinterpret_cast<lds_u32*>(s_shp + 4 * (lane >> 3)) = w;
      }
    } else {
      for (int g = tid; g < (C + 7) / 8; g += blockDim.x) {
        uint32_t w = 0;
        for (int b = 0; b < 8 && 8 * g + b < C; ++b) w |= (uint32_t)min(exp_of_bits(sb[8 * g + b]) - emin, 15) << (4 * b);
        *reinterpret_cast<lds_u32*>(s_shp + 4 * g) = w;
      }
    }
    if (wave == 0) {
      // bias32: double sum over codebooks in ascending order, 64 offsets per
      // coalesced load, summed in order through readlane (all lanes alike)
      double sum = 0.0;
      for (int j0 = 0; j0 < C; j0 += 64) {
        const float ov = j0 == 0 ? off0 : a.offset[min(j0 + lane, C - 1)];
        const int n = min(64, C - j0);
        for (int l = 0; l < n; ++l) sum += (double)__int_as_float(__builtin_amdgcn_readlane(__float_as_int(ov), l));
      }
      if (lane == 0) s_misc[2] = __float_as_int((float)sum);
    }
  }
  __syncthreads();

  // ---------------- per-wavefront chunk loop ----------------
  // accumulate-phase lane mapping
  const int lpr_log2 = 6 - a.rw_log2;
  const int ar = lane >> lpr_log2;                  // row of the chunk
  const int cg = lane & ((1 << lpr_log2) - 1);      // first column quad
  const int LPR = 1 << lpr_log2;
  const lds_t* lq[UQ];
#pragma unroll
  for (int u = 0; u < UQ; ++u) lq[u] = s_lut + min(cg + u * LPR, nq - 1) * kQB;
  // register-resident tree: when C divides 64, lane l always handles
  // codebook l % C of rows l / C + j * (64 / C), j < RW * C / 64
  float t0 = 0, t1 = 0, t2 = 0, t3 = 0, t4 = 0, t5 = 0, t6 = 0, t7 = 0, t8 = 0, t9 = 0, t10 = 0,
        t11 = 0, t12 = 0, t13 = 0, t14 = 0;
  int sc0 = 0, sc1 = 0, sc2 = 0, sc3 = 0;
  int cl = 0, er0 = 0, erstep = 1, enr = 0;
  if (kEnc && a.enc_reg == 1) {
    cl = lane & (C - 1);
    er0 = lane >> a.c_log2;
    erstep = 64 >> a.c_log2;
    enr = (RW * C) >> 6;
    const lds_f32* th = s_thr + cl;
    t0 = th[0]; t1 = th[C]; t2 = th[2 * C]; t3 = th[3 * C]; t4 = th[4 * C]; t5 = th[5 * C];
    t6 = th[6 * C]; t7 = th[7 * C]; t8 = th[8 * C]; t9 = th[9 * C]; t10 = th[10 * C];
    t11 = th[11 * C]; t12 = th[12 * C]; t13 = th[13 * C]; t14 = th[14 * C];
    sc0 = s_split[cl];
    sc1 = s_split[C + cl];
    sc2 = s_split[2 * C + cl];
    sc3 = s_split[3 * C + cl];
  }
  float step = 1.0f, bias = 0.0f;
  if (kAcc && ELEM == kI8) {
    bias = __int_as_float(uniform(s_misc[2]));
    step = __builtin_ldexpf(1.0f, emin);
  }

  for (; ch < a.nchunks; ch += tw) {
    const int64_t row0 = ch << a.rw_log2;
    const int rows_valid = (int)min<int64_t>(RW, a.N - row0);

    // 1. stage this chunk's rows in LDS, start loading the next chunk (at
    // raised wavefront priority: a wavefront whose rows have arrived issues
    // its next loads ahead of the other wavefronts' walks and sums)
    if (PF > 0) {
      __builtin_amdgcn_s_setprio(2);
      pf.store(kEnc ? sA : sI);
      const int64_t nx = ch + tw;
      if (nx < a.nchunks) {
        const int64_t nrow0 = nx << a.rw_log2;
        pf.load(src0 + nrow0 * src_rs, (int)min<int64_t>(RW, a.N - nrow0), RW, (int)src_rs);
      }
      __builtin_amdgcn_s_setprio(0);
    } else if (kEnc) {
      for (int r = 0; r < rows_valid; ++r) {
        const float* src = a.A + (row0 + r) * a.lda;
        for (int col = lane; col < a.D; col += 64)
          reinterpret_cast<lds_f32*>(sA)[r * a.Dp + col] = src[col];
      }
    } else {
      for (int r = 0; r < rows_valid; ++r) {
        const uint8_t* src = a.idx_in + (row0 + r) * (int64_t)C;
        for (int col = lane; col < C; col += 64) sI[r * a.Cp + col] = src[col];
      }
    }
    wave_sync();

    // 2. encode: 4 comparisons per (row, codebook)
    if (kEnc && a.enc_reg == 1) {
      const lds_f32* xa = reinterpret_cast<const lds_f32*>(sA);
      for (int j = 0; j < enr; j += 2) {  // two rows per step: 8 independent loads
        const int ra = er0 + j * erstep;
        const int rb = er0 + min(j + 1, enr - 1) * erstep;
        const lds_f32* pa = xa + ra * a.Dp;
        const lds_f32* pb = xa + rb * a.Dp;
        const float a0 = pa[sc0], a1 = pa[sc1], a2 = pa[sc2], a3 = pa[sc3];
        const float b0 = pb[sc0], b1 = pb[sc1], b2 = pb[sc2], b3 = pb[sc3];
        sI[ra * a.Cp + cl] = (uint8_t)tree_walk(a0, a1, a2, a3, MDN_TREE_ARGS);
        const int ib = tree_walk(b0, b1, b2, b3, MDN_TREE_ARGS);
        if (j + 1 < enr) sI[rb * a.Cp + cl] = (uint8_t)ib;
      }
    } else if (kEnc && a.enc_reg == 2) {
      // C a multiple of 64: lane l walks codebooks l, l + 64, ... for every
      // row of the chunk, with that codebook's tree and split columns in
      // registers (two rows per step: 8 independent loads)
      const lds_f32* xa = reinterpret_cast<const lds_f32*>(sA);
      for (int cb = lane; cb < C; cb += 64) {
        const lds_f32* th = s_thr + cb;
        const float u0 = th[0], u1 = th[C], u2 = th[2 * C], u3 = th[3 * C], u4 = th[4 * C], u5 = th[5 * C],
                    u6 = th[6 * C], u7 = th[7 * C], u8 = th[8 * C], u9 = th[9 * C], u10 = th[10 * C],
                    u11 = th[11 * C], u12 = th[12 * C], u13 = th[13 * C], u14 = th[14 * C];
        const int q0 = s_split[cb], q1 = s_split[C + cb], q2 = s_split[2 * C + cb], q3 = s_split[3 * C + cb];
        for (int r = 0; r < RW; r += 2) {
          const int rb = min(r + 1, RW - 1);
          const lds_f32* pa = xa + r * a.Dp;
          const lds_f32* pb = xa + rb * a.Dp;
          const float a0 = pa[q0], a1 = pa[q1], a2 = pa[q2], a3 = pa[q3];
          const float b0 = pb[q0], b1 = pb[q1], b2 = pb[q2], b3 = pb[q3];
          sI[r * a.Cp + cb] = (uint8_t)tree_walk(a0, a1, a2, a3, u0, u1, u2, u3, u4, u5, u6, u7, u8, u9, u10, u11,
                                                 u12, u13, u14);
          const int ib = tree_walk(b0, b1, b2, b3, u0, u1, u2, u3, u4, u5, u6, u7, u8, u9, u10, u11, u12, u13, u14);
          if (r + 1 < RW) sI[rb * a.Cp + cb] = (uint8_t)ib;
        }
      }
    } else if (kEnc) {
      // four independent walks per lane at a time, level by level, so their
      // dependent threshold reads overlap; (row, codebook) pairs past the
      // chunk repeat the lane's first pair and are not stored
      const lds_f32* xa = reinterpret_cast<const lds_f32*>(sA);
      const int npair = RW * C;
      for (int p0 = lane; p0 < npair; p0 += 256) {
        int i[4], c[4], r[4];
        const lds_f32* xr[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int p = (p0 + 64 * q < npair) ? p0 + 64 * q : p0;
          r[q] = (C == 1) ? p : (int)__umulhi((uint32_t)p, a.c_magic);
          c[q] = p - r[q] * C;
          xr[q] = xa + r[q] * a.Dp;
          i[q] = (xr[q][s_split[c[q]]] > s_thr[c[q]]) ? 1 : 0;
        }
#pragma unroll
        for (int t = 1; t < kLevels; ++t)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            i[q] = 2 * i[q] + ((xr[q][s_split[t * C + c[q]]] > s_thr[((1 << t) - 1 + i[q]) * C + c[q]]) ? 1 : 0);
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (p0 + 64 * q < npair) sI[r[q] * a.Cp + c[q]] = (uint8_t)i[q];
      }
    }
    if (kEnc) {
      wave_sync();
      if (a.idx_out != nullptr) {
        if (a.Cp == C && ((reinterpret_cast<uintptr_t>(a.idx_out) & 3) == 0)) {
          uint32_t* dst = reinterpret_cast<uint32_t*>(a.idx_out + row0 * C);
          const lds_u32* s32 = reinterpret_cast<const lds_u32*>(sI);
          const int n32 = (rows_valid * C) >> 2;
          for (int u = lane; u < n32; u += 64) dst[u] = s32[u];
        } else {
          for (int r = 0; r < rows_valid; ++r)
            for (int c = lane; c < C; c += 64) a.idx_out[(row0 + r) * C + c] = sI[r * a.Cp + c];
        }
      }
    }

    // 3. accumulate + 4. epilogue
    if (kAcc) {
      const lds_t* ir = sI + ar * a.Cp;
      const int64_t row = row0 + ar;
      int iacc[UQ][4];
      float facc[UQ][4];
#pragma unroll
      for (int u = 0; u < UQ; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) { iacc[u][e] = 0; facc[u][e] = 0.0f; }
      if (ELEM == kI8) {
        if (maxsh <= 6)
          accumulate<ELEM, UQ, true>(ir, lq, C, a.lut_rs, s_shp, s_sh, iacc, facc);
        else
          accumulate<ELEM, UQ, false>(ir, lq, C, a.lut_rs, s_shp, s_sh, iacc, facc);
      } else {
        accumulate<ELEM, UQ, false>(ir, lq, C, a.lut_rs, s_shp, s_sh, iacc, facc);
      }
      if (ar < rows_valid) {
#pragma unroll
        for (int u = 0; u < UQ; ++u) {
          const int q = cg + u * LPR;
          if (q < nq) {
            const int mloc = 4 * q;
            float o[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
              o[e] = (ELEM == kI8) ? __builtin_fmaf((float)iacc[u][e], step, bias) : facc[u][e];
            float* yp = a.y ? a.y + row * a.M + m0 + mloc : nullptr;
            int32_t* ap = (ELEM == kI8 && a.acc) ? a.acc + row * a.M + m0 + mloc : nullptr;
            if (a.vec_out && mloc + 4 <= mt) {
              if (yp) __builtin_nontemporal_store((f32x4){o[0], o[1], o[2], o[3]}, reinterpret_cast<f32x4*>(yp));
              if (ap) __builtin_nontemporal_store((u32x4){(uint32_t)iacc[u][0], (uint32_t)iacc[u][1],
                                                          (uint32_t)iacc[u][2], (uint32_t)iacc[u][3]},
                                                  reinterpret_cast<u32x4*>(ap));
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                if (mloc + e < mt) {
                  if (yp) yp[e] = o[e];
                  if (ap) ap[e] = iacc[u][e];
                }
              }
            }
          }
        }
      }
    }
    wave_sync();  // the next iteration overwrites this wavefront's LDS buffers
  }
}

// ---------------------------------------------------------------------------
// Instantiation table.  pf: 16-byte units prefetched per lane per chunk
// (0 = synchronous generic staging); uq: column quads per lane.
#define MDN_PF_LIST(X, MODE, ELEM, UQ) \
  X(MODE, ELEM, 0, UQ) X(MODE, ELEM, 1, UQ) X(MODE, ELEM, 2, UQ) X(MODE, ELEM, 4, UQ) \
  X(MODE, ELEM, 8, UQ) X(MODE, ELEM, 9, UQ) X(MODE, ELEM, 16, UQ)

// Per (device, kernel, block, LDS size): the LDS attribute is raised once and
// the number of resident workgroups per CU is queried once (a full cache only
// means querying again).
int launch_prepare(const void* fn, int block, int lds, hipError_t* err) {
  struct Entry { int dev; const void* fn; int block, lds, n; };
  static Entry cache[256];
  static int used = 0;
  static std::mutex mu;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = -1;
  std::lock_guard<std::mutex> lock(mu);
  for (int i = 0; i < used; ++i)
    if (cache[i].dev == dev && cache[i].fn == fn && cache[i].block == block && cache[i].lds == lds) return cache[i].n;
  if (lds > 64 * 1024) {
    const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) { *err = e; return 0; }
  }
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, block, lds) != hipSuccess || n < 1) n = 1;
  if (used < 256) cache[used++] = Entry{dev, fn, block, lds, n};
  return n;
}

// Compute units of the current device, queried once per device.
int device_cus() {
  constexpr int kDevs = 64;
  static std::atomic<int> cus[kDevs] = {};
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = 0;
  if (dev >= 0 && dev < kDevs) {
    const int v = cus[dev].load();
    if (v != 0) return v;
  }
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1) n = 256;
  if (dev >= 0 && dev < kDevs) cus[dev].store(n);
  return n;
}

// The persistent grid never exceeds what is resident at once, so no wave of
// workgroups runs after the first has drained.
template <int MODE, int ELEM, int PF, int UQ>
static hipError_t launch_one(const KArgs& a, dim3 grid, dim3 block, hipStream_t stream) {
  const void* fn = reinterpret_cast<const void*>(&path_kernel<MODE, ELEM, PF, UQ>);
  hipError_t err = hipSuccess;
  const int per_cu = launch_prepare(fn, (int)block.x, a.L.total, &err);
  if (err != hipSuccess) return err;
  const int64_t resident = (int64_t)per_cu * device_cus();
  int64_t gx = (int64_t)grid.x;
  const int64_t cap = resident / (int64_t)grid.y;
  if (gx > cap) gx = cap > 0 ? cap : 1;
  grid.x = (unsigned)gx;
  hipLaunchKernelGGL((path_kernel<MODE, ELEM, PF, UQ>), grid, block, a.L.total, stream, a);
  return hipGetLastError();
}

#define MDN_CASE(MODE, ELEM, PF, UQ)                                         \
  if (mode == MODE && elem == ELEM && pf == PF && uq == UQ) {                \
    return launch_one<MODE, ELEM, PF, UQ>(a, grid, block, stream);           \
  }

hipError_t launch_path(int mode, int elem, int pf, int uq, const KArgs& a, dim3 grid, dim3 block,
                       hipStream_t stream) {
  // encode-only kernels ignore elem and uq
  if (mode == kEncode) { elem = kI8; uq = 1; }
  MDN_PF_LIST(MDN_CASE, kEncode, kI8, 1)
  MDN_PF_LIST(MDN_CASE, kFused, kI8, 1)
  MDN_PF_LIST(MDN_CASE, kFused, kI8, 2)
  MDN_PF_LIST(MDN_CASE, kFused, kI8, 4)
  MDN_PF_LIST(MDN_CASE, kFused, kF32, 1)
  MDN_PF_LIST(MDN_CASE, kFused, kF32, 2)
  MDN_PF_LIST(MDN_CASE, kFused, kF32, 4)
  MDN_PF_LIST(MDN_CASE, kAccum, kI8, 1)
  MDN_PF_LIST(MDN_CASE, kAccum, kI8, 2)
  MDN_PF_LIST(MDN_CASE, kAccum, kI8, 4)
  MDN_PF_LIST(MDN_CASE, kAccum, kF32, 1)
  MDN_PF_LIST(MDN_CASE, kAccum, kF32, 2)
  MDN_PF_LIST(MDN_CASE, kAccum, kF32, 4)
  return hipErrorInvalidValue;
}

}  // namespace mdn
