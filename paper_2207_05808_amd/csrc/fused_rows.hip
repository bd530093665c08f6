// Fused encode + lookup-accumulate for int8 tables of 64 codebooks with at
// most 512 output columns, for calls with many rows (§1, §2.1 of McCarter &
// Dronen: 4 comparisons per codebook encode a row; the product is the sum over
// codebooks of the selected table rows).  The table (64 x 16 x M bytes) is too
// large for LDS, so it streams through LDS 4 codebooks at a time, while HBM
// carries the rows of A in and the outputs out: the encode (HBM-bound) and the
// sums (LDS-bound) run in the same kernel, at the same time.
//
// One 1024-thread workgroup per CU owns a contiguous block of rows and runs a
// pipeline of steps, one barrier each.  Step g uses codebook tile g % 16
// (codebooks 4 (g % 16) .. + 3), staged in LDS buffer g % 2 as 16-bit
// offset-binary fields u = (q + 128) << (e_c - e_min), two columns per dword,
// in the lane-slot order of the row-uniform accumulate (lane l owns columns
// 4l..4l+3 and 256+4l..256+4l+3; slot permuted within each 256-byte span so
// that reads and staging writes cover all 64 banks).  While no 16-bit field
// can carry into the next (255 sum_c 2^(e_c - e_min) <= 65535) a plain 32-bit
// add sums two columns.
//
// Roles (wavefront-uniform):
//  * producers, wavefronts 0-3: at step g they write table tile (g + 1) % 16
//    into the other buffer (from registers loaded a step earlier) and load
//    tile (g + 2) % 16; and they encode the 12 rows that start at step g + 2
//    (lane = codebook; its 15 thresholds and 4 split columns in registers;
//    the 4 compared values gathered two steps ahead), writing the index bytes
//    to a ring of index rows in LDS (and to idx_out when the caller asks);
//  * consumers, wavefronts 4-15: each keeps 16 rows in flight, row slot j in
//    registers as 4 dwords of fields per lane.  A row in slot j starts at a
//    step g0 = j (mod 16) and takes tiles g0, g0 + 1, ... (mod 16): 16 steps,
//    every codebook once (integer sums commute).  At each step a consumer adds
//    the step's tile to its 16 rows (one 16-byte LDS read per lane per
//    codebook: the table row a codebook selects is uniform over the wavefront,
//    its index byte read from the ring), then retires slot (g + 1) % 16, whose
//    row has seen all 16 tiles: convert, layer output, store (2 KB), and the
//    slot starts a new row at the next step.  So each consumer retires and
//    starts one row per step (12 rows per step per workgroup) and the output
//    work is spread evenly over the steps.
// The first 15 steps fill the slots and the last 15 drain them.
//
// When the table's block exponents are too far apart for 16-bit fields the
// kernel only encodes: every row's 64 index bytes go to idx_out, or, when the
// caller gave none, to the first 64 bytes of the row's own output row (M >= 16
// floats).  The host always follows this kernel with the row-uniform
// accumulate in a mode that does nothing unless the fields did not fit; that
// kernel reads a row's indices before it writes the row.
#include "internal.hpp"

#include <climits>
#include <type_traits>

namespace mdn {

namespace {

typedef uint32_t fu32x4 __attribute__((ext_vector_type(4)));
typedef float ff32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char flds_t;
typedef __attribute__((address_space(3))) uint32_t flds_u32;
typedef __attribute__((address_space(3))) uint8_t flds_u8;
typedef __attribute__((address_space(3))) fu32x4 flds_u32x4;
typedef __attribute__((address_space(3))) ff32x4 flds_f32x4;
typedef __attribute__((address_space(3))) float flds_f32;

constexpr int kFBufDword3 = 0x00020000;   // raw, unswizzled buffer descriptor (gfx9 family)
constexpr int kFOob = INT_MAX;            // buffer offset past any descriptor range: reads zero
constexpr int kFProd = 4;                 // producer wavefronts
constexpr int kFCons = 12;                // consumer wavefronts = rows started per step
constexpr int kFTiles = 16;               // codebook tiles per row (64 codebooks / 4)
constexpr int kFRowBytes = 1024;          // LDS bytes of one staged table row (512 16-bit fields)
constexpr int kFTileBytes = 4 * 16 * kFRowBytes;   // one of the two tile buffers (64 KB)
constexpr int kFRowsPerProd = kFCons / kFProd;      // rows each producer encodes per step (3)
constexpr int kFDepth = 3;                // consumer table-read items in flight (2 reads each)
constexpr int kFRingStep = kFCons * 64 + 4;   // ring bytes per step: 12 rows of 64 indices, + 4 so that the
                                              // 16 slots' index words (different steps) hit different banks

__device__ __forceinline__ int funi(int v) { return __builtin_amdgcn_readfirstlane(v); }

// the step barrier, with nothing scheduled across it (the compiler would
// otherwise start converting the table tile just requested and wait for it
// before the barrier)
__device__ __forceinline__ void fstep_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  __syncthreads();
  __builtin_amdgcn_sched_barrier(0);
}

// a uniform value pinned to a scalar register (the compiler otherwise keeps
// some uniform floats in vector registers, which the consumers cannot spare).
// The s_nop gives the VALU write of the source register the wait states a
// v_readfirstlane needs before it reads that register: the compiler inserts
// them for its own instructions but cannot see into this asm.
__device__ __forceinline__ float fsgpr(float v) {
  float r;
  asm volatile("s_nop 4\n\tv_readfirstlane_b32 %0, %1" : "=s"(r) : "v"(v));
  return r;
}

// the lane id, recomputed where it is used (never hoisted into a live register)
__device__ __forceinline__ int flane() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// Leaf of the balanced 4-level tree: at level t the node is i (0 <= i < 2^t),
// its threshold is thresholds[2^t - 1 + i] (heap order); x_t > threshold
// (strict: ties and NaN go to 0) is the next bit, the root's the highest.
// (thresholds passed by value: selects of values, never of addresses)
struct FTree {
  float t0, t1, t2, t3, t4, t5, t6, t7, t8, t9, t10, t11, t12, t13, t14;
};
__device__ __forceinline__ int fwalk(float x0, float x1, float x2, float x3, const FTree T) {
  const bool b0 = x0 > T.t0;
  const bool b1 = x1 > (b0 ? T.t2 : T.t1);
  const float v2 = b0 ? (b1 ? T.t6 : T.t5) : (b1 ? T.t4 : T.t3);
  const bool b2 = x2 > v2;
  const float lo = b1 ? (b2 ? T.t10 : T.t9) : (b2 ? T.t8 : T.t7);
  const float hi = b1 ? (b2 ? T.t14 : T.t13) : (b2 ? T.t12 : T.t11);
  const bool b3 = x3 > (b0 ? hi : lo);
  return ((int)b0 << 3) | ((int)b1 << 2) | ((int)b2 << 1) | (int)b3;
}

template <int CTRL>
__device__ __forceinline__ float fdpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}

// max / sum over the 64 lanes, the same value in every lane (DPP within rows
// of 16 lanes, then the four row results through readlane)
template <bool MAX>
__device__ __forceinline__ float freduce64(float x) {
  auto op = [](float a, float b) { return MAX ? __builtin_fmaxf(a, b) : a + b; };
  x = op(x, fdpp<0xB1>(x));    // quad_perm [1,0,3,2]
  x = op(x, fdpp<0x4E>(x));    // quad_perm [2,3,0,1]
  x = op(x, fdpp<0x141>(x));   // row_half_mirror
  x = op(x, fdpp<0x140>(x));   // row_mirror
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return op(op(r0, r1), op(r2, r3));
}

}  // namespace

__global__ void __launch_bounds__(1024) fenc_kernel(const FArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  flds_t* smem = (flds_t*)smem_raw;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = funi(tid >> 6);
  const int M = a.M;
  const int64_t rb0 = (int64_t)blockIdx.x * a.rows_per_block;   // this workgroup's first row
  const int64_t left = a.N - rb0;
  if (left <= 0) return;   // uniform: no rows for this workgroup
  const int rows_b = (int)(left < a.rows_per_block ? left : a.rows_per_block);

  // ---------------- dequantization constants, computed by every wavefront
  // alone (lane l holds codebook l): e_min, shifts, sum of 2^sh, bias32
  const uint32_t sbits = __float_as_uint(a.scale[lane]);
  const int e_c = (int)((sbits >> 23) & 0xffu) - 127;
  int emin = e_c;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) emin = min(emin, __shfl_xor(emin, o));
  const int sh = min(e_c - emin, 30);
  int pw = sh <= 14 ? (1 << sh) : (1 << 15);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) pw += __shfl_xor(pw, o);
  const int S = funi(pw);                 // sum of 2^sh (saturated per codebook at 2^15)
  const bool fields = S <= 257;           // 255 * S <= 65535

  // the 15 thresholds and 4 split columns of codebook `lane` (clamped to
  // [0, D): memory safety only)
  auto load_tree = [&](FTree& T, int (&sp)[4]) {
    const float* th = a.thr + lane * 15;
    T = FTree{th[0], th[1], th[2], th[3], th[4], th[5], th[6], th[7], th[8], th[9], th[10], th[11], th[12], th[13],
              th[14]};
#pragma unroll
    for (int t = 0; t < 4; ++t) sp[t] = (int)min((unsigned)a.split[lane * 4 + t], (unsigned)(a.D - 1));
  };

  if (!fields) {
    // ---------------- encode only: each wavefront walks whole rows
    FTree T;
    int sp[4];
    load_tree(T, sp);
    for (int r = wave; r < rows_b; r += 16) {
      const int64_t row = rb0 + r;
      const float* Ar = a.A + row * a.lda;
      const int k = fwalk(Ar[sp[0]], Ar[sp[1]], Ar[sp[2]], Ar[sp[3]], T);
      uint8_t* dst = a.idx_out ? a.idx_out + row * 64 : reinterpret_cast<uint8_t*>(a.y + row * M);
      dst[lane] = (uint8_t)k;
    }
    return;
  }

  // bias32: double sum over codebooks in ascending order
  double bsum = 0.0;
  {
    const float ov = a.offset[lane];
#pragma unroll 8
    for (int j = 0; j < 64; ++j) bsum += (double)__int_as_float(__builtin_amdgcn_readlane(__float_as_int(ov), j));
  }
  const float bias32 = (float)bsum;
  const float step = __builtin_ldexpf(1.0f, emin);

  flds_t* s_tab = smem;                                   // two tile buffers, 64 KB each
  flds_t* s_ring = smem + a.off_ring;                     // [kFRing steps][12 rows][64 bytes] (+ 4 per step)
  flds_f32x4* s_bias = reinterpret_cast<flds_f32x4*>(smem + a.off_bias);
  if (a.bias_lds)   // column biases of the layer output, staged once
    for (int m = tid; m < M; m += 1024) reinterpret_cast<flds_f32*>(s_bias)[m] = a.col_bias[m];

  const int nsteps = (rows_b + kFCons - 1) / kFCons;   // steps at which rows start
  // + the steps that drain the last rows, rounded up to whole cycles of the 16
  // tiles (the consumer loop is unrolled over one cycle; extra steps start no rows)
  const int total = (nsteps + kFTiles - 1 + kFTiles - 1) / kFTiles * kFTiles;

  if (wave < kFProd) {
    // ======================================================= producers
    const int pw4 = wave;                 // 0..3
    const int ptid = tid;                 // 0..255
    const int tp = ptid & 15;             // 16 columns of each half of the slice
    const int trq = ptid >> 4;            // prototype (staged row within each codebook)
    FTree T;
    int sp[4];
    load_tree(T, sp);

    // ---- table tiles: thread (trq, tp) stages prototype trq of the tile's 4
    // codebooks, columns 16 tp.. of each 256-column half: 8 units of 16 bytes
    const __amdgpu_buffer_rsrc_t trs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(a.lut), 0, 64 * 16 * M, kFBufDword3);
    fu32x4 tv[4][2];
    auto load_tile = [&](int t) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int base = ((4 * t + j) * 16 + trq) * M + 16 * tp;
        asm volatile("" : "+v"(base));
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const bool ok = 256 * h + 16 * tp < M;   // M % 16 == 0: units are whole
          tv[j][h] = __builtin_amdgcn_raw_buffer_load_b128(trs, ok ? base + 256 * h : kFOob, 0, 0);
        }
      }
    };
    typedef unsigned short us2 __attribute__((ext_vector_type(2)));
    auto store_tile = [&](int t, int buf) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int shj = __builtin_amdgcn_readlane(sh, 4 * t + j);   // uniform: codebook 4 t + j
        const us2 s2 = {(unsigned short)shj, (unsigned short)shj};
        int base = buf * kFTileBytes + (j * 16 + trq) * kFRowBytes + tp * 64;
        asm volatile("" : "+v"(base));
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          uint32_t w[4];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const uint32_t u = tv[j][h][i] ^ 0x80808080u;   // q + 128 per byte
            // (shifted unconditionally: a select between shifted and unshifted
            // values costs more than the shift by 0 it would save)
            w[2 * h] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(us2, __builtin_amdgcn_perm(0u, u, 0x0c010c00u)) << s2);
            w[2 * h + 1] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(us2, __builtin_amdgcn_perm(0u, u, 0x0c030c02u)) << s2);
          }
          // lane 4 tp + i's slot sits at position 4 tp + (i + tp / 4) % 4
          *reinterpret_cast<flds_u32x4*>(s_tab + base + 16 * ((i + (tp >> 2)) & 3)) =
              (fu32x4){w[0], w[1], w[2], w[3]};
        }
      }
    };

    // ---- encode: rows starting at step s are local rows 12 s + k (k the
    // consumer); this wavefront walks k = 3 pw4 .. 3 pw4 + 2.  Rows past the
    // block lie past the descriptor's range and read zeros (a valid walk whose
    // result is never used); the host keeps every such offset below 2^31.
    const __amdgpu_buffer_rsrc_t ars = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(a.A + rb0 * a.lda), 0, (int)((int64_t)rows_b * a.lda * 4), kFBufDword3);
    // (the whole offset in the lane's VGPR offset, which the range check
    // covers; no select, so no branch and no wait on the loads in flight)
    const int ldab = (int)(a.lda * 4);
    auto gather = [&](int s, float (&x)[kFRowsPerProd][4]) {
#pragma unroll
      for (int q = 0; q < kFRowsPerProd; ++q) {
        const int rowoff = (kFCons * s + kFRowsPerProd * pw4 + q) * ldab;   // uniform
#pragma unroll
        for (int t = 0; t < 4; ++t)
          x[q][t] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ars, rowoff + 4 * sp[t], 0, 0));
        __builtin_amdgcn_sched_barrier(0);   // a row's 4 loads (the same cache lines) issued together
      }
    };
    auto walk_rows = [&](int s, const float (&x)[kFRowsPerProd][4]) {
      flds_u8* ring = reinterpret_cast<flds_u8*>(s_ring + (s % kFRing) * kFRingStep);
#pragma unroll
      for (int q = 0; q < kFRowsPerProd; ++q) {
        const int k = kFRowsPerProd * pw4 + q;
        const int leaf = fwalk(x[q][0], x[q][1], x[q][2], x[q][3], T);
        ring[k * 64 + lane] = (uint8_t)leaf;
        const int lr = kFCons * s + k;
        if (a.idx_out && lr < rows_b) a.idx_out[(rb0 + lr) * 64 + lane] = (uint8_t)leaf;
      }
    };

    float xa[kFRowsPerProd][4], xb[kFRowsPerProd][4];
    load_tile(0);
    gather(0, xa);
    gather(1, xb);
    store_tile(0, 0);
    load_tile(1);
    walk_rows(0, xa);
    walk_rows(1, xb);
    gather(2, xa);
    gather(3, xb);
    __syncthreads();   // tile 0, the index rows of steps 0 and 1, the bias row
    // step g: tile (g + 1) % 16 into buffer (g + 1) % 2 (its readers, step
    // g - 1, finished before the last barrier), load tile (g + 2) % 16, walk
    // the rows of step g + 2 (gathered at step g - 2), gather step g + 4's
    auto pstep = [&](int g, float (&x)[kFRowsPerProd][4]) {
      store_tile((g + 1) & (kFTiles - 1), (g + 1) & 1);
      load_tile((g + 2) & (kFTiles - 1));
      walk_rows(g + 2, x);
      gather(g + 4, x);
    };
    for (int g = 0; g < total; g += 2) {   // total is a multiple of 16
      pstep(g, xa);
      fstep_barrier();
      pstep(g + 1, xb);
      fstep_barrier();
    }
    return;
  }

  // ========================================================= consumers
  const int k = wave - kFProd;   // 0..11: the row this wavefront starts at each step
  // the lane's slot of staged row (c_local * 16 + p) of buffer b: position
  // (lane & ~3) + ((lane & 3) + lane / 16) % 4 of 16 bytes
  const uint32_t lane_slot =
      (uint32_t)(uintptr_t)(s_tab + 16 * ((lane & ~3) + (((lane & 3) + (lane >> 4)) & 3)));
  // index word (codebooks 4 (g % 16) .. + 3) of the row in slot jl = lane %
  // 16 at step g: that row started at step g - ((g - jl) % 16)
  auto ring_read = [&](int g) -> uint32_t {
    const int jl = flane() & 15;
    const int d = (g - jl) & (kFTiles - 1);
    int slot = (g % kFRing) - d;
    if (slot < 0) slot += kFRing;
    const int off = a.off_ring + slot * kFRingStep + k * 64 + 4 * (g & (kFTiles - 1));
    return *reinterpret_cast<const flds_u32*>(smem + off);
  };

  uint32_t acc[kFTiles][4];
#pragma unroll
  for (int j = 0; j < kFTiles; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[j][e] = 0u;

  const int off128 = 128 * S;
  const float st = fsgpr(step), bz = fsgpr(bias32);   // scalar registers for the whole loop
  // retire the row in slot U at step g: it started at step g - 15.  Outputs
  // go half by half (lane l: columns 4l..4l+3, then 256+4l..256+4l+3), so few
  // registers are needed beside the 16 slots.
  auto retire = [&](uint32_t (&ac)[4], int g, auto actc) {
    constexpr int ACT = decltype(actc)::value;
    constexpr bool SOFTMAX = ACT == 3;
    const int gs = g - (kFTiles - 1);
    const int lr = kFCons * gs + k;
    if (gs >= 0 && lr < rows_b) {   // uniform
      const int64_t row = rb0 + lr;
      const int l4 = 4 * flane();
      // output i (0..3) of half h: 16-bit field (i & 1) of dword 2 h + i / 2
      auto outs = [&](int h, int (&o)[4]) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t w = ac[2 * h + (i >> 1)];
          o[i] = (int)((i & 1) ? (w >> 16) : (w & 0xffffu)) - off128;
        }
      };
      auto zs = [&](int h, float (&z)[4]) {   // y, then the layer output's bias and ReLU
        int o[4];
        outs(h, o);
        const int col = l4 + 256 * h;
        ff32x4 b4 = {0.0f, 0.0f, 0.0f, 0.0f};
        if (ACT != 0 && a.bias_lds && col < M) b4 = s_bias[col >> 2];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = __builtin_fmaf((float)o[i], st, bz);
          if (ACT != 0) {
            v = v + b4[i];
            if (ACT == 2) v = (v > 0.0f) ? v : 0.0f;
          }
          z[i] = v;
        }
      };
      if (SOFTMAX) {
        // row softmax: the whole row is in this wavefront
        float vmax = -__builtin_inff();
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          float z[4];
          zs(h, z);
          if (l4 + 256 * h < M)
#pragma unroll
            for (int i = 0; i < 4; ++i) vmax = __builtin_fmaxf(vmax, z[i]);
        }
        vmax = freduce64<true>(vmax);
        float sum = 0.0f;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          float z[4];
          zs(h, z);
          if (l4 + 256 * h < M)
#pragma unroll
            for (int i = 0; i < 4; ++i) sum += expf(z[i] - vmax);
        }
        const float rs = 1.0f / freduce64<false>(sum);   // correctly rounded reciprocal, then products
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int col = l4 + 256 * h;
          if (col >= M) continue;
          float z[4];
          zs(h, z);
          __builtin_nontemporal_store((ff32x4){expf(z[0] - vmax) * rs, expf(z[1] - vmax) * rs,
                                               expf(z[2] - vmax) * rs, expf(z[3] - vmax) * rs},
                                      reinterpret_cast<ff32x4*>(a.y + row * M + col));
        }
      } else {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int col = l4 + 256 * h;
          if (col >= M) continue;
          float z[4];
          zs(h, z);
          __builtin_nontemporal_store((ff32x4){z[0], z[1], z[2], z[3]}, reinterpret_cast<ff32x4*>(a.y + row * M + col));
        }
      }
      if (a.acc) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int col = l4 + 256 * h;
          if (col >= M) continue;
          int o[4];
          outs(h, o);
          __builtin_nontemporal_store((fu32x4){(uint32_t)o[0], (uint32_t)o[1], (uint32_t)o[2], (uint32_t)o[3]},
                                      reinterpret_cast<fu32x4*>(a.acc + row * M + col));
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) ac[e] = 0u;
  };

  __syncthreads();   // tile 0, the index rows of steps 0 and 1, the bias row
  uint32_t vi = ring_read(0);
  // step g = g0 + u of one cycle: tile u in buffer u % 2; slot (u + 1) % 16
  // retires (u a compile-time constant: every slot index is static)
  auto cstep = [&](int g, auto uc, auto actc) {
    constexpr int u = decltype(uc)::value;
    uint32_t d[kFTiles];   // index words of the 16 slots' rows (uniform)
#pragma unroll
    for (int j = 0; j < kFTiles; ++j) d[j] = __builtin_amdgcn_readlane(vi, j);
    vi = ring_read(g + 1);   // next step's words: every row they name is already in the ring
    uint32_t lane_buf = lane_slot + (u & 1) * kFTileBytes;
    asm volatile("" : "+v"(lane_buf));
    auto slot_of = [&](int cb, int p) -> const flds_t* {
      uint32_t adr;
      asm("v_lshl_add_u32 %0, %1, 10, %2" : "=v"(adr) : "s"(p), "v"(lane_buf));
      return (const flds_t*)(uintptr_t)adr + cb * 16 * kFRowBytes;
    };
    // items i = (codebook pair cp = 2 (i / 16), slot j = i % 16), software
    // pipelined kFDepth deep: the reads of items i + 1 .. i + kFDepth - 1 are
    // in flight while item i is summed (12 consumer wavefronts need about 6
    // KB each in flight to cover the LDS latency)
    constexpr int NI = 2 * kFTiles;
    fu32x4 v0[kFDepth], v1[kFDepth];
    auto rd = [&](int i, fu32x4& x0, fu32x4& x1) {
      const int cp = 2 * (i / kFTiles);
      const uint32_t dw = d[i % kFTiles];
      x0 = *reinterpret_cast<const flds_u32x4*>(slot_of(cp, (dw >> (8 * cp)) & 15));
      x1 = *reinterpret_cast<const flds_u32x4*>(slot_of(cp + 1, (dw >> (8 * cp + 8)) & 15));
    };
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < kFDepth - 1; ++i) rd(i, v0[i], v1[i]);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      __builtin_amdgcn_sched_barrier(0);
      if (i + kFDepth - 1 < NI) rd(i + kFDepth - 1, v0[(i + kFDepth - 1) % kFDepth], v1[(i + kFDepth - 1) % kFDepth]);
      __builtin_amdgcn_sched_barrier(0);
      const int j = i % kFTiles;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[j][e] += v0[i % kFDepth][e] + v1[i % kFDepth][e];
        asm("" : "+v"(acc[j][e]));   // opaque: no reassociation across codebook pairs
      }
    }
    retire(acc[(u + 1) & (kFTiles - 1)], g, actc);
    fstep_barrier();
  };
  // one copy of the loop per layer output, so the running loop holds only its own
  auto cycles = [&](auto actc) {
    for (int g0 = 0; g0 < total; g0 += kFTiles) {
#define MDN_CSTEP(U) cstep(g0 + U, std::integral_constant<int, U>{}, actc);
      MDN_CSTEP(0) MDN_CSTEP(1) MDN_CSTEP(2) MDN_CSTEP(3) MDN_CSTEP(4) MDN_CSTEP(5) MDN_CSTEP(6) MDN_CSTEP(7)
      MDN_CSTEP(8) MDN_CSTEP(9) MDN_CSTEP(10) MDN_CSTEP(11) MDN_CSTEP(12) MDN_CSTEP(13) MDN_CSTEP(14) MDN_CSTEP(15)
#undef MDN_CSTEP
    }
  };
  switch (a.act) {
    case 0: cycles(std::integral_constant<int, 0>{}); break;
    case 1: cycles(std::integral_constant<int, 1>{}); break;
    case 2: cycles(std::integral_constant<int, 2>{}); break;
    default: cycles(std::integral_constant<int, 3>{}); break;
  }
}

hipError_t launch_fenc(const FArgs& f, int blocks, hipStream_t stream) {
  hipError_t err = hipSuccess;
  launch_prepare(reinterpret_cast<const void*>(&fenc_kernel), 1024, f.lds_total, &err);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(fenc_kernel, dim3((unsigned)blocks), dim3(1024), f.lds_total, stream, f);
  return hipGetLastError();
}

}  // namespace mdn
