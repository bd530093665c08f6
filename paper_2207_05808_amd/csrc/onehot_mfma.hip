// Lookup-accumulate as an int8 matrix product on the matrix cores.
//
// The encoder's output for a row is the concatenation of C one-hot vectors of
// length 16 (§2.2 of McCarter & Dronen), and the lookup-accumulate is the
// product of that 0/1 row with the stacked tables (§1: the sum over codebooks
// of the selected table rows).  For int8 tables in block floating point the
// exact integer sum is acc = sum_c 2^sh_c q_c[idx_c] with sh_c = e_c - e_min;
// with the one-hot entry of codebook c set to 2^sh_c instead of 1, acc is one
// int8 x int8 -> int32 product over K = 16 C, which the matrix cores compute
// exactly (int32 wraps only past the documented bound, and every partial sum
// obeys the same bound).  One-hot entries must fit int8, so the codebooks
// are taken in shift groups of width 7 (2^0 .. 2^6), the highest group
// first, with the sums shifted left by 7 between groups: a table whose shifts
// are all below 7 (the common case) takes one pass.
//
// Sparse products.  A one-hot operand has at most one nonzero in every group
// of 4 consecutive K values, so it is 2:4 sparse, and the sparse product
// v_smfmac_i32_32x32x64_i8 covers 64 K values (4 codebooks) in about the time
// of one 32-value dense product: the one-hot operand goes as the compressed
// sparse operand (two stored values and their 2-bit positions per group,
// built in registers from the index bytes), the table as the dense one.
//
// Why the matrix cores: summed by gathers, each lookup reads 2 bytes of LDS
// (a 16-bit field per column), and on layers with hundreds of output columns
// the LDS, not HBM, sets the time.  The products do 8 times the arithmetic of
// the gathers but on units that are otherwise idle, and read the table from
// LDS once per 64 rows.
//
// Layout.  A workgroup (8 wavefronts) owns one column slice of W = 32 WB
// columns for its lifetime, staged once into LDS transposed, as [codebook]
// [column][16 prototypes] bytes, so the table operand of a product (32
// columns x 64 K values) is two 16-byte reads per lane.  Each wavefront takes
// tiles of 64 rows (two 32-row blocks) of the workgroup's row range
// independently (no barrier after the prologue): per 4 codebooks it reads WB
// table operands one step ahead, builds the compressed one-hot operands of
// its two row blocks, and issues 2 WB products.  Index rows come in 8-byte
// chunks, each reloaded with the next tile's as soon as its last product step
// has been issued.  Results come out with the columns across the lanes and
// the rows in registers; y = fmaf(float(acc), 2^e_min, bias32) (the offsets'
// double sum, codebooks ascending, rounded once), then the layer output's
// bias and ReLU, and dword streaming stores, each writing two whole 128-byte
// row segments.
//
// Workgroups are numbered so that the slices of one row group run on one XCD,
// or on as few as the group's slices fill (block b runs on XCD b % 8): the
// index rows of a group are read into one or two L2s, not eight.
#include "internal.hpp"

#include <climits>
#include <type_traits>
#include <utility>

namespace mdn {

namespace {

typedef int32_t mi32x4 __attribute__((ext_vector_type(4)));
typedef int32_t mi32x8 __attribute__((ext_vector_type(8)));
typedef int32_t mi32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t mu32x2 __attribute__((ext_vector_type(2)));
typedef float mf32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char mlds_t;
typedef __attribute__((address_space(3))) mi32x4 mlds_i32x4;
typedef __attribute__((address_space(3))) mu32x2 mlds_u32x2;
typedef __attribute__((address_space(3))) uint32_t mlds_u32;
typedef __attribute__((address_space(3))) uint8_t mlds_u8;
typedef __attribute__((address_space(3))) int32_t mlds_i32;
typedef __attribute__((address_space(3))) float mlds_f32;
typedef __attribute__((address_space(3))) mf32x4 mlds_f32x4;

constexpr int kMWaves = 8;      // wavefronts per workgroup
constexpr int kMTileRows = 64;  // rows per wavefront tile: two blocks of 32
constexpr int kMGroupBits = 7;  // one-hot entries 2^0 .. 2^6 fit int8
constexpr int kMBufDword3 = 0x00020000;   // raw, unswizzled buffer descriptor (gfx9 family)
static_assert(30 / 7 + 1 <= kMaccGroups, "shifts up to 30 (clamped, as everywhere) in whole groups of 7");

__device__ __forceinline__ int muni(int v) { return __builtin_amdgcn_readfirstlane(v); }

// f(integral_constant<int, I>) for I = 0, 1, ..., in order, unrolled
template <typename F, int... I>
__device__ __forceinline__ void mfor(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}

// 4 x 4 transpose of dwords over the four lanes of every quad: dword e of
// lane u on entry is dword u of lane e on return (the same two stages)
__device__ __forceinline__ void mquad_transpose_dw(mi32x4& x, int lane) {
  const int b0 = lane & 1, b1 = (lane >> 1) & 1;
  mi32x4 z;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int v = __builtin_amdgcn_mov_dpp(x[e ^ 1], 0xB1, 0xf, 0xf, false);
    z[e] = b0 == (e & 1) ? x[e] : v;
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int v = __builtin_amdgcn_mov_dpp(z[e ^ 2], 0x4E, 0xf, 0xf, false);
    x[e] = b1 == ((e >> 1) & 1) ? z[e] : v;
  }
}

// The 2:4-compressed one-hot operand of a codebook: its 16 prototypes in
// groups of 4, two stored values per group, each with a 2-bit position.  The
// group x / 4 holding prototype x stores (v, 0) at positions (x % 4, x % 4 +
// 1 mod 4), the other groups (0, 0) at positions (0, 1).  So the stored
// values are v at byte 2 (x / 4) of the codebook's 8 bytes, and the position
// bits 0x4444 ^ (d(x % 4) << 4 (x / 4)), d = 0, 13, 10, 7 (the xor of 0x4
// with the group's two positions).  For the 4 index bytes of w at once:
// lo, hi = the low and high bytes of those 16 position bits (per byte of w),
// sh16 = 16 (x / 4) per byte (the shift of v within the 8 bytes).  A byte
// table of 0x44 ^ (d(x % 4) << 4 (x / 4 % 2)) for x % 8, looked up with
// v_perm, gives the varying byte; the other byte is 0x44.
__device__ __forceinline__ void msparse_fields(uint32_t w, uint32_t& lo, uint32_t& hi, uint32_t& sh16) {
  constexpr uint32_t kT8lo = 0x434E4944u;   // x % 8 = 0..3: 0x44, 0x49, 0x4E, 0x43
  constexpr uint32_t kT8hi = 0x34E49444u;   // x % 8 = 4..7: 0x44, 0x94, 0xE4, 0x34
  const uint32_t t = __builtin_amdgcn_perm(kT8hi, kT8lo, w & 0x07070707u);
  const uint32_t big = ((w >> 3) & 0x01010101u) * 0xffu;   // 0xff in the bytes with x >= 8
  lo = (big & 0x44444444u) | (~big & t);
  hi = (big & t) | (~big & 0x44444444u);
  sh16 = (w << 2) & 0x30303030u;                          // 16 (x / 4) per byte
}

}  // namespace

// C16: codebooks in units of 16 (padded codebooks have one-hot entries 0);
// WB: 32-column blocks per wavefront (W = 32 WB columns per slice)
template <int C16, int WB>
__global__ void __launch_bounds__(kMWaves * 64) macc_kernel(const MArgs a) {
  constexpr int W = 32 * WB;
  constexpr int CP = 16 * C16;                 // staged codebooks
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  mlds_t* s_tab = (mlds_t*)smem_raw;           // [CP][W][16] bytes (off 0)
  mlds_u8* s_val = reinterpret_cast<mlds_u8*>(s_tab + a.off_val);      // [kMaccGroups][CP] one-hot entries
  mlds_i32* s_sh = reinterpret_cast<mlds_i32*>(s_tab + a.off_sh);      // [CP] shifts (-1: padding)
  mlds_i32* s_misc = reinterpret_cast<mlds_i32*>(s_tab + a.off_misc);  // bias32 bits, e_min, max shift
  mlds_f32* s_bias = reinterpret_cast<mlds_f32*>(s_tab + a.off_bias);  // [W] column biases of the slice

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = muni(tid >> 6);
  const int C = a.C, M = a.M;
  const int64_t N = a.N;

  // ---------------- this workgroup's slice and rows
  const int b = blockIdx.x;
  int slice, group;
  if (a.xcd_map) {
    // (group, slice) pairs in group-major order, a contiguous run of them per
    // XCD (block b runs on XCD b % 8): the slices of a row group share an L2
    const int gi = (b & 7) * (int)(gridDim.x >> 3) + (b >> 3);
    slice = gi % a.nslices;
    group = gi / a.nslices;
  } else {
    slice = b % a.nslices;
    group = b / a.nslices;
  }
  const int col0 = slice * W;
  const int64_t r0 = (int64_t)group * a.rows_per_group;
  if (r0 >= N) return;   // uniform: no rows for this workgroup
  const int64_t r1 = min(N, r0 + a.rows_per_group);

  // ---------------- block exponents, shifts, the offsets' sum
  if (tid == 0) { s_misc[1] = INT_MAX; s_misc[2] = 0; }
  __syncthreads();
  const uint32_t* sb = reinterpret_cast<const uint32_t*>(a.scale);
  for (int c = tid; c < C; c += kMWaves * 64) atomicMin((int*)&s_misc[1], (int)((sb[c] >> 23) & 0xffu) - 127);
  __syncthreads();
  const int emin = muni(s_misc[1]);
  for (int c = tid; c < CP; c += kMWaves * 64) {
    const int sh = c < C ? min((int)((sb[c] >> 23) & 0xffu) - 127 - emin, 30) : -1;
    s_sh[c] = sh;
    atomicMax((int*)&s_misc[2], sh);
  }
  if (wave == 0) {   // double sum over codebooks in ascending order, rounded once
    double sum = 0.0;
    for (int c0 = 0; c0 < C; c0 += 64) {
      const float ov = a.offset[min(c0 + lane, C - 1)];
      const int n = min(64, C - c0);
      for (int j = 0; j < n; ++j) sum += (double)__int_as_float(__builtin_amdgcn_readlane(__float_as_int(ov), j));
    }
    if (lane == 0) s_misc[0] = __float_as_int((float)sum);
  }
  if (a.bias_lds)   // zeros past the last column
    for (int m = tid; m < W; m += kMWaves * 64) s_bias[m] = col0 + m < M ? a.col_bias[col0 + m] : 0.0f;

  // ---------------- the table slice, transposed: LDS byte (c W + m) 16 + p =
  // q[c][p][col0 + m].  A unit is 4 prototypes x 4 columns of one codebook:
  // four dword loads (one per prototype row) and a 4 x 4 byte transpose.
  {
    constexpr int units = CP * 4 * (W / 4);
    for (int u = tid; u < units; u += kMWaves * 64) {
      const int m4 = u % (W / 4);
      const int pg = (u / (W / 4)) & 3;
      const int c = u / (W / 4) / 4;
      const int col = col0 + 4 * m4;
      uint32_t d[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t e = ((int64_t)c * 16 + 4 * pg + r) * M + col;
        d[r] = (c < C && col < M) ? *reinterpret_cast<const uint32_t*>(a.lut + e) : 0u;
      }
      const uint32_t lo01 = __builtin_amdgcn_perm(d[1], d[0], 0x05010400u);   // d0.0 d1.0 d0.1 d1.1
      const uint32_t hi01 = __builtin_amdgcn_perm(d[1], d[0], 0x07030602u);   // d0.2 d1.2 d0.3 d1.3
      const uint32_t lo23 = __builtin_amdgcn_perm(d[3], d[2], 0x05010400u);
      const uint32_t hi23 = __builtin_amdgcn_perm(d[3], d[2], 0x07030602u);
      mlds_u32* dst = reinterpret_cast<mlds_u32*>(s_tab + ((c * W + 4 * m4) * 16 + 4 * pg));
      dst[0] = __builtin_amdgcn_perm(lo23, lo01, 0x05040100u);    // column + 0: d0.0 d1.0 d2.0 d3.0
      dst[4] = __builtin_amdgcn_perm(lo23, lo01, 0x07060302u);    // column + 1
      dst[8] = __builtin_amdgcn_perm(hi23, hi01, 0x05040100u);    // column + 2
      dst[12] = __builtin_amdgcn_perm(hi23, hi01, 0x07060302u);   // column + 3
    }
  }
  __syncthreads();
  const int maxsh = muni(s_misc[2]);
  const int ngroups = maxsh / kMGroupBits + 1;
  for (int u = tid; u < ngroups * CP; u += kMWaves * 64) {
    const int g = u / CP, c = u % CP;
    const int sh = s_sh[c];
    // the one-hot entry of codebook c in shift group g: 2^(sh_c - 7 g) when
    // its shift is in the group, else 0
    s_val[u] = (sh >= 0 && sh / kMGroupBits == g) ? (uint8_t)(1u << (sh - kMGroupBits * g)) : (uint8_t)0;
  }
  __syncthreads();
  const float step = __builtin_ldexpf(1.0f, emin);
  const float bias32 = __int_as_float(muni(s_misc[0]));

  // ---------------- row tiles
  const int h = lane >> 5;    // half-wavefront: codebook 16 j + 8 h + i of the pair
  const int ml = lane & 31;   // table operand: column; one-hot operand and results: row
  const uint32_t lane_tab = (uint32_t)(uintptr_t)(s_tab + (h * W + ml) * 16);
  const int cvalid = (C + 15) >> 4;   // index chunks of 16 codebooks that exist
  const int64_t ntiles = (r1 - r0 + kMTileRows - 1) / kMTileRows;

  // index bytes of codebooks 16 j + 8 h .. + 7 of the lane's two rows
  auto load_idx = [&](int64_t t, mu32x2 (&ix)[2][C16]) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      int64_t row = r0 + t * kMTileRows + 32 * rb + ml;
      row = row < N ? row : N - 1;
      const uint8_t* src = a.idx + row * C + 8 * h;
#pragma unroll
      for (int j = 0; j < C16; ++j)
        ix[rb][j] = j < cvalid ? *reinterpret_cast<const mu32x2*>(src + 16 * j) : (mu32x2){0u, 0u};
    }
  };

  // index chunks of the current tile; chunk j is reloaded with the next
  // tile's as soon as the last product step that reads it has been issued
  mu32x2 ixc[2][C16];
  const bool plain = a.y && !a.acc && col0 + W <= M;   // uniform
  const bool whole = a.y && col0 + W <= M;               // (the int32 sums too, whole tiles only)
  // the layer output of 4 consecutive columns from slice column lc: bias,
  // then ReLU (act 2)
  auto layer_out = [&](mf32x4 z, int lc) -> mf32x4 {
    if (a.act != 0) {
      const mf32x4 bb = a.bias_lds ? *reinterpret_cast<const mlds_f32x4*>(s_bias + lc)
                                   : (mf32x4){0.0f, 0.0f, 0.0f, 0.0f};
      z = z + bb;
      if (a.act == 2)
#pragma unroll
        for (int e = 0; e < 4; ++e) z[e] = z[e] > 0.0f ? z[e] : 0.0f;
    }
    return z;
  };
  int64_t t = wave;
  if (t < ntiles) load_idx(t, ixc);
  for (; t < ntiles; t += kMWaves) {
    const bool more = t + kMWaves < ntiles;   // uniform
    mi32x16 acc[2][WB];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int cb = 0; cb < WB; ++cb) acc[rb][cb] = (mi32x16){};
    for (int g = ngroups - 1; g >= 0; --g) {
      if (g != ngroups - 1) {
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int cb = 0; cb < WB; ++cb) acc[rb][cb] <<= kMGroupBits;
      }
      const mlds_t* vrow = reinterpret_cast<const mlds_t*>(s_val) + g * CP + 8 * h;
      mu32x2 vv[C16];   // one-hot entries of the lane's codebooks in this group
#pragma unroll
      for (int j = 0; j < C16; ++j) vv[j] = *reinterpret_cast<const mlds_u32x2*>(vrow + 16 * j);
      // (the index bytes opaque here: their extraction stays inside the group
      // loop instead of being hoisted out of it into more registers)
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int j = 0; j < C16; ++j) asm volatile("" : "+v"(ixc[rb][j]));
      {
        // sparse product step s (j = s / 4, i = s % 4) covers codebooks
        // 16 j + 2 i + {0, 1, 8, 9}: the lane's one-hot operand (row ml)
        // holds 16 j + 8 h + 2 i + k in groups 4 k .. 4 k + 3 (k = 0, 1);
        // its table operand (column ml) holds 16 j + 2 i + h in bytes 0-15
        // and 16 j + 8 + 2 i + h in bytes 16-31.  Table operands are read one
        // step ahead; the compressed one-hot operands are built in registers.
        auto load_tab = [&](auto sc, mi32x8 (&Bt)[WB]) {
          constexpr int st = decltype(sc)::value;
          constexpr int j = st / 4, i = st % 4;
#pragma unroll
          for (int cb = 0; cb < WB; ++cb) {
            const mi32x4 lo = *reinterpret_cast<const mlds_i32x4*>((const mlds_t*)(uintptr_t)lane_tab +
                                                                   ((16 * j + 2 * i) * W + 32 * cb) * 16);
            const mi32x4 hi = *reinterpret_cast<const mlds_i32x4*>((const mlds_t*)(uintptr_t)lane_tab +
                                                                   ((16 * j + 8 + 2 * i) * W + 32 * cb) * 16);
            Bt[cb] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          }
        };
        mi32x8 Ta[WB], Tb[WB];
        load_tab(std::integral_constant<int, 0>{}, Ta);
        mfor([&](auto sc) {
          constexpr int st = decltype(sc)::value;
          constexpr int j = st / 4, i = st % 4;
          mi32x8(&cur)[WB] = (st & 1) ? Tb : Ta;
          mi32x8(&nxt)[WB] = (st & 1) ? Ta : Tb;
          if constexpr (st + 1 < 4 * C16) load_tab(std::integral_constant<int, st + 1>{}, nxt);
          // bytes 2 i, 2 i + 1 of the chunk: dword i / 2, bytes 2 (i % 2) and
          // 2 (i % 2) + 1; the work on a whole dword (4 codebooks, two steps)
          // is shared by its two steps
          const uint32_t vw = vv[j][i >> 1] >> (16 * (i & 1));
#pragma unroll
          for (int rb = 0; rb < 2; ++rb) {
            const uint32_t w = ixc[rb][j][i >> 1];
            uint32_t lo, hi, sh16;
            msparse_fields(w, lo, hi, sh16);
            const int ix = (int)__builtin_amdgcn_perm(hi, lo, (i & 1) ? 0x07030602u : 0x05010400u);
            const int p0 = 16 * (i & 1);   // bit offset of the step's first byte
            const uint64_t q0 = (uint64_t)(vw & 0xffu) << ((sh16 >> p0) & 0xffu);
            const uint64_t q1 = (uint64_t)((vw >> 8) & 0xffu) << ((sh16 >> (p0 + 8)) & 0xffu);
            const mi32x4 A = {(int)(uint32_t)q0, (int)(uint32_t)(q0 >> 32), (int)(uint32_t)q1,
                              (int)(uint32_t)(q1 >> 32)};
#pragma unroll
            for (int cb = 0; cb < WB; ++cb)
              acc[rb][cb] = __builtin_amdgcn_smfmac_i32_32x32x64_i8(A, cur[cb], acc[rb][cb], ix, 0, 0);
          }
          if constexpr (st % 4 == 3) {
            // chunk j has been read for the last time in this pass: in the
            // last pass, start loading the next tile's
            if (g == 0 && more && j < cvalid) {
#pragma unroll
              for (int rb = 0; rb < 2; ++rb) {
                int64_t row = r0 + (t + kMWaves) * kMTileRows + 32 * rb + ml;
                row = row < N ? row : N - 1;
                ixc[rb][j] = *reinterpret_cast<const mu32x2*>(a.idx + row * C + 8 * h + 16 * j);
              }
            }
          }
          __builtin_amdgcn_sched_barrier(0);
        }, std::make_integer_sequence<int, 4 * C16>{});
      }
    }

    {
      // ---------------- epilogue of the sparse products: lane (ml, h)
      // holds column ml of each 32 x 32 block, rows 8 q + 4 h .. + 3 in
      // registers 4 q .. 4 q + 3
      if (whole && r0 + (t + 1) * kMTileRows <= r1) {
        // every row of the tile exists: dword stores, each writing two whole
        // 128-byte row segments (lanes 0-31 one row, 32-63 another), with no
        // vector work for addresses (the row offsets are scalar offsets of a
        // buffer store; the host keeps a group's outputs below 2^31 bytes),
        // as streaming stores (aux 2: nt).  Against the transposed 16-byte
        // stores below: 0.46 against 0.48 ms on a 1M x 512 output.
        const __amdgpu_buffer_rsrc_t yrs =
            __builtin_amdgcn_make_buffer_rsrc(a.y + r0 * M, 0, (int)((r1 - r0) * M * 4), kMBufDword3);
        // (two copies of the loop, so that the outputs-only one carries
        // nothing for the sums)
        auto stores = [&](auto with_sums) {
          constexpr bool SUMS = decltype(with_sums)::value;
          const __amdgpu_buffer_rsrc_t ars = __builtin_amdgcn_make_buffer_rsrc(
              SUMS ? a.acc + r0 * M : nullptr, 0, SUMS ? (int)((r1 - r0) * M * 4) : 0, kMBufDword3);
#pragma unroll
          for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int cb = 0; cb < WB; ++cb) {
              const int lc = 32 * cb + ml;
              const float bb = a.act != 0 && a.bias_lds ? s_bias[lc] : 0.0f;
              const int voff = (int)(((t * kMTileRows + 32 * rb + 4 * h) * (int64_t)M + col0 + lc) * 4);
#pragma unroll
              for (int r = 0; r < 16; ++r) {
                float z = __builtin_fmaf((float)acc[rb][cb][r], step, bias32);
                if (a.act != 0) {
                  z = z + bb;
                  if (a.act == 2) z = z > 0.0f ? z : 0.0f;
                }
                const int soff = __builtin_amdgcn_readfirstlane((8 * (r >> 2) + (r & 3)) * M * 4);
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(z), yrs, voff, soff, 2);
                if (SUMS) __builtin_amdgcn_raw_buffer_store_b32((uint32_t)acc[rb][cb][r], ars, voff, soff, 2);
              }
            }
        };
        if (a.acc)
          stores(std::true_type{});
        else
          stores(std::false_type{});
        continue;
      }
      if (plain) {
        // (the last tile of a group, rows past its end skipped) a dword
        // transpose over each quad of lanes gives lane 4 a + u row
        // 8 q + 4 h + u, columns 4 a .. 4 a + 3: a store instruction writes
        // 8 whole 128-byte row segments, as streaming stores
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int cb = 0; cb < WB; ++cb) {
            const int lc = 32 * cb + 4 * (ml >> 2);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              mi32x4 x;
#pragma unroll
              for (int e = 0; e < 4; ++e)
                x[e] = __float_as_int(__builtin_fmaf((float)acc[rb][cb][4 * q + e], step, bias32));
              mquad_transpose_dw(x, lane);
              const int64_t row = r0 + t * kMTileRows + 32 * rb + 8 * q + 4 * h + (ml & 3);
              if (row < r1)
                __builtin_nontemporal_store(layer_out(__builtin_bit_cast(mf32x4, x), lc),
                                            reinterpret_cast<mf32x4*>(a.y + row * M + col0 + lc));
            }
          }
        continue;
      }
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int cb = 0; cb < WB; ++cb) {
          const int lc = 32 * cb + ml;
          if (col0 + lc >= M) continue;
          const float bb = a.act != 0 && a.bias_lds ? s_bias[lc] : 0.0f;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int64_t row = r0 + t * kMTileRows + 32 * rb + 8 * (r >> 2) + 4 * h + (r & 3);
            if (row >= r1) continue;
            const int sv = acc[rb][cb][r];
            if (a.y) {
              float z = __builtin_fmaf((float)sv, step, bias32);
              if (a.act != 0) {
                z = z + bb;
                if (a.act == 2) z = z > 0.0f ? z : 0.0f;
              }
              a.y[row * M + col0 + lc] = z;
            }
            if (a.acc) a.acc[row * M + col0 + lc] = sv;
          }
        }
    }
  }
}

int macc_width(int C) { return C <= 64 ? 128 : 64; }

hipError_t launch_macc(const MArgs& m, int blocks, hipStream_t stream) {
  const void* fn = m.C <= 64 ? reinterpret_cast<const void*>(&macc_kernel<4, 4>)
                             : reinterpret_cast<const void*>(&macc_kernel<8, 2>);
  hipError_t err = hipSuccess;
  launch_prepare(fn, kMWaves * 64, m.lds_total, &err);
  if (err != hipSuccess) return err;
  if (m.C <= 64)
    hipLaunchKernelGGL((macc_kernel<4, 4>), dim3((unsigned)blocks), dim3(kMWaves * 64), m.lds_total,
                       stream, m);
  else
    hipLaunchKernelGGL((macc_kernel<8, 2>), dim3((unsigned)blocks), dim3(kMWaves * 64), m.lds_total,
                       stream, m);
  return hipGetLastError();
}

}  // namespace mdn
