// Lookup-accumulate with one output row per lane, for fp32 tables (§1 of
// McCarter & Dronen: the product is the sum over codebooks of the table rows
// the encoder selected; fp32 tables are summed in ascending codebook order,
// each sum starting from +0.0f).
//
// A work item is 1024 rows x 64 output columns: each of the 16 wavefronts of
// a 1024-thread workgroup takes 64 rows, one per lane, and every lane keeps
// the 64 sums of its row in registers.  The table's column slice is staged
// 16 codebooks at a time, [16 codebooks][16 prototypes][64 columns], into one
// of two LDS buffers; the next tile (or the next work item's first tile) is
// loaded straight into the other buffer (buffer_load ... lds, no registers)
// while the current one is summed.  A lane reads the staged row its own index
// selects: one address per codebook (a bit-field extract and a multiply-add),
// then 16 reads of 16 bytes whose offsets are immediates, so almost all of
// the vector work is the four fp32 adds per read.  Staged rows are 17 units
// of 16 bytes (the 17th a copy of the 16th), which puts the 16 prototypes of
// a codebook in 16 different LDS bank groups: the lanes of one read see no
// bank conflict whatever their indices (lanes with equal indices share the
// access).
//
// Each lane stores 16 bytes of its own row per store instruction, so one
// instruction touches 64 rows; these are ordinary (cached) stores, which the
// L2 merges into whole lines: as streaming stores they left the L2 as partial
// lines, written 3.7 times over with a read of each (6.3 against 4.6 ms on the
// 524288 x 1024 output of a 256-codebook layer).
//
// Work items are numbered with the column tile fastest, and a grid of whole
// XCD multiples gives each XCD runs of consecutive items, so the 16 column
// tiles of a row block mostly share one L2 for the index rows.
//
// int8 tables take the same scheme with 16-bit fields (rlane_i8_kernel,
// below) when their field sums fit.
#include "internal.hpp"

#include <climits>
#include <utility>

namespace mdn {

namespace {

typedef uint32_t lu32x4 __attribute__((ext_vector_type(4)));
typedef float lf32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char llds_t;
typedef __attribute__((address_space(3))) lu32x4 llds_u32x4;
typedef __attribute__((address_space(3))) lf32x4 llds_f32x4;
typedef __attribute__((address_space(3))) float llds_f32;
typedef __attribute__((address_space(3))) int32_t llds_i32;
typedef unsigned short lus2 __attribute__((ext_vector_type(2)));

constexpr int kLBufDword3 = 0x00020000;          // raw, unswizzled buffer descriptor (gfx9 family)
constexpr int kLVmcnt0 = 0x0F70;                 // s_waitcnt vmcnt(0), other counters unconstrained
constexpr int kLWaves = 16;                      // wavefronts per workgroup
constexpr int kLRows = kLWaves * 64;             // rows per work item
constexpr int kLUnits = kRowLaneCols / 4;        // 16-byte units per staged row (16)
constexpr int kLRowStride = (kLUnits + 1) * 16;  // 272: one pad unit per staged row
constexpr int kLCbStride = 16 * kLRowStride;     // 4352 bytes per codebook
constexpr int kLTileBytes = kRowLaneCT * kLCbStride;   // 69632 bytes per buffer
constexpr int kLStageLoads = kLTileBytes / 1024;       // 68 direct loads of 1 KB per tile
constexpr int kLStagePerWave = (kLStageLoads + kLWaves - 1) / kLWaves;   // 5 (waves 0-3), else 4
static_assert(kLTileBytes % 1024 == 0, "tile buffers are whole direct loads");
static_assert((kRowLaneCT - 1) * kLCbStride + (kLUnits - 1) * 16 <= 65535, "read offsets fit the immediate");

__device__ __forceinline__ int luni(int v) { return __builtin_amdgcn_readfirstlane(v); }

// f(integral_constant<int, I>) for I = 0, 1, ..., in order, unrolled
template <typename F, int... I>
__device__ __forceinline__ void lfor(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}

// 4 x 4 transpose of 16-byte elements over the four lanes of every quad:
// element k of lane q (its position in the quad) on entry is element q of
// lane k on return.  Two exchange stages, with the partner lane q ^ 1 (on
// element k ^ 1), then q ^ 2 (on k ^ 2): a DPP move and a select each.
__device__ __forceinline__ void quad_transpose(lu32x4 (&x)[4], int lane) {
  constexpr int kSwap1 = 0xB1;   // quad_perm [1, 0, 3, 2]
  constexpr int kSwap2 = 0x4E;   // quad_perm [2, 3, 0, 1]
  const int b0 = lane & 1, b1 = (lane >> 1) & 1;
  lu32x4 z[4];
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t t = (uint32_t)__builtin_amdgcn_mov_dpp((int)x[k ^ 1][e], kSwap1, 0xf, 0xf, false);
      z[k][e] = b0 == (k & 1) ? x[k][e] : t;
    }
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t t = (uint32_t)__builtin_amdgcn_mov_dpp((int)z[k ^ 2][e], kSwap2, 0xf, 0xf, false);
      x[k][e] = b1 == ((k >> 1) & 1) ? z[k][e] : t;
    }
}

template <int D>
__global__ void __launch_bounds__(1024) rlane_f32_kernel(const TArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  llds_t* s_tab = (llds_t*)smem_raw;   // two tile buffers (off_tab == 0)
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = luni(tid >> 6);
  const int C = a.C, M = a.M, ntm = a.ntm;
  const int64_t N = a.N;
  const int T = C / kRowLaneCT;   // tiles per work item (C % 16 == 0)

  const __amdgpu_buffer_rsrc_t trs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.lut), 0, (int)((int64_t)C * 16 * M * 4), kLBufDword3);
  // this lane's part of direct load j of a tile: unit g of the tile's 272-byte
  // rows (row rr = codebook * 16 + prototype, unit u; the pad unit repeats
  // unit 15), as a byte offset from the tile's first table element
  int rel[kLStagePerWave];
#pragma unroll
  for (int j = 0; j < kLStagePerWave; ++j) {
    const int g = (wave + kLWaves * j) * 64 + lane;
    const int rr = g / (kLUnits + 1), u = g % (kLUnits + 1);
    rel[j] = rr * M * 4 + min(u, kLUnits - 1) * 16;
  }
  auto stage = [&](int t, int m0, int buf) {
    const int sbase = (t * kRowLaneCT * 16 * M + m0) * 4;
#pragma unroll
    for (int j = 0; j < kLStagePerWave; ++j) {
      const int i = wave + kLWaves * j;
      if (j + 1 < kLStagePerWave || i < kLStageLoads)   // uniform
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            trs, (__attribute__((address_space(3))) void*)(s_tab + buf * kLTileBytes + i * 1024), 16, rel[j], sbase,
            0, 0);
    }
  };
  auto publish = [&]() {   // this wavefront's direct loads are in LDS, then the barrier
    __builtin_amdgcn_s_waitcnt(kLVmcnt0);   // (as a builtin the compiler knows every load has completed)
    __syncthreads();
  };

  // work item numbering: with a grid of whole multiples of 8, workgroup b
  // (dispatched to XCD b % 8) takes positions within its XCD's run
  const int G = gridDim.x;
  const int pos = (G % 8 == 0) ? (int)((blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3)) : (int)blockIdx.x;
  const int64_t nwork = a.nwork;
  const int64_t stride = a.idx_stride;
  auto lane_row = [&](int64_t w) { return min((w / ntm) * kLRows + (int64_t)wave * 64 + lane, N - 1); };

  llds_f32x4* s_bias = reinterpret_cast<llds_f32x4*>(s_tab + a.off_bias);
  if (a.bias_lds)   // (col_bias is only 4-byte aligned: one float per load); zeros up to whole column tiles
    for (int m = tid; m < ntm * kRowLaneCols; m += kLWaves * 64)
      reinterpret_cast<llds_f32*>(s_bias)[m] = m < M ? a.col_bias[m] : 0.0f;

  int gb = 0;   // buffer of the current tile (alternates over the whole sequence)
  lu32x4 kc = {0u, 0u, 0u, 0u};   // index bytes of the current tile's 16 codebooks (this lane's row)
  lu32x4 kn = kc;                 // those of the next tile
  if (pos < nwork) {
    stage(0, (int)(pos % ntm) * kRowLaneCols, 0);
    kc = *reinterpret_cast<const lu32x4*>(a.idx + lane_row(pos) * stride);
    publish();
    asm volatile("" : "+v"(kc));
  }
  for (int64_t w = pos; w < nwork; w += G) {
    const int mt = (int)(w % ntm);
    const int m0 = mt * kRowLaneCols;
    const int64_t row = (w / ntm) * kLRows + (int64_t)wave * 64 + lane;   // this lane's output row
    const int64_t wn = w + G;
    const int64_t rown = lane_row(w);
    const int64_t rown_next = wn < nwork ? lane_row(wn) : rown;   // the next work item's
    const int mn0 = (int)(wn % ntm) * kRowLaneCols;
    float acc[4 * kLUnits];
#pragma unroll
    for (int i = 0; i < 4 * kLUnits; ++i) acc[i] = 0.0f;

    for (int t = 0; t < T; ++t) {
      // the other buffer's readers (the previous tile) finished before the last barrier
      if (t + 1 < T) {
        kn = *reinterpret_cast<const lu32x4*>(a.idx + rown * stride + kRowLaneCT * (t + 1));
        stage(t + 1, m0, gb ^ 1);
      } else if (wn < nwork) {
        kn = *reinterpret_cast<const lu32x4*>(a.idx + rown_next * stride);
        stage(0, mn0, gb ^ 1);
      }
      const uint32_t base = (uint32_t)gb * kLTileBytes;
      uint32_t adr = 0;
      lu32x4 v[D + 1];
      // step s reads unit s % 16 of codebook s / 16; reads run D steps ahead
      auto read = [&](auto S) {
        constexpr int s = decltype(S)::value;
        constexpr int cb = s / kLUnits, u = s % kLUnits;
        if constexpr (u == 0) {
          const uint32_t k = __builtin_amdgcn_ubfe(kc[cb >> 2], 8 * (cb & 3), 4);
          adr = k * (uint32_t)kLRowStride + base;
        }
        v[s % (D + 1)] = *reinterpret_cast<const llds_u32x4*>((const llds_t*)(uintptr_t)adr + cb * kLCbStride + u * 16);
      };
      auto step = [&](auto S) {
        constexpr int s = decltype(S)::value;
        constexpr int u = s % kLUnits;
        if constexpr (s + D < kRowLaneCT * kLUnits) read(std::integral_constant<int, s + D>{});
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int e = 0; e < 4; ++e)   // codebooks ascending; each sum stays in its register
          asm("v_add_f32 %0, %0, %1" : "+v"(acc[4 * u + e]) : "v"(v[s % (D + 1)][e]));
        __builtin_amdgcn_sched_barrier(0);
      };
      lfor(read, std::make_integer_sequence<int, D>{});
      lfor(step, std::make_integer_sequence<int, kRowLaneCT * kLUnits>{});
      publish();   // the next tile visible; every reader of this buffer done
      gb ^= 1;
      kc = kn;
      asm volatile("" : "+v"(kc), "+v"(kn));   // (the loads have completed: no waits for them later)
    }

    // ---------------- epilogue: row `row`, columns m0 .. m0 + 63, one unit at a time
    lf32x4* yr = reinterpret_cast<lf32x4*>(a.y + min(row, N - 1) * M + m0);
    auto z_of = [&](int u) {   // sum, or the layer output: + column bias (act 1), then ReLU (act 2)
      lf32x4 z = {acc[4 * u], acc[4 * u + 1], acc[4 * u + 2], acc[4 * u + 3]};
      if (a.act != 0) {
        const lf32x4 b4 = a.bias_lds ? s_bias[(m0 >> 2) + u] : (lf32x4){0.0f, 0.0f, 0.0f, 0.0f};   // padded past M
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          z[e] = z[e] + b4[e];
          if (a.act == 2) z[e] = (z[e] > 0.0f) ? z[e] : 0.0f;
        }
      }
      return z;
    };
#pragma unroll
    for (int u = 0; u < kLUnits; ++u) {
      const lf32x4 z = z_of(u);
      if (row < N && m0 + 4 * u < M) yr[u] = z;   // M % 4 == 0: whole units
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}


// y for int8 tables whose 16-bit field sums fit: 255 sum_c 2^sh_c <= 65535, with
// sh_c = e_c - e_min from the exponents of the codebook scales (each term
// saturated at 2^15; the row-uniform kernel, launched after this one, makes
// the same test and does the other case with 32-bit sums).  One row per lane
// over 128 columns: a staged entry is the 16-bit field u = (q + 128) << sh_c,
// so a 16-byte read holds 8 columns, and one v_add3_u32 adds two codebooks to
// two columns (no field carries into the next, as the exact total fits).  The
// int32 sum is the field minus 128 sum_c 2^sh_c, and y = sum * 2^e_min + the
// offsets' sum (a single fma), as in the row-uniform kernel.
//
// A workgroup keeps one 128-column tile of the table for its lifetime and
// streams row blocks; the table tiles cycle through the codebooks, and since
// integer sums do not depend on their order, wavefront w joins the cycle at
// its own phase (w T / 16 tiles, T tiles per cycle) and sums any T
// consecutive tiles for a set of rows.  The wavefronts' output stores are
// then spread over the tiles instead of coming all at once from every CU
// (which left the LDS idle while HBM took the burst).  The table goes through
// registers: each thread loads 32 bytes of the tile after next while the
// current tile is summed, and at the start of a tile widens the registers it
// loaded one tile earlier and writes them to the free buffer.
template <int DI, bool XPOSE>
__global__ void __launch_bounds__(1024) rlane_i8_kernel(const TArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  llds_t* s_tab = (llds_t*)smem_raw;   // two tile buffers (off_tab == 0)
  llds_i32* s_sh = reinterpret_cast<llds_i32*>(s_tab + a.off_sh);
  llds_i32* s_misc = reinterpret_cast<llds_i32*>(s_tab + a.off_misc);   // offsets' sum (bits), e_min, sum of 2^sh
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = luni(tid >> 6);
  const int C = a.C, M = a.M, ntm = a.ntm;
  const int64_t N = a.N;
  const int T = C / kRowLaneCT;   // tiles per work item (C % 16 == 0, T >= 2)

  // ---------------- block exponents, shifts, their sum and the offsets' sum
  if (tid == 0) { s_misc[1] = INT_MAX; s_misc[2] = 0; }
  __syncthreads();
  const uint32_t* sb = reinterpret_cast<const uint32_t*>(a.scale);
  for (int c = tid; c < C; c += kLWaves * 64) atomicMin((int*)&s_misc[1], (int)((sb[c] >> 23) & 0xffu) - 127);
  __syncthreads();
  const int emin = luni(s_misc[1]);
  for (int c = tid; c < C; c += kLWaves * 64) {
    const int sh = min((int)((sb[c] >> 23) & 0xffu) - 127 - emin, 30);
    s_sh[c] = sh;
    atomicAdd((int*)&s_misc[2], sh <= 14 ? (1 << sh) : (1 << 15));
  }
  if (wave == 0) {   // the offsets' sum: double, codebooks in ascending order, rounded once
    double sum = 0.0;
    for (int c0 = 0; c0 < C; c0 += 64) {
      const float ov = a.offset[min(c0 + lane, C - 1)];
      const int n = min(64, C - c0);
      for (int j = 0; j < n; ++j) sum += (double)__int_as_float(__builtin_amdgcn_readlane(__float_as_int(ov), j));
    }
    if (lane == 0) s_misc[0] = __float_as_int((float)sum);
  }
  llds_f32x4* s_bias = reinterpret_cast<llds_f32x4*>(s_tab + a.off_bias);
  if (a.bias_lds)   // (col_bias is only 4-byte aligned: one float per load); zeros up to whole column tiles
    for (int m = tid; m < ntm * kRowLaneColsI8; m += kLWaves * 64)
      reinterpret_cast<llds_f32*>(s_bias)[m] = m < M ? a.col_bias[m] : 0.0f;
  __syncthreads();
  const int S = luni(s_misc[2]);
  if (S > 257) return;   // 32-bit sums: the row-uniform kernel does this call (uniform over the workgroup)
  const float step = __builtin_ldexpf(1.0f, emin);
  const float bias = __int_as_float(luni(s_misc[0]));

  // ---------------- staging: thread t widens 32 columns (32 (t % 4)..) of staged
  // row t / 4 of a tile (codebook t / 64 of the tile: one per wavefront)
  const __amdgpu_buffer_rsrc_t trs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.lut), 0, (int)((int64_t)C * 16 * M), kLBufDword3);
  const int srow = tid >> 2, spart = tid & 3;
  lu32x4 tv[2];
  // (the offsets are derived at each call through an empty asm, so the
  // compiler does not keep precomputed ones in registers)
  auto load_tile = [&](int t, int m0) {
    int col = m0 + 32 * spart;
    asm volatile("" : "+v"(col));
    const int base = (t * kRowLaneCT * 16 + srow) * M + col;
#pragma unroll
    for (int h = 0; h < 2; ++h)   // M % 16 == 0: units are whole
      tv[h] = __builtin_amdgcn_raw_buffer_load_b128(trs, col + 16 * h < M ? base + 16 * h : INT_MAX, 0, 0);
  };
  auto store_tile = [&](int t, int buf) {
    const unsigned short sh = (unsigned short)luni(s_sh[t * kRowLaneCT + wave]);
    const lus2 s2 = {sh, sh};
    llds_t* dst = s_tab + buf * kLTileBytes + srow * kLRowStride + spart * 64;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      uint32_t w[8];   // fields of columns (2i, 2i + 1)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t u = tv[h][i] ^ 0x80808080u;   // q + 128 per byte
        w[2 * i] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(lus2, __builtin_amdgcn_perm(0u, u, 0x0c010c00u)) << s2);
        w[2 * i + 1] =
            __builtin_bit_cast(uint32_t, __builtin_bit_cast(lus2, __builtin_amdgcn_perm(0u, u, 0x0c030c02u)) << s2);
      }
      *reinterpret_cast<llds_u32x4*>(dst + 32 * h) = (lu32x4){w[0], w[1], w[2], w[3]};
      *reinterpret_cast<llds_u32x4*>(dst + 32 * h + 16) = (lu32x4){w[4], w[5], w[6], w[7]};
    }
  };

  // ---------------- this workgroup's column tile and row blocks (the grid is
  // a multiple of the column tiles: gpt workgroups per column tile)
  const int gpt = (int)gridDim.x / ntm;
  const int m0 = (int)(blockIdx.x % ntm) * kRowLaneColsI8;
  const int64_t rb0 = blockIdx.x / ntm;
  const int64_t nrb = (N + kLRows - 1) / kLRows;
  const int K = (int)((nrb - rb0 + gpt - 1) / gpt);   // row blocks rb0, rb0 + gpt, ... below nrb
  if (K <= 0) return;   // (uniform)
  const bool spread = K >= 4;   // phases pay off over a few row blocks only
  const int phi = spread ? (wave * T) >> 4 : 0;   // this wavefront's first tile
  const int stot = K * T + (spread ? (15 * T) >> 4 : 0);   // tiles this workgroup stages
  const int64_t stride = a.idx_stride;
  // this lane's row in its row set k (clamped)
  auto lane_row = [&](int k) {
    const int64_t r = (rb0 + (int64_t)k * gpt) * kLRows + wave * 64;   // (uniform)
    return min(r + lane, N - 1);
  };
  // index bytes of tile s for this lane (zeros outside its row sets)
  auto idx_of = [&](int s) -> lu32x4 {
    const int rel = s - phi;
    if (rel < 0 || rel >= K * T) return (lu32x4){0u, 0u, 0u, 0u};   // (uniform)
    return *reinterpret_cast<const lu32x4*>(a.idx + lane_row(rel / T) * stride + kRowLaneCT * (s % T));
  };

  int gb = 0;
  load_tile(0, m0);
  lu32x4 kc = idx_of(0);   // index bytes of the current tile's 16 codebooks (this lane's row)
  lu32x4 kn = kc;          // those of the next tile
  store_tile(0, 0);
  if (stot > 1) load_tile(1 % T, m0);
  __syncthreads();
  asm volatile("" : "+v"(kc));
  uint32_t acc[4 * kLUnits];   // fields of columns m0 + 8u + 2e, + 1 in word 4u + e
#pragma unroll
  for (int i = 0; i < 4 * kLUnits; ++i) acc[i] = 0u;
  const int off128 = 128 * S;

  for (int s = 0; s < stot; ++s) {
    // the next tile (registers) into the free buffer, whose readers finished
    // before the last barrier; then the tile after it into the registers
    if (s + 1 < stot) {
      kn = idx_of(s + 1);
      store_tile((s + 1) % T, gb ^ 1);
      if (s + 2 < stot) load_tile((s + 2) % T, m0);
    }
    const int rel = s - phi;
    const bool active = rel >= 0 && rel < K * T;   // (uniform per wavefront)
    if (active) {
      const uint32_t base = (uint32_t)gb * kLTileBytes;
      uint32_t adr0 = 0, adr1 = 0;
      lu32x4 v[DI + 1][2];
      // item i: codebooks 2 (i / 16) and 2 (i / 16) + 1, unit i % 16; reads run DI items ahead
      auto read = [&](auto I) {
        constexpr int i = decltype(I)::value;
        constexpr int cb = 2 * (i / kLUnits), u = i % kLUnits;
        if constexpr (u == 0) {
          adr0 = __builtin_amdgcn_ubfe(kc[cb >> 2], 8 * (cb & 3), 4) * (uint32_t)kLRowStride + base;
          adr1 = __builtin_amdgcn_ubfe(kc[cb >> 2], 8 * (cb & 3) + 8, 4) * (uint32_t)kLRowStride + base;
        }
        v[i % (DI + 1)][0] =
            *reinterpret_cast<const llds_u32x4*>((const llds_t*)(uintptr_t)adr0 + cb * kLCbStride + u * 16);
        v[i % (DI + 1)][1] =
            *reinterpret_cast<const llds_u32x4*>((const llds_t*)(uintptr_t)adr1 + (cb + 1) * kLCbStride + u * 16);
      };
      auto step = [&](auto I) {
        constexpr int i = decltype(I)::value;
        constexpr int u = i % kLUnits;
        if constexpr (i + DI < kRowLaneCT / 2 * kLUnits) read(std::integral_constant<int, i + DI>{});
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int e = 0; e < 4; ++e)   // each sum stays in its register
          asm("v_add3_u32 %0, %1, %2, %0" : "+v"(acc[4 * u + e]) : "v"(v[i % (DI + 1)][0][e]), "v"(v[i % (DI + 1)][1][e]));
        __builtin_amdgcn_sched_barrier(0);
      };
      lfor(read, std::make_integer_sequence<int, DI>{});
      lfor(step, std::make_integer_sequence<int, kRowLaneCT / 2 * kLUnits>{});
    }
    __syncthreads();   // the next tile visible; every reader of this buffer done
    gb ^= 1;
    kc = kn;
    asm volatile("" : "+v"(kc), "+v"(kn));   // (the loads have completed: no waits for them later)

    if (active && rel % T == T - 1) {
      // ---------------- this wavefront's row set is complete (the others sum
      // the next tile meanwhile): y for columns m0 .. m0 + 127, 16 at a time
      int64_t rq = (rb0 + (int64_t)(rel / T) * gpt) * kLRows + (int64_t)wave * 64;   // the wavefront's first row
      asm volatile("" : "+v"(rq));   // (derived here, not kept across the tiles)
#pragma unroll
      for (int g = 0; g < kLUnits / 2; ++g) {
        const bool cols_ok = m0 + 16 * g < M;   // M % 16 == 0: whole groups
        lu32x4 x[4];   // element k: columns 16 g + 4 k ..
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          lf32x4 b4 = {0.0f, 0.0f, 0.0f, 0.0f};
          if (a.act != 0 && a.bias_lds) b4 = s_bias[(m0 >> 2) + 4 * g + k];   // padded past M
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t f = acc[8 * g + 2 * k + (e >> 1)];
            const int sum = (int)((e & 1) ? (f >> 16) : (f & 0xffffu)) - off128;
            float z = __builtin_fmaf((float)sum, step, bias);
            if (a.act != 0) {   // + column bias, then ReLU
              z = z + b4[e];
              if (a.act == 2) z = (z > 0.0f) ? z : 0.0f;
            }
            x[k][e] = __float_as_uint(z);
          }
        }
        if constexpr (XPOSE) {
          // lane q of each quad takes columns 4 q .. 4 q + 3 of the 16 for the
          // quad's four rows: a store instruction then writes 64 contiguous
          // bytes of 16 rows instead of 16 bytes of 64 rows (a quarter of the
          // L2 write requests, for tables whose row sets end often)
          quad_transpose(x, lane);
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const int64_t r = rq + (lane & ~3) + k;
            if (r < N && cols_ok) *reinterpret_cast<lu32x4*>(a.y + r * M + m0 + 16 * g + 4 * (lane & 3)) = x[k];
          }
        } else {
          const int64_t r = rq + lane;
          if (r < N && cols_ok) {
            lu32x4* yr = reinterpret_cast<lu32x4*>(a.y + r * M + m0 + 16 * g);
#pragma unroll
            for (int k = 0; k < 4; ++k) yr[k] = x[k];
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int i = 0; i < 4 * kLUnits; ++i) acc[i] = 0u;
    }
  }
}

}  // namespace

hipError_t launch_rlane_f32(const TArgs& t, int cus, hipStream_t stream) {
  constexpr int D = 4;
  const void* fn = reinterpret_cast<const void*>(&rlane_f32_kernel<D>);
  hipError_t err = hipSuccess;
  const int per_cu = launch_prepare(fn, kLWaves * 64, t.lds_total, &err);
  if (err != hipSuccess) return err;
  int64_t blocks = t.nwork;
  const int64_t resident = (int64_t)per_cu * cus;
  if (blocks > resident) blocks = resident;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(rlane_f32_kernel<D>, dim3((unsigned)blocks), dim3(kLWaves * 64), t.lds_total, stream, t);
  return hipGetLastError();
}

hipError_t launch_rlane_i8(const TArgs& t, int cus, hipStream_t stream) {
  constexpr int DI = 2;
  // quad-transposed stores below 128 codebooks (row sets end every C / 16
  // tiles: more wavefronts store per tile)
  const bool xpose = t.C < 128;
  const void* fn = xpose ? reinterpret_cast<const void*>(&rlane_i8_kernel<DI, true>)
                         : reinterpret_cast<const void*>(&rlane_i8_kernel<DI, false>);
  hipError_t err = hipSuccess;
  const int per_cu = launch_prepare(fn, kLWaves * 64, t.lds_total, &err);
  if (err != hipSuccess) return err;
  // whole multiples of the column tiles, each workgroup streaming row blocks
  // of one of them
  const int64_t resident = (int64_t)per_cu * cus;
  int64_t gpt = (t.nwork < resident ? t.nwork : resident) / t.ntm;
  if (gpt < 1) gpt = 1;
  const int64_t blocks = gpt * t.ntm;
  if (xpose)
    hipLaunchKernelGGL((rlane_i8_kernel<DI, true>), dim3((unsigned)blocks), dim3(kLWaves * 64), t.lds_total, stream, t);
  else
    hipLaunchKernelGGL((rlane_i8_kernel<DI, false>), dim3((unsigned)blocks), dim3(kLWaves * 64), t.lds_total, stream, t);
  return hipGetLastError();
}

}  // namespace mdn
