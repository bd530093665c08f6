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

}  // namespace mdn
