// Offline table construction for one layer: T = P B (§2.2), then 8-bit block
// floating point quantization (§1).  Not on the inference hot path; it turns
// prototypes and weights into the tables the hot path reads.
//
// T[c][k][m] = sum_d P[c][k][d] * B[d][m] is a double sum over d ascending;
// the products of two fp32 values are exact in double and the library is
// built with -ffp-contract=off, so every entry is one well-defined double.
//
// Quantization of codebook c over its 16 x M entries:
//   offset o_c = (float)((min + max) / 2),  r_c = max |T - o_c|,
//   e_c        = smallest e in [-126, 127] with r_c <= 127 * 2^e,
//   e_c       <- max(e_c, max_c' e_c' - cap)   (127 * C * 2^cap < 2^24),
//   q          = round-half-even((T - o_c) * 2^-e_c),  |q| <= 127.
// Three launches: per-codebook statistics (one workgroup per codebook; the
// exponents are parked in scale_out as integers), codes, then scales.
#include "internal.hpp"

namespace mdn {

constexpr int kBuildThreads = 256;
// the statistics pass: one workgroup of kStatsThreads per codebook, kStatsILP
// entries of a thread evaluated together (their sums are independent chains,
// each in its own order)
constexpr int kStatsThreads = 1024;
constexpr int kStatsILP = 4;

__device__ __forceinline__ double table_entry(const float* __restrict__ P, const float* __restrict__ B,
                                              int D, int M, int64_t row, int m) {
  const float* p = P + row * D;
  double s = 0.0;
  for (int d = 0; d < D; ++d) s = __dadd_rn(s, __dmul_rn((double)p[d], (double)B[(int64_t)d * M + m]));
  return s;
}

// where the quantizer's entries come from: T = P B computed on the fly, or a
// given double table (a fitted one)
struct SrcPB {
  const float* P;
  const float* B;
  int D, M;
  __device__ double at(int64_t row, int m) const { return table_entry(P, B, D, M, row, m); }
  // entries e0 + q stride (q < kStatsILP) of codebook c's 16 x M block: the
  // sums run side by side, each over d ascending; entries past `per` read a
  // valid entry and are ignored
  __device__ void at_many(int c, int e0, int stride, int per, double* t) const {
    const float* p[kStatsILP];
    const float* b[kStatsILP];
#pragma unroll
    for (int q = 0; q < kStatsILP; ++q) {
      const int e = min(e0 + q * stride, per - 1);
      const int k = e / M, m = e - k * M;
      p[q] = P + ((int64_t)c * kK + k) * D;
      b[q] = B + m;
      t[q] = 0.0;
    }
    for (int d = 0; d < D; ++d)
#pragma unroll
      for (int q = 0; q < kStatsILP; ++q)
        t[q] = __dadd_rn(t[q], __dmul_rn((double)p[q][d], (double)b[q][(int64_t)d * M]));
  }
};
struct SrcT {
  const double* T;
  int M;
  __device__ double at(int64_t row, int m) const { return T[row * M + m]; }
  __device__ void at_many(int c, int e0, int stride, int per, double* t) const {
#pragma unroll
    for (int q = 0; q < kStatsILP; ++q) {
      const int e = min(e0 + q * stride, per - 1);
      t[q] = T[(int64_t)c * kK * M + e];
    }
  }
};

template <int NT>
__device__ double block_reduce(double v, bool take_max, double* s_red) {
  const int tid = threadIdx.x;
  s_red[tid] = v;
  __syncthreads();
  for (int w = NT / 2; w > 0; w >>= 1) {
    if (tid < w) {
      const double o = s_red[tid + w];
      s_red[tid] = take_max ? fmax(s_red[tid], o) : fmin(s_red[tid], o);
    }
    __syncthreads();
  }
  const double r = s_red[0];
  __syncthreads();
  return r;
}

template <class Src>
__global__ void __launch_bounds__(kStatsThreads)
table_stats_kernel(const Src src, int M, float* __restrict__ scale_out, float* __restrict__ offset_out) {
  __shared__ double s_red[kStatsThreads];
  const int c = blockIdx.x;
  const int per = kK * M;
  double lo = __builtin_inf(), hi = -__builtin_inf();
  for (int e0 = threadIdx.x; e0 < per; e0 += kStatsILP * kStatsThreads) {
    double t[kStatsILP];
    src.at_many(c, e0, kStatsThreads, per, t);
#pragma unroll
    for (int q = 0; q < kStatsILP; ++q)
      if (e0 + q * kStatsThreads < per) {
        lo = fmin(lo, t[q]);
        hi = fmax(hi, t[q]);
      }
  }
  lo = block_reduce<kStatsThreads>(lo, false, s_red);
  hi = block_reduce<kStatsThreads>(hi, true, s_red);
  const float o = (float)__ddiv_rn(__dadd_rn(lo, hi), 2.0);
  double r = 0.0;
  for (int e0 = threadIdx.x; e0 < per; e0 += kStatsILP * kStatsThreads) {
    double t[kStatsILP];
    src.at_many(c, e0, kStatsThreads, per, t);
#pragma unroll
    for (int q = 0; q < kStatsILP; ++q)
      if (e0 + q * kStatsThreads < per) r = fmax(r, fabs(__dsub_rn(t[q], (double)o)));
  }
  r = block_reduce<kStatsThreads>(r, true, s_red);
  if (threadIdx.x == 0) {
    int ex = -126;
    while (ex < 127 && r > 127.0 * __builtin_ldexp(1.0, ex)) ++ex;
    offset_out[c] = o;
    reinterpret_cast<int*>(scale_out)[c] = ex;  // parked exponent, replaced by table_scale_kernel
  }
}

__device__ int max_parked_exponent(const float* __restrict__ scale_out, int C, int* s_max) {
  if (threadIdx.x == 0) *s_max = -126;
  __syncthreads();
  const int* parked = reinterpret_cast<const int*>(scale_out);
  for (int c = threadIdx.x; c < C; c += blockDim.x) atomicMax(s_max, parked[c]);
  __syncthreads();
  return *s_max;
}

template <class Src>
__global__ void __launch_bounds__(kBuildThreads)
table_codes_kernel(const Src src, int C, int M, int cap, const float* __restrict__ scale_out,
                   const float* __restrict__ offset_out, int8_t* __restrict__ lut) {
  __shared__ int s_max;
  const int emax = max_parked_exponent(scale_out, C, &s_max);
  const int64_t total = (int64_t)C * kK * M;
  for (int64_t e = (int64_t)blockIdx.x * kBuildThreads + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * kBuildThreads) {
    const int64_t row = e / M;
    const int m = (int)(e - row * M);
    const int c = (int)(row / kK);
    const int ex = max(reinterpret_cast<const int*>(scale_out)[c], emax - cap);
    const double t = src.at(row, m);
    const double q = rint(__dmul_rn(__dsub_rn(t, (double)offset_out[c]), __builtin_ldexp(1.0, -ex)));
    lut[e] = (int8_t)(int)fmin(127.0, fmax(-127.0, q));
  }
}

__global__ void table_scale_kernel(float* __restrict__ scale_out, int C, int cap) {
  __shared__ int s_max;
  const int emax = max_parked_exponent(scale_out, C, &s_max);
  // every thread has read its exponents before any is replaced
  int ex[4];
  for (int j = 0; j < 4; ++j) {
    const int c = threadIdx.x + j * blockDim.x;
    ex[j] = c < C ? max(reinterpret_cast<const int*>(scale_out)[c], emax - cap) : 0;
  }
  __syncthreads();
  for (int j = 0; j < 4; ++j) {
    const int c = threadIdx.x + j * blockDim.x;
    if (c < C) scale_out[c] = __builtin_ldexpf(1.0f, ex[j]);
  }
}

__global__ void __launch_bounds__(kBuildThreads)
table_f32_kernel(const float* __restrict__ P, const float* __restrict__ B, int C, int D, int M,
                 float* __restrict__ lut) {
  const int64_t total = (int64_t)C * kK * M;
  for (int64_t e = (int64_t)blockIdx.x * kBuildThreads + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * kBuildThreads) {
    const int64_t row = e / M;
    const int m = (int)(e - row * M);
    lut[e] = (float)table_entry(P, B, D, M, row, m);
  }
}

static unsigned grid_for(int64_t total) {
  const int64_t g = (total + kBuildThreads - 1) / kBuildThreads;
  return (unsigned)(g < 65536 ? (g > 0 ? g : 1) : 65536);
}

template <class Src>
static hipError_t quantize(const Src& src, int C, int M, int8_t* lut, float* scale, float* offset, int cap,
                           hipStream_t stream) {
  hipLaunchKernelGGL(table_stats_kernel<Src>, dim3(C), dim3(kStatsThreads), 0, stream, src, M, scale, offset);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(table_codes_kernel<Src>, dim3(grid_for((int64_t)C * kK * M)), dim3(kBuildThreads), 0,
                     stream, src, C, M, cap, scale, offset, lut);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // C <= 4 * 256 codebooks per single-workgroup scale pass
  hipLaunchKernelGGL(table_scale_kernel, dim3(1), dim3(256), 0, stream, scale, C, cap);
  return hipGetLastError();
}

hipError_t launch_build_lut(const float* P, const float* B, int C, int D, int M, int8_t* lut,
                            float* scale, float* offset, int cap, hipStream_t stream) {
  return quantize(SrcPB{P, B, D, M}, C, M, lut, scale, offset, cap, stream);
}

hipError_t launch_quantize_lut(const double* T, int C, int M, int8_t* lut, float* scale, float* offset, int cap,
                               hipStream_t stream) {
  return quantize(SrcT{T, M}, C, M, lut, scale, offset, cap, stream);
}

hipError_t launch_build_lut_f32(const float* P, const float* B, int C, int D, int M, float* lut,
                                hipStream_t stream) {
  hipLaunchKernelGGL(table_f32_kernel, dim3(grid_for((int64_t)C * kK * M)), dim3(kBuildThreads), 0,
                     stream, P, B, C, D, M, lut);
  return hipGetLastError();
}

}  // namespace mdn
