// Model-aware table fit, Eq. 3 of McCarter & Dronen (§2.2), with an affine
// layer output (bias and identity, which cancel): the table T minimising
// ||Y - G T||^2 + lambda ||T - T0||^2 solves the normal equations
//     (G^T G + lambda I) T = G^T Y + lambda T0,
// G the one-hot encoder output (G[n][16c + k] = 1 iff idx[n][c] = k), Y = AB
// the layer's exact outputs on training rows and T0 = P0 B the prototype
// table.  Offline: it turns training data into a table for the hot path.
//
// Steps (each its own launch family):
//   gram    H = G^T G, integer counts: H[16c + k][16c' + k'] is the number of
//           rows whose codebook-c index is k and codebook-c' index is k'.
//           Workgroups own an 8 x 8 block of codebook pairs and a row chunk,
//           count in LDS, then add their nonzero counts to H (integer
//           atomics: the result does not depend on their order).
//   scatter R = G^T Y in double: a stable counting sort lists each
//           codebook's rows bucket by bucket (ascending within a bucket),
//           then one wavefront per (codebook, 64 columns), lane = column,
//           sums each bucket's rows in that order: every entry is the sum of
//           its rows in ascending row order.
//   solve   A = H + lambda I (double), B = R + lambda T0; A = L L^T by a
//           blocked right-looking Cholesky factorisation (panels of 32:
//           diagonal block in one workgroup, the rows below it, then the
//           trailing update), then blocked forward and backward substitution
//           over the M columns of B, in place.
// Every multiply-subtract is one fused multiply-add, and every entry takes
// its terms in the same order as the unblocked algorithm (k ascending in the
// factor and forward pass, descending in the backward pass), so the result
// does not depend on the blocking.
#include "internal.hpp"

namespace mdn {

namespace {

constexpr int kNB = 32;        // panel / block width of the factorisation and the solves
constexpr int kGB = 8;         // codebooks per side of a Gram pair block
constexpr int kGW = kGB * kK;  // 128: counts per side of a pair block

__global__ void __launch_bounds__(256) fill_i32_kernel(int32_t* __restrict__ p, int64_t n) {
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n; e += (int64_t)gridDim.x * 256) p[e] = 0;
}

// ------------------------------------------------------------------ gram
__global__ void __launch_bounds__(256)
gram_kernel(const uint8_t* __restrict__ idx, int64_t N, int C, int nbc, int64_t chunk_rows,
            int32_t* __restrict__ H) {
  __shared__ int s_cnt[kGW * kGW];   // 64 KB
  const int tid = threadIdx.x;
  const int npair = nbc * nbc;
  const int pair = blockIdx.x % npair;
  const int64_t chunk = blockIdx.x / npair;
  const int c1 = (pair / nbc) * kGB, c2 = (pair % nbc) * kGB;
  const int n1 = min(kGB, C - c1), n2 = min(kGB, C - c2);
  for (int e = tid; e < kGW * kGW; e += 256) s_cnt[e] = 0;
  __syncthreads();
  const int64_t r0 = chunk * chunk_rows;
  const int64_t r1 = min(N, r0 + chunk_rows);
  for (int64_t n = r0 + tid; n < r1; n += 256) {
    const uint8_t* ir = idx + n * C;
    int ka[kGB], kb[kGB];
#pragma unroll
    for (int a = 0; a < kGB; ++a) ka[a] = a < n1 ? (int)(ir[c1 + a] & 15) : 0;
#pragma unroll
    for (int b = 0; b < kGB; ++b) kb[b] = b < n2 ? (int)(ir[c2 + b] & 15) : 0;
#pragma unroll
    for (int a = 0; a < kGB; ++a)
#pragma unroll
      for (int b = 0; b < kGB; ++b)
        if (a < n1 && b < n2) atomicAdd(&s_cnt[(a * kK + ka[a]) * kGW + b * kK + kb[b]], 1);
  }
  __syncthreads();
  const int64_t n16 = (int64_t)C * kK;
  for (int e = tid; e < kGW * kGW; e += 256) {
    const int v = s_cnt[e];
    const int ra = e / kGW, rb = e % kGW;
    if (v != 0 && ra < n1 * kK && rb < n2 * kK) atomicAdd(&H[(c1 * kK + ra) * n16 + c2 * kK + rb], v);
  }
}

// --------------------------------------------------------------- scatter
// R[16c + k][m] = sum over rows n (ascending) with idx[n][c] = k of Y[n][m].
//
// partition: one wavefront per codebook lists the rows bucket by bucket,
// ascending within each bucket (a stable counting sort: per 64-row batch, one
// ballot per bucket gives each row its rank among the batch's rows of its
// bucket), perm[c][start_k ..] = rows of bucket k, start[c][k] the bucket
// starts (start[c][16] = N).  Each codebook's list is followed by 128 entries
// of row 0, read (and ignored) by the last two batches of the scatter.
constexpr int kPermPad = 128;

__global__ void __launch_bounds__(64)
partition_kernel(const uint8_t* __restrict__ idx, int64_t N, int C, int32_t* __restrict__ perm,
                 int32_t* __restrict__ start) {
  const int lane = threadIdx.x;
  const int c = blockIdx.x;
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));   // lanes below this one
  int64_t cnt[kK];
#pragma unroll
  for (int k = 0; k < kK; ++k) cnt[k] = 0;
  for (int64_t n0 = 0; n0 < N; n0 += 64) {
    const int key = (n0 + lane < N) ? (int)(idx[(n0 + lane) * C + c] & 15) : kK;
#pragma unroll
    for (int k = 0; k < kK; ++k) cnt[k] += __popcll(__ballot(key == k));
  }
  int64_t pos[kK];
  int64_t run = 0;
#pragma unroll
  for (int k = 0; k < kK; ++k) {
    pos[k] = run;
    if (lane == 0) start[c * (kK + 1) + k] = (int32_t)run;
    run += cnt[k];
  }
  if (lane == 0) start[c * (kK + 1) + kK] = (int32_t)N;
  int32_t* pc = perm + (int64_t)c * (N + kPermPad);
  pc[N + lane] = 0;
  pc[N + 64 + lane] = 0;
  for (int64_t n0 = 0; n0 < N; n0 += 64) {
    const int key = (n0 + lane < N) ? (int)(idx[(n0 + lane) * C + c] & 15) : kK;
#pragma unroll
    for (int k = 0; k < kK; ++k) {
      const uint64_t mask = __ballot(key == k);
      if (key == k) pc[pos[k] + __popcll(mask & lt)] = (int32_t)(n0 + lane);
      pos[k] += __popcll(mask);
    }
  }
}

// scatter: one wavefront per (codebook, 64-column tile), lane = column.  The
// codebook's row list is walked in batches of kSR positions (64 for float
// inputs, 32 for double; the next batch's loads in flight while the current
// one is added); a running double
// sum takes the rows in list order and is stored and restarted at each
// bucket end, so every entry is its bucket's rows summed in ascending order.
// V: float (targets Y) or double (gradient residuals); kSR positions per batch
template <class V, int kSR>
__global__ void __launch_bounds__(64)
scatter_kernel(const int32_t* __restrict__ perm, const int32_t* __restrict__ start, int64_t N, int C,
               const V* __restrict__ Y, int M, double* __restrict__ R) {
  __shared__ V s_v[kSR][64];
  const int lane = threadIdx.x;
  const int ntile = (M + 63) / 64;
  const int c = blockIdx.x / ntile;
  const int m = (blockIdx.x % ntile) * 64 + lane;
  const bool ok = m < M;
  const V* yc = Y + min(m, M - 1);
  const int32_t* pc = perm + (int64_t)c * (N + kPermPad);
  const int32_t* sc = start + c * (kK + 1);
  double* rc = R + (int64_t)c * kK * M + m;
  int k = 0;
  int64_t end = sc[1];   // end of bucket k
  double acc = 0.0;
  // store and restart the sums of every bucket that ends at position p
  auto close_buckets = [&](int64_t p) {
    while (k < kK && end == p) {
      if (ok) rc[(int64_t)k * M] = acc;
      acc = 0.0;
      ++k;
      end = (k < kK) ? sc[k + 1] : -1;
    }
  };
  // positions past N read the padding (row 0) and columns past M column
  // M - 1: every load is valid, unused values are ignored; the row numbers
  // are uniform (scalar loads)
  V v[kSR], vn[kSR];
  if (N > 0) {
#pragma unroll
    for (int j = 0; j < kSR; ++j) v[j] = yc[(int64_t)pc[j] * M];
  }
  for (int64_t p0 = 0; p0 < N; p0 += kSR) {
    const int32_t* pn = pc + p0 + kSR;
#pragma unroll
    for (int j = 0; j < kSR; ++j) vn[j] = yc[(int64_t)pn[j] * M];
    if (end >= p0 + kSR) {
      // the whole batch lies in bucket k
#pragma unroll
      for (int j = 0; j < kSR; ++j) acc = __dadd_rn(acc, (double)v[j]);
    } else {
      // a bucket ends inside the batch (at most 16 + 1 batches): position by
      // position, the values parked in LDS (this lane's own column)
#pragma unroll
      for (int j = 0; j < kSR; ++j) s_v[j][lane] = v[j];
#pragma unroll 1
      for (int j = 0; j < kSR; ++j) {
        close_buckets(p0 + j);
        if (p0 + j < N) acc = __dadd_rn(acc, (double)s_v[j][lane]);
      }
    }
#pragma unroll
    for (int j = 0; j < kSR; ++j) v[j] = vn[j];
  }
  close_buckets(N);
}

// -------------------------------------------------------------- assemble
// A = H + lambda I (lower triangle and diagonal; the strict upper triangle
// is never read), B = R + lambda T0 (in place in B).
__global__ void __launch_bounds__(256)
assemble_kernel(const int32_t* __restrict__ H, int64_t n, double lam, double* __restrict__ A,
                double* __restrict__ B, const float* __restrict__ T0, int64_t nb_total) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n * n; e += stride) {
    const int64_t i = e / n, j = e - (e / n) * n;
    if (j <= i) A[e] = (double)H[e] + (i == j ? lam : 0.0);
  }
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < nb_total; e += stride)
    B[e] = __dadd_rn(B[e], __dmul_rn(lam, (double)T0[e]));
}

// ---------------------------------------------------------- factorisation
// diagonal block [j0, j0 + jb) of the panel: unblocked right-looking in LDS
__global__ void __launch_bounds__(256) potrf_diag_kernel(double* __restrict__ A, int64_t n, int j0, int jb) {
  __shared__ double a[kNB][kNB + 1];
  const int tid = threadIdx.x;
  for (int e = tid; e < kNB * kNB; e += 256) {
    const int i = e / kNB, j = e % kNB;
    a[i][j] = (i < jb && j <= i) ? A[(j0 + i) * n + j0 + j] : 0.0;
  }
  __syncthreads();
  for (int j = 0; j < jb; ++j) {
    if (tid == 0) a[j][j] = __dsqrt_rn(a[j][j]);
    __syncthreads();
    const double d = a[j][j];
    for (int i = j + 1 + tid; i < jb; i += 256) a[i][j] = __ddiv_rn(a[i][j], d);
    __syncthreads();
    // update of the columns right of j: entry (i, q), j < q <= i, term k = j
    for (int e = tid; e < kNB * kNB; e += 256) {
      const int i = e / kNB, q = e % kNB;
      if (q > j && q <= i && i < jb) a[i][q] = __fma_rn(-a[i][j], a[q][j], a[i][q]);
    }
    __syncthreads();
  }
  for (int e = tid; e < kNB * kNB; e += 256) {
    const int i = e / kNB, j = e % kNB;
    if (i < jb && j <= i) A[(j0 + i) * n + j0 + j] = a[i][j];
  }
}

// rows [j0 + jb, n) of the panel: L21 = A21 L11^-T, one row per thread
__global__ void __launch_bounds__(256) trsm_panel_kernel(double* __restrict__ A, int64_t n, int j0, int jb) {
  __shared__ double l[kNB][kNB + 1];
  const int tid = threadIdx.x;
  for (int e = tid; e < kNB * kNB; e += 256) {
    const int i = e / kNB, j = e % kNB;
    l[i][j] = (i < jb && j <= i) ? A[(j0 + i) * n + j0 + j] : 0.0;
  }
  __syncthreads();
  const int64_t row = (int64_t)j0 + jb + (int64_t)blockIdx.x * 256 + tid;
  if (row >= n) return;
  double* ar = A + row * n + j0;
  double x[kNB];
#pragma unroll
  for (int j = 0; j < kNB; ++j) x[j] = j < jb ? ar[j] : 0.0;
#pragma unroll
  for (int j = 0; j < kNB; ++j) {
    if (j < jb) {
      x[j] = __ddiv_rn(x[j], l[j][j]);
#pragma unroll
      for (int q = j + 1; q < kNB; ++q) x[q] = __fma_rn(-x[j], l[q][j], x[q]);
    }
  }
#pragma unroll
  for (int j = 0; j < kNB; ++j)
    if (j < jb) ar[j] = x[j];
}

// trailing update: A[i][q] -= sum_{k in panel, ascending} L[i][k] L[q][k] for
// j0 + jb <= q <= i < n; a 32 x 32 tile per workgroup (lower tiles only)
__global__ void __launch_bounds__(256) syrk_kernel(double* __restrict__ A, int64_t n, int j0, int jb) {
  __shared__ double li[kNB][kNB + 1];
  __shared__ double lq[kNB][kNB + 1];
  const int tid = threadIdx.x;
  // tile (ti, tq), ti >= tq, from the linear block index
  int ti = 0;
  const int b = blockIdx.x;
  while ((ti + 1) * (ti + 2) / 2 <= b) ++ti;
  const int tq = b - ti * (ti + 1) / 2;
  const int64_t s = (int64_t)j0 + jb;
  const int64_t i0 = s + (int64_t)ti * kNB, q0 = s + (int64_t)tq * kNB;
  for (int e = tid; e < kNB * kNB; e += 256) {
    const int r = e / kNB, k = e % kNB;
    li[r][k] = (i0 + r < n && k < jb) ? A[(i0 + r) * n + j0 + k] : 0.0;
    lq[r][k] = (q0 + r < n && k < jb) ? A[(q0 + r) * n + j0 + k] : 0.0;
  }
  __syncthreads();
  const int ty = tid / 16, tx = tid % 16;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int r = ty + 16 * a, q = tx + 16 * c;
      const int64_t gi = i0 + r, gq = q0 + q;
      if (gi < n && gq <= gi) {
        double v = A[gi * n + gq];
        for (int k = 0; k < jb; ++k) v = __fma_rn(-li[r][k], lq[q][k], v);
        A[gi * n + gq] = v;
      }
    }
}

// ------------------------------------------------------------------ solves
// B [n][M] in place.  Forward: z_i = (b_i - sum_{k < i} L[i][k] z_k) / L[i][i],
// k ascending; backward: t_i = (z_i - sum_{k > i} L[k][i] t_k) / L[i][i], k
// descending.  Blocks of 32 rows; the diagonal block one column per thread,
// the update of the other rows as 32 x 64 tiles.
template <bool FWD>
__global__ void __launch_bounds__(256) trsv_diag_kernel(const double* __restrict__ A, int64_t n, double* __restrict__ B,
                                                         int M, int i0, int ib) {
  __shared__ double l[kNB][kNB + 1];
  const int tid = threadIdx.x;
  for (int e = tid; e < kNB * kNB; e += 256) {
    const int i = e / kNB, j = e % kNB;
    l[i][j] = (i < ib && j <= i) ? A[(i0 + i) * n + i0 + j] : 0.0;
  }
  __syncthreads();
  const int64_t m = (int64_t)blockIdx.x * 256 + tid;
  if (m >= M) return;
  double x[kNB];
#pragma unroll
  for (int i = 0; i < kNB; ++i) x[i] = i < ib ? B[(i0 + i) * (int64_t)M + m] : 0.0;
  if (FWD) {
#pragma unroll
    for (int i = 0; i < kNB; ++i) {
      if (i < ib) {
        x[i] = __ddiv_rn(x[i], l[i][i]);
#pragma unroll
        for (int q = i + 1; q < kNB; ++q) x[q] = __fma_rn(-l[q][i], x[i], x[q]);
      }
    }
  } else {
#pragma unroll
    for (int i = kNB - 1; i >= 0; --i) {
      if (i < ib) {
        x[i] = __ddiv_rn(x[i], l[i][i]);
#pragma unroll
        for (int q = 0; q < i; ++q) x[q] = __fma_rn(-l[i][q], x[i], x[q]);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < kNB; ++i)
    if (i < ib) B[(i0 + i) * (int64_t)M + m] = x[i];
}

// FWD: rows r >= i0 + ib get the block's terms, k ascending: b_r -= L[r][k] z_k.
// !FWD: rows r < i0 get them, k descending: b_r -= L[k][r] t_k.
template <bool FWD>
__global__ void __launch_bounds__(256) trsv_update_kernel(const double* __restrict__ A, int64_t n, double* __restrict__ B,
                                                           int M, int i0, int ib) {
  __shared__ double lr[kNB][kNB + 1];   // lr[r][k]: the coefficient of block row k in row r
  __shared__ double z[kNB][64];
  const int tid = threadIdx.x;
  const int ntm = (M + 63) / 64;
  const int64_t r0 = FWD ? (int64_t)i0 + ib + (int64_t)(blockIdx.x / ntm) * kNB : (int64_t)(blockIdx.x / ntm) * kNB;
  const int64_t rend = FWD ? n : i0;
  const int64_t m0 = (int64_t)(blockIdx.x % ntm) * 64;
  for (int e = tid; e < kNB * kNB; e += 256) {
    const int r = e / kNB, k = e % kNB;
    const int64_t gr = r0 + r;
    double v = 0.0;
    if (gr < rend && k < ib) v = FWD ? A[gr * n + i0 + k] : A[(i0 + k) * n + gr];
    lr[r][k] = v;
  }
  for (int e = tid; e < kNB * 64; e += 256) {
    const int k = e / 64, c = e % 64;
    z[k][c] = (k < ib && m0 + c < M) ? B[(i0 + k) * (int64_t)M + m0 + c] : 0.0;
  }
  __syncthreads();
  const int c = tid % 64;
  const int rr = tid / 64;   // rows rr, rr + 4, ..., 8 per thread
  if (m0 + c >= M) return;
#pragma unroll
  for (int a = 0; a < kNB / 4; ++a) {
    const int r = rr + 4 * a;
    const int64_t gr = r0 + r;
    if (gr >= rend) continue;
    double v = B[gr * (int64_t)M + m0 + c];
    if (FWD) {
      for (int k = 0; k < ib; ++k) v = __fma_rn(-lr[r][k], z[k][c], v);
    } else {
      for (int k = ib - 1; k >= 0; --k) v = __fma_rn(-lr[r][k], z[k][c], v);
    }
    B[gr * (int64_t)M + m0 + c] = v;
  }
}

// ------------------------------------------- nonlinear output: gradient descent
// z_n = (sum_c T[c][idx[n][c]][.], c ascending) + b.  One wavefront per row,
// lanes over columns; the row's indices are uniform (scalar loads).
__device__ __forceinline__ double wave_max(double v) {
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ double wave_sum(double v) {
  for (int o = 32; o > 0; o >>= 1) v = __dadd_rn(v, __shfl_xor(v, o));
  return v;
}

// Softmax of the row held in out[0..M) (in place): maximum subtracted, exp,
// sum, division.
__device__ void softmax_row_inplace(double* __restrict__ out, int M, int lane) {
  double mx = -__builtin_inf();
  for (int m = lane; m < M; m += 64) mx = fmax(mx, out[m]);
  mx = wave_max(mx);
  double sum = 0.0;
  for (int m = lane; m < M; m += 64) {
    const double e = exp(__dsub_rn(out[m], mx));
    out[m] = e;
    sum = __dadd_rn(sum, e);
  }
  sum = wave_sum(sum);
  for (int m = lane; m < M; m += 64) out[m] = __ddiv_rn(out[m], sum);
}

// P = sigma(Y + b): ReLU (act 2) or row softmax (acts 3 and 4), in double
__global__ void __launch_bounds__(256)
target_kernel(const float* __restrict__ Y, int64_t N, int M, const float* __restrict__ bias, int act,
              double* __restrict__ P) {
  const int lane = threadIdx.x & 63;
  for (int64_t n = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); n < N; n += (int64_t)gridDim.x * 4) {
    double* pr = P + n * M;
    for (int m = lane; m < M; m += 64) {
      const double z = __dadd_rn((double)Y[n * M + m], bias ? (double)bias[m] : 0.0);
      pr[m] = (act == 2) ? (z > 0.0 ? z : 0.0) : z;
    }
    if (act >= 3) softmax_row_inplace(pr, M, lane);
  }
}

// D = dObjective / dz per row: ReLU 2 (relu(z) - P) [z > 0]; softmax with the
// KL divergence softmax(z) - P; softmax with the squared error 2 p (d - s),
// p = softmax(z), d = p - P, s = sum_m d_m p_m (the softmax Jacobian
// diag(p) - p p^T applied to 2 d).
__global__ void __launch_bounds__(256)
resid_kernel(const uint8_t* __restrict__ idx, int64_t N, int C, const double* __restrict__ T, int M,
             const float* __restrict__ bias, int act, const double* __restrict__ P, double* __restrict__ D) {
  const int lane = threadIdx.x & 63;
  for (int64_t n = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); n < N; n += (int64_t)gridDim.x * 4) {
    const uint8_t* ir = idx + n * C;
    double* dr = D + n * M;
    const double* pr = P + n * M;
    for (int m = lane; m < M; m += 64) {
      double s = 0.0;
      for (int c = 0; c < C; ++c) s = __dadd_rn(s, T[((int64_t)c * kK + (ir[c] & 15)) * M + m]);
      const double z = __dadd_rn(s, bias ? (double)bias[m] : 0.0);
      dr[m] = (act == 2) ? (z > 0.0 ? __dmul_rn(2.0, __dsub_rn(z, pr[m])) : 0.0) : z;
    }
    if (act == 3) {
      softmax_row_inplace(dr, M, lane);
      for (int m = lane; m < M; m += 64) dr[m] = __dsub_rn(dr[m], pr[m]);
    } else if (act == 4) {
      softmax_row_inplace(dr, M, lane);
      double s = 0.0;
      for (int m = lane; m < M; m += 64) s = __dadd_rn(s, __dmul_rn(__dsub_rn(dr[m], pr[m]), dr[m]));
      s = wave_sum(s);
      for (int m = lane; m < M; m += 64) {
        const double p = dr[m];
        dr[m] = __dmul_rn(2.0, __dmul_rn(p, __dsub_rn(__dsub_rn(p, pr[m]), s)));
      }
    }
  }
}

// T = T - eta (R + 2 lambda (T - T0))
__global__ void __launch_bounds__(256)
gd_update_kernel(double* __restrict__ T, const float* __restrict__ T0, const double* __restrict__ R, double lam,
                 double eta, int64_t total) {
  const double two_lam = __dmul_rn(2.0, lam);
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const double g = __dadd_rn(R[e], __dmul_rn(two_lam, __dsub_rn(T[e], (double)T0[e])));
    T[e] = __dsub_rn(T[e], __dmul_rn(eta, g));
  }
}

__global__ void __launch_bounds__(256) copy_f32_f64_kernel(const float* __restrict__ a, double* __restrict__ b,
                                                           int64_t total) {
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256)
    b[e] = (double)a[e];
}

unsigned grid_1d(int64_t total, int per) {
  int64_t g = (total + per - 1) / per;
  if (g < 1) g = 1;
  if (g > 65536) g = 65536;
  return (unsigned)g;
}

}  // namespace

hipError_t launch_gram(const uint8_t* idx, int64_t N, int C, int32_t* H, int cus, hipStream_t stream) {
  const int64_t n16 = (int64_t)C * kK;
  hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_1d(n16 * n16, 256)), dim3(256), 0, stream, H, n16 * n16);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || N == 0) return e;
  const int nbc = (C + kGB - 1) / kGB;
  const int64_t npair = (int64_t)nbc * nbc;
  // about four workgroups per CU in all, chunks of at least 256 rows
  int64_t chunks = ((int64_t)4 * cus + npair - 1) / npair;
  const int64_t max_chunks = (N + 255) / 256;
  if (chunks > max_chunks) chunks = max_chunks;
  if (chunks < 1) chunks = 1;
  const int64_t chunk_rows = (N + chunks - 1) / chunks;
  chunks = (N + chunk_rows - 1) / chunk_rows;
  hipLaunchKernelGGL(gram_kernel, dim3((unsigned)(npair * chunks)), dim3(256), 0, stream, idx, N, C, nbc,
                     chunk_rows, H);
  return hipGetLastError();
}

hipError_t launch_partition(const uint8_t* idx, int64_t N, int C, int32_t* perm, int32_t* start,
                            hipStream_t stream) {
  hipLaunchKernelGGL(partition_kernel, dim3((unsigned)C), dim3(64), 0, stream, idx, N, C, perm, start);
  return hipGetLastError();
}

template <class V, int kSR>
hipError_t launch_scatter_sorted(const int32_t* perm, const int32_t* start, int64_t N, int C, const V* Y, int M,
                                 double* R, hipStream_t stream) {
  const int ntile = (M + 63) / 64;
  hipLaunchKernelGGL((scatter_kernel<V, kSR>), dim3((unsigned)(C * ntile)), dim3(64), 0, stream, perm, start, N, C,
                     Y, M, R);
  return hipGetLastError();
}

hipError_t launch_scatter(const uint8_t* idx, int64_t N, int C, const float* Y, int M, double* R,
                          int32_t* perm, int32_t* start, hipStream_t stream) {
  hipError_t e = launch_partition(idx, N, C, perm, start, stream);
  if (e != hipSuccess) return e;
  return launch_scatter_sorted<float, 64>(perm, start, N, C, Y, M, R, stream);
}

hipError_t launch_fit_ridge(const uint8_t* idx, int64_t N, int C, const float* Y, int M, const float* T0,
                            double lam, double* T, int32_t* H, double* A, int32_t* perm, int32_t* start,
                            int cus, hipStream_t stream) {
  const int64_t n = (int64_t)C * kK;
  hipError_t e = launch_gram(idx, N, C, H, cus, stream);
  if (e != hipSuccess) return e;
  e = launch_scatter(idx, N, C, Y, M, T, perm, start, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(assemble_kernel, dim3(grid_1d(n * n, 256)), dim3(256), 0, stream, H, n, lam, A, T, T0,
                     n * M);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  for (int j0 = 0; j0 < n; j0 += kNB) {
    const int jb = (int)((n - j0) < kNB ? (n - j0) : kNB);
    hipLaunchKernelGGL(potrf_diag_kernel, dim3(1), dim3(256), 0, stream, A, n, j0, jb);
    const int64_t below = n - j0 - jb;
    if (below > 0) {
      hipLaunchKernelGGL(trsm_panel_kernel, dim3(grid_1d(below, 256)), dim3(256), 0, stream, A, n, j0, jb);
      const int64_t tiles = (below + kNB - 1) / kNB;
      hipLaunchKernelGGL(syrk_kernel, dim3((unsigned)(tiles * (tiles + 1) / 2)), dim3(256), 0, stream, A, n, j0,
                         jb);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const int ntm = (M + 63) / 64;
  for (int i0 = 0; i0 < n; i0 += kNB) {   // forward
    const int ib = (int)((n - i0) < kNB ? (n - i0) : kNB);
    hipLaunchKernelGGL(trsv_diag_kernel<true>, dim3(grid_1d(M, 256)), dim3(256), 0, stream, A, n, T, M, i0, ib);
    const int64_t below = n - i0 - ib;
    if (below > 0)
      hipLaunchKernelGGL(trsv_update_kernel<true>, dim3((unsigned)(((below + kNB - 1) / kNB) * ntm)), dim3(256), 0,
                         stream, A, n, T, M, i0, ib);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const int64_t last = ((n - 1) / kNB) * kNB;
  for (int64_t i0 = last; i0 >= 0; i0 -= kNB) {   // backward
    const int ib = (int)((n - i0) < kNB ? (n - i0) : kNB);
    hipLaunchKernelGGL(trsv_diag_kernel<false>, dim3(grid_1d(M, 256)), dim3(256), 0, stream, A, n, T, M, (int)i0,
                       ib);
    if (i0 > 0)
      hipLaunchKernelGGL(trsv_update_kernel<false>, dim3((unsigned)(((i0 + kNB - 1) / kNB) * ntm)), dim3(256), 0,
                         stream, A, n, T, M, (int)i0, ib);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_fit_gd(const uint8_t* idx, int64_t N, int C, const float* Y, int M, const float* bias, int act,
                         const float* T0, double lam, double eta, int iters, double* T, double* P, double* D,
                         double* R, int32_t* perm, int32_t* start, hipStream_t stream) {
  const int64_t total = (int64_t)C * kK * M;
  hipLaunchKernelGGL(copy_f32_f64_kernel, dim3(grid_1d(total, 256)), dim3(256), 0, stream, T0, T, total);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || iters == 0) return e;
  if ((e = launch_partition(idx, N, C, perm, start, stream)) != hipSuccess) return e;
  const unsigned rows = grid_1d((N + 3) / 4, 1);   // 4 rows per workgroup, rows looped past 65536 groups
  if (N > 0) {
    hipLaunchKernelGGL(target_kernel, dim3(rows), dim3(256), 0, stream, Y, N, M, bias, act, P);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  for (int it = 0; it < iters; ++it) {
    if (N > 0) {
      hipLaunchKernelGGL(resid_kernel, dim3(rows), dim3(256), 0, stream, idx, N, C, T, M, bias, act, P, D);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if ((e = launch_scatter_sorted<double, 32>(perm, start, N, C, D, M, R, stream)) != hipSuccess) return e;
    hipLaunchKernelGGL(gd_update_kernel, dim3(grid_1d(total, 256)), dim3(256), 0, stream, T, T0, R, lam, eta, total);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace mdn
