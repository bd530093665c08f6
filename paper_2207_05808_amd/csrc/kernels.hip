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

namespace mdn {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
#define MDN_CONST __attribute__((address_space(4)))

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Exponent of a normal fp32 power of two: scale = 2^e.
__device__ __forceinline__ int exp_of_bits(uint32_t bits) { return (int)((bits >> 23) & 0xffu) - 127; }

__device__ __forceinline__ uint32_t bfe(uint32_t v, int off, int width) {
  return __builtin_amdgcn_ubfe(v, off, width);
}

// Rows of a strided 2-D byte array, RW rows per chunk, prefetched in 16-byte
// units through VGPRs.  Unit j of lane l is u = l + 64 j; it belongs to row
// u / upr and column unit u % upr.
template <int PF, bool NT>
struct Prefetch {
  u32x4 buf[PF > 0 ? PF : 1];
  int goff[PF > 0 ? PF : 1];   // byte offset from the chunk's first row in global memory
  int loff[PF > 0 ? PF : 1];   // byte offset in the LDS buffer, -1 when idle
  int rrow[PF > 0 ? PF : 1];   // row within the chunk (1 << 30 when idle)

  __device__ __forceinline__ void init(int lane, int rw, int upr, int64_t src_rs, int lds_rs) {
#pragma unroll
    for (int j = 0; j < PF; ++j) {
      const int u = lane + 64 * j;
      if (u < rw * upr) {
        const int r = u / upr;
        const int col = u - r * upr;
        goff[j] = (int)(r * src_rs) + col * 16;
        loff[j] = r * lds_rs + col * 16;
        rrow[j] = r;
      } else {
        goff[j] = 0;
        loff[j] = -1;
        rrow[j] = 1 << 30;
      }
    }
  }
  __device__ __forceinline__ void load(const char* base, int rows_valid) {
#pragma unroll
    for (int j = 0; j < PF; ++j) {
      if (rrow[j] < rows_valid) {
        const u32x4* p = reinterpret_cast<const u32x4*>(base + goff[j]);
        buf[j] = NT ? __builtin_nontemporal_load(p) : *p;
      }
    }
  }
  __device__ __forceinline__ void store(char* lds) const {
#pragma unroll
    for (int j = 0; j < PF; ++j)
      if (loff[j] >= 0) *reinterpret_cast<u32x4*>(lds + loff[j]) = buf[j];
  }
};

template <int MODE, int ELEM, int PF, int UQ>
__global__ void __launch_bounds__(512) path_kernel(const KArgs a) {
  constexpr bool kEnc = MODE != kAccum;
  constexpr bool kAcc = MODE != kEncode;
  constexpr int kQB = ELEM == kI8 ? 4 : 16;  // bytes of one 4-column quad of a LUT row
  extern __shared__ __attribute__((aligned(16))) char smem[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int nw = blockDim.x >> 6;
  const int C = a.C;
  const int m0 = blockIdx.y * a.Mt;
  const int mt = min(a.Mt, a.M - m0);   // columns of this tile
  const int nq = (mt + 3) >> 2;         // column quads of this tile

  char* s_lut = smem + a.L.lut;
  float* s_thr = reinterpret_cast<float*>(smem + a.L.thr);
  int* s_split = reinterpret_cast<int*>(smem + a.L.split);
  int* s_misc = reinterpret_cast<int*>(smem + a.L.misc);

  // ---------------- workgroup prologue ----------------
  if (kAcc) {
    const int rows = C * kK;
    // quads per LDS row, padded to a power of two so the index split is a shift
    int qlog = 0;
    while ((1 << qlog) < nq) ++qlog;
    const int total = rows << qlog;
    if (ELEM == kI8) {
      if (a.vec_out) {  // M % 4 == 0 and 4-byte aligned table: dword copies
        const uint32_t* src = reinterpret_cast<const uint32_t*>(a.lut);
        const int m4 = a.M >> 2;
        for (int u = tid; u < total; u += blockDim.x) {
          const int row = u >> qlog, q = u & ((1 << qlog) - 1);
          if (q < nq)
            *reinterpret_cast<uint32_t*>(s_lut + row * a.lut_rs + 4 * q) =
                src[(int64_t)row * m4 + (m0 >> 2) + q];
        }
      } else {
        const int8_t* src = reinterpret_cast<const int8_t*>(a.lut);
        for (int u = tid; u < (rows << (qlog + 2)); u += blockDim.x) {
          const int row = u >> (qlog + 2), j = u & ((4 << qlog) - 1);
          if (j < 4 * nq)
            s_lut[row * a.lut_rs + j] = (j < mt) ? src[(int64_t)row * a.M + m0 + j] : (int8_t)0;
        }
      }
    } else {
      const float* src = reinterpret_cast<const float*>(a.lut);
      for (int u = tid; u < (rows << (qlog + 2)); u += blockDim.x) {
        const int row = u >> (qlog + 2), j = u & ((4 << qlog) - 1);
        if (j < 4 * nq)
          *reinterpret_cast<float*>(s_lut + row * a.lut_rs + 4 * j) =
              (j < mt) ? src[(int64_t)row * a.M + m0 + j] : 0.0f;
      }
    }
  }
  if (kEnc) {
    for (int u = tid; u < C * 16; u += blockDim.x) {
      const int c = u >> 4, j = u & 15;
      s_thr[u] = (j < kNodes) ? a.thr[c * kNodes + j] : 0.0f;
    }
    for (int u = tid; u < C * kLevels; u += blockDim.x) {
      const unsigned s = (unsigned)a.split[u];
      s_split[u] = (int)min(s, (unsigned)(a.D - 1));  // memory safety only
    }
  }
  if (kAcc && ELEM == kI8) {
    if (tid == 0) { s_misc[0] = 1 << 30; s_misc[1] = 0; }
    __syncthreads();
    const uint32_t* sb = reinterpret_cast<const uint32_t*>(a.scale);
    for (int c = tid; c < C; c += blockDim.x) atomicMin(&s_misc[0], exp_of_bits(sb[c]));
    __syncthreads();
    const int emin = s_misc[0];
    for (int c = tid; c < C; c += blockDim.x) atomicMax(&s_misc[1], exp_of_bits(sb[c]) - emin);
    if (tid == 0) {
      double s = 0.0;  // bias32: double sum over codebooks in ascending order
      for (int c = 0; c < C; ++c) s += (double)a.offset[c];
      s_misc[2] = __float_as_int((float)s);
      s_misc[3] = __float_as_int(__builtin_ldexpf(1.0f, emin));
    }
  }
  __syncthreads();

  // ---------------- per-wavefront chunk loop ----------------
  const int RW = a.RW;
  float* sA = reinterpret_cast<float*>(smem + a.L.a) + (size_t)wave * RW * a.Dp;
  uint8_t* sI = reinterpret_cast<uint8_t*>(smem + a.L.idx) + (size_t)wave * RW * a.Cp;
  const int64_t tw = (int64_t)gridDim.x * nw;
  int64_t ch = (int64_t)blockIdx.x * nw + wave;

  // source rows of this mode: rows of A (encode) or of idx (accumulate)
  const char* src0 = kEnc ? reinterpret_cast<const char*>(a.A) : reinterpret_cast<const char*>(a.idx_in);
  const int64_t src_rs = kEnc ? a.lda * 4 : (int64_t)C;  // bytes between rows
  Prefetch<PF, kEnc> pf;
  if (PF > 0) {
    if (kEnc) pf.init(lane, RW, a.D >> 2, src_rs, a.Dp * 4);
    else      pf.init(lane, RW, C >> 4, src_rs, a.Cp);
    if (ch < a.nchunks) {
      const int64_t row0 = ch << a.rw_log2;
      pf.load(src0 + row0 * src_rs, (int)min<int64_t>(RW, a.N - row0));
    }
  }

  // accumulate-phase lane mapping
  const int lpr_log2 = 6 - a.rw_log2;
  const int ar = lane >> lpr_log2;                  // row of the chunk
  const int cg = lane & ((1 << lpr_log2) - 1);      // first column quad
  const int LPR = 1 << lpr_log2;
  int emin = 0, maxsh = 0;
  float step = 1.0f, bias = 0.0f;
  if (kAcc && ELEM == kI8) {
    emin = uniform(s_misc[0]);
    maxsh = uniform(s_misc[1]);
    bias = __int_as_float(uniform(s_misc[2]));
    step = __int_as_float(uniform(s_misc[3]));
  }
  const MDN_CONST uint32_t* cscale = (const MDN_CONST uint32_t*)(uintptr_t)a.scale;

  for (; ch < a.nchunks; ch += tw) {
    const int64_t row0 = ch << a.rw_log2;
    const int rows_valid = (int)min<int64_t>(RW, a.N - row0);

    // 1. stage this chunk's rows in LDS
    if (PF > 0) {
      pf.store(kEnc ? reinterpret_cast<char*>(sA) : reinterpret_cast<char*>(sI));
      const int64_t nx = ch + tw;
      if (nx < a.nchunks) {
        const int64_t nrow0 = nx << a.rw_log2;
        pf.load(src0 + nrow0 * src_rs, (int)min<int64_t>(RW, a.N - nrow0));
      }
    } else if (kEnc) {
      for (int r = 0; r < rows_valid; ++r) {
        const float* src = a.A + (row0 + r) * a.lda;
        for (int col = lane; col < a.D; col += 64) sA[r * a.Dp + col] = src[col];
      }
    } else {
      for (int r = 0; r < rows_valid; ++r) {
        const uint8_t* src = a.idx_in + (row0 + r) * (int64_t)C;
        for (int col = lane; col < C; col += 64) sI[r * a.Cp + col] = src[col];
      }
    }
    wave_sync();

    // 2. encode: 4 comparisons per (row, codebook)
    if (kEnc) {
      for (int p = lane; p < RW * C; p += 64) {
        const int r = (C == 1) ? p : (int)__umulhi((uint32_t)p, a.c_magic);
        const int c = p - r * C;
        const float* xr = sA + r * a.Dp;
        const int* sp = s_split + c * kLevels;
        const float* th = s_thr + c * 16;
        int i = (xr[sp[0]] > th[0]) ? 1 : 0;
        i = 2 * i + ((xr[sp[1]] > th[1 + i]) ? 1 : 0);
        i = 2 * i + ((xr[sp[2]] > th[3 + i]) ? 1 : 0);
        i = 2 * i + ((xr[sp[3]] > th[7 + i]) ? 1 : 0);
        sI[r * a.Cp + c] = (uint8_t)i;
      }
      wave_sync();
      if (a.idx_out != nullptr) {
        if (a.Cp == C && ((reinterpret_cast<uintptr_t>(a.idx_out) & 3) == 0)) {
          uint32_t* dst = reinterpret_cast<uint32_t*>(a.idx_out + row0 * C);
          const uint32_t* s32 = reinterpret_cast<const uint32_t*>(sI);
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
      const uint8_t* ir = sI + ar * a.Cp;
      const char* lut_lane = s_lut + cg * kQB;
      const int64_t row = row0 + ar;
      if (ELEM == kI8) {
        int acc[UQ][4];
#pragma unroll
        for (int u = 0; u < UQ; ++u)
#pragma unroll
          for (int b = 0; b < 4; ++b) acc[u][b] = 0;
        if (maxsh <= 6) {
          for (int c0 = 0; c0 < C; c0 += 4) {
            const uint32_t kw = *reinterpret_cast<const uint32_t*>(ir + c0);
#pragma unroll
            for (int b = 0; b < 4; ++b) {
              const int c = c0 + b;
              if (c < C) {
                const int w = 1 << (exp_of_bits(cscale[c]) - emin);
                const int k = (int)bfe(kw, 8 * b, 4);
                const char* rowp = lut_lane + (c * kK + k) * a.lut_rs;
#pragma unroll
                for (int u = 0; u < UQ; ++u) {
                  if (UQ == 1 || cg + u * LPR < nq) {
                    const int v = *reinterpret_cast<const int*>(rowp + u * LPR * kQB);
                    acc[u][0] = __builtin_amdgcn_sdot4(v, w, acc[u][0], false);
                    acc[u][1] = __builtin_amdgcn_sdot4(v, w << 8, acc[u][1], false);
                    acc[u][2] = __builtin_amdgcn_sdot4(v, w << 16, acc[u][2], false);
                    acc[u][3] = __builtin_amdgcn_sdot4(v, w << 24, acc[u][3], false);
                  }
                }
              }
            }
          }
        } else {
          for (int c0 = 0; c0 < C; c0 += 4) {
            const uint32_t kw = *reinterpret_cast<const uint32_t*>(ir + c0);
#pragma unroll
            for (int b = 0; b < 4; ++b) {
              const int c = c0 + b;
              if (c < C) {
                const int sh = exp_of_bits(cscale[c]) - emin;
                const int k = (int)bfe(kw, 8 * b, 4);
                const char* rowp = lut_lane + (c * kK + k) * a.lut_rs;
#pragma unroll
                for (int u = 0; u < UQ; ++u) {
                  if (UQ == 1 || cg + u * LPR < nq) {
                    const int v = *reinterpret_cast<const int*>(rowp + u * LPR * kQB);
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                      acc[u][e] += __builtin_amdgcn_sbfe(v, 8 * e, 8) << sh;
                  }
                }
              }
            }
          }
        }
        if (ar < rows_valid) {
#pragma unroll
          for (int u = 0; u < UQ; ++u) {
            const int q = cg + u * LPR;
            if (q < nq) {
              const int mloc = 4 * q;
              float o[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) o[e] = __builtin_fmaf((float)acc[u][e], step, bias);
              float* yp = a.y ? a.y + row * a.M + m0 + mloc : nullptr;
              int32_t* ap = a.acc ? a.acc + row * a.M + m0 + mloc : nullptr;
              if (a.vec_out && mloc + 4 <= mt) {
                if (yp) __builtin_nontemporal_store((f32x4){o[0], o[1], o[2], o[3]}, reinterpret_cast<f32x4*>(yp));
                if (ap) __builtin_nontemporal_store((u32x4){(uint32_t)acc[u][0], (uint32_t)acc[u][1],
                                                            (uint32_t)acc[u][2], (uint32_t)acc[u][3]},
                                                    reinterpret_cast<u32x4*>(ap));
              } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                  if (mloc + e < mt) {
                    if (yp) yp[e] = o[e];
                    if (ap) ap[e] = acc[u][e];
                  }
                }
              }
            }
          }
        }
      } else {
        float acc[UQ][4];
#pragma unroll
        for (int u = 0; u < UQ; ++u)
#pragma unroll
          for (int b = 0; b < 4; ++b) acc[u][b] = 0.0f;
        for (int c0 = 0; c0 < C; c0 += 4) {
          const uint32_t kw = *reinterpret_cast<const uint32_t*>(ir + c0);
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const int c = c0 + b;
            if (c < C) {
              const int k = (int)bfe(kw, 8 * b, 4);
              const char* rowp = lut_lane + (c * kK + k) * a.lut_rs;
#pragma unroll
              for (int u = 0; u < UQ; ++u) {
                if (UQ == 1 || cg + u * LPR < nq) {
                  const f32x4 v = *reinterpret_cast<const f32x4*>(rowp + u * LPR * kQB);
                  acc[u][0] = acc[u][0] + v.x;
                  acc[u][1] = acc[u][1] + v.y;
                  acc[u][2] = acc[u][2] + v.z;
                  acc[u][3] = acc[u][3] + v.w;
                }
              }
            }
          }
        }
        if (ar < rows_valid) {
#pragma unroll
          for (int u = 0; u < UQ; ++u) {
            const int q = cg + u * LPR;
            if (q < nq) {
              const int mloc = 4 * q;
              float* yp = a.y + row * a.M + m0 + mloc;
              if (a.vec_out && mloc + 4 <= mt) {
                __builtin_nontemporal_store((f32x4){acc[u][0], acc[u][1], acc[u][2], acc[u][3]},
                                            reinterpret_cast<f32x4*>(yp));
              } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                  if (mloc + e < mt) yp[e] = acc[u][e];
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

#define MDN_CASE(MODE, ELEM, PF, UQ)                                                  \
  if (mode == MODE && elem == ELEM && pf == PF && uq == UQ) {                         \
    hipLaunchKernelGGL((path_kernel<MODE, ELEM, PF, UQ>), grid, block, a.L.total,     \
                       stream, a);                                                    \
    return hipGetLastError();                                                         \
  }

static hipError_t set_lds_limit(int mode, int elem, int pf, int uq, int bytes);

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
  (void)set_lds_limit;
  return hipErrorInvalidValue;
}

static hipError_t set_lds_limit(int, int, int, int, int) { return hipSuccess; }

}  // namespace mdn
