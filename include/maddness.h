/*
 * maddness.h -- C ABI of the MI355X (gfx950) library for the inference path
 * of the MADDNESS-style approximate matrix product studied in McCarter &
 * Dronen, "Look-ups are not (yet) all you need for deep learning inference".
 *
 * The product A B (A: N x D activations, B: D x M weights known in advance,
 * §1) is approximated by product quantization: each row of A is hashed, per
 * codebook c, to one of K = 16 prototypes by a balanced 4-level binary tree
 * (§1; §2.1: four comparisons per codebook), and the result is the sum over the C
 * codebooks of the rows of precomputed tables T_c = P_c B (§1; §2.2) picked
 * by those indices.  The tables are stored in 8-bit block floating point
 * (§1): int8 codes with a power-of-two scale and an fp32 offset per codebook.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every array argument is a DEVICE pointer owned by the caller.  The
 *    library keeps no pointer after the call returns; the caller keeps the
 *    buffers alive until the work on `stream` has completed.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).  The
 *    calls only enqueue work on it: no host synchronisation and no device
 *    allocation, so every call can be captured in a HIP graph.  Where a call
 *    needs device memory beyond its inputs and outputs, the caller passes it:
 *    the index array of the fused entry points for tables too large for
 *    their single-launch kernels or where two phases are faster
 *    (maddness_matmul_index_bytes), and the
 *    workspaces of the table fit.
 *  - Row-major layouts.  A has row stride `lda` (elements, lda >= D); every
 *    other array is dense.
 *  - Return value: MADDNESS_OK or an error status (never aborts, never
 *    throws).  Argument checks run before any HIP call, so they work on a
 *    machine without a GPU.  N == 0 is valid and enqueues nothing.
 *  - Device-array CONTENTS are preconditions that the hot path does not
 *    check: split dims in [0, D) (kernels clamp them for memory safety only),
 *    indices in [0, 16), scales exact normal fp32 powers of two with
 *    128 * sum_c 2^(e_c - e_min) <= 2^31 (so that no sum of int8 codes,
 *    -128 included, leaves int32).  Violations give unspecified values,
 *    never out-of-bounds accesses.
 *  - Output arrays must not overlap each other or any input array of the same
 *    call (kernels may read inputs, indices in particular, through the scalar
 *    cache while outputs are being written).  Inputs may overlap each other.
 *  - Thread safety: the global state is a per-kernel cache of launch
 *    attributes and the per-device address of maddness_matmul_noalloc's
 *    scratch array, each filled once under a mutex; concurrent calls on
 *    different streams are independent, except calls of
 *    maddness_matmul_noalloc on one device (see there).
 */
#ifndef MADDNESS_H
#define MADDNESS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    MADDNESS_OK = 0,
    MADDNESS_EINVAL = 1,       /* bad size, NULL or misaligned pointer      */
    MADDNESS_EHIP = 2,         /* a HIP runtime call or a launch failed     */
    MADDNESS_EUNSUPPORTED = 3, /* shape beyond what the kernels handle      */
    MADDNESS_ENOMEM = 4        /* reserved: no entry point allocates         */
};

/* Layer output sigma for maddness_matmul_act[_f32] (§2.2: the bias term
   composed with an elementwise or a row-wise nonlinearity). */
enum {
    MADDNESS_ACT_NONE = 0,     /* y                                          */
    MADDNESS_ACT_BIAS = 1,     /* z = y + bias[m]                            */
    MADDNESS_ACT_RELU = 2,     /* z > 0 ? z : +0                             */
    MADDNESS_ACT_SOFTMAX = 3   /* softmax of z over the M outputs of a row   */
};

/* Objectives of the gradient-descent table fit, maddness_fit_lut_gd (§2.2,
   Eq. 3 with a nonlinear layer output; the bias is added first). */
enum {
    MADDNESS_FIT_RELU_SQERR = 2,     /* ReLU, squared error                       */
    MADDNESS_FIT_SOFTMAX_KLD = 3,    /* row softmax, KL divergence (as in §3.1)   */
    MADDNESS_FIT_SOFTMAX_SQERR = 4   /* row softmax, squared error (Eq. 3)        */
};

#define MADDNESS_K 16          /* prototypes per codebook (4-bit indices)   */
#define MADDNESS_LEVELS 4      /* tree depth: comparisons per codebook      */
#define MADDNESS_NODES 15      /* thresholds per codebook                   */

/* Library version (major * 10000 + minor * 100 + patch). */
int maddness_version(void);

/* Static string naming a status code; never NULL. */
const char* maddness_status_string(int status);

/*
 * Encoding function (§1: map each subvector to the index of one of K
 * prototypes, a log2(K)-bit integer; §1 and §2.1: a balanced binary tree
 * with four comparisons per codebook, K = 16).
 *
 *   A           [N][lda] fp32, row n at A + n * lda, D columns used.
 *   split_dims  [C][4] int32: the column of A compared at tree level t.
 *               A GLOBAL column index, so any permutation of the input
 *               dimensions (the subspace partitioning of §2.1) is folded in.
 *   thresholds  [C][15] fp32 in heap order: node i (0 <= i < 2^t) of level t
 *               is thresholds[c][2^t - 1 + i].
 *   idx_out     [N][C] uint8, written with values in [0, 16).
 *
 * idx[n][c] = i_4 where i_0 = 0 and
 *   i_{t+1} = 2 i_t + (A[n][split[c][t]] > thresholds[c][2^t - 1 + i_t]);
 * the comparison is strict (ties and NaN go to the 0 branch), so the root
 * decision is the most significant bit.
 *
 * EINVAL: a NULL array (when N > 0), N < 0, D <= 0, C <= 0, lda < D,
 * split_dims/thresholds/A not 4-byte aligned.  EUNSUPPORTED: C > 512.
 */
int maddness_encode(const float* A, int64_t N, int32_t D, int64_t lda,
                    const int32_t* split_dims, const float* thresholds,
                    int32_t C, uint8_t* idx_out, void* stream);

/*
 * Lookup-accumulate over 8-bit block floating point tables (§1: the result
 * is the sum over codebooks of the table rows picked by the indices; tables
 * quantized to 8-bit block floating point).
 *
 *   idx     [N][C] uint8 in [0, 16).
 *   lut     [C][16][M] int8 codes q.
 *   scale   [C] fp32, each an exact normal power of two 2^e_c.
 *   offset  [C] fp32 o_c.  The table entry is 2^e_c * q + o_c.
 *   acc_out [N][M] int32 or NULL:  acc = sum_c q[c][idx[n][c]][m] << (e_c - e_min),
 *           exact (no overflow under the precondition above).
 *   y_out   [N][M] fp32 or NULL (not both NULL):
 *           y = fmaf((float)acc, 2^e_min, bias32), where
 *           bias32 = (float)(sum_c offset[c] accumulated in double, c = 0..C-1).
 *           (float)acc is exact while |acc| <= 2^24, which tables from
 *           maddness_build_lut always satisfy, and y is then the single
 *           rounding of acc 2^e_min + bias32; a larger |acc| (possible only
 *           with other tables) is rounded to fp32 before the fma.
 *
 * EINVAL: a NULL required array, both outputs NULL, N < 0, C <= 0, M <= 0,
 * misaligned scale/offset/acc_out/y_out.  EUNSUPPORTED: C > 512.
 */
int maddness_lut_accumulate(const uint8_t* idx, int64_t N, int32_t C,
                            const int8_t* lut, const float* scale,
                            const float* offset, int32_t M,
                            int32_t* acc_out, float* y_out, void* stream);

/*
 * Rounded 8-bit summation over codebooks (§1 names it as the summation of
 * MADDNESS's 8-bit tables; this library's reading, R20): an approximate
 * alternative to the exact sum of maddness_lut_accumulate.  Every scale must
 * be the same power of two 2^e (a precondition, as for the other device
 * contents; maddness_build_lut_shared makes such tables).  Per output, the
 * biased codes u_c = q_c + 128 of codebooks 0..C-1, followed by P - C copies
 * of 128 (P = the smallest power of two >= C), are reduced by a balanced
 * tree in codebook order whose nodes are rounded byte averages
 * (a + b + 1) >> 1; with r the root,
 *   acc = P * (r - 128),   y = fl32(acc * 2^e + bias32)   (bias32 as above).
 * The estimate satisfies 0 <= acc - sum_c q_c <= P log2(P) / 2.
 * Same arguments and errors as maddness_lut_accumulate; idx must also be
 * 16-byte aligned (EINVAL otherwise), and C > 128 gives EUNSUPPORTED (the
 * kernel keeps the table's whole column slice and a batch of index rows in
 * LDS).
 */
int maddness_lut_accumulate_avg(const uint8_t* idx, int64_t N, int32_t C,
                                const int8_t* lut, const float* scale,
                                const float* offset, int32_t M,
                                int32_t* acc_out, float* y_out, void* stream);

/*
 * Lookup-accumulate over an unquantized fp32 table [C][16][M]:
 *   y[n][m] = (((0 + T[0][idx0][m]) + T[1][idx1][m]) + ...) in fp32, codebooks
 * in ascending order (a fixed order, so the result is deterministic).
 * EINVAL / EUNSUPPORTED as above.
 */
int maddness_lut_accumulate_f32(const uint8_t* idx, int64_t N, int32_t C,
                                const float* lut, int32_t M, float* y_out,
                                void* stream);

/*
 * Fused encode + lookup-accumulate: the whole inference path for one layer
 * (§1).  Same arguments and results as maddness_encode followed by
 * maddness_lut_accumulate; y_out is required, acc_out is an optional extra
 * output.  When the table [C][16][M] fits the single-launch kernels the
 * indices never leave the chip and idx_out is optional (written when given).
 * Otherwise the rows are encoded into idx_out and then accumulated, and
 * idx_out is required: EINVAL when it is NULL.  One case sits between: int8
 * tables of 64 codebooks and 16 <= M <= 512 columns at 98304 rows or more
 * run as one launch without idx_out, but given an 8-byte aligned idx_out
 * with M >= 128 they run faster in two phases through it (encode, then the
 * lookup-accumulate as a one-hot int8 product on the matrix cores, §2.2's
 * encoder output taken as a 0/1 matrix).  maddness_matmul_index_bytes tells
 * which case a call is.
 */
int maddness_matmul(const float* A, int64_t N, int32_t D, int64_t lda,
                    const int32_t* split_dims, const float* thresholds,
                    int32_t C, const int8_t* lut, const float* scale,
                    const float* offset, int32_t M, float* y_out,
                    int32_t* acc_out, uint8_t* idx_out, void* stream);

/* Fused encode + fp32-table accumulate (unquantized mode); see above,
   idx_out included. */
int maddness_matmul_f32(const float* A, int64_t N, int32_t D, int64_t lda,
                        const int32_t* split_dims, const float* thresholds,
                        int32_t C, const float* lut, int32_t M, float* y_out,
                        uint8_t* idx_out, void* stream);

/*
 * Fused encode + lookup-accumulate followed by the layer output sigma
 * (§2.2: deep learning needs sigma(A B), the bias term composed with a
 * nonlinearity -- elementwise such as ReLU, or row-wise such as softmax for
 * a classifier).  y is formed exactly as by maddness_matmul, then
 *   z[n][m] = fl32(y[n][m] + col_bias[m])   (act >= MADDNESS_ACT_BIAS;
 *                                            col_bias NULL: no bias)
 *   MADDNESS_ACT_RELU:    out = z > 0 ? z : +0 (bit-exact, -0 and NaN give +0)
 *   MADDNESS_ACT_SOFTMAX: out[n][m] = exp(z[n][m] - max_j z[n][j]) /
 *                         sum_j exp(z[n][j] - max_j z[n][j]), evaluated in
 *                         fp32 (expf, any summation order): each entry is
 *                         within (|z - max| + M + 5) * 2^-24 relative of the
 *                         exact value (plus underflow below 2^-126).
 * col_bias [M] fp32, 4-byte aligned.  idx_out [N][C] receives the indices;
 * it is optional or required as for maddness_matmul.  EINVAL: act outside
 * 0..3, plus the conditions of maddness_matmul.
 */
int maddness_matmul_act(const float* A, int64_t N, int32_t D, int64_t lda,
                        const int32_t* split_dims, const float* thresholds,
                        int32_t C, const int8_t* lut, const float* scale,
                        const float* offset, int32_t M, const float* col_bias,
                        int32_t act, float* y_out, uint8_t* idx_out,
                        void* stream);

/* The same with an unquantized fp32 table (see maddness_matmul_f32). */
int maddness_matmul_act_f32(const float* A, int64_t N, int32_t D, int64_t lda,
                            const int32_t* split_dims, const float* thresholds,
                            int32_t C, const float* lut, int32_t M,
                            const float* col_bias, int32_t act, float* y_out,
                            uint8_t* idx_out, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops or harnesses that forbid allocation, even through
 * a caching allocator): maddness_matmul with the same arguments and results,
 * except that idx_out is optional for every shape.  When the table does not
 * fit the single-launch kernels and idx_out is NULL, the indices go through
 * a scratch array inside the library: a 32 MiB static device array on each
 * device the library runs on, held until the process ends, whose address is
 * resolved once per device on its first such call.  Rows are processed in
 * chunks of (32 MiB / C) rounded down to a multiple of 256 rows (at least
 * 65536), each encoded into the scratch array and accumulated from it, so no
 * call size exceeds it.  Calls that take the scratch path share the device's
 * array: two such calls on one device whose work overlaps (different
 * streams, or different host threads without ordering) race on it and give
 * unspecified results; calls on one stream are ordered and safe.  The array
 * keeps the last call's indices; nothing is read before it is written, so
 * nothing needs clearing.  Allocates nothing.  EHIP if the scratch address
 * cannot be resolved; otherwise the errors of maddness_matmul.
 */
int maddness_matmul_noalloc(const float* A, int64_t N, int32_t D, int64_t lda,
                            const int32_t* split_dims, const float* thresholds,
                            int32_t C, const int8_t* lut, const float* scale,
                            const float* offset, int32_t M, float* y_out,
                            int32_t* acc_out, uint8_t* idx_out, void* stream);

/*
 * Device bytes of idx_out that the fused entry points use for this call: 0
 * when the call runs as one launch (idx_out optional), N * C when the indices
 * go through memory: required there, except for the shapes above that also
 * run as one launch without it (slower).  The answer depends on
 * the shape, on whether the table is fp32 (f32 != 0), on act (the layer
 * output of maddness_matmul_act[_f32]; 0 for maddness_matmul[_f32]) and on
 * the alignment of A, so pass the A of the call.  Returns -1 for arguments
 * the entry points reject with EINVAL, -3 for shapes they reject with
 * EUNSUPPORTED.  Makes no HIP call.
 */
int64_t maddness_matmul_index_bytes(const float* A, int64_t N, int32_t D, int64_t lda, int32_t C,
                                    int32_t M, int32_t f32, int32_t act);

/*
 * Offline table construction (§2.2: T = P B) followed by 8-bit block
 * floating point quantization (§1).
 *
 *   P      [C][16][D] fp32 prototypes (zero outside codebook c's subspace).
 *   B      [D][M] fp32 weights.
 *   T[c][k][m] = sum_d P[c][k][d] * B[d][m], a double sum over d ascending
 *   (each product is exact in double).  Per codebook, over its 16 x M
 *   entries: offset o_c = (float)((min + max) / 2); r_c = max |T - o_c|;
 *   e_c = the smallest integer in [-126, 127] with r_c <= 127 * 2^e_c, then
 *   raised to at least max_c e_c - cap, cap the largest integer with
 *   127 * C * 2^cap < 2^24 (so acc stays exact in fp32); codes
 *   q = round-half-even((T - o_c) / 2^e_c) in [-127, 127]; scale = 2^e_c.
 *
 *   lut_out [C][16][M] int8, scale_out [C] fp32, offset_out [C] fp32.
 * EINVAL: NULL, non-positive sizes, 127 * C >= 2^24, misaligned P/B/scale/offset.
 */
int maddness_build_lut(const float* P, const float* B, int32_t C, int32_t D,
                       int32_t M, int8_t* lut_out, float* scale_out,
                       float* offset_out, void* stream);

/* The same quantization with one block exponent shared by every codebook
   (cap = 0: e_c = max_c e_c), as maddness_lut_accumulate_avg requires. */
int maddness_build_lut_shared(const float* P, const float* B, int32_t C,
                              int32_t D, int32_t M, int8_t* lut_out,
                              float* scale_out, float* offset_out, void* stream);

/* Same table T = P B, each entry rounded to fp32 (unquantized mode). */
int maddness_build_lut_f32(const float* P, const float* B, int32_t C,
                           int32_t D, int32_t M, float* lut_out, void* stream);

/*
 * 8-bit block floating point quantization (§1; the quantizer of
 * maddness_build_lut) of a given table T [C][16][M] (double, device), e.g. a
 * fitted one.  shared != 0 gives every codebook the same exponent (as
 * maddness_build_lut_shared).  EINVAL / EUNSUPPORTED as for
 * maddness_build_lut; T must be 8-byte aligned.
 */
int maddness_quantize_lut(const double* T, int32_t C, int32_t M, int32_t shared,
                          int8_t* lut_out, float* scale_out, float* offset_out,
                          void* stream);

/*
 * Model-aware table fit (§2.2, Eq. 3) with an affine layer output, where the
 * bias cancels: the table T [C][16][M] minimising
 *     sum_n || Y[n] - sum_c T[c][idx[n][c]] ||^2 + lambda || T - T0 ||^2
 * over training rows n, Y = AB the layer's exact outputs [N][M] (fp32),
 * idx [N][C] their encoder indices, T0 = P0 B the prototype table (fp32,
 * [C][16][M]).  With G the one-hot encoder output (G[n][16c + k] = 1 iff
 * idx[n][c] = k) the minimiser solves (G^T G + lambda I) T = G^T Y +
 * lambda T0; it is computed in double (T_out, [C][16][M], 8-byte aligned) by
 * a Cholesky factorisation and forward / backward substitution whose every
 * multiply-subtract is one fused multiply-add, terms of an entry taken k
 * ascending (factor, forward pass) or descending (backward pass).
 * workspace: device memory of at least maddness_fit_lut_workspace_bytes(N, C)
 * bytes, 256-byte aligned, caller-owned, contents undefined on return.
 * lambda must be positive and finite (EINVAL); with a rank-deficient G^T G
 * (every row picks one bucket per codebook, so it always is for C > 1) a
 * lambda near the rounding level of G^T G's entries (about N x 1e-16) can
 * leave the factorisation without a positive pivot in double, and the
 * result is then NaN.  C > 256 or N >= 2^31 gives
 * EUNSUPPORTED.  Quantize the result with maddness_quantize_lut, or round it
 * to fp32 for the unquantized mode.
 */
int64_t maddness_fit_lut_workspace_bytes(int64_t N, int32_t C);   /* -1 if out of range */
int maddness_fit_lut_ridge(const uint8_t* idx, int64_t N, int32_t C,
                           const float* Y, int32_t M, const float* T0,
                           double lambda, double* T_out, void* workspace,
                           int64_t workspace_bytes, void* stream);

/*
 * Model-aware table fit (§2.2, Eq. 3) with a nonlinear layer output, by
 * full-batch gradient descent from T = T0 (the paper names the objectives,
 * not an optimiser; eta and iters are the caller's).  With
 * z_n = (sum_c T[c][idx[n][c]][.], c ascending, double) + col_bias and `act`
 * one of the MADDNESS_FIT_* objectives:
 *   RELU_SQERR:    objective sum_n ||relu(Y[n] + b) - relu(z_n)||^2,
 *                  residual 2 (relu(z) - relu(y + b)) [z > 0];
 *   SOFTMAX_KLD:   objective sum_n KL(softmax(Y[n] + b) || softmax(z_n)),
 *                  residual softmax(z) - softmax(y + b);
 *   SOFTMAX_SQERR: objective sum_n ||softmax(z_n) - softmax(Y[n] + b)||^2,
 *                  residual 2 p (d - s) with p = softmax(z),
 *                  d = p - softmax(y + b), s = sum_m d_m p_m;
 * each plus lambda ||T - T0||^2.  A step: R = G^T residual (rows ascending),
 * g = R + 2 lambda (T - T0), T = T - eta g, all in double.  ReLU steps are
 * exactly reproducible; softmax steps differ from another implementation only
 * through exp and the order of the row sums.  col_bias [M] fp32 or NULL
 * (zeros).  workspace: at least maddness_fit_lut_gd_workspace_bytes(N, C, M)
 * device bytes, 256-byte aligned.  EINVAL: another act, lambda < 0, eta <= 0,
 * non-finite values, iters < 0; EUNSUPPORTED: C > 256 or N >= 2^31.
 */
int64_t maddness_fit_lut_gd_workspace_bytes(int64_t N, int32_t C, int32_t M);   /* -1 if out of range */
int maddness_fit_lut_gd(const uint8_t* idx, int64_t N, int32_t C,
                        const float* Y, int32_t M, const float* col_bias,
                        int32_t act, const float* T0, double lambda,
                        double eta, int32_t iters, double* T_out,
                        void* workspace, int64_t workspace_bytes, void* stream);

/*
 * The two sums the normal equations of Eq. 3 are built from:
 * maddness_encoder_gram: H = G^T G [16C][16C] as int32 counts
 *   (H[16c + k][16c' + k'] = number of rows with idx[n][c] = k and
 *   idx[n][c'] = k'); exact.
 * maddness_encoder_scatter: R = G^T Y [16C][M] in double, each entry the sum
 *   of its rows in ascending row order; workspace (device, 256-byte aligned,
 *   at least maddness_encoder_scatter_workspace_bytes(N, C) bytes) holds the
 *   rows listed bucket by bucket.
 * C > 256 or N >= 2^31 gives EUNSUPPORTED.
 */
int maddness_encoder_gram(const uint8_t* idx, int64_t N, int32_t C,
                          int32_t* gram_out, void* stream);
int64_t maddness_encoder_scatter_workspace_bytes(int64_t N, int32_t C);   /* -1 if out of range */
int maddness_encoder_scatter(const uint8_t* idx, int64_t N, int32_t C,
                             const float* Y, int32_t M, double* out,
                             void* workspace, int64_t workspace_bytes,
                             void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MADDNESS_H */
