/*
 * Plain CPU oracle for the MADDNESS-style encode + lookup-accumulate path
 * studied in "Look-ups are not (yet) all you need for deep learning
 * inference" (McCarter & Dronen).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the CPU-baseline leg
 * of the benchmark do.  It shares no code, header, table or helper with the
 * HIP path.
 *
 * Style: scalar loops in the order the method states them, double precision
 * wherever the method leaves the precision open, no blocking, no fusion and
 * no reordering.  OpenMP splits the independent rows across host threads and
 * never changes the order of any sum.  Build with
 *     gcc -O2 -std=c99 -fopenmp -ffp-contract=off -fno-fast-math -fPIC -shared
 * so that no multiply-add is contracted.
 *
 * Readings of points the paper leaves open (the same numbers label them in
 * the tests and in the HIP sources):
 *   R1  a tree node sends x right iff x > threshold (strict; ties and NaN go
 *       left).
 *   R2  one split dimension per (codebook, level), a global column of A.
 *   R3  node (t, i) of codebook c is thresholds[c*15 + 2^t - 1 + i]; the root
 *       decision is the most significant bit of the 4-bit index.
 *   R5  8-bit block floating point: table entry = scale_c * q + offset_c with
 *       q an int8 and scale_c an exact power of two per codebook.
 *   R6  quantizer: offset = midrange, exponent = the smallest that fits every
 *       code in [-127, 127] (no clipping), raised to within `cap` of the
 *       largest exponent so the int32 sum stays exact in fp32.
 *   R7  acc = sum_c q_c 2^(e_c - e_min) exactly in int32: any int8 codes are
 *       admitted when 128 * sum_c 2^(e_c - e_min) <= 2^31.
 *   R9  y = fmaf( float(acc), 2^e_min, bias32 ), with bias32 = fl32( sum_c
 *       offset_c accumulated in double, c ascending ).  float(acc) is exact
 *       while |acc| <= 2^24 (always so for tables from the quantizer, R6), and
 *       y is then one rounding of acc 2^e_min + bias32; a larger |acc| is
 *       rounded to fp32 first (two roundings).
 *   R10 unquantized mode: y = (((0 + T_0) + T_1) + ...) in fp32, c ascending.
 *   R21 model-aware table fit (Eq. 3) with sigma affine (bias and identity,
 *       so the bias cancels): minimise sum_n ||y_n - g_n^T T||^2 +
 *       lambda ||T - T0||^2 over T, squared Frobenius norms with no 1/N, g_n
 *       the one-hot encoder output (G[n][16c + k] = 1 iff idx[n][c] = k),
 *       targets Y = AB and the prototype table T0 = P0 B given in fp32 and
 *       taken exactly, lambda > 0; the minimiser solves the normal equations
 *       (G^T G + lambda I) T = G^T Y + lambda T0, column by column, in
 *       double: Cholesky factor L L^T, then forward and backward
 *       substitution, every multiply-subtract one fused multiply-add, the
 *       terms of an entry taken k ascending (factor, forward pass) or k
 *       descending (backward pass).
 *   R22 Eq. 3 with a nonlinear sigma, by full-batch gradient descent from
 *       T = T0 with a given step eta and iteration count (the paper names
 *       the objectives, not the optimiser).  z_n = (sum_c T[c][idx][.], c
 *       ascending, in double) + b.  ReLU: objective sum_n ||relu(y_n + b) -
 *       relu(z_n)||^2, residual r = 2 (relu(z) - relu(y + b)) [z > 0].
 *       Softmax: objective sum_n KL(softmax(y_n + b) || softmax(z_n)),
 *       residual r = softmax(z) - softmax(y + b).  Softmax with the squared
 *       error of Eq. 3 itself: objective sum_n ||softmax(z_n) -
 *       softmax(y_n + b)||^2; with p = softmax(z), d = p - softmax(y + b)
 *       and s = sum_m d_m p_m (m ascending), the residual (the chain rule
 *       through the softmax Jacobian diag(p) - p p^T) is r_m = 2 p_m (d_m - s).
 *       Step: R = G^T r (rows ascending from 0), g = R + 2 lambda (T - T0),
 *       T = T - eta g.
 *   R19 layer output sigma: z = fl32(y + bias_m); ReLU keeps z when z > 0 and
 *       gives +0 otherwise; softmax is taken over the M outputs of a row.
 *   R20 rounded 8-bit summation: one shared block exponent; biased codes
 *       u = q + 128, padded with 128 to P = 2^L codebooks, combined by a
 *       balanced tree in codebook order of rounded averages (a + b + 1) >> 1;
 *       the sum is estimated as P * (root - 128).
 *
 * Every entry point returns 0 on success and a negative code on a violated
 * precondition (it never aborts): -1 bad size / pointer, -2 a scale that is
 * not an exact normal power of two, -3 an accumulator that could overflow
 * int32, -4 an out-of-range split dimension.
 */
#include <stdint.h>
#include <stddef.h>
#include <math.h>
#include <stdlib.h>

#define ORACLE_K 16      /* prototypes per codebook: 2^4 leaves         */
#define ORACLE_LEVELS 4  /* one comparison per tree level, §2.1              */
#define ORACLE_NODES 15  /* internal nodes of a balanced 4-level tree   */

int oracle_version(void) { return 1; }

int oracle_max_threads(void) {
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Host threads for the row loops of later calls (timing only; n >= 1). */
void oracle_set_threads(int n) {
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/*
 * Encoding function (§1: each subvector is mapped to the index of one of K
 * prototypes, a log2(K)-bit integer; §1 and §2.1: MADDNESS does it with a
 * balanced binary regression tree, one comparison per level, four levels for
 * K = 16).
 * Walk the tree of codebook c from the root: at level t the current node is
 * i (0 <= i < 2^t), its threshold is thresholds[c][2^t - 1 + i], and the
 * compared value is A[n][split[c][t]].  The next node is 2i + bit.
 */
int oracle_encode(const float* A, int64_t N, int32_t D, int64_t lda,
                  const int32_t* split, const float* thr, int32_t C,
                  uint8_t* idx)
{
    if (N < 0 || D <= 0 || C <= 0 || lda < D) return -1;
    if (N > 0 && (!A || !split || !thr || !idx)) return -1;
    for (int64_t j = 0; j < (int64_t)C * ORACLE_LEVELS; ++j)
        if (split[j] < 0 || split[j] >= D) return -4;
    int64_t n;
#pragma omp parallel for schedule(static)
    for (n = 0; n < N; ++n) {
        const float* row = A + n * lda;
        for (int32_t c = 0; c < C; ++c) {
            int i = 0;                                   /* node within level */
            for (int t = 0; t < ORACLE_LEVELS; ++t) {
                float x = row[split[c * ORACLE_LEVELS + t]];
                float v = thr[c * ORACLE_NODES + ((1 << t) - 1) + i];
                int bit = (x > v) ? 1 : 0;               /* R1 */
                i = 2 * i + bit;
            }
            idx[n * C + c] = (uint8_t)i;
        }
    }
    return 0;
}

/* Block exponent of one scale: scale = 2^e exactly, with scale a normal
 * fp32 number (R5).  Returns 0 and writes e, or -2. */
int oracle_block_exponent(float scale, int32_t* e)
{
    if (!(scale > 0.0f) || isinf(scale)) return -2;
    int x;
    float m = frexpf(scale, &x);                         /* scale = m 2^x, m in [0.5,1) */
    if (m != 0.5f) return -2;
    if (x - 1 < -126) return -2;                         /* subnormal scales rejected */
    *e = x - 1;
    return 0;
}

/* Dequantization constants shared by every output (R5, R9): per-codebook
 * shifts sh_c = e_c - e_min, e_min, and bias32.  Also checks that the int32
 * accumulator cannot overflow for any int8 codes (R7): the most negative sum
 * is -128 * sum_c 2^sh_c, which must be >= -2^31, and the largest,
 * 127 * sum_c 2^sh_c, is then below 2^31 - 1. */
int oracle_dequant_params(const float* scale, const float* offset, int32_t C,
                          int32_t* sh, int32_t* e_min, float* bias32)
{
    if (C <= 0 || !scale || !offset || !sh || !e_min || !bias32) return -1;
    int32_t emin = 1000;
    for (int32_t c = 0; c < C; ++c) {
        int32_t e;
        if (oracle_block_exponent(scale[c], &e) != 0) return -2;
        sh[c] = e;
        if (e < emin) emin = e;
    }
    double bound = 0.0;
    for (int32_t c = 0; c < C; ++c) {
        sh[c] -= emin;
        if (sh[c] > 30) return -3;
        bound += 128.0 * ldexp(1.0, sh[c]);
    }
    if (bound > 2147483648.0) return -3;
    double s = 0.0;
    for (int32_t c = 0; c < C; ++c) s += (double)offset[c];
    *e_min = emin;
    *bias32 = (float)s;
    return 0;
}

/*
 * Lookup-accumulate (§1: the approximate inner product is the sum over
 * codebooks of the table rows picked by the indices; 8-bit block floating
 * point tables).  With table entry = 2^e_c q + o_c,
 *     sum_c (2^e_c q_c + o_c) = 2^e_min * sum_c (q_c << sh_c) + sum_c o_c,
 * so the codebook sum is an exact integer acc and the float work is one
 * rounding at the end (R9).  lut is [C][16][M] int8, idx is [N][C].
 * acc_out and y_out may each be NULL (not both).
 */
int oracle_lut_accumulate(const uint8_t* idx, int64_t N, int32_t C,
                          const int8_t* lut, const float* scale,
                          const float* offset, int32_t M,
                          int32_t* acc_out, float* y_out)
{
    if (N < 0 || C <= 0 || M <= 0) return -1;
    if (!acc_out && !y_out) return -1;
    if (N > 0 && (!idx || !lut || !scale || !offset)) return -1;
    int32_t* sh = (int32_t*)malloc(sizeof(int32_t) * (size_t)C);
    if (!sh) return -1;
    int32_t emin;
    float bias32;
    int rc = oracle_dequant_params(scale, offset, C, sh, &emin, &bias32);
    if (rc != 0) { free(sh); return rc; }
    const float step = ldexpf(1.0f, emin);
    for (int64_t n = 0; n < N; ++n)
        for (int32_t c = 0; c < C; ++c)
            if (idx[n * C + c] >= ORACLE_K) { free(sh); return -1; }
    int64_t n;
#pragma omp parallel for schedule(static)
    for (n = 0; n < N; ++n) {
        for (int32_t m = 0; m < M; ++m) {
            int64_t acc = 0;
            for (int32_t c = 0; c < C; ++c) {
                int k = idx[n * C + c];
                int64_t q = lut[((int64_t)c * ORACLE_K + k) * M + m];
                acc += q * ((int64_t)1 << sh[c]);
            }
            if (acc_out) acc_out[n * M + m] = (int32_t)acc;
            if (y_out) y_out[n * M + m] = fmaf((float)acc, step, bias32);
        }
    }
    free(sh);
    return 0;
}

/*
 * Unquantized mode: the table holds fp32 entries T[c][k][m] and the sum over
 * codebooks is taken in fp32, c ascending, starting from +0 (R10).
 */
int oracle_lut_accumulate_f32(const uint8_t* idx, int64_t N, int32_t C,
                              const float* lut, int32_t M, float* y_out)
{
    if (N < 0 || C <= 0 || M <= 0) return -1;
    if (N > 0 && (!idx || !lut || !y_out)) return -1;
    for (int64_t n = 0; n < N; ++n)
        for (int32_t c = 0; c < C; ++c)
            if (idx[n * C + c] >= ORACLE_K) return -1;
    int64_t n;
#pragma omp parallel for schedule(static)
    for (n = 0; n < N; ++n) {
        for (int32_t m = 0; m < M; ++m) {
            float s = 0.0f;
            for (int32_t c = 0; c < C; ++c) {
                int k = idx[n * C + c];
                s = s + lut[((int64_t)c * ORACLE_K + k) * M + m];
            }
            y_out[n * M + m] = s;
        }
    }
    return 0;
}

/*
 * Lookup table T = P B (§2.2): P is the prototype matrix, one block of 16
 * rows per codebook ([C][16][D], zero outside the codebook's subspace), B is
 * the weight matrix [D][M].  Each entry is a double sum over d ascending of
 * exact products of fp32 values.
 */
int oracle_build_table(const float* P, const float* B, int32_t C, int32_t D,
                       int32_t M, double* T)
{
    if (C <= 0 || D <= 0 || M <= 0 || !P || !B || !T) return -1;
    int64_t r;
#pragma omp parallel for schedule(static)
    for (r = 0; r < (int64_t)C * ORACLE_K; ++r) {
        for (int32_t m = 0; m < M; ++m) {
            double s = 0.0;
            for (int32_t d = 0; d < D; ++d)
                s += (double)P[r * D + d] * (double)B[(int64_t)d * M + m];
            T[r * M + m] = s;
        }
    }
    return 0;
}

/* Largest cap with 127 * C * 2^cap < 2^24 (R6): keeps the int32 sum of any
 * C codes, each shifted by at most cap, exactly representable in fp32. */
int oracle_exponent_cap(int32_t C)
{
    if (C <= 0 || 127.0 * C >= 16777216.0) return -1;
    int cap = 0;
    while (127.0 * C * ldexp(1.0, cap + 1) < 16777216.0) ++cap;
    return cap;
}

/*
 * 8-bit block floating point quantization of T (§1; reading R6).
 * Per codebook c over its 16 x M entries: offset o_c = fl32 of the midrange,
 * r_c = max |T - o_c| (in double), e_c = the smallest e in [-126, 127] with
 * r_c <= 127 * 2^e.  Then e_c is raised to at least max_c e_c - cap, and
 * q = round-half-even((T - o_c) / 2^e_c), which always lies in [-127, 127].
 */
static int quantize_table_cap(const double* T, int32_t C, int32_t M, int cap,
                              int8_t* lut, float* scale, float* offset)
{
    const int64_t per = (int64_t)ORACLE_K * M;
    int32_t emax = -126;
    int32_t* ec = (int32_t*)malloc(sizeof(int32_t) * (size_t)C);
    if (!ec) return -1;
    for (int32_t c = 0; c < C; ++c) {
        const double* t = T + c * per;
        double lo = t[0], hi = t[0];
        for (int64_t j = 1; j < per; ++j) {
            if (t[j] < lo) lo = t[j];
            if (t[j] > hi) hi = t[j];
        }
        float o = (float)((lo + hi) / 2.0);
        double r = 0.0;
        for (int64_t j = 0; j < per; ++j) {
            double a = fabs(t[j] - (double)o);
            if (a > r) r = a;
        }
        int32_t e = -126;
        while (e < 127 && r > 127.0 * ldexp(1.0, e)) ++e;
        offset[c] = o;
        ec[c] = e;
        if (e > emax) emax = e;
    }
    for (int32_t c = 0; c < C; ++c) {
        int32_t e = ec[c];
        if (e < emax - cap) e = emax - cap;
        const double* t = T + c * per;
        const double o = (double)offset[c];
        for (int64_t j = 0; j < per; ++j) {
            double q = nearbyint((t[j] - o) / ldexp(1.0, e));
            if (q > 127.0 || q < -127.0) { free(ec); return -3; }  /* cannot happen; guard */
            lut[c * per + j] = (int8_t)q;
        }
        scale[c] = ldexpf(1.0f, e);
    }
    free(ec);
    return 0;
}

int oracle_quantize_table(const double* T, int32_t C, int32_t M,
                          int8_t* lut, float* scale, float* offset)
{
    if (C <= 0 || M <= 0 || !T || !lut || !scale || !offset) return -1;
    int cap = oracle_exponent_cap(C);
    if (cap < 0) return -1;
    return quantize_table_cap(T, C, M, cap, lut, scale, offset);
}

/*
 * The same quantizer with one block exponent shared by every codebook (the
 * floor max_c e_c - cap taken with cap = 0), as the rounded 8-bit averaging
 * accumulate below requires (reading R20).
 */
int oracle_quantize_table_shared(const double* T, int32_t C, int32_t M,
                                 int8_t* lut, float* scale, float* offset)
{
    if (C <= 0 || M <= 0 || !T || !lut || !scale || !offset) return -1;
    return quantize_table_cap(T, C, M, 0, lut, scale, offset);
}

/* Unquantized table: each T entry rounded to fp32 (round to nearest even). */
int oracle_round_table_f32(const double* T, int64_t n, float* out)
{
    if (n < 0 || (n > 0 && (!T || !out))) return -1;
    for (int64_t j = 0; j < n; ++j) out[j] = (float)T[j];
    return 0;
}

/*
 * Layer output sigma(AB) (§2.2: the bias term composed with a nonlinearity,
 * elementwise such as ReLU or row-wise such as softmax; reading R19).
 * act: 0 none, 1 bias only, 2 bias then ReLU, 3 bias then softmax over each
 * row.  y and bias are fp32 (bias may be NULL: no bias); out is [N][M]
 * double.  The bias add is one fp32 rounding, z = fl32(y + bias[m]); ReLU is
 * z if z > 0 else +0 (so -0 and NaN give +0); softmax is evaluated in double
 * from the fp32 z: p_m = exp(z_m - max_j z_j) / sum_j exp(z_j - max_j z_j),
 * the sum taken in ascending j.
 */
int oracle_sigma(const float* y, int64_t N, int32_t M, const float* bias,
                 int32_t act, double* out)
{
    if (N < 0 || M <= 0 || act < 0 || act > 3) return -1;
    if (N > 0 && (!y || !out)) return -1;
    int64_t n;
#pragma omp parallel for schedule(static)
    for (n = 0; n < N; ++n) {
        const float* yr = y + n * M;
        double* o = out + n * M;
        for (int32_t m = 0; m < M; ++m) {
            float z = yr[m];
            if (act >= 1 && bias) z = z + bias[m];
            if (act == 2) z = (z > 0.0f) ? z : 0.0f;
            o[m] = (double)z;
        }
        if (act == 3) {
            double mx = o[0];
            for (int32_t m = 1; m < M; ++m)
                if (o[m] > mx) mx = o[m];
            double sum = 0.0;
            for (int32_t m = 0; m < M; ++m) {
                o[m] = exp(o[m] - mx);
                sum += o[m];
            }
            for (int32_t m = 0; m < M; ++m) o[m] = o[m] / sum;
        }
    }
    return 0;
}

/*
 * Rounded 8-bit summation over codebooks (§1 names it, for MADDNESS's 8-bit
 * tables, without defining it; reading R20).  Every scale must be the same
 * power of two 2^e (else -2).  Per output, the biased codes u_c = q_c + 128
 * (in [1, 255]) of codebooks 0..C-1, followed by P - C copies of 128 (P the
 * smallest power of two >= C), are reduced level by level: node i of the
 * next level is (u_2i + u_2i+1 + 1) >> 1, a rounded byte average.  The root
 * r estimates the mean code + 128, so acc = P * (r - 128) estimates
 * sum_c q_c, and y = fl32(acc * 2^e + bias32) exactly as in R9.
 */
int oracle_lut_accumulate_avg(const uint8_t* idx, int64_t N, int32_t C,
                              const int8_t* lut, const float* scale,
                              const float* offset, int32_t M,
                              int32_t* acc, float* y)
{
    if (N < 0 || C <= 0 || M <= 0 || C > 4096) return -1;
    if (N > 0 && (!idx || !lut || !scale || !offset || !acc || !y)) return -1;
    for (int32_t c = 1; c < C; ++c)
        if (scale[c] != scale[0]) return -2;
    int32_t sh_unused[4096];
    int32_t emin = 0;
    float bias32 = 0.0f;
    int rc = oracle_dequant_params(scale, offset, C, sh_unused, &emin, &bias32);
    if (rc != 0) return rc;
    const float unit = ldexpf(1.0f, emin);   /* 2^e */
    int32_t P = 1;
    while (P < C) P *= 2;
    int64_t n;
#pragma omp parallel for schedule(static)
    for (n = 0; n < N; ++n) {
        int32_t u[4096];
        for (int32_t m = 0; m < M; ++m) {
            for (int32_t c = 0; c < P; ++c) {
                if (c < C) {
                    int k = idx[n * C + c];
                    u[c] = (int32_t)lut[((int64_t)c * ORACLE_K + k) * M + m] + 128;
                } else {
                    u[c] = 128;
                }
            }
            for (int32_t width = P; width > 1; width /= 2)
                for (int32_t i = 0; i < width / 2; ++i)
                    u[i] = (u[2 * i] + u[2 * i + 1] + 1) >> 1;
            const int32_t a = P * (u[0] - 128);
            acc[n * M + m] = a;
            y[n * M + m] = fmaf((float)a, unit, bias32);
        }
    }
    return 0;
}

/*
 * Gram matrix of the one-hot encoder output, H = G^T G (the matrix of the
 * normal equations of Eq. 3 under reading R21): H[16c + k][16c' + k'] counts
 * the rows n with idx[n][c] = k and idx[n][c'] = k'.  H is [16C][16C].
 */
int oracle_encoder_gram(const uint8_t* idx, int64_t N, int32_t C, int64_t* H)
{
    if (N < 0 || C <= 0 || !H || (N > 0 && !idx)) return -1;
    const int64_t n16 = (int64_t)C * ORACLE_K;
    for (int64_t j = 0; j < n16 * n16; ++j) H[j] = 0;
    for (int64_t n = 0; n < N; ++n)
        for (int32_t c = 0; c < C; ++c)
            for (int32_t c2 = 0; c2 < C; ++c2) {
                const int64_t r = (int64_t)c * ORACLE_K + idx[n * C + c];
                const int64_t s = (int64_t)c2 * ORACLE_K + idx[n * C + c2];
                H[r * n16 + s] += 1;
            }
    return 0;
}

/*
 * R = G^T Y (right-hand side of the normal equations of Eq. 3, reading R21):
 * R[16c + k][m] = sum over the rows n with idx[n][c] = k of Y[n][m], summed in
 * double over n ascending.  R is [16C][M].
 */
int oracle_encoder_scatter(const uint8_t* idx, int64_t N, int32_t C,
                           const float* Y, int32_t M, double* R)
{
    if (N < 0 || C <= 0 || M <= 0 || !R || (N > 0 && (!idx || !Y))) return -1;
    const int64_t n16 = (int64_t)C * ORACLE_K;
    for (int64_t j = 0; j < n16 * M; ++j) R[j] = 0.0;
    for (int64_t n = 0; n < N; ++n)
        for (int32_t c = 0; c < C; ++c) {
            const int64_t r = (int64_t)c * ORACLE_K + idx[n * C + c];
            for (int32_t m = 0; m < M; ++m) R[r * M + m] += (double)Y[n * M + m];
        }
    return 0;
}

/*
 * Model-aware table fit, Eq. 3 with sigma affine (reading R21): T [C][16][M]
 * solves (H + lambda I) T = R + lambda T0 with H and R as above.  The
 * matrix is symmetric positive definite for lambda > 0; it is factored as
 * L L^T (Cholesky, textbook order: column j from the columns before it) and
 * each of the M columns is solved by forward then backward substitution.
 * Each multiply-subtract is one fma(); the terms of an entry are taken k
 * ascending, except in the backward pass (k descending).
 * Returns -1 on bad sizes, -2 when lambda is not a positive finite number.
 */
int oracle_fit_lut_ridge(const uint8_t* idx, int64_t N, int32_t C,
                         const float* Y, int32_t M, const float* T0,
                         double lambda, double* T)
{
    if (N < 0 || C <= 0 || M <= 0 || C > 1024 || !T0 || !T) return -1;
    if (!(lambda > 0.0) || !isfinite(lambda)) return -2;
    const int64_t n16 = (int64_t)C * ORACLE_K;
    int64_t* H = (int64_t*)malloc(sizeof(int64_t) * n16 * n16);
    double* L = (double*)malloc(sizeof(double) * n16 * n16);
    double* R = (double*)malloc(sizeof(double) * n16 * M);
    double* z = (double*)malloc(sizeof(double) * n16);
    int rc = (!H || !L || !R || !z) ? -1 : 0;
    if (rc == 0) rc = oracle_encoder_gram(idx, N, C, H);
    if (rc == 0) rc = oracle_encoder_scatter(idx, N, C, Y, M, R);
    if (rc == 0) {
        /* A = H + lambda I, factored in place into its lower triangle */
        for (int64_t i = 0; i < n16; ++i)
            for (int64_t j = 0; j < n16; ++j)
                L[i * n16 + j] = (double)H[i * n16 + j] + (i == j ? lambda : 0.0);
        for (int64_t j = 0; j < n16; ++j) {
            double d = L[j * n16 + j];
            for (int64_t k = 0; k < j; ++k) d = fma(-L[j * n16 + k], L[j * n16 + k], d);
            d = sqrt(d);
            L[j * n16 + j] = d;
            for (int64_t i = j + 1; i < n16; ++i) {
                double v = L[i * n16 + j];
                for (int64_t k = 0; k < j; ++k) v = fma(-L[i * n16 + k], L[j * n16 + k], v);
                L[i * n16 + j] = v / d;
            }
        }
        for (int32_t m = 0; m < M; ++m) {
            /* right-hand side column m: (G^T Y)[.][m] + lambda T0[.][m] */
            for (int64_t i = 0; i < n16; ++i) z[i] = R[i * M + m] + lambda * (double)T0[i * M + m];
            for (int64_t i = 0; i < n16; ++i) {          /* L z' = z */
                double v = z[i];
                for (int64_t k = 0; k < i; ++k) v = fma(-L[i * n16 + k], z[k], v);
                z[i] = v / L[i * n16 + i];
            }
            for (int64_t i = n16 - 1; i >= 0; --i) {     /* L^T t = z' */
                double v = z[i];
                for (int64_t k = n16 - 1; k > i; --k) v = fma(-L[k * n16 + i], z[k], v);
                z[i] = v / L[i * n16 + i];
            }
            for (int64_t i = 0; i < n16; ++i) T[i * M + m] = z[i];
        }
    }
    free(H); free(L); free(R); free(z);
    return rc;
}

/* row softmax in double: maximum subtracted, exp, sum over m ascending */
static void softmax_row(const double* z, int32_t M, double* q)
{
    double mx = z[0];
    for (int32_t m = 1; m < M; ++m) if (z[m] > mx) mx = z[m];
    double sum = 0.0;
    for (int32_t m = 0; m < M; ++m) { q[m] = exp(z[m] - mx); sum += q[m]; }
    for (int32_t m = 0; m < M; ++m) q[m] = q[m] / sum;
}

/*
 * Model-aware table fit, Eq. 3 with a nonlinear layer output (reading R22):
 * act 2 = bias + ReLU with the squared-error objective, act 3 = bias + row
 * softmax with the KL-divergence objective (the alternative §3.1 uses for
 * classifier layers), act 4 = bias + row softmax with the squared-error
 * objective (Eq. 3 as written), each plus lambda ||T - T0||^2.
 * Full-batch gradient descent from T = T0: `iters` steps of size eta.  The
 * bias is optional (NULL = zeros).  T is [C][16][M] double.  Returns -1 on
 * bad sizes, -2 on a bad act, lambda, eta or iteration count.
 */
int oracle_fit_lut_gd(const uint8_t* idx, int64_t N, int32_t C, const float* Y, int32_t M,
                      const float* bias, int32_t act, const float* T0, double lambda, double eta,
                      int32_t iters, double* T)
{
    if (N < 0 || C <= 0 || M <= 0 || !T0 || !T || (N > 0 && (!idx || !Y))) return -1;
    if ((act != 2 && act != 3 && act != 4) || !(lambda >= 0.0) || !isfinite(lambda) || !(eta > 0.0) ||
        !isfinite(eta) || iters < 0)
        return -2;
    const int64_t n16 = (int64_t)C * ORACLE_K;
    double* P = (double*)malloc(sizeof(double) * (N > 0 ? N : 1) * M);   /* sigma of the targets */
    double* R = (double*)malloc(sizeof(double) * n16 * M);
    double* z = (double*)malloc(sizeof(double) * M);
    double* q = (double*)malloc(sizeof(double) * M);
    if (!P || !R || !z || !q) { free(P); free(R); free(z); free(q); return -1; }
    for (int64_t n = 0; n < N; ++n) {
        for (int32_t m = 0; m < M; ++m) z[m] = (double)Y[n * M + m] + (bias ? (double)bias[m] : 0.0);
        if (act == 2) {
            for (int32_t m = 0; m < M; ++m) P[n * M + m] = z[m] > 0.0 ? z[m] : 0.0;
        } else {
            softmax_row(z, M, &P[n * M]);
        }
    }
    for (int64_t j = 0; j < n16 * M; ++j) T[j] = (double)T0[j];
    for (int32_t it = 0; it < iters; ++it) {
        for (int64_t j = 0; j < n16 * M; ++j) R[j] = 0.0;
        for (int64_t n = 0; n < N; ++n) {
            for (int32_t m = 0; m < M; ++m) {
                double sacc = 0.0;
                for (int32_t c = 0; c < C; ++c)
                    sacc += T[((int64_t)c * ORACLE_K + idx[n * C + c]) * M + m];
                z[m] = sacc + (bias ? (double)bias[m] : 0.0);
            }
            if (act == 2) {
                for (int32_t m = 0; m < M; ++m)
                    q[m] = z[m] > 0.0 ? 2.0 * (z[m] - P[n * M + m]) : 0.0;
            } else if (act == 3) {
                softmax_row(z, M, q);
                for (int32_t m = 0; m < M; ++m) q[m] = q[m] - P[n * M + m];
            } else {
                softmax_row(z, M, q);                    /* q = p */
                double sdp = 0.0;
                for (int32_t m = 0; m < M; ++m) sdp += (q[m] - P[n * M + m]) * q[m];
                for (int32_t m = 0; m < M; ++m) {
                    const double d = q[m] - P[n * M + m];
                    q[m] = 2.0 * (q[m] * (d - sdp));
                }
            }
            for (int32_t c = 0; c < C; ++c) {
                const int64_t r = (int64_t)c * ORACLE_K + idx[n * C + c];
                for (int32_t m = 0; m < M; ++m) R[r * M + m] += q[m];
            }
        }
        for (int64_t j = 0; j < n16 * M; ++j) {
            const double g = R[j] + 2.0 * lambda * (T[j] - (double)T0[j]);
            T[j] = T[j] - eta * g;
        }
    }
    free(P); free(R); free(z); free(q);
    return 0;
}
