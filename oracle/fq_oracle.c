/*
 * Plain CPU oracle for the FoldQuantVLA runtime quantized projection.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do.  It shares no code, header or constant with the GPU path.
 *
 * It follows the paper step by step, with no blocking or fusion:
 *   - Sec. III-C: block Hadamard rotation R = I (x) H_b / sqrt(b), H_b the
 *     Sylvester +-1 matrix, applied as a fast Walsh-Hadamard transform.
 *   - Eq. (5), Sec. III-E: dynamic per-token symmetric quantization,
 *     delta_t = r * ||z_t||_inf / q, q = 2^(bits-1) - 1, codes clip(round(z/delta)),
 *     and the zero-token rule (z_t = 0 gives codes 0 and delta 0; Alg. 1 runtime).
 *   - Eq. (8), Sec. III-F: integer output y_jt = s_j * delta_t * sum_c qW_jc qA_ct + b_j.
 *
 * Floating-point contract (the paper fixes no precision or summation order for
 * these steps; the readings are listed in the design notes):
 *   * the transform runs in fp32 as an in-place butterfly with stages
 *     h = 1, 2, 4, ..., b/2, each pair (a, c) -> (a + c, a - c), on the
 *     UNNORMALIZED Sylvester matrix; the 1/sqrt(b) factor is carried by delta
 *     (by Prop. 2 this leaves the codes unchanged in exact arithmetic);
 *   * the per-token division z/delta is one fp32 reciprocal per token,
 *     inv = q / (r*A), followed by one fp32 multiply per element;
 *   * round() is round-half-to-even;
 *   * delta = ((r*A) * c_b) / q in fp32, c_b = the float nearest 1/sqrt(b).
 * Build with -ffp-contract=off so no multiply-add is fused.
 *
 * The integer contraction is a brute-force int64 triple loop (eq. (8) is the
 * definition), and the dequantization is done in double.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
static int omp_thread_slot(void) { return omp_get_thread_num(); }
int fqo_max_threads(void) { return omp_get_max_threads(); }
void fqo_set_threads(int n) { if (n > 0) omp_set_num_threads(n); }
#else
static int omp_thread_slot(void) { return 0; }
int fqo_max_threads(void) { return 1; }
void fqo_set_threads(int n) { (void)n; }
#endif

#define FQO_OK 0
#define FQO_BAD_ARG 1

static float bf16_bits_to_float(uint16_t h) {
    uint32_t u = ((uint32_t)h) << 16; /* bf16 is the top half of an fp32 */
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

static int is_pow2(int64_t b) { return b >= 1 && (b & (b - 1)) == 0; }

/* c_b: the float nearest to 1/sqrt(b) (Sec. III-C normalization of H_b). */
float fqo_inv_sqrt_b(int64_t b) {
    return (float)(1.0 / sqrt((double)b));
}

/* Unnormalized Sylvester FWHT of one block of length b, in place, fp32.
 * Stage h pairs index j with j + h inside every 2h-aligned group. */
void fqo_fwht_block_f32(float *v, int64_t b) {
    for (int64_t h = 1; h < b; h *= 2) {
        for (int64_t i = 0; i < b; i += 2 * h) {
            for (int64_t j = i; j < i + h; ++j) {
                float a = v[j];
                float c = v[j + h];
                v[j] = a + c;
                v[j + h] = a - c;
            }
        }
    }
}

/* Eq. (5) on one transformed token u[0..K) (unnormalized coordinates). */
static void quantize_token(const float *u, int64_t K, int bits, float r, float cb,
                           int8_t *code, float *delta) {
    const int q = (1 << (bits - 1)) - 1;
    float A = 0.0f;
    for (int64_t c = 0; c < K; ++c) {
        float m = fabsf(u[c]);
        if (m > A) A = m;
    }
    if (A == 0.0f) { /* zero-token rule */
        for (int64_t c = 0; c < K; ++c) code[c] = 0;
        *delta = 0.0f;
        return;
    }
    const float rA = r * A;
    const float inv = (float)q / rA;
    for (int64_t c = 0; c < K; ++c) {
        float t = u[c] * inv;
        float k = rintf(t); /* round half to even (default rounding mode) */
        if (k > (float)q) k = (float)q;
        if (k < (float)-q) k = (float)-q;
        code[c] = (int8_t)k;
    }
    *delta = (rA * cb) / (float)q;
}

static int check_args(int64_t M, int64_t K, int64_t b, int bits, float r, int64_t ld) {
    if (M < 0 || K < 1 || !is_pow2(b) || K % b != 0) return FQO_BAD_ARG;
    if (bits != 4 && bits != 8) return FQO_BAD_ARG;
    if (!(r > 0.0f && r <= 1.0f)) return FQO_BAD_ARG;
    if (ld < K) return FQO_BAD_ARG;
    return FQO_OK;
}

/* One row: optional per-channel multiplier before the rotation (fold-before S^-1,
 * Sec. III-C), blockwise FWHT, optional per-channel multiplier after it (fold-after
 * P^-1, Sec. III-C), quantize.  Each multiplier is one fp32 rounding per element. */
static void transform_row(float *v, const float *chan_mult, const float *post_mult, int64_t K,
                          int64_t b) {
    if (chan_mult)
        for (int64_t c = 0; c < K; ++c) v[c] = v[c] * chan_mult[c];
    for (int64_t k0 = 0; k0 < K; k0 += b) fqo_fwht_block_f32(v + k0, b);
    if (post_mult)
        for (int64_t c = 0; c < K; ++c) v[c] = v[c] * post_mult[c];
}

static void transform_quantize_row(float *v, const float *chan_mult, const float *post_mult,
                                   int64_t K, int64_t b, int bits, float r, float cb,
                                   int8_t *code, float *delta) {
    transform_row(v, chan_mult, post_mult, K, b);
    quantize_token(v, K, bits, r, cb, code, delta);
}

/* The prologue's transform alone (multipliers and the unnormalized butterfly), fp32 rows
 * z [M, K]: the coordinates in which Sec. III-F collects calibration tokens and rounds the
 * folded weights.  x is bf16 bits (is_bf16) or fp32. */
int fqo_transform(const void *x, int is_bf16, int64_t ldx, const float *chan_mult,
                  const float *post_mult, int64_t M, int64_t K, int64_t b, float *z) {
    if (check_args(M, K, b, 4, 1.0f, ldx)) return FQO_BAD_ARG;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < M; ++t) {
        float *row = z + t * K;
        for (int64_t c = 0; c < K; ++c)
            row[c] = is_bf16 ? bf16_bits_to_float(((const uint16_t *)x)[t * ldx + c])
                             : ((const float *)x)[t * ldx + c];
        transform_row(row, chan_mult, post_mult, K, b);
    }
    return FQO_OK;
}

/* Activation prologue (Alg. 1 runtime, first two steps) on bf16 tokens.
 * x: [M, ldx] bf16 bit patterns; chan_mult: [K] or NULL (fold-before S^-1);
 * post_mult: [K] or NULL (fold-after P^-1); codes: [M, K] int8 (unpacked);
 * delta: [M]; scratch: [nthreads * K] floats. */
int fqo_fwht_quant_bf16(const uint16_t *x, int64_t ldx, const float *chan_mult,
                        const float *post_mult, int64_t M, int64_t K, int64_t b, int bits,
                        float r, int8_t *codes, float *delta, float *scratch) {
    if (check_args(M, K, b, bits, r, ldx)) return FQO_BAD_ARG;
    const float cb = fqo_inv_sqrt_b(b);
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < M; ++t) {
        float *v = scratch + (int64_t)omp_thread_slot() * K;
        for (int64_t c = 0; c < K; ++c) v[c] = bf16_bits_to_float(x[t * ldx + c]);
        transform_quantize_row(v, chan_mult, post_mult, K, b, bits, r, cb, codes + t * K, delta + t);
    }
    return FQO_OK;
}

/* Same on fp32 rows.  With r = 1, chan_mult = s (fold-before S) and post_mult = p
 * (fold-after P), this is the offline weight rounding: row j of W S R^T P equals
 * p . R (s . w_j) because H_b is symmetric, and RTN with a per-output-channel scale
 * (Sec. III-E/F, Alg. 1 offline) rounds it with the same per-row rule. */
int fqo_fwht_quant_f32(const float *x, int64_t ldx, const float *chan_mult, const float *post_mult,
                       int64_t M, int64_t K, int64_t b, int bits, float r, int8_t *codes,
                       float *delta, float *scratch) {
    if (check_args(M, K, b, bits, r, ldx)) return FQO_BAD_ARG;
    const float cb = fqo_inv_sqrt_b(b);
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < M; ++t) {
        float *v = scratch + (int64_t)omp_thread_slot() * K;
        memcpy(v, x + t * ldx, (size_t)K * sizeof(float));
        transform_quantize_row(v, chan_mult, post_mult, K, b, bits, r, cb, codes + t * K, delta + t);
    }
    return FQO_OK;
}

/* Canonical signed-INT4 nibble packing: byte i of a row holds channel 2i in the
 * low nibble and channel 2i+1 in the high nibble, two's complement. */
int fqo_pack_int4(const int8_t *codes, int64_t M, int64_t K, uint8_t *out) {
    if (M < 0 || K < 0 || K % 2) return FQO_BAD_ARG;
    for (int64_t t = 0; t < M; ++t)
        for (int64_t i = 0; i < K / 2; ++i) {
            uint8_t lo = (uint8_t)codes[t * K + 2 * i] & 0x0F;
            uint8_t hi = (uint8_t)codes[t * K + 2 * i + 1] & 0x0F;
            out[t * (K / 2) + i] = (uint8_t)(lo | (hi << 4));
        }
    return FQO_OK;
}

/* Eq. (8) accumulator: acc[t, j] = sum_c qA[t, c] * qW[j, c], brute force in int64. */
int fqo_gemm_i64(const int8_t *qa, const int8_t *qw, int64_t M, int64_t N, int64_t K,
                 int64_t *acc) {
    if (M < 0 || N < 0 || K < 0) return FQO_BAD_ARG;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < M; ++t)
        for (int64_t j = 0; j < N; ++j) {
            int64_t s = 0;
            for (int64_t c = 0; c < K; ++c) s += (int64_t)qa[t * K + c] * (int64_t)qw[j * K + c];
            acc[t * N + j] = s;
        }
    return FQO_OK;
}

/* Eq. (8) rescale: y[t, j] = s_w[j] * delta[t] * acc[t, j] + bias[j], in double. */
int fqo_dequant(const int64_t *acc, const float *delta, const float *s_w, const float *bias,
                int64_t M, int64_t N, double *y) {
    if (M < 0 || N < 0) return FQO_BAD_ARG;
    for (int64_t t = 0; t < M; ++t)
        for (int64_t j = 0; j < N; ++j) {
            double v = (double)s_w[j] * (double)delta[t] * (double)acc[t * N + j];
            if (bias) v += (double)bias[j];
            y[t * N + j] = v;
        }
    return FQO_OK;
}

/* Weight-only INT4 projection: the paper keeps GR00T's adaptive layer-norm modulation
 * at floating-point activations times INT4 weights (Sec. III-A).  The weights are
 * rounded per output channel (codes q, scales s); the activations stay bf16 and are
 * not quantized.  acc[t, j] = sum_c x[t, c] * q[j, c] and y[t, j] = s_j acc[t, j] + b_j,
 * both in double (every product of a bf16 and a small integer is exact in double). */
int fqo_w4a16(const uint16_t *x, int64_t ldx, const int8_t *qw, const float *s_w,
              const float *bias, int64_t M, int64_t N, int64_t K, double *acc, double *y) {
    if (M < 0 || N < 0 || K < 1 || ldx < K) return FQO_BAD_ARG;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < M; ++t)
        for (int64_t j = 0; j < N; ++j) {
            double a = 0.0;
            for (int64_t c = 0; c < K; ++c)
                a += (double)bf16_bits_to_float(x[t * ldx + c]) * (double)qw[j * K + c];
            acc[t * N + j] = a;
            double v = (double)s_w[j] * a;
            if (bias) v += (double)bias[j];
            y[t * N + j] = v;
        }
    return FQO_OK;
}

/* Stored composite rotation (Sec. III-C, the action expert's optional transform): a
 * channel permutation followed by per-block orthogonal b x b matrices, R = B P, in place
 * of the block Hadamard.  The paper fixes neither the permutation ("zigzag") nor how the
 * block matrices are made ("SVD-Hadamard"); both are inputs here.  Per token:
 *   v_c = fl(x_c * s^-1_c)                (optional fold-before, original channel order)
 *   w_c = v_perm[c]                       (gather; perm = NULL is the identity)
 *   u_{kb+i} = fma chain over j = 0..b-1 ascending of Q_k[i][j] * w_{kb+j}, from +0
 *   u_c = fl(u_c * p^-1_c)                (optional fold-after)
 * then eq. (5) with c_b = 1 (the blocks are orthonormal, nothing is deferred to delta).
 * blocks: [K/b][b][b] fp32, Q_k row-major.  scratch: [nthreads * 2K] floats. */
static void rotate_quantize_row(const float *x, const int32_t *perm, const float *blocks,
                                const float *chan_mult, const float *post_mult, int64_t K,
                                int64_t b, int bits, float r, int8_t *code, float *delta,
                                float *v, float *u) {
    for (int64_t c = 0; c < K; ++c) v[c] = chan_mult ? x[c] * chan_mult[c] : x[c];
    for (int64_t k0 = 0; k0 < K; k0 += b) {
        const float *Q = blocks + k0 * b;  /* block k0 / b: b * b entries */
        for (int64_t i = 0; i < b; ++i) {
            float acc = 0.0f;
            for (int64_t j = 0; j < b; ++j) {
                const int64_t src = perm ? (int64_t)perm[k0 + j] : k0 + j;
                acc = fmaf(Q[i * b + j], v[src], acc);
            }
            u[k0 + i] = post_mult ? acc * post_mult[k0 + i] : acc;
        }
    }
    quantize_token(u, K, bits, r, 1.0f, code, delta);
}

static int check_perm(const int32_t *perm, int64_t K) {
    if (!perm) return FQO_OK;
    for (int64_t c = 0; c < K; ++c)
        if (perm[c] < 0 || perm[c] >= K) return FQO_BAD_ARG;
    return FQO_OK;
}

int fqo_rotate_quant_bf16(const uint16_t *x, int64_t ldx, const int32_t *perm, const float *blocks,
                          const float *chan_mult, const float *post_mult, int64_t M, int64_t K,
                          int64_t b, int bits, float r, int8_t *codes, float *delta, float *scratch) {
    if (check_args(M, K, b, bits, r, ldx) || check_perm(perm, K) || !blocks) return FQO_BAD_ARG;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < M; ++t) {
        float *row = scratch + (int64_t)omp_thread_slot() * 3 * K;
        for (int64_t c = 0; c < K; ++c) row[c] = bf16_bits_to_float(x[t * ldx + c]);
        rotate_quantize_row(row, perm, blocks, chan_mult, post_mult, K, b, bits, r, codes + t * K,
                            delta + t, row + K, row + 2 * K);
    }
    return FQO_OK;
}

int fqo_rotate_quant_f32(const float *x, int64_t ldx, const int32_t *perm, const float *blocks,
                         const float *chan_mult, const float *post_mult, int64_t M, int64_t K,
                         int64_t b, int bits, float r, int8_t *codes, float *delta, float *scratch) {
    if (check_args(M, K, b, bits, r, ldx) || check_perm(perm, K) || !blocks) return FQO_BAD_ARG;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < M; ++t) {
        float *row = scratch + (int64_t)omp_thread_slot() * 3 * K;
        rotate_quantize_row(x + t * ldx, perm, blocks, chan_mult, post_mult, K, b, bits, r,
                            codes + t * K, delta + t, row + K, row + 2 * K);
    }
    return FQO_OK;
}

/* GPTQ in the transformed coordinates (eq. (7), Sec. III-F): the columns of each folded
 * weight row are rounded in order, and each rounding error is pushed onto the columns not
 * yet rounded through U, the upper Cholesky factor of the damped inverse second moment
 * (H^-1 = U^T U), in the lazy-batch form of the GPTQ method: within a block of `blk`
 * columns the error goes to the block's later columns at once, to the columns after the
 * block once per block.  Exact arithmetic is the same as the one-column-at-a-time form.
 *
 * Floating-point contract (fp64 throughout; the paper fixes no precision):
 *   A = max_c |w_c| over the fp32 row (exact), q = 2^(bits-1) - 1;
 *   scale = fl32((A * scale_mult) / q) in fp32 (the round-to-nearest weight rule's scale);
 *   inv = q / A and step = A / q in fp64;
 *   column c: code = clamp(rint(w_c * inv), -q, q); e = (w_c - code * step) / U[c][c];
 *     each later column c' of the block: w_c' = fma(-e, U[c][c'], w_c');
 *   after the block [i1, i2): each column c' >= i2: acc = fma chain over k = i1..i2-1
 *     ascending of e_k * U[k][c'] from +0, then w_c' = w_c' - acc.
 * A zero row gives codes 0 and scale 0.  w: fp32 [N, ldw] folded rows (the unnormalized
 * transform's coordinates); U: fp64 [K, K] row-major (entries below the diagonal unused);
 * codes: int8 [N, K]; scales: fp32 [N]; scratch: nthreads * (K + blk) doubles. */
int fqo_gptq_sweep(const float *w, int64_t ldw, const double *U, int64_t N, int64_t K, int bits,
                   int64_t blk, float scale_mult, int8_t *codes, float *scales, double *scratch) {
    if (N < 0 || K < 1 || ldw < K || blk < 1 || (bits != 4 && bits != 8)) return FQO_BAD_ARG;
    const int q = (1 << (bits - 1)) - 1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t j = 0; j < N; ++j) {
        double *wr = scratch + (int64_t)omp_thread_slot() * (K + blk);
        double *e = wr + K;
        const float *src = w + j * ldw;
        int8_t *code = codes + j * K;
        float A = 0.0f;
        for (int64_t c = 0; c < K; ++c) {
            float m = fabsf(src[c]);
            if (m > A) A = m;
        }
        if (A == 0.0f) {
            for (int64_t c = 0; c < K; ++c) code[c] = 0;
            scales[j] = 0.0f;
            continue;
        }
        scales[j] = (A * scale_mult) / (float)q;
        const double inv = (double)q / (double)A, step = (double)A / (double)q;
        for (int64_t c = 0; c < K; ++c) wr[c] = (double)src[c];
        for (int64_t i1 = 0; i1 < K; i1 += blk) {
            const int64_t i2 = i1 + blk < K ? i1 + blk : K;
            for (int64_t c = i1; c < i2; ++c) {
                double k = rint(wr[c] * inv); /* round half to even */
                if (k > q) k = q;
                if (k < -q) k = -q;
                code[c] = (int8_t)k;
                const double err = (wr[c] - k * step) / U[c * K + c];
                e[c - i1] = err;
                for (int64_t c2 = c + 1; c2 < i2; ++c2) wr[c2] = fma(-err, U[c * K + c2], wr[c2]);
            }
            for (int64_t c2 = i2; c2 < K; ++c2) {
                double acc = 0.0;
                for (int64_t k = i1; k < i2; ++k) acc = fma(e[k - i1], U[k * K + c2], acc);
                wr[c2] = wr[c2] - acc;
            }
        }
    }
    return FQO_OK;
}
