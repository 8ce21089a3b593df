/*
 * fq.h -- C ABI of the FoldQuantVLA runtime quantized projection on AMD MI355X (gfx950).
 *
 * The projection (Sec. III-E/F, Alg. 1 runtime) computes, for tokens x_t:
 *   z_t   = P^-1 R S^-1 x_t,  R = I_{K/b} (x) H_b / sqrt(b)   (block Hadamard, Sec. III-C)
 *   qA_t, delta_t = per-token symmetric quantization of z_t       (eq. (5))
 *   c_jt  = sum_c qW_jc qA_ct   (integer accumulation, INT32)     (eq. (8))
 *   y_jt  = s_j delta_t c_jt + b_j                                 (eq. (8))
 * against weights folded and rounded offline: W~ = W S R^T P rounded per output
 * channel to signed INT4 / INT8 codes qW with scales s (Alg. 1 offline).  S and P are
 * the positive diagonal scales of the two fold presets of Sec. III-C: fold-before
 * (S calibrated in the original coordinates, P = I) and fold-after (S = I, P calibrated
 * after the rotation); either may be the identity (NULL).
 *
 * Conventions shared by every entry point:
 *   - Every buffer argument is a DEVICE pointer owned by the caller, except where a
 *     comment says otherwise.  The library never allocates or frees memory; scratch
 *     space comes from a caller-provided workspace.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls enqueue work and
 *     return without synchronizing.  Device-side faults surface at the caller's next
 *     synchronization, as usual in HIP.
 *   - Arguments are validated before anything is enqueued; a failed check returns a
 *     status and enqueues nothing.  fq_last_error() (thread-local) then describes it.
 *   - M = 0 (or N = 0) is a valid no-op.
 *   - Layouts are row-major.  `ld*` arguments are row strides in elements.
 *   - Shape limits: K % 128 == 0, 128 <= K <= 32768, N % 16 == 0, b a power of two
 *     with 1 <= b <= 256 and K % b == 0, bits in {4, 8}, 0 < clip_ratio <= 1; for the
 *     GEMMs M, N <= 2^24 and M * N <= 2^40 (FQ_ERR_UNSUPPORTED beyond).  K is held to
 *     whole 128-channel steps because the kernel-native weight tiles and every k step of
 *     the GEMMs span 128 input channels; the paper's only requirement is that b divides K
 *     (Sec. III-C), and every layer width of the workloads is a multiple of 1024.
 *   - Alignment: every pointer 16-byte aligned; ldx and ldy multiples of 8.
 *   - No aliasing: an output (codes, scales, y, acc_out, a workspace) may not overlap
 *     another output or an input, over the bytes the call touches (FQ_ERR_ALIAS).
 *
 * Numerical contract of the prologue (so that codes are reproducible bit for bit):
 *   the transform is an fp32 butterfly on the UNNORMALIZED Sylvester matrix with
 *   stages h = 1, 2, ..., b/2, pairs (a, c) -> (a + c, a - c), with the optional
 *   S^-1 multiply (one fp32 rounding) before it and the optional P^-1 multiply (one
 *   fp32 rounding) after it; A_t = max_c |u_tc|
 *   over the whole row; inv = q / (r * A_t) (one correctly rounded fp32 division);
 *   code = clamp(rne(u * inv), -q, q); delta_t = ((r * A_t) * c_b) / q with c_b
 *   the float nearest 1/sqrt(b); a zero row gives codes 0 and delta 0.  No fused
 *   multiply-adds.
 */
#ifndef FQ_H_
#define FQ_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FQ_OK = 0,
  FQ_ERR_NULL = 1,        /* a required pointer is NULL */
  FQ_ERR_SHAPE = 2,       /* negative or inconsistent sizes, ld too small */
  FQ_ERR_UNSUPPORTED = 3, /* sizes outside the supported range, bad b / bits / clip ratio */
  FQ_ERR_ALIGN = 4,       /* pointer or leading dimension misaligned */
  FQ_ERR_WORKSPACE = 5,   /* workspace missing or smaller than required */
  FQ_ERR_HIP = 6,         /* a HIP runtime call or kernel launch failed */
  FQ_ERR_ALIAS = 7        /* an output buffer overlaps another output or an input */
} fq_status;

/* Runtime prologue, Alg. 1 runtime steps 1-2 (Sec. III-C transform, eq. (5)).
 *   x_bf16     [M, ldx] bf16 tokens (only the first K columns are read).
 *   smooth_inv [K] fp32 fold-before multiplier S^-1 (Sec. III-C), or NULL for S = I;
 *              multiplied into x once, in fp32, before the rotation.
 *   post_inv   [K] fp32 fold-after multiplier P^-1 (Sec. III-C), or NULL for P = I;
 *              multiplied into the rotated row once, in fp32, before the row absmax.
 *   b          Hadamard block size; bits: 4 or 8 (q = 7 or 127); clip_ratio: r in eq. (5).
 *   a_codes    output codes, canonical layout: bits = 8 -> int8 [M, K];
 *              bits = 4 -> uint8 [M, K/2], byte i of a row = channel 2i in the low
 *              nibble, channel 2i+1 in the high nibble (two's complement).
 *   delta      output fp32 [M] per-token scales (0 for a zero token). */
fq_status fq_fwht_quant(const void *x_bf16, int64_t ldx, const float *smooth_inv,
                        const float *post_inv, int64_t M, int64_t K, int b, int bits,
                        float clip_ratio, void *a_codes, float *delta, void *stream);

/* Offline weight fold and round-to-nearest, Alg. 1 offline (eq. (2), Sec. III-C/F).
 *   w          [N, ldw] fp32 weights of one consumer (row j = output channel j).
 *   col_scale  [K] fp32 S (fold-before smoothing, times a folded norm gain, eq. (4)),
 *              or NULL; multiplied into each row once, in fp32, before the rotation.
 *   post_scale [K] fp32 P (fold-after scale, Sec. III-C), or NULL; multiplied into
 *              each rotated row once, in fp32, before the row absmax.
 *   Row j of W S R^T P is p . R (s . w_j) because H_b is symmetric, so each row is
 *   rounded with the prologue's contract at r = 1: w_codes int8 [N, K] in [-q, q] and
 *   w_scale fp32 [N] (the per-output-channel s_j). */
fq_status fq_quantize_weights(const float *w, int64_t ldw, const float *col_scale,
                              const float *post_scale, int64_t N, int64_t K, int b, int bits,
                              int8_t *w_codes, float *w_scale, void *stream);

/* Prologue with the stored composite rotation (Sec. III-C: the action expert's optional
 * transform, a channel permutation followed by per-block SVD-Hadamard matrices) in place
 * of the block Hadamard: z_t = P^-1 B Pi S^-1 x_t with
 *   perm       int32 [K] or NULL (identity): output position c takes input channel perm[c]
 *              (entries outside [0, K) are clamped, giving wrong codes but no fault);
 *   blocks     fp32 [K/b, b, b], block k's matrix Q_k row-major, applied to positions
 *              [k b, (k+1) b); orthonormal blocks keep the scale (nothing deferred to delta);
 *   b          a power of two, 1 <= b <= 128 (a block's matrix is staged in LDS, 64 KB at
 *              b = 128); K <= 32768 and M <= 2^20.
 * Contract: after the optional S^-1 multiply and the gather, output i of block k is the
 * fp32 fused multiply-add chain over j = 0..b-1 ascending of Q_k[i][j] * w_{kb+j},
 * starting from +0; then the optional P^-1 multiply; then eq. (5) exactly as
 * fq_fwht_quant with c_b = 1.  Codes in the canonical layout, as fq_fwht_quant.
 *   ws         scratch of fq_rotate_quant_workspace_bytes(M, K) bytes (the fp32 rotated
 *              rows); no initialization needed. */
size_t fq_rotate_quant_workspace_bytes(int64_t M, int64_t K);
fq_status fq_rotate_quant(const void *x_bf16, int64_t ldx, const int32_t *perm, const float *blocks,
                          const float *smooth_inv, const float *post_inv, int64_t M, int64_t K, int b,
                          int bits, float clip_ratio, void *a_codes, float *delta, void *ws,
                          size_t ws_bytes, void *stream);

/* Offline weight fold and round-to-nearest for the composite rotation: row j of
 * W S R^T P with R = B Pi is rounded with fq_rotate_quant's contract at r = 1 (fp32 rows
 * [N, ldw], ldw a multiple of 4); w_codes int8 [N, K], w_scale fp32 [N]; ws as above
 * with M = N. */
fq_status fq_quantize_weights_rotated(const float *w, int64_t ldw, const int32_t *perm, const float *blocks,
                                      const float *col_scale, const float *post_scale, int64_t N, int64_t K,
                                      int b, int bits, int8_t *w_codes, float *w_scale, void *ws,
                                      size_t ws_bytes, void *stream);

/* Bytes of the packed, kernel-native weight layout for an [N, K] matrix. */
size_t fq_packed_weight_bytes(int64_t N, int64_t K, int bits);

/* Pack int8 codes [N, K] (values in [-q, q]) into the kernel-native layout that the
 * GEMM entry points read (Sec. III-F: packed signed-INT4 / INT8 weight codes).
 * The layout is opaque; fq_unpack_weights inverts it exactly. */
fq_status fq_pack_weights(const int8_t *w_codes, int64_t N, int64_t K, int bits, void *w_packed,
                          void *stream);
fq_status fq_unpack_weights(const void *w_packed, int64_t N, int64_t K, int bits, int8_t *w_codes,
                            void *stream);

/* Workspace bytes fq_gemm_w4a4 / fq_gemm_w8a8 need for this shape (may be 0). */
size_t fq_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int bits);

/* Integer GEMM with the eq. (8) rescale epilogue (Alg. 1 runtime, consumer loop).
 *   a_codes   canonical activation codes as written by fq_fwht_quant
 *             (w4a4: uint8 [M, K/2] nibbles; w8a8: int8 [M, K]).
 *   delta     fp32 [M]; w_packed: from fq_pack_weights with the same bits;
 *   w_scale   fp32 [N]; bias: fp32 [N] or NULL.
 *   y_bf16    [M, ldy] bf16 output: y = bf16_rne(fp32(acc) * (w_scale[j] * delta[t]) + bias[j]).
 *   acc_out   int32 [M, N] raw accumulators, or NULL (for verification).
 *   ws        scratch of at least fq_gemm_workspace_bytes(M, N, K, bits) bytes (0 when
 *             the shape needs none; ws may then be NULL).  It needs no initialization;
 *             it holds the INT32 partial sums of a split K between the GEMM kernel and
 *             its epilogue, or (W4A4, a few hundred rows at long K) a k-step-major copy
 *             of a_codes that the GEMM reads with coalesced loads.  Calls that share a
 *             workspace race unless they are ordered, e.g. on one stream.
 * Accumulation is exact: |acc| <= K q^2 < 2^31 for K <= 32768 at INT4 and
 * K <= 32768 at INT8 (127^2 * 32768 < 2^31 holds up to K = 133152). */
fq_status fq_gemm_w4a4(const void *a_codes, const float *delta, const void *w_packed,
                       const float *w_scale, const float *bias, void *y_bf16, int64_t ldy,
                       int32_t *acc_out, int64_t M, int64_t N, int64_t K, void *ws,
                       size_t ws_bytes, void *stream);
fq_status fq_gemm_w8a8(const void *a_codes, const float *delta, const void *w_packed,
                       const float *w_scale, const float *bias, void *y_bf16, int64_t ldy,
                       int32_t *acc_out, int64_t M, int64_t N, int64_t K, void *ws,
                       size_t ws_bytes, void *stream);

/* Weight-only INT4 projection (W4A16): the paper runs GR00T's adaptive layer-norm
 * modulation with floating-point activations and INT4 weights (Sec. III-A).
 *   x_bf16    [M, ldx] bf16 activations, not quantized (ldx >= K, multiple of 8).
 *   w_packed  INT4 weights from fq_pack_weights(bits = 4), rounded per output channel,
 *             typically with fq_quantize_weights at b = 1 (no rotation); w_scale fp32 [N].
 *   y_bf16    [M, ldy] bf16: y = bf16_rne(fp32(sum_c x_tc q_jc) * w_scale[j] + bias[j]).
 *   acc_out   fp32 [M, N] sums before the scale, or NULL (for verification).
 *   ws        scratch of fq_gemm_w4a16_workspace_bytes(M, N, K) bytes (fp32 partial sums
 *             of a split K; 0 bytes and NULL allowed when K is not split).
 * The sums are floating point on the bf16 matrix cores (every product of a bf16 and a
 * code is exact in fp32; the additions round), so they agree with an exact sum within
 * (K - 1) 2^-24 sum_c |x_tc q_jc|, not bit for bit.  Same shape limits as the other
 * entry points, and M <= 64 * 65535. */
size_t fq_gemm_w4a16_workspace_bytes(int64_t M, int64_t N, int64_t K);
fq_status fq_gemm_w4a16(const void *x_bf16, int64_t ldx, const void *w_packed, const float *w_scale,
                        const float *bias, void *y_bf16, int64_t ldy, float *acc_out, int64_t M,
                        int64_t N, int64_t K, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes fq_linear needs: the intermediate activation codes and scales, and the
 * split-K partial sums.  Scratch with no initialization requirement.  (The intermediate
 * codes are the canonical nibbles or int8, or for the shapes the k-group GEMM serves the
 * same nibbles stored k-step major: the same bytes in another order.) */
size_t fq_linear_workspace_bytes(int64_t M, int64_t N, int64_t K, int bits);

/* The whole runtime projection for one consumer (Alg. 1 runtime; eqs. (5), (8)):
 * prologue on x, integer GEMM against w_packed, rescale + bias, bf16 out.
 * Same arguments and contracts as fq_fwht_quant followed by fq_gemm_w{4a4,8a8}, and the
 * same output bit for bit; the intermediate codes and scales live in `ws`. */
fq_status fq_linear(const void *x_bf16, int64_t ldx, const float *smooth_inv, const float *post_inv,
                    int64_t M, int64_t K, int64_t N, int b, int bits, float clip_ratio,
                    const void *w_packed, const float *w_scale, const float *bias, void *y_bf16,
                    int64_t ldy, void *ws, size_t ws_bytes, void *stream);

/* fq_linear for callers that cannot allocate memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): the same arguments, kernels and
 * outputs bit for bit, without a workspace argument.  Its scratch is a device array inside
 * the library, fq_linear_static_max_workspace_bytes() = 64 MiB on every device the library
 * runs on, held until the process ends; a shape whose fq_linear_workspace_bytes exceeds it
 * is rejected with FQ_ERR_WORKSPACE before anything is enqueued.  The call allocates and
 * frees nothing (the array's device address is looked up once per device, on the first
 * call made with that device current).  All calls on one device share the array: calls
 * that may overlap on a device (different streams, different threads without ordering)
 * race; calls ordered on one stream do not.  The scratch needs no initialization. */
size_t fq_linear_static_max_workspace_bytes(void);
fq_status fq_linear_static(const void *x_bf16, int64_t ldx, const float *smooth_inv, const float *post_inv,
                           int64_t M, int64_t K, int64_t N, int b, int bits, float clip_ratio,
                           const void *w_packed, const float *w_scale, const float *bias, void *y_bf16,
                           int64_t ldy, void *stream);

/* Static description of a status code, and the thread-local message of the last failure. */
const char *fq_status_string(fq_status s);
const char *fq_last_error(void);

/* ---- GPTQ in the transformed coordinates (eq. (7), Sec. III-F) ----------------------------
 * Offline rounding of folded weights against the second moment G = Z Z^T of calibration
 * tokens taken in the runtime transform's coordinates, with diagonal damping (the GPTQ
 * method the paper names for its four-bit weights).  Four calls:
 *   fq_transform      tokens and weight rows into the transformed coordinates;
 *   fq_gptq_hessian   G = Z Z^T (fp64);
 *   fq_gptq_factor    U with (G + lambda I)^-1 = U^T U;
 *   fq_gptq_sweep     the column sweep, codes and per-output-channel scales.
 * All four take device pointers, enqueue on `stream` and return before the work is done. */

/* The prologue's transform without the quantization: z_t = P^-1 H_b S^-1 x_t, unnormalized
 * (Sylvester +-1 blocks, the same fp32 butterfly, stage order and multiplies as
 * fq_fwht_quant), fp32 rows z [M, K].  x: bf16 rows (x_is_f32 = 0, ldx a multiple of 8) or
 * fp32 rows (x_is_f32 = 1, ldx a multiple of 4); pre_mult / post_mult: fp32 [K] or NULL.
 * K a multiple of 128 in [128, 32768]; b a power of two <= 256 dividing K.  Weight rows go
 * through the same call (x_is_f32 = 1, pre_mult = the fold's S, post_mult = its P): since
 * H_b is symmetric, row j of W S H_b^T P is P H_b (S w_j). */
fq_status fq_transform(const void *x, int x_is_f32, int64_t ldx, const float *pre_mult, const float *post_mult,
                       int64_t M, int64_t K, int b, float *z, void *stream);

/* G = sum_t z_t z_t^T over T transformed tokens z [T, ldz] (fp32), in fp64, written in full
 * (symmetric) to G [K, K]; accumulate != 0 adds to the G already there, so calibration
 * batches can be streamed.  K a multiple of 128, at most 16384.  T = 0 with accumulate = 0
 * clears G. */
fq_status fq_gptq_hessian(const float *z, int64_t ldz, int64_t T, int64_t K, double *G, int accumulate,
                          void *stream);

/* U: fp64 [K, K] upper triangular (zeros below the diagonal) with H^-1 = U^T U, where
 * H = G + lambda I, lambda = damp * mean(diag G) (damp in [0, 1], 0.01 is the GPTQ
 * method's default); an all-zero diagonal gives H = I.  H must be positive definite
 * (damping > 0 guarantees it for a nonzero G); otherwise U holds NaNs.
 * ws: fq_gptq_factor_workspace_bytes(K) bytes (about 2 K^2 doubles), no initialization. */
size_t fq_gptq_factor_workspace_bytes(int64_t K);
fq_status fq_gptq_factor(const double *G, int64_t K, double damp, double *U, void *ws, size_t ws_bytes,
                         void *stream);

/* The GPTQ column sweep over folded weight rows w_t fp32 [N, ldw] (fq_transform's output
 * for the weights, with the same block size b), with U from fq_gptq_factor.  Contract
 * (fp64; the codes are reproducible bit for bit): per row A = max |w|, scale =
 * fl32((A * c_b) / q) with c_b the float nearest 1/sqrt(b) (the block Hadamard's
 * normalization, deferred to the scale exactly as in fq_quantize_weights), inv = q / A and
 * step = A / q; columns in blocks of 128; column c: code = clamp(rint(w_c * inv), -q, q),
 * e = (w_c - code * step) / U[c][c], each later column c' of the block w_c' =
 * fma(-e, U[c][c'], w_c'); after the block, each later column w_c' -= (fma chain over the
 * block's k ascending of e_k * U[k][c'] from +0).  A zero row gives codes 0 and scale 0.
 * w_codes int8 [N, K] (pack with fq_pack_weights); w_scale fp32 [N];
 * ws: fq_gptq_sweep_workspace_bytes(N, K) bytes, no initialization. */
size_t fq_gptq_sweep_workspace_bytes(int64_t N, int64_t K);
fq_status fq_gptq_sweep(const float *w_t, int64_t ldw, const double *U, int64_t N, int64_t K, int b, int bits,
                        int8_t *w_codes, float *w_scale, void *ws, size_t ws_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* FQ_H_ */
