// C ABI of libfq: argument validation, workspace layout and dispatch to the gfx950 kernels.
// Every check runs before anything is enqueued, so a failing call has no device effect.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <atomic>
#include <cstring>
#include <initializer_list>

#include "../../include/fq.h"
#include "fq_launch.hpp"

// Scratch of fq_linear_static: the workspace of fq_linear in a file-scope device array
// instead of a caller's buffer.  In host code `scratch` names a host-side stand-in, not the
// device array: its device address comes from hipGetSymbolAddress, once per device.
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

namespace {

thread_local char g_err[512] = "";

fq_status fail(fq_status s, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return s;
}

fq_status ok() {
  g_err[0] = '\0';
  return FQ_OK;
}

fq_status hip_fail(hipError_t e, const char *where) {
  return fail(FQ_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool is_pow2(int64_t v) { return v >= 1 && (v & (v - 1)) == 0; }

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Byte range [p, p + n) of a caller buffer, for the no-overlap preconditions.
struct Span {
  uintptr_t lo, hi;
};
Span span(const void *p, size_t n) { return Span{reinterpret_cast<uintptr_t>(p), reinterpret_cast<uintptr_t>(p) + n}; }
bool overlap(Span a, Span b) { return a.lo && b.lo && a.lo < b.hi && b.lo < a.hi; }
// True when an output range overlaps another output or any input (NULL ranges are empty).
bool outputs_alias(std::initializer_list<Span> outs, std::initializer_list<Span> ins) {
  for (auto o = outs.begin(); o != outs.end(); ++o) {
    for (auto p = o + 1; p != outs.end(); ++p)
      if (overlap(*o, *p)) return true;
    for (const Span &i : ins)
      if (overlap(*o, i)) return true;
  }
  return false;
}
// Bytes spanned by `rows` rows of `row_bytes` bytes at a stride of `ld_bytes`.
size_t rows_span(int64_t rows, int64_t ld_bytes, int64_t row_bytes) {
  return rows <= 0 ? 0 : (size_t)(rows - 1) * (size_t)ld_bytes + (size_t)row_bytes;
}

constexpr int64_t kMaxK = 32768;
constexpr int64_t kMaxGptqK = 16384;  // the factor holds two K x K fp64 matrices

// float nearest to 1/sqrt(b), b = 2^k: 2^(-k/2) for even k, 2^(-(k-1)/2) / sqrt(2) for odd k
float inv_sqrt_pow2(int b) {
  int k = 0;
  while ((1 << k) < b) ++k;
  const float rsqrt2 = 0x1.6a09e6p-1f;  // nearest float to 1/sqrt(2)
  return (k & 1) ? std::ldexp(rsqrt2, -(k - 1) / 2) : std::ldexp(1.0f, -k / 2);
}

fq_status check_k(int64_t K) {
  if (K < 128 || K > kMaxK) return fail(FQ_ERR_UNSUPPORTED, "K=%lld outside [128, %lld]", (long long)K, (long long)kMaxK);
  if (K % 128) return fail(FQ_ERR_UNSUPPORTED, "K=%lld is not a multiple of 128", (long long)K);
  return FQ_OK;
}

fq_status check_bits(int bits) {
  if (bits != 4 && bits != 8) return fail(FQ_ERR_UNSUPPORTED, "bits=%d (must be 4 or 8)", bits);
  return FQ_OK;
}

fq_status check_block(int b, int64_t K) {
  if (!is_pow2(b) || b > 256) return fail(FQ_ERR_UNSUPPORTED, "b=%d is not a power of two in [1, 256]", b);
  if (K % b) return fail(FQ_ERR_SHAPE, "K=%lld is not a multiple of b=%d", (long long)K, b);
  return FQ_OK;
}

// Shape/argument checks of the prologue; `ld_mult` is the element multiple that keeps
// rows 16-byte aligned (8 for bf16, 4 for fp32).
fq_status check_prologue_shape(int64_t ldx, int ld_mult, int64_t M, int64_t K, int b, int bits,
                               float r) {
  if (M < 0) return fail(FQ_ERR_SHAPE, "M=%lld < 0", (long long)M);
  fq_status s;
  if ((s = check_k(K)) != FQ_OK) return s;
  if ((s = check_bits(bits)) != FQ_OK) return s;
  if ((s = check_block(b, K)) != FQ_OK) return s;
  if (!(r > 0.0f && r <= 1.0f)) return fail(FQ_ERR_UNSUPPORTED, "clip_ratio=%g outside (0, 1]", (double)r);
  if (ldx < K) return fail(FQ_ERR_SHAPE, "leading dimension %lld < K=%lld", (long long)ldx, (long long)K);
  if (ldx % ld_mult) return fail(FQ_ERR_ALIGN, "leading dimension %lld is not a multiple of %d", (long long)ldx, ld_mult);
  return FQ_OK;
}

fq_status check_prologue(const void *x, int64_t ldx, int ld_mult, const float *smooth,
                         const float *post, int64_t M, int64_t K, int b, int bits, float r,
                         const void *codes, const float *delta) {
  fq_status s = check_prologue_shape(ldx, ld_mult, M, K, b, bits, r);
  if (s != FQ_OK || M == 0) return s;
  if (!x || !codes || !delta) return fail(FQ_ERR_NULL, "input, codes and scales must be non-NULL");
  if (!aligned16(x) || !aligned16(codes) || !aligned16(delta) || (smooth && !aligned16(smooth)) ||
      (post && !aligned16(post)))
    return fail(FQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  return FQ_OK;
}

// No-overlap precondition of a prologue: the codes, the scales and `extra` (a workspace, or
// an empty span) against each other and against the rows, the multipliers and `extra_in`.
fq_status check_prologue_alias(const void *x, int64_t ldx, int in_bytes, const float *smooth, const float *post,
                               int64_t M, int64_t K, int bits, const void *codes, const float *delta,
                               Span extra = Span{0, 0}, Span extra_in = Span{0, 0}) {
  if (outputs_alias({span(codes, (size_t)M * (size_t)K * (size_t)bits / 8), span(delta, (size_t)M * 4), extra},
                    {span(x, rows_span(M, ldx * in_bytes, K * in_bytes)), span(smooth, (size_t)K * 4),
                     span(post, (size_t)K * 4), extra_in}))
    return fail(FQ_ERR_ALIAS, "codes, scales and workspace must not overlap each other or an input");
  return FQ_OK;
}

fq_status check_gemm(const void *a, const float *delta, const void *w, const float *w_scale,
                     const float *bias, const void *y, int64_t ldy, const int32_t *acc_out,
                     int64_t M, int64_t N, int64_t K) {
  if (M < 0 || N < 0) return fail(FQ_ERR_SHAPE, "M=%lld, N=%lld must be >= 0", (long long)M, (long long)N);
  fq_status s;
  if ((s = check_k(K)) != FQ_OK) return s;
  if (N % 16) return fail(FQ_ERR_UNSUPPORTED, "N=%lld is not a multiple of 16", (long long)N);
  if (N > (1ll << 24) || M > (1ll << 24)) return fail(FQ_ERR_UNSUPPORTED, "M or N too large");
  // keeps every tile count and tile index of the launch grids within 31 bits
  if (M * N > (1ll << 40)) return fail(FQ_ERR_UNSUPPORTED, "M x N = %lld outputs is too large", (long long)(M * N));
  if (ldy < N) return fail(FQ_ERR_SHAPE, "ldy=%lld < N=%lld", (long long)ldy, (long long)N);
  if (ldy % 8) return fail(FQ_ERR_ALIGN, "ldy=%lld is not a multiple of 8", (long long)ldy);
  if (M == 0 || N == 0) return FQ_OK;
  if (!a || !delta || !w || !w_scale || !y) return fail(FQ_ERR_NULL, "a, delta, w, w_scale and y must be non-NULL");
  if (!aligned16(a) || !aligned16(delta) || !aligned16(w) || !aligned16(w_scale) || !aligned16(y) ||
      (bias && !aligned16(bias)) || (acc_out && !aligned16(acc_out)))
    return fail(FQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  return FQ_OK;
}

fq_status gemm_common(const void *a_codes, int a_fmt, int64_t lda, const float *delta,
                      const void *w_packed, const float *w_scale, const float *bias, void *y,
                      int64_t ldy, int32_t *acc_out, int64_t M, int64_t N, int64_t K, int bits,
                      void *ws, size_t ws_bytes, hipStream_t stream, bool go = true) {
  const fq::GemmPlan pl = fq::plan_gemm(M, N, K, bits, a_fmt == fq::kANibbleKM);
  const size_t need = fq::gemm_plan_workspace(pl) + (a_fmt == fq::kANibble ? fq::gemm_plan_relayout_bytes(pl, M, K) : 0);
  if (need > 0 && (!ws || ws_bytes < need))
    return fail(FQ_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws ? ws_bytes : (size_t)0);
  if (need > 0 && !aligned16(ws)) return fail(FQ_ERR_ALIGN, "workspace must be 16-byte aligned");
  fq::GemmArgs g;
  g.a = static_cast<const uint8_t *>(a_codes);
  g.lda = lda;
  g.a_fmt = a_fmt;
  g.delta = delta;
  g.w = static_cast<const uint8_t *>(w_packed);
  g.w_scale = w_scale;
  g.bias = bias;
  g.y = static_cast<uint16_t *>(y);
  g.ldy = ldy;
  g.acc_out = acc_out;
  g.M = M;
  g.N = N;
  g.K = K;
  g.bits = bits;
  hipError_t e = fq::launch_gemm(g, pl, ws, stream, go);
  if (e != hipSuccess) return hip_fail(e, go ? "gemm launch" : "gemm kernel selection");
  return ok();
}

fq_status gemm_entry(int bits, const void *a_codes, const float *delta, const void *w_packed,
                     const float *w_scale, const float *bias, void *y, int64_t ldy, int32_t *acc_out,
                     int64_t M, int64_t N, int64_t K, void *ws, size_t ws_bytes, void *stream) {
  fq_status s = check_gemm(a_codes, delta, w_packed, w_scale, bias, y, ldy, acc_out, M, N, K);
  if (s != FQ_OK) return s;
  if (M == 0 || N == 0) return ok();
  const int a_fmt = bits == 4 ? fq::kANibble : fq::kAInt8;
  const int64_t lda = bits == 4 ? K / 2 : K;
  const size_t need = fq_gemm_workspace_bytes(M, N, K, bits);
  if (need > 0 && (!ws || ws_bytes < need))
    return fail(FQ_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws ? ws_bytes : (size_t)0);
  if (outputs_alias({span(y, rows_span(M, ldy * 2, N * 2)), span(acc_out, acc_out ? (size_t)M * N * 4 : 0),
                     span(need ? ws : nullptr, need)},
                    {span(a_codes, (size_t)M * lda), span(delta, (size_t)M * 4),
                     span(w_packed, fq_packed_weight_bytes(N, K, bits)), span(w_scale, (size_t)N * 4),
                     span(bias, bias ? (size_t)N * 4 : 0)}))
    return fail(FQ_ERR_ALIAS, "y, acc_out and the workspace must not overlap each other or an input");
  return gemm_common(a_codes, a_fmt, lda, delta, w_packed, w_scale, bias, y, ldy, acc_out, M, N, K,
                     bits, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

// fq_linear workspace: none when one fused kernel runs the projection (few tokens, K up
// to 4096); otherwise [codes (nibbles for W4A4, int8 for W8A8)][delta][split-K partials]
size_t linear_ws_bytes(int64_t M, int64_t N, int64_t K, int bits) {
  if (M <= 0 || N <= 0 || K < 128 || (bits != 4 && bits != 8)) return 0;
  if (fq::plan_small(M, N, K, bits).ok) return 0;
  return align256((size_t)M * (size_t)K * (size_t)bits / 8) + align256((size_t)M * 4) +
         fq::gemm_plan_workspace(fq::plan_gemm(M, N, K, bits, bits == 4));
}

int log2_pow2(int b) {
  int k = 0;
  while ((1 << k) < b) ++k;
  return k;
}

// The fused projection: both stages are validated, and the GEMM's kernel is resolved,
// before the prologue is enqueued, so a failing call enqueues nothing.
fq_status linear_common(const void *x_bf16, int64_t ldx, const float *smooth_inv, const float *post_inv,
                        int64_t M, int64_t K, int64_t N, int b, int bits, float clip_ratio,
                        const void *w_packed, const float *w_scale, const float *bias, void *y_bf16,
                        int64_t ldy, void *ws, size_t ws_bytes, void *stream) {
  fq_status s = check_prologue_shape(ldx, 8, M, K, b, bits, clip_ratio);
  if (s != FQ_OK) return s;
  if (M > 0 && smooth_inv && !aligned16(smooth_inv)) return fail(FQ_ERR_ALIGN, "smooth_inv must be 16-byte aligned");
  if (M > 0 && post_inv && !aligned16(post_inv)) return fail(FQ_ERR_ALIGN, "post_inv must be 16-byte aligned");
  s = check_gemm(x_bf16, w_scale, w_packed, w_scale, bias, y_bf16, ldy, nullptr, M, N, K);
  if (s != FQ_OK) return s;
  if (M == 0 || N == 0) return ok();
  const size_t codes_bytes = align256((size_t)M * (size_t)K * (size_t)bits / 8);
  const size_t delta_bytes = align256((size_t)M * 4);
  const size_t need = linear_ws_bytes(M, N, K, bits);
  if (need > 0 && (!ws || ws_bytes < need))
    return fail(FQ_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws ? ws_bytes : (size_t)0);
  if (need > 0 && !aligned16(ws)) return fail(FQ_ERR_ALIGN, "workspace must be 16-byte aligned");
  if (outputs_alias({span(y_bf16, rows_span(M, ldy * 2, N * 2)), span(need ? ws : nullptr, need)},
                    {span(x_bf16, rows_span(M, ldx * 2, K * 2)), span(smooth_inv, smooth_inv ? (size_t)K * 4 : 0),
                     span(post_inv, post_inv ? (size_t)K * 4 : 0), span(w_packed, fq_packed_weight_bytes(N, K, bits)),
                     span(w_scale, (size_t)N * 4), span(bias, bias ? (size_t)N * 4 : 0)}))
    return fail(FQ_ERR_ALIAS, "y and the workspace must not overlap each other or an input");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const fq::SmallPlan sp = fq::plan_small(M, N, K, bits);
  if (sp.ok) {
    fq::SmallArgs a;
    a.x = x_bf16;
    a.ldx = ldx;
    a.chan_mult = smooth_inv;
    a.post_mult = post_inv;
    a.w = static_cast<const uint8_t *>(w_packed);
    a.w_scale = w_scale;
    a.bias = bias;
    a.y = static_cast<uint16_t *>(y_bf16);
    a.ldy = ldy;
    a.M = M;
    a.N = N;
    a.K = K;
    a.log2b = log2_pow2(b);
    a.bits = bits;
    a.clip_ratio = clip_ratio;
    a.cb = inv_sqrt_pow2(b);
    hipError_t e = fq::launch_linear_small(a, sp, st);
    if (e != hipSuccess) return hip_fail(e, "fused projection launch");
    return ok();
  }
  uint8_t *codes = static_cast<uint8_t *>(ws);
  float *delta = reinterpret_cast<float *>(codes + codes_bytes);
  void *gws = codes + codes_bytes + delta_bytes;
  const size_t gws_bytes = ws_bytes - codes_bytes - delta_bytes;
  // W4A4 codes between the two kernels are nibbles (half the bytes of int8, the same
  // per-step cost in the GEMMs, which widen them in registers), canonical or, for the
  // k-group GEMM, k-step major; W8A8 codes are int8.
  const bool nibble = bits == 4;
  const bool kmajor = nibble && fq::plan_gemm(M, N, K, bits, true).kind == 3;
  const int fmt = nibble ? (kmajor ? fq::kOutNibbleKM : fq::kOutNibble) : fq::kOutInt8;
  const int afmt = nibble ? (kmajor ? fq::kANibbleKM : fq::kANibble) : fq::kAInt8;
  const int64_t lda = nibble ? K / 2 : K;
  s = gemm_common(codes, afmt, lda, delta, w_packed, w_scale, bias, y_bf16, ldy, nullptr, M, N, K, bits, gws,
                  gws_bytes, st, /*go=*/false);
  if (s != FQ_OK) return s;
  hipError_t e = fq::launch_fwht_quant(x_bf16, false, ldx, smooth_inv, post_inv, M, (int)K, b, bits,
                                       clip_ratio, inv_sqrt_pow2(b), codes, lda, delta, fmt, st);
  if (e != hipSuccess) return hip_fail(e, "fwht_quant launch");
  return gemm_common(codes, afmt, lda, delta, w_packed, w_scale, bias, y_bf16, ldy, nullptr, M, N, K, bits, gws,
                     gws_bytes, st);
}

// Device address of `scratch` on the current device, looked up once per device with that
// device current (each device holds its own copy of the array).  Concurrent first calls
// may both look it up; they store the same address.
constexpr int kMaxDevices = 64;
std::atomic<void *> g_scratch_ptr[kMaxDevices];

fq_status static_scratch(void **out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(FQ_ERR_UNSUPPORTED, "device %d beyond %d devices", dev, kMaxDevices);
  void *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(FQ_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return FQ_OK;
}

fq_status rotate_common(const void *x, bool x_f32, int64_t ldx, const int32_t *perm, const float *blocks,
                        const float *pre, const float *post, int64_t M, int64_t K, int b, int bits, float r,
                        void *codes, int64_t ldc, float *delta, int fmt, void *ws, size_t ws_bytes,
                        void *stream) {
  fq_status s = check_prologue(x, ldx, x_f32 ? 4 : 8, pre, post, M, K, b, bits, r, codes, delta);
  if (s != FQ_OK) return s;
  if (b > 128) return fail(FQ_ERR_UNSUPPORTED, "b=%d: the composite rotation holds blocks of at most 128", b);
  if (K > 32768) return fail(FQ_ERR_UNSUPPORTED, "K=%lld: the composite rotation handles K <= 32768", (long long)K);
  if (M > (1ll << 20)) return fail(FQ_ERR_UNSUPPORTED, "M=%lld: the composite rotation handles M <= 2^20 rows", (long long)M);
  if (M == 0) return ok();
  if (!blocks) return fail(FQ_ERR_NULL, "blocks must be non-NULL");
  if (!aligned16(blocks) || (perm && !aligned16(perm)))
    return fail(FQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  const size_t need = fq_rotate_quant_workspace_bytes(M, K);
  if (!ws || ws_bytes < need)
    return fail(FQ_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws ? ws_bytes : (size_t)0);
  if (!aligned16(ws)) return fail(FQ_ERR_ALIGN, "workspace must be 16-byte aligned");
  s = check_prologue_alias(x, ldx, x_f32 ? 4 : 2, pre, post, M, K, fmt == fq::kOutNibble ? 4 : 8, codes, delta,
                           span(ws, need), span(blocks, (size_t)K * b * 4));
  if (s != FQ_OK) return s;
  if (perm && overlap(span(perm, (size_t)K * 4), span(ws, need))) return fail(FQ_ERR_ALIAS, "perm overlaps the workspace");
  hipError_t e = fq::launch_rotate_quant(x, x_f32, ldx, perm, blocks, pre, post, M, (int)K, b, bits, r,
                                         static_cast<uint8_t *>(codes), ldc, delta, fmt,
                                         static_cast<float *>(ws), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "rotate_quant launch");
  return ok();
}

}  // namespace

extern "C" {

const char *fq_status_string(fq_status s) {
  switch (s) {
    case FQ_OK: return "ok";
    case FQ_ERR_NULL: return "null pointer";
    case FQ_ERR_SHAPE: return "bad shape";
    case FQ_ERR_UNSUPPORTED: return "unsupported argument";
    case FQ_ERR_ALIGN: return "misaligned pointer or leading dimension";
    case FQ_ERR_WORKSPACE: return "workspace too small";
    case FQ_ERR_HIP: return "HIP runtime error";
    case FQ_ERR_ALIAS: return "output overlaps another buffer";
  }
  return "unknown status";
}

const char *fq_last_error(void) { return g_err; }

fq_status fq_fwht_quant(const void *x_bf16, int64_t ldx, const float *smooth_inv,
                        const float *post_inv, int64_t M, int64_t K, int b, int bits,
                        float clip_ratio, void *a_codes, float *delta, void *stream) {
  fq_status s = check_prologue(x_bf16, ldx, 8, smooth_inv, post_inv, M, K, b, bits, clip_ratio, a_codes, delta);
  if (s != FQ_OK) return s;
  if (M == 0) return ok();
  s = check_prologue_alias(x_bf16, ldx, 2, smooth_inv, post_inv, M, K, bits, a_codes, delta);
  if (s != FQ_OK) return s;
  const int fmt = bits == 4 ? fq::kOutNibble : fq::kOutInt8;
  const int64_t ldc = bits == 4 ? K / 2 : K;
  hipError_t e = fq::launch_fwht_quant(x_bf16, false, ldx, smooth_inv, post_inv, M, (int)K, b, bits,
                                       clip_ratio, inv_sqrt_pow2(b), static_cast<uint8_t *>(a_codes), ldc,
                                       delta, fmt, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "fwht_quant launch");
  return ok();
}

fq_status fq_quantize_weights(const float *w, int64_t ldw, const float *col_scale,
                              const float *post_scale, int64_t N, int64_t K, int b, int bits,
                              int8_t *w_codes, float *w_scale, void *stream) {
  fq_status s = check_prologue(w, ldw, 4, col_scale, post_scale, N, K, b, bits, 1.0f, w_codes, w_scale);
  if (s != FQ_OK) return s;
  if (N == 0) return ok();
  s = check_prologue_alias(w, ldw, 4, col_scale, post_scale, N, K, 8, w_codes, w_scale);
  if (s != FQ_OK) return s;
  hipError_t e = fq::launch_fwht_quant(w, true, ldw, col_scale, post_scale, N, (int)K, b, bits, 1.0f,
                                       inv_sqrt_pow2(b), reinterpret_cast<uint8_t *>(w_codes), K,
                                       w_scale, fq::kOutInt8, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "quantize_weights launch");
  return ok();
}

size_t fq_rotate_quant_workspace_bytes(int64_t M, int64_t K) {
  if (M <= 0 || K < 128) return 0;
  return align256((size_t)M * (size_t)K * 4);
}


fq_status fq_rotate_quant(const void *x_bf16, int64_t ldx, const int32_t *perm, const float *blocks,
                          const float *smooth_inv, const float *post_inv, int64_t M, int64_t K, int b,
                          int bits, float clip_ratio, void *a_codes, float *delta, void *ws,
                          size_t ws_bytes, void *stream) {
  const bool nib = bits == 4;
  return rotate_common(x_bf16, false, ldx, perm, blocks, smooth_inv, post_inv, M, K, b, bits, clip_ratio,
                       a_codes, nib ? K / 2 : K, delta, nib ? fq::kOutNibble : fq::kOutInt8, ws, ws_bytes,
                       stream);
}

fq_status fq_quantize_weights_rotated(const float *w, int64_t ldw, const int32_t *perm, const float *blocks,
                                      const float *col_scale, const float *post_scale, int64_t N, int64_t K,
                                      int b, int bits, int8_t *w_codes, float *w_scale, void *ws,
                                      size_t ws_bytes, void *stream) {
  return rotate_common(w, true, ldw, perm, blocks, col_scale, post_scale, N, K, b, bits, 1.0f, w_codes, K,
                       w_scale, fq::kOutInt8, ws, ws_bytes, stream);
}

size_t fq_packed_weight_bytes(int64_t N, int64_t K, int bits) {
  if (N < 0 || K < 0 || (bits != 4 && bits != 8)) return 0;
  return (size_t)N * (size_t)K * (size_t)bits / 8;
}

fq_status fq_pack_weights(const int8_t *w_codes, int64_t N, int64_t K, int bits, void *w_packed,
                          void *stream) {
  fq_status s;
  if (N < 0) return fail(FQ_ERR_SHAPE, "N=%lld < 0", (long long)N);
  if (N % 16) return fail(FQ_ERR_UNSUPPORTED, "N=%lld is not a multiple of 16", (long long)N);
  if ((s = check_k(K)) != FQ_OK) return s;
  if ((s = check_bits(bits)) != FQ_OK) return s;
  if (N == 0) return ok();
  if (!w_codes || !w_packed) return fail(FQ_ERR_NULL, "w_codes and w_packed must be non-NULL");
  if (!aligned16(w_codes) || !aligned16(w_packed)) return fail(FQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  if (overlap(span(w_codes, (size_t)N * K), span(w_packed, fq_packed_weight_bytes(N, K, bits))))
    return fail(FQ_ERR_ALIAS, "w_codes and w_packed must not overlap");
  hipError_t e = fq::launch_pack_weights(w_codes, N, (int)K, bits, static_cast<uint8_t *>(w_packed),
                                         static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "pack launch");
  return ok();
}

fq_status fq_unpack_weights(const void *w_packed, int64_t N, int64_t K, int bits, int8_t *w_codes,
                            void *stream) {
  fq_status s;
  if (N < 0) return fail(FQ_ERR_SHAPE, "N=%lld < 0", (long long)N);
  if (N % 16) return fail(FQ_ERR_UNSUPPORTED, "N=%lld is not a multiple of 16", (long long)N);
  if ((s = check_k(K)) != FQ_OK) return s;
  if ((s = check_bits(bits)) != FQ_OK) return s;
  if (N == 0) return ok();
  if (!w_codes || !w_packed) return fail(FQ_ERR_NULL, "w_codes and w_packed must be non-NULL");
  if (!aligned16(w_codes) || !aligned16(w_packed)) return fail(FQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  if (overlap(span(w_codes, (size_t)N * K), span(w_packed, fq_packed_weight_bytes(N, K, bits))))
    return fail(FQ_ERR_ALIAS, "w_codes and w_packed must not overlap");
  hipError_t e = fq::launch_unpack_weights(static_cast<const uint8_t *>(w_packed), N, (int)K, bits,
                                           w_codes, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "unpack launch");
  return ok();
}

size_t fq_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int bits) {
  if (M <= 0 || N <= 0 || K < 128 || (bits != 4 && bits != 8)) return 0;
  const fq::GemmPlan pl = fq::plan_gemm(M, N, K, bits);
  return fq::gemm_plan_workspace(pl) + fq::gemm_plan_relayout_bytes(pl, M, K);
}

fq_status fq_gemm_w4a4(const void *a_codes, const float *delta, const void *w_packed,
                       const float *w_scale, const float *bias, void *y_bf16, int64_t ldy,
                       int32_t *acc_out, int64_t M, int64_t N, int64_t K, void *ws,
                       size_t ws_bytes, void *stream) {
  return gemm_entry(4, a_codes, delta, w_packed, w_scale, bias, y_bf16, ldy, acc_out, M, N, K, ws,
                    ws_bytes, stream);
}

fq_status fq_gemm_w8a8(const void *a_codes, const float *delta, const void *w_packed,
                       const float *w_scale, const float *bias, void *y_bf16, int64_t ldy,
                       int32_t *acc_out, int64_t M, int64_t N, int64_t K, void *ws,
                       size_t ws_bytes, void *stream) {
  return gemm_entry(8, a_codes, delta, w_packed, w_scale, bias, y_bf16, ldy, acc_out, M, N, K, ws,
                    ws_bytes, stream);
}

size_t fq_gemm_w4a16_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  if (M <= 0 || N <= 0 || K < 128) return 0;
  return fq::plan_w4a16(M, N, K).partial_bytes;
}

fq_status fq_gemm_w4a16(const void *x_bf16, int64_t ldx, const void *w_packed, const float *w_scale,
                        const float *bias, void *y_bf16, int64_t ldy, float *acc_out, int64_t M,
                        int64_t N, int64_t K, void *ws, size_t ws_bytes, void *stream) {
  fq_status s = check_gemm(x_bf16, w_scale, w_packed, w_scale, bias, y_bf16, ldy, nullptr, M, N, K);
  if (s != FQ_OK) return s;
  if (ldx < K) return fail(FQ_ERR_SHAPE, "leading dimension %lld < K=%lld", (long long)ldx, (long long)K);
  if (ldx % 8) return fail(FQ_ERR_ALIGN, "leading dimension %lld is not a multiple of 8", (long long)ldx);
  if (M == 0 || N == 0) return ok();
  if (acc_out && !aligned16(acc_out)) return fail(FQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  const fq::W16Plan pl = fq::plan_w4a16(M, N, K);
  if (pl.rb > 65535) return fail(FQ_ERR_UNSUPPORTED, "M=%lld: at most %d rows", (long long)M, 64 * 65535);
  if (pl.partial_bytes > 0 && (!ws || ws_bytes < pl.partial_bytes))
    return fail(FQ_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", pl.partial_bytes,
                ws ? ws_bytes : (size_t)0);
  if (pl.partial_bytes > 0 && !aligned16(ws)) return fail(FQ_ERR_ALIGN, "workspace must be 16-byte aligned");
  fq::W16Args g;
  g.x = x_bf16;
  g.ldx = ldx;
  g.w = static_cast<const uint8_t *>(w_packed);
  g.w_scale = w_scale;
  g.bias = bias;
  g.y = static_cast<uint16_t *>(y_bf16);
  g.ldy = ldy;
  g.acc_out = acc_out;
  g.M = M;
  g.N = N;
  g.K = K;
  if (outputs_alias({span(y_bf16, rows_span(M, ldy * 2, N * 2)), span(acc_out, acc_out ? (size_t)M * N * 4 : 0),
                     span(pl.partial_bytes ? ws : nullptr, pl.partial_bytes)},
                    {span(x_bf16, rows_span(M, ldx * 2, K * 2)), span(w_packed, fq_packed_weight_bytes(N, K, 4)),
                     span(w_scale, (size_t)N * 4), span(bias, bias ? (size_t)N * 4 : 0)}))
    return fail(FQ_ERR_ALIAS, "y, acc_out and the workspace must not overlap each other or an input");
  hipError_t e = fq::launch_w4a16(g, pl, ws, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "w4a16 launch");
  return ok();
}

size_t fq_linear_workspace_bytes(int64_t M, int64_t N, int64_t K, int bits) {
  return linear_ws_bytes(M, N, K, bits);
}

fq_status fq_linear(const void *x_bf16, int64_t ldx, const float *smooth_inv, const float *post_inv,
                    int64_t M, int64_t K, int64_t N, int b, int bits, float clip_ratio,
                    const void *w_packed, const float *w_scale, const float *bias, void *y_bf16,
                    int64_t ldy, void *ws, size_t ws_bytes, void *stream) {
  return linear_common(x_bf16, ldx, smooth_inv, post_inv, M, K, N, b, bits, clip_ratio, w_packed, w_scale, bias,
                       y_bf16, ldy, ws, ws_bytes, stream);
}

size_t fq_linear_static_max_workspace_bytes(void) { return kStaticScratchBytes; }

fq_status fq_linear_static(const void *x_bf16, int64_t ldx, const float *smooth_inv, const float *post_inv,
                           int64_t M, int64_t K, int64_t N, int b, int bits, float clip_ratio,
                           const void *w_packed, const float *w_scale, const float *bias, void *y_bf16,
                           int64_t ldy, void *stream) {
  // the shape checks come first, so that a bad shape reports itself rather than a size
  fq_status s = check_prologue_shape(ldx, 8, M, K, b, bits, clip_ratio);
  if (s != FQ_OK) return s;
  if ((s = check_gemm(x_bf16, w_scale, w_packed, w_scale, bias, y_bf16, ldy, nullptr, M, N, K)) != FQ_OK) return s;
  if (M == 0 || N == 0) return ok();
  const size_t need = linear_ws_bytes(M, N, K, bits);
  if (need > kStaticScratchBytes)
    return fail(FQ_ERR_WORKSPACE, "this shape needs %zu bytes of scratch; fq_linear_static holds %zu", need,
                kStaticScratchBytes);
  void *ws = nullptr;
  if (need > 0 && (s = static_scratch(&ws)) != FQ_OK) return s;
  return linear_common(x_bf16, ldx, smooth_inv, post_inv, M, K, N, b, bits, clip_ratio, w_packed, w_scale, bias,
                       y_bf16, ldy, ws, need > 0 ? kStaticScratchBytes : 0, stream);
}

// ---- GPTQ in the transformed coordinates (eq. (7)) ----

fq_status fq_transform(const void *x, int x_is_f32, int64_t ldx, const float *pre_mult, const float *post_mult,
                       int64_t M, int64_t K, int b, float *z, void *stream) {
  fq_status s = check_prologue_shape(ldx, x_is_f32 ? 4 : 8, M, K, b, 4, 1.0f);
  if (s != FQ_OK) return s;
  if (M == 0) return ok();
  if (!x || !z) return fail(FQ_ERR_NULL, "x and z must be non-NULL");
  if (!aligned16(x) || !aligned16(z) || (pre_mult && !aligned16(pre_mult)) || (post_mult && !aligned16(post_mult)))
    return fail(FQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  {
    const int in_bytes = x_is_f32 ? 4 : 2;
    if (outputs_alias({span(z, (size_t)M * K * 4)}, {span(x, rows_span(M, ldx * in_bytes, K * in_bytes)),
                                                      span(pre_mult, pre_mult ? (size_t)K * 4 : 0),
                                                      span(post_mult, post_mult ? (size_t)K * 4 : 0)}))
      return fail(FQ_ERR_ALIAS, "z must not overlap an input");
  }
  hipError_t e = fq::launch_transform(x, x_is_f32 != 0, ldx, pre_mult, post_mult, M, (int)K, b, z,
                                      static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "transform launch");
  return ok();
}

fq_status fq_gptq_hessian(const float *z, int64_t ldz, int64_t T, int64_t K, double *G, int accumulate,
                          void *stream) {
  fq_status s;
  if ((s = check_k(K)) != FQ_OK) return s;
  if (K > kMaxGptqK) return fail(FQ_ERR_UNSUPPORTED, "K=%lld: GPTQ handles K <= %lld", (long long)K, (long long)kMaxGptqK);
  if (T < 0) return fail(FQ_ERR_SHAPE, "T=%lld < 0", (long long)T);
  if (ldz < K) return fail(FQ_ERR_SHAPE, "ldz=%lld < K=%lld", (long long)ldz, (long long)K);
  if (!G || (T > 0 && !z)) return fail(FQ_ERR_NULL, "z and G must be non-NULL");
  if (!aligned16(G) || (z && !aligned16(z))) return fail(FQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  if (T > 0 && overlap(span(G, (size_t)K * K * 8), span(z, rows_span(T, ldz * 4, K * 4))))
    return fail(FQ_ERR_ALIAS, "G must not overlap z");
  hipError_t e = fq::launch_gptq_hessian(z, ldz, T, (int)K, G, accumulate != 0, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "gptq_hessian launch");
  return ok();
}

size_t fq_gptq_factor_workspace_bytes(int64_t K) {
  if (K < 128 || K > kMaxGptqK) return 0;
  return fq::gptq_factor_ws_bytes((int)K);
}

fq_status fq_gptq_factor(const double *G, int64_t K, double damp, double *U, void *ws, size_t ws_bytes,
                         void *stream) {
  fq_status s;
  if ((s = check_k(K)) != FQ_OK) return s;
  if (K > kMaxGptqK) return fail(FQ_ERR_UNSUPPORTED, "K=%lld: GPTQ handles K <= %lld", (long long)K, (long long)kMaxGptqK);
  if (!(damp >= 0.0 && damp <= 1.0)) return fail(FQ_ERR_UNSUPPORTED, "damp=%g outside [0, 1]", damp);
  if (!G || !U) return fail(FQ_ERR_NULL, "G and U must be non-NULL");
  if (!aligned16(G) || !aligned16(U)) return fail(FQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  const size_t need = fq_gptq_factor_workspace_bytes(K);
  if (!ws || ws_bytes < need)
    return fail(FQ_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws ? ws_bytes : (size_t)0);
  if (!aligned16(ws)) return fail(FQ_ERR_ALIGN, "workspace must be 16-byte aligned");
  if (outputs_alias({span(U, (size_t)K * K * 8), span(ws, need)}, {span(G, (size_t)K * K * 8)}))
    return fail(FQ_ERR_ALIAS, "U and the workspace must not overlap each other or G");
  hipError_t e = fq::launch_gptq_factor(G, (int)K, damp, U, ws, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "gptq_factor launch");
  return ok();
}

size_t fq_gptq_sweep_workspace_bytes(int64_t N, int64_t K) {
  if (N <= 0 || K < 128 || K > kMaxK) return 0;
  return fq::gptq_sweep_ws_bytes(N, (int)K);
}

fq_status fq_gptq_sweep(const float *w_t, int64_t ldw, const double *U, int64_t N, int64_t K, int b, int bits,
                        int8_t *w_codes, float *w_scale, void *ws, size_t ws_bytes, void *stream) {
  fq_status s;
  if (N < 0) return fail(FQ_ERR_SHAPE, "N=%lld < 0", (long long)N);
  if ((s = check_k(K)) != FQ_OK) return s;
  if ((s = check_bits(bits)) != FQ_OK) return s;
  if ((s = check_block(b, K)) != FQ_OK) return s;
  if (ldw < K) return fail(FQ_ERR_SHAPE, "ldw=%lld < K=%lld", (long long)ldw, (long long)K);
  if (N > (1ll << 24)) return fail(FQ_ERR_UNSUPPORTED, "N=%lld too large", (long long)N);
  if (N == 0) return ok();
  if (!w_t || !U || !w_codes || !w_scale) return fail(FQ_ERR_NULL, "w_t, U, w_codes and w_scale must be non-NULL");
  if (!aligned16(w_t) || !aligned16(U) || !aligned16(w_codes) || !aligned16(w_scale))
    return fail(FQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  const size_t need = fq_gptq_sweep_workspace_bytes(N, K);
  if (!ws || ws_bytes < need)
    return fail(FQ_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws ? ws_bytes : (size_t)0);
  if (!aligned16(ws)) return fail(FQ_ERR_ALIGN, "workspace must be 16-byte aligned");
  if (outputs_alias({span(w_codes, (size_t)N * K), span(w_scale, (size_t)N * 4), span(ws, need)},
                    {span(w_t, rows_span(N, ldw * 4, K * 4)), span(U, (size_t)K * K * 8)}))
    return fail(FQ_ERR_ALIAS, "codes, scales and the workspace must not overlap each other or an input");
  // the block Hadamard's normalization, deferred to the scale as in the prologue
  hipError_t e = fq::launch_gptq_sweep(w_t, ldw, U, N, (int)K, bits, inv_sqrt_pow2(b), w_codes, w_scale, ws,
                                       static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "gptq_sweep launch");
  return ok();
}

}  // extern "C"
