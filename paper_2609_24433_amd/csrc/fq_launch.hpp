// Host-side launchers of the gfx950 kernels (internal to libfq; not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <atomic>

namespace fq {

// A kernel launched with more than 64 KB of dynamic LDS must first raise its limit with
// hipFuncSetAttribute, on every device it runs on.  `done` (one per kernel
// instantiation) records the devices already raised, 64 at most; concurrent first
// launches may both set the attribute, which is harmless.
template <typename Kern>
inline hipError_t allow_dynamic_lds(Kern kern, size_t lds, std::atomic<uint64_t> &done) {
  if (lds <= 65536) return hipSuccess;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  const uint64_t bit = 1ull << dev;
  if (done.load(std::memory_order_acquire) & bit) return hipSuccess;
  e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  done.fetch_or(bit, std::memory_order_release);
  return hipSuccess;
}

// Output layouts of the prologue.
constexpr int kOutNibble = 0;    // canonical signed-INT4: channel 2i low nibble of byte i
constexpr int kOutInt8 = 1;      // canonical int8, one byte per channel
constexpr int kOutNibbleKM = 2;  // the same nibbles k-step major: [K/128][M][64 B]

// Activation operand formats of the GEMM.
constexpr int kANibble = 0;    // canonical nibbles (widened in the kernel)
constexpr int kAInt8 = 1;      // canonical int8 (W8A8)
constexpr int kANibbleKM = 2;  // nibbles k-step major: [K/128][M][64 B] (plan kind 3)

hipError_t launch_fwht_quant(const void *x, bool x_is_f32, int64_t ldx, const float *chan_mult,
                             const float *post_mult, int64_t M, int K, int b, int bits, float clip_ratio, float cb,
                             uint8_t *codes, int64_t ld_codes, float *delta, int out_fmt,
                             hipStream_t s);

// Composite-rotation prologue (permutation + per-block matrices, b <= 128) through the fp32
// workspace z [M, K].
hipError_t launch_rotate_quant(const void *x, bool x_is_f32, int64_t ldx, const int32_t *perm,
                               const float *blocks, const float *chan_mult, const float *post_mult,
                               int64_t M, int K, int b, int bits, float clip_ratio, uint8_t *codes,
                               int64_t ld_codes, float *delta, int out_fmt, float *z, hipStream_t s);

hipError_t launch_pack_weights(const int8_t *codes, int64_t N, int K, int bits, uint8_t *packed,
                               hipStream_t s);
hipError_t launch_unpack_weights(const uint8_t *packed, int64_t N, int K, int bits, int8_t *codes,
                                 hipStream_t s);

// GEMM plan: which kernel, its tiling and its split of K.
struct GemmPlan {
  int kind;     // 0 = streaming (M <= 64), 1 = tiled, 2 = streaming with one K range per wave (long K),
                // 3 = k groups (INT4, a few hundred rows, long K; k-step-major codes)
  int mt;       // streaming: 16-row tiles covering M
  int kt, wk;   // streaming: k steps per wave, wave groups along K per workgroup
  int wc;       // streaming: 16-channel wave columns per workgroup
  int rb;       // streaming: row blocks of 16 mt rows (the grid's z dimension)
  int bm, bn;   // tiled: workgroup tile
  int stages;   // tiled: depth of the LDS load ring
  int loader;   // tiled: 1 = a fifth wave issues the ring loads
  int order;    // tiled: tile order (bit 0: down the rows first; bit 1: no XCD grouping)
  int splits;   // K slices (each slice: ksteps k steps); > 1 adds an epilogue kernel
  int ksteps;   // 128-wide k steps per slice
  int64_t tiles;        // output tiles along the grid's x dimension
  size_t partial_bytes; // split-K INT32 partials [splits][M][N]
};

// kmajor_codes: the caller writes the activation codes k-step major at no extra cost (the
// fused projection's prologue), which widens the k-group plan's range
GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, int bits, bool kmajor_codes = false);
// scratch of the GEMM itself (split-K partials); a kind-3 plan fed canonical codes also
// needs gemm_plan_relayout_bytes for their k-step-major copy
size_t gemm_plan_workspace(const GemmPlan &pl);
size_t gemm_plan_relayout_bytes(const GemmPlan &pl, int64_t M, int64_t K);

// k-group GEMM (fq_gemm_kg.hip), plan kind 3: INT4 codes k-step major (a_fmt kANibbleKM).
struct KgParams {
  const uint8_t *a;  // [K/128][M][64 B]
  const float *delta;
  const uint8_t *w;
  const float *w_scale;
  const float *bias;
  uint16_t *y;
  int64_t ldy;
  int32_t *acc_out;
  int M, N, K;
};
size_t kgroup_lds_bytes();
// a_canonical != NULL: first convert those canonical codes into a_kmajor (M K/2 bytes),
// which p.a must point to.  go = false only resolves the kernel and raises its LDS limit.
hipError_t launch_gemm_kgroup(const KgParams &p, const uint8_t *a_canonical, uint8_t *a_kmajor, hipStream_t s,
                              bool go);

struct GemmArgs {
  const uint8_t *a;
  int64_t lda;  // bytes per activation row
  int a_fmt;
  const float *delta;
  const uint8_t *w;
  const float *w_scale;
  const float *bias;
  uint16_t *y;
  int64_t ldy;
  int32_t *acc_out;
  int64_t M, N, K;
  int bits;
};

// ws: at least gemm_plan_workspace(pl) bytes of scratch (no initialization needed).
// go = false launches nothing: it only resolves the plan's kernel and raises its LDS
// limit, returning an error when the plan has no kernel.
hipError_t launch_gemm(const GemmArgs &g, const GemmPlan &pl, void *ws, hipStream_t s, bool go = true);

// The fused projection for few tokens (fq_small.hip): one kernel per call, each workgroup
// quantizing its own r rows and multiplying them against 64 ncw output channels.
struct SmallPlan {
  bool ok;          // false: the shape is outside what the fused kernel handles
  int r, cpt, ncw;  // rows per workgroup, 16-channel chunks per prologue thread, 64-channel groups per workgroup / 64
  int rb, groups;   // grid: output-channel groups x row blocks
};
struct SmallArgs {
  const void *x;  // bf16 [M, ldx]
  int64_t ldx;
  const float *chan_mult, *post_mult;
  const uint8_t *w;
  const float *w_scale, *bias;
  uint16_t *y;
  int64_t ldy;
  int64_t M, N, K;
  int log2b, bits;
  float clip_ratio, cb;
};
SmallPlan plan_small(int64_t M, int64_t N, int64_t K, int bits);
// go = false resolves the kernel and raises its LDS limit without launching.
hipError_t launch_linear_small(const SmallArgs &a, const SmallPlan &pl, hipStream_t s, bool go = true);

// Weight-only INT4 (bf16 activations) projection.
struct W16Plan {
  int mt, kt;           // 16-row tiles per workgroup, k steps per wave group (4 groups)
  bool one;             // a single token: only its row is staged, and K up to 16384 needs no split
  int splits, rb;       // K slices, row blocks
  int64_t tiles;        // 16-channel weight tiles
  size_t partial_bytes; // fp32 partials [splits][M][N] when K is split
};
struct W16Args {
  const void *x;        // bf16 [M, ldx]
  int64_t ldx;
  const uint8_t *w;
  const float *w_scale;
  const float *bias;
  uint16_t *y;
  int64_t ldy;
  float *acc_out;
  int64_t M, N, K;
};
W16Plan plan_w4a16(int64_t M, int64_t N, int64_t K);
hipError_t launch_w4a16(const W16Args &g, const W16Plan &pl, void *ws, hipStream_t s);

// GPTQ in the transformed coordinates (fq_gptq.hip)
hipError_t launch_transform(const void *x, bool x_is_f32, int64_t ldx, const float *pre, const float *post,
                            int64_t M, int K, int b, float *z, hipStream_t s);
hipError_t launch_gptq_hessian(const float *z, int64_t ldz, int64_t T, int K, double *G, bool accumulate,
                               hipStream_t s);
size_t gptq_factor_ws_bytes(int K);
hipError_t launch_gptq_factor(const double *G, int K, double damp, double *U, void *ws, hipStream_t s);
size_t gptq_sweep_ws_bytes(int64_t N, int K);
hipError_t launch_gptq_sweep(const float *w, int64_t ldw, const double *U, int64_t N, int K, int bits,
                             float scale_mult, int8_t *codes, float *scales, void *ws, hipStream_t s);

}  // namespace fq
