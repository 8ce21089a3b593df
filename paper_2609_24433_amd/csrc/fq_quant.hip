// Runtime prologue of the quantized projection (Sec. III-C transform, eq. (5) quantizer):
// per token row, blockwise Sylvester FWHT in fp32, row absmax, symmetric round-to-nearest
// quantization and packing.  The same kernel rounds offline weight rows (r = 1).
//
// Work layout: a row of K channels is split into 16-channel chunks.  A workgroup of NT
// threads holds RPW = NT / TPR rows (one row of K / 32 threads for K >= 8192, else rows of
// K / 16 threads in 256-thread workgroups); thread tau of a row owns chunks
// c*TPR + chunk_lane(tau), so a wave's lanes hold consecutive chunks.
//   loads: every chunk of the thread is requested up front (coalesced 16-byte loads);
//   stages h = 1..8: the optional per-channel multiplier, then the butterfly inside each
//           chunk, in registers;
//   stages h = 16..b/2: lane exchanges (a b-block spans b/16 <= 16 lanes of one wave),
//           no LDS; an upper lane keeps the negated difference (lane_stage), undone by the
//           sign it multiplies into 1 / (r A);
//   the row absmax is reduced over the row's lanes (DPP / swizzle) and waves (LDS), and
//   each thread quantizes, packs and stores its chunks in natural channel order (nibbles
//   through a biased bit pattern that packs without masks; no clamp when r = 1).
// Every stage is the pair update (a, c) -> (a + c, a - c) in fp32 in ascending h, so the
// result does not depend on where the data lives; no multiply-add is contracted.
#include "fq_codes.hpp"
#include "fq_device.hpp"
#include "fq_launch.hpp"

namespace fq {

struct QuantParams {
  const void *x;
  int64_t ldx;  // elements
  const float *chan_mult;  // fold-before S^-1, before the rotation (or NULL)
  const float *post_mult;  // fold-after P^-1, after the rotation (or NULL)
  int64_t M;
  int K;
  int bits;
  float clip_ratio;
  float cb;  // float nearest 1/sqrt(b)
  uint8_t *codes;
  int64_t ld_codes;  // bytes per output row (64 for k-step-major nibbles)
  int64_t kstride;   // nibbles: bytes between the 128-channel k steps of a row (64 canonical)
  float *delta;
  int out_fmt;
  int tpr_log2;
};

// In-place butterfly over n consecutive register values, stages h = 1 .. hmax/2.
template <int N, int HMAX>
__device__ __forceinline__ void butterfly(float (&v)[N]) {
#pragma unroll
  for (int h = 1; h < HMAX; h *= 2) {
#pragma unroll
    for (int i = 0; i < N; i += 2 * h) {
#pragma unroll
      for (int j = i; j < i + h; ++j) {
        float a = v[j], c = v[j + h];
        v[j] = a + c;
        v[j + h] = a - c;
      }
    }
  }
}

// Position of thread tau's chunks inside the row: bits 2 and 3 of tau swapped (tau is a
// multiple-of-16 range, so the swap stays inside the row's lanes).  Chunk index bit 2 (the
// stage h = 64) then lies on lane bit 3, whose exchange is a DPP row rotation by 8, and the
// LDS-crossbar swizzle (lane xor 4) is left to the stage h = 128 of b = 256 only.  A wave
// still loads and stores the same 64 consecutive chunks, so every access stays coalesced.
__device__ __forceinline__ int chunk_lane(int tau) {
  return (tau & ~12) | ((tau & 4) << 1) | ((tau & 8) >> 1);
}

// NT threads per workgroup; a row is handled by TPR = 2^tpr_log2 >= 16 consecutive
// threads, thread tau owning CPT chunks (chunk c * TPR + chunk_lane(tau)).  CLAMP: the
// clip ratio is below 1, so |u * inv| can exceed q + 1/2 and codes saturate.  OUT: nibble
// or int8 codes.  MULT: a fold multiplier is given (chan_mult or post_mult, either may still
// be NULL).  Fixing these at compile time leaves the common path without branches.
template <typename Tin, int LOG2B, int CPT, int NT, bool CLAMP, int OUT, bool MULT>
__global__ __launch_bounds__(NT) void fwht_quant_kernel(QuantParams p) {
  constexpr int B = 1 << LOG2B;
  constexpr int B1 = B < 16 ? B : 16;              // stages done inside a chunk
  constexpr int NWAVES = NT / kWave;
  // lane masks of the stages h = 16, 32, 64, 128 (chunk index bits 0, 1, 2, 3; see chunk_lane)
  constexpr int SMASK = (B >= 32 ? 1 : 0) | (B >= 64 ? 2 : 0) | (B >= 128 ? 8 : 0) | (B >= 256 ? 4 : 0);
  __shared__ float red[NWAVES];

  const int tid = threadIdx.x;
  const int TPR = 1 << p.tpr_log2;
  const int RPW = NT >> p.tpr_log2;
  const int row_local = tid >> p.tpr_log2;
  const int tau = tid & (TPR - 1);
  const int lam = chunk_lane(tau);
  const int64_t row = (int64_t)blockIdx.x * RPW + row_local;
  const bool row_ok = row < p.M;
  const int64_t row_c = row_ok ? row : p.M - 1;  // loads of rows past M read row M - 1
  const int K = p.K;
  const int nchunks = K >> 4;
  const int q = (1 << (p.bits - 1)) - 1;
  const float qf = (float)q;

  // ---- all loads first (branch-free: out-of-range chunks read chunk 0) ----------------
  // (the optional multipliers are read where they are applied: kept in registers from
  // here, they would cost 32 VGPRs per chunk whether used or not)
  Chunk<Tin> raw[CPT];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int j = c * TPR + lam;
    const int jc = j < nchunks ? j : 0;
    load_chunk<Tin>(p.x, row_c * p.ldx + (int64_t)jc * 16, raw[c]);
  }

  // ---- pass 1: optional multiplier, stages h < 16 in registers -------------------------
  float v1[CPT][16];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    unpack_chunk<Tin>(raw[c], v1[c]);
    if (MULT && p.chan_mult) {
      const int j = c * TPR + lam;
      const float4 *m4 = reinterpret_cast<const float4 *>(p.chan_mult + (j < nchunks ? j : 0) * 16);
      float4 cm[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) cm[i] = m4[i];
      mul_chunk(v1[c], cm);
    }
    butterfly<16, B1>(v1[c]);
  }

  // ---- stages h = 16 .. b/2: a b-block is b/16 chunks held by lanes of one 16-lane row
  // (TPR >= 16), so every stage is a lane exchange, no LDS round trip ----
  if constexpr (B >= 32) lane_stage<1, CPT>(v1, tau);
  if constexpr (B >= 64) lane_stage<2, CPT>(v1, tau);
  if constexpr (B >= 128) lane_stage<8, CPT>(v1, tau);
  if constexpr (B >= 256) lane_stage<4, CPT>(v1, tau);

  // ---- optional fold-after multiplier (Sec. III-C), one fp32 rounding per element -------
  if (MULT && p.post_mult) {
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int j = c * TPR + lam;
      const float4 *m4 = reinterpret_cast<const float4 *>(p.post_mult + (j < nchunks ? j : 0) * 16);
      float4 pm[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) pm[i] = m4[i];
      mul_chunk(v1[c], pm);
    }
  }

  // ---- row absmax: own chunks, then the row's lanes, then the row's waves ---------------
  float amax = 0.0f;
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int j = c * TPR + lam;
    if (j < nchunks) {
#pragma unroll
      for (int i = 0; i < 16; ++i) amax = fmaxf(amax, fabsf(v1[c][i]));
    }
  }
  {
    const int lim = TPR < kWave ? TPR : kWave;
    amax = fmaxf(amax, lane_xor<1>(amax));
    amax = fmaxf(amax, lane_xor<2>(amax));
    amax = fmaxf(amax, lane_xor<4>(amax));
    amax = fmaxf(amax, lane_xor<8>(amax));
    if (lim > 16) amax = fmaxf(amax, lane_xor<16>(amax));
    if (lim > 32) amax = fmaxf(amax, __shfl_xor(amax, 32, kWave));
    if (TPR > kWave) {
      if ((tid & (kWave - 1)) == 0) red[tid / kWave] = amax;
      __syncthreads();
      const int w0 = (row_local * TPR) / kWave;
      amax = red[w0];
      for (int w = 1; w < TPR / kWave; ++w) amax = fmaxf(amax, red[w0 + w]);
    }
  }

  const bool zero = !(amax > 0.0f);
  const float rA = p.clip_ratio * amax;
  const float inv = zero ? 0.0f : qf / rA;
  if (row_ok && tau == 0) p.delta[row] = zero ? 0.0f : (rA * p.cb) / qf;
  // the lane stages leave this lane's values multiplied by sgn (lane_stage); sgn * inv
  // gives the same products as inv on the true values
  const float sgn = (__builtin_popcount(tau & SMASK) & 1) ? -1.0f : 1.0f;
  const float inv_l = inv * sgn;

  // ---- quantize and pack in natural channel order ------------------------------------
  // Without the clamp the bound |u * inv| < q + 1/2 needs a finite inv (a row absmax below
  // q / FLT_MAX lies outside the supported range; such a row keeps the clamp).
  if (row_ok) {
    uint8_t *row_out = p.codes + row * p.ld_codes;
    const float lim = qf + 0.49f;
    const bool clamp = CLAMP || !__builtin_isfinite(inv);
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int j = c * TPR + lam;
      if (j < nchunks) {
        if constexpr (OUT == kOutNibble) {
          uint32_t cc[16];
          if (clamp) {
#pragma unroll
            for (int i = 0; i < 16; ++i) cc[i] = quantize_bits_biased<true>(v1[c][i], inv_l, lim);
          } else {
#pragma unroll
            for (int i = 0; i < 16; ++i) cc[i] = quantize_bits_biased<false>(v1[c][i], inv_l, lim);
          }
          *reinterpret_cast<uint2 *>(row_out + (int64_t)(j >> 3) * p.kstride + (j & 7) * 8) =
              pack_chunk_nibbles_biased(cc);
        } else {
          int cc[16];
          if (clamp) {
#pragma unroll
            for (int i = 0; i < 16; ++i) cc[i] = quantize_bits(v1[c][i], inv_l, lim);
          } else {
#pragma unroll
            for (int i = 0; i < 16; ++i) cc[i] = __float_as_int(v1[c][i] * inv_l + 12582912.0f);
          }
          *reinterpret_cast<uint4 *>(row_out + (int64_t)j * 16) = pack_chunk_int8(cc);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------------------

// Threads per row and chunks per thread: two 16-channel chunks per thread once a row has
// 512 chunks or more (K >= 8192: one row per workgroup of K / 32 threads, at most 1024),
// one chunk per thread below that (rows of at most 256 chunks share 256-thread
// workgroups).  Measured at K = 16384 against four chunks per 256-thread row: M = 816
// 7.6 against 8.3 us, M = 4096 26.6 against 27.4 us (b = 128); at K 1024 .. 4096 one chunk
// per thread stays ahead.  Every row has at least 16 threads (chunk_lane).
struct QuantShape {
  int nt, cpt, tpr_log2;
};

static QuantShape quant_shape(int K) {
  const int nchunks = K / 16;
  int tpr = 16;
  while (tpr < nchunks) tpr *= 2;
  QuantShape q;
  q.cpt = 1;
  if (tpr >= 512) {
    tpr /= 2;
    q.cpt = 2;
  }
  q.nt = tpr > 256 ? tpr : 256;
  q.tpr_log2 = 0;
  while ((1 << q.tpr_log2) < tpr) ++q.tpr_log2;
  return q;
}

template <typename Tin, int LOG2B, int CPT, int NT, bool CLAMP, int OUT, bool MULT>
static hipError_t launch_one(const QuantParams &p, int grid, hipStream_t s) {
  hipLaunchKernelGGL((fwht_quant_kernel<Tin, LOG2B, CPT, NT, CLAMP, OUT, MULT>), dim3(grid), dim3(NT), 0, s, p);
  return hipGetLastError();
}

template <typename Tin, int LOG2B, bool CLAMP, int OUT, bool MULT>
static hipError_t launch_c(const QuantParams &p, const QuantShape &q, int grid, hipStream_t s) {
  if (q.nt == 256 && q.cpt == 1) return launch_one<Tin, LOG2B, 1, 256, CLAMP, OUT, MULT>(p, grid, s);
  if (q.nt == 256 && q.cpt == 2) return launch_one<Tin, LOG2B, 2, 256, CLAMP, OUT, MULT>(p, grid, s);
  if (q.nt == 512 && q.cpt == 2) return launch_one<Tin, LOG2B, 2, 512, CLAMP, OUT, MULT>(p, grid, s);
  if (q.nt == 1024 && q.cpt == 2) return launch_one<Tin, LOG2B, 2, 1024, CLAMP, OUT, MULT>(p, grid, s);
  return hipErrorInvalidValue;
}

template <typename Tin, int LOG2B, bool CLAMP, int OUT>
static hipError_t launch_m(const QuantParams &p, const QuantShape &q, int grid, hipStream_t s) {
  return (p.chan_mult || p.post_mult) ? launch_c<Tin, LOG2B, CLAMP, OUT, true>(p, q, grid, s)
                                      : launch_c<Tin, LOG2B, CLAMP, OUT, false>(p, q, grid, s);
}

// bf16 activations: every clip ratio and code width; fp32 rows are the offline weights
// (r = 1, int8 codes) only.
template <typename Tin, int LOG2B>
static hipError_t launch_b(const QuantParams &p, const QuantShape &q, int grid, hipStream_t s) {
  const bool clamp = p.clip_ratio != 1.0f;
  if constexpr (sizeof(Tin) == 4) {
    if (clamp || p.out_fmt != kOutInt8) return hipErrorInvalidValue;
    return launch_m<Tin, LOG2B, false, kOutInt8>(p, q, grid, s);
  } else {
    if (p.out_fmt == kOutNibble)
      return clamp ? launch_m<Tin, LOG2B, true, kOutNibble>(p, q, grid, s)
                   : launch_m<Tin, LOG2B, false, kOutNibble>(p, q, grid, s);
    return clamp ? launch_m<Tin, LOG2B, true, kOutInt8>(p, q, grid, s)
                 : launch_m<Tin, LOG2B, false, kOutInt8>(p, q, grid, s);
  }
}

template <typename Tin>
static hipError_t launch_t(const QuantParams &p, int log2b, const QuantShape &q, int grid, hipStream_t s) {
  switch (log2b) {
    case 0: return launch_b<Tin, 0>(p, q, grid, s);
    case 1: return launch_b<Tin, 1>(p, q, grid, s);
    case 2: return launch_b<Tin, 2>(p, q, grid, s);
    case 3: return launch_b<Tin, 3>(p, q, grid, s);
    case 4: return launch_b<Tin, 4>(p, q, grid, s);
    case 5: return launch_b<Tin, 5>(p, q, grid, s);
    case 6: return launch_b<Tin, 6>(p, q, grid, s);
    case 7: return launch_b<Tin, 7>(p, q, grid, s);
    case 8: return launch_b<Tin, 8>(p, q, grid, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_fwht_quant(const void *x, bool x_is_f32, int64_t ldx, const float *chan_mult,
                             const float *post_mult, int64_t M, int K, int b, int bits, float clip_ratio, float cb,
                             uint8_t *codes, int64_t ld_codes, float *delta, int out_fmt,
                             hipStream_t s) {
  if (M <= 0) return hipSuccess;
  const QuantShape q = quant_shape(K);
  const int rpw = q.nt >> q.tpr_log2;
  int log2b = 0;
  while ((1 << log2b) < b) ++log2b;
  if ((16 << q.tpr_log2) < b) return hipErrorInvalidValue;  // a block must lie in one wave's lanes
  const int64_t grid64 = (M + rpw - 1) / rpw;
  if (grid64 > 0x7FFFFFFF) return hipErrorInvalidValue;
  QuantParams p;
  p.x = x;
  p.ldx = ldx;
  p.chan_mult = chan_mult;
  p.post_mult = post_mult;
  p.M = M;
  p.K = K;
  p.bits = bits;
  p.clip_ratio = clip_ratio;
  p.cb = cb;
  p.codes = codes;
  p.ld_codes = ld_codes;
  p.kstride = 64;
  p.delta = delta;
  p.out_fmt = out_fmt;
  if (out_fmt == kOutNibbleKM) {  // row r, k step ks at ks * 64 M + 64 r
    p.out_fmt = kOutNibble;
    p.ld_codes = 64;
    p.kstride = 64 * M;
  }
  p.tpr_log2 = q.tpr_log2;
  return x_is_f32 ? launch_t<float>(p, log2b, q, (int)grid64, s)
                  : launch_t<uint16_t>(p, log2b, q, (int)grid64, s);
}

}  // namespace fq
