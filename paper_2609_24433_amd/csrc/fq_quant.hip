// Runtime prologue of the quantized projection (Sec. III-C transform, eq. (5) quantizer):
// per token row, blockwise Sylvester FWHT in fp32, row absmax, symmetric round-to-nearest
// quantization and packing.  The same kernel rounds offline weight rows (r = 1).
//
// Work layout: a row of K channels is split into 16-channel chunks.  A workgroup of NT
// threads (256, or 1024 when there are few rows) holds RPW = NT / TPR rows; thread tau
// of a row owns chunks c*TPR + tau, so consecutive chunks sit in consecutive lanes.
//   loads: every chunk of the thread is requested up front (coalesced 16-byte loads);
//   stages h = 1..8: the optional per-channel multiplier, then the butterfly inside each
//           chunk, in registers;
//   stages h = 16..b/2: lane exchanges (a b-block spans b/16 <= 16 lanes of one wave),
//           no LDS; an upper lane keeps the negated difference (lane_stage), undone by the
//           sign it multiplies into 1 / (r A);
//   the row absmax is reduced over the row's lanes (DPP / swizzle) and waves (LDS), and
//   each thread quantizes, packs and stores its chunks in natural channel order.
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
  int64_t ld_codes;  // bytes per output row
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

// NT threads per workgroup; a row is handled by TPR = 2^tpr_log2 consecutive threads,
// each owning CPT chunks (chunk c * TPR + tau).
template <typename Tin, int LOG2B, int CPT, int NT>
__global__ __launch_bounds__(NT) void fwht_quant_kernel(QuantParams p) {
  constexpr int B = 1 << LOG2B;
  constexpr int B1 = B < 16 ? B : 16;              // stages done inside a chunk
  constexpr int NWAVES = NT / kWave;
  __shared__ float red[NWAVES];

  const int tid = threadIdx.x;
  const int TPR = 1 << p.tpr_log2;
  const int RPW = NT >> p.tpr_log2;
  const int row_local = tid >> p.tpr_log2;
  const int tau = tid & (TPR - 1);
  const int64_t row = (int64_t)blockIdx.x * RPW + row_local;
  const bool row_ok = row < p.M;
  const int64_t row_c = row_ok ? row : p.M - 1;  // loads of rows past M read row M - 1
  const int K = p.K;
  const int nchunks = K >> 4;
  const int q = (1 << (p.bits - 1)) - 1;
  const float qf = (float)q;

  // ---- all loads first (branch-free: out-of-range chunks read chunk 0) ----------------
  // (the optional multipliers are read where they are applied: kept in registers from
  // here, they would cost 32 VGPRs per chunk whether used or not, and with them the kernel
  // holds half the waves per SIMD)
  Chunk<Tin> raw[CPT];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int j = c * TPR + tau;
    const int jc = j < nchunks ? j : 0;
    load_chunk<Tin>(p.x, row_c * p.ldx + (int64_t)jc * 16, raw[c]);
  }

  // ---- pass 1: optional multiplier, stages h < 16 in registers -------------------------
  float v1[CPT][16];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    unpack_chunk<Tin>(raw[c], v1[c]);
    if (p.chan_mult) {
      const int j = c * TPR + tau;
      const float4 *m4 = reinterpret_cast<const float4 *>(p.chan_mult + (j < nchunks ? j : 0) * 16);
      float4 cm[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) cm[i] = m4[i];
      mul_chunk(v1[c], cm);
    }
    butterfly<16, B1>(v1[c]);
  }

  // ---- stages h = 16 .. b/2: a b-block is b/16 consecutive chunks, held by consecutive
  // lanes of one wave (TPR >= b/16 and a multiple of it), so the partner of chunk j in
  // stage h is lane ^ (h/16) and every stage is a lane exchange, no LDS round trip ----
  if constexpr (B >= 32) lane_stage<1, CPT>(v1, tau);
  if constexpr (B >= 64) lane_stage<2, CPT>(v1, tau);
  if constexpr (B >= 128) lane_stage<4, CPT>(v1, tau);
  if constexpr (B >= 256) lane_stage<8, CPT>(v1, tau);

  // ---- optional fold-after multiplier (Sec. III-C), one fp32 rounding per element -------
  if (p.post_mult) {
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int j = c * TPR + tau;
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
    const int j = c * TPR + tau;
    if (j < nchunks) {
#pragma unroll
      for (int i = 0; i < 16; ++i) amax = fmaxf(amax, fabsf(v1[c][i]));
    }
  }
  {
    const int lim = TPR < kWave ? TPR : kWave;
    if (lim > 1) amax = fmaxf(amax, lane_xor<1>(amax));
    if (lim > 2) amax = fmaxf(amax, lane_xor<2>(amax));
    if (lim > 4) amax = fmaxf(amax, lane_xor<4>(amax));
    if (lim > 8) amax = fmaxf(amax, lane_xor<8>(amax));
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
  const float sgn = B >= 32 ? ((__builtin_popcount(tau & (B / 16 - 1)) & 1) ? -1.0f : 1.0f) : 1.0f;
  const float inv_l = inv * sgn;

  // ---- quantize and pack in natural channel order ------------------------------------
  if (row_ok) {
    uint8_t *row_out = p.codes + row * p.ld_codes;
    const float lim = qf + 0.49f;
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int j = c * TPR + tau;
      if (j < nchunks) {
        int cc[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) cc[i] = quantize_bits(v1[c][i], inv_l, lim);
        store_chunk_bits(row_out, j, cc, p.out_fmt);
      }
    }
  }
}

// ---------------------------------------------------------------------------------------

// Threads per workgroup and chunks per thread: wide workgroups (1024 threads, one chunk
// per thread) when there are few rows, so a long row is spread over more threads;
// 256-thread workgroups otherwise.
struct QuantShape {
  int nt, cpt, tpr_log2;
};

static QuantShape quant_shape(int64_t M, int K) {
  const int nchunks = K / 16;
  QuantShape q;
  q.nt = (M < 256 && nchunks > 256) ? 1024 : 256;
  q.cpt = 1;
  while (nchunks > q.nt * q.cpt) q.cpt *= 2;
  int tpr = 8;
  while (tpr < q.nt && tpr * q.cpt < nchunks) tpr *= 2;
  q.tpr_log2 = 0;
  while ((1 << q.tpr_log2) < tpr) ++q.tpr_log2;
  return q;
}

template <typename Tin, int LOG2B, int CPT, int NT>
static hipError_t launch_one(const QuantParams &p, size_t smem, int grid, hipStream_t s) {
  static std::atomic<uint64_t> attr{0};
  hipError_t e = allow_dynamic_lds(&fwht_quant_kernel<Tin, LOG2B, CPT, NT>, smem, attr);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((fwht_quant_kernel<Tin, LOG2B, CPT, NT>), dim3(grid), dim3(NT), smem, s, p);
  return hipGetLastError();
}

template <typename Tin, int LOG2B>
static hipError_t launch_b(const QuantParams &p, const QuantShape &q, size_t smem, int grid,
                           hipStream_t s) {
  if (q.nt == 1024) {
    switch (q.cpt) {
      case 1: return launch_one<Tin, LOG2B, 1, 1024>(p, smem, grid, s);
      case 2: return launch_one<Tin, LOG2B, 2, 1024>(p, smem, grid, s);
      default: return hipErrorInvalidValue;
    }
  }
  switch (q.cpt) {
    case 1: return launch_one<Tin, LOG2B, 1, 256>(p, smem, grid, s);
    case 2: return launch_one<Tin, LOG2B, 2, 256>(p, smem, grid, s);
    case 4: return launch_one<Tin, LOG2B, 4, 256>(p, smem, grid, s);
    case 8: return launch_one<Tin, LOG2B, 8, 256>(p, smem, grid, s);
    default: return hipErrorInvalidValue;
  }
}

template <typename Tin>
static hipError_t launch_t(const QuantParams &p, int log2b, const QuantShape &q, size_t smem, int grid,
                           hipStream_t s) {
  switch (log2b) {
    case 0: return launch_b<Tin, 0>(p, q, smem, grid, s);
    case 1: return launch_b<Tin, 1>(p, q, smem, grid, s);
    case 2: return launch_b<Tin, 2>(p, q, smem, grid, s);
    case 3: return launch_b<Tin, 3>(p, q, smem, grid, s);
    case 4: return launch_b<Tin, 4>(p, q, smem, grid, s);
    case 5: return launch_b<Tin, 5>(p, q, smem, grid, s);
    case 6: return launch_b<Tin, 6>(p, q, smem, grid, s);
    case 7: return launch_b<Tin, 7>(p, q, smem, grid, s);
    case 8: return launch_b<Tin, 8>(p, q, smem, grid, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_fwht_quant(const void *x, bool x_is_f32, int64_t ldx, const float *chan_mult,
                             const float *post_mult, int64_t M, int K, int b, int bits, float clip_ratio, float cb,
                             uint8_t *codes, int64_t ld_codes, float *delta, int out_fmt,
                             hipStream_t s) {
  if (M <= 0) return hipSuccess;
  const QuantShape q = quant_shape(M, K);
  const int rpw = q.nt >> q.tpr_log2;
  int log2b = 0;
  while ((1 << log2b) < b) ++log2b;
  const size_t smem = 0;
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
  p.delta = delta;
  p.out_fmt = out_fmt;
  p.tpr_log2 = q.tpr_log2;
  return x_is_f32 ? launch_t<float>(p, log2b, q, smem, (int)grid64, s)
                  : launch_t<uint16_t>(p, log2b, q, smem, (int)grid64, s);
}

}  // namespace fq
