// Runtime prologue of the quantized projection (Sec. III-C transform, eq. (5) quantizer):
// per token row, blockwise Sylvester FWHT in fp32, row absmax, symmetric round-to-nearest
// quantization and packing.  The same kernel rounds offline weight rows (r = 1).
//
// Work layout: a row of K channels is split into 16-channel chunks.  A workgroup of 256
// threads holds RPW = 256 / TPR rows; thread tau of a row owns chunks c*TPR + tau.
//   pass 1: each thread loads its chunks (coalesced 16-byte loads), applies the optional
//           per-channel multiplier and the butterfly stages h = 1..8 in registers;
//   pass 2 (b > 16): the row goes through LDS once; each thread then holds whole
//           "columns" (channels col + 16*m of one block) and runs stages h = 16..b/2;
//   the row absmax is reduced across the row's threads, codes are formed in registers,
//   and (b > 16) returned to natural order through LDS before packing and storing.
// Every stage is the pair update (a, c) -> (a + c, a - c) in fp32 in ascending h, so the
// result does not depend on where the data lives; no multiply-add is contracted.
#include "fq_device.hpp"
#include "fq_launch.hpp"

namespace fq {

struct QuantParams {
  const void *x;
  int64_t ldx;  // elements
  const float *chan_mult;
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

template <typename Tin>
struct ChunkLoader;

template <>
struct ChunkLoader<uint16_t> {  // bf16 bit patterns
  static __device__ __forceinline__ void load(const void *base, int64_t off, float (&v)[16]) {
    const uint4 *p = reinterpret_cast<const uint4 *>(reinterpret_cast<const uint16_t *>(base) + off);
    uint4 a = p[0], b = p[1];
    uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      v[2 * i] = bf16_lo(w[i]);
      v[2 * i + 1] = bf16_hi(w[i]);
    }
  }
};

template <>
struct ChunkLoader<float> {
  static __device__ __forceinline__ void load(const void *base, int64_t off, float (&v)[16]) {
    const float4 *p = reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(base) + off);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float4 t = p[i];
      v[4 * i] = t.x;
      v[4 * i + 1] = t.y;
      v[4 * i + 2] = t.z;
      v[4 * i + 3] = t.w;
    }
  }
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

__device__ __forceinline__ int quantize1(float u, float inv, float qf) {
  float t = u * inv;
  float k = __builtin_rintf(t);  // round half to even
  k = fminf(fmaxf(k, -qf), qf);
  return (int)k;
}

// Pack 16 codes (natural channel order) and store them for one chunk.
__device__ __forceinline__ void store_chunk(uint8_t *row_out, int chunk, const int (&c)[16],
                                            int out_fmt) {
  if (out_fmt == kOutNibble) {
    uint32_t w0 = 0, w1 = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      uint32_t byte = ((uint32_t)c[2 * i] & 0xFu) | (((uint32_t)c[2 * i + 1] & 0xFu) << 4);
      if (i < 4)
        w0 |= byte << (8 * i);
      else
        w1 |= byte << (8 * (i - 4));
    }
    *reinterpret_cast<uint2 *>(row_out + (int64_t)chunk * 8) = make_uint2(w0, w1);
  } else {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = ((uint32_t)c[4 * i] & 0xFFu) | (((uint32_t)c[4 * i + 1] & 0xFFu) << 8) |
             (((uint32_t)c[4 * i + 2] & 0xFFu) << 16) | (((uint32_t)c[4 * i + 3] & 0xFFu) << 24);
    if (out_fmt == kOutPerm8) {
      // per group of 8 channels: bytes c0 c2 c4 c6 c1 c3 c5 c7 (the order in which the
      // GEMM widens nibble-packed weights)
      uint32_t p0 = __builtin_amdgcn_perm(w[1], w[0], 0x06040200u);
      uint32_t p1 = __builtin_amdgcn_perm(w[1], w[0], 0x07050301u);
      uint32_t p2 = __builtin_amdgcn_perm(w[3], w[2], 0x06040200u);
      uint32_t p3 = __builtin_amdgcn_perm(w[3], w[2], 0x07050301u);
      w[0] = p0;
      w[1] = p1;
      w[2] = p2;
      w[3] = p3;
    }
    *reinterpret_cast<uint4 *>(row_out + (int64_t)chunk * 16) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

template <typename Tin, int LOG2B, int CPT>
__global__ __launch_bounds__(256) void fwht_quant_kernel(QuantParams p) {
  constexpr int B = 1 << LOG2B;
  constexpr int B1 = B < 16 ? B : 16;           // stages done in pass 1
  constexpr int MPU = B > 16 ? B / 16 : 1;      // elements per pass-2 unit
  constexpr int UPT = B > 16 ? 256 * CPT / B : 1;  // pass-2 units per thread
  extern __shared__ float smem[];
  __shared__ float red[4];

  const int tid = threadIdx.x;
  const int TPR = 1 << p.tpr_log2;
  const int RPW = 256 >> p.tpr_log2;
  const int row_local = tid >> p.tpr_log2;
  const int tau = tid & (TPR - 1);
  const int64_t row = (int64_t)blockIdx.x * RPW + row_local;
  const bool row_ok = row < p.M;
  const int K = p.K;
  const int nchunks = K >> 4;
  const int q = (1 << (p.bits - 1)) - 1;
  const float qf = (float)q;

  // ---- pass 1: load, optional multiplier, stages h < 16 ------------------------------
  float v1[CPT][16];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int j = c * TPR + tau;
    if (row_ok && j < nchunks) {
      ChunkLoader<Tin>::load(p.x, row * p.ldx + (int64_t)j * 16, v1[c]);
      if (p.chan_mult) {
        const float4 *m4 = reinterpret_cast<const float4 *>(p.chan_mult + j * 16);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float4 m = m4[i];
          v1[c][4 * i] = v1[c][4 * i] * m.x;
          v1[c][4 * i + 1] = v1[c][4 * i + 1] * m.y;
          v1[c][4 * i + 2] = v1[c][4 * i + 2] * m.z;
          v1[c][4 * i + 3] = v1[c][4 * i + 3] * m.w;
        }
      }
      butterfly<16, B1>(v1[c]);
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) v1[c][i] = 0.0f;
    }
  }

  float amax = 0.0f;
  float v2[UPT][MPU];
  float *srow = smem + (int64_t)row_local * K;
  if constexpr (B > 16) {
    // ---- pass 2: columns through LDS, stages h = 16 .. b/2 ----------------------------
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int j = c * TPR + tau;
      if (j < nchunks) {
        float4 *d = reinterpret_cast<float4 *>(srow + j * 16);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          d[i] = make_float4(v1[c][4 * i], v1[c][4 * i + 1], v1[c][4 * i + 2], v1[c][4 * i + 3]);
      }
    }
    __syncthreads();
    const int nunits = (K / B) * 16;
#pragma unroll
    for (int i = 0; i < UPT; ++i) {
      const int u = i * TPR + tau;
      if (u < nunits) {
        const int base = (u >> 4) * B + (u & 15);
#pragma unroll
        for (int m = 0; m < MPU; ++m) v2[i][m] = srow[base + 16 * m];
        butterfly<MPU, MPU>(v2[i]);
#pragma unroll
        for (int m = 0; m < MPU; ++m) amax = fmaxf(amax, fabsf(v2[i][m]));
      } else {
#pragma unroll
        for (int m = 0; m < MPU; ++m) v2[i][m] = 0.0f;
      }
    }
  } else {
#pragma unroll
    for (int c = 0; c < CPT; ++c)
#pragma unroll
      for (int i = 0; i < 16; ++i) amax = fmaxf(amax, fabsf(v1[c][i]));
  }

  // ---- row absmax across the row's threads -------------------------------------------
  {
    const int lim = TPR < kWave ? TPR : kWave;
    for (int off = lim >> 1; off > 0; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off, kWave));
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

  uint8_t *row_out = p.codes + row * p.ld_codes;
  if constexpr (B > 16) {
    // codes back to natural order through LDS (as bytes), then pack per chunk
    __syncthreads();  // every pass-2 read of srow is done
    int8_t *crow = reinterpret_cast<int8_t *>(smem) + (int64_t)row_local * K;
    const int nunits = (K / B) * 16;
#pragma unroll
    for (int i = 0; i < UPT; ++i) {
      const int u = i * TPR + tau;
      if (u < nunits) {
        const int base = (u >> 4) * B + (u & 15);
#pragma unroll
        for (int m = 0; m < MPU; ++m) crow[base + 16 * m] = (int8_t)(zero ? 0 : quantize1(v2[i][m], inv, qf));
      }
    }
    __syncthreads();
    if (row_ok) {
#pragma unroll
      for (int c = 0; c < CPT; ++c) {
        const int j = c * TPR + tau;
        if (j < nchunks) {
          uint4 raw = *reinterpret_cast<const uint4 *>(crow + j * 16);
          uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
          int cc[16];
#pragma unroll
          for (int i = 0; i < 16; ++i) cc[i] = (int)(int8_t)((w[i >> 2] >> (8 * (i & 3))) & 0xFFu);
          store_chunk(row_out, j, cc, p.out_fmt);
        }
      }
    }
  } else {
    if (row_ok) {
#pragma unroll
      for (int c = 0; c < CPT; ++c) {
        const int j = c * TPR + tau;
        if (j < nchunks) {
          int cc[16];
#pragma unroll
          for (int i = 0; i < 16; ++i) cc[i] = zero ? 0 : quantize1(v1[c][i], inv, qf);
          store_chunk(row_out, j, cc, p.out_fmt);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------------------

static int cpt_for(int K) {
  const int nchunks = K / 16;
  int cpt = 1;
  while (nchunks > 256 * cpt) cpt *= 2;
  return cpt;
}

template <typename Tin, int LOG2B, int CPT>
static void allow_large_lds(size_t smem) {
  // more than 64 KB of dynamic LDS (K > 16384 with b > 16) must be requested explicitly
  if (smem > 65536)
    (void)hipFuncSetAttribute(reinterpret_cast<const void *>(&fwht_quant_kernel<Tin, LOG2B, CPT>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
}

template <typename Tin, int LOG2B>
static hipError_t launch_b(const QuantParams &p, int cpt, size_t smem, int grid, hipStream_t s) {
  if (cpt == 8) allow_large_lds<Tin, LOG2B, 8>(smem);
  switch (cpt) {
    case 1: hipLaunchKernelGGL((fwht_quant_kernel<Tin, LOG2B, 1>), dim3(grid), dim3(256), smem, s, p); break;
    case 2: hipLaunchKernelGGL((fwht_quant_kernel<Tin, LOG2B, 2>), dim3(grid), dim3(256), smem, s, p); break;
    case 4: hipLaunchKernelGGL((fwht_quant_kernel<Tin, LOG2B, 4>), dim3(grid), dim3(256), smem, s, p); break;
    case 8: hipLaunchKernelGGL((fwht_quant_kernel<Tin, LOG2B, 8>), dim3(grid), dim3(256), smem, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename Tin>
static hipError_t launch_t(const QuantParams &p, int log2b, int cpt, size_t smem, int grid,
                           hipStream_t s) {
  switch (log2b) {
    case 0: return launch_b<Tin, 0>(p, cpt, smem, grid, s);
    case 1: return launch_b<Tin, 1>(p, cpt, smem, grid, s);
    case 2: return launch_b<Tin, 2>(p, cpt, smem, grid, s);
    case 3: return launch_b<Tin, 3>(p, cpt, smem, grid, s);
    case 4: return launch_b<Tin, 4>(p, cpt, smem, grid, s);
    case 5: return launch_b<Tin, 5>(p, cpt, smem, grid, s);
    case 6: return launch_b<Tin, 6>(p, cpt, smem, grid, s);
    case 7: return launch_b<Tin, 7>(p, cpt, smem, grid, s);
    case 8: return launch_b<Tin, 8>(p, cpt, smem, grid, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_fwht_quant(const void *x, bool x_is_f32, int64_t ldx, const float *chan_mult,
                             int64_t M, int K, int b, int bits, float clip_ratio, float cb,
                             uint8_t *codes, int64_t ld_codes, float *delta, int out_fmt,
                             hipStream_t s) {
  if (M <= 0) return hipSuccess;
  const int cpt = cpt_for(K);
  int tpr = 8;
  while (tpr < 256 && tpr * cpt * 16 < K) tpr *= 2;
  int tpr_log2 = 0;
  while ((1 << tpr_log2) < tpr) ++tpr_log2;
  const int rpw = 256 / tpr;
  int log2b = 0;
  while ((1 << log2b) < b) ++log2b;
  const size_t smem = b > 16 ? (size_t)rpw * K * sizeof(float) : 0;
  const int64_t grid64 = (M + rpw - 1) / rpw;
  if (grid64 > 0x7FFFFFFF) return hipErrorInvalidValue;
  QuantParams p;
  p.x = x;
  p.ldx = ldx;
  p.chan_mult = chan_mult;
  p.M = M;
  p.K = K;
  p.bits = bits;
  p.clip_ratio = clip_ratio;
  p.cb = cb;
  p.codes = codes;
  p.ld_codes = ld_codes;
  p.delta = delta;
  p.out_fmt = out_fmt;
  p.tpr_log2 = tpr_log2;
  return x_is_f32 ? launch_t<float>(p, log2b, cpt, smem, (int)grid64, s)
                  : launch_t<uint16_t>(p, log2b, cpt, smem, (int)grid64, s);
}

size_t fwht_quant_smem_bytes(int K, int b) {
  const int cpt = cpt_for(K);
  int tpr = 8;
  while (tpr < 256 && tpr * cpt * 16 < K) tpr *= 2;
  return b > 16 ? (size_t)(256 / tpr) * K * sizeof(float) : 0;
}

}  // namespace fq
