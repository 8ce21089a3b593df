// Integer GEMM of the quantized projection with the eq. (8) rescale epilogue, and the
// kernel-native weight packing it reads.
//
// Contraction: acc[t, j] = sum_c qA[t, c] qW[j, c] on the gfx950 INT8 matrix cores
// (v_mfma_i32_16x16x64_i8, INT32 accumulation).  gfx950 has no INT4 matrix instruction,
// so nibble operands are widened in registers to int8 lanes holding 16 * code: one
// shift and two masks per 8 codes.  The scale factor (16 or 256) divides out exactly
// at the end with an arithmetic shift.  The widening interleaves channels
// (0 2 4 6 1 3 5 7 per group of 8); activations and weights go through the same
// interleave, and an integer sum does not depend on its order.
//
// Weight layout (kernel-native, opaque to callers): tiles of 16 output channels x 128
// input channels, tile (nb, kt) at byte offset (nb * K/128 + kt) * tile_bytes; inside a
// tile, lane l of a wave owns channel 16*nb + l%16 and input channels
// 128*kt + 32*(l/16) + [0, 32), stored contiguously at byte l * lane_bytes.  A wave
// therefore fetches a whole tile with one fully coalesced 16/32-byte load per lane.
//
// Two kernels:
//   gemm_stream (M <= 64): the weights are streamed once; each workgroup owns 64 output
//     channels (one 16-channel tile per wave) and one slice of K; activation tiles are
//     shared through LDS; weight tiles go straight from HBM to registers with a
//     several-step prefetch ring.  K slices are combined exactly in INT32 by the last
//     workgroup to finish its output tile.
//   gemm_tile (M > 64): 128 x 128 output tiles, 2 x 2 waves of 64 x 64, both operands
//     double-buffered through LDS, optional split-K with the same exact combination.
#include "fq_device.hpp"
#include "fq_launch.hpp"

#include <cstdlib>
#include <cstring>

namespace fq {

// ----------------------------------------------------------------------------------------
// weight packing

template <int BITS>
__global__ __launch_bounds__(256) void pack_weights_kernel(const int8_t *__restrict__ codes,
                                                           int64_t N, int K,
                                                           uint8_t *__restrict__ packed) {
  const int64_t lane_id = (int64_t)blockIdx.x * 256 + threadIdx.x;  // one lane of one tile
  const int ktiles = K / kTileK;
  const int64_t total = (N / kTileN) * ktiles * kWave;
  if (lane_id >= total) return;
  const int l = (int)(lane_id % kWave);
  const int64_t tile = lane_id / kWave;
  const int64_t nb = tile / ktiles;
  const int kt = (int)(tile % ktiles);
  const int64_t n = nb * kTileN + (l & 15);
  const int k0 = kt * kTileK + 32 * (l >> 4);
  const int8_t *src = codes + n * K + k0;
  uint8_t *dst = packed + tile * tile_bytes(BITS) + l * lane_bytes(BITS);
  const uint4 *s4 = reinterpret_cast<const uint4 *>(src);
  uint4 a = s4[0], b = s4[1];
  if (BITS == 8) {
    reinterpret_cast<uint4 *>(dst)[0] = a;
    reinterpret_cast<uint4 *>(dst)[1] = b;
  } else {
    uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    uint32_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t r = 0;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        uint32_t x = w[2 * i + h];  // 4 codes
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          uint32_t lo = (x >> (16 * k)) & 0xFu;
          uint32_t hi = (x >> (16 * k + 8)) & 0xFu;
          r |= (lo | (hi << 4)) << (8 * (2 * h + k));
        }
      }
      o[i] = r;
    }
    *reinterpret_cast<uint4 *>(dst) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

template <int BITS>
__global__ __launch_bounds__(256) void unpack_weights_kernel(const uint8_t *__restrict__ packed,
                                                             int64_t N, int K,
                                                             int8_t *__restrict__ codes) {
  const int64_t lane_id = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int ktiles = K / kTileK;
  const int64_t total = (N / kTileN) * ktiles * kWave;
  if (lane_id >= total) return;
  const int l = (int)(lane_id % kWave);
  const int64_t tile = lane_id / kWave;
  const int64_t nb = tile / ktiles;
  const int kt = (int)(tile % ktiles);
  const int64_t n = nb * kTileN + (l & 15);
  const int k0 = kt * kTileK + 32 * (l >> 4);
  const uint8_t *src = packed + tile * tile_bytes(BITS) + l * lane_bytes(BITS);
  uint4 *d4 = reinterpret_cast<uint4 *>(codes + n * K + k0);
  if (BITS == 8) {
    d4[0] = reinterpret_cast<const uint4 *>(src)[0];
    d4[1] = reinterpret_cast<const uint4 *>(src)[1];
  } else {
    uint4 s = *reinterpret_cast<const uint4 *>(src);
    uint32_t w[4] = {s.x, s.y, s.z, s.w};
    uint32_t o[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      uint32_t half = (w[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;  // 2 bytes = 4 codes
      uint32_t r = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        int32_t nib = (int32_t)((half >> (4 * k)) & 0xFu);
        nib = (nib ^ 8) - 8;  // sign-extend
        r |= ((uint32_t)nib & 0xFFu) << (8 * k);
      }
      o[i] = r;
    }
    d4[0] = make_uint4(o[0], o[1], o[2], o[3]);
    d4[1] = make_uint4(o[4], o[5], o[6], o[7]);
  }
}

hipError_t launch_pack_weights(const int8_t *codes, int64_t N, int K, int bits, uint8_t *packed,
                               hipStream_t s) {
  const int64_t total = (N / kTileN) * (K / kTileK) * kWave;
  if (total == 0) return hipSuccess;
  const int64_t grid = (total + 255) / 256;
  if (bits == 4)
    hipLaunchKernelGGL(pack_weights_kernel<4>, dim3((unsigned)grid), dim3(256), 0, s, codes, N, K, packed);
  else
    hipLaunchKernelGGL(pack_weights_kernel<8>, dim3((unsigned)grid), dim3(256), 0, s, codes, N, K, packed);
  return hipGetLastError();
}

hipError_t launch_unpack_weights(const uint8_t *packed, int64_t N, int K, int bits, int8_t *codes,
                                 hipStream_t s) {
  const int64_t total = (N / kTileN) * (K / kTileK) * kWave;
  if (total == 0) return hipSuccess;
  const int64_t grid = (total + 255) / 256;
  if (bits == 4)
    hipLaunchKernelGGL(unpack_weights_kernel<4>, dim3((unsigned)grid), dim3(256), 0, s, packed, N, K, codes);
  else
    hipLaunchKernelGGL(unpack_weights_kernel<8>, dim3((unsigned)grid), dim3(256), 0, s, packed, N, K, codes);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------------------
// GEMM

struct GemmParams {
  const uint8_t *a;
  int64_t lda;
  const float *delta;
  const uint8_t *w;
  const float *w_scale;
  const float *bias;
  uint16_t *y;
  int64_t ldy;
  int32_t *acc_out;
  int M, N, K;
  int ksteps;  // k steps of 128 per split
  int32_t *partial;
  uint32_t *counters;
  int red_atomic;  // 1: K slices combine with device atomics into one [M, N] buffer
};

template <int BITS, int AFMT>
struct Fmt {
  static constexpr int arow = AFMT == kANibble ? 64 : 128;  // activation bytes per row per k step
  static constexpr int tb = tile_bytes(BITS);
  static constexpr int lb = lane_bytes(BITS);
  // acc = 2^shift * true sum
  static constexpr int shift = BITS == 8 ? 0 : (AFMT == kANibble ? 8 : 4);
};

// Activation operand of lane (row, g) for k-chunk c from a row of one k step.
template <int AFMT>
__device__ __forceinline__ v4i a_operand(const uint8_t *row, int g, int c) {
  if constexpr (AFMT == kANibble) {
    return widen8(*reinterpret_cast<const v2i *>(row + g * 16 + c * 8));
  } else {
    return *reinterpret_cast<const v4i *>(row + g * 32 + c * 16);
  }
}

// Weight operand of lane l for k-chunk c from one tile.
template <int BITS>
__device__ __forceinline__ v4i w_operand(const uint8_t *tile, int l, int c) {
  if constexpr (BITS == 4) {
    return widen8(*reinterpret_cast<const v2i *>(tile + l * 16 + c * 8));
  } else {
    return *reinterpret_cast<const v4i *>(tile + l * 32 + c * 16);
  }
}

// Eq. (8) epilogue for one 16 x 16 accumulator tile held by a wave: lane l holds rows
// 4*(l/16) + r (r = 0..3) of column l % 16.
template <int SHIFT>
__device__ __forceinline__ void epilogue16(const GemmParams &p, v4i acc, int m_base, int n_base,
                                           int lane) {
  const int n = n_base + (lane & 15);
  if (n >= p.N) return;
  const float sw = p.w_scale[n];
  const float bj = p.bias ? p.bias[n] : 0.0f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int m = m_base + 4 * (lane >> 4) + r;
    if (m < p.M) {
      const int a = acc[r] >> SHIFT;
      if (p.acc_out) p.acc_out[(int64_t)m * p.N + n] = a;
      const float sc = sw * p.delta[m];
      const float yv = (float)a * sc + bj;
      p.y[(int64_t)m * p.ldy + n] = (uint16_t)f32_to_bf16(yv);
    }
  }
}

// Split-K: publish this workgroup's raw partial tile; returns true in the one workgroup
// that arrives last for the output tile, after adding every other slice's partial into
// `acc` (integer addition: exact, order-free).  Partial layout: [split][M][N].
template <int TI, int TJ>
__device__ __forceinline__ bool splitk_combine(const GemmParams &p, v4i (&acc)[TI][TJ],
                                               const int (&m_base)[TI], const int (&n_base)[TJ],
                                               int lane, int split, int nsplit, int tile_id) {
  __shared__ int s_last;
  const int64_t slice = (int64_t)p.M * p.N;
  if (p.red_atomic) {
    // every slice adds into one zeroed [M, N] buffer; the last arrival reads the totals
    // back with exchanges that also re-zero the buffer for the next call
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j) {
        const int n = n_base[j] + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m_base[i] + 4 * (lane >> 4) + r;
          if (m < p.M && n < p.N)
            __hip_atomic_fetch_add(&p.partial[(int64_t)m * p.N + n], acc[i][j][r], __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
      const uint32_t prev = __hip_atomic_fetch_add(&p.counters[tile_id], 1u, __ATOMIC_RELAXED,
                                                   __HIP_MEMORY_SCOPE_AGENT);
      s_last = (prev == (uint32_t)(nsplit - 1));
    }
    __syncthreads();
    if (!s_last) return false;
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j) {
        const int n = n_base[j] + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m_base[i] + 4 * (lane >> 4) + r;
          if (m < p.M && n < p.N)
            acc[i][j][r] = __hip_atomic_exchange(&p.partial[(int64_t)m * p.N + n], 0, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    if (threadIdx.x == 0)
      __hip_atomic_store(&p.counters[tile_id], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return true;
  }
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int n = n_base[j] + (lane & 15);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m_base[i] + 4 * (lane >> 4) + r;
        if (m < p.M && n < p.N) p.partial[split * slice + (int64_t)m * p.N + n] = acc[i][j][r];
      }
    }
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t prev = atomicAdd(&p.counters[tile_id], 1u);
    s_last = (prev == (uint32_t)(nsplit - 1));
  }
  __syncthreads();
  if (!s_last) return false;
  __threadfence();
  for (int z = 0; z < nsplit; ++z) {
    if (z == split) continue;
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j) {
        const int n = n_base[j] + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m_base[i] + 4 * (lane >> 4) + r;
          if (m < p.M && n < p.N)
            acc[i][j][r] += p.partial[z * slice + (int64_t)m * p.N + n];
        }
      }
  }
  if (threadIdx.x == 0) p.counters[tile_id] = 0u;  // ready for the next call
  return true;
}

// ---------------- streaming kernel (M <= 64) ----------------

constexpr int kStreamPF = 4;  // weight k steps in flight per wave

template <int BITS, int AFMT, int MT>
__global__ __launch_bounds__(256) void gemm_stream_kernel(GemmParams p) {
  using F = Fmt<BITS, AFMT>;
  constexpr int AROWP = F::arow + 16;
  constexpr int ASTAGE = MT * 16 * AROWP;
  constexpr int ACHUNKS = MT * 16 * F::arow / 16;
  constexpr int LU4 = F::lb / 16;  // uint4 per lane per weight tile
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * ASTAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int nblk = blockIdx.x;
  const int split = blockIdx.y;
  const int nsplit = gridDim.y;
  const int ktot = p.K / kTileK;
  const int ks_begin = split * p.ksteps;
  const int nk = min(p.ksteps, ktot - ks_begin);
  const int ntile = nblk * 4 + wave;  // this wave's 16-channel tile
  const bool n_ok = ntile * 16 < p.N;

  const uint8_t *wbase = p.w + ((int64_t)ntile * ktot + ks_begin) * F::tb + lane * F::lb;

  // activation tile loader: chunk q -> row q / (arow/16), 16-byte column q % (arow/16)
  uint4 areg[(ACHUNKS + 255) / 256];
  auto load_a = [&](int ks) {
#pragma unroll
    for (int i = 0; i < (ACHUNKS + 255) / 256; ++i) {
      const int q = i * 256 + tid;
      areg[i] = make_uint4(0, 0, 0, 0);
      if (q < ACHUNKS) {
        const int row = q / (F::arow / 16), col = q % (F::arow / 16);
        if (row < p.M)
          areg[i] = *reinterpret_cast<const uint4 *>(p.a + (int64_t)row * p.lda +
                                                     (int64_t)(ks_begin + ks) * F::arow + col * 16);
      }
    }
  };
  auto store_a = [&](int buf) {
#pragma unroll
    for (int i = 0; i < (ACHUNKS + 255) / 256; ++i) {
      const int q = i * 256 + tid;
      if (q < ACHUNKS) {
        const int row = q / (F::arow / 16), col = q % (F::arow / 16);
        *reinterpret_cast<uint4 *>(lds + buf * ASTAGE + row * AROWP + col * 16) = areg[i];
      }
    }
  };

  uint4 wring[kStreamPF][LU4];
#pragma unroll
  for (int s = 0; s < kStreamPF; ++s)
#pragma unroll
    for (int u = 0; u < LU4; ++u)
      wring[s][u] = (n_ok && s < nk) ? reinterpret_cast<const uint4 *>(wbase + (int64_t)s * F::tb)[u]
                                     : make_uint4(0, 0, 0, 0);

  v4i acc[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i] = v4i{0, 0, 0, 0};

  if (nk > 0) {
    load_a(0);
    store_a(0);
  }
  __syncthreads();

  for (int ks0 = 0; ks0 < nk; ks0 += kStreamPF) {
#pragma unroll
    for (int s = 0; s < kStreamPF; ++s) {
      const int ks = ks0 + s;
      if (ks < nk) {
        if (ks + 1 < nk) load_a(ks + 1);
        uint4 wcur[LU4];
#pragma unroll
        for (int u = 0; u < LU4; ++u) wcur[u] = wring[s][u];
        if (n_ok && ks + kStreamPF < nk) {
#pragma unroll
          for (int u = 0; u < LU4; ++u)
            wring[s][u] = reinterpret_cast<const uint4 *>(wbase + (int64_t)(ks + kStreamPF) * F::tb)[u];
        }
        const uint8_t *abuf = lds + (ks & 1) * ASTAGE;
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          v4i bop;
          if constexpr (BITS == 4) {
            v2i h;
            h.x = (int)(c == 0 ? wcur[0].x : wcur[0].z);
            h.y = (int)(c == 0 ? wcur[0].y : wcur[0].w);
            bop = widen8(h);
          } else {
            const uint4 t = wcur[c];
            bop = v4i{(int)t.x, (int)t.y, (int)t.z, (int)t.w};
          }
#pragma unroll
          for (int i = 0; i < MT; ++i) {
            const v4i aop = a_operand<AFMT>(abuf + (i * 16 + (lane & 15)) * AROWP, lane >> 4, c);
            acc[i] = mfma16x16x64(aop, bop, acc[i]);
          }
        }
        if (ks + 1 < nk) store_a((ks + 1) & 1);
        __syncthreads();
      }
    }
  }

  int m_base[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) m_base[i] = i * 16;
  int n_base[1] = {ntile * 16};
  v4i acc2[MT][1];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc2[i][0] = acc[i];
  if (nsplit > 1) {
    if (!splitk_combine<MT, 1>(p, acc2, m_base, n_base, lane, split, nsplit, nblk)) return;
  }
  if (!n_ok) return;
#pragma unroll
  for (int i = 0; i < MT; ++i) epilogue16<F::shift>(p, acc2[i][0], m_base[i], n_base[0], lane);
}

// ---------------- tiled kernel (M > 64) ----------------

template <int BITS, int AFMT, int BM, int BN>
__global__ __launch_bounds__(256) void gemm_tile_kernel(GemmParams p) {
  using F = Fmt<BITS, AFMT>;
  constexpr int AROWP = F::arow + 16;
  constexpr int NT = BN / 16;
  constexpr int ASTAGE = BM * AROWP;
  constexpr int BSTAGE = NT * F::tb;
  constexpr int ACH = BM * F::arow / 16 / 256;  // 16-byte activation chunks per thread
  constexpr int BCH = NT * F::tb / 16 / 256;    // 16-byte weight chunks per thread
  constexpr int TM = BM / 32, TN = NT / 2;      // 16x16 tiles per wave (2 x 2 waves)
  static_assert(ACH >= 1 && BCH >= 1, "tile too small for 256 threads");
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * (ASTAGE + BSTAGE)];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int ntiles_n = (p.N + BN - 1) / BN;
  const int tile_id = blockIdx.x;
  const int tn = tile_id % ntiles_n, tm = tile_id / ntiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const int split = blockIdx.y, nsplit = gridDim.y;
  const int ktot = p.K / kTileK;
  const int ks_begin = split * p.ksteps;
  const int nk = min(p.ksteps, ktot - ks_begin);

  uint4 ar[ACH], br[BCH];
  auto load = [&](int ks) {
    const int kk = ks_begin + ks;
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int q = i * 256 + tid;
      const int row = q / (F::arow / 16), col = q % (F::arow / 16);
      ar[i] = (m0 + row < p.M)
                  ? *reinterpret_cast<const uint4 *>(p.a + (int64_t)(m0 + row) * p.lda +
                                                     (int64_t)kk * F::arow + col * 16)
                  : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int q = i * 256 + tid;
      const int t = q / (F::tb / 16), off = (q % (F::tb / 16)) * 16;
      const int nb = n0 / 16 + t;
      br[i] = (nb * 16 < p.N)
                  ? *reinterpret_cast<const uint4 *>(p.w + ((int64_t)nb * ktot + kk) * F::tb + off)
                  : make_uint4(0, 0, 0, 0);
    }
  };
  auto store = [&](int buf) {
    uint8_t *la = lds + buf * (ASTAGE + BSTAGE);
    uint8_t *lb = la + ASTAGE;
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int q = i * 256 + tid;
      const int row = q / (F::arow / 16), col = q % (F::arow / 16);
      *reinterpret_cast<uint4 *>(la + row * AROWP + col * 16) = ar[i];
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) *reinterpret_cast<uint4 *>(lb + (i * 256 + tid) * 16) = br[i];
  };

  v4i acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = v4i{0, 0, 0, 0};

  if (nk > 0) {
    load(0);
    store(0);
  }
  __syncthreads();
  for (int ks = 0; ks < nk; ++ks) {
    if (ks + 1 < nk) load(ks + 1);
    const uint8_t *la = lds + (ks & 1) * (ASTAGE + BSTAGE);
    const uint8_t *lb = la + ASTAGE;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      v4i af[TM], bf[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = a_operand<AFMT>(la + (wm * (BM / 2) + i * 16 + (lane & 15)) * AROWP, lane >> 4, c);
#pragma unroll
      for (int j = 0; j < TN; ++j) bf[j] = w_operand<BITS>(lb + (wn * TN + j) * F::tb, lane, c);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma16x16x64(af[i], bf[j], acc[i][j]);
    }
    if (ks + 1 < nk) store((ks + 1) & 1);
    __syncthreads();
  }

  int m_base[TM], n_base[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) m_base[i] = m0 + wm * (BM / 2) + i * 16;
#pragma unroll
  for (int j = 0; j < TN; ++j) n_base[j] = n0 + (wn * TN + j) * 16;
  if (nsplit > 1) {
    if (!splitk_combine<TM, TN>(p, acc, m_base, n_base, lane, split, nsplit, tile_id)) return;
  }
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) epilogue16<F::shift>(p, acc[i][j], m_base[i], n_base[j], lane);
}

// ----------------------------------------------------------------------------------------
// planning and launch

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Development tuning override, read once: FQ_TUNE="splits=<n>,red=<0|1>".
struct Tune {
  int splits = 0, red = -1;
};
static Tune read_tune() {
  Tune t;
  const char *e = getenv("FQ_TUNE");
  if (!e) return t;
  const char *s = strstr(e, "splits=");
  if (s) t.splits = atoi(s + 7);
  s = strstr(e, "red=");
  if (s) t.red = atoi(s + 4);
  return t;
}

GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, int bits) {
  (void)bits;
  static const Tune tune = read_tune();
  GemmPlan pl{};
  const int ktot = (int)(K / kTileK);
  if (M <= 64) {
    pl.kind = 0;
    pl.mt = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
    const int64_t nblk = (N + 63) / 64;
    // aim for about two workgroups per compute unit, slices of at least 4 k steps
    int64_t want = (512 + nblk - 1) / nblk;
    int64_t maxs = ktot / 4 > 0 ? ktot / 4 : 1;
    int64_t s = want < maxs ? want : maxs;
    if (s < 1) s = 1;
    pl.ksteps = (int)((ktot + s - 1) / s);
    pl.splits = (ktot + pl.ksteps - 1) / pl.ksteps;
    pl.tiles = nblk;
  } else {
    pl.kind = 1;
    pl.bm = 128;
    pl.bn = 128;
    const int64_t tiles = ((M + 127) / 128) * ((N + 127) / 128);
    int64_t s = 1;
    while (tiles * s < 256 && s < 4 && ktot / (s * 2) >= 8) s *= 2;
    pl.ksteps = (int)((ktot + s - 1) / s);
    pl.splits = (ktot + pl.ksteps - 1) / pl.ksteps;
    pl.tiles = tiles;
  }
  if (tune.splits > 0) {
    int64_t sp = tune.splits < ktot ? tune.splits : ktot;
    pl.ksteps = (int)((ktot + sp - 1) / sp);
    pl.splits = (ktot + pl.ksteps - 1) / pl.ksteps;
  }
  pl.red_atomic = tune.red == 1 ? 1 : 0;
  if (pl.tiles > kMaxCounters) {  // too many output tiles to count: no split
    pl.ksteps = ktot;
    pl.splits = 1;
  }
  pl.partial_bytes = pl.splits > 1 ? align256((size_t)(pl.red_atomic ? 1 : pl.splits) * M * N * 4) : 0;
  pl.counter_bytes = pl.splits > 1 ? kCounterRegionBytes : 0;
  return pl;
}

size_t gemm_plan_workspace(const GemmPlan &pl) { return pl.partial_bytes + pl.counter_bytes; }

template <int BITS, int AFMT>
static hipError_t launch_gemm_t(const GemmParams &p, const GemmPlan &pl, hipStream_t s) {
  if (pl.kind == 0) {
    dim3 grid((unsigned)pl.tiles, (unsigned)pl.splits);
    switch (pl.mt) {
      case 1: hipLaunchKernelGGL((gemm_stream_kernel<BITS, AFMT, 1>), grid, dim3(256), 0, s, p); break;
      case 2: hipLaunchKernelGGL((gemm_stream_kernel<BITS, AFMT, 2>), grid, dim3(256), 0, s, p); break;
      default: hipLaunchKernelGGL((gemm_stream_kernel<BITS, AFMT, 4>), grid, dim3(256), 0, s, p); break;
    }
  } else {
    dim3 grid((unsigned)pl.tiles, (unsigned)pl.splits);
    hipLaunchKernelGGL((gemm_tile_kernel<BITS, AFMT, 128, 128>), grid, dim3(256), 0, s, p);
  }
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs &g, const GemmPlan &pl, void *ws, size_t gap, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  GemmParams p;
  p.a = g.a;
  p.lda = g.lda;
  p.delta = g.delta;
  p.w = g.w;
  p.w_scale = g.w_scale;
  p.bias = g.bias;
  p.y = g.y;
  p.ldy = g.ldy;
  p.acc_out = g.acc_out;
  p.M = (int)g.M;
  p.N = (int)g.N;
  p.K = (int)g.K;
  p.ksteps = pl.ksteps;
  p.red_atomic = pl.red_atomic;
  // counters first, at a fixed offset, so that calls of any shape can share a workspace
  p.counters = pl.splits > 1 ? reinterpret_cast<uint32_t *>(ws) : nullptr;
  p.partial = pl.splits > 1 ? reinterpret_cast<int32_t *>(reinterpret_cast<uint8_t *>(ws) +
                                                          kCounterRegionBytes + gap)
                            : nullptr;
  if (g.bits == 4)
    return g.a_fmt == kANibble ? launch_gemm_t<4, kANibble>(p, pl, s) : launch_gemm_t<4, kAInt8>(p, pl, s);
  return launch_gemm_t<8, kAInt8>(p, pl, s);
}

}  // namespace fq
