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
//           no LDS;
//   the row absmax is reduced over the row's lanes (DPP / swizzle) and waves (LDS), and
//   each thread quantizes, packs and stores its chunks in natural channel order.
// Every stage is the pair update (a, c) -> (a + c, a - c) in fp32 in ascending h, so the
// result does not depend on where the data lives; no multiply-add is contracted.
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

// Raw 16-channel chunk as loaded: bf16 = 2 x 16 bytes, fp32 = 4 x 16 bytes.
template <typename Tin>
struct Chunk {
  static constexpr int U4 = sizeof(Tin) == 2 ? 2 : 4;
  uint4 u[U4];
};

template <typename Tin>
__device__ __forceinline__ void load_chunk(const void *base, int64_t off, Chunk<Tin> &c) {
  const uint4 *p = reinterpret_cast<const uint4 *>(reinterpret_cast<const Tin *>(base) + off);
#pragma unroll
  for (int i = 0; i < Chunk<Tin>::U4; ++i) c.u[i] = p[i];
}

template <typename Tin>
__device__ __forceinline__ void unpack_chunk(const Chunk<Tin> &c, float (&v)[16]) {
  if constexpr (sizeof(Tin) == 2) {
    const uint32_t w[8] = {c.u[0].x, c.u[0].y, c.u[0].z, c.u[0].w, c.u[1].x, c.u[1].y, c.u[1].z, c.u[1].w};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      v[2 * i] = bf16_lo(w[i]);
      v[2 * i + 1] = bf16_hi(w[i]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[4 * i] = __uint_as_float(c.u[i].x);
      v[4 * i + 1] = __uint_as_float(c.u[i].y);
      v[4 * i + 2] = __uint_as_float(c.u[i].z);
      v[4 * i + 3] = __uint_as_float(c.u[i].w);
    }
  }
}

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

// code = clamp(rne(u * inv), -q, q), returned as the fp32 bit pattern 0x4B400000 + code,
// whose low byte is the two's-complement code.  t is first clamped to
// [-(q + 0.49), q + 0.49]: every t that rounds to a value beyond +-q lands on +-(q + 0.49),
// which rounds to +-q, and no other t moves, so the clamp after rounding is implied.
// Adding 1.5 * 2^23 then rounds to the nearest integer, ties to even, exactly as rint
// does for |t| < 2^22.
__device__ __forceinline__ int quantize_bits(float u, float inv, float lim) {
  const float t = __builtin_amdgcn_fmed3f(u * inv, -lim, lim);
  return __float_as_int(t + 12582912.0f);
}

// Pack 16 quantized bit patterns (natural channel order; low byte = code) and store them.
__device__ __forceinline__ void store_chunk_bits(uint8_t *row_out, int chunk, const int (&c)[16],
                                                 int out_fmt) {
  if (out_fmt == kOutNibble) {
    uint32_t w[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      uint32_t b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        b[i] = ((uint32_t)c[8 * h + 2 * i] & 0xFu) | ((uint32_t)c[8 * h + 2 * i + 1] << 4);
      // low bytes of b[0..3] -> one word
      const uint32_t lo = __builtin_amdgcn_perm(b[1], b[0], 0x0c0c0400u);
      const uint32_t hi = __builtin_amdgcn_perm(b[3], b[2], 0x04000c0cu);
      w[h] = lo | hi;
    }
    *reinterpret_cast<uint2 *>(row_out + (int64_t)chunk * 8) = make_uint2(w[0], w[1]);
  } else {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t lo = __builtin_amdgcn_perm((uint32_t)c[4 * i + 1], (uint32_t)c[4 * i], 0x0c0c0400u);
      const uint32_t hi = __builtin_amdgcn_perm((uint32_t)c[4 * i + 3], (uint32_t)c[4 * i + 2], 0x04000c0cu);
      w[i] = lo | hi;
    }
    *reinterpret_cast<uint4 *>(row_out + (int64_t)chunk * 16) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// Value of lane (l ^ M) of the wave, for M < 32: DPP quad permutations for 1 and 2, a
// 16-lane row rotation by 8 for 8, the LDS crossbar's bit-mask swizzle (no memory) for 4
// and 16.  Pure data movement: the butterfly sums stay bit-exact.
template <int M>
__device__ __forceinline__ float lane_xor(float v) {
  const int x = __float_as_int(v);
  int r;
  if constexpr (M == 1) r = __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false);       // quad_perm 1,0,3,2
  else if constexpr (M == 2) r = __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false);  // quad_perm 2,3,0,1
  else if constexpr (M == 8) r = __builtin_amdgcn_update_dpp(0, x, 0x128, 0xF, 0xF, false); // row_ror:8
  else r = __builtin_amdgcn_ds_swizzle(x, (M << 10) | 0x1F);                                // xor M in 32 lanes
  return __int_as_float(r);
}

// Butterfly stage h = 16 M across lanes: chunk j pairs with chunk j ^ M, held by lane ^ M.
// The lower chunk keeps a + c, the upper one a - c, as fma(+-1, own, partner): one
// rounding of the exact sum or difference, the same as the add or subtract.
template <int M, int CPT>
__device__ __forceinline__ void lane_stage(float (&v)[CPT][16], int tau) {
  const float sgn = (tau & M) ? -1.0f : 1.0f;
#pragma unroll
  for (int c = 0; c < CPT; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) v[c][i] = __builtin_fmaf(sgn, v[c][i], lane_xor<M>(v[c][i]));
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
  Chunk<Tin> raw[CPT];
  float4 cm[CPT][4], pm[CPT][4];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int j = c * TPR + tau;
    const int jc = j < nchunks ? j : 0;
    load_chunk<Tin>(p.x, row_c * p.ldx + (int64_t)jc * 16, raw[c]);
    if (p.chan_mult) {
      const float4 *m4 = reinterpret_cast<const float4 *>(p.chan_mult + jc * 16);
#pragma unroll
      for (int i = 0; i < 4; ++i) cm[c][i] = m4[i];
    }
    if (p.post_mult) {
      const float4 *m4 = reinterpret_cast<const float4 *>(p.post_mult + jc * 16);
#pragma unroll
      for (int i = 0; i < 4; ++i) pm[c][i] = m4[i];
    }
  }

  // ---- pass 1: optional multiplier, stages h < 16 in registers -------------------------
  float v1[CPT][16];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    unpack_chunk<Tin>(raw[c], v1[c]);
    if (p.chan_mult) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v1[c][4 * i] = v1[c][4 * i] * cm[c][i].x;
        v1[c][4 * i + 1] = v1[c][4 * i + 1] * cm[c][i].y;
        v1[c][4 * i + 2] = v1[c][4 * i + 2] * cm[c][i].z;
        v1[c][4 * i + 3] = v1[c][4 * i + 3] * cm[c][i].w;
      }
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
    for (int c = 0; c < CPT; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v1[c][4 * i] = v1[c][4 * i] * pm[c][i].x;
        v1[c][4 * i + 1] = v1[c][4 * i + 1] * pm[c][i].y;
        v1[c][4 * i + 2] = v1[c][4 * i + 2] * pm[c][i].z;
        v1[c][4 * i + 3] = v1[c][4 * i + 3] * pm[c][i].w;
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
        for (int i = 0; i < 16; ++i) cc[i] = quantize_bits(v1[c][i], inv, lim);
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
  static bool attr = false;  // more than 64 KB of dynamic LDS must be requested once
  if (smem > 65536 && !attr) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&fwht_quant_kernel<Tin, LOG2B, CPT, NT>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
    attr = true;
  }
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

// ---------------------------------------------------------------------------------------
// Stored composite rotation (Sec. III-C, the action expert's optional transform in place of
// the block Hadamard): gather by a channel permutation, then per-block orthogonal b x b
// matrices, as two kernels through an fp32 workspace z [M, K]:
//   rot_transform_kernel: a workgroup takes one block and R rows.  The block's matrix goes
//     to LDS transposed (4 x 4 sub-blocks: coalesced 16-byte loads, 16-byte writes), the
//     rows' gathered, pre-multiplied inputs w_j = x[perm[kb + j]] * s_inv[perm[kb + j]]
//     transposed as well; both are XOR-swizzled so that the transposing writes are free of
//     bank conflicts.  Thread (g, h) owns TR rows times TI outputs and, for j = 0..b-1
//     ascending, reads TI matrix entries (one 16-byte read) and TR inputs (broadcast) and
//     advances each output's fma chain Q[i][j] * w_j from +0: the register-tiled form of the
//     per-output chain, whose order it keeps.  Then the optional fold-after multiplier;
//   rot_quant_kernel: one workgroup per row: row absmax, eq. (5) with c_b = 1 (the
//     blocks are orthonormal), canonical packing.
// Permutation entries are clamped into [0, K): a bad permutation gives wrong codes, never
// an out-of-bounds read.

template <int B>
struct RotShape {
  static constexpr int TI = B < 4 ? B : 4;  // outputs per thread
  static constexpr int NI = B / TI;         // output groups per block
  static constexpr int NRG = 256 / NI;      // row groups per workgroup
  static constexpr int QSW = (B / 4 < 8 ? (B >= 4 ? B / 4 : 1) : 8) - 1;  // matrix chunk swizzle mask
};

template <int B, int TR>
constexpr int rot_rows() { return RotShape<B>::NRG * TR; }

template <int B, int TR>
constexpr size_t rot_lds_bytes() {
  return ((size_t)B * B + (size_t)B * rot_rows<B, TR>()) * sizeof(float);
}

template <typename Tin, int B, int TR>
__global__ __launch_bounds__(256) void rot_transform_kernel(const void *x, int64_t ldx, const int32_t *perm,
                                                            const float *blocks, const float *chan_mult,
                                                            const float *post_mult, int64_t M, int K, float *z) {
  using S = RotShape<B>;
  constexpr int R = rot_rows<B, TR>();
  // input swizzle mask; with four rows per thread it keeps each thread's rows one aligned
  // 16-byte group (two LDS reads per j in all, few enough for the lgkm counter to track a
  // whole prefetched group)
  constexpr int VSW = ((R < 32 ? R : 32) - 1) & (TR == 4 ? ~3 : ~0);
  extern __shared__ __attribute__((aligned(16))) float rot_lds[];
  // qt[j * B + 4 * (c ^ sw(j)) + u] = Q[4 c + u][j], sw(j) = (j / 4) & QSW
  // vt[j * R + (r ^ (j & VSW))] = w_j of row r
  float *qt = rot_lds;
  float *vt = rot_lds + B * B;
  const int tid = threadIdx.x;
  const int kblk = blockIdx.x;
  const int64_t row0 = (int64_t)blockIdx.y * R;
  const float *Q = blocks + (int64_t)kblk * B * B;
  // Thread (rr, j) gathers channel perm[kb + j] for rows rr, rr + 256/b, ...: one
  // permutation entry and multiplier per thread.  Loads go out in dependency order
  // (permutation, matrix, inputs) and all before the first LDS write, so the matrix's
  // round trip overlaps the permutation's and the gather's.
  constexpr int JR = 256 / B, NV = R / JR;
  const int j = tid % B, rr = tid / B;
  int src = perm ? perm[kblk * B + j] : kblk * B + j;
  constexpr int NBK = B / 4, NSB = NBK * NBK, NQ = B >= 4 ? (NSB + 255) / 256 : 1;
  float4 tq[NQ][4];
  if constexpr (B >= 4) {
    // sub-block (ib, jb) = rows 4 ib.. of columns 4 jb..; lanes take consecutive jb
#pragma unroll
    for (int k = 0; k < NQ; ++k) {
      const int sb = tid + 256 * k;
      if (NSB % 256 == 0 || sb < NSB) {
        const int jb = sb % NBK, ib = sb / NBK;
#pragma unroll
        for (int u = 0; u < 4; ++u) tq[k][u] = *reinterpret_cast<const float4 *>(Q + (4 * ib + u) * B + 4 * jb);
      }
    }
  }
  src = min(max(src, 0), K - 1);
  const float cm = chan_mult ? chan_mult[src] : 1.0f;
  // rows past M load row M - 1 (no branch, so every load is in flight at once) and store 0
  using Raw = typename std::conditional<sizeof(Tin) == 2, uint16_t, float>::type;
  Raw raw[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int64_t row = min(row0 + rr + JR * k, M - 1);
    raw[k] = reinterpret_cast<const Raw *>(x)[row * ldx + src];
  }
  __builtin_amdgcn_sched_barrier(0);  // every load above issues before the first use below
  if constexpr (B >= 4) {
#pragma unroll
    for (int k = 0; k < NQ; ++k) {
      const int sb = tid + 256 * k;
      if (NSB % 256 == 0 || sb < NSB) {
        const int jb = sb % NBK, ib = sb / NBK;
        const int col = 4 * (ib ^ (jb & S::QSW));
        float *d = qt + 4 * jb * B + col;
        *reinterpret_cast<float4 *>(d) = float4{tq[k][0].x, tq[k][1].x, tq[k][2].x, tq[k][3].x};
        *reinterpret_cast<float4 *>(d + B) = float4{tq[k][0].y, tq[k][1].y, tq[k][2].y, tq[k][3].y};
        *reinterpret_cast<float4 *>(d + 2 * B) = float4{tq[k][0].z, tq[k][1].z, tq[k][2].z, tq[k][3].z};
        *reinterpret_cast<float4 *>(d + 3 * B) = float4{tq[k][0].w, tq[k][1].w, tq[k][2].w, tq[k][3].w};
      }
    }
  } else {
    if (tid < B * B) qt[(tid / B) * B + tid % B] = Q[(tid % B) * B + tid / B];
  }
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const bool in = row0 + rr + JR * k < M;
    float v;
    if constexpr (sizeof(Tin) == 2)
      v = bf16_lo(raw[k]);
    else
      v = raw[k];
    vt[j * R + ((rr + JR * k) ^ (j & VSW))] = in ? (chan_mult ? v * cm : v) : 0.0f;
  }
  __syncthreads();
  const int h = tid % S::NI, g = tid / S::NI;
  const int r0 = g * TR;
  float acc[TR][S::TI];
#pragma unroll
  for (int t = 0; t < TR; ++t)
#pragma unroll
    for (int c = 0; c < S::TI; ++c) acc[t][c] = 0.0f;
  if constexpr (S::TI == 4) {
    // groups of 4 j, double-buffered in registers: group jg + 1 is read while group jg is
    // multiplied, so LDS latency overlaps the fma chains
    constexpr int NG = B / 4;
    float4 qa[2][4];
    float va[2][4][TR];
    auto load_group = [&](int buf, int jg) {
      const int col = 4 * (h ^ (jg & S::QSW));
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = 4 * jg + u;
        qa[buf][u] = *reinterpret_cast<const float4 *>(qt + j * B + col);
        if constexpr (TR == 4) {
          const float4 w4 = *reinterpret_cast<const float4 *>(vt + j * R + (r0 ^ (j & VSW)));
          va[buf][u][0] = w4.x; va[buf][u][1] = w4.y; va[buf][u][2] = w4.z; va[buf][u][3] = w4.w;
        } else {
#pragma unroll
          for (int t = 0; t < TR; ++t) va[buf][u][t] = vt[j * R + ((r0 + t) ^ (j & VSW))];
        }
      }
    };
    auto fma_group = [&](int buf) {
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int t = 0; t < TR; ++t) {
          const float w = va[buf][u][t];
          acc[t][0] = __builtin_fmaf(qa[buf][u].x, w, acc[t][0]);
          acc[t][1] = __builtin_fmaf(qa[buf][u].y, w, acc[t][1]);
          acc[t][2] = __builtin_fmaf(qa[buf][u].z, w, acc[t][2]);
          acc[t][3] = __builtin_fmaf(qa[buf][u].w, w, acc[t][3]);
        }
    };
    load_group(0, 0);
#pragma unroll 1
    for (int jg = 0; jg < NG; jg += 2) {
      if (jg + 1 < NG) load_group(1, jg + 1);
      fma_group(0);
      if (jg + 1 < NG) {
        if (jg + 2 < NG) load_group(0, jg + 2);
        fma_group(1);
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < B; ++j) {
#pragma unroll
      for (int t = 0; t < TR; ++t) {
        const float w = vt[j * R + ((r0 + t) ^ (j & VSW))];
#pragma unroll
        for (int c = 0; c < S::TI; ++c) acc[t][c] = __builtin_fmaf(qt[j * B + c], w, acc[t][c]);
      }
    }
  }
  const int c_out = kblk * B + h * S::TI;
#pragma unroll
  for (int t = 0; t < TR; ++t) {
    const int64_t row = row0 + r0 + t;
    if (row < M) {
#pragma unroll
      for (int c = 0; c < S::TI; ++c) {
        float v = acc[t][c];
        if (post_mult) v = v * post_mult[c_out + c];
        z[row * K + c_out + c] = v;
      }
    }
  }
}

// One workgroup per row; thread t owns 16-channel chunks t, t + 256, ... (K <= 32768).
__global__ __launch_bounds__(256) void rot_quant_kernel(const float *z, int64_t M, int K, int bits, float clip_ratio,
                                                        uint8_t *codes, int64_t ld_codes, float *delta, int out_fmt) {
  constexpr int CPT = 8;
  __shared__ float red[4];
  const int tid = threadIdx.x;
  const int64_t row = blockIdx.x;
  const int nchunks = K >> 4;
  const float *zr = z + row * K;
  float v[CPT][16];
  float amax = 0.0f;
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    // chunks past the row's end reread its last chunk (no branch, so every load is in
    // flight at once) and are left out of the maximum
    const int j = min(c * 256 + tid, nchunks - 1);
    const float4 *s4 = reinterpret_cast<const float4 *>(zr + j * 16);
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const float4 t = s4[q4];
      v[c][4 * q4] = t.x; v[c][4 * q4 + 1] = t.y; v[c][4 * q4 + 2] = t.z; v[c][4 * q4 + 3] = t.w;
    }
  }
#pragma unroll
  for (int c = 0; c < CPT; ++c)
    if (c * 256 + tid < nchunks)
#pragma unroll
      for (int e = 0; e < 16; ++e) amax = fmaxf(amax, fabsf(v[c][e]));
  amax = fmaxf(amax, lane_xor<1>(amax));
  amax = fmaxf(amax, lane_xor<2>(amax));
  amax = fmaxf(amax, lane_xor<4>(amax));
  amax = fmaxf(amax, lane_xor<8>(amax));
  amax = fmaxf(amax, lane_xor<16>(amax));
  amax = fmaxf(amax, __shfl_xor(amax, 32, kWave));
  if ((tid & 63) == 0) red[tid >> 6] = amax;
  __syncthreads();
  amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const int q = (1 << (bits - 1)) - 1;
  const float qf = (float)q;
  const bool zero = !(amax > 0.0f);
  const float rA = clip_ratio * amax;
  const float inv = zero ? 0.0f : qf / rA;
  if (tid == 0) delta[row] = zero ? 0.0f : (rA * 1.0f) / qf;
  uint8_t *row_out = codes + row * ld_codes;
  const float lim = qf + 0.49f;
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int j = c * 256 + tid;
    if (j < nchunks) {
      int cc[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) cc[e] = quantize_bits(v[c][e], inv, lim);
      store_chunk_bits(row_out, j, cc, out_fmt);
    }
  }
}

template <typename Tin, int B, int TR>
static hipError_t launch_rot_tr(const void *x, int64_t ldx, const int32_t *perm, const float *blocks,
                                const float *chan_mult, const float *post_mult, int64_t M, int K, float *z,
                                hipStream_t s) {
  constexpr size_t lds = rot_lds_bytes<B, TR>();
  static_assert(lds <= 160 * 1024, "LDS budget");
  static bool attr = false;  // more than 64 KB of dynamic LDS must be requested once
  if (lds > 65536 && !attr) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&rot_transform_kernel<Tin, B, TR>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr = true;
  }
  constexpr int R = rot_rows<B, TR>();
  const int64_t gy = (M + R - 1) / R;
  if (gy > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL((rot_transform_kernel<Tin, B, TR>), dim3((unsigned)(K / B), (unsigned)gy), dim3(256), lds, s,
                     x, ldx, perm, blocks, chan_mult, post_mult, M, K, z);
  return hipGetLastError();
}

// Four rows per thread when that still gives a grid of at least one workgroup per compute
// unit (with b = 128 two such workgroups fill a compute unit's LDS), else one (small M:
// more workgroups, each loading its block's matrix once).
template <typename Tin, int B>
static hipError_t launch_rot_b(const void *x, int64_t ldx, const int32_t *perm, const float *blocks,
                               const float *chan_mult, const float *post_mult, int64_t M, int K, float *z,
                               hipStream_t s) {
  const int64_t wide = (K / B) * ((M + rot_rows<B, 4>() - 1) / rot_rows<B, 4>());
  return wide >= 256 ? launch_rot_tr<Tin, B, 4>(x, ldx, perm, blocks, chan_mult, post_mult, M, K, z, s)
                     : launch_rot_tr<Tin, B, 1>(x, ldx, perm, blocks, chan_mult, post_mult, M, K, z, s);
}

template <typename Tin>
static hipError_t launch_rot_t(const void *x, int64_t ldx, const int32_t *perm, const float *blocks,
                               const float *chan_mult, const float *post_mult, int64_t M, int K, int b,
                               float *z, hipStream_t s) {
  switch (b) {
    case 1: return launch_rot_b<Tin, 1>(x, ldx, perm, blocks, chan_mult, post_mult, M, K, z, s);
    case 2: return launch_rot_b<Tin, 2>(x, ldx, perm, blocks, chan_mult, post_mult, M, K, z, s);
    case 4: return launch_rot_b<Tin, 4>(x, ldx, perm, blocks, chan_mult, post_mult, M, K, z, s);
    case 8: return launch_rot_b<Tin, 8>(x, ldx, perm, blocks, chan_mult, post_mult, M, K, z, s);
    case 16: return launch_rot_b<Tin, 16>(x, ldx, perm, blocks, chan_mult, post_mult, M, K, z, s);
    case 32: return launch_rot_b<Tin, 32>(x, ldx, perm, blocks, chan_mult, post_mult, M, K, z, s);
    case 64: return launch_rot_b<Tin, 64>(x, ldx, perm, blocks, chan_mult, post_mult, M, K, z, s);
    case 128: return launch_rot_b<Tin, 128>(x, ldx, perm, blocks, chan_mult, post_mult, M, K, z, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_rotate_quant(const void *x, bool x_is_f32, int64_t ldx, const int32_t *perm,
                               const float *blocks, const float *chan_mult, const float *post_mult,
                               int64_t M, int K, int b, int bits, float clip_ratio, uint8_t *codes,
                               int64_t ld_codes, float *delta, int out_fmt, float *z, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (K > 256 * 8 * 16 || M > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipError_t e = x_is_f32 ? launch_rot_t<float>(x, ldx, perm, blocks, chan_mult, post_mult, M, K, b, z, s)
                          : launch_rot_t<uint16_t>(x, ldx, perm, blocks, chan_mult, post_mult, M, K, b, z, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(rot_quant_kernel, dim3((unsigned)M), dim3(256), 0, s, z, M, K, bits, clip_ratio, codes,
                     ld_codes, delta, out_fmt);
  return hipGetLastError();
}

}  // namespace fq
