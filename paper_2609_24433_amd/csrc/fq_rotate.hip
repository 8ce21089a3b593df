#include <type_traits>

#include "fq_codes.hpp"
#include "fq_device.hpp"
#include "fq_launch.hpp"

namespace fq {

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
    // the reads past the last group re-read it (valid LDS, results unused): no branch in
    // the loop, so the two register sets keep their registers instead of being copied
    load_group(0, 0);
#pragma unroll 1
    for (int jg = 0; jg < NG; jg += 2) {
      load_group(1, jg + 1 < NG ? jg + 1 : NG - 1);
      fma_group(0);
      load_group(0, jg + 2 < NG ? jg + 2 : NG - 1);
      if constexpr (NG % 2 == 0) {
        fma_group(1);
      } else {
        if (jg + 1 < NG) fma_group(1);
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
  float pm[S::TI];
#pragma unroll
  for (int c = 0; c < S::TI; ++c) pm[c] = post_mult ? post_mult[c_out + c] : 1.0f;
#pragma unroll
  for (int t = 0; t < TR; ++t) {
    const int64_t row = row0 + r0 + t;
    if (row < M) {
      float v[S::TI];
#pragma unroll
      for (int c = 0; c < S::TI; ++c) v[c] = post_mult ? acc[t][c] * pm[c] : acc[t][c];
      if constexpr (S::TI == 4) {
        *reinterpret_cast<float4 *>(z + row * K + c_out) = float4{v[0], v[1], v[2], v[3]};
      } else {
#pragma unroll
        for (int c = 0; c < S::TI; ++c) z[row * K + c_out + c] = v[c];
      }
    }
  }
}

// One workgroup per row; thread t owns 16-channel chunks t, t + 256, ... (K <= 32768).
template <int CPT>
__global__ __launch_bounds__(256) void rot_quant_kernel(const float *z, int64_t M, int K, int bits, float clip_ratio,
                                                        uint8_t *codes, int64_t ld_codes, float *delta, int out_fmt) {
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
  static std::atomic<uint64_t> attr{0};
  hipError_t e = allow_dynamic_lds(&rot_transform_kernel<Tin, B, TR>, lds, attr);
  if (e != hipSuccess) return e;
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
  // chunks per thread: the fewest that cover the row (no thread rereads a chunk it does not own)
  const int nch = K / 16;
  if (nch <= 256)
    hipLaunchKernelGGL(rot_quant_kernel<1>, dim3((unsigned)M), dim3(256), 0, s, z, M, K, bits, clip_ratio, codes,
                       ld_codes, delta, out_fmt);
  else if (nch <= 512)
    hipLaunchKernelGGL(rot_quant_kernel<2>, dim3((unsigned)M), dim3(256), 0, s, z, M, K, bits, clip_ratio, codes,
                       ld_codes, delta, out_fmt);
  else if (nch <= 1024)
    hipLaunchKernelGGL(rot_quant_kernel<4>, dim3((unsigned)M), dim3(256), 0, s, z, M, K, bits, clip_ratio, codes,
                       ld_codes, delta, out_fmt);
  else
    hipLaunchKernelGGL(rot_quant_kernel<8>, dim3((unsigned)M), dim3(256), 0, s, z, M, K, bits, clip_ratio, codes,
                       ld_codes, delta, out_fmt);
  return hipGetLastError();
}

}  // namespace fq
