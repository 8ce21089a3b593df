// The whole runtime projection for a few tokens in ONE kernel (Alg. 1 runtime: the
// Sec. III-C transform, the eq. (5) quantizer, the eq. (8) integer contraction and
// rescale).  For M <= 64 tokens and K <= 2048 the two-kernel path (prologue, then GEMM)
// spends most of its time on the second launch and on the dependency between the two;
// here every workgroup quantizes its own R rows itself, with exactly the prologue's fp32
// arithmetic (the helpers of fq_codes.hpp), while its weight tiles stream into registers,
// and then multiplies them.  Workgroups that share rows repeat those rows' prologue; the
// planner keeps that repetition small.
//
// Workgroup: 8 waves, R <= 8 rows [m0, m0 + R), NC = 128 NCW output channels: wave w owns
// the 16-channel tiles w + 8 i (i < NCW) over the whole of K.
//   loads, in this order: the prologue waves their row (with R <= 4 rows, waves 2r and
//     2r + 1 hold row r as 8-channel chunks, 128 lanes per row; with 8 rows, wave r holds
//     row r as 16-channel chunks; chunk c * lanes + lane, coalesced, in registers), every
//     wave the scales and biases of its tiles, then its weight tiles (one 16- or 32-byte
//     load per lane per tile and k step, in registers);
//   prologue (once the row has landed: loads complete in issue order): the blockwise
//     butterfly (stages inside a chunk in registers, the rest across lanes), the row
//     absmax across the wave (and the row's two waves through LDS), eq. (5); the codes go to LDS
//     already in the MFMA operand format (INT4 codes widened to int8 x 16, exactly as the
//     GEMM kernels widen them), 16-byte units XOR-swizzled by row so that the reads of 16
//     rows hit distinct banks, and delta_t to LDS;
//   one barrier, then each wave runs its tiles over all k steps on v_mfma_i32_16x16x64_i8
//     (activation operands from LDS, all read before the first MFMA; weight operands from
//     registers, widened as they are used; two accumulator chains per tile, even and odd
//     steps, added at the end: integer sums are exact in any order).  MFMA rows past R
//     read a valid row and are discarded;
//   the rescale y = bf16_rne(fp32(acc) (s_j delta_t) + b_j) is stored directly from the
//     MFMA layout (a row's 16 columns of a tile are 32 contiguous bytes).
#include "fq_codes.hpp"
#include "fq_device.hpp"
#include "fq_launch.hpp"

namespace fq {

struct SmallParams {
  const uint16_t *x;       // bf16 [M, ldx]
  int64_t ldx;
  const float *chan_mult;  // fold-before S^-1 or NULL
  const float *post_mult;  // fold-after P^-1 or NULL
  const uint8_t *w;        // kernel-native weight tiles
  const float *w_scale;    // [N]
  const float *bias;       // [N] or NULL
  uint16_t *y;             // bf16 [M, ldy]
  int64_t ldy;
  int M, N, K;
  int log2b;
  float clip_ratio;
  float cb;                // float nearest 1/sqrt(b)
};

constexpr int kSmallThreads = 64 * 8;

template <int BITS, int R, int CPT, int NCW>
struct SmallShape {
  static constexpr int NW = 8;                       // waves
  static constexpr int NT = kSmallThreads;
  static constexpr int NC = 16 * NW * NCW;           // output channels per workgroup
  static constexpr int TB = tile_bytes(BITS);        // bytes of one 16 x 128 weight tile
  static constexpr int LB = lane_bytes(BITS);        // a lane's bytes of one tile
  static constexpr int KMAX = 1024 * CPT;            // longest row: CPT chunks per lane
  static constexpr int KTMAX = KMAX / kTileK;        // k steps of the longest row
  static constexpr int ABYTES = R * KMAX;            // the rows' codes, one byte per code
  static constexpr int SHIFT = BITS == 4 ? 8 : 0;    // both operands widened x16 for INT4
  static constexpr size_t LDS = (size_t)ABYTES + 64; // codes | delta (8 floats) | row maxima (8)
  static_assert(R >= 1 && R <= NW, "one wave per row");
};

// Registers for the weights: NCW tiles x K / 128 steps x lane_bytes / 4.
static bool small_fits(int bits, int cpt, int ncw) {
  return ncw * 8 * cpt * (bits == 4 ? 4 : 8) <= 64;
}

// 16-byte unit u of row r of the codes, swizzled by the row's low 3 bits
__device__ __forceinline__ int code_unit(int r, int u) { return u ^ (r & 7); }

// v[c] *= m[CW j .. CW j + CW) for chunk j = c * tpr + t (chunk 0 past the row's end).
template <int CPT, int CW>
__device__ __forceinline__ void mul_chunks_cw(float (&v)[CPT][CW], const float *m, int tpr, int t, int nchunks) {
  float4 mv[CPT][CW / 4];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int j = c * tpr + t;
    const float4 *m4 = reinterpret_cast<const float4 *>(m + (j < nchunks ? j : 0) * CW);
#pragma unroll
    for (int i = 0; i < CW / 4; ++i) mv[c][i] = m4[i];
  }
#pragma unroll
  for (int c = 0; c < CPT; ++c)
#pragma unroll
    for (int i = 0; i < CW / 4; ++i) {
      v[c][4 * i] = v[c][4 * i] * mv[c][i].x;
      v[c][4 * i + 1] = v[c][4 * i + 1] * mv[c][i].y;
      v[c][4 * i + 2] = v[c][4 * i + 2] * mv[c][i].z;
      v[c][4 * i + 3] = v[c][4 * i + 3] * mv[c][i].w;
    }
}

template <int BITS, int R, int CPT, int NCW>
__global__ __launch_bounds__(kSmallThreads) void linear_small_kernel(SmallParams p) {
  using S = SmallShape<BITS, R, CPT, NCW>;
  constexpr int KT = S::KTMAX;
  constexpr int LU = S::LB / 16;  // 16-byte loads per lane per tile and k step
  // Prologue layout: up to 4 rows take two waves each (8-channel chunks, 128 lanes per
  // row); 8 rows take one wave each (16-channel chunks).  Both give the same codes.
  constexpr int WPR = R <= 4 ? 2 : 1;   // waves per row
  constexpr int CW = 16 / WPR;          // channels per chunk
  constexpr int TPR = 64 * WPR;         // lanes per row
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int K = p.K;
  const int ktot = K / kTileK;
  const int nch = K / CW;  // chunks per row
  uint8_t *al = lds;       // codes: row r at r * K, 16-channel chunk j at unit code_unit(r, j)
  float *dl = reinterpret_cast<float *>(lds + S::ABYTES);
  float *red = dl + 8;     // per-wave row maxima

  const int m0 = blockIdx.y * R;
  const int nt0 = blockIdx.x * (S::NC / 16);  // first 16-channel tile of the workgroup
  const int ntiles = p.N / 16;
  const int g = lane >> 4, cl = lane & 15;
  const bool pro = wave < R * WPR;            // a prologue wave
  const int r = wave / WPR;                   // its row
  const int t = (wave % WPR) * 64 + lane;     // its lane within the row

  // ---- loads: the row, the epilogue's scales, then the weight tiles ------------------------
  uint4 raw[CPT][CW / 8];
  if (pro) {
    const int mc = min(m0 + r, p.M - 1);  // rows past M repeat row M - 1 (never stored)
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int j = c * TPR + t;
      const uint4 *src = reinterpret_cast<const uint4 *>(p.x + (int64_t)mc * p.ldx + (int64_t)(j < nch ? j : 0) * CW);
#pragma unroll
      for (int u = 0; u < CW / 8; ++u) raw[c][u] = src[u];
    }
  }
  float sw[NCW], bj[NCW];
  const uint8_t *wtile[NCW];
#pragma unroll
  for (int i = 0; i < NCW; ++i) {
    const int tt = min(nt0 + wave + S::NW * i, ntiles - 1);  // tiles past N re-read the last one
    const int n = tt * 16 + cl;
    sw[i] = p.w_scale[n];
    bj[i] = p.bias ? p.bias[n] : 0.0f;
    wtile[i] = p.w + (int64_t)tt * ktot * S::TB + lane * S::LB;
  }
  // steps past this K re-read its last step (never multiplied)
  uint4 wr[NCW][KT][LU];
#pragma unroll
  for (int i = 0; i < NCW; ++i)
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int u = 0; u < LU; ++u)
        wr[i][kt][u] = reinterpret_cast<const uint4 *>(wtile[i] + (int64_t)min(kt, ktot - 1) * S::TB)[u];

  // ---- prologue of row m0 + r, bit for bit the standalone prologue's arithmetic --------------
  float v[CPT][CW];
  float amax = 0.0f;
  if (pro) {
#pragma unroll
    for (int c = 0; c < CPT; ++c)
#pragma unroll
      for (int u = 0; u < CW / 8; ++u) {
        const uint32_t w4[4] = {raw[c][u].x, raw[c][u].y, raw[c][u].z, raw[c][u].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          v[c][8 * u + 2 * i] = bf16_lo(w4[i]);
          v[c][8 * u + 2 * i + 1] = bf16_hi(w4[i]);
        }
      }
    if (p.chan_mult) mul_chunks_cw<CPT, CW>(v, p.chan_mult, TPR, t, nch);
    row_transform<CPT, CW>(v, p.log2b, t);
    if (p.post_mult) mul_chunks_cw<CPT, CW>(v, p.post_mult, TPR, t, nch);
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      if (c * TPR + t < nch) {
#pragma unroll
        for (int i = 0; i < CW; ++i) amax = fmaxf(amax, fabsf(v[c][i]));
      }
    }
    // across the wave's 64 lanes (max is order-free)
    amax = fmaxf(amax, lane_xor<1>(amax));
    amax = fmaxf(amax, lane_xor<2>(amax));
    amax = fmaxf(amax, lane_xor<4>(amax));
    amax = fmaxf(amax, lane_xor<8>(amax));
    amax = fmaxf(amax, lane_xor<16>(amax));
    amax = fmaxf(amax, __shfl_xor(amax, 32, kWave));
    if constexpr (WPR > 1) {
      if (lane == 0) red[wave] = amax;
    }
  }
  if constexpr (WPR > 1) {
    lds_barrier();  // every wave's row maximum is in LDS
    if (pro) amax = fmaxf(red[r * WPR], red[r * WPR + 1]);
  }
  if (pro) {
    const int q = (1 << (BITS - 1)) - 1;
    const float qf = (float)q;
    const bool zero = !(amax > 0.0f);
    const float rA = p.clip_ratio * amax;
    const float inv = (zero ? 0.0f : qf / rA) * row_sign<CW>(p.log2b, t);  // see lane_stage
    if (t == 0) dl[r] = zero ? 0.0f : (rA * p.cb) / qf;
    const float lim = qf + 0.49f;
    // no clamp at r = 1 (|u * inv| < q + 1/2; see quantize_bits_biased) unless inv is not finite
    const bool clamp = p.clip_ratio != 1.0f || !__builtin_isfinite(inv);
    uint8_t *row_l = al + r * K;
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int j = c * TPR + t;
      if (j < nch) {
        // the chunk's part of one MFMA operand (CW channels, stored as the MFMA consumes
        // it: INT4 widened to int8 x 16, INT8 as is), at its place in the row's k step
        if constexpr (BITS == 4) {
          uint32_t cb[CW];
          if (clamp) {
#pragma unroll
            for (int i = 0; i < CW; ++i) cb[i] = quantize_bits_biased<true>(v[c][i], inv, lim);
          } else {
#pragma unroll
            for (int i = 0; i < CW; ++i) cb[i] = quantize_bits_biased<false>(v[c][i], inv, lim);
          }
          uint32_t w[CW / 4];
#pragma unroll
          for (int h = 0; h < CW / 8; ++h) widen_biased8(cb + 8 * h, w[2 * h], w[2 * h + 1]);
          if constexpr (CW == 16)
            *reinterpret_cast<uint4 *>(row_l + code_unit(r, j) * 16) = make_uint4(w[0], w[1], w[2], w[3]);
          else
            *reinterpret_cast<uint2 *>(row_l + code_unit(r, j >> 1) * 16 + (j & 1) * 8) = make_uint2(w[0], w[1]);
        } else {
          int cc[CW];
          if (clamp) {
#pragma unroll
            for (int i = 0; i < CW; ++i) cc[i] = quantize_bits(v[c][i], inv, lim);
          } else {
#pragma unroll
            for (int i = 0; i < CW; ++i) cc[i] = __float_as_int(v[c][i] * inv + 12582912.0f);
          }
          if constexpr (CW == 16) {
            *reinterpret_cast<uint4 *>(row_l + code_unit(r, j) * 16) = pack_chunk_int8(cc);
          } else {
            uint2 op;
            op.x = __builtin_amdgcn_perm((uint32_t)cc[1], (uint32_t)cc[0], 0x0c0c0400u) |
                   __builtin_amdgcn_perm((uint32_t)cc[3], (uint32_t)cc[2], 0x04000c0cu);
            op.y = __builtin_amdgcn_perm((uint32_t)cc[5], (uint32_t)cc[4], 0x0c0c0400u) |
                   __builtin_amdgcn_perm((uint32_t)cc[7], (uint32_t)cc[6], 0x04000c0cu);
            *reinterpret_cast<uint2 *>(row_l + code_unit(r, j >> 1) * 16 + (j & 1) * 8) = op;
          }
        }
      }
    }
  }
  lds_barrier();  // the codes and the scales are in LDS

  // ---- GEMM over the whole of K ---------------------------------------------------------------
  // Steps past this K take zero activation operands (they add nothing), so that the MFMA
  // loop runs straight through.
  const int rr = cl & (R - 1);  // MFMA row -> a valid row of the block
  const uint8_t *arow = al + rr * K;
  v4i ar[KT][2];
#pragma unroll
  for (int kt = 0; kt < KT; ++kt)
#pragma unroll
    for (int c = 0; c < 2; ++c)
      ar[kt][c] = kt < ktot ? *reinterpret_cast<const v4i *>(arow + code_unit(rr, kt * 8 + 2 * g + c) * 16)
                            : v4i{0, 0, 0, 0};
  v4i acc[2][NCW];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int i = 0; i < NCW; ++i) acc[h][i] = v4i{0, 0, 0, 0};
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) {
#pragma unroll
    for (int i = 0; i < NCW; ++i) {
      v4i b0, b1;
      if constexpr (BITS == 4) {
        b0 = widen8(v2i{(int)wr[i][kt][0].x, (int)wr[i][kt][0].y});
        b1 = widen8(v2i{(int)wr[i][kt][0].z, (int)wr[i][kt][0].w});
      } else {
        b0 = __builtin_bit_cast(v4i, wr[i][kt][0]);
        b1 = __builtin_bit_cast(v4i, wr[i][kt][1]);
      }
      acc[kt & 1][i] = mfma16x16x64(ar[kt][0], b0, acc[kt & 1][i]);
      acc[kt & 1][i] = mfma16x16x64(ar[kt][1], b1, acc[kt & 1][i]);
    }
  }

  // ---- rescale and store straight from the MFMA layout ----------------------------------------
  // lane (g, cl) holds rows 4 g + e of column cl; the deltas of rows 4 g .. 4 g + 3 in one
  // read (rows past R read the spare words after the deltas and are never stored)
  const float4 d4 = *reinterpret_cast<const float4 *>(dl + 4 * g);
  const float dr[4] = {d4.x, d4.y, d4.z, d4.w};
  const int rows_here = min(R, p.M - m0) - 4 * g;  // valid rows from 4 g on
  uint16_t *yrow = p.y + (int64_t)(m0 + 4 * g) * p.ldy;
#pragma unroll
  for (int i = 0; i < NCW; ++i) {
    const v4i tsum = acc[0][i] + acc[1][i];
    const int n = (nt0 + wave + S::NW * i) * 16 + cl;
    if (n < p.N) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (e < rows_here) {
          const float val = (float)(tsum[e] >> S::SHIFT) * (sw[i] * dr[e]) + bj[i];
          yrow[(int64_t)e * p.ldy + n] = (uint16_t)f32_to_bf16(val);
        }
    }
  }
}

// ---------------------------------------------------------------------------------------
// plan and launch

template <int BITS, int R, int CPT, int NCW>
static hipError_t launch_small_t(const SmallParams &p, dim3 grid, hipStream_t s, bool go) {
  constexpr size_t lds = SmallShape<BITS, R, CPT, NCW>::LDS;
  static_assert(lds <= 64 * 1024, "LDS budget");
  static std::atomic<uint64_t> attr{0};
  hipError_t e = allow_dynamic_lds(&linear_small_kernel<BITS, R, CPT, NCW>, lds, attr);
  if (e != hipSuccess || !go) return e;
  hipLaunchKernelGGL((linear_small_kernel<BITS, R, CPT, NCW>), grid, dim3(SmallShape<BITS, R, CPT, NCW>::NT), lds, s, p);
  return hipGetLastError();
}

SmallPlan plan_small(int64_t M, int64_t N, int64_t K, int bits) {
  SmallPlan pl{};
  pl.ok = false;
  if (M < 1 || M > 64 || K > 2048 || (bits == 8 && K > 1024)) return pl;
  const int cpt = K <= 1024 ? 1 : 2;
  // Per-workgroup cycles: the prologue (~1400 cycles of VALU issue per 1024 channels of a
  // wave, plus latency: rows of two waves for R <= 4, one wave for R = 8, so two waves per
  // SIMD at R = 4 and 8), then the MFMAs and the weight widening of 2 waves per SIMD;
  // grids beyond one workgroup per compute unit run in rounds.  The weight stream
  // overlaps the prologue.
  double best = 1e30;
  for (int R : {1, 2, 4, 8}) {
    for (int ncw : {1, 2}) {
      if (!small_fits(bits, cpt, ncw)) continue;
      const int nc = 128 * ncw;
      const int64_t rb = (M + R - 1) / R, groups = (N + nc - 1) / nc;
      const double rounds = (double)((rb * groups + 255) / 256);
      const double pro = R <= 4 ? (R <= 2 ? 700.0 : 1400.0) * cpt + 1000.0 : 2800.0 * cpt + 800.0;
      const double mma = 2.0 * ncw * (K / 64) * (16.0 + (bits == 4 ? 12.0 : 0.0));
      const double cost = rounds * (pro + mma + 300.0);
      if (cost < best) {
        best = cost;
        pl.ok = true;
        pl.r = R;
        pl.cpt = cpt;
        pl.ncw = ncw;
        pl.rb = (int)rb;
        pl.groups = (int)groups;
      }
    }
  }
  return pl;
}

// Only shapes whose weight tiles fit the registers are built.
template <int BITS, int R, int CPT, int NCW>
static hipError_t launch_small_fit(const SmallParams &p, dim3 grid, hipStream_t s, bool go) {
  if constexpr (NCW * 8 * CPT * (BITS == 4 ? 4 : 8) <= 64) return launch_small_t<BITS, R, CPT, NCW>(p, grid, s, go);
  return hipErrorInvalidValue;
}

template <int BITS, int R, int CPT>
static hipError_t launch_small_ncw(const SmallParams &p, const SmallPlan &pl, dim3 grid, hipStream_t s, bool go) {
  switch (pl.ncw) {
    case 1: return launch_small_fit<BITS, R, CPT, 1>(p, grid, s, go);
    case 2: return launch_small_fit<BITS, R, CPT, 2>(p, grid, s, go);
    default: return hipErrorInvalidValue;
  }
}

template <int BITS, int R>
static hipError_t launch_small_cpt(const SmallParams &p, const SmallPlan &pl, dim3 grid, hipStream_t s, bool go) {
  switch (pl.cpt) {
    case 1: return launch_small_ncw<BITS, R, 1>(p, pl, grid, s, go);
    case 2: return launch_small_ncw<BITS, R, 2>(p, pl, grid, s, go);
    default: return hipErrorInvalidValue;
  }
}

template <int BITS>
static hipError_t launch_small_r(const SmallParams &p, const SmallPlan &pl, dim3 grid, hipStream_t s, bool go) {
  switch (pl.r) {
    case 1: return launch_small_cpt<BITS, 1>(p, pl, grid, s, go);
    case 2: return launch_small_cpt<BITS, 2>(p, pl, grid, s, go);
    case 4: return launch_small_cpt<BITS, 4>(p, pl, grid, s, go);
    case 8: return launch_small_cpt<BITS, 8>(p, pl, grid, s, go);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_linear_small(const SmallArgs &a, const SmallPlan &pl, hipStream_t s, bool go) {
  if (!pl.ok) return hipErrorInvalidValue;
  SmallParams p;
  p.x = static_cast<const uint16_t *>(a.x);
  p.ldx = a.ldx;
  p.chan_mult = a.chan_mult;
  p.post_mult = a.post_mult;
  p.w = a.w;
  p.w_scale = a.w_scale;
  p.bias = a.bias;
  p.y = a.y;
  p.ldy = a.ldy;
  p.M = (int)a.M;
  p.N = (int)a.N;
  p.K = (int)a.K;
  p.log2b = a.log2b;
  p.clip_ratio = a.clip_ratio;
  p.cb = a.cb;
  const dim3 grid((unsigned)pl.groups, (unsigned)pl.rb);
  return a.bits == 4 ? launch_small_r<4>(p, pl, grid, s, go) : launch_small_r<8>(p, pl, grid, s, go);
}

}  // namespace fq
