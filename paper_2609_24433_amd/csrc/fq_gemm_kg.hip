// Tiled INT4 GEMM for a few hundred to ~1000 tokens at long K (eq. (8) contraction and
// rescale), where 128 x 128 output tiles would leave most compute units idle unless K is
// split across workgroups (and a second kernel adds the slices).
//
// Workgroup: 4 waves, one 128 x 64 output tile (8 x 4 tiles of 16 x 16); wave w owns the
// k steps w, w + 4, w + 8, ... of the whole of K, so the tile needs no split of K across
// workgroups and its four partial sums add up through LDS at the end (exact integers).
// Every wave streams its own operands straight from L2 into registers, three register sets
// deep (the loads of steps ks + 4 and ks + 8 are in flight while step ks is multiplied; two
// sets measured the same to 6% slower at M = 816, K 16384 -> N 2048), with buffer
// loads: one SGPR descriptor per operand, a fixed per-lane offset and a per-step scalar
// offset, so the loop carries no address arithmetic.  No operand goes through LDS.
//
// Activation codes come k-step major: the 64 bytes (128 nibble codes) of row r for k step
// ks sit at ks * 64 M + 64 r, so a row tile's operand of one step is 1 KB contiguous
// (16 rows x 64 bytes), one coalesced load.  Read from the canonical row-major layout the
// same operand is 16 half cache lines and the kernel measured 30% slower; the fused
// projection's prologue writes this layout directly and the GEMM entry point converts
// canonical codes first (codes_kmajor_kernel).
//
// MFMA and widening as in the other GEMM kernels: v_mfma_i32_16x16x64_i8 on nibbles widened
// to int8 x 16 (channels interleaved 0 2 4 6 1 3 5 7 in both operands), INT32 accumulators
// in AGPRs (this file is built without the VGPR accumulator form: 128 accumulators plus two
// register sets of operands do not fit in 256 VGPRs), the factor 256 shifted out at the end.
#include "fq_device.hpp"
#include "fq_launch.hpp"

namespace fq {

namespace {

constexpr int kKgTI = 8;    // 16-row tiles per workgroup tile
constexpr int kKgTJ = 4;    // 16-column tiles per workgroup tile
constexpr int kKgWaves = 4; // k groups
constexpr int kKgShift = 8; // both operands widened x 16
constexpr int kKgSets = 3;  // operand register sets: loads run two k steps ahead
constexpr size_t kKgPartLds = (size_t)kKgWaves * kKgTI * kKgTJ * 1024;  // the k groups' sums
constexpr int kKgOutStride = 16 * kKgTJ * 2 + 16;                        // bf16 staging row, padded
constexpr size_t kKgLds = kKgPartLds + (size_t)16 * kKgTI * kKgOutStride;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_of(const void *base, int64_t bytes) {
  const int n = bytes < 0x7fffffff ? (int)bytes : 0x7fffffff;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, n, 0x00020000);
}

__global__ __launch_bounds__(64 * kKgWaves) void gemm_kgroup_kernel(KgParams p) {
  constexpr int TI = kKgTI, TJ = kKgTJ, KG = kKgWaves, NB = TI * TJ;
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ntn = (p.N + 16 * TJ - 1) / (16 * TJ);
  const int tn = blockIdx.x % ntn, tm = blockIdx.x / ntn;
  const int m0 = tm * 16 * TI, n0 = tn * 16 * TJ;
  const int ktot = p.K / kTileK;
  const int astep = p.M * 64;  // bytes of one k step of the k-major codes

  // per-lane operand offsets: row 16 i + l % 16 (rows past M repeat row M - 1, never
  // stored), 16 bytes per lane group (channels 32 (l / 16) + [0, 32) of the step)
  uint32_t aoff[TI];
#pragma unroll
  for (int i = 0; i < TI; ++i) aoff[i] = (uint32_t)min(m0 + 16 * i + (lane & 15), p.M - 1) * 64u + 16u * (lane >> 4);
  // weight tile (nb, ks) at (nb K/128 + ks) KB, lane l's 16 bytes at 16 l (tiles past N
  // re-read the last one, never stored)
  uint32_t boff[TJ];
#pragma unroll
  for (int j = 0; j < TJ; ++j) boff[j] = (uint32_t)min(n0 / 16 + j, p.N / 16 - 1) * (uint32_t)ktot * 1024u + lane * 16;
  const __amdgpu_buffer_rsrc_t arsrc = buffer_of(p.a, (int64_t)ktot * astep);
  const __amdgpu_buffer_rsrc_t brsrc = buffer_of(p.w, (int64_t)(p.N / 16) * ktot * 1024);

  v4i acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) acc[i][j] = v4i{0, 0, 0, 0};
  constexpr int NSET = kKgSets;
  v4i ra[NSET][TI], rb[NSET][TJ];
  auto load = [&](v4i (&ra_)[TI], v4i (&rb_)[TJ], int ks) {
#pragma unroll
    for (int i = 0; i < TI; ++i) ra_[i] = __builtin_amdgcn_raw_buffer_load_b128(arsrc, aoff[i], ks * astep, 0);
#pragma unroll
    for (int j = 0; j < TJ; ++j) rb_[j] = __builtin_amdgcn_raw_buffer_load_b128(brsrc, boff[j], ks * 1024, 0);
  };
  // both 64-channel chunks of a step: the widened weight operands of the chunk, then each
  // row tile's widened activation operand against the four of them
  auto compute = [&](const v4i (&ra_)[TI], const v4i (&rb_)[TJ]) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      v4i wb[TJ];
#pragma unroll
      for (int j = 0; j < TJ; ++j) wb[j] = widen8(c == 0 ? v2i{rb_[j].x, rb_[j].y} : v2i{rb_[j].z, rb_[j].w});
#pragma unroll
      for (int i = 0; i < TI; ++i) {
        const v4i wa = widen8(c == 0 ? v2i{ra_[i].x, ra_[i].y} : v2i{ra_[i].z, ra_[i].w});
#pragma unroll
        for (int j = 0; j < TJ; ++j) acc[i][j] = mfma16x16x64(wa, wb[j], acc[i][j]);
      }
    }
  };
  // NSET steps per loop trip, one per register set, each set's loads issued NSET - 1 steps
  // before its multiplies (the scheduling walls keep the compiler from sinking them); the
  // last nk mod NSET steps after the loop, so the accumulators flow through a single path
  // (a conditional trip end made the compiler copy them between AGPR sets every trip).  A
  // load past the wave's last step re-reads step K/128 - 1 (in bounds, never multiplied).
  const int nk = ktot > wave ? (ktot - wave + KG - 1) / KG : 0;
  const int klast = ktot - 1;
  int ks = wave;
#pragma unroll
  for (int q = 0; q < NSET - 1; ++q) load(ra[q], rb[q], min(ks + q * KG, klast));
  int t = 0;
  for (; t + NSET - 1 < nk; t += NSET) {
#pragma unroll
    for (int q = 0; q < NSET; ++q) {
      load(ra[(q + NSET - 1) % NSET], rb[(q + NSET - 1) % NSET], min(ks + (q + NSET - 1) * KG, klast));
      __builtin_amdgcn_sched_barrier(0);
      compute(ra[q], rb[q]);
      __builtin_amdgcn_sched_barrier(0);
    }
    ks += NSET * KG;
  }
#pragma unroll
  for (int q = 0; q < NSET - 1; ++q)
    if (t + q < nk) compute(ra[q], rb[q]);

  // ---- the k groups' sums: every wave leaves its 32 tiles in LDS (lane-major, 1 KB per
  // tile), then wave w adds up column tile w of all four and rescales it ----
  v4i *part = reinterpret_cast<v4i *>(lds);
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) part[(wave * NB + i * TJ + j) * 64 + lane] = acc[i][j];
  __syncthreads();
  static_assert(TJ == KG, "one column tile per wave in the final sum");
  const int j = wave;
  const int g = lane >> 4, cl = lane & 15;
  v4i fin[TI];
#pragma unroll
  for (int i = 0; i < TI; ++i) {
    v4i s = part[(i * TJ + j) * 64 + lane];
#pragma unroll
    for (int q = 1; q < KG; ++q) {
      const v4i u = part[(q * NB + i * TJ + j) * 64 + lane];
      s.x += u.x;
      s.y += u.y;
      s.z += u.z;
      s.w += u.w;
    }
    fin[i] = s;
  }
  // rescale factors: the rows' delta_t (rows past M read row M - 1, never stored) and the
  // column's s_j and b_j
  float dt[TI][4];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) dt[i][r] = p.delta[min(m0 + 16 * i + 4 * g + r, p.M - 1)];
  const int n = n0 + 16 * j + cl;
  const int nc = min(n, p.N - 1);
  const float sw = p.w_scale[nc];
  const float bj = p.bias ? p.bias[nc] : 0.0f;
  if (p.acc_out) {
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + 16 * i + 4 * g + r;
        if (m < p.M && n < p.N) p.acc_out[(int64_t)m * p.N + n] = fin[i][r] >> kKgShift;
      }
  }
  // bf16 y = fp32(acc) (s_j delta_t) + b_j, staged in LDS (after the partial sums) so that
  // the tile leaves in 16-byte row chunks
  uint8_t *out = lds + kKgPartLds;
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = 16 * i + 4 * g + r;
      const float v = (float)(fin[i][r] >> kKgShift) * (sw * dt[i][r]) + bj;
      *reinterpret_cast<uint16_t *>(out + row * kKgOutStride + (16 * j + cl) * 2) = (uint16_t)f32_to_bf16(v);
    }
  __syncthreads();
  constexpr int CPR = 16 * TJ / 8;  // 16-byte chunks per staged row
  for (int q = threadIdx.x; q < 16 * TI * CPR; q += 64 * KG) {
    const int row = q / CPR, ch = q % CPR;
    const int m = m0 + row, nn = n0 + ch * 8;
    if (m < p.M && nn < p.N)
      *reinterpret_cast<uint4 *>(p.y + (int64_t)m * p.ldy + nn) = *reinterpret_cast<const uint4 *>(out + row * kKgOutStride + ch * 16);
  }
}

// Canonical nibble codes [M][K/2] -> k-step major [K/128][M][64 B], 16 bytes per thread.
// Thread u takes 16-byte chunk c = 16 kq + u % 16 of row r = (u / 16) % M, kq = u / (16 M):
// a wave reads 4 rows x 256 contiguous bytes (whole cache lines) and writes, for each of
// the 4 k steps those bytes hold, 4 consecutive rows x 64 bytes (256 contiguous bytes).
// (Read as a quarter step per thread, the rows' cache lines were fetched twice.)
__global__ __launch_bounds__(256) void codes_kmajor_kernel(const uint8_t *__restrict__ src, uint8_t *__restrict__ dst,
                                                            int M, int K) {
  const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int cpr = K / 32;  // 16-byte chunks per row (4 per k step)
  const int64_t rowunits = (int64_t)M * 16;
  const int kq = (int)(u / rowunits);
  const int rem = (int)(u - (int64_t)kq * rowunits);
  const int r = rem >> 4;
  const int c = 16 * kq + (rem & 15);
  if (c >= cpr) return;
  const int ks = c >> 2;
  *reinterpret_cast<uint4 *>(dst + (int64_t)ks * 64 * M + (int64_t)r * 64 + (c & 3) * 16) =
      *reinterpret_cast<const uint4 *>(src + (int64_t)r * (K / 2) + (int64_t)c * 16);
}

}  // namespace

size_t kgroup_lds_bytes() { return kKgLds; }

hipError_t launch_gemm_kgroup(const KgParams &p, const uint8_t *a_canonical, uint8_t *a_kmajor, hipStream_t s,
                              bool go) {
  static std::atomic<uint64_t> attr{0};
  hipError_t e = allow_dynamic_lds(&gemm_kgroup_kernel, kKgLds, attr);
  if (e != hipSuccess || !go) return e;
  if (a_canonical) {
    const int64_t units = (int64_t)((p.K / 32 + 15) / 16) * p.M * 16;  // 16-chunk row groups, rounded up
    hipLaunchKernelGGL(codes_kmajor_kernel, dim3((unsigned)((units + 255) / 256)), dim3(256), 0, s, a_canonical,
                       a_kmajor, p.M, p.K);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int64_t tiles = ((int64_t)(p.M + 16 * kKgTI - 1) / (16 * kKgTI)) * ((p.N + 16 * kKgTJ - 1) / (16 * kKgTJ));
  hipLaunchKernelGGL(gemm_kgroup_kernel, dim3((unsigned)tiles), dim3(64 * kKgWaves), kKgLds, s, p);
  return hipGetLastError();
}

}  // namespace fq
