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
// Two GEMM kernels:
//   gemm_stream (M <= 64): streams the weights once; a workgroup owns 16, 32 or 64
//     output channels, a block of rows (all M, or 16 when the grid would be small) and
//     a slice of K (split again between up to 4 wave groups that add up in LDS); the
//     activation slice is staged to LDS in one batch.
//   gemm_tile (M > 64): 128 x 128 output tiles (64 x 128 when the larger tiles would
//     leave half the compute units idle) fed through a ring of LDS stages, with a
//     register-level software pipeline and an optional load-issuing fifth wave.
// When K is split across workgroups, each slice writes its raw INT32 tile to a
// partial buffer and a small epilogue kernel adds the slices (exact) and rescales;
// the kernel boundary orders the two, so no atomics or cache-wide fences are needed.
// Output tiles are staged through LDS so that global stores are 16-byte coalesced.
#include "fq_device.hpp"
#include "fq_launch.hpp"
#include <type_traits>


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
  int ksteps;        // k steps of 128 per K slice
  int32_t *partial;  // [slices][M][N] raw accumulators when K is split
  int order;         // tiled: bit 0 = tile ids run down the rows first; bit 1 = no XCD grouping
};

template <int BITS, int AFMT>
struct Fmt {
  static constexpr int arow = AFMT == kANibble ? 64 : 128;  // activation bytes per row per k step
  static constexpr int tb = tile_bytes(BITS);
  static constexpr int lb = lane_bytes(BITS);
  // acc = 2^shift * true sum
  static constexpr int shift = BITS == 8 ? 0 : (AFMT == kANibble ? 8 : 4);
};

// Weight operand of lane l for k-chunk c from one tile.
template <int BITS>
__device__ __forceinline__ v4i w_operand(const uint8_t *tile, int l, int c) {
  if constexpr (BITS == 4) {
    return widen8(*reinterpret_cast<const v2i *>(tile + l * 16 + c * 8));
  } else {
    return *reinterpret_cast<const v4i *>(tile + l * 32 + c * 16);
  }
}


// ---------------- output stage ----------------
//
// A wave holds 16 x 16 accumulator tiles in the MFMA layout (lane l: rows 4*(l/16)+r,
// column l%16).  The workgroup's whole R x C output tile is written to LDS first and
// then leaves in 16-byte row chunks: either the final bf16 y (eq. (8) rescale applied
// by the lane that owns the value) or the raw INT32 slice of a split K.

struct EpiParams {  // per-lane rescale factors, loaded before the main loop
  float sw, bj;
};

__device__ __forceinline__ float rescale(int acc_shifted, float sw, float dt, float bj) {
  return (float)acc_shifted * (sw * dt) + bj;
}

// Stage one wave's tile (rows row0 + 16 i + 4 g + r, cols col0 + 16 j + l%16) in LDS.
// mode_final: bf16 with rescale; else raw int32.
template <int TI, int TJ, int SHIFT, bool FINAL>
__device__ __forceinline__ void stage_tiles(uint8_t *lds, int C, const v4i (&acc)[TI][TJ], int row0,
                                            int col0, int lane, const float (&dt)[TI][4],
                                            const EpiParams (&ep)[TJ]) {
  const int g = lane >> 4, cl = lane & 15;
  const int stride = FINAL ? C * 2 + 16 : C * 4 + 16;
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = row0 + 16 * i + 4 * g + r, col = col0 + 16 * j + cl;
        if constexpr (FINAL) {
          const float v = rescale(acc[i][j][r] >> SHIFT, ep[j].sw, dt[i][r], ep[j].bj);
          *reinterpret_cast<uint16_t *>(lds + row * stride + col * 2) = (uint16_t)f32_to_bf16(v);
        } else {
          *reinterpret_cast<int32_t *>(lds + row * stride + col * 4) = acc[i][j][r];
        }
      }
}

// Copy the staged R x C tile (origin m0, n0) to global memory in 16-byte chunks.
template <bool FINAL>
__device__ __forceinline__ void store_staged(const uint8_t *lds, int R, int C, int m0, int n0,
                                             const GemmParams &p, int split, int nthreads) {
  const int stride = FINAL ? C * 2 + 16 : C * 4 + 16;
  const int cpr = FINAL ? C / 8 : C / 4;  // 16-byte chunks per row
  for (int q = threadIdx.x; q < R * cpr; q += nthreads) {
    const int row = q / cpr, ch = q % cpr;
    const int m = m0 + row;
    const int n = n0 + ch * (FINAL ? 8 : 4);
    if (m < p.M && n < p.N) {
      const uint4 v = *reinterpret_cast<const uint4 *>(lds + row * stride + ch * 16);
      if constexpr (FINAL)
        *reinterpret_cast<uint4 *>(p.y + (int64_t)m * p.ldy + n) = v;
      else
        *reinterpret_cast<uint4 *>(p.partial + ((int64_t)split * p.M + m) * p.N + n) = v;
    }
  }
}

// Raw accumulators for verification (acc_out != NULL): direct stores, not a fast path.
template <int TI, int TJ, int SHIFT>
__device__ __forceinline__ void store_acc_out(const GemmParams &p, const v4i (&acc)[TI][TJ],
                                              int m_base, int n_base, int lane) {
  const int g = lane >> 4, cl = lane & 15;
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m_base + 16 * i + 4 * g + r, n = n_base + 16 * j + cl;
        if (m < p.M && n < p.N) p.acc_out[(int64_t)m * p.N + n] = acc[i][j][r] >> SHIFT;
      }
}

template <int TI, int TJ>
__device__ __forceinline__ void load_epi(const GemmParams &p, int m_base, int n_base, int lane,
                                         float (&dt)[TI][4], EpiParams (&ep)[TJ]) {
  const int g = lane >> 4, cl = lane & 15;
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = min(m_base + 16 * i + 4 * g + r, p.M - 1);
      dt[i][r] = p.delta[m];
    }
#pragma unroll
  for (int j = 0; j < TJ; ++j) {
    const int n = min(n_base + 16 * j + cl, p.N - 1);
    ep[j].sw = p.w_scale[n];
    ep[j].bj = p.bias ? p.bias[n] : 0.0f;
  }
}

// ---------------- split-K epilogue ----------------
// Adds the K slices of the raw INT32 partials (exact, fixed order), divides out the
// widening scale and applies the eq. (8) rescale; 4 output columns per thread.  The loads
// of up to 8 slices and of the rescale factors are all issued before the first add, so a
// thread waits for one round trip rather than one per slice.
template <int SHIFT>
__global__ __launch_bounds__(256) void splitk_epilogue_kernel(GemmParams p, int slices) {
  const int cpr = p.N / 4;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)p.M * cpr) return;
  const int m = (int)(idx / cpr), n = (int)(idx % cpr) * 4;
  const float dt = p.delta[m];
  const float4 sw = *reinterpret_cast<const float4 *>(p.w_scale + n);
  const float4 bj = p.bias ? *reinterpret_cast<const float4 *>(p.bias + n) : make_float4(0.f, 0.f, 0.f, 0.f);
  const int4 *src = reinterpret_cast<const int4 *>(p.partial + (int64_t)m * p.N + n);
  const int64_t zs = (int64_t)p.M * p.N / 4;  // int4 stride between slices
  int a[4] = {0, 0, 0, 0};
  for (int z0 = 0; z0 < slices; z0 += 8) {
    int4 v[8];
#pragma unroll
    for (int z = 0; z < 8; ++z)
      if (z0 + z < slices) v[z] = src[(z0 + z) * zs];
#pragma unroll
    for (int z = 0; z < 8; ++z)
      if (z0 + z < slices) {
        a[0] += v[z].x; a[1] += v[z].y; a[2] += v[z].z; a[3] += v[z].w;
      }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) a[i] >>= SHIFT;
  if (p.acc_out) *reinterpret_cast<int4 *>(p.acc_out + (int64_t)m * p.N + n) = make_int4(a[0], a[1], a[2], a[3]);
  const uint32_t o0 = f32_to_bf16(rescale(a[0], sw.x, dt, bj.x)) | (f32_to_bf16(rescale(a[1], sw.y, dt, bj.y)) << 16);
  const uint32_t o1 = f32_to_bf16(rescale(a[2], sw.z, dt, bj.z)) | (f32_to_bf16(rescale(a[3], sw.w, dt, bj.w)) << 16);
  *reinterpret_cast<uint2 *>(p.y + (int64_t)m * p.ldy + n) = make_uint2(o0, o1);
}

// Waits until at most `later` ring stages of LPS loads each are still in flight.
template <int LPS, int MAXL>
__device__ __forceinline__ void wait_ring(int later) {
  static_assert(MAXL * LPS < 64, "vmcnt range");
  if constexpr (MAXL >= 4) { if (later >= 4) { wait_vmcnt<4 * LPS>(); return; } }
  if constexpr (MAXL >= 3) { if (later == 3) { wait_vmcnt<3 * LPS>(); return; } }
  if constexpr (MAXL >= 2) { if (later == 2) { wait_vmcnt<2 * LPS>(); return; } }
  if constexpr (MAXL >= 1) { if (later == 1) { wait_vmcnt<LPS>(); return; } }
  wait_vmcnt<0>();
}

// ---------------- streaming kernel (M <= 64) ----------------
//
// Workgroup = WC x WK waves (WC, WK = 1, 2 or 4): 16 WC output channels (one 16-channel
// tile per wave column) x MT 16-row tiles (row block blockIdx.z) x a K slice of WK * KT
// k steps; wave group kg takes KT consecutive steps.  Fewer wave columns spread a narrow projection's weights over more compute units.
// Every wave first issues the loads of all KT of its weight tiles into registers; the
// activation slice (MT * 16 rows) then goes to LDS with direct-to-LDS loads, all in
// flight at once.  The slice's 16-byte chunks are XOR-swizzled inside each row so that
// the 16 rows a wave reads at once hit distinct banks without padding (a direct-to-LDS
// wave instruction fills one contiguous KB).  The MFMA loop double-buffers its
// activation operands in registers, one k step ahead.  The WK groups add up through
// LDS and the 64-channel tile leaves through the LDS output stage.

template <int AROW>
__device__ __forceinline__ int slice_swizzle(int row) {
  // chunks per row; rows per 256 bytes of LDS when a row is shorter than that
  constexpr int CPR = AROW / 16;
  constexpr int RP = AROW >= 256 ? 1 : 256 / AROW;
  constexpr int MASK = CPR < 16 ? CPR - 1 : 15;
  return (row / RP) & MASK;
}

// Activation slice -> LDS with direct loads, swizzled 16-byte chunks.  Wave w fills the
// KBs [w IA, (w+1) IA), whole rows of the slice.  The swizzle of row kb RPK + lr splits
// into swz(kb RPK) ^ swz(lr), so a lane's offset is fixed up to one XOR with a
// wave-uniform value and the row pointer advances by a uniform stride.  Rows past M read
// the KB's first row and (KFULL false) chunks past the end of K read chunk 0: both reach
// only dropped results.  A KB holding only rows past M is not loaded.
template <int AROW, int IA, int SLICE_KB, bool KFULL>
__device__ __forceinline__ void stage_slice(const uint8_t *abase, int64_t lda, int M, int wave, int lane,
                                            int valid_cols, uint8_t *lds) {
  constexpr int CPR = AROW / 16;  // 16-byte chunks per row
  if constexpr (CPR >= 64) {
    // a KB is 1/KPR of one row: row uniform, lane chunk h 64 + (lane ^ swz(row))
    constexpr int KPR = CPR / 64;
    constexpr int RPW = IA / KPR;  // rows per wave
    static_assert(IA % KPR == 0, "a wave loads whole rows");
    const int row0 = wave * RPW;
    const uint8_t *rp = abase + (int64_t)row0 * lda;
#pragma unroll
    for (int rr = 0; rr < RPW; ++rr, rp += lda) {
      const int row = row0 + rr;
      if (row * KPR >= SLICE_KB || row >= M) break;
      const int x = lane ^ slice_swizzle<AROW>(row);
#pragma unroll
      for (int h = 0; h < KPR; ++h) {
        int col = h * 64 + x;
        if (!KFULL && col >= valid_cols) col = 0;
        load_to_lds16(rp + (uint32_t)(col * 16), lds + (row * KPR + h) * 1024);
      }
    }
  } else {
    // a KB holds RPK whole rows: lane -> row lr = lane / CPR, chunk pos = lane % CPR
    constexpr int RPK = 64 / CPR;
    const int lr = lane / CPR, pos = lane % CPR;
    const int px = pos ^ slice_swizzle<AROW>(lr);
    const int kb0 = wave * IA;
    const uint8_t *rp = abase + (int64_t)kb0 * RPK * lda;
    const uint32_t lro = (uint32_t)(lr * lda);
#pragma unroll
    for (int i = 0; i < IA; ++i, rp += RPK * lda) {
      const int kb = kb0 + i;
      const int row = kb * RPK;  // first row of the KB
      if (kb >= SLICE_KB || row >= M) break;
      int col = px ^ slice_swizzle<AROW>(row);
      if (!KFULL && col >= valid_cols) col = 0;
      const uint32_t ro = row + RPK <= M || lr < M - row ? lro : 0u;
      load_to_lds16(rp + (ro + (uint32_t)(col * 16)), lds + kb * 1024);
    }
  }
}

template <int BITS, int AFMT, int MT, int KT, int WK, int WC>
__global__ __launch_bounds__(64 * WC * WK) void gemm_stream_kernel(GemmParams p) {
  using F = Fmt<BITS, AFMT>;
  constexpr int NTHREADS = 64 * WC * WK;
  constexpr int NWAVES = WC * WK;
  constexpr int NCOL = 16 * WC;             // output channels per workgroup
  constexpr int LU4 = F::lb / 16;           // 16-byte loads per lane per weight tile
  constexpr int AROW = WK * KT * F::arow;   // activation bytes per row in the slice
  constexpr int ROWS = MT * 16;
  constexpr int CPR = AROW / 16;            // 16-byte chunks per row
  constexpr int SLICE_KB = ROWS * AROW / 1024;
  constexpr int IA = (SLICE_KB + NWAVES - 1) / NWAVES;  // direct-to-LDS loads per wave
  static_assert(ROWS * AROW % 1024 == 0, "slice must be whole KB");
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: scalar index math
  const int wn = wave % WC, kg = wave / WC;
  const int nblk = blockIdx.x;
  const int split = blockIdx.y;
  const int nsplit = gridDim.y;
  const int ktot = p.K / kTileK;
  const int slice_begin = split * WK * KT;
  const int ks_begin = slice_begin + kg * KT;
  const int nk = max(0, min(KT, ktot - ks_begin));
  const int ntile = nblk * WC + wn;
  const bool n_ok = ntile * 16 < p.N;
  const int m0 = blockIdx.z * ROWS;      // first row of this workgroup's row block
  const int mz = min(ROWS, p.M - m0);    // its rows (>= 1)

  // 1. activation slice -> LDS (see stage_slice)
  {
    const uint8_t *abase = p.a + (int64_t)m0 * p.lda + (int64_t)slice_begin * F::arow;
    const int valid_cols = min(WK * KT, ktot - slice_begin) * (F::arow / 16);
    if (valid_cols == CPR)
      stage_slice<AROW, IA, SLICE_KB, true>(abase, p.lda, mz, wave, lane, valid_cols, lds);
    else
      stage_slice<AROW, IA, SLICE_KB, false>(abase, p.lda, mz, wave, lane, valid_cols, lds);
  }

  // rescale factors of the row tiles this wave group finishes (i = kg mod WK)
  float dt[MT][4];
  EpiParams ep[1];
  if (nsplit == 1) {
    const int g = lane >> 4, cl = lane & 15;
#pragma unroll
    for (int i = 0; i < MT; ++i)
      if (i % WK == kg)
#pragma unroll
        for (int r = 0; r < 4; ++r) dt[i][r] = p.delta[min(m0 + 16 * i + 4 * g + r, p.M - 1)];
    const int n = min(ntile * 16 + cl, p.N - 1);
    ep[0].sw = p.w_scale[n];
    ep[0].bj = p.bias ? p.bias[n] : 0.0f;
  }

  // 2. then all weight tiles of this wave, in k order.  Vector loads complete in issue
  // order, so once everything but the weights has landed the slice is in LDS, and the
  // MFMAs of step kt start when tile kt arrives, while later tiles are still streaming.
  // Loads are unconditional (a step past the end of K re-reads the last tile, never
  // used) so that no branch sits between them.
  sched_wall();
  uint4 wreg[KT][LU4];
  const uint8_t *wtile = p.w + (int64_t)min(ntile, p.N / 16 - 1) * ktot * F::tb + lane * F::lb;
  if (nk == KT) {
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int u = 0; u < LU4; ++u)
        wreg[kt][u] = reinterpret_cast<const uint4 *>(wtile + (int64_t)(ks_begin + kt) * F::tb)[u];
  } else {
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int u = 0; u < LU4; ++u)
        wreg[kt][u] = reinterpret_cast<const uint4 *>(wtile + (int64_t)min(ks_begin + kt, ktot - 1) * F::tb)[u];
  }

  sched_wall();
  wait_vmcnt<KT * LU4>();
  lds_barrier();

  // 3. MFMA over the wave's k steps, activation operands one step ahead in registers
  v4i acc[MT][1];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i][0] = v4i{0, 0, 0, 0};
  const int r16 = lane & 15, g = lane >> 4;
  auto load_a = [&](int kt, v4i (&dst)[MT][2]) {
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const int row = i * 16 + r16;
      const uint8_t *rp = lds + row * AROW;
      const int swz = slice_swizzle<AROW>(row);
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        if constexpr (AFMT == kANibble) {
          const int chunk = (kg * KT + kt) * 4 + g;  // 64-byte rows per step: 4 chunks
          dst[i][c] = widen8(*reinterpret_cast<const v2i *>(rp + ((chunk ^ swz) * 16) + c * 8));
        } else {
          const int chunk = (kg * KT + kt) * 8 + 2 * g + c;
          dst[i][c] = *reinterpret_cast<const v4i *>(rp + ((chunk ^ swz) * 16));
        }
      }
    }
  };
  v4i abuf[2][MT][2];
  load_a(0, abuf[0]);
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) {
    if (kt + 1 < KT) load_a(kt + 1, abuf[(kt + 1) & 1]);
    if (kt < nk) {
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        v4i bop;
        if constexpr (BITS == 4) {
          v2i h;
          h.x = (int)(c == 0 ? wreg[kt][0].x : wreg[kt][0].z);
          h.y = (int)(c == 0 ? wreg[kt][0].y : wreg[kt][0].w);
          bop = widen8(h);
        } else {
          const uint4 t = wreg[kt][c];
          bop = v4i{(int)t.x, (int)t.y, (int)t.z, (int)t.w};
        }
#pragma unroll
        for (int i = 0; i < MT; ++i) acc[i][0] = mfma16x16x64(abuf[kt & 1][i][c], bop, acc[i][0]);
      }
    }
  }

  // 4. every wave group leaves its tiles in LDS; wave group kg adds up row tiles
  // i = kg mod WK (exact integer sums) and stages them; the tile leaves through the stage
  __syncthreads();  // the activation slice is no longer read
  uint8_t *stage = lds + (WK > 1 ? (size_t)WK * WC * MT * 64 * 16 : 0);
  if constexpr (WK > 1) {
    v4i *red = reinterpret_cast<v4i *>(lds);
#pragma unroll
    for (int i = 0; i < MT; ++i) red[((kg * WC + wn) * MT + i) * 64 + lane] = acc[i][0];
    __syncthreads();
#pragma unroll
    for (int i = 0; i < MT; ++i)
      if (i % WK == kg) {
        v4i t = red[(wn * MT + i) * 64 + lane];
#pragma unroll
        for (int g2 = 1; g2 < WK; ++g2) t += red[((g2 * WC + wn) * MT + i) * 64 + lane];
        acc[i][0] = t;
      }
  }
#pragma unroll
  for (int i = 0; i < MT; ++i)
    if (i % WK == kg) {
      const v4i t[1][1] = {{acc[i][0]}};
      const float d[1][4] = {{dt[i][0], dt[i][1], dt[i][2], dt[i][3]}};
      if (p.acc_out && nsplit == 1 && n_ok) store_acc_out<1, 1, F::shift>(p, t, m0 + 16 * i, ntile * 16, lane);
      if (nsplit == 1)
        stage_tiles<1, 1, F::shift, true>(stage, NCOL, t, 16 * i, wn * 16, lane, d, ep);
      else
        stage_tiles<1, 1, F::shift, false>(stage, NCOL, t, 16 * i, wn * 16, lane, d, ep);
    }
  __syncthreads();
  if (nsplit == 1)
    store_staged<true>(stage, ROWS, NCOL, m0, nblk * NCOL, p, 0, NTHREADS);
  else
    store_staged<false>(stage, ROWS, NCOL, m0, nblk * NCOL, p, split, NTHREADS);
}

template <int BITS, int AFMT, int MT, int KT, int WK, int WC>
static size_t stream_lds_bytes() {
  const size_t slice = (size_t)MT * 16 * (WK * KT * Fmt<BITS, AFMT>::arow);
  const size_t red = WK > 1 ? (size_t)WK * WC * MT * 64 * 16 : 0;
  const size_t out = red + (size_t)MT * 16 * (16 * WC * 4 + 16);
  return slice > out ? slice : out;
}

// ---------------- streaming kernel, one K range per wave (M <= 64, long K, INT4) ----------------
//
// Workgroup = WK waves, NCW 16-channel tiles (16 NCW output channels), one 16-row block
// (blockIdx.z) and a K slice of WK * KT steps (blockIdx.y).  Wave kg owns the steps
// [kg KT, (kg + 1) KT) of the slice for every tile of the workgroup: it stages its own part
// of the activation slice (16 rows x KT steps of nibble codes) in its own LDS region with
// direct-to-LDS loads (16-byte chunks XOR-swizzled by row, as in the kernel above), then
// loads its NCW x KT weight tiles into registers, and multiplies as soon as its own part
// has landed: no wave waits for another before the final sum, and each widened activation
// operand serves all NCW tiles.  Steps past K find zero activation codes in LDS.  At the
// end the waves' sums add up through LDS (exact integers) and wave i rescales tile i.
template <int KT, int WK, int NCW>
__global__ __launch_bounds__(64 * WK) void gemm_stream_kw_kernel(GemmParams p) {
  using F = Fmt<4, kANibble>;
  constexpr int AROW = KT * F::arow;            // bytes of one row in a wave's part
  constexpr int PART = 16 * AROW;               // a wave's part: 16 rows
  constexpr int KPR = AROW / 1024;              // direct-to-LDS loads (1 KB each) per row
  constexpr int NCOL = 16 * NCW;
  static_assert(AROW % 1024 == 0 && NCW <= WK, "whole-KB rows; one finishing wave per tile");
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];

  const int lane = threadIdx.x & 63;
  const int kg = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nblk = blockIdx.x, split = blockIdx.y, nsplit = gridDim.y;
  const int ktot = p.K / kTileK;
  const int ks_begin = split * WK * KT + kg * KT;
  const int nk = max(0, min(KT, ktot - ks_begin));
  const int m0 = blockIdx.z * 16;
  const int mz = min(16, p.M - m0);  // rows of the block (>= 1)
  uint8_t *part = lds + kg * PART;

  // rescale factors first (every wave loads them; wave i < NCW uses those of tile i), so
  // that only the weight tiles are issued after the slice
  float dt[1][4];
  EpiParams ep[1];
  const int ntile_own = nblk * NCW + (kg < NCW ? kg : 0);
  load_epi<1, 1>(p, m0, ntile_own * 16, lane, dt, ep);

  // 1. this wave's part of the slice: row r < mz, KT * 4 chunks, chunk c at unit c ^ r.
  // Units of chunks past K are written with zeros instead (a partial last slice), so their
  // MFMAs add nothing and the loop below needs no masking
  sched_wall();
  {
    const uint8_t *abase = p.a + (int64_t)m0 * p.lda + (int64_t)ks_begin * F::arow;
    const int valid = nk * (F::arow / 16);
    if (valid == KT * 4) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if (r >= mz) break;
#pragma unroll
        for (int h = 0; h < KPR; ++h)
          load_to_lds16(abase + (int64_t)r * p.lda + (uint32_t)((((h * 64 + lane) ^ r)) * 16),
                        part + r * AROW + h * 1024);
      }
    } else {
      for (int r = 0; r < mz; ++r)
        for (int h = 0; h < KPR; ++h) {
          const int c = (h * 64 + lane) ^ r;
          if (c < valid)
            load_to_lds16(abase + (int64_t)r * p.lda + (uint32_t)(c * 16), part + r * AROW + h * 1024);
          else
            lds_write16_untracked(part + r * AROW + (h * 64 + lane) * 16, make_uint4(0u, 0u, 0u, 0u));
        }
    }
  }

  // 2. the weight tiles of every tile of the workgroup, in k order (steps past K re-read
  // the last step, never used with a nonzero operand), as untracked loads: step kt waits
  // for exactly its own tiles below.  The compiler takes an untracked load's register as
  // written at once, so no control flow may separate the loads from their waits: at a
  // join the register allocator may copy a register whose data has not landed.
  sched_wall();
  v4i wreg[NCW][KT];
  const uint8_t *wt[NCW];
#pragma unroll
  for (int i = 0; i < NCW; ++i)
    wt[i] = p.w + (int64_t)min(nblk * NCW + i, p.N / 16 - 1) * ktot * F::tb + lane * F::lb;
#pragma unroll
  for (int kt = 0; kt < KT; ++kt)
#pragma unroll
    for (int i = 0; i < NCW; ++i)
      wreg[i][kt] = global_load16_untracked(wt[i] + (int64_t)min(ks_begin + kt, ktot - 1) * F::tb);
  sched_wall();

  // 3. MFMA over the wave's steps once this wave's slice loads have landed (they were
  // issued before the weights, and loads complete in issue order).  The slice is read with
  // untracked LDS reads: the compiler cannot tell this wave's region from the ones other
  // waves' direct-to-LDS loads are filling.  Each read is waited for (lgkmcnt) before its
  // value is used, one step ahead of the MFMAs; step kt waits (vmcnt) until only the
  // tiles of later steps are in flight.
  wait_vmcnt<NCW * KT>();
  const int r16 = lane & 15, g = lane >> 4;
  const uint8_t *rp = part + r16 * AROW;
  auto load_a = [&](int kt) -> v4i {
    return __builtin_bit_cast(v4i, lds_read16_untracked(rp + (((kt * 4 + g) ^ r16) * 16)));
  };
  v4i acc[2][NCW];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int i = 0; i < NCW; ++i) acc[h][i] = v4i{0, 0, 0, 0};
  v4i araw = load_a(0);
  auto step = [&](auto kt_c) {
    constexpr int kt = decltype(kt_c)::value;
    sched_wall();
    if constexpr (NCW == 2)
      vm_wait_on<(KT - 1 - kt) * NCW>(wreg[0][kt], wreg[1][kt]);
    else
      vm_wait_on<(KT - 1 - kt) * NCW>(wreg[0][kt]);
    lgkm_wait_on(araw);
    const v4i cur = araw;
    if constexpr (kt + 1 < KT) araw = load_a(kt + 1);
    const v4i a0 = widen8(v2i{cur.x, cur.y});
    const v4i a1 = widen8(v2i{cur.z, cur.w});
#pragma unroll
    for (int i = 0; i < NCW; ++i) {
      const v4i w = wreg[i][kt];
      acc[0][i] = mfma16x16x64(a0, widen8(v2i{w.x, w.y}), acc[0][i]);
      acc[1][i] = mfma16x16x64(a1, widen8(v2i{w.z, w.w}), acc[1][i]);
    }
  };
  static_for<KT>(step);

  // 4. the waves' sums add up through LDS (the slice is no longer read); wave i < NCW
  // finishes tile i
  __syncthreads();
  v4i *red = reinterpret_cast<v4i *>(lds);
#pragma unroll
  for (int i = 0; i < NCW; ++i) red[(kg * NCW + i) * 64 + lane] = acc[0][i] + acc[1][i];
  __syncthreads();
  uint8_t *stage = lds + (size_t)WK * NCW * 64 * 16;
  if (kg < NCW) {
    v4i t = red[kg * 64 + lane];
#pragma unroll
    for (int w = 1; w < WK; ++w) t += red[(w * NCW + kg) * 64 + lane];
    const v4i tt[1][1] = {{t}};
    if (p.acc_out && nsplit == 1) store_acc_out<1, 1, F::shift>(p, tt, m0, ntile_own * 16, lane);
    if (nsplit == 1)
      stage_tiles<1, 1, F::shift, true>(stage, NCOL, tt, 0, kg * 16, lane, dt, ep);
    else
      stage_tiles<1, 1, F::shift, false>(stage, NCOL, tt, 0, kg * 16, lane, dt, ep);
  }
  __syncthreads();
  if (nsplit == 1)
    store_staged<true>(stage, 16, NCOL, m0, nblk * NCOL, p, 0, 64 * WK);
  else
    store_staged<false>(stage, 16, NCOL, m0, nblk * NCOL, p, split, 64 * WK);
}

template <int KT, int WK, int NCW>
static constexpr size_t stream_kw_lds_bytes() {
  constexpr size_t slice = (size_t)WK * 16 * KT * 64;
  constexpr size_t fin = (size_t)WK * NCW * 64 * 16 + 16 * (16 * NCW * 4 + 16);
  return slice > fin ? slice : fin;
}

// ---------------- tiled kernel (M > 64) ----------------
//
// BM x BN output tile per workgroup (2 x 2 waves), k steps of 128 channels.  Operands
// move HBM/L2 -> LDS with gfx950's direct-to-LDS loads (global_load_lds_dwordx4: each
// wave instruction fills one contiguous KB of LDS, no registers involved) into a ring of
// STAGES buffers, so loads for later k steps are in flight while step ks is multiplied.
// Activation rows are XOR-swizzled in 16-byte chunks so the 16 rows a wave reads at
// once fall into distinct LDS banks; weight tiles keep their lane-contiguous
// kernel-native layout, which is already conflict-free.
//
// The loop is software-pipelined at the register level: after the one barrier per k step,
// the whole next step's operands are read from LDS into a second register set while the
// current step's 32 MFMAs run, one read per two MFMAs.  Every read is 16 bytes per lane
// (an 8-byte nibble operand brings both 64-wide chunks at once): 8-byte reads at a 16-byte
// lane stride put two lanes on every bank and doubled the LDS time.  With at most one
// workgroup per compute unit, a fifth wave issues the ring loads.  Measured at M = 816:
// ~1000-1150 cycles per k step against 512 of MFMA issue; removing the ring loads changes
// nothing, removing the LDS operand reads leaves ~700, the MFMA + widening loop alone ~660.

template <int AFMT>
__device__ __forceinline__ int a_swizzle(int row) {
  return AFMT == kANibble ? ((row >> 1) & 3) : ((row >> 1) & 7);
}

// Optional logical tile order that keeps consecutive tiles (same activation rows) on one
// XCD: the hardware hands workgroup p to XCD p % 8.
__device__ __forceinline__ int xcd_remap(int p, int total) {
  if ((total & 7) != 0) return p;
  return (p & 7) * (total >> 3) + (p >> 3);
}

template <int BITS, int AFMT, int BM, int BN, int STAGES, int LW>
__global__ __launch_bounds__(256 + 64 * LW) void gemm_tile_kernel(GemmParams p) {
  using F = Fmt<BITS, AFMT>;
  constexpr int CPR = F::arow / 16;
  constexpr int NT = BN / 16;
  constexpr int ASTAGE = BM * F::arow;
  constexpr int BSTAGE = NT * F::tb;
  constexpr int STAGE = ASTAGE + BSTAGE;
  constexpr int NLW = LW ? 1 : 4;                // waves that issue the ring loads
  constexpr int IA = BM * CPR / (64 * NLW);
  constexpr int IB = BSTAGE / 1024 / NLW;
  constexpr int LPS = IA + IB;
  constexpr int TM = BM / 32, TN = NT / 2;       // 2 x 2 waves of 64 x 64
  static_assert(IA >= 1 && IB >= 1, "tile too small");
  using AOp = typename std::conditional<AFMT == kANibble, v2i, v4i>::type;
  using BOp = typename std::conditional<BITS == 4, v2i, v4i>::type;
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = (wave >> 1) & 1, wn = wave & 1;
  const int lw = LW ? 0 : wave;                  // index among the loading waves
  const int ntiles_n = (p.N + BN - 1) / BN;
  const int ntiles_m = (p.M + BM - 1) / BM;
  const int total = ntiles_n * ntiles_m * gridDim.y;
  const int lin = blockIdx.x + blockIdx.y * gridDim.x;
  const int logical = (p.order & 2) ? lin : xcd_remap(lin, total);
  const int tile_id = logical % (ntiles_n * ntiles_m);
  const int split = logical / (ntiles_n * ntiles_m);
  const int nsplit = gridDim.y;
  const int tn = (p.order & 1) ? tile_id / ntiles_m : tile_id % ntiles_n;
  const int tm = (p.order & 1) ? tile_id % ntiles_m : tile_id / ntiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const int ktot = p.K / kTileK;
  const int ks_begin = split * p.ksteps;
  const int nk = min(p.ksteps, ktot - ks_begin);

  const uint8_t *asrc[IA];
#pragma unroll
  for (int i = 0; i < IA; ++i) {
    const int slot = (lw * IA + i) * 64 + lane;
    const int row = slot / CPR, pos = slot % CPR;
    const int logical_chunk = pos ^ a_swizzle<AFMT>(row);
    const int grow = min(m0 + row, p.M - 1);
    asrc[i] = p.a + (int64_t)grow * p.lda + (int64_t)ks_begin * F::arow + logical_chunk * 16;
  }
  const uint8_t *bsrc[IB];
#pragma unroll
  for (int i = 0; i < IB; ++i) {
    const int j = lw * IB + i;                   // KB index inside the weight stage
    const int t = j / (F::tb / 1024), h = j % (F::tb / 1024);
    const int nb = min(n0 / 16 + t, p.N / 16 - 1);
    bsrc[i] = p.w + ((int64_t)nb * ktot + ks_begin) * F::tb + h * 1024 + lane * 16;
  }
  // Loads k step ks into its ring slot.  Past the slice end the source is clamped to the last
  // step: those loads only fill a slot that is never read again, and they keep the number of
  // loads in flight constant so that one vmcnt wait fits every step.
  auto issue = [&](int ks) {
    uint8_t *st = lds + (ks % STAGES) * STAGE;
    const int kc = min(ks, nk - 1);
#pragma unroll
    for (int i = 0; i < IA; ++i)
      load_to_lds16(asrc[i] + (int64_t)kc * F::arow, st + (lw * IA + i) * 1024);
#pragma unroll
    for (int i = 0; i < IB; ++i)
      load_to_lds16(bsrc[i] + (int64_t)kc * F::tb, st + ASTAGE + (lw * IB + i) * 1024);
  };

  // per-lane LDS byte offsets of this wave's operands inside a stage, chunk 0
  int aoff[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int row = wm * (BM / 2) + i * 16 + (lane & 15);
    const int g = lane >> 4;
    aoff[i] = AFMT == kANibble ? row * F::arow + ((g ^ a_swizzle<AFMT>(row)) * 16)
                               : row * F::arow + (((2 * g) ^ a_swizzle<AFMT>(row)) * 16);
  }
  const int boff = ASTAGE + wn * TN * F::tb + lane * (BITS == 4 ? 16 : 32);

  // Raw operands of a whole k step (both 64-wide chunks); two sets, for even and odd steps.
  // Every LDS read is 16 bytes per lane: a nibble operand brings both chunks' 8-byte halves
  // at once (lanes 16 bytes apart, conflict-free; 8-byte reads of one half would put two
  // lanes on every bank), an int8 operand one chunk.
  constexpr int RA = AFMT == kANibble ? 1 : 2;   // activation reads per row tile per step
  constexpr int RB = BITS == 4 ? 1 : 2;          // weight reads per column tile per step
  v4i ar[2][RA][TM];
  v4i br[2][RB][TN];
  constexpr int NREAD = RA * TM + RB * TN;       // LDS reads per wave per step
  // read r of step ks into `set`: activation reads first, then weight reads
  auto read_one = [&](int set, int ks, int r) {
    const uint8_t *st = lds + (ks % STAGES) * STAGE;
    if (r < RA * TM) {
      const int c = r / TM, i = r % TM;
      // int8 rows: chunk 1 is the next 16-byte chunk, whose swizzled position is chunk 0's ^ 16
      ar[set][c][i] = *reinterpret_cast<const v4i *>(st + (aoff[i] ^ (c * 16)));
    } else {
      const int q = r - RA * TM, c = q / TN, j = q % TN;
      br[set][c][j] = *reinterpret_cast<const v4i *>(st + boff + j * F::tb + c * 16);
    }
  };
  // operands of chunk c from a raw set
  auto a_op = [&](int set, int c, int i) -> v4i {
    if constexpr (AFMT == kANibble) {
      const v4i &t = ar[set][0][i];
      return widen8(c == 0 ? v2i{t.x, t.y} : v2i{t.z, t.w});
    } else {
      return ar[set][c][i];
    }
  };
  auto b_op = [&](int set, int c, int j) -> v4i {
    if constexpr (BITS == 4) {
      const v4i &t = br[set][0][j];
      return widen8(c == 0 ? v2i{t.x, t.y} : v2i{t.z, t.w});
    } else {
      return br[set][c][j];
    }
  };

  v4i acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = v4i{0, 0, 0, 0};
  // One k step: after the step barrier (stage ks + 1 has landed; every wave finished
  // reading stage ks, whose slot the next issue refills), step ks is multiplied from one
  // register set while step ks + 1 is read into the other.  The reads are spread one per
  // two MFMAs: issued in a burst, the four waves' reads fill the compute unit's LDS queue
  // and stall the in-order wave, MFMA issue included.
  auto step = [&](int cur, int ks, bool more) {
    if (more) {
      if (!LW) wait_vmcnt<(STAGES - 2) * LPS>();
      lds_barrier();
      if (!LW) issue(ks + STAGES);
    }
    int r = 0;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      v4i wa[TM];
#pragma unroll
      for (int i = 0; i < TM; ++i) wa[i] = a_op(cur, c, i);
      // weight tile outer: one widened weight operand live at a time
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const v4i wb = b_op(cur, c, j);
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          __builtin_amdgcn_sched_barrier(0);
          acc[i][j] = mfma16x16x64(wa[i], wb, acc[i][j]);
          if (more && ((j * TM + i) & 1) == 1 && r < NREAD) {
            __builtin_amdgcn_sched_barrier(0);
            read_one(cur ^ 1, ks + 1, r);
            ++r;
          }
        }
      }
    }
    // smaller tiles have fewer MFMAs per step than reads (int8 operands): the rest now
    if (more) {
#pragma unroll
      for (; r < NREAD; ++r) {
        __builtin_amdgcn_sched_barrier(0);
        read_one(cur ^ 1, ks + 1, r);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  if (LW && wave == 4) {
    // loader wave: keeps the ring full; one barrier per step, like the MFMA waves
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s) issue(s);
    wait_vmcnt<(STAGES - 2) * LPS>();
    lds_barrier();
    issue(STAGES - 1);
    for (int ks = 0; ks < nk - 1; ++ks) {
      wait_vmcnt<(STAGES - 2) * LPS>();
      lds_barrier();
      issue(ks + STAGES);
    }
  } else {
    if (!LW) {
#pragma unroll
      for (int s = 0; s < STAGES - 1; ++s) issue(s);
      wait_vmcnt<(STAGES - 2) * LPS>();
    }
    lds_barrier();
#pragma unroll
    for (int r = 0; r < NREAD; ++r) read_one(0, 0, r);
    if (!LW) issue(STAGES - 1);
    int ks = 0;
    for (; ks + 2 < nk; ks += 2) {
      step(0, ks, true);
      step(1, ks + 1, true);
    }
    if (ks + 1 < nk) {
      step(0, ks, true);
      step(1, ks + 1, false);
    } else {
      step(0, ks, false);
    }
  }

  const int m_wave = m0 + wm * (BM / 2), n_wave = n0 + wn * (BN / 2);
  const bool mma_wave = !(LW && wave == 4);
  const bool out_wave = mma_wave;  // the loader wave holds no results
  float dt[TM][4];
  EpiParams ep[TN];
  if (nsplit == 1 && out_wave) load_epi<TM, TN>(p, m_wave, n_wave, lane, dt, ep);
  __syncthreads();  // also drains the ring's trailing loads before the LDS is reused
  if (out_wave) {
    if (nsplit == 1) {
      if (p.acc_out) store_acc_out<TM, TN, F::shift>(p, acc, m_wave, n_wave, lane);
      stage_tiles<TM, TN, F::shift, true>(lds, BN, acc, wm * (BM / 2), wn * (BN / 2), lane, dt, ep);
    } else {
      stage_tiles<TM, TN, F::shift, false>(lds, BN, acc, wm * (BM / 2), wn * (BN / 2), lane, dt, ep);
    }
  }
  __syncthreads();
  if (nsplit == 1)
    store_staged<true>(lds, BM, BN, m0, n0, p, 0, 256 + 64 * LW);
  else
    store_staged<false>(lds, BM, BN, m0, n0, p, split, 256 + 64 * LW);
}

template <int BITS, int AFMT, int BM, int BN, int STAGES>
static constexpr size_t tile_lds_bytes() {
  // ring; then the k-group hand-over (BM * BN int32) or the staged output, one after the other
  constexpr size_t ring = (size_t)STAGES * (BM * Fmt<BITS, AFMT>::arow + BN / 16 * Fmt<BITS, AFMT>::tb);
  constexpr size_t out = (size_t)BM * (BN * 4 + 16);
  return ring > out ? ring : out;
}

// ----------------------------------------------------------------------------------------
// planning and launch

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, int bits, bool kmajor_codes) {
  GemmPlan pl{};
  const int ktot = (int)(K / kTileK);
  if (M <= 64) {
    // Weight streaming.  A workgroup stages its activation slice (the rows of its row
    // block, the slice's k steps) in LDS once for its wave columns of 16 channels; 4 wave groups of kt steps
    // split the slice and add up in LDS.  A slice holds as many k steps as LDS allows
    // (32 of nibble codes, 16 of int8 codes: 128 KB for 64 rows), so K up to 4096 (W4A4)
    // needs no split-K epilogue kernel.  Then the fewest wave columns that keep the grid
    // within one workgroup per compute unit, which spreads a narrow projection's weight
    // stream over more compute units.  These shapes measured fastest at M = 50.
    pl.kind = 0;
    pl.mt = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
    if (ktot < 4) {
      pl.wk = 1;
      pl.kt = ktot >= 2 ? 2 : 1;
    } else {
      const int cap = bits == 4 ? 32 : 16;
      const int per = ktot < cap ? ktot : cap;  // k steps per slice
      pl.wk = 4;
      pl.kt = per <= 4 ? 1 : (per <= 8 ? 2 : (per <= 16 ? 4 : 8));
    }
    pl.ksteps = pl.kt * pl.wk;
    pl.splits = (ktot + pl.ksteps - 1) / pl.ksteps;
    pl.wc = 4;
    for (int wc = 1; wc < 4; wc *= 2)
      if (((N + 16 * wc - 1) / (16 * wc)) * pl.splits <= 256) {
        pl.wc = wc;
        break;
      }
    pl.tiles = (N + 16 * pl.wc - 1) / (16 * pl.wc);
    // A grid that fills at most half the compute units also splits the rows: one 16-row
    // tile per workgroup, so each workgroup widens a quarter of the activation codes
    // (M = 50) and four times as many compute units share the weight stream.  Sibling
    // row blocks read the same weights; when the tile count is a multiple of 8 they run
    // on one XCD (workgroups go round-robin over the 8 XCDs) and its L2 serves the repeats.
    pl.rb = 1;
    if (M > 16 && pl.tiles * pl.splits <= 128) {
      pl.mt = 1;
      pl.rb = (int)((M + 15) / 16);
    }
    // Long K (nibble codes, K >= 16384): one K range per wave (gemm_stream_kw_kernel),
    // 16-row blocks, 8 waves of 16 steps each (the whole of K = 16384 in one slice, 128 KB
    // of LDS, no split-K epilogue).  32 output channels per workgroup when that grid still
    // holds >= 256 workgroups, else 16; up to 32 rows the plan needs a grid of >= 128
    // workgroups to keep the weight stream wide enough.  Each row block streams the weights
    // again (its siblings share them through the XCD's L2); each wave waits only for its
    // own slice part.  Measured at M = 50, K 16384 -> N 2048: 11.1 us with four wave groups
    // sharing one slice, 9.5 us this way.  Shorter K stays on the kernel above (site D of
    // the action expert, K 4096: 3.3 against 3.5 us this way).
    if (bits == 4 && ktot >= 128) {
      const int rb = (int)((M + 15) / 16);
      const int splits = (ktot + 127) / 128;
      int ncw = 2;
      if (((N + 31) / 32) * rb * splits < 256) ncw = 1;
      const int64_t tiles = (N + 16 * ncw - 1) / (16 * ncw);
      if (M > 32 || tiles * rb * splits >= 128) {
        pl.kind = 2;
        pl.mt = 1;
        pl.rb = rb;
        pl.wk = 8;
        pl.kt = 16;
        pl.ksteps = 128;
        pl.splits = splits;
        pl.wc = ncw;
        pl.tiles = tiles;
      }
    }
  } else {
    // INT4 at long K where 128 x 128 tiles would not fill the chip without splitting K (a
    // few hundred to ~1000 rows, N ~ 2048): 128 x 64 tiles with the K range split across
    // the workgroup's four waves instead (gemm_kgroup_kernel, no partial buffer, no second
    // kernel).  Measured at M = 816, K 16384 -> N 2048 against the split 128 x 128 plan:
    // 31 against 43 us on one GPU (fed k-step-major codes).  Short K (fewer than 64 steps
    // per tile) and grids of fewer than 160 tiles stay on the LDS-ring kernel below.
    // With k-step-major codes for free (no conversion kernel), grids of up to 1023 such
    // tiles at K >= 16384 take it too: K 16384 -> N 2048 at M = 1600 / 2048 / 3072 in
    // 56.5 / 58.3 / 85.4 against 63.3 / 64.1 / 103.8 us on the LDS-ring kernel; at 1024
    // tiles (M = 4096) the two measured the same and at K = 8192 the ring kernel led.
    // Byte offsets into the codes and the weights are 32-bit in that kernel.
    if (bits == 4 && ktot >= 64 && M * K / 2 < (int64_t(1) << 31) && N * K / 2 < (int64_t(1) << 31)) {
      const int64_t t128 = ((M + 127) / 128) * ((N + 127) / 128);
      const int64_t tkg = ((M + 127) / 128) * ((N + 63) / 64);
      const bool wide = kmajor_codes && ktot >= 128 && tkg < 1024;
      if ((t128 < 200 || wide) && tkg >= 160) {
        pl.kind = 3;
        pl.tiles = tkg;
        pl.splits = 1;
        pl.ksteps = ktot;
        pl.partial_bytes = 0;
        return pl;
      }
    }
    pl.kind = 1;
    // K slices: split a grid of fewer than 200 tiles while each slice keeps >= 32 steps
    auto slices = [&](int64_t tiles) {
      int64_t s = 1;
      while (tiles * s < 200 && s < 4 && ktot / (s * 2) >= 32) s *= 2;
      return s;
    };
    // 128 x 128 tiles; 64 x 128 when the 128-row grid, split included, would leave half
    // the compute units idle (measured: M = 256, K 16384 -> N 2048 in 19.0 against
    // 24.0 us; M = 816, K 2048 -> N 2048 in 9.7 against 13.1 us; at M = 816,
    // K 16384 -> N 2048 the split 128-row grid stays ahead, 39.7 against 43.1 us)
    pl.bm = 128;
    pl.bn = 128;
    {
      const int64_t t128 = ((M + 127) / 128) * ((N + 127) / 128);
      if (t128 * slices(t128) <= 128) pl.bm = 64;
    }
    const int64_t tiles = ((M + pl.bm - 1) / pl.bm) * ((N + pl.bn - 1) / pl.bn);
    int64_t s = slices(tiles);
    pl.ksteps = (int)((ktot + s - 1) / s);
    pl.splits = (ktot + pl.ksteps - 1) / pl.ksteps;
    pl.tiles = tiles;
    // One workgroup per compute unit: 4 ring stages, and for INT4 a fifth wave that issues
    // the ring loads so the MFMA waves never stall on load issue (INT8 tiles need twice
    // the loads per step, more than one wave issues in time: there the MFMA waves load,
    // 2-7% faster measured at M = 130 .. 816).  Two per compute unit: 3 stages, no
    // loader wave; the second workgroup already overlaps the loads.
    const bool lone = tiles * pl.splits <= 256;
    pl.loader = lone && bits == 4 ? 1 : 0;
    pl.stages = lone ? 4 : 3;
    // Tile ids in workgroup order, rows of tiles along N (measured 2-4% faster at M = 816
    // than grouping consecutive tiles on one XCD or running down the rows first).
    pl.order = 2;
  }
  pl.partial_bytes = pl.splits > 1 ? align256((size_t)pl.splits * M * N * 4) : 0;
  return pl;
}

size_t gemm_plan_workspace(const GemmPlan &pl) { return pl.partial_bytes; }

size_t gemm_plan_relayout_bytes(const GemmPlan &pl, int64_t M, int64_t K) {
  return pl.kind == 3 ? align256((size_t)M * (size_t)K / 2) : 0;
}

// Every launcher below takes `go`: false resolves the kernel the plan selects and raises
// its dynamic-LDS limit without launching anything, so that a caller can find out whether
// a plan is launchable before it enqueues other work.
template <int BITS, int AFMT, int MT, int KT, int WK, int WC>
static hipError_t launch_stream(const GemmParams &p, dim3 grid, hipStream_t s, bool go) {
  const size_t lds = stream_lds_bytes<BITS, AFMT, MT, KT, WK, WC>();
  static std::atomic<uint64_t> attr{0};
  hipError_t e = allow_dynamic_lds(&gemm_stream_kernel<BITS, AFMT, MT, KT, WK, WC>, lds, attr);
  if (e != hipSuccess || !go) return e;
  hipLaunchKernelGGL((gemm_stream_kernel<BITS, AFMT, MT, KT, WK, WC>), grid, dim3(64 * WC * WK), lds, s, p);
  return hipGetLastError();
}

template <int KT, int WK, int NCW>
static hipError_t launch_stream_kw(const GemmParams &p, dim3 grid, hipStream_t s, bool go) {
  constexpr size_t lds = stream_kw_lds_bytes<KT, WK, NCW>();
  static_assert(lds <= 160 * 1024, "LDS budget");
  static std::atomic<uint64_t> attr{0};
  hipError_t e = allow_dynamic_lds(&gemm_stream_kw_kernel<KT, WK, NCW>, lds, attr);
  if (e != hipSuccess || !go) return e;
  hipLaunchKernelGGL((gemm_stream_kw_kernel<KT, WK, NCW>), grid, dim3(64 * WK), lds, s, p);
  return hipGetLastError();
}

template <int BITS, int AFMT, int MT, int WC>
static hipError_t launch_stream_wc(const GemmParams &p, int kt, int wk, dim3 grid, hipStream_t s, bool go) {
  if (wk == 4) {
    switch (kt) {
      case 1: return launch_stream<BITS, AFMT, MT, 1, 4, WC>(p, grid, s, go);
      case 2: return launch_stream<BITS, AFMT, MT, 2, 4, WC>(p, grid, s, go);
      case 4: return launch_stream<BITS, AFMT, MT, 4, 4, WC>(p, grid, s, go);
      case 8:
        if constexpr (AFMT == kANibble) return launch_stream<BITS, AFMT, MT, 8, 4, WC>(p, grid, s, go);
        return hipErrorInvalidValue;  // a 32-step int8 slice does not fit in LDS
      default: return hipErrorInvalidValue;
    }
  }
  if (wk == 1) {
    switch (kt) {
      case 1: return launch_stream<BITS, AFMT, MT, 1, 1, WC>(p, grid, s, go);
      case 2: return launch_stream<BITS, AFMT, MT, 2, 1, WC>(p, grid, s, go);
      default: return hipErrorInvalidValue;
    }
  }
  return hipErrorInvalidValue;
}

template <int BITS, int AFMT, int MT>
static hipError_t launch_stream_mt(const GemmParams &p, int kt, int wk, int wc, dim3 grid, hipStream_t s, bool go) {
  switch (wc) {
    case 1: return launch_stream_wc<BITS, AFMT, MT, 1>(p, kt, wk, grid, s, go);
    case 2: return launch_stream_wc<BITS, AFMT, MT, 2>(p, kt, wk, grid, s, go);
    case 4: return launch_stream_wc<BITS, AFMT, MT, 4>(p, kt, wk, grid, s, go);
    default: return hipErrorInvalidValue;
  }
}

template <int BITS, int AFMT, int BM, int BN, int ST, int LW>
static hipError_t launch_tile(const GemmParams &p, dim3 grid, hipStream_t s, bool go) {
  constexpr size_t lds = tile_lds_bytes<BITS, AFMT, BM, BN, ST>();
  static_assert(lds <= 160 * 1024, "LDS budget");
  static std::atomic<uint64_t> attr{0};
  hipError_t e = allow_dynamic_lds(&gemm_tile_kernel<BITS, AFMT, BM, BN, ST, LW>, lds, attr);
  if (e != hipSuccess || !go) return e;
  hipLaunchKernelGGL((gemm_tile_kernel<BITS, AFMT, BM, BN, ST, LW>), grid, dim3(256 + 64 * LW), lds, s, p);
  return hipGetLastError();
}

template <int BITS, int AFMT, int BM, int BN>
static hipError_t launch_tile_shape(const GemmParams &p, const GemmPlan &pl, dim3 grid, hipStream_t s, bool go) {
  if (pl.stages != 3 && pl.stages != 4) return hipErrorInvalidValue;
  if (pl.loader) {
    // one wave's loads of STAGES - 2 steps must fit the 6-bit vmcnt: 4 stages only for INT4
    if constexpr (BITS == 4)
      return pl.stages == 4 ? launch_tile<BITS, AFMT, BM, BN, 4, 1>(p, grid, s, go)
                            : launch_tile<BITS, AFMT, BM, BN, 3, 1>(p, grid, s, go);
    else
      return pl.stages == 3 ? launch_tile<BITS, AFMT, BM, BN, 3, 1>(p, grid, s, go) : hipErrorInvalidValue;
  }
  return pl.stages == 4 ? launch_tile<BITS, AFMT, BM, BN, 4, 0>(p, grid, s, go)
                        : launch_tile<BITS, AFMT, BM, BN, 3, 0>(p, grid, s, go);
}

template <int BITS, int AFMT>
static hipError_t launch_gemm_t(const GemmParams &p, const GemmPlan &pl, hipStream_t s, bool go) {
  hipError_t e;
  if (pl.kind == 2) {
    dim3 grid((unsigned)pl.tiles, (unsigned)pl.splits, (unsigned)pl.rb);
    e = hipErrorInvalidValue;
    if constexpr (BITS == 4 && AFMT == kANibble) {
      if (pl.kt == 16 && pl.wk == 8 && pl.wc == 1) e = launch_stream_kw<16, 8, 1>(p, grid, s, go);
      if (pl.kt == 16 && pl.wk == 8 && pl.wc == 2) e = launch_stream_kw<16, 8, 2>(p, grid, s, go);
    }
  } else if (pl.kind == 0) {
    dim3 grid((unsigned)pl.tiles, (unsigned)pl.splits, (unsigned)pl.rb);
    switch (pl.mt) {
      case 1: e = launch_stream_mt<BITS, AFMT, 1>(p, pl.kt, pl.wk, pl.wc, grid, s, go); break;
      case 2: e = launch_stream_mt<BITS, AFMT, 2>(p, pl.kt, pl.wk, pl.wc, grid, s, go); break;
      case 4: e = launch_stream_mt<BITS, AFMT, 4>(p, pl.kt, pl.wk, pl.wc, grid, s, go); break;
      default: e = hipErrorInvalidValue; break;
    }
  } else {
    dim3 grid((unsigned)pl.tiles, (unsigned)pl.splits);
    if (pl.bm == 64 && pl.bn == 128)
      e = launch_tile_shape<BITS, AFMT, 64, 128>(p, pl, grid, s, go);
    else if (pl.bm == 128 && pl.bn == 128)
      e = launch_tile_shape<BITS, AFMT, 128, 128>(p, pl, grid, s, go);
    else
      e = hipErrorInvalidValue;
  }
  if (e != hipSuccess || pl.splits == 1 || !go) return e;
  const int64_t threads = (int64_t)p.M * (p.N / 4);
  const unsigned blocks = (unsigned)((threads + 255) / 256);
  hipLaunchKernelGGL((splitk_epilogue_kernel<Fmt<BITS, AFMT>::shift>), dim3(blocks), dim3(256), 0, s, p,
                     pl.splits);
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs &g, const GemmPlan &pl, void *ws, hipStream_t s, bool go) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (pl.kind == 3) {
    // k groups: k-step-major codes as given, or canonical ones converted into ws first
    if (g.bits != 4) return hipErrorInvalidValue;
    KgParams kp;
    kp.delta = g.delta;
    kp.w = g.w;
    kp.w_scale = g.w_scale;
    kp.bias = g.bias;
    kp.y = g.y;
    kp.ldy = g.ldy;
    kp.acc_out = g.acc_out;
    kp.M = (int)g.M;
    kp.N = (int)g.N;
    kp.K = (int)g.K;
    if (g.a_fmt == kANibbleKM) {
      kp.a = g.a;
      return launch_gemm_kgroup(kp, nullptr, nullptr, s, go);
    }
    if (g.a_fmt != kANibble || g.lda != g.K / 2) return hipErrorInvalidValue;
    kp.a = static_cast<const uint8_t *>(ws);
    return launch_gemm_kgroup(kp, g.a, static_cast<uint8_t *>(ws), s, go);
  }
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
  p.partial = pl.splits > 1 ? reinterpret_cast<int32_t *>(ws) : nullptr;
  p.order = pl.order;
  if (g.bits == 4)
    return g.a_fmt == kANibble ? launch_gemm_t<4, kANibble>(p, pl, s, go) : hipErrorInvalidValue;
  return launch_gemm_t<8, kAInt8>(p, pl, s, go);
}

// ----------------------------------------------------------------------------------------
// Weight-only INT4 projection (W4A16): bf16 activations times the packed INT4 weight
// tiles, y = bf16_rne(s_j sum_c x_tc q_jc + b_j), the sum in fp32 on the bf16 matrix cores
// (v_mfma_f32_16x16x32_bf16).  The paper runs GR00T's adaptive layer-norm modulation this
// way (Sec. III-A).  Same streaming design as the W4A4 kernel: a workgroup owns one
// 16-channel weight tile column, a block of MT 16-row tiles and a K slice split between 4
// wave groups; the bf16 activation slice goes to LDS first (swizzled direct-to-LDS
// loads), the weight tiles follow in k order, and each k step's MFMAs start when its tile
// lands.  A weight nibble becomes a bf16 exactly: sign-extending bit-field extract,
// int -> fp32 (|code| <= 8), the fp32's upper half.  MFMA c of a 128-wide k step takes,
// from lane group g, channels 32 g + 8 c + [0, 8): the lane's own weight bytes 4c..4c+3 and
// the matching 16 bytes of the activation row, so both operands use one k order.

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

struct W16Params {
  const uint8_t *x;      // bf16 [M, ldx]
  int64_t ldx;           // elements
  const uint8_t *w;      // packed INT4 tiles
  const float *w_scale;  // [N]
  const float *bias;     // [N] or NULL
  uint16_t *y;           // bf16 [M, ldy]
  int64_t ldy;
  float *acc_out;        // fp32 [M, N] or NULL
  float *partial;        // fp32 [splits][M][N] when K is split
  int M, N, K;
};

// 8 nibble codes (channels 2i in the low, 2i + 1 in the high nibble of byte i) -> 8 bf16
// in channel order.
__device__ __forceinline__ bf16x8 nibbles_to_bf16(uint32_t w) {
  uint32_t r[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float e = (float)((int32_t)(w << (28 - 8 * i)) >> 28);
    const float o = (float)((int32_t)(w << (24 - 8 * i)) >> 28);
    r[i] = __builtin_amdgcn_perm(__float_as_uint(o), __float_as_uint(e), 0x07060302u);
  }
  const uint4 v = make_uint4(r[0], r[1], r[2], r[3]);
  return __builtin_bit_cast(bf16x8, v);
}

template <int MT, int KT, bool ONE>
__global__ __launch_bounds__(256) void w4a16_stream_kernel(W16Params p) {
  constexpr int WK = 4;
  constexpr int AROW = WK * KT * 256;  // bf16 bytes per row of the slice (128 channels per step)
  constexpr int ROWS = MT * 16;        // rows of the output tile
  // ONE (a single token): LDS holds that row only and every MFMA row reads it, so a slice
  // of 128 k steps (K = 16384) takes 32 KB and K needs no split
  constexpr int LROWS = ONE ? 1 : ROWS;
  static_assert(!ONE || MT == 1, "single-token slices have one row tile");
  constexpr int CPR = AROW / 16;
  constexpr int SLICE_KB = LROWS * AROW / 1024;
  constexpr int IA = SLICE_KB / WK;
  static_assert(LROWS * AROW % (1024 * WK) == 0, "slice must split into whole KBs per wave");
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int kg = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ntile = blockIdx.x, split = blockIdx.y, nsplit = gridDim.y;
  const int m0 = blockIdx.z * ROWS;
  const int mz = min(ROWS, p.M - m0);
  const int ktot = p.K / kTileK;
  const int slice_begin = split * WK * KT;
  const int ks_begin = slice_begin + kg * KT;
  const int nk = max(0, min(KT, ktot - ks_begin));

  // 1. bf16 activation slice -> LDS
  {
    const uint8_t *abase = p.x + ((int64_t)m0 * p.ldx + (int64_t)slice_begin * kTileK) * 2;
    const int valid_cols = min(WK * KT, ktot - slice_begin) * (kTileK * 2 / 16);
    if constexpr (ONE) {
      // wave kg fills KBs [kg IA, (kg + 1) IA) of the one row (a single row is not swizzled);
      // 16-byte chunks past the end of K read chunk 0
#pragma unroll
      for (int i = 0; i < IA; ++i) {
        const int kb = kg * IA + i;
        int col = kb * 64 + lane;
        if (col >= valid_cols) col = 0;
        load_to_lds16(abase + (uint32_t)(col * 16), lds + kb * 1024);
      }
    } else if (valid_cols == CPR) {
      stage_slice<AROW, IA, SLICE_KB, true>(abase, p.ldx * 2, mz, kg, lane, valid_cols, lds);
    } else {
      stage_slice<AROW, IA, SLICE_KB, false>(abase, p.ldx * 2, mz, kg, lane, valid_cols, lds);
    }
  }
  // 2. this wave's weight tiles, in k order, unconditionally (clamped past the end of K)
  sched_wall();
  uint4 wreg[KT];
  const uint8_t *wtile = p.w + (int64_t)ntile * ktot * tile_bytes(4) + lane * lane_bytes(4);
#pragma unroll
  for (int kt = 0; kt < KT; ++kt)
    wreg[kt] = *reinterpret_cast<const uint4 *>(wtile + (int64_t)min(ks_begin + kt, ktot - 1) * tile_bytes(4));
  sched_wall();
  wait_vmcnt<KT>();
  lds_barrier();

  // 3. MFMAs: per k step, 4 chunks of 32 channels, MT row tiles each
  v4f acc[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i] = v4f{0.f, 0.f, 0.f, 0.f};
  const int r16 = lane & 15, g = lane >> 4;
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) {
    if (kt < nk) {
      const uint32_t wd[4] = {wreg[kt].x, wreg[kt].y, wreg[kt].z, wreg[kt].w};
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const bf16x8 b = nibbles_to_bf16(wd[c]);
#pragma unroll
        for (int i = 0; i < MT; ++i) {
          const int row = ONE ? 0 : i * 16 + r16;
          const int chunk = (kg * KT + kt) * 16 + 4 * g + c;
          const uint4 av = *reinterpret_cast<const uint4 *>(lds + row * AROW + ((chunk ^ slice_swizzle<AROW>(row)) * 16));
          acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, av), b, acc[i], 0, 0, 0);
        }
      }
    }
  }

  // 4. wave groups add up through LDS (fixed order); group kg finishes row tiles kg mod 4
  __syncthreads();  // the slice is no longer read
  v4f *red = reinterpret_cast<v4f *>(lds);
#pragma unroll
  for (int i = 0; i < MT; ++i) red[(kg * MT + i) * 64 + lane] = acc[i];
  __syncthreads();
  const int n = ntile * 16 + r16;
  const float sw = p.w_scale[n];
  const float bj = p.bias ? p.bias[n] : 0.0f;
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    if (i % WK != kg) continue;
    v4f t = red[i * 64 + lane];
#pragma unroll
    for (int g2 = 1; g2 < WK; ++g2) t += red[(g2 * MT + i) * 64 + lane];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + i * 16 + 4 * g + r;
      if (m >= p.M) continue;
      if (nsplit > 1) {
        p.partial[((int64_t)split * p.M + m) * p.N + n] = t[r];
      } else {
        if (p.acc_out) p.acc_out[(int64_t)m * p.N + n] = t[r];
        p.y[(int64_t)m * p.ldy + n] = (uint16_t)f32_to_bf16(t[r] * sw + bj);
      }
    }
  }
}

// Adds the fp32 K slices in fixed order and applies the scale and bias; 4 columns per thread.
__global__ __launch_bounds__(256) void w4a16_splitk_epilogue_kernel(W16Params p, int slices) {
  const int cpr = p.N / 4;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)p.M * cpr) return;
  const int m = (int)(idx / cpr), n = (int)(idx % cpr) * 4;
  const float4 sw = *reinterpret_cast<const float4 *>(p.w_scale + n);
  const float4 bj = p.bias ? *reinterpret_cast<const float4 *>(p.bias + n) : make_float4(0.f, 0.f, 0.f, 0.f);
  const float4 *src = reinterpret_cast<const float4 *>(p.partial + (int64_t)m * p.N + n);
  const int64_t zs = (int64_t)p.M * p.N / 4;
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int z0 = 0; z0 < slices; z0 += 8) {
    float4 v[8];
#pragma unroll
    for (int z = 0; z < 8; ++z)
      if (z0 + z < slices) v[z] = src[(z0 + z) * zs];
#pragma unroll
    for (int z = 0; z < 8; ++z)
      if (z0 + z < slices) {
        a.x += v[z].x; a.y += v[z].y; a.z += v[z].z; a.w += v[z].w;
      }
  }
  if (p.acc_out) *reinterpret_cast<float4 *>(p.acc_out + (int64_t)m * p.N + n) = a;
  const uint32_t o0 = f32_to_bf16(a.x * sw.x + bj.x) | (f32_to_bf16(a.y * sw.y + bj.y) << 16);
  const uint32_t o1 = f32_to_bf16(a.z * sw.z + bj.z) | (f32_to_bf16(a.w * sw.w + bj.w) << 16);
  *reinterpret_cast<uint2 *>(p.y + (int64_t)m * p.ldy + n) = make_uint2(o0, o1);
}

W16Plan plan_w4a16(int64_t M, int64_t N, int64_t K) {
  W16Plan pl{};
  const int ktot = (int)(K / kTileK);
  if (M == 1 && ktot > 16) {
    // a single token: LDS holds its row only (KT KB, not 16 rows' worth), so many
    // workgroups share a compute unit.  K up to 8192 in one slice (no split-K epilogue);
    // longer K in slices of 32 k steps, which spreads the weight stream and its nibble
    // widening over more compute units (measured at K 16384 -> N 2048: 8.9 us against
    // 10.6 us for one 128-step slice per 16 channels).
    pl.one = true;
    pl.mt = 1;
    const int per = (ktot + 3) / 4;  // k steps per wave group
    pl.kt = per <= 8 ? 8 : (per <= 16 ? 16 : 8);
    pl.splits = (ktot + 4 * pl.kt - 1) / (4 * pl.kt);
    pl.tiles = N / 16;
    pl.rb = 1;
    pl.partial_bytes = pl.splits > 1 ? align256((size_t)pl.splits * M * N * 4) : 0;
    return pl;
  }
  pl.mt = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  // k steps per slice that fit 64 KB of LDS for 16 mt rows, so that two workgroups share
  // a compute unit (measured against 128 KB slices at K 16384 -> N 2048: M = 16 12.1
  // against 13.2 us, M = 32 17.4 against 19.5 us)
  const int smax = 16 / pl.mt;
  const int per = ktot < smax ? ktot : smax;
  pl.kt = per <= 4 ? 1 : (per <= 8 ? 2 : 4);
  pl.splits = (ktot + 4 * pl.kt - 1) / (4 * pl.kt);
  pl.tiles = N / 16;
  pl.rb = (int)((M + 16 * pl.mt - 1) / (16 * pl.mt));
  pl.partial_bytes = pl.splits > 1 ? align256((size_t)pl.splits * M * N * 4) : 0;
  return pl;
}

template <int MT, int KT, bool ONE = false>
static hipError_t launch_w16(const W16Params &p, dim3 grid, hipStream_t s) {
  constexpr size_t slice = (size_t)(ONE ? 1 : MT * 16) * 4 * KT * 256;
  constexpr size_t red = (size_t)4 * MT * 64 * 16;
  constexpr size_t lds = slice > red ? slice : red;
  static_assert(lds <= 160 * 1024, "LDS budget");
  static std::atomic<uint64_t> attr{0};
  hipError_t e = allow_dynamic_lds(&w4a16_stream_kernel<MT, KT, ONE>, lds, attr);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((w4a16_stream_kernel<MT, KT, ONE>), grid, dim3(256), lds, s, p);
  return hipGetLastError();
}

static hipError_t launch_w16_one(const W16Params &p, int kt, dim3 grid, hipStream_t s) {
  switch (kt) {
    case 4: return launch_w16<1, 4, true>(p, grid, s);
    case 8: return launch_w16<1, 8, true>(p, grid, s);
    case 16: return launch_w16<1, 16, true>(p, grid, s);
    default: return launch_w16<1, 32, true>(p, grid, s);
  }
}

template <int MT>
static hipError_t launch_w16_kt(const W16Params &p, int kt, dim3 grid, hipStream_t s) {
  switch (kt) {
    case 1: return launch_w16<MT, 1>(p, grid, s);
    case 2: return launch_w16<MT, 2>(p, grid, s);
    case 4: if constexpr (MT <= 2) return launch_w16<MT, 4>(p, grid, s); else return hipErrorInvalidValue;
    default: if constexpr (MT == 1) return launch_w16<MT, 8>(p, grid, s); else return hipErrorInvalidValue;
  }
}

hipError_t launch_w4a16(const W16Args &g, const W16Plan &pl, void *ws, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  W16Params p;
  p.x = static_cast<const uint8_t *>(g.x);
  p.ldx = g.ldx;
  p.w = g.w;
  p.w_scale = g.w_scale;
  p.bias = g.bias;
  p.y = g.y;
  p.ldy = g.ldy;
  p.acc_out = g.acc_out;
  p.partial = pl.splits > 1 ? reinterpret_cast<float *>(ws) : nullptr;
  p.M = (int)g.M;
  p.N = (int)g.N;
  p.K = (int)g.K;
  const dim3 grid((unsigned)pl.tiles, (unsigned)pl.splits, (unsigned)pl.rb);
  hipError_t e;
  if (pl.one) {
    e = launch_w16_one(p, pl.kt, grid, s);
  } else switch (pl.mt) {
    case 1: e = launch_w16_kt<1>(p, pl.kt, grid, s); break;
    case 2: e = launch_w16_kt<2>(p, pl.kt, grid, s); break;
    default: e = launch_w16_kt<4>(p, pl.kt, grid, s); break;
  }
  if (e != hipSuccess || pl.splits == 1) return e;
  const int64_t threads = (int64_t)p.M * (p.N / 4);
  hipLaunchKernelGGL(w4a16_splitk_epilogue_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, p,
                     pl.splits);
  return hipGetLastError();
}

}  // namespace fq
