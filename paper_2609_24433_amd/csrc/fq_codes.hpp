// Device helpers shared by the prologue kernels: eq. (5) rounding to a code bit pattern,
// canonical packing of 16 codes, and cross-lane reads inside a wave.
#pragma once

#include "fq_device.hpp"
#include "fq_launch.hpp"

namespace fq {

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

}  // namespace fq
