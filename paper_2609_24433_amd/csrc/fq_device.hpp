// Device-side helpers shared by the gfx950 kernels of the quantized projection.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fq {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// Kernel-native weight tile: 16 output channels x 128 input channels.  Lane l of a
// wave owns channel n = l % 16 and the 32 input channels [32*(l/16), 32*(l/16)+32)
// of the tile; it stores them contiguously (16 bytes of nibbles or 32 bytes of int8).
// MFMA k-chunk c (0 or 1) of the tile consumes, from every lane, the 16 channels
// 32*(l/16) + 16*c + [0, 16).  Activation operands use the same channel mapping.
constexpr int kTileN = 16;
constexpr int kTileK = 128;
__host__ __device__ constexpr int tile_bytes(int bits) { return bits == 4 ? 1024 : 2048; }
__host__ __device__ constexpr int lane_bytes(int bits) { return bits == 4 ? 16 : 32; }

// bf16 bit pattern -> fp32 (exact).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// fp32 -> bf16 with round-to-nearest-even (NaN kept quiet).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// Signed nibbles -> int8 lanes scaled by 16.  Word w holds channels 0..7 (channel 2i in
// the low nibble of byte i).  lo gets 16*{c0,c2,c4,c6}, hi gets 16*{c1,c3,c5,c7}.
__device__ __forceinline__ void widen_nibbles(uint32_t w, uint32_t &lo, uint32_t &hi) {
  lo = (w << 4) & 0xF0F0F0F0u;
  hi = w & 0xF0F0F0F0u;
}

// 16 nibble-packed channels (8 bytes) -> MFMA operand of 16 int8 lanes (x16).
__device__ __forceinline__ v4i widen8(v2i p) {
  uint32_t a0, a1, b0, b1;
  widen_nibbles((uint32_t)p.x, a0, a1);
  widen_nibbles((uint32_t)p.y, b0, b1);
  v4i r;
  r.x = (int)a0;
  r.y = (int)a1;
  r.z = (int)b0;
  r.w = (int)b1;
  return r;
}

__device__ __forceinline__ v4i mfma16x16x64(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

}  // namespace fq
