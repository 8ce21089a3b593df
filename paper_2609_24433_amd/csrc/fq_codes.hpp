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

// Nibble codes in biased form, for the prologue kernel: clamp (when the clip ratio can push
// |u * inv| past q + 1/2) and add 1.5 * 2^23 + 8, which rounds exactly as quantize_bits does
// (the added integer is even, so ties still go to even) and leaves the bit pattern
// 0x4B400000 + code + 8: the low nibble holds code + 8 in [1, 15] and bits 4..15 are zero.
// With r = 1 no clamp is needed: |u| <= A, inv = fl(q / A), so |fl(u * inv)| <= q (1 + 2^-24)^2
// < q + 1/2 and the rounded value never passes q.
template <bool CLAMP>
__device__ __forceinline__ uint32_t quantize_bits_biased(float u, float inv, float lim) {
  const float t = CLAMP ? __builtin_amdgcn_fmed3f(u * inv, -lim, lim) : u * inv;
  return __float_as_uint(t + 12582920.0f);
}

// (a << S) | b as one instruction; written out so that the compiler keeps the two-level
// combination below instead of re-associating it into separate shifts.
template <int S>
__device__ __forceinline__ uint32_t lshl_or(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_lshl_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "i"(S), "v"(b));
  return r;
}

// 16 biased bit patterns (natural channel order) -> canonical nibbles, 8 bytes.  Byte 0 of
// (odd << 4) | even is (c_odd + 8) << 4 | (c_even + 8) and its byte 1 is zero, so two such
// words combine with one more shift-or, two halves with a byte permute, and one xor with 0x8
// per nibble turns code + 8 into the two's-complement nibble.
__device__ __forceinline__ uint2 pack_chunk_nibbles_biased(const uint32_t (&c)[16]) {
  uint32_t w[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    uint32_t pb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) pb[i] = lshl_or<4>(c[8 * h + 2 * i + 1], c[8 * h + 2 * i]);
    const uint32_t lo = lshl_or<8>(pb[1], pb[0]);
    const uint32_t hi = lshl_or<8>(pb[3], pb[2]);
    w[h] = __builtin_amdgcn_perm(hi, lo, 0x05040100u) ^ 0x88888888u;
  }
  return make_uint2(w[0], w[1]);
}

// 8 biased bit patterns (channels 0..7, see quantize_bits_biased) straight to the INT4
// MFMA operand words, the form widen_nibbles gives from the packed nibbles: lo holds
// 16 * {c0, c2, c4, c6}, hi 16 * {c1, c3, c5, c7}, one int8 lane each.  Two shift-ors and a
// byte permute gather four (code + 8) bytes; shifting them up a nibble gives 16 (code + 8),
// and xor 0x80 per byte subtracts the 128 (mod 256).
__device__ __forceinline__ void widen_biased8(const uint32_t *b, uint32_t &lo, uint32_t &hi) {
  const uint32_t le = __builtin_amdgcn_perm(lshl_or<8>(b[6], b[4]), lshl_or<8>(b[2], b[0]), 0x05040100u);
  const uint32_t ho = __builtin_amdgcn_perm(lshl_or<8>(b[7], b[5]), lshl_or<8>(b[3], b[1]), 0x05040100u);
  lo = (le << 4) ^ 0x80808080u;
  hi = (ho << 4) ^ 0x80808080u;
}

// Pack 16 quantized bit patterns (natural channel order; low byte = code) into canonical
// nibbles (8 bytes: channel 2i in the low nibble of byte i) or int8 (16 bytes).
__device__ __forceinline__ uint2 pack_chunk_nibbles(const int (&c)[16]) {
  uint32_t w[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    uint32_t b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) b[i] = ((uint32_t)c[8 * h + 2 * i] & 0xFu) | ((uint32_t)c[8 * h + 2 * i + 1] << 4);
    // low bytes of b[0..3] -> one word
    const uint32_t lo = __builtin_amdgcn_perm(b[1], b[0], 0x0c0c0400u);
    const uint32_t hi = __builtin_amdgcn_perm(b[3], b[2], 0x04000c0cu);
    w[h] = lo | hi;
  }
  return make_uint2(w[0], w[1]);
}

__device__ __forceinline__ uint4 pack_chunk_int8(const int (&c)[16]) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t lo = __builtin_amdgcn_perm((uint32_t)c[4 * i + 1], (uint32_t)c[4 * i], 0x0c0c0400u);
    const uint32_t hi = __builtin_amdgcn_perm((uint32_t)c[4 * i + 3], (uint32_t)c[4 * i + 2], 0x04000c0cu);
    w[i] = lo | hi;
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// Pack chunk `chunk` of a row and store it at its canonical place in row_out.
__device__ __forceinline__ void store_chunk_bits(uint8_t *row_out, int chunk, const int (&c)[16],
                                                 int out_fmt) {
  if (out_fmt == kOutNibble)
    *reinterpret_cast<uint2 *>(row_out + (int64_t)chunk * 8) = pack_chunk_nibbles(c);
  else
    *reinterpret_cast<uint4 *>(row_out + (int64_t)chunk * 16) = pack_chunk_int8(c);
}

// Value of lane (l ^ M) of the wave, for M < 32: DPP quad permutations for 1 and 2, a
// 16-lane row rotation by 8 for 8, the LDS crossbar's bit-mask swizzle (no memory) for 4
// and 16.  Every lane's source is valid, so the DPP moves need no old value.  Pure data
// movement: the butterfly sums stay bit-exact.
template <int M>
__device__ __forceinline__ float lane_xor(float v) {
  const int x = __float_as_int(v);
  int r;
  if constexpr (M == 1) r = __builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false);       // quad_perm 1,0,3,2
  else if constexpr (M == 2) r = __builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false);  // quad_perm 2,3,0,1
  else if constexpr (M == 8) r = __builtin_amdgcn_mov_dpp(x, 0x128, 0xF, 0xF, false); // row_ror:8
  else r = __builtin_amdgcn_ds_swizzle(x, (M << 10) | 0x1F);                          // xor M in 32 lanes
  return __int_as_float(r);
}

// ---- the prologue's per-chunk arithmetic (one 16-channel chunk per register array) ----

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

// v *= m elementwise (one fp32 rounding per element): the fold multipliers.
__device__ __forceinline__ void mul_chunk(float (&v)[16], const float4 (&m)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[4 * i] = v[4 * i] * m[i].x;
    v[4 * i + 1] = v[4 * i + 1] * m[i].y;
    v[4 * i + 2] = v[4 * i + 2] * m[i].z;
    v[4 * i + 3] = v[4 * i + 3] * m[i].w;
  }
}

// One butterfly stage of span H inside a chunk of CW registers: (a, c) -> (a + c, a - c).
template <int H, int CW = 16>
__device__ __forceinline__ void chunk_stage(float (&v)[CW]) {
#pragma unroll
  for (int i = 0; i < CW; i += 2 * H) {
#pragma unroll
    for (int j = i; j < i + H; ++j) {
      float a = v[j], c = v[j + H];
      v[j] = a + c;
      v[j + H] = a - c;
    }
  }
}

// Butterfly stage h = CW M across lanes: chunk j pairs with chunk j ^ M, held by lane ^ M.
// Each lane computes own + s * partner with s = -1 on the upper lane, as one fma (the exact
// sum or difference, rounded once): the lower lane gets a + c, the upper one c - a, the
// negation of a - c (round to nearest even is symmetric, so bit for bit -(a - c)).  Both
// partners carry the same sign (it depends only on the chunk index bits below M), so every
// later stage stays the same pair update up to that sign; row_sign() gives the sign a lane
// carries after the whole transform.  In this form the partner is a multiplicand, which lets
// the compiler fold a DPP lane move into the multiply-add.
// own + s * partner for every value of a chunk, the partner read through a DPP lane move
// folded into v_fmac_f32 (one instruction per value).  The leading s_nop covers the DPP
// read-after-write wait states for values written just before the block; inside the block
// every instruction reads and writes its own register.
#define FQ_FMAC(i, CTL) "v_fmac_f32_dpp %" #i ", %" #i ", %[s] " CTL "\n\t"
#define FQ_FMAC8(CTL)                                                                             \
  FQ_FMAC(0, CTL) FQ_FMAC(1, CTL) FQ_FMAC(2, CTL) FQ_FMAC(3, CTL) FQ_FMAC(4, CTL) FQ_FMAC(5, CTL) \
  FQ_FMAC(6, CTL) FQ_FMAC(7, CTL)
#define FQ_FMAC16(CTL)                                                                              \
  FQ_FMAC8(CTL) FQ_FMAC(8, CTL) FQ_FMAC(9, CTL) FQ_FMAC(10, CTL) FQ_FMAC(11, CTL) FQ_FMAC(12, CTL) \
  FQ_FMAC(13, CTL) FQ_FMAC(14, CTL) FQ_FMAC(15, CTL)
#define FQ_DPP_FMAC_CHUNK(NAME, CTL)                                                               \
  __device__ __forceinline__ void NAME(float (&v)[16], float s) {                                 \
    asm("s_nop 4\n\t" FQ_FMAC16(CTL)                                                             \
        : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]),      \
          "+v"(v[7]), "+v"(v[8]), "+v"(v[9]), "+v"(v[10]), "+v"(v[11]), "+v"(v[12]), "+v"(v[13]),   \
          "+v"(v[14]), "+v"(v[15])                                                                \
        : [s] "v"(s));                                                                            \
  }                                                                                               \
  __device__ __forceinline__ void NAME(float (&v)[8], float s) {                                  \
    asm("s_nop 4\n\t" FQ_FMAC8(CTL)                                                              \
        : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]),      \
          "+v"(v[7])                                                                              \
        : [s] "v"(s));                                                                            \
  }
FQ_DPP_FMAC_CHUNK(fmac_xor1, "quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf")
FQ_DPP_FMAC_CHUNK(fmac_xor2, "quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf")
FQ_DPP_FMAC_CHUNK(fmac_xor8, "row_ror:8 row_mask:0xf bank_mask:0xf")
#undef FQ_DPP_FMAC_CHUNK
#undef FQ_FMAC16
#undef FQ_FMAC8
#undef FQ_FMAC

template <int M, int CPT, int CW = 16>
__device__ __forceinline__ void lane_stage(float (&v)[CPT][CW], int tau) {
  const float s = (tau & M) ? -1.0f : 1.0f;
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    if constexpr (M == 1) fmac_xor1(v[c], s);
    else if constexpr (M == 2) fmac_xor2(v[c], s);
    else if constexpr (M == 8) fmac_xor8(v[c], s);
    else {
#pragma unroll
      for (int i = 0; i < CW; ++i) v[c][i] = __builtin_fmaf(lane_xor<M>(v[c][i]), s, v[c][i]);
    }
  }
}

// Sign of the values lane tau holds after row_transform(log2b): -1 when an odd number of
// its lane stages left it on the upper side.  |value| and value * (sign * inv) are those of
// the true transform exactly.
template <int CW = 16>
__device__ __forceinline__ float row_sign(int log2b, int tau) {
  constexpr int L = CW == 16 ? 4 : 3;  // stages inside a chunk
  const int lanes = log2b > L ? (1 << (log2b - L)) - 1 : 0;
  return (__builtin_popcount(tau & lanes) & 1) ? -1.0f : 1.0f;
}

// The blockwise unnormalized Sylvester transform of a row held as CW-channel chunks
// c * TPR + tau by consecutive lanes: stages h = 1 .. b/2 in ascending order, h < CW
// inside each chunk and h >= CW across lanes (a b-block is b/CW consecutive chunks in
// consecutive lanes of one wave).  b = 2^log2b is uniform across the wave, so the stage
// branches are too.  The result does not depend on CW: every stage is the same pair
// update in the same order.
template <int CPT, int CW = 16>
__device__ __forceinline__ void row_transform(float (&v)[CPT][CW], int log2b, int tau) {
  static_assert(CW == 8 || CW == 16, "chunk width");
  constexpr int L = CW == 16 ? 4 : 3;  // stages inside a chunk
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    if (log2b > 0) chunk_stage<1, CW>(v[c]);
    if (log2b > 1) chunk_stage<2, CW>(v[c]);
    if (log2b > 2) chunk_stage<4, CW>(v[c]);
    if constexpr (CW == 16)
      if (log2b > 3) chunk_stage<8, CW>(v[c]);
  }
  if (log2b > L) lane_stage<1, CPT, CW>(v, tau);
  if (log2b > L + 1) lane_stage<2, CPT, CW>(v, tau);
  if (log2b > L + 2) lane_stage<4, CPT, CW>(v, tau);
  if (log2b > L + 3) lane_stage<8, CPT, CW>(v, tau);
  if constexpr (CW == 8)
    if (log2b > L + 4) lane_stage<16, CPT, CW>(v, tau);
}

}  // namespace fq
