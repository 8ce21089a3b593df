// Device-side helpers shared by the gfx950 kernels of the quantized projection.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

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

// fp32 -> bf16 bit pattern, round to nearest even: gfx950's v_cvt_pk_bf16_f32 (one
// instruction instead of five for the integer rounding it replaces; checked equal to that
// rounding on 16.7 million inputs covering ties, denormals and infinities; a NaN stays a
// quiet NaN).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
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

__device__ __forceinline__ void lds_fence() { asm volatile("" ::: "memory"); }

// f(std::integral_constant<int, i>) for i = 0 .. N-1 in order, each i a compile-time constant.
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F &f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Instruction-scheduling wall: the compiler moves nothing across it.
__device__ __forceinline__ void sched_wall() { __builtin_amdgcn_sched_barrier(0); }

// Workgroup barrier that waits only for this wave's LDS accesses.  __syncthreads() also
// waits for every outstanding global load (vmcnt(0)), which would drain a prefetch ring.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4) | (0 << 8));  // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  lds_fence();
}

// 16 bytes per lane from global memory straight into LDS; a wave fills the contiguous
// KB at `lds_dst` (lane l -> lds_dst + 16 l).  The builtin exists only for the device
// pass, so the host pass (which only needs the kernel stub) sees an empty body.
__device__ __forceinline__ void load_to_lds16(const void *src, void *lds_dst) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_global_load_lds(src, lds_dst, 16, 0, 0);
#else
  (void)src;
  (void)lds_dst;
#endif
}

// 16-byte LDS read the compiler does not track.  The compiler cannot tell LDS locations
// written by direct-to-LDS loads from the ones read here, so it would hold an ordinary
// LDS read until every such load in flight has landed; a kernel that reads one region
// while another region is still being filled issues its own waits instead: a
// wait_vmcnt for the loads that fill the region (and a barrier), and lgkm_wait_all()
// before the result is used.
__device__ __forceinline__ uint4 lds_read16_untracked(const void *p) {
  uint4 v;
  const uint32_t a = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a) : "memory");
  return v;
}
__device__ __forceinline__ float lds_read4_untracked(const void *p) {
  float v;
  const uint32_t a = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
  asm volatile("ds_read_b32 %0, %1" : "=v"(v) : "v"(a) : "memory");
  return v;
}
__device__ __forceinline__ void lgkm_wait_all() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// 16-byte global load the compiler does not track: it places no wait of its own for the
// result, which a kernel that streams many loads into registers needs when the compiler's
// bookkeeping would otherwise make the first use wait for every load in flight.  The
// caller waits with vm_wait_on before using the value.
__device__ __forceinline__ v4i global_load16_untracked(const void *p) {
  v4i v;
  asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(v) : "v"(p) : "memory");
  return v;
}
// s_waitcnt vmcnt(N) tied to a and b, results of untracked loads: no use of them moves
// above the wait.
template <int N>
__device__ __forceinline__ void vm_wait_on(v4i &a, v4i &b) {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%2)" : "+v"(a), "+v"(b) : "i"(N) : "memory");
}
template <int N>
__device__ __forceinline__ void vm_wait_on(v4i &a) {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%1)" : "+v"(a) : "i"(N) : "memory");
}
// lgkmcnt(0) tied to v, the result of an untracked read: no use of v moves above the wait.
__device__ __forceinline__ void lgkm_wait_on(v4i &v) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(v)::"memory");
}
// LDS writes the compiler does not track (same reason); an lds_barrier() orders them.
__device__ __forceinline__ void lds_write4_untracked(void *p, float v) {
  const uint32_t a = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
  asm volatile("ds_write_b32 %0, %1" ::"v"(a), "v"(v) : "memory");
}
__device__ __forceinline__ void lds_write8_untracked(void *p, uint2 v) {
  const uint32_t a = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
  const v2i w{(int)v.x, (int)v.y};
  asm volatile("ds_write_b64 %0, %1" ::"v"(a), "v"(w) : "memory");
}
__device__ __forceinline__ void lds_write16_untracked(void *p, uint4 v) {
  const uint32_t a = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
  const v4i w{(int)v.x, (int)v.y, (int)v.z, (int)v.w};
  asm volatile("ds_write_b128 %0, %1" ::"v"(a), "v"(w) : "memory");
}

// s_waitcnt vmcnt(n) leaving the other counters alone (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}


}  // namespace fq
