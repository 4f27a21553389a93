// CDNA4 (gfx950) building blocks shared by the fused kernels: vector types,
// matrix-core wrappers, cross-lane exchanges and the bias-tile transpose.
//
// Matrix-core layouts (64 lanes, lane L, n = L % 16, g = L / 16):
// v_mfma_f32_16x16x32_bf16: A holds row n, k-slots 8g..8g+7; B holds column n,
// k-slots 8g..8g+7; the accumulator holds rows 4g..4g+3 of column n.
// v_mfma_f32_16x16x16_bf16: the same with k-slots 4g..4g+3.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dcp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 u) { return __builtin_bit_cast(bf16x8, u); }
__device__ __forceinline__ bf16x4 as_bf16x4(u32x2 u) { return __builtin_bit_cast(bf16x4, u); }
__device__ __forceinline__ bf16x2 as_bf16x2(uint32_t u) { return __builtin_bit_cast(bf16x2, u); }

__device__ __forceinline__ f32x4 mfma32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma16(bf16x4 a, bf16x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

// Exchange between lane halves: x's lanes 32..63 <-> y's lanes 0..31.
__device__ __forceinline__ void swap32(float& x, float& y) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(y), false, false);
  x = __uint_as_float(r[0]);
  y = __uint_as_float(r[1]);
}
// Exchange between 16-lane rows: x's odd rows <-> y's even rows.
__device__ __forceinline__ void swap16(float& x, float& y) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(y), false, false);
  x = __uint_as_float(r[0]);
  y = __uint_as_float(r[1]);
}

// Sum / max over the four lanes n, n+16, n+32, n+48; every lane gets the same bits.
__device__ __forceinline__ float sum4(float x) {
  float a = x, b = x;
  swap32(a, b);
  x = a + b;
  a = x;
  b = x;
  swap16(a, b);
  return a + b;
}
__device__ __forceinline__ float max4(float x) {
  float a = x, b = x;
  swap32(a, b);
  x = fmaxf(a, b);
  a = x;
  b = x;
  swap16(a, b);
  return fmaxf(a, b);
}

// b[k][i] holds (row n, head 4g+i, key k) for the tile's 16 keys. After this,
// b[4a + r][i] holds (row n, head 4a+i, key 4g+r): the QK^T accumulator layout
// of head 4a+i. A 4x4 exchange of 4x4 blocks between the lane groups, done
// with two rounds of cross-lane swaps (bit 1 of the group, then bit 0).
__device__ __forceinline__ void transpose_bias(float (&b)[16][4]) {
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int i = 0; i < 4; ++i) swap32(b[4 * c + r][i], b[4 * (c + 2) + r][i]);
#pragma unroll
  for (int c = 0; c < 4; c += 2)
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int i = 0; i < 4; ++i) swap16(b[4 * c + r][i], b[4 * (c + 1) + r][i]);
}

// ---- direct-to-LDS loads and explicit waits
// The DMA loads below are issued from inline asm, so the compiler neither
// counts them nor inserts waits for them: every wait on their data is an
// explicit s_waitcnt with a compile-time count. (Ops the compiler cannot see
// only make its own waits stricter, never looser, because vector-memory
// loads complete in issue order.)
constexpr uint32_t kRawBufferFlags = 0x00020000u;
constexpr int kOutOfRange = 0x7FFFFF00;  // offset past every record: the load moves no data

// 16 bytes per lane from buffer r at byte offset voff into LDS at
// lds_base + 16 * lane (lds_base: wave-uniform LDS byte address). Waits for
// this wave's outstanding LDS reads first, so a slot being refilled is never
// still being read.
__device__ __forceinline__ void dma_b128(__amdgpu_buffer_rsrc_t r, int voff, uint32_t lds_base) {
  uint32_t saved;
  asm volatile(
      "s_waitcnt lgkmcnt(0)\n\t"
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "buffer_load_dwordx4 %1, %2, 0 offen lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(voff), "s"(r), "s"(lds_base)
      : "memory");
}

// The four loads of one key of the pair tensor stream, 4 x 1 KB into LDS at
// lds_base, non-temporal (data read exactly once, so it does not displace the
// reused K/V tiles in the caches), under one M0: the instruction offset (1024 i
// for load i) is added to the LDS and to the global address alike, so voff_i
// is load i's global offset minus 1024 i. Waits for this wave's LDS reads
// first, like dma_b128.
__device__ __forceinline__ void dma_key_stream(__amdgpu_buffer_rsrc_t r, int v0, int v1, int v2, int v3,
                                               uint32_t lds_base) {
  uint32_t saved;
  asm volatile(
      "s_waitcnt lgkmcnt(0)\n\t"
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %6\n\t"
      "buffer_load_dwordx4 %1, %5, 0 offen nt lds\n\t"
      "buffer_load_dwordx4 %2, %5, 0 offen offset:1024 nt lds\n\t"
      "buffer_load_dwordx4 %3, %5, 0 offen offset:2048 nt lds\n\t"
      "buffer_load_dwordx4 %4, %5, 0 offen offset:3072 nt lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(v0), "v"(v1), "v"(v2), "v"(v3), "s"(r), "s"(lds_base)
      : "memory");
}

// Wait until at most N of this wave's vector-memory loads are outstanding.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Workgroup barrier without the memory-model fence (which would also wait for
// every outstanding DMA load). It first waits for this wave's own LDS reads
// and writes (lgkmcnt(0)): gfx950 has the back-off barrier, so the compiler
// does not drain LDS operations before s_barrier by itself, and a read still
// in flight there could otherwise be overtaken by another wave's refill of the
// same LDS after the barrier. The "memory" clobbers keep every LDS access on
// its side of the barrier.
__device__ __forceinline__ void barrier_lds() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)reinterpret_cast<uintptr_t>(p);
}

}  // namespace dcp
