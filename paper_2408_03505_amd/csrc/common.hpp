// Shared device helpers for the gfx950 (CDNA4) kernels: bf16 conversion,
// MFMA operand types, wave-level reductions and the 8x8 register transpose
// used to stage contraction-strided operands into LDS.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace optimus {

typedef uint16_t bf16_t;
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf2f(bf16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// Round-to-nearest-even fp32 -> bf16 (hardware conversion on gfx950).
__device__ __forceinline__ bf16_t f2bf(float f) {
  __bf16 b = static_cast<__bf16>(f);
  return __builtin_bit_cast(bf16_t, b);
}

// Two fp32 -> packed bf16 pair (lo in bits 0..15).
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  return static_cast<uint32_t>(f2bf(lo)) | (static_cast<uint32_t>(f2bf(hi)) << 16);
}

__device__ __forceinline__ float lo_bf(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t v) {
  return __builtin_bit_cast(bf16x8_t, v);
}

__device__ __forceinline__ f32x16_t mfma32(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Workgroup barrier for hand-overs through LDS: waits for this wave's LDS
// (and scalar) accesses only.  __syncthreads() also drains every outstanding
// global load, which would stall loads issued ahead for later work.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Sum / max over the 64 lanes of a wave (butterfly; every lane gets the result).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// 8x8 transpose of bf16 held as eight 16-byte rows: in[j] holds elements
// (j, 0..7); out[i] receives elements (0..7, i).  Each output dword packs
// two 16-bit halves taken from consecutive input rows (v_perm_b32).
__device__ __forceinline__ void transpose8x8(const u32x4_t in[8], u32x4_t out[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t sel = (i & 1) ? 0x07060302u : 0x05040100u;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      out[i][p] = __builtin_amdgcn_perm(in[2 * p + 1][i >> 1], in[2 * p][i >> 1], sel);
    }
  }
}

__device__ __forceinline__ u32x4_t ldg16(const bf16_t *p) {
  return *reinterpret_cast<const u32x4_t *>(p);
}

__device__ __forceinline__ void stg16(bf16_t *p, u32x4_t v) {
  *reinterpret_cast<u32x4_t *>(p) = v;
}

// Streaming (non-temporal) 16-byte stores, for outputs that the writing
// kernel does not read again.
__device__ __forceinline__ void stg16_nt(bf16_t *p, u32x4_t v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4_t *>(p));
}
__device__ __forceinline__ void stg16_nt(float *p, f32x4_t v) {
  __builtin_nontemporal_store(v, reinterpret_cast<f32x4_t *>(p));
}

}  // namespace optimus
