// Direct HBM -> LDS loads and LDS transpose reads shared by the GEMM and
// attention kernels (gfx950).
#pragma once

#include "common.hpp"

namespace optimus {

typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char lds_char;

constexpr int kRsrcWord3 = 0x00020000;  // raw buffer, 32-bit dwords, gfx9 data format

// 128-bit buffer resource: base, byte extent and the raw-buffer format word.
__device__ __forceinline__ u32x4_t make_rsrc(const void *base, uint32_t nbytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return u32x4_t{static_cast<uint32_t>(a), static_cast<uint32_t>(a >> 32) & 0xffffu, nbytes,
                 static_cast<uint32_t>(kRsrcWord3)};
}

// One 16-byte-per-lane buffer load written straight to LDS at
// lds_addr + 16 * lane.  Issued as inline asm so that the compiler does not
// wrap every later LDS access and barrier in a full vmcnt(0) wait; the
// kernel waits on vmcnt itself.  M0 (the LDS base of the DMA) is saved and
// restored around the load; s_nop covers the M0-write hazard.
__device__ __forceinline__ void buffer_load_lds16(const u32x4_t &rsrc, uint32_t lds_addr, uint32_t voff,
                                                  uint32_t soff) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %2, %3, %4 offen lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_addr), "v"(voff), "s"(rsrc), "s"(soff)
      : "memory");
}

// The 4-byte-per-lane form: writes lds_addr + 4 * lane.
__device__ __forceinline__ void buffer_load_lds4(const u32x4_t &rsrc, uint32_t lds_addr, uint32_t voff,
                                                 uint32_t soff) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "buffer_load_dword %2, %3, %4 offen lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_addr), "v"(voff), "s"(rsrc), "s"(soff)
      : "memory");
}

__device__ __forceinline__ bf16x8_t lds_read_tr(const lds_char *a, const lds_char *b) {
  const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      reinterpret_cast<__attribute__((address_space(3))) i16x4_t *>(const_cast<lds_char *>(a)));
  const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      reinterpret_cast<__attribute__((address_space(3))) i16x4_t *>(const_cast<lds_char *>(b)));
  typedef short i16x8_t __attribute__((ext_vector_type(8)));
  const i16x8_t v{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8_t, v);
}

// s_waitcnt vmcnt(N) lgkmcnt(L) (gfx9 encoding; L = 15 leaves LDS alone).
template <int N, int L = 15>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64 && L >= 0 && L < 16, "waitcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (L << 8));
}

}  // namespace optimus
