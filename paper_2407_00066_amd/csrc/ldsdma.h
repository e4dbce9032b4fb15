// Buffer-load and LDS helpers of the LDS-ring GEMM kernels (gemm.hip): raw
// buffer resources with 31-bit offsets, 16-byte loads
// straight into LDS (buffer_load ... lds), explicit wait counts and 16-byte
// LDS fragment reads.  Device code only; nothing here is part of the ABI.
#pragma once

#include "cts_internal.h"

namespace cts {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr uint32_t kOob = 0x80000000u;   // every operand is < 2^31 bytes

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t nbytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                           static_cast<int>(nbytes), 0x00020000);
}

__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

template <int BK> __device__ __forceinline__ int swz_key(int row) {
  if (BK == 128) return row & 15;
  return BK == 64 ? ((row >> 1) & 7) : ((row >> 2) & 3);
}

// The inline assembly below exists only in the device compilation pass (the
// host pass of a HIP translation unit never executes kernel bodies).
template <int N> __device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
#endif
}

template <int N> __device__ __forceinline__ void wait_lgkmcnt() {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
#endif
}

// 16-byte LDS read issued as assembly: its completion is waited for with
// wait_lgkmcnt, and pin() ties the fragment to that wait.
__device__ __forceinline__ void lds_read16(bf16x8& dst, uint32_t addr) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("ds_read_b128 %0, %1" : "=v"(dst) : "v"(addr) : "memory");
#endif
}

// 16-byte buffer load of each lane straight into LDS: lane l's chunk lands at
// lds + 16*l (lds must be the same for the whole wave); out-of-range lanes
// write zeros.
__device__ __forceinline__ void load16_lds(__amdgpu_buffer_rsrc_t r, char* lds, uint32_t voff,
                                           uint32_t soff = 0) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voff,
                                           soff, 0, 0);
#endif
}

// 4-byte buffer load of each lane into LDS, used as an L2 prefetch: the data
// lands in a scratch LDS slot nobody reads, only the cache fill matters.
__device__ __forceinline__ void load4_lds(__amdgpu_buffer_rsrc_t r, void* lds, uint32_t voff,
                                          uint32_t soff) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 4, voff,
                                           soff, 0, 0);
#endif
}

__device__ __forceinline__ void pin(bf16x8& v) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("" : "+v"(v));
#endif
}

}  // namespace cts
