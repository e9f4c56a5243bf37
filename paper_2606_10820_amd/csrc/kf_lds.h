// kf_lds.h -- explicit LDS and buffer-load helpers for gfx950 kernels that
// stage tiles with direct-to-LDS buffer loads.
//
// Operand tiles travel from global memory straight into LDS (buffer loads
// with the lds modifier: no register staging).  The compiler cannot track
// those LDS writes against ordinary LDS reads and would wait for every
// outstanding load before each read, which serialises a pipeline; so kernels
// read their tiles with explicit ds_read instructions and manage both
// counters themselves: vmcnt before the barrier that publishes a stage,
// lgkmcnt before the instructions that consume the reads.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kf {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));  // one 16-byte chunk
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));  // one 8-byte piece
typedef __attribute__((address_space(3))) void* lds_ptr;

__device__ inline uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}

// Raw buffer resource over [base, base + bytes): loads at or past `bytes`
// return zero (and write zero to LDS for the lds form) instead of faulting.
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

// 16 bytes per lane, global byte offset voff + soff, into LDS at dst + 16 * lane
// (dst is uniform across the wavefront).
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff,
                                      void* dst) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr)dst, 16, voff, soff, 0, 0);
}

__device__ __forceinline__ u32x4 ds_read16(uint32_t addr) {
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr) : "memory");
  return v;
}

template <int OFF>
__device__ __forceinline__ u32x4 ds_read16_off(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF) : "memory");
  return v;
}

// Transposing 8-byte read of 16-bit data (gfx950).  In each group of 16 lanes,
// lane 4e + q supplies the address of four consecutive elements (row e, columns
// 4q..4q+3 of a 4 x 16 block); lane i receives column i: the elements of rows
// 0..3 at column i, in row order.
template <int OFF>
__device__ __forceinline__ u32x2 ds_read_tr16_off(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  u32x2 v;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF) : "memory");
  return v;
}

__device__ __forceinline__ void lgkm_wait0() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }


// Keeps a value's consumers after the preceding wait.
__device__ __forceinline__ void pin(u32x4& v) { asm volatile("" : "+v"(v)); }
__device__ __forceinline__ void pin(u32x2& v) { asm volatile("" : "+v"(v)); }

// s_waitcnt with vmcnt = N and the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

}  // namespace kf
