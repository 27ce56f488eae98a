// Device helpers shared by the attention kernels of libvico (gfx950 only).
#pragma once

#include "vico_internal.h"

namespace vico {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) void lds_void;
typedef __amdgpu_buffer_rsrc_t rsrc_t;

constexpr float kLn2 = 0.6931471805599453f;
constexpr int kNumXcd = 8;
constexpr uint32_t kOutOfRange = 0x80000000u;
// Largest lane sum of one half's 16 probabilities accepted against the
// running max; it bounds each of them by 2^8 (exp2 of at most 8), far inside
// the fp32 and bf16 range.
constexpr float kLaneSumLimit = 256.0f;

// Logical work-group id for physical id `pid` so that each XCD receives a
// contiguous block of logical ids (hardware dispatches ids round-robin over
// the XCDs).  A bijection on [0, n).
__device__ __forceinline__ int xcd_remap(int pid, int n) {
  const int xcd = pid % kNumXcd, local = pid / kNumXcd;
  const int per = n / kNumXcd, rem = n % kNumXcd;
  return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

// Combine lane l with lane l^32 (the two halves of one query row's keys).
__device__ __forceinline__ float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Raw buffer resource over `bytes` bytes (stride 0, 32-bit data format).
// Reads at offsets >= bytes return zero.
__device__ __forceinline__ rsrc_t make_rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, 0x00020000);
}

// 16 bytes per lane from a buffer straight into LDS: lane i writes lds + 16*i.
// Kept in a device-only function: used inline in a kernel body, the builtin
// makes the host compilation pass drop the kernel's launch stub.
__device__ __forceinline__ void load_lds16(rsrc_t r, lds_void* lds, uint32_t voffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds, 16, voffset, 0, 0, 0);
}

// s_waitcnt immediate: vmcnt(n), lgkmcnt(0), expcnt not waited for.
constexpr uint32_t waitcnt_vm_lgkm0(uint32_t n) { return 0x0070u | n; }

// Work-group barrier that waits for nothing by itself.  __syncthreads()
// carries a work-group release fence, and the compiler implements that by
// waiting for every outstanding load, including direct-to-LDS prefetches that
// are meant to stay in flight across the barrier.  Callers wait for what they
// need with s_waitcnt first; the "memory" clobber keeps the compiler from
// moving memory accesses across the barrier.
__device__ __forceinline__ void barrier_keep_loads() { asm volatile("s_barrier" ::: "memory"); }

}  // namespace vico
