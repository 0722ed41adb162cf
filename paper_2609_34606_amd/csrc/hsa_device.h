// Device-side helpers shared by the HSA kernels (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hsa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;

// ---------------------------------------------------------------- bf16
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Round two floats to bf16 (nearest-even) and pack: a in the low half
// (a single v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  const bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// ---------------------------------------------------------------- MFMA
// D[32x32] += A[32x16] * B[16x32]. Lane l supplies A row (l % 32), k =
// 8*(l/32)..+8, and B column (l % 32), same k range. Result register r of
// lane l holds row 8*(r/4) + 4*(l/32) + (r%4), column l % 32.
__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

// ---------------------------------------------------------------- feature map
// elu(x) + 1
__device__ __forceinline__ float phi(float x) { return x > 0.f ? x + 1.f : __expf(x); }

// ---------------------------------------------------------------- memory
__device__ __forceinline__ u32x4 ld_global16(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
__device__ __forceinline__ u32x4 ld_lds16(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// Asynchronous 16-byte global -> LDS copy: lane i of the wave writes the 16
// bytes at gptr to lds_wave_base + 16*i. lds_wave_base must be wave-uniform.
__device__ __forceinline__ void g2lds16(const void* gptr, void* lds_wave_base) {
  __builtin_amdgcn_global_load_lds(gptr,
                                   (__attribute__((address_space(3))) void*)lds_wave_base,
                                   16, 0, 0);
}

// The same copy issued from inline assembly. hipcc's wait-count pass stops
// using partial LDS counts (it waits lgkmcnt(0) before every use of an LDS
// read) as soon as a global_load_lds it knows of is in flight; issued this
// way the copy is invisible to it, and LDS operand reads can be pipelined
// with exact lgkmcnt(N) waits. The caller orders the copies itself with
// wait_vmcnt and a barrier before the data is read. Since the vector-memory
// counter retires in order, the compiler's own vmcnt waits stay correct
// (copies it does not count only make them wait longer).
__device__ __forceinline__ void g2lds16_hidden(const void* gptr, void* lds_wave_base) {
  const uint32_t la = (uint32_t)(uintptr_t)lds_wave_base;
  // (one wait state between the write of m0 and the copy that reads it)
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(gptr), "s"(la)
               : "memory", "m0");
}

// s_waitcnt vmcnt(N) with the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

// Workgroup barrier for LDS tiles filled by prefetch. __syncthreads() (and
// any LDS release fence) makes every wave wait for all of its outstanding
// global loads, because global_load_lds writes LDS under the vector-memory
// counter; that would drain a prefetch ring at each tile. This barrier waits
// only for the wave's own LDS reads and writes; the caller makes the
// global_load_lds data of the tile it is about to read complete with
// wait_vmcnt before it. The memory clobber keeps the compiler from moving
// memory accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Load through the constant address space: for data that no thread writes
// while the kernel runs, read at a wave-uniform address. The compiler then
// uses a scalar load (counted by lgkmcnt), which leaves the vmcnt
// accounting of in-flight tile loads untouched.
template <typename T>
__device__ __forceinline__ T ld_const(const T* p) {
  return *(const __attribute__((address_space(4))) T*)(p);
}
// int2 through one 8-byte scalar load (the vector type has no constructor
// from a constant-address-space lvalue)
__device__ __forceinline__ int2 ld_const(const int2* p) {
  const int64_t v = *(const __attribute__((address_space(4))) int64_t*)(p);
  return make_int2((int)(uint32_t)v, (int)(uint32_t)(v >> 32));
}

__device__ __forceinline__ int clampi(int x, int lo, int hi) { return x < lo ? lo : (x > hi ? hi : x); }

}  // namespace hsa
