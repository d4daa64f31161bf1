// Device-side helpers shared by the gfx950 kernels of libhydra.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hydra {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

// D = A * B + C on one 16x16 output tile with a K = 32 step, bf16 inputs,
// fp32 accumulation.  Lane l supplies row (l % 16) of A and column (l % 16)
// of B, each as eight consecutive k values of k-group (l / 16); the result
// lane l holds is D[4 * (l / 16) + i][l % 16], i = 0..3.
__device__ __forceinline__ f32x4_t mfma16(const uint4& a, const uint4& b, const f32x4_t& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                 c, 0, 0, 0);
}

// Raw buffer resource over [base, base + bytes): a 16-byte load whose byte
// offset lies at or past `bytes` returns zeros instead of touching memory,
// which is how ragged tiles and K tails are zero-filled.
typedef __attribute__((__vector_size__(4 * sizeof(int)))) int i32x4_t;
constexpr int kOutOfRange = int(0x80000000u);  // offset that is always past the range

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, int byte_off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0));
}

// Raw buffer descriptor as four dwords (base, base_hi | stride 0, bytes,
// format), for use by inline assembly.  All fields must be wave-uniform.
__device__ __forceinline__ i32x4_t make_rsrc_raw(const void* base, uint32_t bytes) {
  const uint64_t p = (uint64_t)(uintptr_t)base;
  return i32x4_t{(int)(uint32_t)p, (int)((uint32_t)(p >> 32) & 0xFFFFu), (int)bytes, 0x00020000};
}

// 16 bytes per lane copied from a buffer straight into LDS (no register
// staging): lane i writes [lds_base + 16 i, lds_base + 16 i + 16).  lds_base
// must be wave-uniform; an out-of-range offset writes zeros.  Issued through
// inline assembly so that the compiler does not add its own (conservative)
// waits for it: the callers wait explicitly with wait_vm_barrier before any
// wave reads the copied data.  M0 is set here; nothing else in these kernels
// uses M0.
__device__ __forceinline__ void dma16(const i32x4_t& rsrc, const void* lds_base, int byte_off) {
  const uint32_t lds_addr = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)lds_base;
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :: "s"(lds_addr), "v"(byte_off), "s"(rsrc) : "memory");
}

// Wait until at most N of this wave's vector-memory loads (including LDS
// copies) are still in flight and all of its LDS operations are done, then
// join the workgroup barrier.  The empty asm statements stop the compiler
// from moving memory accesses across the barrier.
template <int N>
__device__ __forceinline__ void wait_vm_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt is a 6-bit field");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | (((N >> 4) & 3) << 14));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;

// D = A * B + C on one 32x32 output tile with a K = 16 step, bf16 inputs,
// fp32 accumulation.  Lane l supplies row (l % 32) of A and column (l % 32)
// of B, each as eight consecutive k values of k-group (l / 32); element
// 4 i + e of the result lane l holds is D[8 i + 4 (l / 32) + e][l % 32].
__device__ __forceinline__ f32x16_t mfma32(const uint4& a, const uint4& b, const f32x16_t& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                 c, 0, 0, 0);
}

__device__ __forceinline__ float bf16_to_f32(uint32_t u16) { return __uint_as_float(u16 << 16); }

// float -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// e^x and ln x from the hardware base-2 transcendental units:
// e^x = 2^(x log2 e), ln x = log2(x) ln 2.
constexpr float kLog2e = 1.4426950408889634f;
__device__ __forceinline__ float exp_e(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }
__device__ __forceinline__ float log_e(float x) { return __builtin_amdgcn_logf(x) * 0.6931471805599453f; }

// Merge two (running max, sum of exp(v - max)) pairs.  The products and the
// sum are rounded separately (no contraction), so merge(a, b) == merge(b, a)
// bit for bit.  An empty side has m = -inf and s = 0.
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) {
    m = mn;
    s = 0.f;
    return;
  }
  s = __fadd_rn(__fmul_rn(s, exp_e(m - mn)), __fmul_rn(s2, exp_e(m2 - mn)));
  m = mn;
}

}  // namespace hydra
