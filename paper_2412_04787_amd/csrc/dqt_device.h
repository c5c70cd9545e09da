// Device-side helpers shared by the libdqt kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dqt {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef int i32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kWave = 64;

// ---------------------------------------------------------------- bf16
// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}
// Two fp32 -> packed bf16 pair (lo in bits 0-15), round to nearest even; one
// v_cvt_pk_bf16_f32 on gfx950.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) {
  return __uint_as_float(b << 16);
}

// ---------------------------------------------------------------- e4m3
// OCP E4M3 ("fn"): 1 sign, 4 exponent (bias 7), 3 fraction bits, max 448.
// Round to nearest even, saturate to +-448, keep the sign of zero.
__device__ __forceinline__ uint32_t f32_to_e4m3(float v) {
  const uint32_t sign = (__float_as_uint(v) >> 24) & 0x80u;
  const float a = fabsf(v);
  uint32_t code;
  if (!(a < 448.0f)) {
    code = 0x7Eu;
  } else if (a < 0.015625f) {                  // below 2^-6: subnormal grid 2^-9
    code = (uint32_t)rintf(a * 512.0f);        // exact scaling, ties to even
  } else {
    const uint32_t ab = __float_as_uint(a);
    const uint32_t r = ab + 0x7FFFFu + ((ab >> 20) & 1u);  // RNE to 3 fraction bits
    code = (r >> 20) - (120u << 3);                       // exponent bias 127 -> 7
    code = code > 0x7Eu ? 0x7Eu : code;
  }
  return code | sign;
}

// Four fp32 values -> four OCP e4m3 bytes (value i in byte i), each equal to
// f32_to_e4m3 of the value: the hardware conversion (round to nearest even;
// equal to f32_to_e4m3 for every fp32 of magnitude below 449, all bit
// patterns compared on the GPU) after |v| is clamped to 448 with v's sign,
// which gives f32_to_e4m3's saturation of large values and of NaN.
__device__ __forceinline__ float e4m3_sat(float v) { return copysignf(fminf(fabsf(v), 448.0f), v); }
__device__ __forceinline__ uint32_t f32x4_to_e4m3x4(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(e4m3_sat(a), e4m3_sat(b), 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(e4m3_sat(c), e4m3_sat(d), w, true);
  return (uint32_t)w;
}

// Four fp32 values -> four int8 codes clip(round(v), -128, 127) (value i in
// byte i; round to nearest even; NaN gives -128 like fmaxf): after the clip,
// adding 1.5 * 2^23 rounds to an integer to nearest even and leaves it, in
// two's complement, in the low byte of the sum's bits.
__device__ __forceinline__ uint32_t f32x4_to_i8x4(float a, float b, float c, float d) {
  auto q = [](float v) { return __float_as_uint(fminf(fmaxf(v, -128.0f), 127.0f) + 12582912.0f); };
  return (q(a) & 0xFFu) | ((q(b) & 0xFFu) << 8) | ((q(c) & 0xFFu) << 16) | (q(d) << 24);
}

// E4M3 byte -> fp32 (exact).  NaN codes are not produced by this library.
__device__ __forceinline__ float e4m3_to_f32(uint32_t c) {
  const uint32_t e = (c >> 3) & 0xFu, m = c & 7u;
  float mag;
  if (e == 0) {
    mag = (float)m * 0.001953125f;             // m * 2^-9
  } else {
    mag = __uint_as_float(((e + 120u) << 23) | (m << 20));
  }
  return (c & 0x80u) ? -mag : mag;
}

// ---------------------------------------------------------------- ternary
// Four 2-bit codes of one byte, one per output byte (bits 0-1 of each).
__device__ __forceinline__ uint32_t spread_codes(uint32_t b) {
  return (b & 3u) | ((b << 6) & 0x300u) | ((b << 12) & 0x30000u) | ((b << 18) & 0x3000000u);
}
// Code (0, 1, 2) -> int8 (-1, 0, 1), four at a time, via byte permute.
__device__ __forceinline__ uint32_t codes_to_i8x4(uint32_t spread) {
  return __builtin_amdgcn_perm(0u, 0x000100FFu, spread);
}
// Code (0, 1, 2) -> e4m3 (-1.0, 0, +1.0) bytes (0xB8, 0x00, 0x38).
__device__ __forceinline__ uint32_t codes_to_e4m3x4(uint32_t spread) {
  return __builtin_amdgcn_perm(0u, 0x003800B8u, spread);
}
// Code (0, 1, 2) -> bf16 bits of -1, 0, +1.
__device__ __forceinline__ uint32_t code_to_bf16_bits(uint32_t code) {
  return (uint32_t)((0x00003F800000BF80ull >> (16u * code)) & 0xFFFFu);
}
__device__ __forceinline__ float code_to_f32(uint32_t code) {
  return (float)((int)code - 1);
}

// ---------------------------------------------------------------- LDS DMA
using lds_u8 = __attribute__((address_space(3))) uint8_t;
// One direct-to-LDS load per lane (global_load_lds_dwordx4: 16 bytes, or
// global_load_lds_dword: 4 bytes); the wave's chunks land at consecutive
// positions from the wave-uniform LDS address l (passed in M0).  Issued as
// inline asm so that the compiler, which cannot tell which LDS bytes the
// DMA writes, does not wait for all outstanding DMA before every later LDS
// access; callers wait for their DMA explicitly (vmcnt) before a barrier
// publishes it.  Nothing else in these kernels uses M0.
__device__ __forceinline__ void dma16(const uint8_t* g, lds_u8* l) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)l);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(g), "s"(m0) : "memory");
}
// The same with the non-temporal hint: for data read once (streaming
// kernels), which should not displace reused lines from the caches.
__device__ __forceinline__ void dma16_nt(const uint8_t* g, lds_u8* l) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)l);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt" : : "v"(g), "s"(m0) : "memory");
}
__device__ __forceinline__ void dma4(const uint8_t* g, lds_u8* l) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)l);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off" : : "v"(g), "s"(m0) : "memory");
}
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// wait until at most n (wave-uniform, 0 <= n <= N) vector memory operations
// of this wave are outstanding
template <int N>
__device__ __forceinline__ void wait_vm_le(int n) {
  if constexpr (N == 0) {
    wait_vm<0>();
  } else {
    if (n >= N) wait_vm<N>();
    else wait_vm_le<N - 1>(n);
  }
}

// ---------------------------------------------------------------- waves
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, kWave));
  return v;
}
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}
__device__ __forceinline__ unsigned long long wave_sum_u64(unsigned long long v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

}  // namespace dqt
