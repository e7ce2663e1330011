// Device-side helpers shared by the gfx950 kernels of the group-masked linear layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gm {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// ---------------------------------------------------------------- bf16 <-> fp32

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

// Round-to-nearest-even fp32 -> bf16 (NaN stays a quiet NaN), one
// v_cvt_pk_bf16_f32 per pair of values.
typedef float f32x2_cvt_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_cvt_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_cvt_t{lo, hi}, bf16x2_cvt_t));
}
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) { return __builtin_bit_cast(uint16_t, __bf16(f)); }

// ---------------------------------------------------------------- 16-byte moves

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ __forceinline__ u32x4 zero16() { return u32x4{0u, 0u, 0u, 0u}; }

// Multiply the 8 bf16 values of a 16-byte vector by s (fp32), rounding back to bf16.
__device__ __forceinline__ u32x4 scale_bf16x8(u32x4 v, float s) {
  u32x4 r;
#pragma unroll
  for (int q = 0; q < 4; ++q) r[q] = pack_bf16x2(bf16_lo(v[q]) * s, bf16_hi(v[q]) * s);
  return r;
}

// Transpose an 8 x 8 block of 16-bit values held as 8 vectors of 8:
// out[c] element j = in[j] element c.
__device__ __forceinline__ void transpose8x8_b16(const u32x4 (&in)[8], u32x4 (&out)[8]) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int q = c >> 1;
    const bool hi = c & 1;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      uint32_t a = in[2 * p][q];
      uint32_t b = in[2 * p + 1][q];
      out[c][p] = hi ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
    }
  }
}

// ---------------------------------------------------------------- MFMA

// v_mfma_f32_16x16x32_bf16: C[16x16] += A[16x32] B[32x16].
// Lane l supplies A row (l % 16), k slice [8 (l/16), 8 (l/16) + 8) and
// B column (l % 16) over the same k slice; it receives C rows 4 (l/16) + j,
// j = 0..3, of column (l % 16).
//
// The MFMA is written in assembly with the accumulator as one tied operand.  With the builtin, this clang often gives
// the result a different register from the accumulator input and moves it
// back (up to one move per MFMA with 64 live accumulators), which cuts the
// issue rate of a 128 x 128 wave tile by a third.  AGPR selects the register
// file of the accumulator: a wave tile keeps most accumulators in AGPRs and
// the rest in arch VGPRs, which leaves the register allocator room in both.
// mfma_init starts an accumulator (C input 0), so no accumulator is written
// by other instructions before the K-loop.  The compiler does not see these
// instructions as MFMAs, so its hazard padding does not cover them; readers
// of the accumulators wait for acc_drain().
template <bool AGPR>
__device__ __forceinline__ void mfma_acc(f32x4& acc, const u32x4& a, const u32x4& b) {
  if constexpr (AGPR)
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
  else
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(acc) : "v"(a), "v"(b));
}

template <bool AGPR>
__device__ __forceinline__ void mfma_init(f32x4& acc, const u32x4& a, const u32x4& b) {
  if constexpr (AGPR)
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=a"(acc) : "v"(a), "v"(b));
  else
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=&v"(acc) : "v"(a), "v"(b));
}

template <bool AGPR>
__device__ __forceinline__ void acc_pin(f32x4& acc) {
  if constexpr (AGPR)
    asm volatile("" : "+a"(acc));
  else
    asm volatile("" : "+v"(acc));
}

// After the last MFMA: 24 wait states (more than the longest MFMA write ->
// VALU read dependency), then every accumulator passes through an empty
// statement that orders its readers after the wait.  Accumulator i lives in
// AGPRs when i < N_AGPR.
template <int N_AGPR, int N>
__device__ __forceinline__ void acc_drain(f32x4 (&acc)[N]) {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
#pragma unroll
  for (int i = 0; i < N; ++i) {
    if (i < N_AGPR) acc_pin<true>(acc[i]); else acc_pin<false>(acc[i]);
  }
}

}  // namespace gm
