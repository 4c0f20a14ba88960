// Device-side helpers shared by the gfx950 kernels of libgraphleap.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gl {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// storage types
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b16) {
  return __uint_as_float(b16 << 16);
}

// round-to-nearest-even float -> bf16 bits (NaN kept quiet)
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// 8 bf16 values packed in a uint4 <-> 8 floats
__device__ __forceinline__ void unpack_bf16x8(const uint4& v, float* f) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

__device__ __forceinline__ uint4 pack_bf16x8(const float* f) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = f32_to_bf16_bits(f[2 * i]) | (f32_to_bf16_bits(f[2 * i + 1]) << 16);
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// ---------------------------------------------------------------------------
// MFMA wrappers.  For both instructions the 16x16 fp32 result sits in 4 VGPRs:
// lane l holds D[4*(l/16) + v][l%16] in element v.  Operand lane l supplies row
// (A) or column (B) l%16; the lane group l/16 selects the slice of the
// contraction axis.  Callers give A and B the same slice per lane group, so
// the exact order of the contraction inside the instruction does not matter.
// ---------------------------------------------------------------------------
__device__ __forceinline__ f32x4 mfma_bf16(const uint4& a, const uint4& b, f32x4 acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
}

__device__ __forceinline__ f32x4 mfma_f32(float a, float b, f32x4 acc) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// compare-exchange helpers on packed unsigned keys
// ---------------------------------------------------------------------------
__device__ __forceinline__ void cas_asc(uint32_t& a, uint32_t& b) {
  const uint32_t lo = min(a, b), hi = max(a, b);
  a = lo;
  b = hi;
}

// Bitonic sort of a register array, ascending.  N is a power of two and every
// index is a compile-time constant after unrolling.
template <int N>
__device__ __forceinline__ void sort_regs_asc(uint32_t* v) {
#pragma unroll
  for (int k = 2; k <= N; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const int l = i ^ j;
        if (l > i) {
          if ((i & k) == 0) cas_asc(v[i], v[l]);
          else cas_asc(v[l], v[i]);
        }
      }
    }
  }
}

}  // namespace gl
