// Device-side helpers shared by the gfx950 kernels of libgraphleap.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gl {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // register-friendly 16-byte vector

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// storage types
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b16) {
  return __uint_as_float(b16 << 16);
}

// round-to-nearest-even float -> bf16 bits: gfx950 converts in hardware
// (v_cvt_pk_bf16_f32, one instruction for two values)
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

__device__ __forceinline__ uint32_t f32x2_to_bf16x2_bits(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
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
  for (int i = 0; i < 4; ++i) w[i] = f32x2_to_bf16x2_bits(f[2 * i], f[2 * i + 1]);
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
// cross-lane moves inside each row of 16 lanes, as DPP modifiers (no LDS trip)
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, false);
}

// value of lane t ^ j (j = 1, 2, 4 or 8) within the lane's row of 16
__device__ __forceinline__ uint32_t lane_xor16(uint32_t v, int j) {
  switch (j) {
    case 1: return dpp_mov<0xB1>(v);                     // quad_perm [1,0,3,2]
    case 2: return dpp_mov<0x4E>(v);                     // quad_perm [2,3,0,1]
    case 4: return dpp_mov<0x1B>(dpp_mov<0x141>(v));     // half-row mirror, then quad reverse
    default: return dpp_mov<0x128>(v);                   // row rotate by 8
  }
}

// value of lane 15 - t within the lane's row of 16
__device__ __forceinline__ uint32_t lane_reverse16(uint32_t v) { return dpp_mov<0x140>(v); }

// min (low) or max (!low) of v and the value of lane t ^ (1 << j) in the
// lane's row of 16.  The minimum and the maximum each read the partner through
// a DPP move of their own whose unused `old` operand is the operation's
// identity, so the compiler folds each move into its v_min_u32 / v_max_u32
// (every lane's source is inside its row, so `old` never reaches a result).
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_min(uint32_t v, uint32_t src) {
  return min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)0xffffffffu, (int)src, CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_max(uint32_t v, uint32_t src) {
  return max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)src, CTRL, 0xF, 0xF, false));
}
// Both results are computed by every lane (a DPP read in lane-divergent
// control flow would see inactive partners) and the wanted one selected.
__device__ __forceinline__ uint32_t lane_cas16(uint32_t v, int j, bool low) {
  uint32_t mn, mx;
  switch (j) {
    case 0: mn = dpp_min<0xB1>(v, v); mx = dpp_max<0xB1>(v, v); break;    // quad_perm [1,0,3,2]
    case 1: mn = dpp_min<0x4E>(v, v); mx = dpp_max<0x4E>(v, v); break;    // quad_perm [2,3,0,1]
    case 2: {                                                              // half-row mirror,
      const uint32_t m = dpp_mov<0x141>(v);                                // then quad reverse
      mn = dpp_min<0x1B>(v, m);
      mx = dpp_max<0x1B>(v, m);
      break;
    }
    default: mn = dpp_min<0x128>(v, v); mx = dpp_max<0x128>(v, v); break;  // row rotate by 8
  }
  return low ? mn : mx;
}

// value of lane (16*(lane/16) + src) for a wave-uniform src in [0, 16)
__device__ __forceinline__ uint32_t row_broadcast16(uint32_t v, int src, int lane) {
  const uint32_t r0 = __builtin_amdgcn_readlane(v, src);
  const uint32_t r1 = __builtin_amdgcn_readlane(v, 16 + src);
  const uint32_t r2 = __builtin_amdgcn_readlane(v, 32 + src);
  const uint32_t r3 = __builtin_amdgcn_readlane(v, 48 + src);
  const int g = lane >> 4;
  return g == 0 ? r0 : g == 1 ? r1 : g == 2 ? r2 : r3;
}

// sum of squares of the 8 bf16 values in v, added to acc (packed dot products)
__device__ __forceinline__ float sumsq_bf16x8(const uint4& v, float acc) {
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, v.x), __builtin_bit_cast(bf16x2, v.x), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, v.y), __builtin_bit_cast(bf16x2, v.y), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, v.z), __builtin_bit_cast(bf16x2, v.z), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, v.w), __builtin_bit_cast(bf16x2, v.w), acc, false);
  return acc;
}

__device__ __forceinline__ float sumsq_f32x4(const uint4& v, float acc) {
  const float4 f = __builtin_bit_cast(float4, v);
  return fmaf(f.x, f.x, fmaf(f.y, f.y, fmaf(f.z, f.z, fmaf(f.w, f.w, acc))));
}

// erf by Abramowitz and Stegun, Handbook of Mathematical Functions, formula
// 7.1.26: for z >= 0, erf z = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) e^{-z^2}
// with t = 1 / (1 + p z), absolute error at most 1.5e-7; odd in z.  About a
// dozen instructions, against twice that for the library erff, and far below
// the bf16 rounding of every output it feeds.
__device__ __forceinline__ float erf_as7126(float z) {
  const float a = fabsf(z);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, a, 1.f));
  float q = fmaf(t, 1.061405429f, -1.453152027f);
  q = fmaf(t, q, 1.421413741f);
  q = fmaf(t, q, -0.284496736f);
  q = fmaf(t, q, 0.254829592f);
  const float r = fmaf(-(t * q), __expf(-a * a), 1.f);
  return copysignf(r, z);
}

// GELU x * Phi(x) = x/2 (1 + erf(x / sqrt 2)).
__device__ __forceinline__ float gelu_f32(float x) {
  return 0.5f * x * (1.f + erf_as7126(x * 0.70710678118654752f));
}

// 1 / max(||k||, 1e-12) from the squared norm, with the hardware reciprocal
// square root (about 1 ulp); both kNN kernels use it for their key rows.
__device__ __forceinline__ float key_rnorm(float ss) {
  return __builtin_amdgcn_rsqf(fmaxf(ss, 1e-24f));
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
