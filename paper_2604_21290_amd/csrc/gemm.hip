// Tiled MFMA GEMM for the fully connected layers of the path:
//   out[R, Cout] = act_out(act_in(A)[R, K] W[Cout, K]^T + b) + residual
//   * the MRConv update over materialised [x | m] rows for wide channels
//     (Sec. II-A Eq. 3; the W_x / W_m split of Sec. IV-C2 is the two halves of
//     the contraction axis), where the fused MRConv tile would stream all of W
//     through every 16- or 32-node workgroup;
//   * FC1, FC2 + residual and the FFN of the full ViG block (Eq. 11, 14, 15):
//     act_in = GELU gives sigma(U~) W_out^T, act_out = GELU the FFN's hidden
//     layer, residual the two skip connections.
// A workgroup owns a 128 x 128 output tile, so W is read once per 128 rows
// and A once per 128 output channels.
//   - 4 waves in a 2 x 2 layout; each wave holds a 64 x 64 accumulator block
//     (4 x 4 MFMA tiles of 16 x 16) in registers.
//   - The contraction runs in steps of 64 bytes per row (32 bf16 or 16 fp32
//     channels).  Both operands are K-contiguous, so one 16-byte vector per
//     lane is exactly an MFMA operand slice.  A step's A and B tiles
//     (128 rows x 64 bytes each) pass through LDS, double-buffered: the
//     global loads of step s+1 are in flight while step s is multiplied, and
//     one barrier per step separates the buffers.
//   - act_in is applied to A's elements as they are staged (fp32, rounded back
//     to the storage type, as if the caller had stored sigma(A)).
//   - Epilogue in fp32: + bias, act_out, + residual, rounded once.
#include "gl_device.h"
#include "gl_kernels.h"

namespace gl {

constexpr int kGmBM = 128, kGmBN = 128, kGmThreads = 256;
constexpr int kGmStep = 64;                // bytes per row per contraction step
constexpr int kGmRow = kGmStep + 16;       // LDS row stride (spreads rows over banks)
constexpr int kGmTile = kGmBM * kGmRow;    // one operand tile: 10 KB

size_t gemm_smem_bytes() { return (size_t)4 * kGmTile; }

// GELU of the 16-byte vector's elements, rounded back to the storage type.
template <int DT>
__device__ __forceinline__ u32x4 gelu_vec(u32x4 v) {
  if (DT) {
    float f[8];
    unpack_bf16x8(__builtin_bit_cast(uint4, v), f);
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = gelu_f32(f[i]);
    return __builtin_bit_cast(u32x4, pack_bf16x8(f));
  }
  float4 f = __builtin_bit_cast(float4, v);
  f.x = gelu_f32(f.x);
  f.y = gelu_f32(f.y);
  f.z = gelu_f32(f.z);
  f.w = gelu_f32(f.w);
  return __builtin_bit_cast(u32x4, f);
}

template <int DT, int ACT_IN, int ACT_OUT>
__global__ __launch_bounds__(kGmThreads) void gemm_nt_kernel(GemmArgs a) {
  extern __shared__ __align__(16) char smem[];
  constexpr int ES = DT ? 2 : 4;
  const int R = a.R, K = a.K, Cout = a.Cout;
  const int rowb = K * ES;                  // a multiple of 16
  const int nsteps = (rowb + kGmStep - 1) / kGmStep;
  const int ntn = (Cout + kGmBN - 1) / kGmBN;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = blk / ntn, nt = blk - mt * ntn;
  const int m0 = mt * kGmBM, n0 = nt * kGmBN;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, t = lane & 15;
  const int wm = w >> 1, wn = w & 1;

  // staging: vector v = tid + 256 i of a tile is row v / 4, 16-byte slot v % 4
  const char* Ab = static_cast<const char*>(a.A);
  const char* Wb = static_cast<const char*>(a.W);
  const char* ag[2];
  const char* bg[2];
  int slot[2], lo[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int v = tid + kGmThreads * i, r = v >> 2;
    slot[i] = (v & 3) * 16;
    ag[i] = Ab + (size_t)min(m0 + r, R - 1) * rowb + slot[i];
    bg[i] = Wb + (size_t)min(n0 + r, Cout - 1) * rowb + slot[i];
    lo[i] = r * kGmRow + slot[i];
  }
  u32x4 ra[2], rb[2];
  auto gload = [&](int s) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const bool in = s * kGmStep + slot[i] < rowb;
      const int off = in ? s * kGmStep : 0;
      ra[i] = *reinterpret_cast<const u32x4*>(ag[i] + off);
      rb[i] = *reinterpret_cast<const u32x4*>(bg[i] + off);
      if (!in) ra[i] = rb[i] = u32x4{0, 0, 0, 0};
    }
  };
  auto act = [&]() {
    if (ACT_IN) {
#pragma unroll
      for (int i = 0; i < 2; ++i) ra[i] = gelu_vec<DT>(ra[i]);
    }
  };
  auto sstore = [&](int buf) {
    char* sa = smem + buf * 2 * kGmTile;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      *reinterpret_cast<u32x4*>(sa + lo[i]) = ra[i];
      *reinterpret_cast<u32x4*>(sa + kGmTile + lo[i]) = rb[i];
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  gload(0);
  act();
  sstore(0);
  __syncthreads();
  for (int s = 0; s < nsteps; ++s) {
    if (s + 1 < nsteps) gload(s + 1);
    const char* sa = smem + (s & 1) * 2 * kGmTile;
    uint4 af[4], bf[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      af[i] = *reinterpret_cast<const uint4*>(sa + (wm * 64 + i * 16 + t) * kGmRow + g * 16);
      bf[i] = *reinterpret_cast<const uint4*>(sa + kGmTile + (wn * 64 + i * 16 + t) * kGmRow + g * 16);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (DT) {
          acc[i][j] = mfma_bf16(af[i], bf[j], acc[i][j]);
        } else {
          const float4 x4 = __builtin_bit_cast(float4, af[i]);
          const float4 y4 = __builtin_bit_cast(float4, bf[j]);
          acc[i][j] = mfma_f32(x4.x, y4.x, acc[i][j]);
          acc[i][j] = mfma_f32(x4.y, y4.y, acc[i][j]);
          acc[i][j] = mfma_f32(x4.z, y4.z, acc[i][j]);
          acc[i][j] = mfma_f32(x4.w, y4.w, acc[i][j]);
        }
      }
    if (s + 1 < nsteps) {
      act();
      sstore((s + 1) & 1);
    }
    __syncthreads();
  }

  // -- epilogue: lane (g, t) of tile (i, j) holds rows 4g..4g+3, column t --------
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n = n0 + wn * 64 + j * 16 + t;
    if (n >= Cout) continue;
    float bn = 0.f;
    if (a.bias) {
      bn = DT ? bf16_bits_to_f32(static_cast<const uint16_t*>(a.bias)[n])
              : static_cast<const float*>(a.bias)[n];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = m0 + wm * 64 + i * 16 + 4 * g + v;
        if (row >= R) continue;
        float y = acc[i][j][v] + bn;
        if (ACT_OUT) y = gelu_f32(y);
        const size_t o = (size_t)row * Cout + n;
        if (a.residual) {
          y += DT ? bf16_bits_to_f32(static_cast<const uint16_t*>(a.residual)[o])
                  : static_cast<const float*>(a.residual)[o];
        }
        if (DT) static_cast<uint16_t*>(a.out)[o] = (uint16_t)f32_to_bf16_bits(y);
        else static_cast<float*>(a.out)[o] = y;
      }
  }
}

hipError_t launch_gemm_nt(const GemmArgs& a, int dt_bf16, hipStream_t stream, hipEvent_t ev0,
                          hipEvent_t ev1) {
  const int nm = (a.R + kGmBM - 1) / kGmBM, nn = (a.Cout + kGmBN - 1) / kGmBN;
  const dim3 grid(nm * nn), block(kGmThreads);
  const int v = (dt_bf16 ? 4 : 0) + (a.act_in ? 2 : 0) + (a.act_out ? 1 : 0);
  static const void* const fns[8] = {
      (const void*)&gemm_nt_kernel<0, 0, 0>, (const void*)&gemm_nt_kernel<0, 0, 1>,
      (const void*)&gemm_nt_kernel<0, 1, 0>, (const void*)&gemm_nt_kernel<0, 1, 1>,
      (const void*)&gemm_nt_kernel<1, 0, 0>, (const void*)&gemm_nt_kernel<1, 0, 1>,
      (const void*)&gemm_nt_kernel<1, 1, 0>, (const void*)&gemm_nt_kernel<1, 1, 1>};
  const void* fn = fns[v];
  return launch_with_smem(fn, grid, block, gemm_smem_bytes(), stream, ev0, ev1, a);
}

}  // namespace gl
