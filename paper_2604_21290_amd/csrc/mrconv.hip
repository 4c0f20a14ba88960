// Fused max-relative graph convolution for gfx950 (Sec. II-A Eq. 2-3; the
// W_x / W_m split of Sec. IV-C2).
//
// One workgroup = 4 waves = TM = 16*RT consecutive nodes of the flattened
// [B*N] node axis.
//   1. gather: for each node and each 16-byte channel vector, the k neighbour
//      key rows are read (consecutive lanes read consecutive vectors of the
//      same row, so every neighbour row is one coalesced burst), their
//      elementwise maximum is taken (exact in the storage type), x_i is
//      subtracted in fp32 and the result rounded once.  [x_i | m_i] is
//      written straight into the LDS A-tile; no edge tensor and no [B,N,2C]
//      concatenation is ever written to memory.
//   2. FC on MFMA: out[TM, Cout] = A[TM, 2C] W^T + b.  The contraction runs
//      over the concatenated axis, so columns 0..C-1 of W meet x_i and
//      columns C..2C-1 meet m_i in one accumulation.  Each wave owns every
//      4th 16-column output tile; W rows are read from L2 as MFMA B operands.
#include "gl_device.h"
#include "gl_kernels.h"

namespace gl {

constexpr int kMrThreads = 256;

template <int DT>
__device__ __forceinline__ void load_vec(const char* p, float* f) {
  if (DT) {
    unpack_bf16x8(*reinterpret_cast<const uint4*>(p), f);
  } else {
    const float4 v = *reinterpret_cast<const float4*>(p);
    f[0] = v.x; f[1] = v.y; f[2] = v.z; f[3] = v.w;
  }
}

template <int DT>
__device__ __forceinline__ void store_vec(char* p, const float* f) {
  if (DT) *reinterpret_cast<uint4*>(p) = pack_bf16x8(f);
  else *reinterpret_cast<float4*>(p) = make_float4(f[0], f[1], f[2], f[3]);
}

template <int DT, int RT>
__global__ __launch_bounds__(kMrThreads) void mrconv_kernel(
    const void* __restrict__ x, const void* __restrict__ keys, const int32_t* __restrict__ idx,
    const void* __restrict__ W, const void* __restrict__ bias, void* __restrict__ out, int R,
    int N, int M, int C, int Cout, int k, int lds_row) {
  extern __shared__ __align__(16) char smem[];
  constexpr int TM = 16 * RT;
  constexpr int ES = DT ? 2 : 4;
  constexpr int VEC = 16 / ES;
  char* sA = smem;
  int32_t* sIdx = reinterpret_cast<int32_t*>(smem + TM * lds_row);

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, t = lane & 15;
  const int row0 = blockIdx.x * TM;
  const int CG = C / VEC;

  // -- neighbour lists of the tile -------------------------------------------
  for (int e = tid; e < TM * k; e += kMrThreads) {
    const int r = e / k, tt = e - r * k, row = row0 + r;
    const int j = row < R ? idx[(size_t)row * k + tt] : 0;
    sIdx[e] = min(max(j, 0), M - 1);
  }
  __syncthreads();

  // -- gather-max into the LDS A-tile ------------------------------------------
  for (int e = tid; e < TM * CG; e += kMrThreads) {
    const int r = e / CG, cg = e - r * CG, row = row0 + r;
    char* dst = sA + r * lds_row + cg * 16;
    float xf[VEC], mx[VEC];
    if (row < R) {
      const int b = row / N;
      load_vec<DT>(static_cast<const char*>(x) + ((size_t)row * C + cg * VEC) * ES, xf);
      const char* kbase = static_cast<const char*>(keys) + ((size_t)b * M * C + cg * VEC) * ES;
#pragma unroll
      for (int i = 0; i < VEC; ++i) mx[i] = -INFINITY;
      const int32_t* nb = sIdx + r * k;
      for (int tt = 0; tt < k; ++tt) {
        float kf[VEC];
        load_vec<DT>(kbase + (size_t)nb[tt] * C * ES, kf);
#pragma unroll
        for (int i = 0; i < VEC; ++i) mx[i] = fmaxf(mx[i], kf[i]);
      }
#pragma unroll
      for (int i = 0; i < VEC; ++i) mx[i] -= xf[i];
    } else {
#pragma unroll
      for (int i = 0; i < VEC; ++i) xf[i] = mx[i] = 0.f;
    }
    store_vec<DT>(dst, xf);
    store_vec<DT>(dst + C * ES, mx);
  }
  __syncthreads();

  // -- FC on MFMA ---------------------------------------------------------------
  const int K2 = 2 * C;
  const int NCT = (Cout + 15) >> 4;
  const char* Wb = static_cast<const char*>(W);
  for (int p = 0; 4 * (4 * p) + w < NCT; ++p) {
    f32x4 acc[RT][4];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int c4 = 0; c4 < 4; ++c4) acc[rt][c4] = f32x4{0.f, 0.f, 0.f, 0.f};
    int nrow[4];
    bool nvalid[4];
#pragma unroll
    for (int c4 = 0; c4 < 4; ++c4) {
      const int ct = w + 4 * (4 * p + c4);
      nrow[c4] = ct * 16 + t;
      nvalid[c4] = ct < NCT && nrow[c4] < Cout;
    }
    if (DT) {
      for (int s = 0; s < (K2 + 31) / 32; ++s) {
        const int kk = s * 32 + g * 8;
        const bool kin = kk < K2;
        uint4 a[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          a[rt] = kin ? *reinterpret_cast<const uint4*>(sA + (rt * 16 + t) * lds_row + kk * 2)
                      : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4) {
          const uint4 bw = (kin && nvalid[c4])
                               ? *reinterpret_cast<const uint4*>(Wb + ((size_t)nrow[c4] * K2 + kk) * 2)
                               : make_uint4(0, 0, 0, 0);
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) acc[rt][c4] = mfma_bf16(a[rt], bw, acc[rt][c4]);
        }
      }
    } else {
      for (int s = 0; s < (K2 + 15) / 16; ++s) {
        const int kk = s * 16 + g * 4;
        const bool kin = kk < K2;
        float4 a[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          a[rt] = kin ? *reinterpret_cast<const float4*>(sA + (rt * 16 + t) * lds_row + kk * 4)
                      : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4) {
          const float4 bw = (kin && nvalid[c4])
                                ? *reinterpret_cast<const float4*>(Wb + ((size_t)nrow[c4] * K2 + kk) * 4)
                                : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) {
            acc[rt][c4] = mfma_f32(a[rt].x, bw.x, acc[rt][c4]);
            acc[rt][c4] = mfma_f32(a[rt].y, bw.y, acc[rt][c4]);
            acc[rt][c4] = mfma_f32(a[rt].z, bw.z, acc[rt][c4]);
            acc[rt][c4] = mfma_f32(a[rt].w, bw.w, acc[rt][c4]);
          }
        }
      }
    }
    // -- epilogue: + bias, round once, store ------------------------------------
#pragma unroll
    for (int c4 = 0; c4 < 4; ++c4) {
      if (!nvalid[c4]) continue;
      const int n = nrow[c4];
      float bn = 0.f;
      if (bias) {
        bn = DT ? bf16_bits_to_f32(static_cast<const uint16_t*>(bias)[n])
                : static_cast<const float*>(bias)[n];
      }
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = row0 + rt * 16 + 4 * g + v;
          if (row >= R) continue;
          const float y = acc[rt][c4][v] + bn;
          if (DT) static_cast<uint16_t*>(out)[(size_t)row * Cout + n] = (uint16_t)f32_to_bf16_bits(y);
          else static_cast<float*>(out)[(size_t)row * Cout + n] = y;
        }
      }
    }
  }
}

int mrconv_lds_row_bytes(int C, int dt_bf16) { return 2 * C * (dt_bf16 ? 2 : 4) + 16; }

int mrconv_row_tiles(int C, int k, int dt_bf16, size_t lds_limit) {
  const int row = mrconv_lds_row_bytes(C, dt_bf16);
  for (int rt = 4; rt >= 1; rt >>= 1) {
    const size_t need = (size_t)16 * rt * (row + 4 * k);
    if (need <= lds_limit) return rt;
  }
  return 0;
}

hipError_t launch_mrconv(const void* x, const void* keys, const int32_t* idx, const void* W,
                         const void* bias, void* out, int B, int N, int M, int C, int Cout, int k,
                         int dt_bf16, int rt, hipStream_t stream) {
  const int R = B * N;
  const int lds_row = mrconv_lds_row_bytes(C, dt_bf16);
  const int TM = 16 * rt;
  const size_t lds = (size_t)TM * (lds_row + 4 * k);
  dim3 grid((R + TM - 1) / TM), block(kMrThreads);
#define GL_MR_LAUNCH(DT, RT)                                                                     \
  do {                                                                                           \
    if (lds > 65536) {                                                                           \
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&mrconv_kernel<DT, RT>),  \
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);  \
      if (e != hipSuccess) return e;                                                             \
    }                                                                                            \
    hipLaunchKernelGGL((mrconv_kernel<DT, RT>), grid, block, lds, stream, x, keys, idx, W, bias, \
                       out, R, N, M, C, Cout, k, lds_row);                                       \
  } while (0)
  if (dt_bf16) {
    if (rt == 4) GL_MR_LAUNCH(1, 4);
    else if (rt == 2) GL_MR_LAUNCH(1, 2);
    else GL_MR_LAUNCH(1, 1);
  } else {
    if (rt == 4) GL_MR_LAUNCH(0, 4);
    else if (rt == 2) GL_MR_LAUNCH(0, 2);
    else GL_MR_LAUNCH(0, 1);
  }
#undef GL_MR_LAUNCH
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// r x r average pooling of the node grid into key nodes (pyramid stages).
// One thread per (image, key node, 16-byte channel vector).
// ---------------------------------------------------------------------------
template <int DT>
__global__ __launch_bounds__(256) void pool_kernel(const void* __restrict__ x,
                                                   void* __restrict__ keys, int B, int H, int W,
                                                   int C, int r) {
  constexpr int ES = DT ? 2 : 4;
  constexpr int VEC = 16 / ES;
  const int CG = C / VEC;
  const int Wr = W / r, Mo = (H / r) * Wr;
  const long total = (long)B * Mo * CG;
  const long e = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= total) return;
  const int cg = (int)(e % CG);
  const int o = (int)((e / CG) % Mo);
  const int b = (int)(e / ((long)CG * Mo));
  const int p = o / Wr, q = o - p * Wr;
  float acc[VEC];
#pragma unroll
  for (int i = 0; i < VEC; ++i) acc[i] = 0.f;
  const char* xb = static_cast<const char*>(x) + ((size_t)b * H * W * C + cg * VEC) * ES;
  for (int u = 0; u < r; ++u) {
    for (int v = 0; v < r; ++v) {
      float f[VEC];
      load_vec<DT>(xb + (size_t)((p * r + u) * W + (q * r + v)) * C * ES, f);
#pragma unroll
      for (int i = 0; i < VEC; ++i) acc[i] += f[i];
    }
  }
  const float inv = 1.f / (float)(r * r);
#pragma unroll
  for (int i = 0; i < VEC; ++i) acc[i] *= inv;
  store_vec<DT>(static_cast<char*>(keys) + ((size_t)(b * Mo + o) * C + cg * VEC) * ES, acc);
}

hipError_t launch_pool(const void* x, void* keys, int B, int H, int W, int C, int r, int dt_bf16,
                       hipStream_t stream) {
  const int VEC = dt_bf16 ? 8 : 4;
  const long total = (long)B * (H / r) * (W / r) * (C / VEC);
  dim3 grid((unsigned)((total + 255) / 256)), block(256);
  if (dt_bf16) hipLaunchKernelGGL(pool_kernel<1>, grid, block, 0, stream, x, keys, B, H, W, C, r);
  else hipLaunchKernelGGL(pool_kernel<0>, grid, block, 0, stream, x, keys, B, H, W, C, r);
  return hipGetLastError();
}

}  // namespace gl
