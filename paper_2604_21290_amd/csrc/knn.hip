// Fused dilated kNN graph build for gfx950 (Sec. II-B Eq. 4; Sec. IV-B; Alg. 2).
//
// One workgroup = 4 waves = 16 query rows of one image.  Keys are processed in
// chunks of 256 (16 MFMA tiles of 16 keys):
//   1. Gram tile on MFMA: G = Q K^T over the raw stored values (bf16 products
//      are exact in fp32), while the lanes also accumulate the key rows'
//      squared norms from the same operand registers;
//   2. distance epilogue in fp32 on the accumulator registers:
//      d1 = (1 + n_j) - 2 r_i r_j G_ij, which is the squared distance between
//      the L2-normalised rows minus the per-row constant n_i - 1 (rank
//      preserving within a row); it is quantised to fixed point and packed
//      with the key index into one 32-bit key (distance high, index low), so
//      a plain unsigned compare orders by (distance, index);
//   3. the packed keys of the chunk go to an LDS strip [16][256];
//   4. each query row is owned by 16 lanes of one wave; the row's running
//      sorted list of the K' = k*dilation smallest keys lives in registers
//      (element e = lane + 16*reg).  Chunk candidates below the list's K'-th
//      key pass a threshold filter, are sorted per lane, and are merged 16 at
//      a time (one per lane): bitonic sort across the 16 lanes, then a
//      bitonic merge into the list that keeps its K' smallest.
// The N x M distance matrix never leaves the chip; the only global write is
// idx[B, N, k] (ranks 0, d, 2d, ... of the list).
#include "gl_device.h"
#include "gl_kernels.h"

namespace gl {

constexpr int kKnnRows = 16;     // query rows per workgroup
constexpr int kKnnChunk = 256;   // keys per chunk
constexpr int kKnnThreads = 256;

// Sort one value per lane across each aligned group of 16 lanes (ascending).
__device__ __forceinline__ uint32_t sort16_lanes(uint32_t c, int t) {
#pragma unroll
  for (int s = 1; s <= 4; ++s) {
#pragma unroll
    for (int j = s - 1; j >= 0; --j) {
      const uint32_t p = __shfl_xor(c, 1 << j);
      const bool up = ((t >> s) & 1) == 0;
      const bool lower = ((t >> j) & 1) == 0;
      c = (lower == up) ? min(c, p) : max(c, p);
    }
  }
  return c;
}

// Merge a sorted run of 16 (one per lane, `c`) into the sorted list L of
// 16*R elements (element e = t + 16*a), keeping the 16*R smallest, sorted.
template <int R>
__device__ __forceinline__ void merge16_into_list(uint32_t* L, uint32_t c, int lane, int t) {
  // half-cleaner against the reversed run: only the last 16 list slots can change
  const uint32_t crev = __shfl(c, (lane & 48) | (15 - t));
  L[R - 1] = min(L[R - 1], crev);
  // bitonic merge: strides 16*h inside a lane, then 8,4,2,1 across lanes
#pragma unroll
  for (int h = R / 2; h >= 1; h >>= 1) {
#pragma unroll
    for (int a = 0; a < R; ++a)
      if ((a & h) == 0) cas_asc(L[a], L[a + h]);
  }
#pragma unroll
  for (int j = 3; j >= 0; --j) {
#pragma unroll
    for (int a = 0; a < R; ++a) {
      const uint32_t p = __shfl_xor(L[a], 1 << j);
      L[a] = ((t >> j) & 1) ? max(L[a], p) : min(L[a], p);
    }
  }
}

template <int R>
__device__ __forceinline__ uint32_t list_element(const uint32_t* L, int e, int lane) {
  uint32_t v = L[0];
#pragma unroll
  for (int a = 1; a < R; ++a)
    if ((e >> 4) == a) v = L[a];
  return __shfl(v, (lane & 48) | (e & 15));
}

template <int DT, int R>
__global__ __launch_bounds__(kKnnThreads) void knn_kernel(
    const void* __restrict__ xv, const void* __restrict__ kv, int N, int C, int M, int k,
    int dil, int KK, int ib, float qscale, uint32_t qmax, int32_t* __restrict__ idx_out) {
  __shared__ float s_qr[kKnnRows];
  __shared__ uint32_t s_strip[kKnnRows][kKnnChunk];

  constexpr int ES = DT ? 2 : 4;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, t = lane & 15;
  const int b = blockIdx.y, row0 = blockIdx.x * kKnnRows;
  const char* xb = static_cast<const char*>(xv) + (size_t)b * N * C * ES;
  const char* kb = static_cast<const char*>(kv) + (size_t)b * M * C * ES;

  // -- query inverse norms, 16 threads per row --------------------------------
  {
    const int r = tid >> 4, part = tid & 15;
    const int row = min(row0 + r, N - 1);
    float ss = 0.f;
    if (DT) {
      const uint16_t* p = reinterpret_cast<const uint16_t*>(xb) + (size_t)row * C;
      for (int c = part * 8; c < C; c += 128) {
        float f[8];
        unpack_bf16x8(*reinterpret_cast<const uint4*>(p + c), f);
#pragma unroll
        for (int e = 0; e < 8; ++e) ss = fmaf(f[e], f[e], ss);
      }
    } else {
      const float* p = reinterpret_cast<const float*>(xb) + (size_t)row * C;
      for (int c = part * 4; c < C; c += 64) {
        const float4 v = *reinterpret_cast<const float4*>(p + c);
        ss = fmaf(v.x, v.x, ss);
        ss = fmaf(v.y, v.y, ss);
        ss = fmaf(v.z, v.z, ss);
        ss = fmaf(v.w, v.w, ss);
      }
    }
    ss += __shfl_xor(ss, 8);
    ss += __shfl_xor(ss, 4);
    ss += __shfl_xor(ss, 2);
    ss += __shfl_xor(ss, 1);
    if (part == 0) s_qr[r] = 1.f / fmaxf(sqrtf(ss), 1e-12f);
  }
  __syncthreads();
  float qr[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) qr[v] = s_qr[4 * g + v];

  const int arow = min(row0 + t, N - 1);  // MFMA A-operand row of this lane
  uint32_t L[R];
#pragma unroll
  for (int a = 0; a < R; ++a) L[a] = 0xffffffffu;
  uint32_t tau = 0xffffffffu;
  const int ksteps = DT ? (C + 31) / 32 : (C + 15) / 16;

  for (int chunk0 = 0; chunk0 < M; chunk0 += kKnnChunk) {
    const int nvalid = min(kKnnChunk, M - chunk0);
    const int ntiles = (nvalid + 15) >> 4;
    // -- Gram + epilogue: wave w takes tiles w, w+4, ... -------------------------
    for (int tt = w; tt < ntiles; tt += 4) {
      const int key0 = chunk0 + tt * 16;
      const int krow = min(key0 + t, M - 1);
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      float ss = 0.f;
      if (DT) {
        const uint16_t* qa = reinterpret_cast<const uint16_t*>(xb) + (size_t)arow * C;
        const uint16_t* kp = reinterpret_cast<const uint16_t*>(kb) + (size_t)krow * C;
        for (int s = 0; s < ksteps; ++s) {
          const int c = s * 32 + g * 8;
          uint4 a = make_uint4(0, 0, 0, 0), bb = make_uint4(0, 0, 0, 0);
          if (c < C) {
            a = *reinterpret_cast<const uint4*>(qa + c);
            bb = *reinterpret_cast<const uint4*>(kp + c);
          }
          acc = mfma_bf16(a, bb, acc);
          float f[8];
          unpack_bf16x8(bb, f);
#pragma unroll
          for (int e = 0; e < 8; ++e) ss = fmaf(f[e], f[e], ss);
        }
      } else {
        const float* qa = reinterpret_cast<const float*>(xb) + (size_t)arow * C;
        const float* kp = reinterpret_cast<const float*>(kb) + (size_t)krow * C;
        for (int s = 0; s < ksteps; ++s) {
          const int c = s * 16 + g * 4;
          float4 a = make_float4(0.f, 0.f, 0.f, 0.f), bb = a;
          if (c < C) {
            a = *reinterpret_cast<const float4*>(qa + c);
            bb = *reinterpret_cast<const float4*>(kp + c);
          }
          acc = mfma_f32(a.x, bb.x, acc);
          acc = mfma_f32(a.y, bb.y, acc);
          acc = mfma_f32(a.z, bb.z, acc);
          acc = mfma_f32(a.w, bb.w, acc);
          ss = fmaf(bb.x, bb.x, ss);
          ss = fmaf(bb.y, bb.y, ss);
          ss = fmaf(bb.z, bb.z, ss);
          ss = fmaf(bb.w, bb.w, ss);
        }
      }
      ss += __shfl_xor(ss, 16);
      ss += __shfl_xor(ss, 32);
      const int j = key0 + t;
      const float m2rj = -2.f / fmaxf(sqrtf(ss), 1e-12f);
      const float base = ss > 0.f ? 2.f : 1.f;  // 1 + n_j
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float d1 = fmaf(acc[v] * m2rj, qr[v], base);
        uint32_t q = (uint32_t)(fmaxf(d1, 0.f) * qscale);
        q = min(q, qmax);
        s_strip[4 * g + v][tt * 16 + t] = (j < M) ? ((q << ib) | (uint32_t)j) : 0xffffffffu;
      }
    }
    __syncthreads();
    // -- selection: wave w owns rows 4w .. 4w+3, lanes 16g..16g+15 own row 4w+g --
    uint32_t v[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const int col = t + 16 * m;
      v[m] = (col < nvalid) ? s_strip[4 * w + g][col] : 0xffffffffu;
    }
    __syncthreads();  // the strip is free for the next chunk

    bool pass = false;
#pragma unroll
    for (int m = 0; m < 16; ++m) pass |= v[m] < tau;
    if (__any(pass)) {
#pragma unroll
      for (int m = 0; m < 16; ++m) v[m] = v[m] < tau ? v[m] : 0xffffffffu;
      sort_regs_asc<16>(v);
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        if (!__any(v[m] < tau)) break;
        const uint32_t c = sort16_lanes(v[m], t);
        merge16_into_list<R>(L, c, lane, t);
        tau = list_element<R>(L, KK - 1, lane);
      }
    }
  }

  // -- dilation and output: idx[b, row, e/dil] = index of list element e ------
  const int row = row0 + 4 * w + g;
  if (row < N) {
    int32_t* o = idx_out + ((size_t)b * N + row) * k;
    const uint32_t mask = (1u << ib) - 1u;
#pragma unroll
    for (int a = 0; a < R; ++a) {
      const int e = t + 16 * a;
      if (e < KK && (e % dil) == 0) o[e / dil] = (int32_t)(L[a] & mask);
    }
  }
}

hipError_t launch_knn(const void* x, const void* keys, int B, int N, int C, int M, int k,
                      int dil, int dt_bf16, int32_t* idx_out, hipStream_t stream) {
  const int KK = k * dil;
  int ib = 1;
  while ((1 << ib) < M) ++ib;
  const float qscale = (float)(1u << (30 - ib));
  const uint32_t qmax = (1u << (32 - ib)) - 2u;
  dim3 grid((N + kKnnRows - 1) / kKnnRows, B), block(kKnnThreads);
#define GL_KNN_LAUNCH(DT, R)                                                              \
  hipLaunchKernelGGL((knn_kernel<DT, R>), grid, block, 0, stream, x, keys, N, C, M, k, dil, \
                     KK, ib, qscale, qmax, idx_out)
  if (dt_bf16) {
    if (KK <= 16) GL_KNN_LAUNCH(1, 1);
    else if (KK <= 32) GL_KNN_LAUNCH(1, 2);
    else GL_KNN_LAUNCH(1, 4);
  } else {
    if (KK <= 16) GL_KNN_LAUNCH(0, 1);
    else if (KK <= 32) GL_KNN_LAUNCH(0, 2);
    else GL_KNN_LAUNCH(0, 4);
  }
#undef GL_KNN_LAUNCH
  return hipGetLastError();
}

}  // namespace gl
