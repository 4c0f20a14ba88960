// Fused dilated kNN graph build for gfx950 (Sec. II-B Eq. 4; Sec. IV-B; Alg. 2).
//
// One workgroup = 4 waves = 16 query rows of one image.
//   0. the 16 query rows are staged in LDS once, and their inverse norms
//      computed from there;
//   1. keys are processed in chunks of 256 (16 MFMA tiles of 16 keys); wave w
//      computes tiles w, w+4, w+8, w+12, two at a time, with all operand
//      loads of a batch of k-steps issued before the MFMAs that use them.
//      The Gram G = Q K^T contracts the raw stored values (bf16 products are
//      exact in fp32) and the key rows' squared norms accumulate from the
//      same operand registers;
//   2. distance epilogue in fp32 on the accumulators:
//      d1 = (1 + n_j) - 2 r_i r_j G_ij, the squared distance between the
//      L2-normalised rows minus the per-row constant n_i - 1 (rank
//      preserving within a row), quantised to fixed point and packed with the
//      key index into one 32-bit key (distance high, index low), so one
//      unsigned compare orders by (distance, index);
//   3. the packed keys of the chunk go to an LDS strip [16][256];
//   4. each query row is owned by 16 lanes of one wave; the row's running
//      sorted list of the K' = k*dilation smallest keys lives in registers
//      (element e = lane + 16*reg).  Chunk candidates below the list's K'-th
//      key pass a threshold filter, are sorted per lane, and are merged 16 at
//      a time: bitonic sort across the 16 lanes, then a bitonic merge into
//      the list that keeps its K' smallest.
// The N x M distance matrix never leaves the chip; the only global write is
// idx[B, N, k] (ranks 0, d, 2d, ... of the list).
#include "gl_device.h"
#include "gl_kernels.h"

namespace gl {

constexpr int kKnnRows = 16;     // query rows per workgroup
constexpr int kKnnChunk = 256;   // keys per chunk
constexpr int kKnnThreads = 256;
constexpr int kKnnKU = 4;        // k-steps whose operands are loaded as one batch

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

size_t knn_smem_bytes(int C, int dt_bf16) {
  const size_t qstride = (size_t)C * (dt_bf16 ? 2 : 4) + 16;
  return kKnnRows * qstride + (size_t)kKnnRows * kKnnChunk * 4 + kKnnRows * 4;
}

// One 16-row query tile of one image: rows row0 .. row0+15 of x_b against
// all M keys of keys_b; writes idx_b[row, 0..k-1].  smem holds
// knn_smem_bytes(C) bytes.  Called by all 256 threads of the workgroup.
template <int DT, int R>
__device__ __forceinline__ void knn_tile(char* smem, const char* __restrict__ xb,
                                         const char* __restrict__ kb, int N, int C, int M, int k,
                                         int dil, int KK, int ib, float qscale, uint32_t qmax,
                                         int row0, int32_t* __restrict__ idx_b) {
  constexpr int ES = DT ? 2 : 4;
  constexpr int VEC = 16 / ES;
  const int qstride = C * ES + 16;
  char* sQ = smem;
  uint32_t* sStrip = reinterpret_cast<uint32_t*>(smem + kKnnRows * qstride);
  float* sQr = reinterpret_cast<float*>(sStrip + kKnnRows * kKnnChunk);

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, t = lane & 15;
  const int CG = C / VEC;

  // -- stage the query tile ------------------------------------------------------
  for (int e = tid; e < kKnnRows * CG; e += kKnnThreads) {
    const int r = e / CG, cg = e - r * CG;
    const int row = min(row0 + r, N - 1);
    *reinterpret_cast<uint4*>(sQ + r * qstride + cg * 16) =
        *reinterpret_cast<const uint4*>(xb + ((size_t)row * C + cg * VEC) * ES);
  }
  __syncthreads();
  {
    const int r = tid >> 4, part = tid & 15;
    float ss = 0.f;
    for (int cg = part; cg < CG; cg += 16) {
      float f[VEC];
      if (DT) {
        unpack_bf16x8(*reinterpret_cast<const uint4*>(sQ + r * qstride + cg * 16), f);
      } else {
        const float4 v = *reinterpret_cast<const float4*>(sQ + r * qstride + cg * 16);
        f[0] = v.x; f[1] = v.y; f[2] = v.z; f[3] = v.w;
      }
#pragma unroll
      for (int e = 0; e < VEC; ++e) ss = fmaf(f[e], f[e], ss);
    }
    ss += __shfl_xor(ss, 8);
    ss += __shfl_xor(ss, 4);
    ss += __shfl_xor(ss, 2);
    ss += __shfl_xor(ss, 1);
    if (part == 0) sQr[r] = 1.f / fmaxf(sqrtf(ss), 1e-12f);
  }
  __syncthreads();
  float qr[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) qr[v] = sQr[4 * g + v];

  uint32_t L[R];
#pragma unroll
  for (int a = 0; a < R; ++a) L[a] = 0xffffffffu;
  uint32_t tau = 0xffffffffu;
  // contraction steps: 32 channels (bf16) or 16 channels (fp32, 4 MFMAs) each
  const int KSTEP = DT ? 32 : 16;
  const int ksteps = (C + KSTEP - 1) / KSTEP;
  const char* qa = sQ + t * qstride;  // this lane's A-operand row

  for (int chunk0 = 0; chunk0 < M; chunk0 += kKnnChunk) {
    const int nvalid = min(kKnnChunk, M - chunk0);
    const int ntiles = (nvalid + 15) >> 4;
    // -- Gram + epilogue: wave w takes tiles (w, w+4), then (w+8, w+12) -----------
    for (int tt0 = w; tt0 < ntiles; tt0 += 8) {
      const int tt1 = tt0 + 4;
      const bool has1 = tt1 < ntiles;
      const int kr0 = min(chunk0 + tt0 * 16 + t, M - 1);
      const int kr1 = min(chunk0 + (has1 ? tt1 : tt0) * 16 + t, M - 1);
      const char* kp0 = kb + (size_t)kr0 * C * ES;
      const char* kp1 = kb + (size_t)kr1 * C * ES;
      f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = acc0;
      float ss0 = 0.f, ss1 = 0.f;
      for (int s0 = 0; s0 < ksteps; s0 += kKnnKU) {
        uint4 b0[kKnnKU], b1[kKnnKU];
        bool in[kKnnKU];
#pragma unroll
        for (int u = 0; u < kKnnKU; ++u) {
          const int c = (s0 + u) * KSTEP + g * (KSTEP / 4);
          in[u] = (s0 + u < ksteps) && c < C;
          const int cl = in[u] ? c : 0;
          b0[u] = *reinterpret_cast<const uint4*>(kp0 + (size_t)cl * ES);
          b1[u] = *reinterpret_cast<const uint4*>(kp1 + (size_t)cl * ES);
        }
#pragma unroll
        for (int u = 0; u < kKnnKU; ++u) {
          const int c = (s0 + u) * KSTEP + g * (KSTEP / 4);
          uint4 a = *reinterpret_cast<const uint4*>(qa + (size_t)(in[u] ? c : 0) * ES);
          if (!in[u]) a = b0[u] = b1[u] = make_uint4(0, 0, 0, 0);
          if (DT) {
            acc0 = mfma_bf16(a, b0[u], acc0);
            acc1 = mfma_bf16(a, b1[u], acc1);
            float f[8];
            unpack_bf16x8(b0[u], f);
#pragma unroll
            for (int e = 0; e < 8; ++e) ss0 = fmaf(f[e], f[e], ss0);
            unpack_bf16x8(b1[u], f);
#pragma unroll
            for (int e = 0; e < 8; ++e) ss1 = fmaf(f[e], f[e], ss1);
          } else {
            const float4 af = __builtin_bit_cast(float4, a);
            const float4 f0 = __builtin_bit_cast(float4, b0[u]);
            const float4 f1 = __builtin_bit_cast(float4, b1[u]);
            acc0 = mfma_f32(af.x, f0.x, acc0);
            acc0 = mfma_f32(af.y, f0.y, acc0);
            acc0 = mfma_f32(af.z, f0.z, acc0);
            acc0 = mfma_f32(af.w, f0.w, acc0);
            acc1 = mfma_f32(af.x, f1.x, acc1);
            acc1 = mfma_f32(af.y, f1.y, acc1);
            acc1 = mfma_f32(af.z, f1.z, acc1);
            acc1 = mfma_f32(af.w, f1.w, acc1);
            ss0 = fmaf(f0.x, f0.x, fmaf(f0.y, f0.y, fmaf(f0.z, f0.z, fmaf(f0.w, f0.w, ss0))));
            ss1 = fmaf(f1.x, f1.x, fmaf(f1.y, f1.y, fmaf(f1.z, f1.z, fmaf(f1.w, f1.w, ss1))));
          }
        }
      }
      ss0 += __shfl_xor(ss0, 16);
      ss0 += __shfl_xor(ss0, 32);
      ss1 += __shfl_xor(ss1, 16);
      ss1 += __shfl_xor(ss1, 32);
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        if (p == 1 && !has1) break;
        const int tt = p ? tt1 : tt0;
        const float ss = p ? ss1 : ss0;
        const f32x4 acc = p ? acc1 : acc0;
        const int j = chunk0 + tt * 16 + t;
        const float m2rj = -2.f / fmaxf(sqrtf(ss), 1e-12f);
        const float base = ss > 0.f ? 2.f : 1.f;  // 1 + n_j
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float d1 = fmaf(acc[v] * m2rj, qr[v], base);
          uint32_t q = (uint32_t)(fmaxf(d1, 0.f) * qscale);
          q = min(q, qmax);
          sStrip[(4 * g + v) * kKnnChunk + tt * 16 + t] =
              (j < M) ? ((q << ib) | (uint32_t)j) : 0xffffffffu;
        }
      }
    }
    __syncthreads();
    // -- selection: wave w owns rows 4w .. 4w+3, lanes 16g..16g+15 own row 4w+g --
    uint32_t v[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const int col = t + 16 * m;
      v[m] = (col < nvalid) ? sStrip[(4 * w + g) * kKnnChunk + col] : 0xffffffffu;
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

  // -- dilation and output: idx[row, e/dil] = index of list element e ---------
  const int row = row0 + 4 * w + g;
  if (row < N) {
    int32_t* o = idx_b + (size_t)row * k;
    const uint32_t mask = (1u << ib) - 1u;
#pragma unroll
    for (int a = 0; a < R; ++a) {
      const int e = t + 16 * a;
      if (e < KK && (e % dil) == 0) o[e / dil] = (int32_t)(L[a] & mask);
    }
  }
}

template <int DT, int R>
__global__ __launch_bounds__(kKnnThreads) void knn_kernel(KnnArgs a) {
  extern __shared__ __align__(16) char smem[];
  const int nt = (a.N + kKnnRows - 1) / kKnnRows;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int b = blk / nt, tile = blk - b * nt;
  constexpr int ES = DT ? 2 : 4;
  knn_tile<DT, R>(smem, static_cast<const char*>(a.x) + (size_t)b * a.N * a.C * ES,
                  static_cast<const char*>(a.keys) + (size_t)b * a.M * a.C * ES, a.N, a.C, a.M,
                  a.k, a.dil, a.KK, a.ib, a.qscale, a.qmax, tile * kKnnRows,
                  a.idx + (size_t)b * a.N * a.k);
}

KnnArgs make_knn_args(const void* x, const void* keys, int B, int N, int C, int M, int k, int dil,
                      int32_t* idx) {
  KnnArgs a;
  a.x = x;
  a.keys = keys;
  a.idx = idx;
  a.B = B;
  a.N = N;
  a.C = C;
  a.M = M;
  a.k = k;
  a.dil = dil;
  a.KK = k * dil;
  a.ib = 1;
  while ((1 << a.ib) < M) ++a.ib;
  a.qscale = (float)(1u << (30 - a.ib));
  a.qmax = (1u << (32 - a.ib)) - 2u;
  return a;
}

int knn_list_regs(int KK) { return KK <= 16 ? 1 : KK <= 32 ? 2 : 4; }

hipError_t launch_knn(const void* x, const void* keys, int B, int N, int C, int M, int k,
                      int dil, int dt_bf16, int32_t* idx_out, hipStream_t stream,
                      hipEvent_t ev0, hipEvent_t ev1) {
  const KnnArgs a = make_knn_args(x, keys, B, N, C, M, k, dil, idx_out);
  const size_t smem = knn_smem_bytes(C, dt_bf16);
  const dim3 grid(B * ((N + kKnnRows - 1) / kKnnRows)), block(kKnnThreads);
  const int R = knn_list_regs(a.KK);
  const void* fn = nullptr;
  if (dt_bf16) {
    fn = R == 1 ? (const void*)&knn_kernel<1, 1> : R == 2 ? (const void*)&knn_kernel<1, 2>
                                                          : (const void*)&knn_kernel<1, 4>;
  } else {
    fn = R == 1 ? (const void*)&knn_kernel<0, 1> : R == 2 ? (const void*)&knn_kernel<0, 2>
                                                          : (const void*)&knn_kernel<0, 4>;
  }
  return launch_with_smem(fn, grid, block, smem, stream, ev0, ev1, a);
}

}  // namespace gl
