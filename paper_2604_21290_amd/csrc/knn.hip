// Standalone kNN graph kernel and its launcher (the tile itself is in knn_tile.h).
#include "knn_tile.h"

namespace gl {

size_t knn_smem_bytes(int C, int dt_bf16) {
  (void)C;
  (void)dt_bf16;
  return (size_t)kKnnRows * kKnnChunk * 4;
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
  if (knn_use_stream(M, C, dt_bf16)) return launch_knn_stream(a, dt_bf16, stream, ev0, ev1);
  if (knn_use_resident(B, N, M, C, dt_bf16)) return launch_knn_resident(a, stream, ev0, ev1);
  if (knn_use_wide(M, C, dt_bf16)) return launch_knn_wide(a, stream, ev0, ev1);
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
