// Standalone LDS-staged kNN kernel and its launcher (the tile itself is in
// knn_wide.h).
#include "knn_wide.h"

namespace gl {

// Used from C = 128 on, by the standalone build and by the one-launch block
// alike, so that every schedule ranks the same packed keys.  Standalone it is
// 1.1-2.5x faster than the in-register kernel at C = 192-640; inside the
// one-launch block it makes the ViG-Ti stack 15 % faster.
bool knn_use_wide(int M, int C, int dt_bf16) {
  return dt_bf16 && M <= kWdMaxKeys && C >= 128 && C % 8 == 0;
}

template <int R, int QW, int KROWS>
__global__ __launch_bounds__(kWdThreads) void knn_wide_kernel(KnnArgs a) {
  extern __shared__ __align__(16) char smem[];
  knn_wide_tile<R, QW, KROWS>(smem, a, xcd_remap(blockIdx.x, gridDim.x));
}

template <int R, int QW>
const void* wide_fn_rows(int KROWS) {
  switch (KROWS) {
    case 64: return (const void*)&knn_wide_kernel<R, QW, 64>;
    case 128: return (const void*)&knn_wide_kernel<R, QW, 128>;
    case 224: return (const void*)&knn_wide_kernel<R, QW, 224>;
    default: return (const void*)&knn_wide_kernel<R, QW, 256>;
  }
}

template <int QW>
const void* wide_fn(int R, int KROWS) {
  return R == 1 ? wide_fn_rows<1, QW>(KROWS) : R == 2 ? wide_fn_rows<2, QW>(KROWS) : wide_fn_rows<4, QW>(KROWS);
}

hipError_t launch_knn_wide(const KnnArgs& a, hipStream_t stream, hipEvent_t ev0, hipEvent_t ev1) {
  const int R = knn_list_regs(a.KK), KROWS = knn_wide_key_rows(a.M);
  const void* fn = wide_fn<kWdQW>(R, KROWS);
  const size_t smem = wide_smem<kWdQW>(a.M);
  const dim3 grid(a.B * ((a.N + 16 * kWdQW - 1) / (16 * kWdQW))), block(kWdThreads);
  return launch_with_smem(fn, grid, block, smem, stream, ev0, ev1, a);
}

}  // namespace gl
