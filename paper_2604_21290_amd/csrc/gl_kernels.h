// Kernel launchers of libgraphleap (host-callable; argument checks are done
// by the C ABI layer before any of these is called).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace gl {

hipError_t launch_knn(const void* x, const void* keys, int B, int N, int C, int M, int k,
                      int dil, int dt_bf16, int32_t* idx_out, hipStream_t stream);

int mrconv_lds_row_bytes(int C, int dt_bf16);
// Largest row-tile count (1, 2 or 4 tiles of 16 nodes) whose LDS need fits
// lds_limit bytes; 0 if none does.
int mrconv_row_tiles(int C, int k, int dt_bf16, size_t lds_limit);

hipError_t launch_mrconv(const void* x, const void* keys, const int32_t* idx, const void* W,
                         const void* bias, void* out, int B, int N, int M, int C, int Cout, int k,
                         int dt_bf16, int rt, hipStream_t stream);

hipError_t launch_pool(const void* x, void* keys, int B, int H, int W, int C, int r, int dt_bf16,
                       hipStream_t stream);

}  // namespace gl
