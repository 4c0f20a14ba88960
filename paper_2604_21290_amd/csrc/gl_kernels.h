// Kernel launchers of libgraphleap (host-callable; argument checks are done
// by the C ABI layer before any of these is called).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>

namespace gl {

struct KnnArgs {
  const void* x;      // [B, N, C] queries
  const void* keys;   // [B, M, C] keys (== x when unpooled)
  int32_t* idx;       // [B, N, k]
  int B, N, C, M, k, dil, KK, ib;
  float qscale;       // 2^(30 - ib): fixed-point scale of the packed distance
  uint32_t qmax;      // largest packed distance of a real key
};

struct MrArgs {
  const void* x;      // [B*N, C]
  const void* keys;   // [B, M, C]
  const int32_t* idx; // [B*N, k]
  const void* W;      // [Cout, 2C]
  const void* bias;   // [Cout] or null
  void* out;          // [B*N, Cout]
  int R, N, M, C, Cout, k;
  int heads;          // > 1: W is block-diagonal by heads (Cout == C); zero blocks are skipped
  int col_tiles;      // > 0: each workgroup computes col_tiles 16-column output tiles of its
                      // nodes (small grids: the output columns split over several workgroups)
  int act_out;        // 1: GELU on each output before its one rounding (the full block's
                      // sigma(U~), which only FC2 reads); dense updates only
};

struct GemmArgs {
  const void* A;         // [R, K], K contiguous
  const void* W;         // [Cout, K], K contiguous
  const void* bias;      // [Cout] or null
  const void* residual;  // [R, Cout] or null (may be `out` itself)
  void* out;             // [R, Cout]
  int R, K, Cout;
  int act_in, act_out;   // 0 none, 1 GELU (on A's elements / on the pre-residual output)
};

// Workgroups are dispatched round-robin over the 8 XCDs (workgroup id mod 8).
// Map dispatch ids so that consecutive logical ids (neighbouring tiles of the
// same image, which share key rows) land on the same XCD and its L2.
__device__ __forceinline__ int xcd_remap(int L, int nb) {
  const int q = nb >> 3, r = nb & 7;
  const int xcd = L & 7, slot = L >> 3;
  return xcd < r ? xcd * (q + 1) + slot : r * (q + 1) + (xcd - r) * q + slot;
}

// Launch fn(args) with `smem` bytes of dynamic LDS.  When ev0/ev1 are given the
// launch itself stamps them (start and end of this dispatch).
template <class A>
hipError_t launch_with_smem(const void* fn, dim3 grid, dim3 block, size_t smem, hipStream_t s,
                            hipEvent_t ev0, hipEvent_t ev1, const A& args) {
  if (smem > 65536) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
  }
  void* argv[] = {const_cast<A*>(&args)};
  if (ev0 || ev1) return hipExtLaunchKernel(fn, grid, block, argv, smem, s, ev0, ev1, 0);
  return hipLaunchKernel(fn, grid, block, argv, smem, s);
}

size_t knn_smem_bytes(int C, int dt_bf16);
int knn_list_regs(int KK);
KnnArgs make_knn_args(const void* x, const void* keys, int B, int N, int C, int M, int k, int dil,
                      int32_t* idx);
hipError_t launch_knn(const void* x, const void* keys, int B, int N, int C, int M, int k,
                      int dil, int dt_bf16, int32_t* idx_out, hipStream_t stream,
                      hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);

// Large key sets (M > 256) use the kernel that streams key chunks through LDS.
bool knn_use_stream(int M, int C, int dt_bf16);
hipError_t launch_knn_stream(const KnnArgs& a, int dt_bf16, hipStream_t stream, hipEvent_t ev0,
                             hipEvent_t ev1);
// bf16 rows of C >= 128 against at most 256 keys use the LDS-staged kernel.
bool knn_use_wide(int M, int C, int dt_bf16);
hipError_t launch_knn_wide(const KnnArgs& a, hipStream_t stream, hipEvent_t ev0, hipEvent_t ev1);
// Many query rows (B * ceil(N / 64) >= 384 workgroups) of 33..160 bf16
// channels against at most 256 keys: keys resident in LDS, 64 rows per
// workgroup; its packed keys equal those of the one-launch block's build
// role for the same shape (in-register tile below C = 128, wide tile above).
bool knn_use_resident(int B, int N, int M, int C, int dt_bf16);
hipError_t launch_knn_resident(const KnnArgs& a, hipStream_t stream, hipEvent_t ev0,
                               hipEvent_t ev1);
// The build cannot be a role of the one-launch block: streamed keys, or the
// LDS-staged tile with more key rows than the block's variants stage (224).
inline bool knn_separate(int M, int C, int dt_bf16) {
  return knn_use_stream(M, C, dt_bf16) || (knn_use_wide(M, C, dt_bf16) && M > 224);
}

int mrconv_lds_row_bytes(int C, int dt_bf16);
size_t mrconv_smem_bytes(int C, int k, int dt_bf16, int rt);
// Row tiles of 16 nodes per workgroup (2 or 1) whose LDS need fits lds_limit; 0 if none.
int mrconv_row_tiles(int C, int k, int dt_bf16, size_t lds_limit);
int mrconv_k_bucket(int k);
// MRConv.  Narrow channels: one fused kernel (gather into the LDS A-tile,
// FC from it).  Wide channels (mrconv_use_split): a gather kernel writes
// [x | m] to split_ws (mrconv_split_ws_bytes), then the tiled GEMM.
hipError_t launch_mrconv(const void* x, const void* keys, const int32_t* idx, const void* W,
                         const void* bias, void* out, int B, int N, int M, int C, int Cout, int k,
                         int dt_bf16, int rt, void* split_ws, hipStream_t stream,
                         hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
// The same with the arguments packed (a.heads > 1 for the multi-head update).
hipError_t launch_mrconv_args(const MrArgs& a, int dt_bf16, int rt, void* split_ws,
                              hipStream_t stream, hipEvent_t ev0 = nullptr,
                              hipEvent_t ev1 = nullptr);
bool mrconv_use_split(int C, int Cout, int dt_bf16, int rt, int R);
// The GEMM pass alone of the two-pass form, on [x | m] rows already in split_ws.
hipError_t launch_mrconv_gemm(const MrArgs& a, int dt_bf16, const void* split_ws,
                              hipStream_t stream, hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
int mrconv_col_tiles(int R, int Cout, int rt);
size_t mrconv_split_ws_bytes(int R, int C, int dt_bf16);
// Multi-head update with per-head weights Wh [H, hd, 2hd] on MFMA (hd a
// multiple of 4; mrconv_headw_steps > 0), or the dense block-diagonal W
// expanded from Wh (launch_expand_heads) for the others.
int mrconv_headw_steps(int hd, int dt_bf16);
hipError_t launch_mrconv_headw(const MrArgs& a, int dt_bf16, int rt, hipStream_t stream);
hipError_t launch_expand_heads(const void* Wh, void* Wd, int C, int heads, int dt_bf16,
                               hipStream_t stream);
size_t gemm_smem_bytes();
hipError_t launch_gemm_nt(const GemmArgs& a, int dt_bf16, hipStream_t stream, hipEvent_t ev0,
                          hipEvent_t ev1);

MrArgs make_mr_args(const void* x, const void* keys, const int32_t* idx, const void* W,
                    const void* bias, void* out, int B, int N, int M, int C, int Cout, int k);
// One block: the build tiles of ka and the update tiles of ma in one grid.
hipError_t launch_block(const KnnArgs& ka, const MrArgs& ma, int dt_bf16, int rt,
                        hipStream_t stream, hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
// Two-pass updates (wide W): the build tiles of ka and the gather tiles of
// ma, which write [x | m] rows to xcat, in one grid (bf16, a build the block
// can host: block_hosts_build); launch_mrconv_gemm then finishes the update.
bool block_hosts_build(int B, int N, int M, int C, int R, int dt_bf16);
hipError_t launch_block_gather(const KnnArgs& ka, const MrArgs& ma, void* xcat,
                               hipStream_t stream, hipEvent_t ev0 = nullptr);

// r x r average (key pooling) or, with max_pool, maximum (inter-stage node
// reduction) of the H x W node grid.
hipError_t launch_pool(const void* x, void* keys, int B, int H, int W, int C, int r, int dt_bf16,
                       hipStream_t stream, bool max_pool = false);

}  // namespace gl
