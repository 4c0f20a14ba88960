// One GraphLeap block in a single launch (Sec. III Eq. 10-12; Sec. IV-A).
//
// The lookahead makes the graph build for block l+1 and the feature update of
// block l independent: both read only X^l.  So one grid holds both kinds of
// workgroup -- kNN build tiles writing Ghat^(l+1) and MRConv update tiles
// writing X^(l+1) -- and they run side by side on the CUs, the one-GPU
// counterpart of the paper's concurrently running Graph Construction Engine
// and Feature Update Engine.  No event or second stream orders them; the next
// block's launch follows in stream order.
//
// Workgroup ids are split between the roles in groups of 8 (one per XCD), so
// both roles spread over every XCD from the first wave of dispatch on.
//
// Updates in the two-pass form (wide W) cannot be a tile of this grid; their
// first pass, the gather of [x_i | m_i] rows, also reads only X^l, so it
// shares a grid with the build tiles instead (block_gather_kernel), and the
// GEMM pass follows in stream order.
#include "knn_tile.h"
#include "knn_wide.h"
#include "mrconv_tile.h"

namespace gl {

constexpr int kBlockWideWaves = 2;     // waves per SIMD the LDS-staged variant is compiled for
constexpr bool kBlockWideDB = true;    // its build role with two staging register sets
constexpr bool kBlockWideT3 = true;    // its update role gathering in one round
constexpr int kBlockGatherRows = 32;   // nodes per gather tile of block_gather_kernel

// Role of dispatch id i among nb build and nu update workgroups; j is the
// workgroup's index within its role.
__device__ __forceinline__ bool block_role_is_build(int i, int nb, int nu, int* j) {
  const int P = (min(nb, nu) >> 3) << 3;
  if (i < 2 * P) {
    const int grp = i >> 4, pos = i & 15;
    *j = grp * 8 + (pos & 7);
    return pos < 8;
  }
  const int i2 = i - 2 * P;
  if (i2 < nb - P) {
    *j = P + i2;
    return true;
  }
  *j = P + i2 - (nb - P);
  return false;
}

// Both roles of one launch.  WK > 0: the build role is the LDS-staged tile
// (32 query rows, WK key rows staged) instead of the in-register one (16 query
// rows); that variant takes 74 KB of LDS, so two workgroups per CU, and is
// compiled for two waves per SIMD, which leaves it the registers for the
// tile's second staging set and for a one-round gather.
template <int DT, int R, int RT, int KB, int WK, bool ACT>
__device__ __forceinline__ void block_body(char* smem, const KnnArgs& ka, const MrArgs& ma, int nb, int nu) {
  constexpr int ES = DT ? 2 : 4;
  int j;
  if (block_role_is_build(blockIdx.x, nb, nu, &j)) {
    j = xcd_remap(j, nb);
    if constexpr (WK > 0) {
      knn_wide_tile<R, kWdQW, WK, kBlockWideDB, true>(smem, ka, j);
    } else {
      const int nt = (ka.N + kKnnRows - 1) / kKnnRows;
      const int b = j / nt, tile = j - b * nt;
      knn_tile<DT, R>(smem, static_cast<const char*>(ka.x) + (size_t)b * ka.N * ka.C * ES,
                      static_cast<const char*>(ka.keys) + (size_t)b * ka.M * ka.C * ES, ka.N, ka.C,
                      ka.M, ka.k, ka.dil, ka.KK, ka.ib, ka.qscale, ka.qmax, tile * kKnnRows,
                      ka.idx + (size_t)b * ka.N * ka.k);
    }
  } else {
    j = xcd_remap(j, nu);
    mrconv_tile<DT, RT, KB, false, (WK > 0) && kBlockWideT3, false, false, ACT>(smem, ma, j * 16 * RT);
  }
}

// ACT: the update role's GELU epilogue (ma.act_out, the full block).
template <int DT, int R, int RT, int KB, int WK, bool ACT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3, 8))) void block_kernel(KnnArgs ka, MrArgs ma, int nb, int nu) {
  extern __shared__ __align__(16) char smem[];
  block_body<DT, R, RT, KB, WK, ACT>(smem, ka, ma, nb, nu);
}

template <int DT, int R, int RT, int KB, int WK, bool ACT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(kBlockWideWaves, 8))) void block_kernel_wide(KnnArgs ka, MrArgs ma, int nb, int nu) {
  extern __shared__ __align__(16) char smem[];
  block_body<DT, R, RT, KB, WK, ACT>(smem, ka, ma, nb, nu);
}

template <int DT, int R, int RT, int WK, bool ACT>
const void* block_fn_kb(int KB) {
  if constexpr (WK > 0) {
    switch (KB) {
      case 9: return (const void*)&block_kernel_wide<DT, R, RT, 9, WK, ACT>;
      case 16: return (const void*)&block_kernel_wide<DT, R, RT, 16, WK, ACT>;
      case 32: return (const void*)&block_kernel_wide<DT, R, RT, 32, WK, ACT>;
      default: return (const void*)&block_kernel_wide<DT, R, RT, 64, WK, ACT>;
    }
  } else {
    switch (KB) {
      case 9: return (const void*)&block_kernel<DT, R, RT, 9, WK, ACT>;
      case 16: return (const void*)&block_kernel<DT, R, RT, 16, WK, ACT>;
      case 32: return (const void*)&block_kernel<DT, R, RT, 32, WK, ACT>;
      default: return (const void*)&block_kernel<DT, R, RT, 64, WK, ACT>;
    }
  }
}

template <int DT, int R, int WK, bool ACT>
const void* block_fn_rt(int RT, int KB) {
  return RT == 2 ? block_fn_kb<DT, R, 2, WK, ACT>(KB) : block_fn_kb<DT, R, 1, WK, ACT>(KB);
}

template <int DT, int WK, bool ACT>
const void* block_fn_r(int R, int RT, int KB) {
  return R == 1 ? block_fn_rt<DT, 1, WK, ACT>(RT, KB)
                : R == 2 ? block_fn_rt<DT, 2, WK, ACT>(RT, KB) : block_fn_rt<DT, 4, WK, ACT>(RT, KB);
}

template <int DT, int WK = 0>
const void* block_fn(int R, int RT, int KB, int act) {
  return act ? block_fn_r<DT, WK, true>(R, RT, KB) : block_fn_r<DT, WK, false>(R, RT, KB);
}

// Key rows the build role stages when it is the LDS-staged tile (the
// standalone build would use that kernel too), else 0: 128 up to 128 keys,
// 224 up to 224.  Larger key sets are not built inside the block.
int block_wide_rows(const KnnArgs& ka, int dt_bf16) {
  if (!knn_use_wide(ka.M, ka.C, dt_bf16)) return 0;
  return ka.M <= 128 ? 128 : 224;
}

// The build tiles (LDS-staged, WK key rows) and the gather tiles of a
// two-pass update in one grid.
template <int R, int KB, int WK>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(kBlockWideWaves, 8))) void block_gather_kernel(KnnArgs ka, MrArgs ma, void* xcat, int nb, int ng) {
  extern __shared__ __align__(16) char smem[];
  int j;
  if (block_role_is_build(blockIdx.x, nb, ng, &j))
    knn_wide_tile<R, kWdQW, WK, kBlockWideDB, true>(smem, ka, xcd_remap(j, nb));
  else
    mr_gather_tile<1, KB>(ma, xcd_remap(j, ng), kBlockGatherRows, reinterpret_cast<int32_t*>(smem),
                          xcat);
}

template <int R, int WK>
const void* block_gather_fn_kb(int KB) {
  switch (KB) {
    case 9: return (const void*)&block_gather_kernel<R, 9, WK>;
    case 16: return (const void*)&block_gather_kernel<R, 16, WK>;
    case 32: return (const void*)&block_gather_kernel<R, 32, WK>;
    default: return (const void*)&block_gather_kernel<R, 64, WK>;
  }
}

template <int WK>
const void* block_gather_fn(int R, int KB) {
  return R == 1 ? block_gather_fn_kb<1, WK>(KB)
                : R == 2 ? block_gather_fn_kb<2, WK>(KB) : block_gather_fn_kb<4, WK>(KB);
}

// The LDS-staged build tile with at most 224 key rows (knn_separate's
// complement among the LDS-staged shapes), and build and gather tiles that
// fit the chip in one round at two workgroups per CU (the build tile's LDS):
// past that the gather, which alone runs many workgroups per CU, loses more
// to the shared LDS than the overlap gains (ViG-B: 15.3 K -> 14.5 K layers/s).
bool block_hosts_build(int B, int N, int M, int C, int R, int dt_bf16) {
  if (!knn_use_wide(M, C, dt_bf16) || M > 224) return false;
  const long nb = (long)B * ((N + 16 * kWdQW - 1) / (16 * kWdQW));
  const long ng = (R + kBlockGatherRows - 1) / kBlockGatherRows;
  return nb + ng <= 512;
}

hipError_t launch_block_gather(const KnnArgs& ka, const MrArgs& ma, void* xcat,
                               hipStream_t stream, hipEvent_t ev0) {
  if (!knn_use_wide(ka.M, ka.C, 1) || ka.M > 224 || !xcat) return hipErrorInvalidValue;
  const int wk = block_wide_rows(ka, 1);
  const int qr = 16 * kWdQW;
  const int nb = ka.B * ((ka.N + qr - 1) / qr);
  const int ng = (ma.R + kBlockGatherRows - 1) / kBlockGatherRows;
  const size_t wsm = wk == 128 ? WideGeom<kWdQW, 128>::kSmem : WideGeom<kWdQW, 224>::kSmem;
  const size_t smem = std::max(wsm, (size_t)kBlockGatherRows * 64 * sizeof(int32_t));
  const int R = knn_list_regs(ka.KK), KB = mrconv_k_bucket(ma.k);
  const void* fn = wk == 224 ? block_gather_fn<224>(R, KB) : block_gather_fn<128>(R, KB);
  struct {
    KnnArgs ka;
    MrArgs ma;
    void* xcat;
    int nb, ng;
  } args{ka, ma, xcat, nb, ng};
  void* argv[] = {&args.ka, &args.ma, &args.xcat, &args.nb, &args.ng};
  if (smem > 65536) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
  }
  const dim3 grid(nb + ng), block(256);
  if (ev0) return hipExtLaunchKernel(fn, grid, block, argv, smem, stream, ev0, nullptr, 0);
  return hipLaunchKernel(fn, grid, block, argv, smem, stream);
}

hipError_t launch_block(const KnnArgs& ka, const MrArgs& ma, int dt_bf16, int rt,
                        hipStream_t stream, hipEvent_t ev0, hipEvent_t ev1) {
  const int wk = block_wide_rows(ka, dt_bf16);
  const bool wide = wk > 0;
  const int qr = wide ? 16 * kWdQW : kKnnRows;
  const int nb = ka.B * ((ka.N + qr - 1) / qr);
  const int TM = 16 * rt;
  const int nu = (ma.R + TM - 1) / TM;
  const size_t wsm = wk == 128 ? WideGeom<kWdQW, 128>::kSmem : WideGeom<kWdQW, 224>::kSmem;
  const size_t smem = std::max(wide ? wsm : knn_smem_bytes(ka.C, dt_bf16),
                               mrconv_smem_bytes(ma.C, ma.k, dt_bf16, rt));
  const int R = knn_list_regs(ka.KK), KB = mrconv_k_bucket(ma.k);
  const int act = ma.act_out;
  const void* fn = wk == 224 ? block_fn<1, 224>(R, rt, KB, act)
                   : wk == 128 ? block_fn<1, 128>(R, rt, KB, act)
                   : dt_bf16 ? block_fn<1>(R, rt, KB, act) : block_fn<0>(R, rt, KB, act);
  const dim3 grid(nb + nu), block(256);
  struct {
    KnnArgs ka;
    MrArgs ma;
    int nb, nu;
  } args{ka, ma, nb, nu};
  void* argv[] = {&args.ka, &args.ma, &args.nb, &args.nu};
  if (smem > 65536) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
  }
  if (ev0 || ev1) return hipExtLaunchKernel(fn, grid, block, argv, smem, stream, ev0, ev1, 0);
  return hipLaunchKernel(fn, grid, block, argv, smem, stream);
}

MrArgs make_mr_args(const void* x, const void* keys, const int32_t* idx, const void* W,
                    const void* bias, void* out, int B, int N, int M, int C, int Cout, int k) {
  MrArgs a;
  a.x = x;
  a.keys = keys;
  a.idx = idx;
  a.W = W;
  a.bias = bias;
  a.out = out;
  a.R = B * N;
  a.N = N;
  a.M = M;
  a.C = C;
  a.Cout = Cout;
  a.k = k;
  a.heads = 1;
  a.col_tiles = 0;
  a.act_out = 0;
  return a;
}

}  // namespace gl
