// Standalone MRConv and key-pooling kernels and their launchers (the MRConv
// tile itself is in mrconv_tile.h).
#include "mrconv_tile.h"

namespace gl {

int mrconv_lds_row_bytes(int C, int dt_bf16) { return 2 * C * (dt_bf16 ? 2 : 4) + 16; }

size_t mrconv_smem_bytes(int C, int k, int dt_bf16, int rt) {
  return (size_t)16 * rt * (mrconv_lds_row_bytes(C, dt_bf16) + 4 * k);
}

int mrconv_row_tiles(int C, int k, int dt_bf16, size_t lds_limit) {
  // two row tiles (32 nodes) per workgroup unless the LDS tile does not fit
  for (int rt = 2; rt >= 1; rt >>= 1)
    if (mrconv_smem_bytes(C, k, dt_bf16, rt) <= lds_limit) return rt;
  return 0;
}

// The lean tile: layers of at most 16 output tiles of 16 columns over at least
// one node tile of 32 per CU.  There more workgroups in flight hide the
// gather's latency better than more work per wave does, and (on 64-node
// tiles) each workgroup's pass over W serves twice the nodes.
bool mrconv_use_lean(int C, int Cout, int row_tiles) {
  return Cout <= 256 && C <= 256 && row_tiles >= 256;
}

int mrconv_k_bucket(int k) { return k <= 9 ? 9 : k <= 16 ? 16 : k <= 32 ? 32 : 64; }

template <int DT, int RT, int KB, bool ACT = false>
__global__ __launch_bounds__(kMrThreads) __attribute__((amdgpu_waves_per_eu(3, 8))) void mrconv_kernel(MrArgs a) {
  extern __shared__ __align__(16) char smem[];
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  mrconv_tile<DT, RT, KB, false, false, false, false, ACT>(smem, a, blk * 16 * RT);
}

// Narrow layers over many node tiles: one output tile per wave and pass and
// one gather task per thread (78 VGPRs at k <= 9: six waves per SIMD).
template <int DT, int RT, int KB, bool ACT = false>
__global__ __launch_bounds__(kMrThreads) __attribute__((amdgpu_waves_per_eu(4, 8))) void mrconv_lean_kernel(MrArgs a) {
  extern __shared__ __align__(16) char smem[];
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  mrconv_tile<DT, RT, KB, false, false, false, true, ACT>(smem, a, blk * 16 * RT);
}

// Small grids: workgroup blk computes output-column group blk % ncg (a.col_tiles
// 16-column tiles) of node tile blk / ncg.  Few workgroups run, so the kernel is
// not held to three waves per SIMD.
template <int DT, int RT, int KB, bool ACT = false>
__global__ __launch_bounds__(kMrThreads) void mrconv_cols_kernel(MrArgs a) {
  extern __shared__ __align__(16) char smem[];
  const int nct = (a.Cout + 15) >> 4;
  const int ncg = (nct + a.col_tiles - 1) / a.col_tiles;
  const int blk = blockIdx.x, cg = blk % ncg;
  const int tile0 = cg * a.col_tiles;
  mrconv_tile<DT, RT, KB, false, false, true, false, ACT>(smem, a, (blk / ncg) * 16 * RT, tile0,
                                                          min(nct, tile0 + a.col_tiles));
}

// The multi-head update: the per-tile step tests need registers the
// three-waves-per-SIMD budget does not leave, so this one is not held to it.
template <int DT, int RT, int KB>
__global__ __launch_bounds__(kMrThreads) void mrconv_heads_kernel(MrArgs a) {
  extern __shared__ __align__(16) char smem[];
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  mrconv_tile<DT, RT, KB, true>(smem, a, blk * 16 * RT);
}

template <int DT, int RT, bool HEADS = false, bool COLS = false, bool LEAN = false, bool ACT = false>
const void* mrconv_fn_kb(int KB) {
  if constexpr (LEAN) {
    switch (KB) {
      case 9: return (const void*)&mrconv_lean_kernel<DT, RT, 9, ACT>;
      case 16: return (const void*)&mrconv_lean_kernel<DT, RT, 16, ACT>;
      case 32: return (const void*)&mrconv_lean_kernel<DT, RT, 32, ACT>;
      default: return (const void*)&mrconv_lean_kernel<DT, RT, 64, ACT>;
    }
  } else if constexpr (COLS) {
    switch (KB) {
      case 9: return (const void*)&mrconv_cols_kernel<DT, RT, 9, ACT>;
      case 16: return (const void*)&mrconv_cols_kernel<DT, RT, 16, ACT>;
      case 32: return (const void*)&mrconv_cols_kernel<DT, RT, 32, ACT>;
      default: return (const void*)&mrconv_cols_kernel<DT, RT, 64, ACT>;
    }
  } else if constexpr (HEADS) {
    switch (KB) {
      case 9: return (const void*)&mrconv_heads_kernel<DT, RT, 9>;
      case 16: return (const void*)&mrconv_heads_kernel<DT, RT, 16>;
      case 32: return (const void*)&mrconv_heads_kernel<DT, RT, 32>;
      default: return (const void*)&mrconv_heads_kernel<DT, RT, 64>;
    }
  } else {
    switch (KB) {
      case 9: return (const void*)&mrconv_kernel<DT, RT, 9, ACT>;
      case 16: return (const void*)&mrconv_kernel<DT, RT, 16, ACT>;
      case 32: return (const void*)&mrconv_kernel<DT, RT, 32, ACT>;
      default: return (const void*)&mrconv_kernel<DT, RT, 64, ACT>;
    }
  }
}

// The dense variants' table, with or without the GELU epilogue (a.act_out).
template <int DT, int RT, bool COLS = false, bool LEAN = false>
const void* mrconv_fn_act(int KB, int act) {
  return act ? mrconv_fn_kb<DT, RT, false, COLS, LEAN, true>(KB)
             : mrconv_fn_kb<DT, RT, false, COLS, LEAN, false>(KB);
}

// Gather-only workgroup of the two-pass MRConv: kMrGatherRows nodes.
template <int DT, int KB>
__global__ __launch_bounds__(kMrThreads) void mr_gather_kernel(MrArgs a, void* xcat) {
  __shared__ int32_t sIdx[kMrGatherRows * 64];
  mr_gather_tile<DT, KB>(a, xcd_remap(blockIdx.x, gridDim.x), kMrGatherRows, sIdx, xcat);
}

template <int DT>
const void* gather_fn_kb(int KB) {
  switch (KB) {
    case 9: return (const void*)&mr_gather_kernel<DT, 9>;
    case 16: return (const void*)&mr_gather_kernel<DT, 16>;
    case 32: return (const void*)&mr_gather_kernel<DT, 32>;
    default: return (const void*)&mr_gather_kernel<DT, 64>;
  }
}

// Column groups of a small grid: a layer of at most 64 node tiles with more than
// four 16-column output tiles runs one workgroup per (node tile, group of four
// output tiles); 0 = no split.
int mrconv_col_tiles(int R, int Cout, int rt) {
  const int row_tiles = (R + 16 * rt - 1) / (16 * rt);
  return row_tiles <= 64 && (Cout + 15) / 16 > 4 ? 4 : 0;
}

// The fused tile streams all of W (of its column group) through every workgroup
// of 16*rt nodes; beyond 8 KB of W per node (or when the tile does not fit LDS)
// the two-pass form, which reads W once per 64 or 128 nodes, is used.
bool mrconv_use_split(int C, int Cout, int dt_bf16, int rt, int R) {
  if (rt < 1) return true;
  const int ct = mrconv_col_tiles(R, Cout, rt);
  const int cols = ct ? (16 * ct < Cout ? 16 * ct : Cout) : Cout;
  const size_t wbytes = (size_t)cols * 2 * C * (dt_bf16 ? 2 : 4);
  return wbytes / (size_t)(16 * rt) > 8192;
}

size_t mrconv_split_ws_bytes(int R, int C, int dt_bf16) {
  return (size_t)R * 2 * C * (dt_bf16 ? 2 : 4);
}

hipError_t launch_mrconv(const void* x, const void* keys, const int32_t* idx, const void* W,
                         const void* bias, void* out, int B, int N, int M, int C, int Cout, int k,
                         int dt_bf16, int rt, void* split_ws, hipStream_t stream, hipEvent_t ev0,
                         hipEvent_t ev1) {
  return launch_mrconv_args(make_mr_args(x, keys, idx, W, bias, out, B, N, M, C, Cout, k), dt_bf16,
                            rt, split_ws, stream, ev0, ev1);
}

// The second pass of the two-pass MRConv: out = act_out([x | m] W^T + b).
hipError_t launch_mrconv_gemm(const MrArgs& a, int dt_bf16, const void* split_ws,
                              hipStream_t stream, hipEvent_t ev0, hipEvent_t ev1) {
  GemmArgs ga;
  ga.A = split_ws;
  ga.W = a.W;
  ga.bias = a.bias;
  ga.residual = nullptr;
  ga.out = a.out;
  ga.R = a.R;
  ga.K = 2 * a.C;
  ga.Cout = a.Cout;
  ga.act_in = 0;
  ga.act_out = a.act_out;
  return launch_gemm_nt(ga, dt_bf16, stream, ev0, ev1);
}

hipError_t launch_mrconv_args(const MrArgs& a0, int dt_bf16, int rt, void* split_ws,
                              hipStream_t stream, hipEvent_t ev0, hipEvent_t ev1) {
  MrArgs a = a0;
  const int C = a.C, Cout = a.Cout, k = a.k;
  const int KB = mrconv_k_bucket(k);
  // the multi-head update (W = per-head Wh) always takes the fused tile
  if (a.heads > 1 && (rt < 1 || a.act_out)) return hipErrorInvalidValue;
  if (a.heads <= 1 && mrconv_use_split(C, Cout, dt_bf16, rt, a.R)) {
    if (!split_ws) return hipErrorInvalidValue;
    const dim3 g1((a.R + kMrGatherRows - 1) / kMrGatherRows), blk(kMrThreads);
    const void* fg = dt_bf16 ? gather_fn_kb<1>(KB) : gather_fn_kb<0>(KB);
    void* argv[] = {&a, &split_ws};
    hipError_t e = ev0 ? hipExtLaunchKernel(fg, g1, blk, argv, 0, stream, ev0, nullptr, 0)
                       : hipLaunchKernel(fg, g1, blk, argv, 0, stream);
    if (e != hipSuccess) return e;
    return launch_mrconv_gemm(a, dt_bf16, split_ws, stream, nullptr, ev1);
  }
  const int TM = 16 * rt;
  const size_t smem = mrconv_smem_bytes(C, k, dt_bf16, rt);
  const int row_tiles = (a.R + TM - 1) / TM;
  // A grid of a few node tiles (a single image) leaves most CUs idle while each
  // workgroup streams all of W in batches; there the output columns are split
  // into groups of four 16-column tiles (one per wave), each group its own
  // workgroup (the gather is repeated per group, W is read once per group).
  const int nct = (Cout + 15) >> 4;
  a.col_tiles = a.heads <= 1 ? mrconv_col_tiles(a.R, Cout, rt) : 0;
  const int ncg = a.col_tiles ? (nct + a.col_tiles - 1) / a.col_tiles : 1;
  const dim3 grid(row_tiles * ncg), block(kMrThreads);
  const void* fn;
  const int act = a.act_out;
  if (a.col_tiles > 0) {
    fn = dt_bf16 ? (rt == 2 ? mrconv_fn_act<1, 2, true>(KB, act) : mrconv_fn_act<1, 1, true>(KB, act))
                 : (rt == 2 ? mrconv_fn_act<0, 2, true>(KB, act) : mrconv_fn_act<0, 1, true>(KB, act));
  } else if (a.heads > 1) {
    fn = dt_bf16 ? (rt == 2 ? mrconv_fn_kb<1, 2, true>(KB) : mrconv_fn_kb<1, 1, true>(KB))
                 : (rt == 2 ? mrconv_fn_kb<0, 2, true>(KB) : mrconv_fn_kb<0, 1, true>(KB));
  } else if (mrconv_use_lean(a.C, Cout, row_tiles)) {
    // 64-node tiles when they fit 64 KB of LDS (measured 2-3 % faster than 32)
    if (mrconv_smem_bytes(C, k, dt_bf16, 4) <= 65536) {
      fn = dt_bf16 ? mrconv_fn_act<1, 4, false, true>(KB, act) : mrconv_fn_act<0, 4, false, true>(KB, act);
      return launch_with_smem(fn, dim3((a.R + 63) / 64), block, mrconv_smem_bytes(C, k, dt_bf16, 4),
                              stream, ev0, ev1, a);
    }
    fn = dt_bf16 ? (rt == 2 ? mrconv_fn_act<1, 2, false, true>(KB, act) : mrconv_fn_act<1, 1, false, true>(KB, act))
                 : (rt == 2 ? mrconv_fn_act<0, 2, false, true>(KB, act) : mrconv_fn_act<0, 1, false, true>(KB, act));
  } else {
    fn = dt_bf16 ? (rt == 2 ? mrconv_fn_act<1, 2>(KB, act) : mrconv_fn_act<1, 1>(KB, act))
                 : (rt == 2 ? mrconv_fn_act<0, 2>(KB, act) : mrconv_fn_act<0, 1>(KB, act));
  }
  return launch_with_smem(fn, grid, block, smem, stream, ev0, ev1, a);
}

// ---------------------------------------------------------------------------
// Multi-head update with per-head weights (Sec. II-A; the per-head W_x,h and
// W_m,h of Sec. IV-C2): output channel o of head h = o / hd only meets head
// h's hd channels of x_i and of m_i.  Per workgroup (TM nodes):
//   1. the gather of the fused tile writes [x_i | m_i] rows into LDS;
//   2. the FC runs per head on MFMA: a unit is (head h, 16-column tile c of
//      the head's outputs); its contraction covers only head h's channels,
//      ceil(hd / KSTEP) steps in the x half and as many in the m half.  A and
//      B operands past the head's last channel are zero, so nothing of the
//      neighbouring heads enters.  B comes straight from Wh [H, hd, 2hd]: row
//      o of Wh viewed as [C, 2hd] is output o's [W_x,h | W_m,h] row, so a
//      lane's 8 (bf16) or 4 (fp32) k-values are contiguous.
//   Units are dealt to the 4 waves round-robin; the B operands of a wave's
//   next unit are requested while the current one finishes, the first ones
//   ahead of the gather.
// hd must be a multiple of 4 (operand loads of 4 channels never straddle a
// head) and at most KSH * KSTEP.
// ---------------------------------------------------------------------------
// B operand: Wh row o, k-values kl .. kl+KV-1 of half `half` (zero past hd,
// and for a column past the head's last output).
template <int DT>
__device__ __forceinline__ uint4 mr_wh_operand(const char* Wh, int o, bool ov, int hd, int half,
                                               int kl) {
  if (DT) {
    const char* p = Wh + ((size_t)o * 2 * hd + half * hd + kl) * 2;
    const uint2 lo = (ov && kl < hd) ? *reinterpret_cast<const uint2*>(p) : make_uint2(0, 0);
    const uint2 hi = (ov && kl + 4 < hd) ? *reinterpret_cast<const uint2*>(p + 8) : make_uint2(0, 0);
    return make_uint4(lo.x, lo.y, hi.x, hi.y);
  } else {
    const char* p = Wh + ((size_t)o * 2 * hd + half * hd + kl) * 4;
    return (ov && kl < hd) ? *reinterpret_cast<const uint4*>(p) : make_uint4(0, 0, 0, 0);
  }
}

// A operand from the LDS row: channels kl .. kl+KV-1 of head h in half `half`
// (zero past hd).
template <int DT>
__device__ __forceinline__ uint4 mr_head_a_operand(const char* rowp, int C, int h, int hd, int half,
                                                   int kl) {
  if (DT) {
    const char* p = rowp + (size_t)(half * C + h * hd + kl) * 2;
    const uint2 lo = kl < hd ? *reinterpret_cast<const uint2*>(p) : make_uint2(0, 0);
    const uint2 hi = kl + 4 < hd ? *reinterpret_cast<const uint2*>(p + 8) : make_uint2(0, 0);
    return make_uint4(lo.x, lo.y, hi.x, hi.y);
  } else {
    const char* p = rowp + (size_t)(half * C + h * hd + kl) * 4;
    return kl < hd ? *reinterpret_cast<const uint4*>(p) : make_uint4(0, 0, 0, 0);
  }
}

template <int DT, int RT, int KB, int KSH>
__global__ __launch_bounds__(kMrThreads) void mrconv_headw_kernel(MrArgs a) {
  extern __shared__ __align__(16) char smem[];
  constexpr int TM = 16 * RT;
  constexpr int ES = DT ? 2 : 4;
  constexpr int KSTEP = DT ? 32 : 16;
  constexpr int KV = KSTEP / 4;  // k-values per lane and step
  const int C = a.C, k = a.k, M = a.M, R = a.R, H = a.heads, hd = C / H;
  const int lds_row = 2 * C * ES + 16;
  char* sA = smem;
  int32_t* sIdx = reinterpret_cast<int32_t*>(smem + TM * lds_row);
  const int row0 = xcd_remap(blockIdx.x, gridDim.x) * TM;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, t = lane & 15;

  for (int e = tid; e < TM * k; e += kMrThreads) {
    const int r = e / k, tt = e - r * k, row = row0 + r;
    const int j = row < R ? a.idx[(size_t)row * k + tt] : 0;
    sIdx[e] = min(max(j, 0), M - 1) * (C * ES / 16);
  }

  const int nch = (hd + 15) >> 4;  // 16-column tiles per head
  const int U = H * nch;           // units
  const char* Wh = static_cast<const char*>(a.W);
  uint4 bw[2][KSH];
  auto load_b = [&](int u) {
    const int h = u / nch, ol = (u - h * nch) * 16 + t;
    const int o = h * hd + min(ol, hd - 1);
#pragma unroll
    for (int half = 0; half < 2; ++half)
#pragma unroll
      for (int s = 0; s < KSH; ++s)
        bw[half][s] = mr_wh_operand<DT>(Wh, o, ol < hd, hd, half, s * KSTEP + g * KV);
  };
  if (w < U) load_b(w);
  __syncthreads();
  mr_gather_rows<DT, KB>(a, row0, TM, sIdx, sA, lds_row);
  __syncthreads();

  for (int u = w; u < U; u += 4) {
    const int h = u / nch, ol = (u - h * nch) * 16 + t;
    f32x4 acc[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int half = 0; half < 2; ++half)
#pragma unroll
      for (int s = 0; s < KSH; ++s) {
        if (s * KSTEP >= hd) continue;  // uniform
        const int kl = s * KSTEP + g * KV;
        const uint4 bv = bw[half][s];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          const uint4 av =
              mr_head_a_operand<DT>(sA + (size_t)(rt * 16 + t) * lds_row, C, h, hd, half, kl);
          if (DT) {
            acc[rt] = mfma_bf16(av, bv, acc[rt]);
          } else {
            const float4 x4 = __builtin_bit_cast(float4, av);
            const float4 w4 = __builtin_bit_cast(float4, bv);
            acc[rt] = mfma_f32(x4.x, w4.x, acc[rt]);
            acc[rt] = mfma_f32(x4.y, w4.y, acc[rt]);
            acc[rt] = mfma_f32(x4.z, w4.z, acc[rt]);
            acc[rt] = mfma_f32(x4.w, w4.w, acc[rt]);
          }
        }
      }
    if (u + 4 < U) load_b(u + 4);
    // epilogue: + bias, round once, store (columns past the head are not)
    if (ol < hd) {
      const int o = h * hd + ol;
      float bn = 0.f;
      if (a.bias) {
        bn = DT ? bf16_bits_to_f32(static_cast<const uint16_t*>(a.bias)[o])
                : static_cast<const float*>(a.bias)[o];
      }
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = row0 + rt * 16 + 4 * g + v;
          if (row >= R) continue;
          const size_t off = (size_t)row * C + o;
          const float y = acc[rt][v] + bn;
          if (DT) static_cast<uint16_t*>(a.out)[off] = (uint16_t)f32_to_bf16_bits(y);
          else static_cast<float*>(a.out)[off] = y;
        }
    }
  }
}

// k-steps per half the per-head kernel is compiled for (0: hd is not a
// multiple of 4 or wider than 8 steps).
int mrconv_headw_steps(int hd, int dt_bf16) {
  if (hd < 4 || hd % 4) return 0;
  const int ks = (hd + (dt_bf16 ? 32 : 16) - 1) / (dt_bf16 ? 32 : 16);
  return ks <= 1 ? 1 : ks <= 2 ? 2 : ks <= 4 ? 4 : ks <= 8 ? 8 : 0;
}

template <int DT, int RT, int KSH>
const void* headw_fn_kb(int KB) {
  switch (KB) {
    case 9: return (const void*)&mrconv_headw_kernel<DT, RT, 9, KSH>;
    case 16: return (const void*)&mrconv_headw_kernel<DT, RT, 16, KSH>;
    case 32: return (const void*)&mrconv_headw_kernel<DT, RT, 32, KSH>;
    default: return (const void*)&mrconv_headw_kernel<DT, RT, 64, KSH>;
  }
}

template <int DT, int RT>
const void* headw_fn(int KSH, int KB) {
  return KSH == 1 ? headw_fn_kb<DT, RT, 1>(KB) : KSH == 2 ? headw_fn_kb<DT, RT, 2>(KB)
       : KSH == 4 ? headw_fn_kb<DT, RT, 4>(KB) : headw_fn_kb<DT, RT, 8>(KB);
}

hipError_t launch_mrconv_headw(const MrArgs& a, int dt_bf16, int rt, hipStream_t stream) {
  const int hd = a.C / a.heads;
  const int KSH = mrconv_headw_steps(hd, dt_bf16);
  if (!KSH || rt < 1 || a.Cout != a.C) return hipErrorInvalidValue;
  // few node tiles: 16-node tiles fill more CUs
  if (rt == 2 && (a.R + 31) / 32 < 256) rt = 1;
  const int TM = 16 * rt, KB = mrconv_k_bucket(a.k);
  const void* fn = dt_bf16 ? (rt == 2 ? headw_fn<1, 2>(KSH, KB) : headw_fn<1, 1>(KSH, KB))
                           : (rt == 2 ? headw_fn<0, 2>(KSH, KB) : headw_fn<0, 1>(KSH, KB));
  const dim3 grid((a.R + TM - 1) / TM), block(kMrThreads);
  return launch_with_smem(fn, grid, block, mrconv_smem_bytes(a.C, a.k, dt_bf16, rt), stream,
                          nullptr, nullptr, a);
}

// Dense [C, 2C] = [W_x | W_m] from per-head Wh [H, hd, 2hd]: zero outside the
// heads' diagonal blocks of each half.  One thread per element of the output.
template <int DT>
__global__ __launch_bounds__(256) void expand_heads_kernel(const void* __restrict__ Wh,
                                                           void* __restrict__ Wd, int C, int hd) {
  constexpr int ES = DT ? 2 : 4;
  const long e = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= (long)C * 2 * C) return;
  const int o = (int)(e / (2 * C)), jj = (int)(e - (long)o * 2 * C);
  const int half = jj >= C, j = jj - half * C;
  const int h = o / hd;
  const bool in = j / hd == h;
  const long src = ((long)o * 2 * hd) + half * hd + (j - h * hd);
  if (ES == 2) {
    static_cast<uint16_t*>(Wd)[e] = in ? static_cast<const uint16_t*>(Wh)[src] : (uint16_t)0;
  } else {
    static_cast<float*>(Wd)[e] = in ? static_cast<const float*>(Wh)[src] : 0.f;
  }
}

hipError_t launch_expand_heads(const void* Wh, void* Wd, int C, int heads, int dt_bf16,
                               hipStream_t stream) {
  const long n = (long)C * 2 * C;
  const dim3 grid((unsigned)((n + 255) / 256)), block(256);
  if (dt_bf16) hipLaunchKernelGGL(expand_heads_kernel<1>, grid, block, 0, stream, Wh, Wd, C, C / heads);
  else hipLaunchKernelGGL(expand_heads_kernel<0>, grid, block, 0, stream, Wh, Wd, C, C / heads);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// r x r pooling of the node grid, stride r: the average (key nodes of pyramid
// stages) or the maximum (node reduction between pyramid stages, Sec. IV-E).
// One thread per (image, output node, 16-byte channel vector).  For the
// window sizes the pyramids use (RR = 2, 4) all r*r loads of a thread are
// issued before any is summed, so the window costs one memory round trip;
// other r (RR = 0) loop.  The window is summed in row-major order either way.
// The maximum of stored values is exact; the average is accumulated in fp32
// and rounded once.
// ---------------------------------------------------------------------------
template <int DT, bool MAX, int RR>
__global__ __launch_bounds__(128) void pool_kernel(const void* __restrict__ x,
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
  for (int i = 0; i < VEC; ++i) acc[i] = MAX ? -INFINITY : 0.f;
  const char* xb = static_cast<const char*>(x) + ((size_t)b * H * W * C + cg * VEC) * ES;
  auto add = [&](const float* f) {
#pragma unroll
    for (int i = 0; i < VEC; ++i) acc[i] = MAX ? fmaxf(acc[i], f[i]) : acc[i] + f[i];
  };
  if constexpr (RR > 0) {
    uint4 raw[RR * RR];
#pragma unroll
    for (int u = 0; u < RR; ++u)
#pragma unroll
      for (int v = 0; v < RR; ++v)
        raw[u * RR + v] = *reinterpret_cast<const uint4*>(
            xb + (size_t)((p * RR + u) * W + (q * RR + v)) * C * ES);
#pragma unroll
    for (int i = 0; i < RR * RR; ++i) {
      float f[VEC];
      load_vec<DT>(reinterpret_cast<const char*>(&raw[i]), f);
      add(f);
    }
  } else {
    for (int u = 0; u < r; ++u) {
      for (int v = 0; v < r; ++v) {
        float f[VEC];
        load_vec<DT>(xb + (size_t)((p * r + u) * W + (q * r + v)) * C * ES, f);
        add(f);
      }
    }
  }
  if (!MAX) {
    const float inv = 1.f / (float)(r * r);
#pragma unroll
    for (int i = 0; i < VEC; ++i) acc[i] *= inv;
  }
  store_vec<DT>(static_cast<char*>(keys) + ((size_t)(b * Mo + o) * C + cg * VEC) * ES, acc);
}

template <int DT, bool MAX>
const void* pool_fn(int r) {
  return r == 2 ? (const void*)&pool_kernel<DT, MAX, 2>
         : r == 4 ? (const void*)&pool_kernel<DT, MAX, 4> : (const void*)&pool_kernel<DT, MAX, 0>;
}

hipError_t launch_pool(const void* x, void* keys, int B, int H, int W, int C, int r, int dt_bf16,
                       hipStream_t stream, bool max_pool) {
  const int VEC = dt_bf16 ? 8 : 4;
  const long total = (long)B * (H / r) * (W / r) * (C / VEC);
  const void* fn = max_pool ? (dt_bf16 ? pool_fn<1, true>(r) : pool_fn<0, true>(r))
                            : (dt_bf16 ? pool_fn<1, false>(r) : pool_fn<0, false>(r));
  dim3 grid((unsigned)((total + 127) / 128)), block(128);
  void* argv[] = {&x, &keys, &B, &H, &W, &C, &r};
  return hipLaunchKernel(fn, grid, block, argv, 0, stream);
}

}  // namespace gl
