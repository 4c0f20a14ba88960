// Fused max-relative graph convolution for gfx950 (Sec. II-A Eq. 2-3; the
// W_x / W_m split of Sec. IV-C2), and r x r key pooling for pyramid stages.
//
// One MRConv workgroup = 4 waves = TM = 16*RT consecutive nodes of the
// flattened [B*N] node axis.
//   1. gather: for each node and each 16-byte channel vector, the neighbour
//      key rows are read with all loads of the vector in flight at once
//      (the neighbour loop is unrolled to a compile-time bucket KB >= k; the
//      slots past k repeat the first neighbour, which leaves the maximum
//      unchanged).  Consecutive lanes read consecutive vectors of the same
//      row, so every neighbour row is one coalesced burst.  The maximum is
//      exact in the storage type; x_i is subtracted in fp32 and the result
//      rounded once.  [x_i | m_i] goes straight into the LDS A-tile: no edge
//      tensor and no [B,N,2C] concatenation is ever written to memory.
//   2. FC on MFMA: out[TM, Cout] = A[TM, 2C] W^T + b.  The contraction runs
//      over the concatenated axis, so columns 0..C-1 of W meet x_i and columns
//      C..2C-1 meet m_i in one accumulation.  Each wave owns every 4th
//      16-column output tile; W rows stream from L2 as MFMA B operands, a
//      batch of k-steps at a time.
#pragma once

#include "gl_device.h"
#include "gl_kernels.h"

namespace gl {

constexpr int kMrThreads = 256;
constexpr int kMrKU = 4;  // k-steps of W operands loaded as one batch

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

// W operands of k-steps s0 .. s0+kMrKU-1 for the wave's output tiles
// w + 4*(4p + c4), c4 < 4 (16 columns each).  Tiles past Cout are not loaded
// (their registers keep zeros); k past 2C reads column 0, a real W element
// that meets a zero A operand.
// Multi-head update (a.heads > 1, Cout == C): does the 16-column output tile
// starting at n0 need contraction step s?  Only the channels of the heads the
// tile's columns belong to, in the x half and in the m half, are non-zero in
// the block-diagonal W.  Wave-uniform.
__device__ __forceinline__ bool mr_step_needed(const MrArgs& a, int n0, int s, int kstep) {
  if (a.heads <= 1) return true;
  const int hd = a.C / a.heads;
  const int lo = (n0 / hd) * hd, hi = (min(n0 + 15, a.Cout - 1) / hd + 1) * hd;
  const int k0 = s * kstep, k1 = k0 + kstep;
  return (k0 < hi && k1 > lo) || (k0 < a.C + hi && k1 > a.C + lo);
}

// COLS: only output tiles tile0 .. tile_end-1 (a column group of a small grid),
// one tile per wave and pass, with the W operands of kMrKUCols k-steps per batch.
constexpr int kMrKUCols = 12;
// LEAN: one output tile per wave and pass and one gather task per thread and
// round, for layers of few output tiles that run many node tiles: the
// registers saved buy more waves per SIMD.
template <bool COLS, bool LEAN = false> struct MrBatch {
  static constexpr int KU = COLS ? kMrKUCols : kMrKU;   // k-steps per batch of W operands
  static constexpr int NC = COLS || LEAN ? 1 : 4;       // output tiles per wave and pass
};

template <int DT, bool HEADS, bool COLS = false, bool LEAN = false>
__device__ __forceinline__ void mr_load_w(uint4 (&bw)[(MrBatch<COLS, LEAN>::KU)][(MrBatch<COLS, LEAN>::NC)],
                                          const MrArgs& a, const char* Wb, int w, int p, int s0,
                                          int K2, int Cout, int g, int t, int tile0 = 0,
                                          int tile_end = 0) {
  constexpr int ES = DT ? 2 : 4;
  constexpr int KSTEP = DT ? 32 : 16;
  constexpr int KU = MrBatch<COLS, LEAN>::KU, NC = MrBatch<COLS, LEAN>::NC;
#pragma unroll
  for (int c4 = 0; c4 < NC; ++c4) {
    const int n0 = ((COLS ? tile0 : 0) + w + 4 * (NC * p + c4)) * 16;
    if (COLS ? n0 >= tile_end * 16 : n0 >= Cout) continue;  // wave-uniform
    const char* wrow = Wb + (size_t)min(n0 + t, Cout - 1) * K2 * ES;
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      if (HEADS && !mr_step_needed(a, n0, s0 + u, KSTEP)) continue;  // wave-uniform
      const int kk = (s0 + u) * KSTEP + g * (KSTEP / 4);
      bw[u][c4] = *reinterpret_cast<const uint4*>(wrow + (size_t)(kk < K2 ? kk : 0) * ES);
    }
  }
}

// Gather-max of TM nodes from flattened node row0 (Eq. 2): row r of dst
// (dst + r * dst_stride, LDS or global memory) receives [x_i | m_i] with
// m_i = max_t keys[idx[i, t]] - x_i.  sIdx holds the TM x k neighbour lists,
// each entry j (clamped to [0, M)) stored as its row offset in 16-byte vectors,
// j * C / VEC, so a load address is one shift-add.  Rows past R are not
// written.  Called by all 256 threads.
// T3: three tasks per thread in flight instead of two (a caller with registers
// to spare takes the 32-node tile's 768 tasks of C = 192 in one round).
template <int DT, int KB, bool T3 = false, bool LEAN = false>
__device__ __forceinline__ void mr_gather_rows(const MrArgs& a, int row0, int TM,
                                               const int32_t* sIdx, char* dst, size_t dst_stride) {
  constexpr int ES = DT ? 2 : 4;
  constexpr int VEC = 16 / ES;
  const int C = a.C, k = a.k, M = a.M, N = a.N, R = a.R;
  const int tid = threadIdx.x;
  const int CG = C / VEC;
  // Each task is one (node, 16-byte channel vector); with a small neighbour
  // bucket two tasks keep their loads in flight together.
  constexpr int KG = KB < 16 ? KB : 16;    // neighbour loads in flight per group
  constexpr int TPT = KB <= 9 && !LEAN ? (T3 ? 3 : 2) : 1;  // tasks per thread per iteration
  const int ntask = TM * CG;
  for (int e0 = tid; e0 < ntask; e0 += TPT * kMrThreads) {
    float mx[TPT][VEC];
    uint4 xraw[TPT];
    const char* kbase[TPT];
    const int32_t* nb[TPT];
#pragma unroll
    for (int q = 0; q < TPT; ++q) {
      const int e = min(e0 + q * kMrThreads, ntask - 1);
      const int r = e / CG, cg = e - r * CG;
      const int row = min(row0 + r, R - 1);
      const int b = row / N;
      xraw[q] = *reinterpret_cast<const uint4*>(static_cast<const char*>(a.x) +
                                                ((size_t)row * C + cg * VEC) * ES);
      kbase[q] = static_cast<const char*>(a.keys) + ((size_t)b * M * C + cg * VEC) * ES;
      nb[q] = sIdx + r * k;
#pragma unroll
      for (int i = 0; i < VEC; ++i) mx[q][i] = -INFINITY;
    }
#pragma unroll 1
    for (int t0 = 0; t0 < KB; t0 += KG) {
      uint4 raw[TPT][KG];
#pragma unroll
      for (int q = 0; q < TPT; ++q)
#pragma unroll
        for (int u = 0; u < KG; ++u) {
          const int tt = t0 + u;
          const uint32_t jo = (uint32_t)nb[q][tt < k ? tt : 0];
          raw[q][u] = *reinterpret_cast<const uint4*>(kbase[q] + ((size_t)jo << 4));
        }
#pragma unroll
      for (int q = 0; q < TPT; ++q)
#pragma unroll
        for (int u = 0; u < KG; ++u) {
          float kf[VEC];
          if (DT) unpack_bf16x8(raw[q][u], kf);
          else { const float4 v = __builtin_bit_cast(float4, raw[q][u]); kf[0] = v.x; kf[1] = v.y; kf[2] = v.z; kf[3] = v.w; }
#pragma unroll
          for (int i = 0; i < VEC; ++i) mx[q][i] = fmaxf(mx[q][i], kf[i]);
        }
    }
#pragma unroll
    for (int q = 0; q < TPT; ++q) {
      const int e = e0 + q * kMrThreads;
      if (e >= ntask) continue;
      const int r = e / CG, cg = e - r * CG;
      float xf[VEC];
      if (DT) unpack_bf16x8(xraw[q], xf);
      else { const float4 v = __builtin_bit_cast(float4, xraw[q]); xf[0] = v.x; xf[1] = v.y; xf[2] = v.z; xf[3] = v.w; }
#pragma unroll
      for (int i = 0; i < VEC; ++i) mx[q][i] -= xf[i];
      if (row0 + r >= R) continue;
      char* d = dst + (size_t)r * dst_stride + cg * 16;
      *reinterpret_cast<uint4*>(d) = xraw[q];
      store_vec<DT>(d + C * ES, mx[q]);
    }
  }
}

// Gather-only tile of the two-pass MRConv: the [x_i | m_i] rows of TM nodes
// from flattened node blk * TM, written to xcat [R, 2C].  sIdx: TM * k ints of
// LDS.  Called by all 256 threads.
constexpr int kMrGatherRows = 16;  // nodes per workgroup of the gather kernel

template <int DT, int KB>
__device__ __forceinline__ void mr_gather_tile(const MrArgs& a, int blk, int TM, int32_t* sIdx,
                                               void* xcat) {
  constexpr int ES = DT ? 2 : 4;
  const int row0 = blk * TM;
  for (int e = threadIdx.x; e < TM * a.k; e += kMrThreads) {
    const int r = e / a.k, tt = e - r * a.k, row = row0 + r;
    const int j = row < a.R ? a.idx[(size_t)row * a.k + tt] : 0;
    sIdx[e] = min(max(j, 0), a.M - 1) * (a.C * ES / 16);
  }
  __syncthreads();
  const size_t stride = (size_t)2 * a.C * ES;
  mr_gather_rows<DT, KB>(a, row0, TM, sIdx, static_cast<char*>(xcat) + row0 * stride, stride);
}

// TM = 16*RT nodes starting at flattened node row0.  smem holds
// mrconv_smem_bytes(C, k, RT) bytes.  Called by all 256 threads.
// HEADS: the multi-head update (a.heads > 1), which skips the zero blocks of W.
// COLS: only the 16-column output tiles tile0 .. tile_end-1 (tile_end within
// the layer's tiles), the column group of a small grid.
// ACT: GELU on each output before its rounding (a.act_out; compiled in only
// for the full block's update, so the other updates carry none of its code).
template <int DT, int RT, int KB, bool HEADS = false, bool T3 = false, bool COLS = false,
          bool LEAN = false, bool ACT = false>
__device__ __forceinline__ void mrconv_tile(char* smem, const MrArgs& a, int row0, int tile0 = 0,
                                            int tile_end = 0) {
  constexpr int TM = 16 * RT;
  constexpr int ES = DT ? 2 : 4;
  const int C = a.C, k = a.k, M = a.M, R = a.R, Cout = a.Cout;
  const int lds_row = 2 * C * ES + 16;
  char* sA = smem;
  int32_t* sIdx = reinterpret_cast<int32_t*>(smem + TM * lds_row);

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, t = lane & 15;

  // -- neighbour lists of the tile ---------------------------------------------
  for (int e = tid; e < TM * k; e += kMrThreads) {
    const int r = e / k, tt = e - r * k, row = row0 + r;
    const int j = row < R ? a.idx[(size_t)row * k + tt] : 0;
    sIdx[e] = min(max(j, 0), M - 1) * (C * ES / 16);
  }

  // -- FC geometry; the first batch of W operands is requested here, after the
  //    lists (loads return in order) and ahead of the gather, so its latency
  //    overlaps the gather's ------------------------------------------------------
  const int K2 = 2 * C;
  const int KSTEP = DT ? 32 : 16;
  const int ksteps = (K2 + KSTEP - 1) / KSTEP;
  const int NCT = (Cout + 15) >> 4;
  const char* Wb = static_cast<const char*>(a.W);
  // output tiles past Cout are never loaded: their operands stay zero (their
  // results are not stored either)
  constexpr int KU = MrBatch<COLS, LEAN>::KU, NC = MrBatch<COLS, LEAN>::NC;
  uint4 bw[KU][NC] = {};
  const int T0 = COLS ? tile0 : 0, TE = COLS ? tile_end : NCT;
  if (T0 + w < TE) mr_load_w<DT, HEADS, COLS, LEAN>(bw, a, Wb, w, 0, 0, K2, Cout, g, t, tile0, tile_end);
  __syncthreads();

  mr_gather_rows<DT, KB, T3, LEAN>(a, row0, TM, sIdx, sA, lds_row);
  __syncthreads();

  // -- FC on MFMA -----------------------------------------------------------------
  // PIPE (the one-launch block's update role, which has the registers): the W
  // operands of the next batch of k-steps are requested before the current
  // batch is multiplied, so no batch after the first waits on its own loads.
  constexpr bool PIPE = T3 && !HEADS && !COLS && !LEAN;
  uint4 bw2[KU][NC] = {};
  for (int p = 0; T0 + w + 4 * NC * p < TE; ++p) {
    f32x4 acc[RT][NC];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int c4 = 0; c4 < NC; ++c4) acc[rt][c4] = f32x4{0.f, 0.f, 0.f, 0.f};
    bool nvalid[NC];
#pragma unroll
    for (int c4 = 0; c4 < NC; ++c4)
      nvalid[c4] = COLS ? T0 + w + 4 * (NC * p + c4) < TE : (w + 4 * (NC * p + c4)) * 16 < Cout;
    auto batch = [&](const uint4 (&bv4)[KU][NC], int s0) {
      bool kin[KU];
#pragma unroll
      for (int u = 0; u < KU; ++u) kin[u] = (s0 + u) * KSTEP + g * (KSTEP / 4) < K2;
#pragma unroll
      for (int u = 0; u < KU; ++u) {
        const int kk = (s0 + u) * KSTEP + g * (KSTEP / 4);
        uint4 af[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          af[rt] = kin[u] ? *reinterpret_cast<const uint4*>(sA + (rt * 16 + t) * lds_row + kk * ES)
                          : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int c4 = 0; c4 < NC; ++c4) {
          if (HEADS && !mr_step_needed(a, (w + 4 * (NC * p + c4)) * 16, s0 + u, KSTEP)) continue;
          // past 2C the A operand is zero and bv a real W element (column 0)
          const uint4 bv = bv4[u][c4];
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) {
            if (DT) {
              acc[rt][c4] = mfma_bf16(af[rt], bv, acc[rt][c4]);
            } else {
              const float4 x4 = __builtin_bit_cast(float4, af[rt]);
              const float4 w4 = __builtin_bit_cast(float4, bv);
              acc[rt][c4] = mfma_f32(x4.x, w4.x, acc[rt][c4]);
              acc[rt][c4] = mfma_f32(x4.y, w4.y, acc[rt][c4]);
              acc[rt][c4] = mfma_f32(x4.z, w4.z, acc[rt][c4]);
              acc[rt][c4] = mfma_f32(x4.w, w4.w, acc[rt][c4]);
            }
          }
        }
      }
    };
    if constexpr (PIPE) {
      // batches in pairs: bw holds batch s0 (for the first pass, requested
      // before the gather), bw2 batch s0 + KU; each set is refilled while
      // the other is multiplied.  Past the contraction nothing is multiplied.
      if (p != 0) mr_load_w<DT, HEADS, COLS, LEAN>(bw, a, Wb, w, p, 0, K2, Cout, g, t, tile0, tile_end);
      for (int s0 = 0; s0 < ksteps; s0 += 2 * KU) {
        if (s0 + KU < ksteps)
          mr_load_w<DT, HEADS, COLS, LEAN>(bw2, a, Wb, w, p, s0 + KU, K2, Cout, g, t, tile0, tile_end);
        batch(bw, s0);
        if (s0 + 2 * KU < ksteps)
          mr_load_w<DT, HEADS, COLS, LEAN>(bw, a, Wb, w, p, s0 + 2 * KU, K2, Cout, g, t, tile0, tile_end);
        if (s0 + KU < ksteps) batch(bw2, s0 + KU);
      }
    } else {
      for (int s0 = 0; s0 < ksteps; s0 += KU) {
        if (p != 0 || s0 != 0)
          mr_load_w<DT, HEADS, COLS, LEAN>(bw, a, Wb, w, p, s0, K2, Cout, g, t, tile0, tile_end);
        batch(bw, s0);
      }
    }
    // -- epilogue: + bias, [GELU], round once, store -----------------------------
    // a full tile (all TM nodes below R, Cout a multiple of 16; uniform)
    // stores without per-lane guards
    const bool full = row0 + TM <= R && (Cout & 15) == 0;
#pragma unroll
    for (int c4 = 0; c4 < NC; ++c4) {
      if (!nvalid[c4]) continue;  // wave-uniform
      const int n = (T0 + w + 4 * (NC * p + c4)) * 16 + t;
      const int nc = min(n, Cout - 1);
      float bn = 0.f;
      if (a.bias) {
        bn = DT ? bf16_bits_to_f32(static_cast<const uint16_t*>(a.bias)[nc])
                : static_cast<const float*>(a.bias)[nc];
      }
      auto put = [&](int rt, int v) {
        const size_t o = (size_t)(row0 + rt * 16 + 4 * g + v) * Cout + n;
        float y = acc[rt][c4][v] + bn;
        if constexpr (ACT) y = gelu_f32(y);
        if (DT) static_cast<uint16_t*>(a.out)[o] = (uint16_t)f32_to_bf16_bits(y);
        else static_cast<float*>(a.out)[o] = y;
      };
      if (full) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int v = 0; v < 4; ++v) put(rt, v);
      } else {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (n < Cout && row0 + rt * 16 + 4 * g + v < R) put(rt, v);
      }
    }
  }
}

}  // namespace gl
