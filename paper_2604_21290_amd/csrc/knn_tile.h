// Fused dilated kNN graph build for gfx950 (Sec. II-B Eq. 4; Sec. IV-B; Alg. 2).
//
// One workgroup = 4 waves = 16 query rows of one image.
//   1. keys are processed in chunks of 256 (16 MFMA tiles of 16 keys); wave w
//      computes tiles w, w+4, w+8, w+12 together, with the operand loads of a
//      batch of k-steps for all four tiles issued before the MFMAs use them.
//      The Gram G = Q K^T contracts the raw stored values (bf16 products are
//      exact in fp32); the query and key rows' squared norms accumulate from
//      the same operand registers (packed dot products);
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
#pragma once

#include "gl_device.h"
#include "gl_kernels.h"

namespace gl {

constexpr int kKnnRows = 16;     // query rows per workgroup
constexpr int kKnnChunk = 256;   // keys per chunk
constexpr int kKnnThreads = 256;
constexpr int kKnnKU = 3;        // k-steps whose operands are loaded as one batch
constexpr int kKnnTPP = 4;       // key tiles of a chunk per wave, computed in one pass

// Sort one value per lane across each aligned row of 16 lanes (ascending).
// All cross-lane moves are DPP modifiers within the row.
__device__ __forceinline__ uint32_t sort16_lanes(uint32_t c, int t) {
#pragma unroll
  for (int s = 1; s <= 4; ++s) {
#pragma unroll
    for (int j = s - 1; j >= 0; --j) {
      const bool up = ((t >> s) & 1) == 0;
      const bool lower = ((t >> j) & 1) == 0;
      c = lane_cas16(c, j, lower == up);
    }
  }
  return c;
}

// Merge a sorted run of 16 (one per lane, `c`) into the sorted list L of
// 16*R elements (element e = t + 16*a), keeping the 16*R smallest, sorted.
template <int R>
__device__ __forceinline__ void merge16_into_list(uint32_t* L, uint32_t c, int t) {
  // half-cleaner against the reversed run: only the last 16 list slots can change
  L[R - 1] = min(L[R - 1], lane_reverse16(c));
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
      L[a] = lane_cas16(L[a], j, ((t >> j) & 1) == 0);
    }
  }
}

// List element e (wave-uniform) of each row, broadcast to the row's 16 lanes.
template <int R>
__device__ __forceinline__ uint32_t list_element(const uint32_t* L, int e, int lane) {
  // register select by masks (a select chain can be lowered to an indexed
  // private-memory load)
  uint32_t v = 0;
#pragma unroll
  for (int a = 0; a < R; ++a) v |= L[a] & (0u - (uint32_t)((e >> 4) == a));
  return row_broadcast16(v, e & 15, lane);
}

// The 4 smallest of a lane's 16 values, ascending, in v[0..3]; v[4..15] hold
// the other 12 in no order.  Four sorted groups of 4 (five comparators each),
// then three merges that keep the 4 smallest of two sorted groups sorted
// (a half-cleaner against the reversed second group, then a 4-element
// bitonic sort): 44 compare-exchanges against the full bitonic sort's 80.
__device__ __forceinline__ void top4_regs_asc(uint32_t (&v)[16]) {
#pragma unroll
  for (int q = 0; q < 16; q += 4) {
    cas_asc(v[q], v[q + 1]);
    cas_asc(v[q + 2], v[q + 3]);
    cas_asc(v[q], v[q + 2]);
    cas_asc(v[q + 1], v[q + 3]);
    cas_asc(v[q + 1], v[q + 2]);
  }
  auto merge4 = [&](int a, int b) {
#pragma unroll
    for (int i = 0; i < 4; ++i) cas_asc(v[a + i], v[b + 3 - i]);
    cas_asc(v[a], v[a + 2]);
    cas_asc(v[a + 1], v[a + 3]);
    cas_asc(v[a], v[a + 1]);
    cas_asc(v[a + 2], v[a + 3]);
  };
  merge4(0, 4);
  merge4(8, 12);
  merge4(0, 8);
}

// Merge this lane's 16 candidates v (one row per 16 lanes) into the row's
// sorted list L of the KK smallest keys; tau is the list's KK-th key (all ones
// while the list is not full).  Candidates not below tau are dropped first; the
// rest are sorted per lane and merged 16 at a time, smallest first.
template <int R>
__device__ __forceinline__ void select_chunk(uint32_t* L, uint32_t& tau, uint32_t (&v)[16], int KK,
                                             int t, int lane) {
  bool pass = false;
#pragma unroll
  for (int m = 0; m < 16; ++m) pass |= v[m] < tau;
  if (__any(pass)) {
#pragma unroll
    for (int m = 0; m < 16; ++m) v[m] = v[m] < tau ? v[m] : 0xffffffffu;
    if constexpr (R == 1) {
      // A list of at most 16 rarely takes more than each lane's 4 smallest:
      // those are ordered first, and the rest only when some lane's fifth
      // smallest is still below the threshold after them.
      top4_regs_asc(v);
#pragma unroll
      for (int m = 0; m < 4; m += 2) {
        if (!__any(v[m] < tau)) return;
        const uint32_t c0 = sort16_lanes(v[m], t);
        const uint32_t c1 = sort16_lanes(v[m + 1], t);
        merge16_into_list<R>(L, c0, t);
        merge16_into_list<R>(L, c1, t);
        tau = list_element<R>(L, KK - 1, lane);
      }
      uint32_t fifth = v[4];
#pragma unroll
      for (int m = 5; m < 16; ++m) fifth = min(fifth, v[m]);
      if (!__any(fifth < tau)) return;
      sort_regs_asc<16>(v);  // v[0..3] are already the smallest four, in order
#pragma unroll
      for (int m = 4; m < 16; m += 2) {
        if (!__any(v[m] < tau)) break;
        const uint32_t c0 = sort16_lanes(v[m], t);
        const uint32_t c1 = sort16_lanes(v[m + 1], t);
        merge16_into_list<R>(L, c0, t);
        merge16_into_list<R>(L, c1, t);
        tau = list_element<R>(L, KK - 1, lane);
      }
      return;
    }
    sort_regs_asc<16>(v);
    // Two layers per pass: their 16-lane sorts are independent chains that
    // the scheduler interleaves.  The second layer may hold no key below the
    // updated tau; merging it then changes nothing among the first KK list
    // elements (keys are unique, so none of them can be displaced).
#pragma unroll
    for (int m = 0; m < 16; m += 2) {
      if (!__any(v[m] < tau)) break;
      const uint32_t c0 = sort16_lanes(v[m], t);
      const uint32_t c1 = sort16_lanes(v[m + 1], t);
      merge16_into_list<R>(L, c0, t);
      merge16_into_list<R>(L, c1, t);
      tau = list_element<R>(L, KK - 1, lane);
    }
  }
}

// One 16-row query tile of one image: rows row0 .. row0+15 of x_b against
// all M keys of keys_b; writes idx_b[row, 0..k-1].  smem holds
// knn_smem_bytes() bytes (the candidate strip).  Called by all 256 threads.
template <int DT, int R>
__device__ __forceinline__ void knn_tile(char* smem, const char* __restrict__ xb,
                                         const char* __restrict__ kb, int N, int C, int M, int k,
                                         int dil, int KK, int ib, float qscale, uint32_t qmax,
                                         int row0, int32_t* __restrict__ idx_b) {
  constexpr int ES = DT ? 2 : 4;
  uint32_t* sStrip = reinterpret_cast<uint32_t*>(smem);

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, t = lane & 15;

  // contraction steps: 32 channels (bf16) or 16 channels (fp32, 4 MFMAs) each
  const int KSTEP = DT ? 32 : 16;
  const int ksteps = (C + KSTEP - 1) / KSTEP;
  // this lane's A-operand row (query row0 + t; rows past N repeat row N-1)
  const char* qg = xb + (size_t)min(row0 + t, N - 1) * C * ES;

  // Operands of one batch: k-steps s0 .. s0+KU-1 of the query rows and of the
  // wave's key tiles w, w+4, w+8, w+12 in the chunk at chunk0 (rows clamped;
  // channels past C read channel 0 and are zeroed when used).  Tiles past the
  // chunk repeat tile w; in bf16 they are multiplied like the others and
  // dropped in the epilogue, since a branch around the MFMAs makes the compiler
  // copy the accumulators between register files at every step.
  uint4 bf[kKnnKU][kKnnTPP], af[kKnnKU];
  auto load_batch = [&](int chunk0, int ntiles, int s0) {
    int kr[kKnnTPP];
#pragma unroll
    for (int p = 0; p < kKnnTPP; ++p) {
      const int tt = w + 4 * p;
      kr[p] = min(chunk0 + (tt < ntiles ? tt : w) * 16 + t, M - 1);
    }
#pragma unroll
    for (int u = 0; u < kKnnKU; ++u) {
      const int c = (s0 + u) * KSTEP + g * (KSTEP / 4);
      const size_t off = (size_t)(c < C ? c : 0) * ES;
      af[u] = *reinterpret_cast<const uint4*>(qg + off);
#pragma unroll
      for (int p = 0; p < kKnnTPP; ++p)
        bf[u][p] = *reinterpret_cast<const uint4*>(kb + (size_t)kr[p] * C * ES + off);
    }
  };
  const int ntiles0 = (min(kKnnChunk, M) + 15) >> 4;
  if (w < ntiles0) load_batch(0, ntiles0, 0);

  uint32_t L[R];
#pragma unroll
  for (int a = 0; a < R; ++a) L[a] = 0xffffffffu;
  uint32_t tau = 0xffffffffu;
  float qr[4] = {0.f, 0.f, 0.f, 0.f};  // inverse norms of rows 4g .. 4g+3 (MFMA output rows)

  for (int chunk0 = 0; chunk0 < M; chunk0 += kKnnChunk) {
    const int nvalid = min(kKnnChunk, M - chunk0);
    const int ntiles = (nvalid + 15) >> 4;
    // -- Gram + epilogue: wave w takes tiles w, w+4, w+8, w+12 in one pass --------
    if (w < ntiles) {
      f32x4 acc[kKnnTPP];
      float ss[kKnnTPP];
      float qss = 0.f;
#pragma unroll
      for (int p = 0; p < kKnnTPP; ++p) {
        acc[p] = f32x4{0.f, 0.f, 0.f, 0.f};
        ss[p] = 0.f;
      }
      for (int s0 = 0; s0 < ksteps; s0 += kKnnKU) {
        if (chunk0 != 0 || s0 != 0) load_batch(chunk0, ntiles, s0);
#pragma unroll
        for (int u = 0; u < kKnnKU; ++u) {
          const int c = (s0 + u) * KSTEP + g * (KSTEP / 4);
          const bool in = c < C;
          const uint4 a = in ? af[u] : make_uint4(0, 0, 0, 0);
          if (chunk0 == 0) qss = DT ? sumsq_bf16x8(a, qss) : sumsq_f32x4(a, qss);
#pragma unroll
          for (int p = 0; p < kKnnTPP; ++p) {
            // (fp32 keeps the test: its four MFMAs per step leave no registers
            // for the extra tile in the one-launch block)
            if (!DT && w + 4 * p >= ntiles) continue;
            const uint4 b = in ? bf[u][p] : make_uint4(0, 0, 0, 0);
            if (DT) {
              acc[p] = mfma_bf16(a, b, acc[p]);
              ss[p] = sumsq_bf16x8(b, ss[p]);
            } else {
              const float4 av = __builtin_bit_cast(float4, a);
              const float4 f = __builtin_bit_cast(float4, b);
              acc[p] = mfma_f32(av.x, f.x, acc[p]);
              acc[p] = mfma_f32(av.y, f.y, acc[p]);
              acc[p] = mfma_f32(av.z, f.z, acc[p]);
              acc[p] = mfma_f32(av.w, f.w, acc[p]);
              ss[p] = sumsq_f32x4(b, ss[p]);
            }
          }
        }
      }
      if (chunk0 == 0) {
        // lane (g, t) summed slice g of query row t; complete the sum, then
        // fetch the inverse norms of the output rows 4g .. 4g+3
        qss += __shfl_xor(qss, 16);
        qss += __shfl_xor(qss, 32);
        const float rq = 1.f / fmaxf(sqrtf(qss), 1e-12f);
#pragma unroll
        for (int v = 0; v < 4; ++v) qr[v] = __shfl(rq, 4 * g + v);
      }
#pragma unroll
      for (int p = 0; p < kKnnTPP; ++p) {
        const int tt = w + 4 * p;
        if (tt >= ntiles) continue;
        float sj = ss[p];
        sj += __shfl_xor(sj, 16);
        sj += __shfl_xor(sj, 32);
        const int j = chunk0 + tt * 16 + t;
        // qscale is a power of two, so scaling the factors scales d1 exactly
        const float m2rjS = -2.f * key_rnorm(sj) * qscale;
        const float baseS = (sj > 0.f ? 2.f : 1.f) * qscale;  // (1 + n_j) * qscale
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float d1s = fmaf(acc[p][v] * m2rjS, qr[v], baseS);
          const uint32_t q = min((uint32_t)fmaxf(d1s, 0.f), qmax);
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

    select_chunk<R>(L, tau, v, KK, t, lane);
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

}  // namespace gl
