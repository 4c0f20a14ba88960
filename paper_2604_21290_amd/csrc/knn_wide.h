// LDS-staged dilated kNN graph build for bf16 rows against at most 256 keys
// (Sec. II-B Eq. 4; Sec. IV-B; Alg. 2), the wide-channel build.
//
// The in-register kernel reads every key row once per 16 query rows; at
// C = 640 that is 13 full passes over the keys of an image through L2 for each
// build.  Here one workgroup = 4 waves = 32 query rows of one image against
// all of its keys, and the contraction is staged through LDS like a GEMM:
//   1. each stage moves 128 bytes (64 channels) of the query rows and of
//      the key rows into LDS, double-buffered, with two register sets so the
//      next two stages' global loads are in flight while one is multiplied.  The thread that moves a
//      16-byte vector adds its squares to that row's norm;
//   2. each wave keeps the Gram block of 16 rows against its share of the
//      key tiles in MFMA accumulators;
//   3. after the last stage the row norms are reduced, and the distance
//      epilogue forms the same packed keys as the in-register kernel
//      (fixed-point d1 = (1 + n_j) - 2 r_i r_j G_ij above the key index) into
//      an LDS block [rows][keys] that reuses the stage buffers;
//   4. each row is selected by 16 lanes with the in-register kernel's
//      filtered sort-and-merge, and ranks 0, d, 2d, ... are written to idx.
// The N x M distances never leave the chip.
#pragma once

#include "knn_tile.h"

namespace gl {

constexpr int kWdStep = 128;                // bytes of each row per stage
constexpr int kWdRow = kWdStep + 16;        // LDS row stride
constexpr int kWdMaxKeys = 256;
constexpr int kWdThreads = 256;

// Key rows staged: M rounded up to a multiple of 32 (one staging vector per
// thread covers 32 rows), bucketed so few variants are compiled.
inline int knn_wide_key_rows(int M) { return M <= 64 ? 64 : M <= 128 ? 128 : M <= 224 ? 224 : 256; }

// QW row tiles of 16 query rows per workgroup (QR = 16 QW rows); the key
// tiles are split over the 4 / QW waves that share a row tile.
template <int QW, int KROWS>
struct WideGeom {
  static constexpr int kQR = 16 * QW;
  static constexpr int kSplit = 4 / QW;
  static constexpr int kBuf = (kQR + KROWS) * kWdRow;                     // one stage buffer
  static constexpr int kNorms = 2 * kBuf;                                 // r_i, r_j, 1 + n_j
  static constexpr size_t kSmem = (size_t)2 * kBuf + (kQR + 2 * KROWS) * 4;
  static constexpr int kNV = (kQR + KROWS) / 32;                          // vectors per thread per stage
  static constexpr int kNKT = KROWS / 16 / kSplit;                        // key tiles per wave at most
};

template <int QW>
inline size_t wide_smem(int M) {
  switch (knn_wide_key_rows(M)) {
    case 64: return WideGeom<QW, 64>::kSmem;
    case 128: return WideGeom<QW, 128>::kSmem;
    case 224: return WideGeom<QW, 224>::kSmem;
    default: return WideGeom<QW, 256>::kSmem;
  }
}

// Row tiles per workgroup: 32 query rows measured faster than 64 at every
// shape tried (ViG-B, ViG-S, pyramid stages 3-4): twice the workgroups, two
// waves per SIMD, for twice the key staging.
constexpr int kWdQW = 2;


// One workgroup's tile: blk is its index among the B * ceil(N / QR) tiles.
// smem holds WideGeom<QW, KROWS>::kSmem bytes.  Called by all 256 threads.
// DB: two staging register sets (else one, for a caller with fewer registers).
// SKIP: the padding stage of an odd stage count, and a wave's last key tile
// when it lies wholly past M, are not multiplied (measured faster in the
// one-launch block, slower standalone; the result is the same: a zero stage
// adds nothing, and tiles past M are masked in the epilogue).
template <int R, int QW, int KROWS, bool DB = true, bool SKIP = false>
__device__ __forceinline__ void knn_wide_tile(char* smem, const KnnArgs& a, int blk) {
  using G = WideGeom<QW, KROWS>;
  constexpr int NV = G::kNV, NKT = G::kNKT, QR = G::kQR, SPLIT = G::kSplit;
  const int N = a.N, C = a.C, M = a.M, k = a.k, dil = a.dil, KK = a.KK, ib = a.ib;
  const int rowb = 2 * C;
  const int nstage = (rowb + kWdStep - 1) / kWdStep;
  const int nkt = (M + 15) >> 4;
  const int nqt = (N + QR - 1) / QR;
  const int b = blk / nqt, q0 = (blk - b * nqt) * QR;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, t = lane & 15;
  // wave w: row tile w % QW, key tiles w / QW + SPLIT * j
  const int wr = w % QW, wk = w / QW;
  const char* xb = static_cast<const char*>(a.x) + (size_t)b * N * rowb;
  const char* kb = static_cast<const char*>(a.keys) + (size_t)b * M * rowb;
  float* sRq = reinterpret_cast<float*>(smem + G::kNorms);   // query 1 / ||x_i||
  float* sRk = sRq + QR;                                      // key 1 / ||k_j||
  float* sNk = sRk + KROWS;                                   // 1 + n_j

  // -- staging: vector i of this thread is row (tid / 8) + 32 i of the stage
  //    (rows 0..QR-1 queries, then keys), 16-byte slot tid % 8.  Rows past N or M
  //    repeat the last row; channels past C read channel 0 and are zeroed.
  const int slot = (tid & 7) * 16;
  const char* src[NV];
  int lo[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int r = (tid >> 3) + 32 * i;
    src[i] = r < QR ? xb + (size_t)min(q0 + r, N - 1) * rowb + slot
                    : kb + (size_t)min(r - QR, M - 1) * rowb + slot;
    lo[i] = r * kWdRow + slot;
  }
  // two register sets: while one stage is multiplied out of LDS, the next is
  // waiting in one set and the one after is on its way into the other
  u32x4 st0[NV], st1[NV];
  float ss[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) ss[i] = 0.f;
  auto gload = [&](u32x4 (&st)[NV], int s) {
    const int off = s * kWdStep + slot < rowb ? s * kWdStep : 0;
#pragma unroll
    for (int i = 0; i < NV; ++i) st[i] = *reinterpret_cast<const u32x4*>(src[i] + off);
  };
  auto sstore = [&](u32x4 (&st)[NV], int s, int buf) {
    char* d = smem + buf * G::kBuf;
    if ((s + 1) * kWdStep <= rowb) {  // wave-uniform: the whole stage is inside C
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        ss[i] = sumsq_bf16x8(__builtin_bit_cast(uint4, st[i]), ss[i]);
        *reinterpret_cast<u32x4*>(d + lo[i]) = st[i];
      }
    } else {
      const bool in = s * kWdStep + slot < rowb;
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const u32x4 v = in ? st[i] : u32x4{0, 0, 0, 0};
        ss[i] = sumsq_bf16x8(__builtin_bit_cast(uint4, v), ss[i]);
        *reinterpret_cast<u32x4*>(d + lo[i]) = v;
      }
    }
  };

  f32x4 acc[NKT];
#pragma unroll
  for (int j = 0; j < NKT; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto multiply = [&](int s) {
    const char* sa = smem + (s & 1) * G::kBuf;
#pragma unroll
    for (int kk = 0; kk < kWdStep / 64; ++kk) {
      const uint4 af = *reinterpret_cast<const uint4*>(sa + (16 * wr + t) * kWdRow + kk * 64 + g * 16);
      // every staged key tile is multiplied (tiles past M hold repeated rows and
      // are masked in the epilogue): standalone, a branch here made the compiler
      // copy the accumulators around it.  With SKIP (accumulators in VGPRs)
      // the wave's last tile is skipped when it lies wholly past M.
#pragma unroll
      for (int j = 0; j < NKT; ++j) {
        const int kt = wk + SPLIT * j;
        if (SKIP && j == NKT - 1 && kt >= nkt) continue;
        const uint4 bf =
            *reinterpret_cast<const uint4*>(sa + (QR + 16 * kt + t) * kWdRow + kk * 64 + g * 16);
        acc[j] = mfma_bf16(af, bf, acc[j]);
      }
    }
  };

  // At the top of step s, stage s is in LDS buffer s & 1 and stage s + 1 is in
  // flight into st1 (even s) or st0 (odd s).  The loop runs whole pairs of
  // steps, so that each register set keeps its role: stages past the last (at
  // most two, plus one when the count is odd) load in-range addresses and are
  // stored as zeros, which add nothing to the accumulators or the norms.  With
  // SKIP the one padding stage of an odd count is not multiplied.
  if constexpr (DB) {
    const int npair = (nstage + 1) >> 1;
    gload(st0, 0);
    gload(st1, 1);
    sstore(st0, 0, 0);
    __syncthreads();
    for (int pr = 0; pr < npair; ++pr) {
      const int s = 2 * pr;
      gload(st0, s + 2);
      multiply(s);
      sstore(st1, s + 1, 1);
      __syncthreads();
      gload(st1, s + 3);
      if (!SKIP || s + 1 < nstage) multiply(s + 1);  // an odd count's last pair has one stage
      sstore(st0, s + 2, 0);
      __syncthreads();
    }
  } else {
    gload(st0, 0);
    sstore(st0, 0, 0);
    __syncthreads();
    for (int s = 0; s < nstage; ++s) {
      if (s + 1 < nstage) gload(st0, s + 1);
      multiply(s);
      if (s + 1 < nstage) sstore(st0, s + 1, (s + 1) & 1);
      __syncthreads();
    }
  }

  // -- row norms: the 8 threads of a row are 8 consecutive lanes ---------------------
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    float v = ss[i];
    v += __shfl_xor(v, 1);
    v += __shfl_xor(v, 2);
    v += __shfl_xor(v, 4);
    const int r = (tid >> 3) + 32 * i;
    if ((tid & 7) == 0) {
      if (r < QR) {
        sRq[r] = 1.f / fmaxf(sqrtf(v), 1e-12f);
      } else {
        sRk[r - QR] = key_rnorm(v);
        sNk[r - QR] = v > 0.f ? 2.f : 1.f;
      }
    }
  }
  __syncthreads();

  // -- distance epilogue into the key block [QR][KROWS] (over the stage buffers) --------
  uint32_t* sKey = reinterpret_cast<uint32_t*>(smem);
  {
    const float qscale = a.qscale;
    const uint32_t qmax = a.qmax;
    float qr[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) qr[v] = sRq[16 * wr + 4 * g + v];
#pragma unroll
    for (int j = 0; j < NKT; ++j) {
      const int kt = wk + SPLIT * j;
      if (kt >= nkt) continue;
      const int col = 16 * kt + t;
      // qscale is a power of two, so scaling the factors scales d1 exactly
      const float m2rjS = -2.f * sRk[col] * qscale;
      const float baseS = sNk[col] * qscale;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float d1s = fmaf(acc[j][v] * m2rjS, qr[v], baseS);
        const uint32_t q = min((uint32_t)fmaxf(d1s, 0.f), qmax);
        sKey[(16 * wr + 4 * g + v) * KROWS + col] = col < M ? ((q << ib) | (uint32_t)col) : 0xffffffffu;
      }
    }
  }
  __syncthreads();

  // -- selection: wave w owns rows 4QW w .. 4QW w + 4QW - 1, four at a time (16 lanes each)
  const uint32_t mask = (1u << ib) - 1u;
#pragma unroll 1
  for (int p = 0; p < QW; ++p) {
    const int rl = 4 * QW * w + 4 * p + g;
    uint32_t v[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const int col = t + 16 * m;
      v[m] = (16 * m < KROWS && col < nkt * 16) ? sKey[rl * KROWS + col] : 0xffffffffu;
    }
    uint32_t L[R];
#pragma unroll
    for (int q = 0; q < R; ++q) L[q] = 0xffffffffu;
    uint32_t tau = 0xffffffffu;
    select_chunk<R>(L, tau, v, KK, t, lane);
    const int row = q0 + rl;
    if (row < N) {
      int32_t* o = a.idx + ((size_t)b * N + row) * k;
#pragma unroll
      for (int q = 0; q < R; ++q) {
        const int e = t + 16 * q;
        if (e < KK && (e % dil) == 0) o[e / dil] = (int32_t)(L[q] & mask);
      }
    }
  }
}

}  // namespace gl
