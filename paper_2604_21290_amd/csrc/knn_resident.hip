// kNN graph build for many query rows against a small key set held in LDS
// (Sec. II-B Eq. 4; Sec. IV-B; Alg. 2).  This is the shape of a pyramid's
// first stage, where the 3136 nodes of a 56 x 56 grid meet the 196 keys of
// its 4 x 4 pooled grid (Sec. IV-E).
//
// The in-register kernel gives a workgroup 16 query rows, and each wave
// loads, norms and multiplies a quarter of the key tiles.  With N >> M that
// key-side work is paid N / 16 times per image.  Here a workgroup of 4 waves
// owns 64 query rows:
//   1. the image's keys (M <= 256 rows, 32 < C <= 128 channels, bf16) are
//      staged into LDS once, and each key's scale pair is computed once from
//      them;
//   2. each wave multiplies its own 16 query rows against every key tile,
//      with B operands read from LDS;
//   3. the accumulators are already laid out as the selection wants them:
//      lanes 16g .. 16g+15 hold keys t of each tile for rows 4g .. 4g+3, one
//      register per row.  So each of a wave's four row groups is selected
//      straight from registers with the filtered sort-and-merge, and no
//      candidate strip goes through LDS.
// The packed keys are bit-identical to those of the kernel the one-launch
// block uses as its build role for the same shape: the in-register tile below
// C = 128, the LDS-staged wide tile from C = 128 on.  The MFMA contraction
// order and the epilogue are the same as both; the norms are summed in the
// order of the kernel matched (per 8-channel slice of each 32-channel step,
// chained over the steps, then (s0 + s1) + (s2 + s3); or per 16-byte slot of
// each 128-byte stage, chained over the stages, then reduced over the eight
// slots as a tree).  So the graph is the same whichever kernel builds it.
#include "knn_tile.h"

namespace gl {

constexpr int kRsRows = 64;  // query rows per four-wave workgroup (16 per wave)

// LDS layout: key rows [KT*16][stride bytes], 64 zero bytes, then the scale
// pairs (-2 r_j 2^(30-ib), (1 + n_j) 2^(30-ib)) [KT*16] as float2.  A row
// holds its 2C bytes and a skew that puts the 16 rows one MFMA operand read
// touches on 16 different 16-byte bank groups: stride / 16 must be odd.  A
// contraction step past C reads the row's zeroed skew bytes and then the next
// row (or the zero bytes after the last), all finite, where the A operand is
// zero.
__host__ __device__ inline int resident_stride(int C) { return 2 * C + ((C / 8) % 2 == 0 ? 16 : 32); }

template <int KT>
inline size_t resident_smem(int C) {
  return (size_t)KT * 16 * resident_stride(C) + 64 + (size_t)KT * 16 * 8;
}

// Key tiles compiled for M keys: 4, 8, 13 (M <= 208) or 16.
inline int knn_resident_tiles(int M) { return M <= 64 ? 4 : M <= 128 ? 8 : M <= 208 ? 13 : 16; }

// bf16, at most 256 keys of 33..160 channels, and enough query rows to give
// the chip at least 384 workgroups of 64 (about 1.5 per CU; past 128 channels
// the LDS holds two workgroups per CU).
bool knn_use_resident(int B, int N, int M, int C, int dt_bf16) {
  return dt_bf16 && M <= 256 && C > 32 && C <= 160 && C % 8 == 0 &&
         (long long)B * ((N + kRsRows - 1) / kRsRows) >= 384;
}

// Five contraction steps (C > 128) stage 70 KB of keys, two workgroups per CU,
// so that variant is compiled for two waves per SIMD.
template <int R, int KS, int KT, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(KS > 4 ? 2 : 4, 8))) void knn_resident_kernel(KnnArgs a) {
  constexpr int NT = 64 * NW, ROWS = 16 * NW;
  extern __shared__ __align__(16) char smem[];
  constexpr int NK = KT * 16;  // key rows staged
  // key tiles that are whole for every M of this bucket (M > 0, 64, 128, 208)
  constexpr int kFull = KT == 4 ? 0 : KT == 8 ? 4 : KT == 13 ? 8 : 13;
  const int N = a.N, C = a.C, M = a.M, k = a.k, dil = a.dil, KK = a.KK, ib = a.ib;
  const int nqt = (N + ROWS - 1) / ROWS;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int b = blk / nqt, q0 = (blk - b * nqt) * ROWS;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, t = lane & 15;
  const int rowb = 2 * C, stride = resident_stride(C), nvec = C / 8;
  const char* xb = static_cast<const char*>(a.x) + (size_t)b * N * rowb;
  const char* kb = static_cast<const char*>(a.keys) + (size_t)b * M * rowb;
  char* sZero = smem + NK * stride;
  float2* sScale = reinterpret_cast<float2*>(sZero + 64);

  // -- this wave's query rows: A operands of every contraction step, issued
  //    first so they travel while the keys are staged
  const char* qg = xb + (size_t)min(q0 + 16 * w + t, N - 1) * rowb;
  uint4 af[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int c = s * 32 + g * 8;
    af[s] = *reinterpret_cast<const uint4*>(qg + (size_t)(c < C ? c : 0) * 2);
  }

  // -- stage the keys: vector i is slot i % nvec of row i / nvec (rows past M
  //    repeat row M-1; indices past the last vector repeat it, so every pass
  //    loads and stores unconditionally).  The image's M rows are one
  //    contiguous range of global memory.
  const int total = NK * nvec;
  const uint32_t magic = (65536u + nvec - 1) / nvec;  // i / nvec = (i * magic) >> 16 for i < 4096
  constexpr int NV = (NK * KS * 4 + NT - 1) / NT;    // passes for the widest rows of KS steps
  uint4 st[NV];
  int dst[NV];
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int i = min(tid + NT * u, total - 1);
    const int r = (int)(((uint32_t)i * magic) >> 16), v = i - r * nvec;
    dst[u] = r * stride + v * 16;
    st[u] = *reinterpret_cast<const uint4*>(kb + ((size_t)min(r, M - 1) * nvec + v) * 16);
  }
#pragma unroll
  for (int u = 0; u < NV; ++u) *reinterpret_cast<uint4*>(smem + dst[u]) = st[u];
  // zero each row's skew bytes and the bytes after the last row: a contraction
  // step past C multiplies them by a zero A operand, and uninitialised LDS may
  // hold NaN patterns (0 * NaN is NaN)
  if (tid < NK) {
    for (int o = rowb; o < stride; o += 16)
      *reinterpret_cast<uint4*>(smem + tid * stride + o) = make_uint4(0, 0, 0, 0);
  }
  if (tid < 4) *reinterpret_cast<uint4*>(sZero + 16 * tid) = make_uint4(0, 0, 0, 0);
  __syncthreads();

  // -- key scale pairs, one thread per key row, summed in the order of the
  //    block's build role for this shape (slices past C add zero there).
  //    Below C = 128 (the in-register tile): slice p, channels s*32 + 8p .. +7
  //    of every step s, chained over s, then (s0 + s1) + (s2 + s3), that
  //    kernel's shuffle order.  From C = 128 (the wide tile): slot p, channels
  //    64 S + 8p .. +7 of every 128-byte stage S, chained over S, then the
  //    xor tree over the eight slots.
  const bool wide = C >= 128;
  const float qscale = a.qscale;
  if (tid < NK) {
    const char* row = smem + tid * stride;
    float sj;
    if (wide) {
      float sl[8];
#pragma unroll
      for (int p = 0; p < 8; ++p) {
        float acc = 0.f;
#pragma unroll
        for (int S = 0; S < (KS + 1) / 2; ++S)
          if (S * 64 + p * 8 < C)
            acc = sumsq_bf16x8(*reinterpret_cast<const uint4*>(row + S * 128 + p * 16), acc);
        sl[p] = acc;
      }
      sj = ((sl[0] + sl[1]) + (sl[2] + sl[3])) + ((sl[4] + sl[5]) + (sl[6] + sl[7]));
    } else {
      float sl[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        float acc = 0.f;
#pragma unroll
        for (int s = 0; s < KS; ++s)
          if (s * 32 + p * 8 < C)
            acc = sumsq_bf16x8(*reinterpret_cast<const uint4*>(row + s * 64 + p * 16), acc);
        sl[p] = acc;
      }
      sj = (sl[0] + sl[1]) + (sl[2] + sl[3]);
    }
    sScale[tid] = make_float2(-2.f * key_rnorm(sj) * qscale, (sj > 0.f ? 2.f : 1.f) * qscale);
  }

  // -- query norms in the same order (lane g holds channels 32 s + 8 g of
  //    step s: slice g of the step, or slot g (even s) / g + 4 (odd s) of
  //    stage s / 2), and the Gram
#pragma unroll
  for (int s = 0; s < KS; ++s)
    if (s * 32 + g * 8 >= C) af[s] = make_uint4(0, 0, 0, 0);
  float qss;
  if (wide) {
    float qa = 0.f, qb = 0.f;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      if (s & 1) qb = sumsq_bf16x8(af[s], qb);
      else qa = sumsq_bf16x8(af[s], qa);
    }
    qa += __shfl_xor(qa, 16);
    qa += __shfl_xor(qa, 32);
    qb += __shfl_xor(qb, 16);
    qb += __shfl_xor(qb, 32);
    qss = qa + qb;
  } else {
    qss = 0.f;
#pragma unroll
    for (int s = 0; s < KS; ++s) qss = sumsq_bf16x8(af[s], qss);
    qss += __shfl_xor(qss, 16);
    qss += __shfl_xor(qss, 32);
  }
  const float rq = 1.f / fmaxf(sqrtf(qss), 1e-12f);
  float qr[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) qr[v] = __shfl(rq, 4 * g + v);

  f32x4 acc[KT];
#pragma unroll
  for (int m = 0; m < KT; ++m) {
    acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
    const char* kr = smem + (16 * m + t) * stride + g * 16;
#pragma unroll
    for (int s = 0; s < KS; ++s)
      acc[m] = mfma_bf16(af[s], *reinterpret_cast<const uint4*>(kr + s * 64), acc[m]);
  }
  __syncthreads();  // the scale pairs are written

  // -- epilogue and selection, one row of each 16-lane group at a time -------
  const uint32_t qmax = a.qmax, mask = (1u << ib) - 1u;
  float2 sc[KT];
#pragma unroll
  for (int m = 0; m < KT; ++m) sc[m] = sScale[16 * m + t];
  // (unrolled: a run-time v would select acc[m][v] and qr[v] out of four
  // registers on every tile)
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    uint32_t c16[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      if (m < KT) {
        const int j = 16 * m + t;
        // qscale is a power of two, so scaling the factors scales d1 exactly
        const float d1s = fmaf(acc[m][v] * sc[m].x, qr[v], sc[m].y);
        const uint32_t q = min((uint32_t)fmaxf(d1s, 0.f), qmax);
        // tiles below the bucket's smallest M hold real keys only
        c16[m] = (m < kFull || j < M) ? ((q << ib) | (uint32_t)j) : 0xffffffffu;
      } else {
        c16[m] = 0xffffffffu;
      }
    }
    uint32_t L[R];
#pragma unroll
    for (int e = 0; e < R; ++e) L[e] = 0xffffffffu;
    uint32_t tau = 0xffffffffu;
    select_chunk<R>(L, tau, c16, KK, t, lane);
    const int row = q0 + 16 * w + 4 * g + v;
    if (row < N) {
      int32_t* o = a.idx + ((size_t)b * N + row) * k;
#pragma unroll
      for (int e = 0; e < R; ++e) {
        const int el = t + 16 * e;
        if (el < KK && (el % dil) == 0) o[el / dil] = (int32_t)(L[e] & mask);
      }
    }
  }
}

template <int R, int KS, int NW>
const void* resident_fn_tiles(int KT) {
  switch (KT) {
    case 4: return (const void*)&knn_resident_kernel<R, KS, 4, NW>;
    case 8: return (const void*)&knn_resident_kernel<R, KS, 8, NW>;
    case 13: return (const void*)&knn_resident_kernel<R, KS, 13, NW>;
    default: return (const void*)&knn_resident_kernel<R, KS, 16, NW>;
  }
}

template <int R, int NW>
const void* resident_fn_steps(int KS, int KT) {
  switch (KS) {
    case 2: return resident_fn_tiles<R, 2, NW>(KT);
    case 3: return resident_fn_tiles<R, 3, NW>(KT);
    case 4: return resident_fn_tiles<R, 4, NW>(KT);
    default: return resident_fn_tiles<R, 5, NW>(KT);
  }
}

template <int NW>
const void* resident_fn(int R, int KS, int KT) {
  return R == 1 ? resident_fn_steps<1, NW>(KS, KT)
         : R == 2 ? resident_fn_steps<2, NW>(KS, KT) : resident_fn_steps<4, NW>(KS, KT);
}

// Eight waves (128 query rows) per workgroup when those workgroups fit the
// chip in one round, one per CU, as in the streamed build: each wave's work is
// the same, and the staged keys and their scales serve twice the rows.
int knn_resident_waves(int B, int N) { return (long long)B * ((N + 127) / 128) <= 256 ? 8 : 4; }

hipError_t launch_knn_resident(const KnnArgs& a, hipStream_t stream, hipEvent_t ev0, hipEvent_t ev1) {
  const int R = knn_list_regs(a.KK), KS = (a.C + 31) / 32, KT = knn_resident_tiles(a.M);
  const int NW = knn_resident_waves(a.B, a.N), rows = 16 * NW;
  const void* fn = NW == 8 ? resident_fn<8>(R, KS, KT) : resident_fn<4>(R, KS, KT);
  const size_t smem = KT == 4 ? resident_smem<4>(a.C) : KT == 8 ? resident_smem<8>(a.C)
                      : KT == 13 ? resident_smem<13>(a.C) : resident_smem<16>(a.C);
  const dim3 grid(a.B * ((a.N + rows - 1) / rows)), block(64 * NW);
  return launch_with_smem(fn, grid, block, smem, stream, ev0, ev1, a);
}

}  // namespace gl
