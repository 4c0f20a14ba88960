// Dilated kNN graph build with keys streamed through LDS, for large key sets
// (Sec. II-B Eq. 4; Sec. IV-B; Alg. 2).
//
// One workgroup = NW waves (4 or 8) = 16 NW query rows of one image; wave w
// owns rows 16w .. 16w+15 and keeps their MFMA A operands (all contraction
// steps) and inverse norms in registers for the whole kernel.
//   1. Keys arrive in chunks of KC rows, loaded cooperatively (16-byte vectors,
//      fully coalesced) into registers while the previous chunk is used, then
//      stored to LDS; each key's distance scale factors are computed once per
//      chunk (two threads per key).
//   2. Four 16-key tiles at a time, the Gram tiles come from four independent
//      MFMA chains with B operands read from LDS.  The epilogue costs two operations per candidate,
//        d1s = qscale * ((1 + n_j) - 2 r_i r_j G_ij)
//      (the fixed-point distance of the in-register kernel, before the
//      floor), followed by a compare against the row's threshold: the
//      K'-th packed key's distance bucket plus one, so no candidate that
//      could enter the list is dropped.
//   3. Every row has a buffer of kStCap LDS slots.  The row's passing keys of
//      a tile are appended densely: a lane's place is the row's count plus
//      the passing lanes before it in its 16-lane group (a wave ballot); a
//      group of tiles in which no candidate of the wave passes skips the
//      packing and stores.  Chunks are visited outwards from the workgroup's
//      own place in the key set, which tightens the thresholds early on image
//      grids.  When some row's buffer could overflow in the next group of
//      tiles, and at the end, the wave merges its 16 rows' buffers into their
//      sorted register lists (ceil(count / 16) layers of 16 per row, 16 lanes
//      per row, the same bitonic merge as the in-register kernel), empties
//      them and refreshes the thresholds.
// Results are identical to the in-register kernel: the same packed keys are
// ranked, and the threshold only skips keys that cannot enter the list.
#include "knn_tile.h"

namespace gl {

constexpr int kStCap = 128;      // candidate slots per row
constexpr int kStSlots = kStCap / 16;  // layers of 16 in a full row buffer
constexpr int kStRowStride = kStCap + 2;  // words per row of slots (rows 4 apart change bank)
constexpr int kStGroup = 4;      // key tiles computed together (independent MFMA chains)
// Four-wave workgroups: narrow rows (<= 4 contraction steps) run two per CU;
// wider rows are register-bound to one, which then gets more LDS and a deeper
// prefetch.  Eight-wave workgroups run one per CU and take the LDS of one.
constexpr int kStWideKS = 12;
__host__ __device__ constexpr int st_max_vec(int KS) { return KS >= kStWideKS ? 20 : 10; }
__host__ __device__ constexpr int st_lds_budget(int KS, int NW) {
  return KS >= kStWideKS || NW == 8 ? 150 * 1024 : 80 * 1024;
}

struct StreamGeom {
  int KC, kstride;
  size_t keys, scales, cand, tau, total;
};

// LDS layout: key chunk (KC rows of kstride bytes), per-key scale pairs,
// candidate slots, per-row thresholds.  A key row holds the KS contraction
// steps the kernel runs (channels past C stay zero) plus 16 bytes that move
// consecutive rows to other banks.  KC is a multiple of 64 (whole groups of 4
// tiles), as large as the budget and the prefetch registers allow, at least
// 64 and at most 384 (the eight-wave narrow rows: 384 at C = 96, where each
// chunk boundary costs a barrier and a merge in every wave).
__host__ __device__ inline StreamGeom stream_geom(int C, int dt_bf16, int KS, int NW) {
  StreamGeom s;
  const int rowb = C * (dt_bf16 ? 2 : 4);
  const int rows = 16 * NW;
  s.kstride = KS * 64 + 16;  // a contraction step is 64 bytes in either type
  const int fixed = rows * kStRowStride * 4 + rows * 4;
  int kc = (st_lds_budget(KS, NW) - fixed) / (s.kstride + 8);
  const int kv = st_max_vec(KS) * 64 * NW * 16 / rowb;  // prefetchable rows
  kc = (kc < kv ? kc : kv) / 64 * 64;
  s.KC = kc > 384 ? 384 : kc < 64 ? 64 : kc;
  s.keys = 0;
  s.scales = s.keys + (size_t)s.KC * s.kstride;
  s.cand = s.scales + (size_t)s.KC * 8;
  s.tau = s.cand + (size_t)rows * kStRowStride * 4;
  s.total = s.tau + rows * 4;
  return s;
}

template <int DT, int MV, int NT>
__device__ __forceinline__ void st_load_chunk(u32x4 (&regs)[MV], const char* kb, int k0,
                                              int M, int C, int CG, int nvec, int e0, int tid) {
  constexpr int ES = DT ? 2 : 4;
  constexpr int VEC = 16 / ES;
#pragma unroll
  for (int i = 0; i < MV; ++i) {
    const int e = min(e0 + tid + i * NT, nvec - 1);
    const int r = e / CG, cg = e - r * CG;
    regs[i] = *reinterpret_cast<const u32x4*>(kb + ((size_t)min(k0 + r, M - 1) * C + cg * VEC) * ES);
  }
}

template <int MV, int NT>
__device__ __forceinline__ void st_store_chunk(const u32x4 (&regs)[MV], char* kbuf,
                                               int kstride, int CG, int nvec, int e0, int tid) {
#pragma unroll
  for (int i = 0; i < MV; ++i) {
    const int e = e0 + tid + i * NT;
    const int ec = min(e, nvec - 1);
    const int r = ec / CG, cg = ec - r * CG;
    if (e < nvec) *reinterpret_cast<u32x4*>(kbuf + r * kstride + cg * 16) = regs[i];
  }
}

// Distance scale factors of the keys of one chunk, two threads per key.  Norms
// are summed in the order of the in-register kernel (per 4-lane-group channel
// slice over the contraction steps, then (s0 + s1) + (s2 + s3)), so both
// kernels rank identical packed keys.
template <int DT, int KS, int NT>
__device__ __forceinline__ void st_chunk_scales(const char* kbuf, float2* ksc, int KC, int kstride,
                                                int k0, int M, int C, float qscale, int tid) {
  constexpr int ES = DT ? 2 : 4;
  constexpr int KSTEP = DT ? 32 : 16;
  const int half = tid & 1;
  for (int r0 = 0; r0 < KC; r0 += NT / 2) {
    const int r = r0 + (tid >> 1);
    const int rr = min(r, KC - 1);
    float sq[2] = {0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int c = s * KSTEP + (2 * half + q) * (KSTEP / 4);
        const uint4 v = *reinterpret_cast<const uint4*>(kbuf + rr * kstride + c * ES);
        sq[q] = DT ? sumsq_bf16x8(v, sq[q]) : sumsq_f32x4(v, sq[q]);
      }
      if (KS > 4 && (s & 3) == 3) __builtin_amdgcn_sched_barrier(0);
    }
    const float pair = sq[0] + sq[1];
    const float other = __shfl_xor(pair, 1);
    const float ss = half ? other + pair : pair + other;  // (s0 + s1) + (s2 + s3)
    const float m2rj = -2.f * key_rnorm(ss);
    const float base = ss > 0.f ? 2.f : 1.f;  // 1 + n_j
    if (half == 0 && r < KC)
      ksc[r] = k0 + r < M ? make_float2(m2rj * qscale, base * qscale) : make_float2(0.f, INFINITY);
  }
}

// Gram tiles t0 .. t0+3 of the chunk in LDS against the wave's 16 query rows.
template <int DT, int KS>
__device__ __forceinline__ void st_gram(f32x4 (&acc)[kStGroup], const uint4 (&af)[KS],
                                        const char* kbuf, int t0, int kstride, int C, int g, int t) {
  constexpr int ES = DT ? 2 : 4;
  constexpr int KSTEP = DT ? 32 : 16;
#pragma unroll
  for (int p = 0; p < kStGroup; ++p) acc[p] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int c = s * KSTEP + g * (KSTEP / 4);  // channels past C read the zero pad
    uint4 bv[kStGroup];
#pragma unroll
    for (int p = 0; p < kStGroup; ++p)
      bv[p] = *reinterpret_cast<const uint4*>(kbuf + ((t0 + p) * 16 + t) * kstride + c * ES);
#pragma unroll
    for (int p = 0; p < kStGroup; ++p) {
      if (DT) {
        acc[p] = mfma_bf16(af[s], bv[p], acc[p]);
      } else {
        const float4 x4 = __builtin_bit_cast(float4, af[s]);
        const float4 y4 = __builtin_bit_cast(float4, bv[p]);
        acc[p] = mfma_f32(x4.x, y4.x, acc[p]);
        acc[p] = mfma_f32(x4.y, y4.y, acc[p]);
        acc[p] = mfma_f32(x4.z, y4.z, acc[p]);
        acc[p] = mfma_f32(x4.w, y4.w, acc[p]);
      }
    }
    // long contractions: keep the scheduler from hoisting every step's B loads
    // (4 registers per tile and step) above the first MFMAs
    if (KS > 4 && (s & 3) == 3) __builtin_amdgcn_sched_barrier(0);
  }
}

// The same in two halves, for the narrow rows: the B operands of a group are
// requested (st_gram_load) one epilogue ahead of the MFMAs that use them
// (st_gram_mma), so no MFMA waits on its own LDS read.
template <int DT, int KS>
__device__ __forceinline__ void st_gram_load(uint4 (&bv)[KS][kStGroup], const char* kbuf, int t0,
                                             int kstride, int g, int t) {
  constexpr int ES = DT ? 2 : 4;
  constexpr int KSTEP = DT ? 32 : 16;
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int c = s * KSTEP + g * (KSTEP / 4);
#pragma unroll
    for (int p = 0; p < kStGroup; ++p)
      bv[s][p] = *reinterpret_cast<const uint4*>(kbuf + ((t0 + p) * 16 + t) * kstride + c * ES);
  }
}

template <int DT, int KS>
__device__ __forceinline__ void st_gram_mma(f32x4 (&acc)[kStGroup], const uint4 (&af)[KS],
                                            const uint4 (&bv)[KS][kStGroup]) {
#pragma unroll
  for (int p = 0; p < kStGroup; ++p) acc[p] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < KS; ++s)
#pragma unroll
    for (int p = 0; p < kStGroup; ++p) {
      if (DT) {
        acc[p] = mfma_bf16(af[s], bv[s][p], acc[p]);
      } else {
        const float4 x4 = __builtin_bit_cast(float4, af[s]);
        const float4 y4 = __builtin_bit_cast(float4, bv[s][p]);
        acc[p] = mfma_f32(x4.x, y4.x, acc[p]);
        acc[p] = mfma_f32(x4.y, y4.y, acc[p]);
        acc[p] = mfma_f32(x4.z, y4.z, acc[p]);
        acc[p] = mfma_f32(x4.w, y4.w, acc[p]);
      }
    }
}

// Merge the wave's buffered candidates of its 16 rows into their sorted lists,
// empty the buffers and refresh the filter thresholds.  L[p] holds row 4p + g
// (16 lanes per row); tS[v] and cnt[v] belong to row 4g + v.  Row r's buffer
// is cand[r * kStRowStride + i], i < its count, densely filled, so a row of n
// candidates is merged in ceil(n / 16) layers of 16.
template <int R>
__device__ __forceinline__ void st_flush(uint32_t (&L)[4][R], float (&tS)[4], int (&cnt)[4],
                                         uint32_t* cand, uint32_t* tauL, int KK, int ib, int lane,
                                         int g, int t) {
  // the counts travel to the lanes that merge the rows (row 4p + g is held by
  // group g's lanes in the lists, counted by group p's lanes)
  if (t == 0) {
#pragma unroll
    for (int v = 0; v < 4; ++v) tauL[4 * g + v] = (uint32_t)cnt[v];
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
  // The rows of two list registers at a time are merged together: their sorts
  // and merges are independent dependency chains, which the scheduler
  // interleaves (one chain alone leaves the VALU waiting on each step).
#pragma unroll
  for (int p0 = 0; p0 < 4; p0 += 2) {
    uint32_t tk[2];
    int n[2];
    const uint32_t* src[2];
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      const int row = 4 * (p0 + pp) + g;
      n[pp] = (int)tauL[row];
      tk[pp] = list_element<R>(L[p0 + pp], KK - 1, lane);
      src[pp] = cand + row * kStRowStride + t;
    }
    for (int m = 0; m < kStSlots; ++m) {
      if (!__any(16 * m < n[0] || 16 * m < n[1])) break;
      uint32_t c[2];
#pragma unroll
      for (int pp = 0; pp < 2; ++pp) {
        const uint32_t x = 16 * m + t < n[pp] ? src[pp][16 * m] : 0xffffffffu;
        c[pp] = x < tk[pp] ? x : 0xffffffffu;
      }
      // a layer with no key below its row's threshold changes nothing among
      // the list's first K' keys (keys are unique)
      if (!__any(c[0] != 0xffffffffu || c[1] != 0xffffffffu)) continue;
      const uint32_t c0 = sort16_lanes(c[0], t);
      const uint32_t c1 = sort16_lanes(c[1], t);
      merge16_into_list<R>(L[p0], c0, t);
      merge16_into_list<R>(L[p0 + 1], c1, t);
      tk[0] = list_element<R>(L[p0], KK - 1, lane);
      tk[1] = list_element<R>(L[p0 + 1], KK - 1, lane);
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
    if (t == 0) {
      tauL[4 * p0 + g] = tk[0];
      tauL[4 * (p0 + 1) + g] = tk[1];
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const uint32_t tk = tauL[4 * g + v];
    tS[v] = tk == 0xffffffffu ? INFINITY : (float)((tk >> ib) + 1u);
    cnt[v] = 0;
  }
}

// Narrow rows (KS <= 4) overlap the next group's Gram tiles with the current
// epilogue and are held to two waves per SIMD.  Medium rows need those
// registers for their A operands and run one group at a time.  Wide rows
// (KS >= kStWideKS) are at one wave per SIMD anyway and overlap again.
template <int DT, int R, int KS, int NW>
__device__ __forceinline__ void knn_stream_body(const KnnArgs& a, int KC, int kstride, char* smem) {
  constexpr int NT = 64 * NW, ROWS = 16 * NW;
  constexpr bool PIPE = KS <= 4 || KS >= kStWideKS;
  constexpr bool SPLIT = KS <= 4;  // B operands one epilogue ahead of their MFMAs
  constexpr int MV = st_max_vec(KS);
  constexpr int ES = DT ? 2 : 4;
  constexpr int VEC = 16 / ES;
  constexpr int KSTEP = DT ? 32 : 16;
  const int N = a.N, C = a.C, M = a.M, k = a.k, dil = a.dil, KK = a.KK, ib = a.ib;
  const float qscale = a.qscale;
  const float qmaxf = (float)a.qmax;
  const int ksteps = (C + KSTEP - 1) / KSTEP;
  const int nqb = (N + ROWS - 1) / ROWS;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int b = blk / nqb, q0 = (blk - b * nqb) * ROWS;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, t = lane & 15;

  const StreamGeom geo = stream_geom(C, DT, KS, NW);
  char* kbuf0 = smem + geo.keys;
  float2* ksc0 = reinterpret_cast<float2*>(smem + geo.scales);
  uint32_t* cand = reinterpret_cast<uint32_t*>(smem + geo.cand) + w * 16 * kStRowStride;
  uint32_t* tauL = reinterpret_cast<uint32_t*>(smem + geo.tau) + w * 16;

  const char* xb = static_cast<const char*>(a.x) + (size_t)b * N * C * ES;
  const char* kb = static_cast<const char*>(a.keys) + (size_t)b * M * C * ES;

  // -- query operands and inverse norms (rows q0 + 16w + t) ----------------------
  uint4 af[KS];
  float qss = 0.f;
  {
    const char* qg = xb + (size_t)min(q0 + 16 * w + t, N - 1) * C * ES;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int c = s * KSTEP + g * (KSTEP / 4);
      const bool in = s < ksteps && c < C;
      af[s] = *reinterpret_cast<const uint4*>(qg + (size_t)(in ? c : 0) * ES);
      if (!in) af[s] = make_uint4(0, 0, 0, 0);
      qss = DT ? sumsq_bf16x8(af[s], qss) : sumsq_f32x4(af[s], qss);
    }
  }
  qss += __shfl_xor(qss, 16);
  qss += __shfl_xor(qss, 32);
  float qr[4];
  {
    const float rq = 1.f / fmaxf(sqrtf(qss), 1e-12f);
#pragma unroll
    for (int v = 0; v < 4; ++v) qr[v] = __shfl(rq, 4 * g + v);
  }

  // -- key chunks ---------------------------------------------------------------------
  const int CG = C / VEC;
  const int nvec = KC * CG;
  u32x4 regs[MV];

  // -- selection state ------------------------------------------------------------
  // L[p]: sorted list of row 4p + g (element e = t + 16*a);  tS[v]: filter
  // threshold of row 4g + v;  cnt[v]: candidates buffered for that row, at
  // cand[(4g + v) * kStRowStride + i], i < cnt[v] (the same in the row's 16
  // lanes).
  uint32_t L[4][R];
#pragma unroll
  for (int p = 0; p < 4; ++p)
#pragma unroll
    for (int q = 0; q < R; ++q) L[p][q] = 0xffffffffu;
  float tS[4] = {INFINITY, INFINITY, INFINITY, INFINITY};
  int cnt[4] = {0, 0, 0, 0};
  uint32_t* myRows = cand + 4 * g * kStRowStride;
  const uint32_t below = (1u << t) - 1u;  // lanes of this lane's 16-lane group before it

  // -- zero pad of the key rows (channels C .. 32 KS); chunk stores leave it alone ----
  {
    const int padv = (kstride - 16 - C * ES) / 16;
    for (int i = tid; i < KC * padv; i += NT) {
      const int r = i / padv;
      *reinterpret_cast<u32x4*>(kbuf0 + r * kstride + C * ES + (i - r * padv) * 16) = u32x4{0, 0, 0, 0};
    }
  }

  // -- main loop --------------------------------------------------------------------
  // One LDS key buffer; the next chunk waits in registers while this one is used.
  char* kbuf = kbuf0;
  const int nchunks = (M + KC - 1) / KC;
  // The chunks are visited outwards from the chunk at the workgroup's own
  // position in the key set (its first query row scaled by M / N): ch0,
  // ch0 + 1, ch0 - 1, ch0 + 2, ... (mod nchunks, each chunk once).  The
  // selected lists do not depend on the order; on image grids a node's
  // nearest keys tend to lie near it, above as well as below in row-major
  // order, so the thresholds tighten within the first few chunks and fewer
  // candidates pass the filter.
  const int ch0 = (int)(((long long)q0 * M / N) / KC);
  auto chunk_at = [&](int c) {
    const int off = (c & 1) ? (c + 1) >> 1 : -(c >> 1);
    const int ch = (ch0 + off) % nchunks;
    return ch < 0 ? ch + nchunks : ch;
  };
  // A chunk of at most MV vectors per thread is prefetched into registers
  // while the previous one is used; larger chunks are copied piecewise when
  // their turn comes.
  // The first chunk is loaded inside the loop too: with its loads issued
  // ahead of the loop, the compiler's wait bookkeeping at the loop head keeps
  // treating their registers as pending and makes every chunk wait for the
  // next chunk's prefetch.
  const bool prefetch = nvec <= MV * NT;
  for (int c = 0; c < nchunks; ++c) {
    const int ch = chunk_at(c);
    const int chn = chunk_at(c + 1 < nchunks ? c + 1 : c);
    const int k0 = ch * KC;
    const int ntl = (min(KC, M - k0) + 15) >> 4;
    if (prefetch) {
      if (c == 0) st_load_chunk<DT, MV, NT>(regs, kb, k0, M, C, CG, nvec, 0, tid);
      st_store_chunk<MV, NT>(regs, kbuf, kstride, CG, nvec, 0, tid);
    } else {
      for (int e0 = 0; e0 < nvec; e0 += MV * NT) {
        st_load_chunk<DT, MV, NT>(regs, kb, k0, M, C, CG, nvec, e0, tid);
        st_store_chunk<MV, NT>(regs, kbuf, kstride, CG, nvec, e0, tid);
      }
    }
    __syncthreads();
    st_chunk_scales<DT, KS, NT>(kbuf, ksc0, KC, kstride, k0, M, C, qscale, tid);
    __syncthreads();
    if (prefetch && c + 1 < nchunks)
      st_load_chunk<DT, MV, NT>(regs, kb, chn * KC, M, C, CG, nvec, 0, tid);
    // Gram tiles of group t0 + 4 are issued before the epilogue of group t0
    // (independent MFMA chains run while the VALU filters).  All KC rows of the
    // key buffer hold finite values (the chunk loader repeats the last key),
    // and the scales of rows past the key set make their distance +inf, so
    // tiles and keys past the end need no test.  Contraction steps past C
    // multiply a zero A operand.
    f32x4 acc[kStGroup];
    uint4 bv[SPLIT ? KS : 1][kStGroup];
    if constexpr (SPLIT) {
      st_gram_load<DT, KS>(bv, kbuf, 0, kstride, g, t);
      st_gram_mma<DT, KS>(acc, af, bv);
    } else if (PIPE) {
      st_gram<DT, KS>(acc, af, kbuf, 0, kstride, C, g, t);
    }
    for (int t0 = 0; t0 < ntl; t0 += kStGroup) {
      // a group adds at most 16 * kStGroup candidates to a row; a row whose
      // list is not full yet is merged as soon as it holds K' candidates
      // (its threshold then drops from infinity)
      bool full = false;
#pragma unroll
      for (int v = 0; v < 4; ++v)
        full |= cnt[v] > kStCap - 16 * kStGroup || (cnt[v] >= KK && tS[v] == INFINITY);
      if (__any(full)) st_flush<R>(L, tS, cnt, cand, tauL, KK, ib, lane, g, t);
      const bool more = t0 + kStGroup < ntl;
      // this group's key scales, read ahead of the next group's B operands
      // (LDS reads return in order)
      float2 sc[kStGroup];
#pragma unroll
      for (int p = 0; p < kStGroup; ++p) sc[p] = ksc0[(t0 + p) * 16 + t];
      f32x4 nxt[kStGroup];
      if constexpr (SPLIT) {
        // unconditional (the last group re-reads group 0): a branch here
        // would make every later LDS wait assume these reads are in flight
        st_gram_load<DT, KS>(bv, kbuf, more ? t0 + kStGroup : 0, kstride, g, t);
      } else if (PIPE) {
        if (more) st_gram<DT, KS>(nxt, af, kbuf, t0 + kStGroup, kstride, C, g, t);
      } else {
        st_gram<DT, KS>(acc, af, kbuf, t0, kstride, C, g, t);
      }
      // The common path per candidate is the distance and one compare; the
      // packing and the store run only for the candidates that pass, and not
      // at all in a group where no lane of the wave has one.  A row's passing
      // candidates of one tile go to consecutive places of its buffer: a
      // lane's place is the row's count plus the passing lanes before it in
      // its 16-lane group (from the wave's ballot).
      float dd[kStGroup][4];
#pragma unroll
      for (int p = 0; p < kStGroup; ++p)
#pragma unroll
        for (int v = 0; v < 4; ++v) dd[p][v] = fmaf(acc[p][v] * sc[p].x, qr[v], sc[p].y);
      // does any candidate pass: one compare per row, on its group minimum
      float dmin[4];
#pragma unroll
      for (int v = 0; v < 4; ++v)
        dmin[v] = fminf(fminf(dd[0][v], dd[1][v]), fminf(dd[2][v], dd[3][v]));
      const bool anyp = (dmin[0] < tS[0]) | (dmin[1] < tS[1]) | (dmin[2] < tS[2]) | (dmin[3] < tS[3]);
      if (__any(anyp)) {
#pragma unroll
        for (int p = 0; p < kStGroup; ++p) {
          const uint32_t j = (uint32_t)(k0 + (t0 + p) * 16 + t);
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const bool ps = dd[p][v] < tS[v];
            const uint32_t gm = (uint32_t)(__ballot(ps) >> (16 * g)) & 0xffffu;
            if (ps) {
              const uint32_t q = (uint32_t)__builtin_amdgcn_fmed3f(dd[p][v], 0.f, qmaxf);
              myRows[v * kStRowStride + cnt[v] + __popc(gm & below)] = (q << ib) | j;
            }
            cnt[v] += __popc(gm);
          }
        }
      }
      if constexpr (SPLIT) {
        if (more) st_gram_mma<DT, KS>(acc, af, bv);
      } else if (PIPE) {
#pragma unroll
        for (int p = 0; p < kStGroup; ++p) acc[p] = nxt[p];
      }
    }
    // Every wave merges what it buffered in this chunk before the barrier: the
    // waves wait for each other there anyway, so merges at the same place in
    // every wave overlap instead of adding up, and the next chunk is filtered
    // with fresh thresholds.
    bool any = false;
#pragma unroll
    for (int v = 0; v < 4; ++v) any |= cnt[v] > 0;
    if (__any(any)) st_flush<R>(L, tS, cnt, cand, tauL, KK, ib, lane, g, t);
    __syncthreads();  // every wave is done with this chunk before it is overwritten
  }

  // -- dilation and output ------------------------------------------------------------
  const uint32_t mask = (1u << ib) - 1u;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int row = q0 + 16 * w + 4 * p + g;
    if (row < N) {
      int32_t* o = a.idx + ((size_t)b * N + row) * k;
#pragma unroll
      for (int q = 0; q < R; ++q) {
        const int e = t + 16 * q;
        if (e < KK && (e % dil) == 0) o[e / dil] = (int32_t)(L[p][q] & mask);
      }
    }
  }
}

template <int DT, int R, int KS, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2, 8))) void knn_stream_kernel_narrow(KnnArgs a, int KC, int kstride) {
  extern __shared__ __align__(16) char smem[];
  knn_stream_body<DT, R, KS, NW>(a, KC, kstride, smem);
}

template <int DT, int R, int KS, int NW>
__global__ __launch_bounds__(64 * NW) void knn_stream_kernel(KnnArgs a, int KC, int kstride) {
  extern __shared__ __align__(16) char smem[];
  knn_stream_body<DT, R, KS, NW>(a, KC, kstride, smem);
}

// Contraction steps compiled into the kernel: the next bucket at or above
// ceil(C / step); steps past C run on a zero A operand.
int knn_stream_ks(int C, int dt_bf16) {
  const int KSTEP = dt_bf16 ? 32 : 16;
  const int ks = (C + KSTEP - 1) / KSTEP;
  for (int b : {2, 3, 4, 6, 8, 12, 16, 20, 24})
    if (ks <= b) return b;
  return 0;
}

// Large key sets.  (For many query rows against a small key set, e.g. 3136
// rows x 196 pooled keys, the in-register kernel measured faster.)
bool knn_use_stream(int M, int C, int dt_bf16) {
  return M > 256 && knn_stream_ks(C, dt_bf16) > 0;
}

// Eight-wave workgroups hold two waves per SIMD, whose 256 registers the
// register-bound wide rows (12 or more steps) exceed: those run four waves.
template <int DT, int R, int NW>
const void* stream_fn_ks(int KS) {
  switch (KS) {
    case 2: return (const void*)&knn_stream_kernel_narrow<DT, R, 2, NW>;
    case 3: return (const void*)&knn_stream_kernel_narrow<DT, R, 3, NW>;
    case 4: return (const void*)&knn_stream_kernel_narrow<DT, R, 4, NW>;
    case 6: return (const void*)&knn_stream_kernel<DT, R, 6, NW>;
    case 8: return (const void*)&knn_stream_kernel<DT, R, 8, NW>;
  }
  if constexpr (NW == 4) {
    switch (KS) {
      case 12: return (const void*)&knn_stream_kernel<DT, R, 12, 4>;
      case 16: return (const void*)&knn_stream_kernel<DT, R, 16, 4>;
      case 20: return (const void*)&knn_stream_kernel<DT, R, 20, 4>;
      default: return (const void*)&knn_stream_kernel<DT, R, 24, 4>;
    }
  }
  return nullptr;
}

template <int NW>
const void* stream_fn(int dt_bf16, int R, int KS) {
  if (dt_bf16)
    return R == 1 ? stream_fn_ks<1, 1, NW>(KS)
           : R == 2 ? stream_fn_ks<1, 2, NW>(KS) : stream_fn_ks<1, 4, NW>(KS);
  return R == 1 ? stream_fn_ks<0, 1, NW>(KS)
         : R == 2 ? stream_fn_ks<0, 2, NW>(KS) : stream_fn_ks<0, 4, NW>(KS);
}

// Eight waves (128 query rows) per workgroup when those workgroups fit the
// chip in one round, one per CU: each wave still sweeps every key, so a
// workgroup's life is set by one wave's sweep, and the keys staged per chunk
// serve twice the rows.  Measured on MI355X: the 448 x 448 ViG-Ti build
// (B = 32, N = M = 784, C = 192) 76.8 -> 61.2 us, the high-resolution one
// (B = 8, N = M = 3136, C = 96) 146.2 -> 137.7 us; graphs identical.
int knn_stream_waves(int B, int N, int KS) {
  return KS <= 8 && (long long)B * ((N + 127) / 128) <= 256 ? 8 : 4;
}

hipError_t launch_knn_stream(const KnnArgs& a, int dt_bf16, hipStream_t stream, hipEvent_t ev0,
                             hipEvent_t ev1) {
  const int KS = knn_stream_ks(a.C, dt_bf16);
  const int NW = knn_stream_waves(a.B, a.N, KS), rows = 16 * NW;
  const StreamGeom geo = stream_geom(a.C, dt_bf16, KS, NW);
  const int R = knn_list_regs(a.KK);
  const void* fn = NW == 8 ? stream_fn<8>(dt_bf16, R, KS) : stream_fn<4>(dt_bf16, R, KS);
  const dim3 grid(a.B * ((a.N + rows - 1) / rows)), block(64 * NW);
  if (KS == 0 || !fn || geo.total > 160 * 1024) return hipErrorInvalidValue;
  struct {
    KnnArgs a;
    int KC, kstride;
  } args{a, geo.KC, geo.kstride};
  void* argv[] = {&args.a, &args.KC, &args.kstride};
  if (geo.total > 65536) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)geo.total);
    if (e != hipSuccess) return e;
  }
  if (ev0 || ev1) return hipExtLaunchKernel(fn, grid, block, argv, geo.total, stream, ev0, ev1, 0);
  return hipLaunchKernel(fn, grid, block, argv, geo.total, stream);
}

}  // namespace gl
