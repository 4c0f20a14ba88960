// Tiled MFMA GEMM for the fully connected layers of the path:
//   out[R, Cout] = act_out(act_in(A)[R, K] W[Cout, K]^T + b) + residual
//   * the MRConv update over materialised [x | m] rows for wide channels
//     (Sec. II-A Eq. 3; the W_x / W_m split of Sec. IV-C2 is the two halves of
//     the contraction axis), where the fused MRConv tile would stream all of W
//     through every 16- or 32-node workgroup;
//   * FC1, FC2 + residual and the FFN of the full ViG block (Eq. 11, 14, 15):
//     act_out = GELU gives the FFN's hidden layer (and, on the wide MRConv
//     update, the full block's sigma(U~)), residual the two skip connections;
//     act_in = GELU is gl_linear's GELU on A.
// A workgroup owns a 64 x 64 or 128 x 128 output tile, so W is read once per
// 64 or 128 rows and A once per 64 or 128 output channels.
//   - 4 waves in a 2 x 2 layout, or 8 in a 4 x 2 layout; each wave holds its
//     block of the tile (2 x 2 ... 2 x 4 MFMA tiles of 16 x 16) in registers.
//   - The contraction runs in stages of 256 bytes per row on the 64 x 64
//     tiles (4 MFMA k-steps: 128 bf16 or 64 fp32 channels) and of 128 bytes
//     on the 128 x 128 tiles.  Both operands are K-contiguous, so one 16-byte
//     vector per lane is exactly an MFMA operand slice.  A stage's A and B
//     tiles pass through LDS, double-buffered, with one barrier per stage.
//     The global loads of stage s+1 are in flight while stage s is multiplied;
//     the 128 x 128 tiles keep three staging register sets, so their loads
//     are issued two stages ahead.
//   - act_in is applied to A's elements as they are staged (fp32, rounded back
//     to the storage type, as if the caller had stored sigma(A)).
//   - Epilogue in fp32: + bias, act_out, + residual, rounded once.
#include "gl_device.h"
#include "gl_kernels.h"

namespace gl {

constexpr int kGm128Waves = 8;  // waves of the 128 x 128 configuration

// Tile configurations: BM x BM output tiles, STEP bytes of K per row per stage.
//   64 x 64, 192 B: contractions of at most 192 bytes per row, one stage;
//   64 x 64, 256 B: short contractions or few tiles (the ViG block's layers);
//   128 x 128, 128 B: large GEMMs (e.g. the ViG-B update), where W and A are
//   re-read half as often.
// NW waves: 4 in a 2 x 2 layout (wave tile BM/2 x BM/2), or 8 in a 4 x 2
// layout (BM/4 x BM/2), which keeps twice as many waves in flight per CU for
// the same LDS.
template <int BM, int STEP, int NW = 4>
struct GemmCfg {
  static constexpr int kThreads = 64 * NW;
  static constexpr int kRow = STEP + 16;                 // LDS row stride
  static constexpr int kTile = BM * kRow;                // one operand tile of one stage
  static constexpr int kVec = BM * STEP / 16 / kThreads; // 16-byte loads per thread, operand
  static constexpr int kWm = NW == 8 ? 4 : 2;            // waves along the rows
  static constexpr int kTpwM = BM / 16 / kWm;            // MFMA tiles per wave, rows
  static constexpr int kTpwN = BM / 32;                  // MFMA tiles per wave, columns
  // 192- and 384-byte steps are only used when the whole contraction is one
  // stage, so their tiles are not double-buffered
  static constexpr size_t kSmem = (size_t)(STEP == 384 || STEP == 192 ? 2 : 4) * kTile;
};

size_t gemm_smem_bytes() { return GemmCfg<128, 128>::kSmem; }

// GELU of the 16-byte vector's elements, rounded back to the storage type.
template <int DT>
__device__ __forceinline__ u32x4 gelu_vec(u32x4 v) {
  if (DT) {
    float f[8];
    unpack_bf16x8(__builtin_bit_cast(uint4, v), f);
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = gelu_f32(f[i]);
    return __builtin_bit_cast(u32x4, pack_bf16x8(f));
  }
  float4 f = __builtin_bit_cast(float4, v);
  f.x = gelu_f32(f.x);
  f.y = gelu_f32(f.y);
  f.z = gelu_f32(f.z);
  f.w = gelu_f32(f.w);
  return __builtin_bit_cast(u32x4, f);
}

template <int DT, int ACT_IN, int ACT_OUT, int BM, int STEP, int NW = 4>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(BM == 128 ? 4 : 1, 8))) void gemm_nt_kernel(GemmArgs a) {
  extern __shared__ __align__(16) char smem[];
  using G = GemmCfg<BM, STEP, NW>;
  constexpr int kGmBM = BM, kGmBN = BM, kGmStep = STEP, kGmRow = G::kRow, kGmTile = G::kTile;
  constexpr int kGmVec = G::kVec, TPWM = G::kTpwM, TPWN = G::kTpwN, SPR = STEP / 16;
  constexpr int kGmThreads = G::kThreads;
  const int R = a.R, K = a.K, Cout = a.Cout;
  const int rowb = K * (DT ? 2 : 4);        // a multiple of 16
  const int nstages = (rowb + kGmStep - 1) / kGmStep;
  const int ntn = (Cout + kGmBN - 1) / kGmBN;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = blk / ntn, nt = blk - mt * ntn;
  const int m0 = mt * kGmBM, n0 = nt * kGmBN;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, t = lane & 15;
  const int wm = w >> 1, wn = w & 1;       // the wave's block: 16 TPWM rows, 16 TPWN columns

  // staging: vector v = tid + 256 i of a tile is row v / SPR, 16-byte slot v % SPR
  const char* Ab = static_cast<const char*>(a.A);
  const char* Wb = static_cast<const char*>(a.W);
  const char* ag[kGmVec];
  const char* bg[kGmVec];
  int slot[kGmVec], lo[kGmVec];
#pragma unroll
  for (int i = 0; i < kGmVec; ++i) {
    const int v = tid + kGmThreads * i, r = v / SPR;
    slot[i] = (v % SPR) * 16;
    ag[i] = Ab + (size_t)min(m0 + r, R - 1) * rowb + slot[i];
    bg[i] = Wb + (size_t)min(n0 + r, Cout - 1) * rowb + slot[i];
    lo[i] = r * kGmRow + slot[i];
  }
  // staging register sets: one for the 64 x 64 tiles (the next stage is in
  // flight while one is multiplied), three for the 128 x 128 tiles (two stages
  // ahead: their long contractions are otherwise bound by the latency of each
  // stage's global loads).  A GELU on A (act_in) keeps one: its staging is
  // VALU work that measured slower with the deeper pipeline.
  constexpr int NSET = BM == 128 && !ACT_IN ? 3 : 1;
  u32x4 ra[NSET][kGmVec], rb[NSET][kGmVec];
  // Slots past the contraction load column 0 and are zeroed when they are
  // stored, not when they arrive: touching a loaded register right after its
  // load makes the wave wait for it there.
  auto gload = [&](int q, int s) {
#pragma unroll
    for (int i = 0; i < kGmVec; ++i) {
      const int off = s * kGmStep + slot[i] < rowb ? s * kGmStep : 0;
      ra[q][i] = *reinterpret_cast<const u32x4*>(ag[i] + off);
      rb[q][i] = *reinterpret_cast<const u32x4*>(bg[i] + off);
    }
  };
  auto sstore = [&](int q, int buf, int s) {
    char* sa = smem + buf * 2 * kGmTile;
#pragma unroll
    for (int i = 0; i < kGmVec; ++i) {
      // an empty asm that uses the loaded registers pins their first use here:
      // otherwise the scheduler hoists the zeroing selects (whose condition is
      // known early) to just after the loads, and the wave waits for loads
      // meant to stay in flight for two more stages
      asm volatile("" : "+v"(ra[q][i]), "+v"(rb[q][i]));
      const bool in = s * kGmStep + slot[i] < rowb;
      const u32x4 va = in ? ra[q][i] : u32x4{0, 0, 0, 0};
      const u32x4 vb = in ? rb[q][i] : u32x4{0, 0, 0, 0};
      *reinterpret_cast<u32x4*>(sa + lo[i]) = ACT_IN ? gelu_vec<DT>(va) : va;
      *reinterpret_cast<u32x4*>(sa + kGmTile + lo[i]) = vb;
    }
  };

  f32x4 acc[TPWM][TPWN];
#pragma unroll
  for (int i = 0; i < TPWM; ++i)
#pragma unroll
    for (int j = 0; j < TPWN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // The residual does not depend on the product.  In the 64 x 64 tiles (short,
  // latency-bound contractions) its elements are requested here, so they
  // arrive during the contraction rather than after it; the 128 x 128 tiles
  // load it in the epilogue (its registers would cost them a wave per SIMD).
  // When the residual is `out` itself, each element is still read before
  // this thread writes it, and the tiles of other workgroups are disjoint.
  constexpr bool kResEarly = BM == 64;
  float res[TPWN][TPWM][4];
  if (kResEarly && a.residual) {
#pragma unroll
    for (int j = 0; j < TPWN; ++j) {
      const int n = min(n0 + wn * 16 * TPWN + j * 16 + t, Cout - 1);
#pragma unroll
      for (int i = 0; i < TPWM; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const size_t o = (size_t)min(m0 + wm * 16 * TPWM + i * 16 + 4 * g + v, R - 1) * Cout + n;
          res[j][i][v] = DT ? bf16_bits_to_f32(static_cast<const uint16_t*>(a.residual)[o])
                            : static_cast<const float*>(a.residual)[o];
        }
    }
  }

  auto multiply = [&](int s) {
    const char* sa = smem + (s & 1) * 2 * kGmTile;
#pragma unroll
    for (int kk = 0; kk < kGmStep / 64; ++kk) {
      uint4 af[TPWM], bf[TPWN];
#pragma unroll
      for (int i = 0; i < TPWM; ++i)
        af[i] = *reinterpret_cast<const uint4*>(sa + (wm * 16 * TPWM + i * 16 + t) * kGmRow +
                                                kk * 64 + g * 16);
#pragma unroll
      for (int j = 0; j < TPWN; ++j)
        bf[j] = *reinterpret_cast<const uint4*>(sa + kGmTile + (wn * 16 * TPWN + j * 16 + t) * kGmRow +
                                                kk * 64 + g * 16);
#pragma unroll
      for (int i = 0; i < TPWM; ++i)
#pragma unroll
        for (int j = 0; j < TPWN; ++j) {
          if (DT) {
            acc[i][j] = mfma_bf16(af[i], bf[j], acc[i][j]);
          } else {
            const float4 x4 = __builtin_bit_cast(float4, af[i]);
            const float4 y4 = __builtin_bit_cast(float4, bf[j]);
            acc[i][j] = mfma_f32(x4.x, y4.x, acc[i][j]);
            acc[i][j] = mfma_f32(x4.y, y4.y, acc[i][j]);
            acc[i][j] = mfma_f32(x4.z, y4.z, acc[i][j]);
            acc[i][j] = mfma_f32(x4.w, y4.w, acc[i][j]);
          }
        }
    }
  };

  if constexpr (NSET == 3) {
    // Stage s is multiplied out of LDS buffer s & 1 while stage s+1 waits in
    // register set (s+1) % 3 and stage s+2 is on its way into set (s+2) % 3;
    // set s % 3, stored to LDS one iteration earlier, then takes stage s+3.
    // The loop runs whole groups of three stages, so each register set keeps
    // its role and no load's wait is merged with another's: stages past the
    // contraction (at most two) load in-range addresses, are stored as zeros
    // and are not multiplied.
    gload(0, 0);
    gload(1, 1);
    gload(2, 2);
    sstore(0, 0, 0);
    __syncthreads();
    for (int s0 = 0; s0 < nstages; s0 += 3) {
#pragma unroll
      for (int u = 0; u < 3; ++u) {
        const int s = s0 + u;
        if (s < nstages) multiply(s);
        sstore((u + 1) % 3, (s + 1) & 1, s + 1);
        gload(u, s + 3);
        __syncthreads();
      }
    }
  } else {
    gload(0, 0);
    sstore(0, 0, 0);
    __syncthreads();
    for (int s = 0; s < nstages; ++s) {
      if (s + 1 < nstages) gload(0, s + 1);
      multiply(s);
      if (s + 1 < nstages) sstore(0, (s + 1) & 1, s + 1);
      __syncthreads();
    }
  }

  // -- epilogue: lane (g, t) of tile (i, j) holds rows 4g..4g+3, column t --------
#pragma unroll
  for (int j = 0; j < TPWN; ++j) {
    const int n = n0 + wn * 16 * TPWN + j * 16 + t;
    if (n >= Cout) continue;
    float bn = 0.f;
    if (a.bias) {
      bn = DT ? bf16_bits_to_f32(static_cast<const uint16_t*>(a.bias)[n])
              : static_cast<const float*>(a.bias)[n];
    }
#pragma unroll
    for (int i = 0; i < TPWM; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = m0 + wm * 16 * TPWM + i * 16 + 4 * g + v;
        if (row >= R) continue;
        float y = acc[i][j][v] + bn;
        if (ACT_OUT) y = gelu_f32(y);
        const size_t o = (size_t)row * Cout + n;
        if (a.residual) {
          if (kResEarly) y += res[j][i][v];
          else y += DT ? bf16_bits_to_f32(static_cast<const uint16_t*>(a.residual)[o])
                       : static_cast<const float*>(a.residual)[o];
        }
        if (DT) static_cast<uint16_t*>(a.out)[o] = (uint16_t)f32_to_bf16_bits(y);
        else static_cast<float*>(a.out)[o] = y;
      }
  }
}

template <int BM, int STEP, int NW = 4>
const void* gemm_fn(int v) {
  static const void* const fns[8] = {
      (const void*)&gemm_nt_kernel<0, 0, 0, BM, STEP, NW>, (const void*)&gemm_nt_kernel<0, 0, 1, BM, STEP, NW>,
      (const void*)&gemm_nt_kernel<0, 1, 0, BM, STEP, NW>, (const void*)&gemm_nt_kernel<0, 1, 1, BM, STEP, NW>,
      (const void*)&gemm_nt_kernel<1, 0, 0, BM, STEP, NW>, (const void*)&gemm_nt_kernel<1, 0, 1, BM, STEP, NW>,
      (const void*)&gemm_nt_kernel<1, 1, 0, BM, STEP, NW>, (const void*)&gemm_nt_kernel<1, 1, 1, BM, STEP, NW>};
  return fns[v];
}

hipError_t launch_gemm_nt(const GemmArgs& a, int dt_bf16, hipStream_t stream, hipEvent_t ev0,
                          hipEvent_t ev1) {
  const int v = (dt_bf16 ? 4 : 0) + (a.act_in ? 2 : 0) + (a.act_out ? 1 : 0);
  const size_t rowb = (size_t)a.K * (dt_bf16 ? 2 : 4);
  // large tiles once they alone give every CU a tile and K is long
  const long tiles128 = (long)((a.R + 127) / 128) * ((a.Cout + 127) / 128);
  if (tiles128 >= 256 && rowb >= 1024) {
    constexpr int NW = kGm128Waves;
    const dim3 grid((unsigned)tiles128), block(64 * NW);
    return launch_with_smem(gemm_fn<128, 128, NW>(v), grid, block, GemmCfg<128, 128, NW>::kSmem,
                            stream, ev0, ev1, a);
  }
  const dim3 grid((unsigned)(((a.R + 63) / 64) * ((a.Cout + 63) / 64)));
  const long tiles64 = (long)grid.x;
  // a one-stage contraction never touches the second LDS buffer: half the
  // LDS, twice the workgroups per CU (K = 80 at the first pyramid stage)
  const bool one = rowb <= 256;
  if (rowb <= 192)
    return launch_with_smem(gemm_fn<64, 192, 4>(v), grid, dim3(256), GemmCfg<64, 192, 4>::kSmem,
                            stream, ev0, ev1, a);
  // rows of 257..384 bytes (K = 129..192 in bf16): one stage, one round trip;
  // 4 waves (measured faster than 8 here, GELU layers included)
  if (rowb > 256 && rowb <= 384)
    return launch_with_smem(gemm_fn<64, 384, 4>(v), grid, dim3(256), GemmCfg<64, 384, 4>::kSmem,
                            stream, ev0, ev1, a);
  // with a GELU on either side the 64 x 64 tile is VALU-heavy, and 8 waves
  // overlap it better; so do small grids (at most 512 tiles, about two per
  // CU), which 8 waves per tile fill better; larger plain products are as
  // fast or faster with 4
  if (a.act_in || a.act_out || tiles64 <= 512)
    return launch_with_smem(gemm_fn<64, 256, 8>(v), grid, dim3(512),
                            GemmCfg<64, 256, 8>::kSmem / (one ? 2 : 1), stream, ev0, ev1, a);
  return launch_with_smem(gemm_fn<64, 256, 4>(v), grid, dim3(256),
                          GemmCfg<64, 256, 4>::kSmem / (one ? 2 : 1), stream, ev0, ev1, a);
}

}  // namespace gl
