// fp32 GEMM with 128 x 128 workgroup tiles and K-tiles of 32, for a K- or
// M-contiguous A and an N- or K-contiguous B.  MFMA 32x32x2 f32 (lane l:
// A[l%32][l/32], B[l/32][l%32]; accumulator v of lane l holds
// C[8(v/4) + 4(l/32) + v%4][l%32]).
//
// W = 8 wavefronts of 64 x 32 (2 x 1 blocks of 32 x 32; 32 MFMAs of 64
// cycles per wavefront and K-tile: two wavefronts per SIMD within one
// workgroup) or W = 16 of 32 x 32 (four per SIMD, for outputs with about
// one tile per CU); one barrier per K-tile.  Two LDS stages
// of 32 KiB; the operands of K-tile t+2 are loaded into registers (16 bytes
// per load) while tile t is multiplied and are written to LDS once tile t+1
// is in place, so a load has a whole K-tile of MFMAs to land.  Two
// workgroups share a CU where the output has tiles for it; where it has
// few (a 4096 x 1024 product has 256), the sixteen-wavefront form gives
// each SIMD four wavefronts to issue from while one waits.
//
// Each operand is staged in its HBM orientation:
//  * K-contiguous (A [m][k], B [n][k]): rows of 32 floats (8 chunks of 16
//    bytes) per m or n; row r keeps logical chunk c at c ^ ((r >> 1) & 7),
//    so that an MFMA operand read (32 rows at one k) touches each bank at
//    most twice;
//  * M- or N-contiguous (A [k][m], B [k][n]): rows of 128 floats per k;
//    row k keeps chunk c at c ^ 8 (k % 2), so that the two k of one read
//    fall on disjoint banks.
// Load q (0 .. 16/W - 1) of wavefront w carries the 1 KiB block W q + w of a stage,
// lane l its 16 bytes at l * 16, so the LDS writes are contiguous and the
// swizzle is applied by choosing which chunk each lane fetches.
#include "gemm_common.h"
#include "launch.h"

namespace fluid {

namespace {

constexpr int FR_T = 128;                   // tile rows = tile columns
constexpr int FR_BK = 32;                   // K per stage
constexpr int FR_STAGE = FR_T * FR_BK * 4;  // bytes per operand and stage (16 KiB)

__device__ __forceinline__ int krow_swz(int r) { return (r >> 1) & 7; }
__device__ __forceinline__ int mnrow_swz(int k) { return (k & 1) << 3; }

}  // namespace

template <int W, bool AK, bool BK, bool RES>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(W / 4, W == 16 ? 4 : W / 2))) void gemm_f32_ring_kernel(GemmParams p) {
  constexpr int NQ = 16 / W;            // 1 KiB blocks per operand, stage and wavefront
  constexpr int WM = W == 16 ? 4 : 2;   // wavefronts along M
  constexpr int WN = W / WM;            // wavefronts along N
  constexpr int IM = 128 / WM / 32;     // 32-row MFMA blocks per wavefront along M
  constexpr int JN = 128 / WN / 32;     // 32-wide MFMA blocks per wavefront along N
  __shared__ __attribute__((aligned(1024))) uint8_t As[2][FR_STAGE];
  __shared__ __attribute__((aligned(1024))) uint8_t Bs[2][FR_STAGE];
  const TileCoord tc = tile_coord(p, FR_T, FR_T);
  // causal attention: a tile entirely above the diagonal is never read; a
  // row block's A is zero past its last row, so K stops there
  if ((p.causal & 1u) && tc.n0 > tc.m0 + FR_T - 1) return;
  const uint32_t kend = (p.causal & 2u) ? min(p.K, tc.m0 + FR_T) : p.K;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int lr = lane & 31, lh = lane >> 5;
  const Rsrc ra = make_rsrc(p.A, p.a_bytes);
  const Rsrc rb = make_rsrc(p.B, p.b_bytes);

  // Load sources: rows of A past M and of B past N are clamped onto row /
  // column 0 (they only feed outputs that are never stored); only k past K
  // has to read as zero.
  int32_t a_off[NQ], b_off[NQ];  // element offset without the K-tile's k0
  int a_k[NQ], b_k[NQ];          // the k (within the K-tile) the lane's piece starts at
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int blk = W * q + wave;
    if constexpr (AK) {
      const int row = 8 * blk + (lane >> 3);
      const int c = (lane & 7) ^ krow_swz(row);
      const uint32_t m = tc.m0 + row;
      a_off[q] = tc.a_base + (m < p.M ? row_off(p, m, p.a_m1, p.a_m2) : 0) + 4 * c;
      a_k[q] = 4 * c;
    } else {
      const int row = 2 * blk + (lane >> 5);
      const int c = (lane & 31) ^ mnrow_swz(row);
      const uint32_t m = tc.m0 + 4 * c;
      a_off[q] = tc.a_base + (m < p.M ? row_off(p, m, p.a_m1, p.a_m2) : 0) + row * p.a_k;
      a_k[q] = row;
    }
    if constexpr (BK) {
      const int row = 8 * blk + (lane >> 3);
      const int c = (lane & 7) ^ krow_swz(row);
      const uint32_t n = tc.n0 + row;
      b_off[q] = tc.b_base + (int32_t)(n < p.N ? n : 0) * p.b_n + 4 * c;
      b_k[q] = 4 * c;
    } else {
      const int row = 2 * blk + (lane >> 5);
      const int c = (lane & 31) ^ mnrow_swz(row);
      const uint32_t n = tc.n0 + 4 * c;
      b_off[q] = tc.b_base + (int32_t)(n < p.N ? n : 0) + row * p.b_k;
      b_k[q] = row;
    }
  }
  // elements per unit of k0 along A's and B's k dim
  const int32_t a_ks = AK ? 1 : p.a_k, b_ks = BK ? 1 : p.b_k;

  struct Regs {
    uint4 a[NQ], b[NQ];
  };
  auto gload = [&](Regs& R, uint32_t k0) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const uint32_t ka = k0 + (uint32_t)a_k[q], kb = k0 + (uint32_t)b_k[q];
      R.a[q] = bload16(ra, ka < kend ? 4u * (uint32_t)(a_off[q] + (int32_t)k0 * a_ks) : kOOB);
      R.b[q] = bload16(rb, kb < kend ? 4u * (uint32_t)(b_off[q] + (int32_t)k0 * b_ks) : kOOB);
    }
  };
  auto lstore = [&](const Regs& R, int st) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int blk = W * q + wave;
      *(uint4*)(As[st] + blk * 1024 + lane * 16) = R.a[q];
      *(uint4*)(Bs[st] + blk * 1024 + lane * 16) = R.b[q];
    }
  };

  // operand element (row of the tile's A or B side, k within the K-tile)
  auto a_at = [&](int st, int m, int k) {
    const uint8_t* s = As[st];
    if constexpr (AK) return *(const float*)(s + m * 128 + (((k >> 2) ^ krow_swz(m)) << 4) + (k & 3) * 4);
    else return *(const float*)(s + k * 512 + (((m >> 2) ^ mnrow_swz(k)) << 4) + (m & 3) * 4);
  };
  auto b_at = [&](int st, int n, int k) {
    const uint8_t* s = Bs[st];
    if constexpr (BK) return *(const float*)(s + n * 128 + (((k >> 2) ^ krow_swz(n)) << 4) + (k & 3) * 4);
    else return *(const float*)(s + k * 512 + (((n >> 2) ^ mnrow_swz(k)) << 4) + (n & 3) * 4);
  };

  f32x16 acc[IM][JN];
#pragma unroll
  for (int i = 0; i < IM; ++i)
#pragma unroll
    for (int j = 0; j < JN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  auto compute = [&](int st) {
#pragma unroll
    for (int s = 0; s < FR_BK / 2; ++s) {
      const int k = 2 * s + lh;
      float a[IM], b[JN];
#pragma unroll
      for (int i = 0; i < IM; ++i) a[i] = a_at(st, wm * 32 * IM + 32 * i + lr, k);
#pragma unroll
      for (int j = 0; j < JN; ++j) b[j] = b_at(st, wn * 32 * JN + 32 * j + lr, k);
#pragma unroll
      for (int i = 0; i < IM; ++i)
#pragma unroll
        for (int j = 0; j < JN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  };

  // K-tile t is multiplied from stage t % 2 while K-tile t+2 travels into
  // registers; tile t+1 (loaded during tile t-1) goes to the other stage
  // after the multiply, and one barrier then makes it visible and frees
  // stage t % 2.  Loads past the end of K read zeros.
  const uint32_t nt = (kend + FR_BK - 1) / FR_BK;
  Regs R;
  if (nt > 0) {
    gload(R, 0);
    lstore(R, 0);
  }
  if (nt > 1) gload(R, FR_BK);
  __syncthreads();
  for (uint32_t t = 0; t < nt; t += 2) {
#define FLUID_FR_STEP(U)                                  \
  if (t + U < nt) {                                       \
    compute(U);                                           \
    if (t + U + 1 < nt) {                                 \
      lstore(R, (U + 1) & 1);                             \
      if (t + U + 2 < nt) gload(R, (t + U + 2) * FR_BK);  \
    }                                                     \
    __syncthreads();                                      \
  }
    FLUID_FR_STEP(0)
    FLUID_FR_STEP(1)
#undef FLUID_FR_STEP
  }

  float* C = (float*)p.C;
#pragma unroll
  for (int i = 0; i < IM; ++i)
#pragma unroll
    for (int j = 0; j < JN; ++j)
      epi16<RES>(p, tc.r_base, tc.m0 + wm * 32 * IM + 32 * i + 4 * lh, tc.n0 + wn * 32 * JN + 32 * j + lr, acc[i][j]);
#pragma unroll
  for (int i = 0; i < IM; ++i)
#pragma unroll
    for (int j = 0; j < JN; ++j) {
      const uint32_t n = tc.n0 + wn * 32 * JN + 32 * j + lr;
#pragma unroll
      for (int vg = 0; vg < 4; ++vg) {
        const uint32_t mb = tc.m0 + wm * 32 * IM + 32 * i + 8 * vg + 4 * lh;
        if (n >= p.N || mb >= p.M) continue;
        if (p.cmode == 2) {
          const int32_t o = tc.c_base + row_off(p, mb, p.c_m1, p.c_m2) + (int32_t)n * p.c_n;
          *(float4*)(C + o) = make_float4(acc[i][j][4 * vg], acc[i][j][4 * vg + 1], acc[i][j][4 * vg + 2], acc[i][j][4 * vg + 3]);
        } else {
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const uint32_t m = mb + t;
            if (m < p.M) C[tc.c_base + row_off(p, m, p.c_m1, p.c_m2) + (int32_t)n * p.c_n] = acc[i][j][4 * vg + t];
          }
        }
      }
    }
}

template <int W>
hipError_t ring_go(const NodeKernel& k, hipStream_t s) {
  const GemmParams& p = k.gemm;
  const dim3 grid(p.tiles_m * p.tiles_n * p.G);
#define FLUID_FR(AKv, BKv)                                                                                  \
  do {                                                                                                      \
    if (p.rop) hipLaunchKernelGGL((gemm_f32_ring_kernel<W, AKv, BKv, true>), grid, dim3(64 * W), 0, s, p); \
    else hipLaunchKernelGGL((gemm_f32_ring_kernel<W, AKv, BKv, false>), grid, dim3(64 * W), 0, s, p);      \
  } while (0)
  const bool ak = k.amode == GM_K, bk = k.bmode == GM_K;
  if (ak && bk) FLUID_FR(true, true);
  else if (ak) FLUID_FR(true, false);
  else if (bk) FLUID_FR(false, true);
  else FLUID_FR(false, false);
#undef FLUID_FR
  return hipGetLastError();
}

// fp32 tile 8: sixteen wavefronts; tile 9: eight
hipError_t launch_gemm_f32_ring(const NodeKernel& k, hipStream_t s) {
  if (k.dtype != DT_F32 || (k.amode != GM_K && k.amode != GM_MN) || (k.bmode != GM_K && k.bmode != GM_MN) ||
      (k.gemm_tile != 8 && k.gemm_tile != 9))
    return hipErrorInvalidValue;
  return k.gemm_tile == 8 ? ring_go<16>(k, s) : ring_go<8>(k, s);
}

}  // namespace fluid
