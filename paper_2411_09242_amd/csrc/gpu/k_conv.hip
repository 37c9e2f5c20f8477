// Convolution (no padding, stride 1, one group) as an implicit GEMM on MFMA
// (gfx950), for any layout of the input and output.
//
//   y[n, o, i, j] = sum_{c, u, v} x[n, c, i+u, j+v] * w[o, c, u, v] + b[o]
//
// Rows m = (n, i, j) are output pixels, columns are output channels o, and
// the reduction runs over k = (c, u, v).  In any layout, x[n, c, i+u, j+v]
// sits at row_offset(m) + col_offset(k) with row_offset = n*sN + i*sH + j*sW
// and col_offset = c*sC + u*sH + v*sW, so the unfolded input matrix is never
// built: each thread keeps the row offsets of its pixels and forms column
// offsets per K-tile.  Two load orders:
//   KORD 0: k = (c, u, v) (the weight's row-major order); a wavefront loads
//           64 consecutive pixels of one k -- coalesced when W is the
//           input's unit-stride dim (NCHW-like layouts);
//   KORD 1: k = (u, v, c); a wavefront loads 16 consecutive k of 4 pixels --
//           coalesced when C is unit-stride (NHWC-like layouts).
// A 64 x 64 output tile per group of 256 threads (4 wavefronts, 2 x 2, each
// 32 x 32 -- or a 32 x 32 tile per single-wavefront group -- with
// v_mfma_f32_32x32x2_f32: lane l reads A[l%32][l/32] and
// B[l/32][l%32]; accumulator v of lane l holds C[8(v/4) + 4(l/32) + v%4][l%32]),
// operands staged in LDS K-major, the next K-tile loaded into registers
// while the current one is multiplied.  KS groups share a workgroup and a
// tile, group g taking K-tiles g, g + KS, ...: KS times the wavefronts and
// K-tiles in flight per tile, for layers with fewer tiles than compute
// units; the groups' partial sums are added through LDS in group order
// (deterministic).  The bias is added in fp32 before the store.
#include "dev.h"
#include "launch.h"

namespace fluid {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

template <int KORD>
__device__ __forceinline__ int32_t conv_col_off(const ConvParams& p, uint32_t k, int32_t* waddr) {
  uint32_t c, u, v;
  if constexpr (KORD == 0) {
    c = fdiv(k, p.khw_div);
    const uint32_t r = k - c * p.KHW;
    u = fdiv(r, p.kw_div);
    v = r - u * p.KW;
  } else {
    u = fdiv(k, p.kwc_div);
    const uint32_t r = k - u * p.KWC;
    v = fdiv(r, p.c_div);
    c = r - v * p.C;
  }
  *waddr = (int32_t)(c * p.KHW + u * p.KW + v);
  return (int32_t)c * p.x_c + (int32_t)u * p.x_h + (int32_t)v * p.x_w;
}

template <int KORD, int KS, int TW>
__global__ __launch_bounds__(64 * (TW / 32) * (TW / 32) * KS) void conv_f32_kernel(ConvParams p) {
  // TW x TW output tile per group of WPG wavefronts ((TW/32)^2, each a
  // 32 x 32 block); NT threads per group
  constexpr int WPG = (TW / 32) * (TW / 32), NT = 64 * WPG;
  constexpr int BM = TW, BN = TW, BK = 16;
  constexpr int AP = BM + 4, BP = BN + 4;
  constexpr int AE = BM * BK / NT, BE = BN * BK / NT;  // elements per thread per K-tile
  constexpr int STAGE = BK * AP + BK * BP;            // one group's A and B tiles
  constexpr int RED = (KS - 1) * 16 * NT;             // partial sums of groups 1 .. KS-1
  constexpr int SMEM = KS * STAGE > RED ? KS * STAGE : RED;
  __shared__ float smem[SMEM];
  // the group index is uniform per wavefront: keep it in a scalar register
  const int grp = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / NT));
  float* As = smem + grp * STAGE;
  float* Bs = As + BK * AP;
  const uint32_t tm = blockIdx.x / p.tiles_n, tn = blockIdx.x - tm * p.tiles_n;
  const uint32_t m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x % NT, lane = tid & 63, wave = tid >> 6;
  const int wm = WPG > 1 ? wave >> 1 : 0, wn = WPG > 1 ? wave & 1 : 0;

  auto row_off = [&](uint32_t m, int32_t sn, int32_t sh, int32_t sw) {
    const uint32_t n = fdiv(m, p.ohw_div);
    const uint32_t r = m - n * p.OHW;
    const uint32_t i = fdiv(r, p.ow_div);
    const uint32_t j = r - i * p.OW;
    return (int32_t)n * sn + (int32_t)i * sh + (int32_t)j * sw;
  };

  // A: AE elements per thread per K-tile; element r of thread t is index
  // t + NT r of the tile, pixel-fastest (KORD 0) or k-fastest (KORD 1)
  int a_m[AE], a_k[AE];
  int32_t a_off[AE];
  bool a_ok[AE];
#pragma unroll
  for (int r = 0; r < AE; ++r) {
    const int idx = tid + NT * r;
    if constexpr (KORD == 0) {
      a_m[r] = idx % BM;
      a_k[r] = idx / BM;
    } else {
      a_k[r] = idx % BK;
      a_m[r] = idx / BK;
    }
    const uint32_t m = m0 + a_m[r];
    a_ok[r] = m < p.M;
    a_off[r] = a_ok[r] ? row_off(m, p.x_n, p.x_h, p.x_w) : 0;
  }
  // B (weights): 16 consecutive k of one channel per 16 lanes
  int b_k[BE], b_n[BE];
  bool b_ok[BE];
#pragma unroll
  for (int r = 0; r < BE; ++r) {
    const int idx = tid + NT * r;
    b_k[r] = idx % BK;
    b_n[r] = idx / BK;
    b_ok[r] = n0 + b_n[r] < p.Co;
  }

  float ra[AE], rb[BE];
  auto gload = [&](uint32_t k0) {
    if constexpr (KORD == 0) {
      // per element its own k
#pragma unroll
      for (int r = 0; r < AE; ++r) {
        const uint32_t k = k0 + a_k[r];
        int32_t wa;
        const int32_t co = k < p.K ? conv_col_off<0>(p, k, &wa) : 0;
        ra[r] = (a_ok[r] && k < p.K) ? p.x[a_off[r] + co] : 0.f;
      }
    } else {
      // one k per thread (NT is a multiple of BK), several pixels
      const uint32_t k = k0 + a_k[0];
      int32_t wa;
      const int32_t co = k < p.K ? conv_col_off<1>(p, k, &wa) : 0;
#pragma unroll
      for (int r = 0; r < AE; ++r) ra[r] = (a_ok[r] && k < p.K) ? p.x[a_off[r] + co] : 0.f;
    }
    {
      const uint32_t k = k0 + b_k[0];
      int32_t wa = 0;
      if (k < p.K) (void)conv_col_off<KORD>(p, k, &wa);
#pragma unroll
      for (int r = 0; r < BE; ++r)
        rb[r] = (b_ok[r] && k < p.K) ? p.w[(int32_t)(n0 + b_n[r]) * (int32_t)p.K + wa] : 0.f;
    }
  };
  auto lstore = [&]() {
#pragma unroll
    for (int r = 0; r < AE; ++r) As[a_k[r] * AP + a_m[r]] = ra[r];
#pragma unroll
    for (int r = 0; r < BE; ++r) Bs[b_k[r] * BP + b_n[r]] = rb[r];
  };

  f32x16 acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.f;
  const int lr = lane & 31, lk = lane >> 5;
  // every group runs the same number of rounds (the barriers are
  // workgroup-wide); a group's K-tile past the end loads zeros
  const uint32_t rounds = (p.K + KS * BK - 1) / (KS * BK);
  gload((uint32_t)grp * BK);
  for (uint32_t r = 0; r < rounds; ++r) {
    __syncthreads();
    lstore();
    __syncthreads();
    if (r + 1 < rounds) gload(((r + 1) * KS + (uint32_t)grp) * BK);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 2) {
      const float a = As[(kk + lk) * AP + wm * 32 + lr];
      const float b = Bs[(kk + lk) * BP + wn * 32 + lr];
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
    }
  }
  if constexpr (KS > 1) {
    // groups 1 .. KS-1 park their sums; group 0 adds them in group order
    __syncthreads();
    if (grp > 0) {
#pragma unroll
      for (int v = 0; v < 16; ++v) smem[((grp - 1) * 16 + v) * NT + tid] = acc[v];
    }
    __syncthreads();
    if (grp > 0) return;
#pragma unroll
    for (int g = 0; g < KS - 1; ++g)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] += smem[(g * 16 + v) * NT + tid];
  }

  const uint32_t o = n0 + wn * 32 + lr;
  if (o >= p.Co) return;
  const float bo = p.bias ? p.bias[o] : 0.f;
#pragma unroll
  for (int vg = 0; vg < 4; ++vg)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const uint32_t m = m0 + wm * 32 + 8 * vg + 4 * lk + t;
      if (m < p.M) p.y[row_off(m, p.y_n, p.y_h, p.y_w) + (int32_t)o * p.y_c] = acc[4 * vg + t] + bo;
    }
}

}  // namespace

hipError_t launch_conv(const NodeKernel& k, hipStream_t s) {
  const ConvParams& p = k.conv;
  const uint32_t tw = k.conv_tile;
  const uint32_t grid = ((p.M + tw - 1) / tw) * p.tiles_n;
#define FLUID_CONV(KO, KSv, TWv) \
  hipLaunchKernelGGL((conv_f32_kernel<KO, KSv, TWv>), dim3(grid), dim3(64 * (TWv / 32) * (TWv / 32) * KSv), 0, s, p)
  if (tw == 64 && k.conv_ks == 1) {
    if (k.conv_kord == 0) FLUID_CONV(0, 1, 64);
    else FLUID_CONV(1, 1, 64);
  } else if (tw == 64 && k.conv_ks == 4) {
    if (k.conv_kord == 0) FLUID_CONV(0, 4, 64);
    else FLUID_CONV(1, 4, 64);
  } else if (tw == 32 && k.conv_ks == 8) {
    if (k.conv_kord == 0) FLUID_CONV(0, 8, 32);
    else FLUID_CONV(1, 8, 32);
  } else {
    return hipErrorInvalidValue;
  }
#undef FLUID_CONV
  return hipGetLastError();
}

}  // namespace fluid
