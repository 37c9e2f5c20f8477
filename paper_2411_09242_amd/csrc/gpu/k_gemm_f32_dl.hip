// fp32 GEMM for small M (the projections of a short sequence: M = 128 or 512
// tokens), MFMA 16x16x4 f32.  Such a GEMM has too few 32 x 32 output tiles to
// fill 256 compute units, and each tile's K loop is short, so it is bound by
// how many loads are in flight, not by the matrix cores.  Here:
//
//  * a workgroup owns one (16 FM) x 32 output tile and W wavefronts split
//    its K range into W contiguous slices; at the end the W partial tiles
//    are summed through LDS in wavefront order (a fixed order: the result
//    does not depend on timing);
//  * operands never pass through LDS: each lane loads exactly the values its
//    MFMAs consume, straight from HBM into registers, four 16-k steps ahead.
//    A K-contiguous operand gives a lane four consecutive k in one 16-byte
//    load (one k per MFMA step); an M-/N-contiguous operand is read 4 bytes
//    per lane, sixteen lanes covering 64 contiguous bytes.  A slice of at
//    most six 16-k groups is loaded whole before its first MFMA: a load
//    past the slice (which the rotating four-group loop issues, reading
//    zeros) costs as much issue time as a real one.
//
// MFMA 16x16x4 f32 operand layout: lane l holds A[l % 16][k = l / 16] and
// B[k = l / 16][l % 16]; the result lane l holds D[4 (l / 16) + v][l % 16].
// Step s of a 16-k group uses, in the k slot l / 16, the real k
// 4 (l / 16) + s, the same for A and B.
#include <type_traits>

#include "gemm_common.h"
#include "launch.h"

namespace fluid {

namespace {

constexpr int SK_TN = 32;            // output tile columns
constexpr int SK_FN = 2;             // 16 x 16 blocks across a tile
constexpr int SK_RP = SK_TN + 1;     // LDS reduction row pitch (floats)
constexpr int SK_DEPTH = 4;          // 16-k groups in flight per wavefront

}  // namespace

// One workgroup's tile: tile `bid` of the product p; red is the workgroup's
// W * 16 SK_FM * SK_RP floats of LDS.
template <int W, int SK_FM, int AM, int BMD, bool RES>
__device__ __forceinline__ void gemm_f32_dl_tile(const GemmParams& p, uint32_t bid, float* red) {
  constexpr int SK_TM = 16 * SK_FM;
  const TileCoord tc = tile_coord_at(p, bid, SK_TM, SK_TN);
  // causal attention: a tile entirely above the diagonal is never read; a
  // row block's A is zero past its last row, so K stops there
  if ((p.causal & 1u) && tc.n0 > tc.m0 + SK_TM - 1) return;
  const uint32_t Kc = (p.causal & 2u) ? min(p.K, tc.m0 + SK_TM) : p.K;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lq = lane >> 4;
  const Rsrc ra = make_rsrc(p.A, p.a_bytes);
  const Rsrc rb = make_rsrc(p.B, p.b_bytes);

  // this wavefront's K slice [kbeg, kend), a multiple of 16 long
  const uint32_t kw = ((Kc + 16u * W - 1u) / (16u * W)) * 16u;
  const uint32_t kbeg = wave * kw;
  const uint32_t kend = min(Kc, kbeg + kw);
  const uint32_t ngroups = kend > kbeg ? (kend - kbeg + 15u) / 16u : 0u;

  // Rows past M and columns past N only feed outputs that are never
  // stored: they are clamped onto row / column 0.  k outside the slice reads
  // as zero (kOOB).
  int32_t a_row[SK_FM];
#pragma unroll
  for (int i = 0; i < SK_FM; ++i) {
    const uint32_t m = tc.m0 + 16 * i + lr;
    a_row[i] = tc.a_base + (m < p.M ? row_off(p, m, p.a_m1, p.a_m2) : 0);
  }
  int32_t b_col[SK_FN];
#pragma unroll
  for (int j = 0; j < SK_FN; ++j) {
    const uint32_t n = tc.n0 + 16 * j + lr;
    b_col[j] = tc.b_base + (int32_t)(n < p.N ? n : 0) * p.b_n;
  }

  // one 16-k group of this lane's operands: [block][step]
  struct Grp {
    float a[SK_FM][4];
    float b[SK_FN][4];
  };
  auto load = [&](Grp& G, uint32_t g) {
    const uint32_t k0 = kbeg + 16u * g + 4u * lq;  // this lane's first k
#pragma unroll
    for (int i = 0; i < SK_FM; ++i) {
      if constexpr (AM == GM_K) {
        const uint4 u = bload16(ra, k0 < kend ? 4u * (uint32_t)(a_row[i] + (int32_t)k0) : kOOB);
        G.a[i][0] = __uint_as_float(u.x); G.a[i][1] = __uint_as_float(u.y);
        G.a[i][2] = __uint_as_float(u.z); G.a[i][3] = __uint_as_float(u.w);
      } else {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const uint32_t k = k0 + s;
          G.a[i][s] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                          ra, k < kend ? 4u * (uint32_t)(a_row[i] + (int32_t)k * p.a_k) : kOOB, 0, 0));
        }
      }
    }
#pragma unroll
    for (int j = 0; j < SK_FN; ++j) {
      if constexpr (BMD == GM_K) {
        const uint4 u = bload16(rb, k0 < kend ? 4u * (uint32_t)(b_col[j] + (int32_t)k0) : kOOB);
        G.b[j][0] = __uint_as_float(u.x); G.b[j][1] = __uint_as_float(u.y);
        G.b[j][2] = __uint_as_float(u.z); G.b[j][3] = __uint_as_float(u.w);
      } else {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const uint32_t k = k0 + s;
          G.b[j][s] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                          rb, k < kend ? 4u * (uint32_t)(b_col[j] + (int32_t)k * p.b_k) : kOOB, 0, 0));
        }
      }
    }
  };

  f32x4 acc[SK_FM][SK_FN];
#pragma unroll
  for (int i = 0; i < SK_FM; ++i)
#pragma unroll
    for (int j = 0; j < SK_FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](const Grp& G) {
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int i = 0; i < SK_FM; ++i)
#pragma unroll
        for (int j = 0; j < SK_FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(G.a[i][s], G.b[j][s], acc[i][j], 0, 0, 0);
  };

  if (ngroups <= 6) {
    // a short slice: all its groups are loaded before the first MFMA, with
    // no load past its end
    auto straight = [&](auto nc) {
      constexpr int n = decltype(nc)::value;
      Grp S[n];
#pragma unroll
      for (int i = 0; i < n; ++i) load(S[i], i);
#pragma unroll
      for (int i = 0; i < n; ++i) compute(S[i]);
    };
    switch (ngroups) {
      case 1: straight(std::integral_constant<int, 1>{}); break;
      case 2: straight(std::integral_constant<int, 2>{}); break;
      case 3: straight(std::integral_constant<int, 3>{}); break;
      case 4: straight(std::integral_constant<int, 4>{}); break;
      case 5: straight(std::integral_constant<int, 5>{}); break;
      case 6: straight(std::integral_constant<int, 6>{}); break;
      default: break;  // an empty slice
    }
  } else {
    // group g travels in register set g % 4, loaded three groups before
    // use; groups past the slice read zeros and their MFMAs are skipped
    Grp G0, G1, G2, G3;
    load(G0, 0);
    load(G1, 1);
    load(G2, 2);
    for (uint32_t g = 0; g < ngroups; g += SK_DEPTH) {
      load(G3, g + 3);
      compute(G0);
      load(G0, g + 4);
      if (g + 1 < ngroups) compute(G1);
      load(G1, g + 5);
      if (g + 2 < ngroups) compute(G2);
      load(G2, g + 6);
      if (g + 3 < ngroups) compute(G3);
    }
  }

  // partial tiles -> LDS, then every thread sums W partials of some outputs
#pragma unroll
  for (int i = 0; i < SK_FM; ++i)
#pragma unroll
    for (int j = 0; j < SK_FN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        red[(wave * SK_TM + 16 * i + 4 * lq + v) * SK_RP + 16 * j + lr] = acc[i][j][v];
  __syncthreads();
  float* C = (float*)p.C;
  if (p.cmode == 2) {
    // M-contiguous C: a thread writes 4 consecutive rows of one column
    for (int e = tid; e < SK_TM * SK_TN / 4; e += 64 * W) {
      const int c = e / (SK_TM / 4), r0 = (e % (SK_TM / 4)) * 4;
      const uint32_t n = tc.n0 + c, m0 = tc.m0 + r0;
      if (n >= p.N) continue;
      float o[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        float sum = 0.f;
        for (int w = 0; w < W; ++w) sum += red[(w * SK_TM + r0 + t) * SK_RP + c];
        o[t] = gemm_epi<RES>(p, tc.r_base, m0 + t, n, sum);
      }
      // four rows m0..m0+3 lie in one M2 run (M2 % 4 == 0 in this mode)
      if (m0 + 3 < p.M) {
        *(float4*)(C + tc.c_base + row_off(p, m0, p.c_m1, p.c_m2) + (int32_t)n * p.c_n) = make_float4(o[0], o[1], o[2], o[3]);
      } else {
        for (int t = 0; t < 4; ++t)
          if (m0 + t < p.M) C[tc.c_base + row_off(p, m0 + t, p.c_m1, p.c_m2) + (int32_t)n * p.c_n] = o[t];
      }
    }
  } else {
    // a thread writes 4 consecutive columns of one row (one 16-byte store
    // when C is N-contiguous)
    for (int e = tid; e < SK_TM * SK_TN / 4; e += 64 * W) {
      const int r = e / (SK_TN / 4), c0 = (e % (SK_TN / 4)) * 4;
      const uint32_t m = tc.m0 + r, n0 = tc.n0 + c0;
      if (m >= p.M) continue;
      float o[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        float sum = 0.f;
        for (int w = 0; w < W; ++w) sum += red[(w * SK_TM + r) * SK_RP + c0 + t];
        o[t] = n0 + t < p.N ? gemm_epi<RES>(p, tc.r_base, m, n0 + t, sum) : sum;
      }
      const int32_t base = tc.c_base + row_off(p, m, p.c_m1, p.c_m2);
      if (p.cmode == 1 && n0 + 3 < p.N && ((uintptr_t)(C + base + (int32_t)n0) & 15u) == 0) {
        *(float4*)(C + base + (int32_t)n0) = make_float4(o[0], o[1], o[2], o[3]);
      } else {
        for (int t = 0; t < 4; ++t)
          if (n0 + t < p.N) C[base + (int32_t)(n0 + t) * p.c_n] = o[t];
      }
    }
  }
}

template <int W, int SK_FM, int AM, int BMD, bool RES>
__global__ __launch_bounds__(64 * W) void gemm_f32_dl_kernel(GemmParams p) {
  __shared__ float red[W * 16 * SK_FM * SK_RP];
  gemm_f32_dl_tile<W, SK_FM, AM, BMD, RES>(p, blockIdx.x, red);
}

// The members of a group share tile shape, operand modes and epilogue
// instance; each workgroup runs one tile of its member.
template <int W, int SK_FM, int AM, int BMD, bool RES>
__global__ __launch_bounds__(64 * W) void gemm_f32_dl_group_kernel(GemmGroup G) {
  __shared__ float red[W * 16 * SK_FM * SK_RP];
  uint32_t i = 0;
  while (i + 1 < G.n && blockIdx.x >= G.tiles[i + 1]) ++i;
  gemm_f32_dl_tile<W, SK_FM, AM, BMD, RES>(G.p[i], blockIdx.x - G.tiles[i], red);
}


hipError_t launch_gemm_f32_dl(const NodeKernel& k, hipStream_t s) {
  const GemmParams& p = k.gemm;
  const dim3 grid(p.tiles_m * p.tiles_n * p.G);
#define FLUID_F32DL(Wv, FMv, AMv, BMv)                                                                     \
  do {                                                                                                     \
    if (p.rop) hipLaunchKernelGGL((gemm_f32_dl_kernel<Wv, FMv, AMv, BMv, true>), grid, dim3(64 * Wv), 0, s, p); \
    else hipLaunchKernelGGL((gemm_f32_dl_kernel<Wv, FMv, AMv, BMv, false>), grid, dim3(64 * Wv), 0, s, p);      \
  } while (0)
#define FLUID_F32DL_W(Wv, FMv)                                                          \
  if (k.amode == GM_K && k.bmode == GM_MN) FLUID_F32DL(Wv, FMv, GM_K, GM_MN);           \
  else if (k.amode == GM_K && k.bmode == GM_K) FLUID_F32DL(Wv, FMv, GM_K, GM_K);        \
  else if (k.amode == GM_MN && k.bmode == GM_MN) FLUID_F32DL(Wv, FMv, GM_MN, GM_MN);    \
  else if (k.amode == GM_MN && k.bmode == GM_K) FLUID_F32DL(Wv, FMv, GM_MN, GM_K);      \
  else return hipErrorInvalidValue;
  // tile 6: 16 x 32 over 8 wavefronts; tile 7: 32 x 32 over 4
  if (k.gemm_tile == 6) {
    FLUID_F32DL_W(8, 1)
  } else {
    FLUID_F32DL_W(4, 2)
  }
#undef FLUID_F32DL_W
#undef FLUID_F32DL
  return hipGetLastError();
}

hipError_t launch_gemm_f32_dl_group(const NodeKernel& k, const GemmGroup& G, hipStream_t s) {
  if (k.dtype != DT_F32 || (k.gemm_tile != 6 && k.gemm_tile != 7) || G.n < 1 || G.n > (uint32_t)kMaxGroup)
    return hipErrorInvalidValue;
  const bool res = k.gemm.rop != 0;
  const dim3 grid(G.tiles[G.n]);
#define FLUID_F32DLG(Wv, FMv, AMv, BMv)                                                                          \
  do {                                                                                                           \
    if (res) hipLaunchKernelGGL((gemm_f32_dl_group_kernel<Wv, FMv, AMv, BMv, true>), grid, dim3(64 * Wv), 0, s, G); \
    else hipLaunchKernelGGL((gemm_f32_dl_group_kernel<Wv, FMv, AMv, BMv, false>), grid, dim3(64 * Wv), 0, s, G);    \
  } while (0)
#define FLUID_F32DLG_W(Wv, FMv)                                                          \
  if (k.amode == GM_K && k.bmode == GM_MN) FLUID_F32DLG(Wv, FMv, GM_K, GM_MN);           \
  else if (k.amode == GM_K && k.bmode == GM_K) FLUID_F32DLG(Wv, FMv, GM_K, GM_K);        \
  else if (k.amode == GM_MN && k.bmode == GM_MN) FLUID_F32DLG(Wv, FMv, GM_MN, GM_MN);    \
  else if (k.amode == GM_MN && k.bmode == GM_K) FLUID_F32DLG(Wv, FMv, GM_MN, GM_K);      \
  else return hipErrorInvalidValue;
  if (k.gemm_tile == 6) {
    FLUID_F32DLG_W(8, 1)
  } else {
    FLUID_F32DLG_W(4, 2)
  }
#undef FLUID_F32DLG_W
#undef FLUID_F32DLG
  return hipGetLastError();
}

}  // namespace fluid
