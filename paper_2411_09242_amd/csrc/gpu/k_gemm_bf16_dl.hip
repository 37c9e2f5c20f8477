// bf16 GEMM for a K-contiguous A and an N-contiguous B (the projection
// shape: activations times a row-major weight) or a K-contiguous B (Q K^T
// with K stored [S, D]), MFMA 32x32x16 bf16 with fp32 accumulate, written
// around three gfx950 features:
//
//  * both operands go from HBM to LDS by direct buffer loads
//    (`buffer_load ... lds`: no registers, no VALU work), each in its
//    natural layout -- A as [m][k] rows of 32 k, an N-contiguous B as [k][n]
//    rows of 128 n, a K-contiguous B as [n][k] rows of 32 k;
//  * B is read back with ds_read_b64_tr_b16, which hands each lane four
//    k-consecutive values of one column n; two such reads make one 8-k MFMA
//    operand, so the N-contiguous weight never needs a VALU transpose;
//  * MFMA 32x32x16 bf16, which a single wavefront per SIMD issues at close
//    to the matrix cores' full rate (the 16x16x32 form reaches about 60%).
//
// Workgroup tile 256 x 128, four wavefronts stacked along M (64 x 128 each).
// Both tiles live in a four-stage LDS ring (24 KiB per stage) and are loaded
// three K-tiles ahead.  One barrier per K-tile, a bare s_barrier behind an
// explicit counter wait: after a wavefront has waited for its own loads of
// tile t, the barrier makes every wavefront's part of tile t visible and
// frees the stage that tile t+3 overwrites (a workgroup fence would wait for
// the later tiles' loads too).
//
// The DMA writes 64 lanes x 16 bytes contiguously, so the bank-conflict
// swizzles are applied by choosing which 16-byte chunk each lane fetches:
//  * A row r (64 bytes) stores chunk c at c ^ (((r >> 1) ^ (r >> 3)) & 3):
//    the 32 rows one A-operand read touches then cover every bank once;
//  * an N-contiguous B row r (256 bytes) stores chunk c at c ^ 4 (r % 4): a
//    transpose read touches four consecutive rows at the same columns,
//    which the swizzle puts in four different 64-byte bank groups; a
//    K-contiguous B is laid out and read like A.
//
// The output tile leaves through LDS when C is N- or M-contiguous, so that
// every lane writes 16 contiguous bytes (an S x S score matrix is mostly
// store traffic): each wavefront parks its 64 x 128 bf16 tile in its own
// 16 KiB of the ring, swizzled so that both the parking writes and the
// 16-byte reads are conflict-free.
#include "gemm_common.h"
#include "launch.h"

namespace fluid {

namespace {

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __attribute__((address_space(3))) uint4 lds_uint4;
typedef __attribute__((address_space(3))) void lds_void;

constexpr int DL_BM = 256, DL_BN = 128, DL_BK = 32;
constexpr int DL_AROWB = DL_BK * 2;              // bytes per A row in LDS (one m)
constexpr int DL_BROWB = DL_BN * 2;              // bytes per B row in LDS (one k)
constexpr int DL_ASTAGE = DL_BM * DL_AROWB;      // 16 KiB
constexpr int DL_BSTAGE = DL_BK * DL_BROWB;      // 8 KiB

__device__ __forceinline__ int a_swz(int r) { return ((r >> 1) ^ (r >> 3)) & 3; }

}  // namespace

// NS = 4: the ring above, one workgroup per CU.  NS = 3: a three-stage ring
// (72 KiB, tiles loaded two ahead) and at most 256 registers per lane
// (VGPRs and AGPRs together), so that two workgroups share a CU and one's
// loads, barrier waits and epilogue overlap the other's MFMAs: faster where
// there are many tiles or K is short (Q K^T, the 11008-wide FFN GEMMs).
template <int BMD, int NS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(NS == 3 ? 2 : 1, NS == 3 ? 2 : 1)))
void gemm_bf16_dl_kernel(GemmParams p) {
  static_assert(NS == 3 || NS == 4, "three or four stages");
  constexpr int BK = DL_BK;
  constexpr int FM = 2, FN = 4;  // wavefront tile 64 x 128 in 32 x 32 blocks
  // one LDS object per stage and operand, so that the compiler can tell a
  // DMA into one stage from reads of another and does not wait for every
  // load in flight
  __shared__ __attribute__((aligned(1024))) uint8_t As0[DL_ASTAGE];
  __shared__ __attribute__((aligned(1024))) uint8_t As1[DL_ASTAGE];
  __shared__ __attribute__((aligned(1024))) uint8_t As2[DL_ASTAGE];
  __shared__ __attribute__((aligned(NS > 3 ? 1024 : 16))) uint8_t As3[NS > 3 ? DL_ASTAGE : 16];
  __shared__ __attribute__((aligned(1024))) uint8_t Bs0[DL_BSTAGE];
  __shared__ __attribute__((aligned(1024))) uint8_t Bs1[DL_BSTAGE];
  __shared__ __attribute__((aligned(1024))) uint8_t Bs2[DL_BSTAGE];
  __shared__ __attribute__((aligned(NS > 3 ? 1024 : 16))) uint8_t Bs3[NS > 3 ? DL_BSTAGE : 16];
  // stage indices are compile-time constants in the loop; only the epilogue
  // selects an A stage (its own wavefront's, < 4) at run time
  auto astage = [&](int st) -> uint8_t* { return st == 0 ? As0 : st == 1 ? As1 : st == 2 ? As2 : As3; };
  auto bstage = [&](int st) -> uint8_t* { return st == 0 ? Bs0 : st == 1 ? Bs1 : st == 2 ? Bs2 : Bs3; };
  const TileCoord tc = tile_coord(p, DL_BM, DL_BN);
  // causal attention: a tile entirely above the diagonal is never read; a
  // row block's A is zero past its last row, so K stops there
  if ((p.causal & 1u) && tc.n0 > tc.m0 + DL_BM - 1) return;
  const uint32_t kend = (p.causal & 2u) ? min(p.K, tc.m0 + DL_BM) : p.K;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: DMA base in M0
  const int lr = lane & 31, lh = lane >> 5;
  const Rsrc ra = make_rsrc(p.A, p.a_bytes);
  const Rsrc rb = make_rsrc(p.B, p.b_bytes);

  // Rows of A past M and columns of B past N only feed outputs that are
  // never stored, so they are clamped onto row / column 0 instead of being
  // masked; only k past K has to read as zero.
  // A DMA: round q of wavefront w fills tile rows 16 (4q + w) .. +15; lane l
  // writes chunk position l % 4 of row l / 4, holding logical chunk
  // (l % 4) ^ swizzle(row).
  int32_t a_src[4];
  int a_chunk[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int row = 16 * (4 * q + wave) + (lane >> 2);
    const uint32_t m = tc.m0 + row;
    a_src[q] = tc.a_base + (m < p.M ? row_off(p, m, p.a_m1, p.a_m2) : 0);
    a_chunk[q] = (lane & 3) ^ a_swz(row);
  }
  // N-contiguous B DMA: round q fills rows 16 q + 4 w .. +3; lane l writes
  // chunk position l % 16 of row l / 16, holding logical chunk
  // (l % 16) ^ 4 (row % 4).  K-contiguous B DMA: like A, round q of
  // wavefront w fills rows (n) 16 (4q + w) .. +15.
  const int b_rsub = lane >> 4;
  const int b_chunk = (lane & 15) ^ (4 * b_rsub);
  const uint32_t b_n = tc.n0 + 8 * b_chunk;
  const int32_t b_col = tc.b_base + (int32_t)(b_n < p.N ? b_n : 0);
  int32_t bk_src[2];
  int bk_chunk[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int row = 16 * (4 * q + wave) + (lane >> 2);
    const uint32_t n = tc.n0 + row;
    bk_src[q] = tc.b_base + (int32_t)(n < p.N ? n : 0) * p.b_n;
    bk_chunk[q] = (lane & 3) ^ a_swz(row);
  }

  auto load = [&](int st, uint32_t k0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t k = k0 + 8 * a_chunk[q];
      const uint32_t off = k < kend ? 2u * (uint32_t)(a_src[q] + (int32_t)k) : kOOB;
      lds_void* dst = (lds_void*)(astage(st) + 16 * (4 * q + wave) * DL_AROWB);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, dst, 16, off, 0, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      if constexpr (BMD == GM_MN) {
        const int row = 16 * q + 4 * wave + b_rsub;
        const uint32_t k = k0 + row;
        const uint32_t off = k < kend ? 2u * (uint32_t)(b_col + (int32_t)k * p.b_k) : kOOB;
        lds_void* dst = (lds_void*)(bstage(st) + (16 * q + 4 * wave) * DL_BROWB);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, dst, 16, off, 0, 0, 0);
      } else {
        const uint32_t k = k0 + 8 * bk_chunk[q];
        const uint32_t off = k < kend ? 2u * (uint32_t)(bk_src[q] + (int32_t)k) : kOOB;
        lds_void* dst = (lds_void*)(bstage(st) + 16 * (4 * q + wave) * DL_AROWB);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, dst, 16, off, 0, 0, 0);
      }
    }
  };
  constexpr int kTile = 6;  // DMA instructions per tile and wavefront

  // A operand of block i, k-step kk: row 64 w + 32 i + l % 32, logical chunk
  // 2 kk + l / 32
  auto a_addr = [&](int st, int i, int kk) {
    const int row = wave * 64 + 32 * i + lr;
    const int chunk = (2 * kk + lh) ^ a_swz(row);
    return (const lds_uint4*)(astage(st) + row * DL_AROWB + chunk * 16);
  };
  // transpose-read addressing: lane l (group g = l / 16, s = l % 16) points
  // at row 8 (g / 2) + 4 h + s / 4 of the 16-k slice, columns
  // 32 j + 16 (g % 2) + 4 (s % 4) .. +3; the read returns column
  // 32 j + (l % 32), rows 8 (l / 32) + 4 h .. +3.
  const int tg = lane >> 4, ts = lane & 15;
  const int t_row = 8 * (tg >> 1) + (ts >> 2);
  const int t_col = 16 * (tg & 1) + 4 * (ts & 3);
  auto b_addr = [&](int st, int kk, int h, int j) {
    const int row = 16 * kk + 4 * h + t_row;  // row % 4 == ts / 4
    const int col = 32 * j + t_col;
    const int chunk = (col >> 3) ^ (4 * (row & 3));
    return (lds_v4i16*)(bstage(st) + row * DL_BROWB + chunk * 16 + (col & 7) * 2);
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  auto compute = [&](int st) {
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) a[i] = __builtin_bit_cast(bf16x8, *a_addr(st, i, kk));
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        if constexpr (BMD == GM_MN) {
          const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(b_addr(st, kk, 0, j));
          const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(b_addr(st, kk, 1, j));
          b[j] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        } else {
          // [n][k] rows like A: row 32 j + l % 32, logical chunk 2 kk + l / 32
          const int row = 32 * j + lr;
          const int chunk = (2 * kk + lh) ^ a_swz(row);
          b[j] = __builtin_bit_cast(bf16x8, *(const lds_uint4*)(bstage(st) + row * DL_AROWB + chunk * 16));
        }
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  };

  // Tile t lives in stage t % NS and is loaded NS - 1 tiles ahead.  Loads
  // past the end of K read zeros, so the loop runs whole groups of NS tiles
  // (padding tiles add zeros).
  const uint32_t nt = (kend + BK - 1) / BK;
#pragma unroll
  for (int u = 0; u < NS - 1; ++u) load(u, u * BK);
  for (uint32_t t = 0; t < nt; t += NS) {
#define FLUID_DL_STEP(U)                                            \
  asm volatile("" ::: "memory");                                    \
  __builtin_amdgcn_s_waitcnt(vmcnt_imm((NS - 2) * kTile));          \
  __builtin_amdgcn_s_barrier();                                     \
  asm volatile("" ::: "memory");                                    \
  load((U + NS - 1) % NS, (t + U + NS - 1) * BK);                   \
  compute(U);
    FLUID_DL_STEP(0)
    FLUID_DL_STEP(1)
    FLUID_DL_STEP(2)
    if constexpr (NS > 3) {
      FLUID_DL_STEP(3)
    }
#undef FLUID_DL_STEP
  }

  uint16_t* C = (uint16_t*)p.C;
  const uint32_t wm0 = tc.m0 + wave * 64;  // first row of this wavefront's tile
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) epi16<false, false>(p, tc.r_base, wm0 + i * 32 + 4 * lh, tc.n0 + j * 32 + lr, acc[i][j]);
  if (p.cmode == 1 || p.cmode == 2) {
    // the padding tiles' loads land in the ring: drain them, and let every
    // wavefront finish its last tile, before the ring is reused
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    __syncthreads();
    // 16 KiB for this wavefront's 64 x 128 tile, as two 8 KiB halves: its
    // own A stage, or with three stages, for wavefront 3, two B stages
    auto half = [&](int h) -> uint16_t* {
      if (NS == 3 && wave == 3) return (uint16_t*)(h ? Bs1 : Bs0);
      return (uint16_t*)(astage(wave) + 8192 * h);
    };
    if (p.cmode == 1) {
      // row-major [64][128], 16-byte chunk c of row r at c ^ (r % 16)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int r = i * 32 + 8 * (v / 4) + 4 * lh + (v % 4), c = j * 32 + lr;
            half(r >> 5)[(r & 31) * 128 + (((c >> 3) ^ (r & 15)) << 3) + (c & 7)] = f32_to_bf16(acc[i][j][v]);
          }
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): own parking writes done
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int r = 4 * u + (lane >> 4), ch = lane & 15;
        const uint4 val = *(const uint4*)&half(r >> 5)[(r & 31) * 128 + ((ch ^ (r & 15)) << 3)];
        const uint32_t m = wm0 + r, n0 = tc.n0 + 8 * ch;
        if (m >= p.M || n0 >= p.N) continue;
        uint16_t* dst = C + tc.c_base + row_off(p, m, p.c_m1, p.c_m2) + (int32_t)n0;
        if (n0 + 8 <= p.N && ((uintptr_t)dst & 15u) == 0) {
          *(uint4*)dst = val;
        } else {
          const uint32_t w[4] = {val.x, val.y, val.z, val.w};
          for (int e = 0; e < 8 && n0 + e < p.N; ++e) dst[e] = (uint16_t)(w[e / 2] >> (16 * (e & 1)));
        }
      }
    } else {
      // column-major [128][64] (rows contiguous), 16-byte chunk c of column
      // n at c ^ ((n / 2) % 8); a lane parks 4 consecutive rows (8 bytes)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int vg = 0; vg < 4; ++vg) {
            const int r0 = i * 32 + 8 * vg + 4 * lh, c = j * 32 + lr;
            const uint32_t lo = (uint32_t)f32_to_bf16(acc[i][j][4 * vg]) | ((uint32_t)f32_to_bf16(acc[i][j][4 * vg + 1]) << 16);
            const uint32_t hi = (uint32_t)f32_to_bf16(acc[i][j][4 * vg + 2]) | ((uint32_t)f32_to_bf16(acc[i][j][4 * vg + 3]) << 16);
            *(uint2*)&half(c >> 6)[(c & 63) * 64 + ((((r0 >> 3) ^ ((c >> 1) & 7))) << 3) + (r0 & 7)] = make_uint2(lo, hi);
          }
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int c = 8 * u + (lane >> 3), ch = lane & 7;
        const uint4 val = *(const uint4*)&half(c >> 6)[(c & 63) * 64 + ((ch ^ ((c >> 1) & 7)) << 3)];
        const uint32_t n = tc.n0 + c, m0 = wm0 + 8 * ch;
        if (n >= p.N || m0 >= p.M) continue;
        const uint32_t m2 = m0 - fdiv(m0, p.m2div) * p.M2;  // position within the M2 run
        uint16_t* dst = C + tc.c_base + row_off(p, m0, p.c_m1, p.c_m2) + (int32_t)n * p.c_n;
        if (m0 + 8 <= p.M && m2 + 8 <= p.M2 && ((uintptr_t)dst & 15u) == 0) {
          *(uint4*)dst = val;
        } else {
          const uint32_t w[4] = {val.x, val.y, val.z, val.w};
          for (int e = 0; e < 8 && m0 + e < p.M; ++e)
            C[tc.c_base + row_off(p, m0 + e, p.c_m1, p.c_m2) + (int32_t)n * p.c_n] = (uint16_t)(w[e / 2] >> (16 * (e & 1)));
        }
      }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const uint32_t n = tc.n0 + j * 32 + lr;
      if (n >= p.N) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const uint32_t m = wm0 + i * 32 + 8 * (v / 4) + 4 * lh + (v % 4);
        if (m < p.M) C[tc.c_base + row_off(p, m, p.c_m1, p.c_m2) + (int32_t)n * p.c_n] = f32_to_bf16(acc[i][j][v]);
      }
    }
}

hipError_t launch_gemm_bf16_dl(const NodeKernel& k, hipStream_t s) {
  const GemmParams& p = k.gemm;
  if (k.dtype != DT_BF16 || k.amode != GM_K || (k.bmode != GM_MN && k.bmode != GM_K)) return hipErrorInvalidValue;
  // a bias epilogue only: activations and the Add / Mul run as their own
  // kernels after these tiles
  if (p.rop || p.act) return hipErrorInvalidValue;
  const dim3 grid(p.tiles_m * p.tiles_n * p.G);
  // tile 8: the three-stage ring, two workgroups per CU
#define FLUID_DL(BMv, NSv) hipLaunchKernelGGL((gemm_bf16_dl_kernel<BMv, NSv>), grid, dim3(256), 0, s, p)
  if (k.gemm_tile == 8) {
    if (k.bmode == GM_MN) FLUID_DL(GM_MN, 3);
    else FLUID_DL(GM_K, 3);
  } else {
    if (k.bmode == GM_MN) FLUID_DL(GM_MN, 4);
    else FLUID_DL(GM_K, 4);
  }
#undef FLUID_DL
  return hipGetLastError();
}

}  // namespace fluid
