// bf16 GEMM with a deep load pipeline (MFMA 32x32x16 bf16, fp32 accumulate).
//
// A bf16 MFMA is 16x faster per flop than an fp32 one, so one 32-wide K-tile
// of a 128 x 128 block is only ~0.1 us of matrix work: loads issued one tile
// ahead arrive after the MFMAs have drained.  Here loads run two K-tiles
// ahead (two register sets, the loop unrolled by two so that every register
// index is a compile-time constant), and LDS is double-buffered so that each
// K-tile costs one barrier.  Workgroup tile BM x 128 (BM = 256 or 128) with
// four wavefronts of (BM/2) x 64.  Operand layouts as in k_gemm.hip: LDS
// holds both operands K-contiguous; an M-/N-contiguous operand is transposed
// in 4 x 4 register blocks on its way into LDS.
#include "gemm_common.h"
#include "launch.h"

namespace fluid {

template <int BM, int AM, int BMD>
__global__ __launch_bounds__(256) void gemm_bf16_pipe_kernel(GemmParams p) {
  constexpr int BN = 128, BK = 32;
  constexpr int FM = BM / 64, FN = 2;  // per wavefront (BM/2) x 64
  constexpr int KP = BK + 8;           // LDS row pitch (elements)
  __shared__ uint16_t As[2 * BM * KP];
  __shared__ uint16_t Bs[2 * BN * KP];
  const TileCoord tc = tile_coord(p, BM, BN);
  // causal attention: a tile entirely above the diagonal is never read; a
  // row block's A is zero past its last row, so K stops there
  if ((p.causal & 1u) && tc.n0 > tc.m0 + BM - 1) return;
  const uint32_t Kc = (p.causal & 2u) ? min(p.K, tc.m0 + BM) : p.K;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const Rsrc ra = make_rsrc(p.A, p.a_bytes);
  const Rsrc rb = make_rsrc(p.B, p.b_bytes);

  // per-thread share of one K-tile: BM*32/256 elements of A, 16 of B
  constexpr int AE = BM * BK / 256;
  constexpr int AN = AM == GM_K ? AE / 8 : AM == GM_MN ? AE / 16 : AE;
  constexpr int BNN = BMD == GM_K ? 2 : BMD == GM_MN ? 1 : 16;
  int a_m[AN], a_k[AN];
  int32_t a_off[AN];
  bool a_ok[AN];
#pragma unroll
  for (int r = 0; r < AN; ++r) {
    const int idx = tid + 256 * r;
    if constexpr (AM == GM_K) kpiece_coord(idx, a_m[r], a_k[r]);
    else if constexpr (AM == GM_MN) mnblock_coord(idx, a_m[r], a_k[r]);
    else { a_k[r] = idx % BK; a_m[r] = idx / BK; }
    const uint32_t m = tc.m0 + a_m[r];
    a_ok[r] = m < p.M;
    a_off[r] = tc.a_base + (a_ok[r] ? row_off(p, m, p.a_m1, p.a_m2) : 0);
  }
  int b_n[BNN], b_k[BNN];
  int32_t b_off[BNN];
  bool b_ok[BNN];
#pragma unroll
  for (int r = 0; r < BNN; ++r) {
    const int idx = tid + 256 * r;
    if constexpr (BMD == GM_K) kpiece_coord(idx, b_n[r], b_k[r]);
    else if constexpr (BMD == GM_MN) mnblock_coord(idx, b_n[r], b_k[r]);
    else { b_k[r] = idx % BK; b_n[r] = idx / BK; }
    b_ok[r] = tc.n0 + b_n[r] < p.N;
    b_off[r] = tc.b_base + (int32_t)(tc.n0 + b_n[r]) * p.b_n;
  }

  // One register set holds one K-tile's share, whatever the load mode.
  struct Regs {
    uint4 ca[AM == GM_K ? AN : 1];
    uint2 ba[AM == GM_MN ? 4 * AN : 1];
    uint16_t sa[AM == GM_GENERIC ? AN : 1];
    uint4 cb[BMD == GM_K ? BNN : 1];
    uint2 bb[BMD == GM_MN ? 4 * BNN : 1];
    uint16_t sb[BMD == GM_GENERIC ? BNN : 1];
  };
  Regs R0, R1;

  // Loads never branch: a piece outside the matrix (row past M or N, k past
  // K) is read from kOOB and arrives as zeros.
  auto gload = [&](Regs& R, uint32_t k0) {
#pragma unroll
    for (int r = 0; r < AN; ++r) {
      if constexpr (AM == GM_K) {
        const uint32_t k = k0 + a_k[r];
        R.ca[r] = bload16(ra, (a_ok[r] && k < Kc) ? 2u * (uint32_t)(a_off[r] + (int32_t)k) : kOOB);
      } else if constexpr (AM == GM_MN) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const uint32_t k = k0 + a_k[r] + t;
          R.ba[4 * r + t] = bload8(ra, (a_ok[r] && k < Kc) ? 2u * (uint32_t)(a_off[r] + (int32_t)k * p.a_k) : kOOB);
        }
      } else {
        const uint32_t k = k0 + a_k[r];
        R.sa[r] = bload2(ra, (a_ok[r] && k < Kc) ? 2u * (uint32_t)(a_off[r] + (int32_t)k * p.a_k) : kOOB);
      }
    }
#pragma unroll
    for (int r = 0; r < BNN; ++r) {
      if constexpr (BMD == GM_K) {
        const uint32_t k = k0 + b_k[r];
        R.cb[r] = bload16(rb, (b_ok[r] && k < Kc) ? 2u * (uint32_t)(b_off[r] + (int32_t)k) : kOOB);
      } else if constexpr (BMD == GM_MN) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const uint32_t k = k0 + b_k[r] + t;
          R.bb[4 * r + t] = bload8(rb, (b_ok[r] && k < Kc) ? 2u * (uint32_t)(b_off[r] + (int32_t)k * p.b_k) : kOOB);
        }
      } else {
        const uint32_t k = k0 + b_k[r];
        R.sb[r] = bload2(rb, (b_ok[r] && k < Kc) ? 2u * (uint32_t)(b_off[r] + (int32_t)k * p.b_k) : kOOB);
      }
    }
  };
  auto lstore = [&](const Regs& R, int st) {
    uint16_t* as = As + st * BM * KP;
    uint16_t* bs = Bs + st * BN * KP;
#pragma unroll
    for (int r = 0; r < AN; ++r) {
      if constexpr (AM == GM_K) {
        *(uint4*)&as[a_m[r] * KP + a_k[r]] = R.ca[r];
      } else if constexpr (AM == GM_MN) {
        uint2 o[4];
        transpose4x4_b16(&R.ba[4 * r], o);
        store_rows4(as, a_m[r], KP, a_k[r], o);
      } else {
        as[a_m[r] * KP + a_k[r]] = R.sa[r];
      }
    }
#pragma unroll
    for (int r = 0; r < BNN; ++r) {
      if constexpr (BMD == GM_K) {
        *(uint4*)&bs[b_n[r] * KP + b_k[r]] = R.cb[r];
      } else if constexpr (BMD == GM_MN) {
        uint2 o[4];
        transpose4x4_b16(&R.bb[4 * r], o);
        store_rows4(bs, b_n[r], KP, b_k[r], o);
      } else {
        bs[b_n[r] * KP + b_k[r]] = R.sb[r];
      }
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int lr = lane & 31, lk = (lane >> 5) * 8;
  auto compute = [&](int st) {
    const uint16_t* as = As + st * BM * KP;
    const uint16_t* bs = Bs + st * BN * KP;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8 a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        a[i] = __builtin_bit_cast(bf16x8, *(const uint4*)&as[(wm * (BM / 2) + i * 32 + lr) * KP + kk + lk]);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        b[j] = __builtin_bit_cast(bf16x8, *(const uint4*)&bs[(wn * 64 + j * 32 + lr) * KP + kk + lk]);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  };

  // K-tile t lives in LDS stage t % 2; register set t % 2 carries it from
  // global memory, issued two tiles before it is stored.  Loads past the
  // last tile read zeros (k >= K) and are never stored, so the loop body
  // has no data-dependent branches and the memory counters stay exact.
  const uint32_t nt = (Kc + BK - 1) / BK;
  gload(R0, 0);
  gload(R1, BK);
  lstore(R0, 0);
  __syncthreads();
  gload(R0, 2 * BK);
  uint32_t t = 0;
  for (; t + 2 <= nt; t += 2) {
    compute(0);            // tile t
    lstore(R1, 1);         // tile t+1
    __syncthreads();
    gload(R1, (t + 3) * BK);
    compute(1);            // tile t+1
    lstore(R0, 0);         // tile t+2 (zeros past the end, never read)
    __syncthreads();
    gload(R0, (t + 4) * BK);
  }
  if (t < nt) compute(0);  // odd tile count: the last tile sits in stage 0

  uint16_t* C = (uint16_t*)p.C;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const uint32_t n = tc.n0 + wn * 64 + j * 32 + lr;
      epi16<false>(p, tc.r_base, tc.m0 + wm * (BM / 2) + i * 32 + 4 * (lane >> 5), n, acc[i][j]);
      if (n >= p.N) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const uint32_t m = tc.m0 + wm * (BM / 2) + i * 32 + 8 * (v / 4) + 4 * (lane >> 5) + (v % 4);
        if (m < p.M) C[tc.c_base + row_off(p, m, p.c_m1, p.c_m2) + (int32_t)n * p.c_n] = f32_to_bf16(acc[i][j][v]);
      }
    }
}

namespace {

template <int BM>
hipError_t pipe_go(const NodeKernel& k, hipStream_t s) {
  const GemmParams& p = k.gemm;
  if (p.rop) return hipErrorInvalidValue;  // the Add / Mul runs as its own kernel after these tiles
  const dim3 grid(p.tiles_m * p.tiles_n * p.G);
#define FLUID_PIPE(AMv, BMv) hipLaunchKernelGGL((gemm_bf16_pipe_kernel<BM, AMv, BMv>), grid, dim3(256), 0, s, p)
  if (k.amode == GM_K && k.bmode == GM_MN) FLUID_PIPE(GM_K, GM_MN);
  else if (k.amode == GM_K && k.bmode == GM_K) FLUID_PIPE(GM_K, GM_K);
  else if (k.amode == GM_K) FLUID_PIPE(GM_K, GM_GENERIC);
  else if (k.amode == GM_MN && k.bmode == GM_MN) FLUID_PIPE(GM_MN, GM_MN);
  else if (k.amode == GM_MN && k.bmode == GM_K) FLUID_PIPE(GM_MN, GM_K);
  else if (k.amode == GM_MN) FLUID_PIPE(GM_MN, GM_GENERIC);
  else if (k.bmode == GM_MN) FLUID_PIPE(GM_GENERIC, GM_MN);
  else if (k.bmode == GM_K) FLUID_PIPE(GM_GENERIC, GM_K);
  else FLUID_PIPE(GM_GENERIC, GM_GENERIC);
#undef FLUID_PIPE
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16_pipe(const NodeKernel& k, hipStream_t s) {
  if (k.dtype != DT_BF16) return hipErrorInvalidValue;
  if ((k.gemm_tile == 6 || k.gemm_tile == 8) && k.amode == GM_K && (k.bmode == GM_MN || k.bmode == GM_K))
    return launch_gemm_bf16_dl(k, s);
  if (k.gemm_tile == 9) return launch_gemm_bf16_qk(k, s);
  if (k.gemm_tile >= 8) return hipErrorInvalidValue;
  return k.gemm_tile == 6 ? pipe_go<256>(k, s) : pipe_go<128>(k, s);
}

}  // namespace fluid
