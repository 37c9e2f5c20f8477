// bf16 GEMM for a K-contiguous A and an N-contiguous B (the projection
// shape: activations times a row-major weight), MFMA 16x16x32 bf16 with fp32
// accumulate, written around two gfx950 features:
//
//  * A never passes through LDS.  The workgroup tile is 256 x 128 with four
//    wavefronts stacked along M, so each wavefront owns 64 rows of A and no
//    other wavefront needs them.  Lane l loads its MFMA operand (8
//    consecutive k of row l % 16) straight from HBM with one 16-byte buffer
//    load; the 16 x 32 operand shape puts four lanes on each row, so one
//    load instruction touches 16 rows of 64 bytes rather than 32 rows of 32.
//  * B goes from HBM to LDS by direct buffer loads (no registers, no VALU),
//    in its natural [k][n] form, and is read back with ds_read_b64_tr_b16,
//    which hands each lane four k-consecutive values of one column n.  Two
//    such reads make one 8-k MFMA operand.
//
// B lives in a four-stage LDS ring of 32 x 128 tiles; both operands are
// fetched three K-tiles ahead.  One barrier per K-tile: after a wavefront has
// waited for its own loads of tile t, the barrier makes every wavefront's
// part of tile t visible and frees the stage that tile t+3 overwrites.  The
// barrier is a bare s_barrier behind an explicit counter wait: a workgroup
// fence would wait for every load in flight, tiles t+1 and t+2 included.
//
// LDS tile rows are 256 bytes (128 bf16) with no padding.  The 16-byte
// chunk c of row r is stored at chunk c ^ (2 (r % 4) + 8 ((r / 8) % 2)): a
// transpose read by half a wavefront touches rows {0..3, 8..11} (+4 h) at
// the same two chunks, and the swizzle gives the eight rows eight different
// 32-byte bank groups.
#include "gemm_common.h"
#include "launch.h"

namespace fluid {

namespace {

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __attribute__((address_space(3))) void lds_void;

// s_waitcnt immediate (gfx9 encoding) waiting until at most n vector-memory
// operations are outstanding; export and LDS counters left unconstrained.
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

constexpr int DL_BM = 256, DL_BN = 128, DL_BK = 32, DL_NS = 4;
constexpr int DL_ROWB = DL_BN * 2;               // bytes per LDS row (one k)
constexpr int DL_STAGEB = DL_BK * DL_ROWB;       // 8 KiB per stage

}  // namespace

__global__ __launch_bounds__(256) void gemm_bf16_dl_kernel(GemmParams p) {
  constexpr int BK = DL_BK, NS = DL_NS;
  constexpr int FM = 4, FN = 8;  // wavefront tile 64 x 128 in 16 x 16 blocks
  // one LDS object per stage, so that the compiler can tell a DMA into one
  // stage from reads of another and does not wait for every load in flight
  __shared__ __attribute__((aligned(1024))) uint8_t Bs0[DL_STAGEB];
  __shared__ __attribute__((aligned(1024))) uint8_t Bs1[DL_STAGEB];
  __shared__ __attribute__((aligned(1024))) uint8_t Bs2[DL_STAGEB];
  __shared__ __attribute__((aligned(1024))) uint8_t Bs3[DL_STAGEB];
  auto stage = [&](int st) -> uint8_t* { return st == 0 ? Bs0 : st == 1 ? Bs1 : st == 2 ? Bs2 : Bs3; };
  const TileCoord tc = tile_coord(p, DL_BM, DL_BN);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: DMA base in M0
  const int lr = lane & 15, lq = lane >> 4;
  const Rsrc ra = make_rsrc(p.A, p.a_bytes);
  const Rsrc rb = make_rsrc(p.B, p.b_bytes);

  // Rows of A past M and columns of B past N only feed outputs that are
  // never stored, so they are clamped onto row / column 0 instead of being
  // masked; only k past K has to read as zero.
  // A: row of fragment i for this lane; 8 k at k0 + 8 lq
  int32_t a_row[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const uint32_t m = tc.m0 + wave * 64 + i * 16 + lr;
    a_row[i] = tc.a_base + (m < p.M ? row_off(p, m, p.a_m1, p.a_m2) : 0);
  }
  // B: each wavefront DMA instruction fills four 256-byte rows; lane l
  // writes chunk position l % 16 of row l / 16 of the instruction, which
  // holds the swizzled logical chunk of that row.  Round q covers rows
  // 16 q + 4 wave .. +3, so row % 4 = l / 16 and (row / 8) % 2 = wave / 2.
  const int b_rsub = lane >> 4;                               // row within the instruction
  const int b_chunk = (lane & 15) ^ (2 * b_rsub + 8 * (wave >> 1));  // logical 16-byte chunk
  const uint32_t b_n = tc.n0 + 8 * b_chunk;
  const int32_t b_col = tc.b_base + (int32_t)(b_n < p.N ? b_n : 0);

  auto load_a = [&](uint4 (&R)[FM], uint32_t k0) {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const uint32_t k = k0 + 8 * lq;
      R[i] = bload16(ra, k < p.K ? 2u * (uint32_t)(a_row[i] + (int32_t)k) : kOOB);
    }
  };
  auto load_b = [&](int st, uint32_t k0) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int row = 16 * q + 4 * wave + b_rsub;
      const uint32_t k = k0 + row;
      const uint32_t off = k < p.K ? 2u * (uint32_t)(b_col + (int32_t)k * p.b_k) : kOOB;
      lds_void* dst = (lds_void*)(stage(st) + (16 * q + 4 * wave) * DL_ROWB);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, dst, 16, off, 0, 0, 0);
    }
  };

  // transpose-read addressing: lane l (group g = l / 16, s = l % 16) points
  // at row 8 g + 4 h + s / 4 of the tile, columns 16 j + 4 (s % 4) .. +3;
  // the read returns column 16 j + l % 16, rows 8 (l / 16) + 4 h .. +3,
  // which is half of the lane's MFMA operand.
  const int tg = lane >> 4, ts = lane & 15;
  const int t_row = 8 * tg + (ts >> 2);                        // + 4 h
  const int t_col = 4 * (ts & 3);                              // + 16 j (elements)
  auto b_addr = [&](int st, int h, int j) {
    const int row = 4 * h + t_row;
    const int col = 16 * j + t_col;
    const int chunk = (col >> 3) ^ (2 * (row & 3) + 8 * ((row >> 3) & 1));
    return (lds_v4i16*)(stage(st) + row * DL_ROWB + chunk * 16 + (col & 7) * 2);
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[i][j][v] = 0.f;

  auto compute = [&](int st, const uint4 (&R)[FM]) {
    bf16x8 b[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(b_addr(st, 0, j));
      const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(b_addr(st, 1, j));
      b[j] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const bf16x8 a = __builtin_bit_cast(bf16x8, R[i]);
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[j], acc[i][j], 0, 0, 0);
    }
  };

  // Tile t: A in register set t % 4, B in stage t % 4.  Loads are issued in
  // the order A(t), B(t) and past the end of K they read zeros, so the loop
  // runs whole groups of four tiles and skips the MFMAs of the padding.
  const uint32_t nt = (p.K + BK - 1) / BK;
  uint4 RA0[FM], RA1[FM], RA2[FM], RA3[FM];
  load_a(RA0, 0);
  load_b(0, 0);
  load_a(RA1, BK);
  load_b(1, BK);
  load_a(RA2, 2 * BK);
  load_b(2, 2 * BK);
  // After the loads of tile t, tiles t+1 and t+2 (2 x (FM + 2) loads) may
  // still be in flight.
  constexpr int kAhead = 2 * (FM + 2);
  for (uint32_t t = 0; t < nt; t += 4) {
#define FLUID_DL_STEP(U, RCUR, RNEXT)                                \
  asm volatile("" ::: "memory");                                     \
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(kAhead));                     \
  __builtin_amdgcn_s_barrier();                                      \
  asm volatile("" ::: "memory");                                     \
  load_a(RNEXT, (t + U + 3) * BK);                                   \
  load_b((U + 3) % NS, (t + U + 3) * BK);                            \
  if (t + U < nt) compute(U, RCUR);
    FLUID_DL_STEP(0, RA0, RA3)
    FLUID_DL_STEP(1, RA1, RA0)
    FLUID_DL_STEP(2, RA2, RA1)
    FLUID_DL_STEP(3, RA3, RA2)
#undef FLUID_DL_STEP
  }

  uint16_t* C = (uint16_t*)p.C;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const uint32_t n = tc.n0 + j * 16 + lr;
      if (n >= p.N) continue;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const uint32_t m = tc.m0 + wave * 64 + i * 16 + 4 * lq + v;
        if (m < p.M) C[tc.c_base + row_off(p, m, p.c_m1, p.c_m2) + (int32_t)n * p.c_n] = f32_to_bf16(acc[i][j][v]);
      }
    }
}

hipError_t launch_gemm_bf16_dl(const NodeKernel& k, hipStream_t s) {
  const GemmParams& p = k.gemm;
  if (k.dtype != DT_BF16 || k.amode != GM_K || k.bmode != GM_MN) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gemm_bf16_dl_kernel, dim3(p.tiles_m * p.tiles_n * p.G), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace fluid
