// Helpers shared by the GEMM kernels: tile coordinates, two-level row
// offsets, MFMA vector types.
#pragma once

#include "dev.h"

namespace fluid {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

struct TileCoord {
  uint32_t m0, n0;
  int32_t a_base, b_base, c_base, r_base;
};

// Buffer resource over [base, base + bytes).  A buffer load at a byte offset
// at or beyond `bytes` returns zeros without touching memory, so tile edges
// are padded by pointing the load at kOOB instead of branching around it
// (data format word as for every gfx9 target).
constexpr uint32_t kOOB = 0x80000000u;
typedef __amdgpu_buffer_rsrc_t Rsrc;
__device__ __forceinline__ Rsrc make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint4 bload16(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ uint2 bload8(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}
__device__ __forceinline__ uint16_t bload2(Rsrc r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}

// s_waitcnt immediate (gfx9 encoding) waiting until at most n vector-memory
// operations are outstanding; export and LDS counters left unconstrained.
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// Tile index -> (batch, tile row, tile column), row-major over tiles.
__device__ __forceinline__ TileCoord tile_coord_at(const GemmParams& p, uint32_t bid, uint32_t BM, uint32_t BN) {
  const uint32_t per_g = p.tiles_m * p.tiles_n;
  const uint32_t g = bid / per_g;
  const uint32_t r = bid - g * per_g;
  const uint32_t tm = r / p.tiles_n;
  const uint32_t tn = r - tm * p.tiles_n;
  const uint32_t g1 = fdiv(g, p.g2div);
  const uint32_t g2 = g - g1 * p.G2;
  TileCoord t;
  t.m0 = tm * BM;
  t.n0 = tn * BN;
  t.a_base = (int32_t)g1 * p.a_g1 + (int32_t)g2 * p.a_g2;
  t.b_base = (int32_t)g1 * p.b_g1 + (int32_t)g2 * p.b_g2;
  t.c_base = (int32_t)g1 * p.c_g1 + (int32_t)g2 * p.c_g2;
  t.r_base = (int32_t)g1 * p.r_g1 + (int32_t)g2 * p.r_g2;
  return t;
}
// One workgroup per tile.
__device__ __forceinline__ TileCoord tile_coord(const GemmParams& p, uint32_t BM, uint32_t BN) {
  return tile_coord_at(p, blockIdx.x, BM, BN);
}

// Offset of row m of A (or C) given the two-level row decomposition.
__device__ __forceinline__ int32_t row_off(const GemmParams& p, uint32_t m, int32_t s1, int32_t s2) {
  const uint32_t m1 = fdiv(m, p.m2div);
  return (int32_t)m1 * s1 + (int32_t)(m - m1 * p.M2) * s2;
}

// ---- epilogue: bias, activation, then the elementwise Add / Mul with R
// Offset of row m of R.  It splits m with R's own copy of the divisor: the
// compiler cannot share that split with the stores' (which would keep the
// split of every row of a tile live from the epilogue to the stores).
__device__ __forceinline__ int32_t r_row_off(const GemmParams& p, uint32_t m) {
  const uint32_t m1 = fdiv(m, p.r_m2div);
  return (int32_t)m1 * p.r_m1 + (int32_t)(m - m1 * p.r_m2div.d) * p.r_m2;
}
__device__ __forceinline__ float epi_load(const GemmParams& p, const void* base, int32_t off) {
  return p.epi_bf16 ? bf16_to_f32(((const uint16_t*)base)[off]) : ((const float*)base)[off];
}
__device__ __forceinline__ float epi_act(const GemmParams& p, float x) {
  if (p.act == 1) return gelu_erf(x);
  if (p.act == 2) return silu(x);
  return x;
}
__device__ __forceinline__ float epi_rop(const GemmParams& p, float x, float r) {
  return p.rop == 1 ? x + r : x * r;
}
// One output value at (m, n) of the batch whose R offset is r_base.  RES:
// the kernel instance that performs the Add / Mul with R (a separate
// instance, so that the others keep their register budget).
template <bool RES>
__device__ __forceinline__ float gemm_epi(const GemmParams& p, int32_t r_base, uint32_t m, uint32_t n, float v) {
  if (p.bias) v += epi_load(p, p.bias, (int32_t)n);
  v = epi_act(p, v);
  if (RES && m < p.M)
    v = epi_rop(p, v, epi_load(p, p.R, r_base + r_row_off(p, m) + (int32_t)n * p.r_n));
  return v;
}
// The 16 accumulators of a 32 x 32 MFMA block (the 32x32 output layout:
// value v of a lane sits at row m_first + 8 (v / 4) + v % 4 of column n).
// ACT false: an instance without the activation step.
template <bool RES, bool ACT = true>
__device__ __forceinline__ void epi16(const GemmParams& p, int32_t r_base, uint32_t m_first, uint32_t n,
                                      f32x16& v) {
  if ((p.bias || (ACT && p.act) || RES) && n < p.N) {
    const float b = p.bias ? epi_load(p, p.bias, (int32_t)n) : 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float x = ACT ? epi_act(p, v[i] + b) : v[i] + b;
      if (RES) {
        const uint32_t m = m_first + 8 * (i / 4) + (i % 4);
        if (m < p.M) x = epi_rop(p, x, epi_load(p, p.R, r_base + r_row_off(p, m) + (int32_t)n * p.r_n));
      }
      v[i] = x;
    }
  }
}


// Four rows of four bf16 (rows[t] = elements 0..3 at k + t) -> four rows of
// four k (out[j] = k .. k+3 of element j).
__device__ __forceinline__ void transpose4x4_b16(const uint2* rows, uint2* out) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint32_t e[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const uint32_t w = (j < 2) ? rows[t].x : rows[t].y;
      e[t] = (j & 1) ? (w >> 16) : (w & 0xffffu);
    }
    out[j] = make_uint2(e[0] | (e[1] << 16), e[2] | (e[3] << 16));
  }
}

// Writes the four transposed rows out[0..3] to LDS rows row0 .. row0+3
// (pitch kp elements) at column kcol.
__device__ __forceinline__ void store_rows4(uint16_t* lds, int row0, int kp, int kcol, const uint2* out) {
#pragma unroll
  for (int j = 0; j < 4; ++j) *(uint2*)&lds[(row0 + j) * kp + kcol] = out[j];
}

// Staging a 32-deep K-tile through LDS rows of pitch 40 elements (80 bytes).
// Thread index -> (row, k) of the piece a thread carries:
//  * K-contiguous operand, 16-byte pieces of 8 k: sixteen consecutive
//    threads take sixteen consecutive rows at one k, so the 16-byte LDS
//    writes of a wavefront hit every bank once (rows 80 bytes apart cover
//    all bank groups); a row's four pieces still come from one 64-byte span
//    of HBM within the same wavefront.
//  * M-/N-contiguous operand, 4 x 4 blocks: eight consecutive threads take
//    the eight k-groups of one 4-row block, so the 8-byte row writes after
//    the in-register transpose spread over all banks instead of landing
//    rows 4 x 80 bytes apart on the same few banks.
__device__ __forceinline__ void kpiece_coord(int idx, int& row, int& k) {
  row = (idx & 15) + 16 * (idx >> 6);
  k = ((idx >> 4) & 3) * 8;
}
__device__ __forceinline__ void mnblock_coord(int idx, int& row, int& k) {
  row = (idx >> 3) * 4;
  k = (idx & 7) * 4;
}

}  // namespace fluid
