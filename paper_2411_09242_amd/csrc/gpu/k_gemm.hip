// Permuted-stride batched GEMM on MFMA (gfx950).
//
//   C[g, m, n] = sum_k A[g, m, k] * B[g, k, n]
//
// Every operand is addressed through its own strides, so any layout the
// planner picks for A, B or C runs without a relayout copy.  A block of 256
// threads (4 wavefronts, 2 x 2) computes a BM x BN tile; operand tiles are
// staged through LDS, where they are stored in the orientation the MFMA
// fragments read, whichever dim is unit-stride in HBM:
//   A: K-contiguous ("k") or M-contiguous ("mn") 16-byte loads, else scalar
//   B: N-contiguous ("mn") or K-contiguous ("k") 16-byte loads, else scalar
//   C: N-contiguous stores, M-contiguous 4-row stores, else scalar.
// fp32 uses v_mfma_f32_32x32x2_f32 (lane l: A[l%32][l/32], B[l/32][l%32]);
// bf16 uses v_mfma_f32_32x32x16_bf16 (lane l: 8 consecutive k of row l%32,
// k-group l/32) with fp32 accumulation.  Accumulator v of lane l holds
// C[8(v/4) + 4(l/32) + v%4][l%32].  The next K-tile is loaded into
// registers while the current one is multiplied.
#include "gemm_common.h"
#include "launch.h"

namespace fluid {

// ============================================================== fp32
// The register budget of four wavefronts per SIMD: four 128 x 128
// workgroups share a compute unit (without it the compiler's 139 registers
// left room for three, and a 1024-tile launch ran a second, quarter-full
// round).
template <int BM, int BN, int AM, int BMD, bool RES>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void gemm_f32_kernel(GemmParams p) {
  constexpr int BK = 16;
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int AP = BM + 4, BP = BN + 4;
  __shared__ float As[BK * AP];
  __shared__ float Bs[BK * BP];
  const TileCoord tc = tile_coord(p, BM, BN);
  // causal attention: a tile entirely above the diagonal is never read; a
  // row block's A is zero past its last row, so K stops there
  if ((p.causal & 1u) && tc.n0 > tc.m0 + BM - 1) return;
  const uint32_t Kc = (p.causal & 2u) ? min(p.K, tc.m0 + BM) : p.K;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // ---- per-thread load plan (rows are fixed across K-tiles)
  constexpr int A_ELEMS = BM * BK / 256;  // 8 or 4
  constexpr int A_VECS = A_ELEMS / 4;
  constexpr int B_ELEMS = BN * BK / 256;
  constexpr int B_VECS = B_ELEMS / 4;
  int32_t a_off[A_ELEMS];
  bool a_ok[A_ELEMS];
  int a_m[A_ELEMS], a_k[A_ELEMS];
  if constexpr (AM == GM_K) {
#pragma unroll
    for (int r = 0; r < A_VECS; ++r) {
      const int idx = tid + 256 * r;
      a_m[r] = idx / (BK / 4);
      a_k[r] = (idx % (BK / 4)) * 4;
      const uint32_t m = tc.m0 + a_m[r];
      a_ok[r] = m < p.M;
      a_off[r] = tc.a_base + (a_ok[r] ? row_off(p, m, p.a_m1, p.a_m2) : 0);
    }
  } else if constexpr (AM == GM_MN) {
#pragma unroll
    for (int r = 0; r < A_VECS; ++r) {
      const int idx = tid + 256 * r;
      a_k[r] = idx / (BM / 4);
      a_m[r] = (idx % (BM / 4)) * 4;
      const uint32_t m = tc.m0 + a_m[r];
      a_ok[r] = m < p.M;
      a_off[r] = tc.a_base + (a_ok[r] ? row_off(p, m, p.a_m1, p.a_m2) : 0);
    }
  } else {
#pragma unroll
    for (int r = 0; r < A_ELEMS; ++r) {
      const int idx = tid + 256 * r;
      a_m[r] = idx % BM;
      a_k[r] = idx / BM;
      const uint32_t m = tc.m0 + a_m[r];
      a_ok[r] = m < p.M;
      a_off[r] = tc.a_base + (a_ok[r] ? row_off(p, m, p.a_m1, p.a_m2) : 0);
    }
  }
  int b_k[B_ELEMS], b_n[B_ELEMS];
  bool b_ok[B_ELEMS];
  if constexpr (BMD == GM_MN) {
#pragma unroll
    for (int r = 0; r < B_VECS; ++r) {
      const int idx = tid + 256 * r;
      b_k[r] = idx / (BN / 4);
      b_n[r] = (idx % (BN / 4)) * 4;
      b_ok[r] = tc.n0 + b_n[r] < p.N;
    }
  } else if constexpr (BMD == GM_K) {
#pragma unroll
    for (int r = 0; r < B_VECS; ++r) {
      const int idx = tid + 256 * r;
      b_n[r] = idx / (BK / 4);
      b_k[r] = (idx % (BK / 4)) * 4;
      b_ok[r] = tc.n0 + b_n[r] < p.N;
    }
  } else {
#pragma unroll
    for (int r = 0; r < B_ELEMS; ++r) {
      const int idx = tid + 256 * r;
      b_n[r] = idx % BN;
      b_k[r] = idx / BN;
      b_ok[r] = tc.n0 + b_n[r] < p.N;
    }
  }

  float ra[A_ELEMS], rb[B_ELEMS];
  const float* A = (const float*)p.A;
  const float* B = (const float*)p.B;
  auto gload = [&](uint32_t k0) {
    if constexpr (AM == GM_K) {
#pragma unroll
      for (int r = 0; r < A_VECS; ++r) {
        const uint32_t k = k0 + a_k[r];
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (a_ok[r] && k < Kc) v = *(const float4*)(A + a_off[r] + (int32_t)k);
        ra[4 * r] = v.x; ra[4 * r + 1] = v.y; ra[4 * r + 2] = v.z; ra[4 * r + 3] = v.w;
      }
    } else if constexpr (AM == GM_MN) {
#pragma unroll
      for (int r = 0; r < A_VECS; ++r) {
        const uint32_t k = k0 + a_k[r];
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (a_ok[r] && k < Kc) v = *(const float4*)(A + a_off[r] + (int32_t)k * p.a_k);
        ra[4 * r] = v.x; ra[4 * r + 1] = v.y; ra[4 * r + 2] = v.z; ra[4 * r + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int r = 0; r < A_ELEMS; ++r) {
        const uint32_t k = k0 + a_k[r];
        ra[r] = (a_ok[r] && k < Kc) ? A[a_off[r] + (int32_t)k * p.a_k] : 0.f;
      }
    }
    if constexpr (BMD == GM_MN) {
#pragma unroll
      for (int r = 0; r < B_VECS; ++r) {
        const uint32_t k = k0 + b_k[r];
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (b_ok[r] && k < Kc) v = *(const float4*)(B + tc.b_base + (int32_t)k * p.b_k + (int32_t)(tc.n0 + b_n[r]));
        rb[4 * r] = v.x; rb[4 * r + 1] = v.y; rb[4 * r + 2] = v.z; rb[4 * r + 3] = v.w;
      }
    } else if constexpr (BMD == GM_K) {
#pragma unroll
      for (int r = 0; r < B_VECS; ++r) {
        const uint32_t k = k0 + b_k[r];
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (b_ok[r] && k < Kc) v = *(const float4*)(B + tc.b_base + (int32_t)k + (int32_t)(tc.n0 + b_n[r]) * p.b_n);
        rb[4 * r] = v.x; rb[4 * r + 1] = v.y; rb[4 * r + 2] = v.z; rb[4 * r + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int r = 0; r < B_ELEMS; ++r) {
        const uint32_t k = k0 + b_k[r];
        rb[r] = (b_ok[r] && k < Kc) ? B[tc.b_base + (int32_t)k * p.b_k + (int32_t)(tc.n0 + b_n[r]) * p.b_n] : 0.f;
      }
    }
  };
  auto lstore = [&]() {
    if constexpr (AM == GM_K) {
#pragma unroll
      for (int r = 0; r < A_VECS; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j) As[(a_k[r] + j) * AP + a_m[r]] = ra[4 * r + j];
    } else if constexpr (AM == GM_MN) {
#pragma unroll
      for (int r = 0; r < A_VECS; ++r)
        *(float4*)&As[a_k[r] * AP + a_m[r]] = make_float4(ra[4 * r], ra[4 * r + 1], ra[4 * r + 2], ra[4 * r + 3]);
    } else {
#pragma unroll
      for (int r = 0; r < A_ELEMS; ++r) As[a_k[r] * AP + a_m[r]] = ra[r];
    }
    if constexpr (BMD == GM_MN) {
#pragma unroll
      for (int r = 0; r < B_VECS; ++r)
        *(float4*)&Bs[b_k[r] * BP + b_n[r]] = make_float4(rb[4 * r], rb[4 * r + 1], rb[4 * r + 2], rb[4 * r + 3]);
    } else if constexpr (BMD == GM_K) {
#pragma unroll
      for (int r = 0; r < B_VECS; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j) Bs[(b_k[r] + j) * BP + b_n[r]] = rb[4 * r + j];
    } else {
#pragma unroll
      for (int r = 0; r < B_ELEMS; ++r) Bs[b_k[r] * BP + b_n[r]] = rb[r];
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int lr = lane & 31, lk = lane >> 5;
  gload(0);
  for (uint32_t k0 = 0; k0 < Kc; k0 += BK) {
    __syncthreads();
    lstore();
    __syncthreads();
    if (k0 + BK < Kc) gload(k0 + BK);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 2) {
      float a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) a[i] = As[(kk + lk) * AP + wm * WM + i * 32 + lr];
#pragma unroll
      for (int j = 0; j < FN; ++j) b[j] = Bs[(kk + lk) * BP + wn * WN + j * 32 + lr];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }

  // ---- epilogue
  float* C = (float*)p.C;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
      epi16<RES>(p, tc.r_base, tc.m0 + wm * WM + i * 32 + 4 * lk, tc.n0 + wn * WN + j * 32 + lr, acc[i][j]);
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const uint32_t n = tc.n0 + wn * WN + j * 32 + lr;
#pragma unroll
      for (int vg = 0; vg < 4; ++vg) {
        const uint32_t mb = tc.m0 + wm * WM + i * 32 + 8 * vg + 4 * lk;
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

// ============================================================== bf16
// LDS holds both operands K-contiguous ([row][k], k fastest) so that each
// lane fetches its 8 bf16 MFMA inputs with one 16-byte LDS read.  An
// M-/N-contiguous HBM operand is transposed on the way in: each thread loads
// a 4(k) x 4(m|n) block with four 8-byte loads and writes four 8-byte rows.
template <int BM, int BN, int AM, int BMD, bool RES>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmParams p) {
  constexpr int BK = 32;
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int KP = BK + 8;  // padded row pitch (elements)
  __shared__ uint16_t As[BM * KP];
  __shared__ uint16_t Bs[BN * KP];
  const TileCoord tc = tile_coord(p, BM, BN);
  // causal attention: a tile entirely above the diagonal is never read; a
  // row block's A is zero past its last row, so K stops there
  if ((p.causal & 1u) && tc.n0 > tc.m0 + BM - 1) return;
  const uint32_t Kc = (p.causal & 2u) ? min(p.K, tc.m0 + BM) : p.K;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const uint16_t* A = (const uint16_t*)p.A;
  const uint16_t* B = (const uint16_t*)p.B;

  // A plan
  constexpr int A_ELEMS = BM * BK / 256;  // 16 or 8
  constexpr int A_CH = A_ELEMS / 8;       // 16-byte chunks (K mode)
  constexpr int A_BL = A_ELEMS / 16;      // 4x4 blocks (MN mode), may be 0
  int a_m[A_ELEMS], a_k[A_ELEMS];
  int32_t a_off[A_ELEMS];
  bool a_ok[A_ELEMS];
  if constexpr (AM == GM_K) {
#pragma unroll
    for (int r = 0; r < A_CH; ++r) {
      const int idx = tid + 256 * r;
      kpiece_coord(idx, a_m[r], a_k[r]);
      const uint32_t m = tc.m0 + a_m[r];
      a_ok[r] = m < p.M;
      a_off[r] = tc.a_base + (a_ok[r] ? row_off(p, m, p.a_m1, p.a_m2) : 0);
    }
  } else if constexpr (AM == GM_MN && A_BL > 0) {
#pragma unroll
    for (int r = 0; r < A_BL; ++r) {
      const int idx = tid + 256 * r;
      mnblock_coord(idx, a_m[r], a_k[r]);
      const uint32_t m = tc.m0 + a_m[r];
      a_ok[r] = m < p.M;
      a_off[r] = tc.a_base + (a_ok[r] ? row_off(p, m, p.a_m1, p.a_m2) : 0);
    }
  } else {
#pragma unroll
    for (int r = 0; r < A_ELEMS; ++r) {
      const int idx = tid + 256 * r;
      a_k[r] = idx % BK;
      a_m[r] = idx / BK;
      const uint32_t m = tc.m0 + a_m[r];
      a_ok[r] = m < p.M;
      a_off[r] = tc.a_base + (a_ok[r] ? row_off(p, m, p.a_m1, p.a_m2) : 0);
    }
  }
  constexpr int B_ELEMS = BN * BK / 256;
  constexpr int B_CH = B_ELEMS / 8;
  constexpr int B_BL = B_ELEMS / 16;
  int b_n[B_ELEMS], b_k[B_ELEMS];
  bool b_ok[B_ELEMS];
  if constexpr (BMD == GM_K) {
#pragma unroll
    for (int r = 0; r < B_CH; ++r) {
      const int idx = tid + 256 * r;
      kpiece_coord(idx, b_n[r], b_k[r]);
      b_ok[r] = tc.n0 + b_n[r] < p.N;
    }
  } else if constexpr (BMD == GM_MN && B_BL > 0) {
#pragma unroll
    for (int r = 0; r < B_BL; ++r) {
      const int idx = tid + 256 * r;
      mnblock_coord(idx, b_n[r], b_k[r]);
      b_ok[r] = tc.n0 + b_n[r] < p.N;
    }
  } else {
#pragma unroll
    for (int r = 0; r < B_ELEMS; ++r) {
      const int idx = tid + 256 * r;
      b_k[r] = idx % BK;
      b_n[r] = idx / BK;
      b_ok[r] = tc.n0 + b_n[r] < p.N;
    }
  }
  constexpr bool A_VEC_K = AM == GM_K;
  constexpr bool A_VEC_MN = AM == GM_MN && A_BL > 0;
  constexpr bool B_VEC_K = BMD == GM_K;
  constexpr bool B_VEC_MN = BMD == GM_MN && B_BL > 0;

  uint4 ca[A_CH > 0 ? A_CH : 1];
  uint2 ba[A_BL > 0 ? A_BL * 4 : 1];
  uint16_t sa[A_ELEMS];
  uint4 cb[B_CH > 0 ? B_CH : 1];
  uint2 bb[B_BL > 0 ? B_BL * 4 : 1];
  uint16_t sb[B_ELEMS];

  auto gload = [&](uint32_t k0) {
    if constexpr (A_VEC_K) {
#pragma unroll
      for (int r = 0; r < A_CH; ++r) {
        const uint32_t k = k0 + a_k[r];
        ca[r] = (a_ok[r] && k < Kc) ? *(const uint4*)(A + a_off[r] + (int32_t)k) : make_uint4(0, 0, 0, 0);
      }
    } else if constexpr (A_VEC_MN) {
#pragma unroll
      for (int r = 0; r < A_BL; ++r)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const uint32_t k = k0 + a_k[r] + t;
          ba[4 * r + t] = (a_ok[r] && k < Kc) ? *(const uint2*)(A + a_off[r] + (int32_t)k * p.a_k) : make_uint2(0, 0);
        }
    } else {
#pragma unroll
      for (int r = 0; r < A_ELEMS; ++r) {
        const uint32_t k = k0 + a_k[r];
        sa[r] = (a_ok[r] && k < Kc) ? A[a_off[r] + (int32_t)k * p.a_k] : (uint16_t)0;
      }
    }
    if constexpr (B_VEC_K) {
#pragma unroll
      for (int r = 0; r < B_CH; ++r) {
        const uint32_t k = k0 + b_k[r];
        cb[r] = (b_ok[r] && k < Kc) ? *(const uint4*)(B + tc.b_base + (int32_t)k + (int32_t)(tc.n0 + b_n[r]) * p.b_n)
                                     : make_uint4(0, 0, 0, 0);
      }
    } else if constexpr (B_VEC_MN) {
#pragma unroll
      for (int r = 0; r < B_BL; ++r)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const uint32_t k = k0 + b_k[r] + t;
          bb[4 * r + t] = (b_ok[r] && k < Kc)
                              ? *(const uint2*)(B + tc.b_base + (int32_t)k * p.b_k + (int32_t)(tc.n0 + b_n[r]))
                              : make_uint2(0, 0);
        }
    } else {
#pragma unroll
      for (int r = 0; r < B_ELEMS; ++r) {
        const uint32_t k = k0 + b_k[r];
        sb[r] = (b_ok[r] && k < Kc) ? B[tc.b_base + (int32_t)k * p.b_k + (int32_t)(tc.n0 + b_n[r]) * p.b_n] : (uint16_t)0;
      }
    }
  };
  auto lstore = [&]() {
    if constexpr (A_VEC_K) {
#pragma unroll
      for (int r = 0; r < A_CH; ++r) *(uint4*)&As[a_m[r] * KP + a_k[r]] = ca[r];
    } else if constexpr (A_VEC_MN) {
#pragma unroll
      for (int r = 0; r < A_BL; ++r) {
        uint2 o[4];
        transpose4x4_b16(&ba[4 * r], o);
        store_rows4(As, a_m[r], KP, a_k[r], o);
      }
    } else {
#pragma unroll
      for (int r = 0; r < A_ELEMS; ++r) As[a_m[r] * KP + a_k[r]] = sa[r];
    }
    if constexpr (B_VEC_K) {
#pragma unroll
      for (int r = 0; r < B_CH; ++r) *(uint4*)&Bs[b_n[r] * KP + b_k[r]] = cb[r];
    } else if constexpr (B_VEC_MN) {
#pragma unroll
      for (int r = 0; r < B_BL; ++r) {
        uint2 o[4];
        transpose4x4_b16(&bb[4 * r], o);
        store_rows4(Bs, b_n[r], KP, b_k[r], o);
      }
    } else {
#pragma unroll
      for (int r = 0; r < B_ELEMS; ++r) Bs[b_n[r] * KP + b_k[r]] = sb[r];
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
  gload(0);
  for (uint32_t k0 = 0; k0 < Kc; k0 += BK) {
    __syncthreads();
    lstore();
    __syncthreads();
    if (k0 + BK < Kc) gload(k0 + BK);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8 a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        uint4 q = *(const uint4*)&As[(wm * WM + i * 32 + lr) * KP + kk + lk];
        a[i] = __builtin_bit_cast(bf16x8, q);
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        uint4 q = *(const uint4*)&Bs[(wn * WN + j * 32 + lr) * KP + kk + lk];
        b[j] = __builtin_bit_cast(bf16x8, q);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }

  uint16_t* C = (uint16_t*)p.C;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const uint32_t n = tc.n0 + wn * WN + j * 32 + lr;
      epi16<RES>(p, tc.r_base, tc.m0 + wm * WM + i * 32 + 4 * (lane >> 5), n, acc[i][j]);
      if (n >= p.N) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const uint32_t m = tc.m0 + wm * WM + i * 32 + 8 * (v / 4) + 4 * (lane >> 5) + (v % 4);
        if (m < p.M) C[tc.c_base + row_off(p, m, p.c_m1, p.c_m2) + (int32_t)n * p.c_n] = f32_to_bf16(acc[i][j][v]);
      }
    }
}

// (the large-tile, deeply pipelined bf16 kernel lives in k_gemm_bf16.hip)

// ============================================================== split-K
// For GEMMs with few output tiles (a 128-token batch gives 24 tiles of
// 64x64 for a 768-wide projection): W wavefronts of one workgroup share one
// (32 FM) x (32 FN) output tile and each takes a contiguous 1/W of the K
// range; partial tiles are summed through LDS at the end (no workspace, no
// atomics).  Operands go straight from global memory into MFMA registers:
// within each 16-wide K step, lane group h = lane / 32 owns k0 + 8h .. k0 +
// 8h + 7 (any pairing of k between A and B is valid as long as both use it),
// so a K-contiguous operand is two 16-byte loads (fp32) or one (bf16) per
// lane, and an M- or N-contiguous operand is a coalesced 32-lane row access.
// Each iteration covers U such steps and the next iteration's loads are
// issued before the current MFMAs (ping-pong registers with compile-time
// indices), so 2 x 16U K-values per wavefront are in flight.
template <typename T, int FM, int FN, int W, int U, bool AVK, bool BVK, bool RES>
__global__ __launch_bounds__(64 * W) void gemm_sk_kernel(GemmParams p) {
  constexpr int TM = 32 * FM, TN = 32 * FN, RP = TN + 1;
  constexpr int KI = 16 * U;  // K values per iteration
  constexpr bool BF = sizeof(T) == 2;
  __shared__ float red[W * TM * RP];
  const TileCoord tc = tile_coord(p, TM, TN);
  // causal attention: a tile entirely above the diagonal is never read; a
  // row block's A is zero past its last row, so K stops there
  if ((p.causal & 1u) && tc.n0 > tc.m0 + TM - 1) return;
  const uint32_t Kc = (p.causal & 2u) ? min(p.K, tc.m0 + TM) : p.K;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int h = lane >> 5, r = lane & 31;
  const T* A = (const T*)p.A;
  const T* B = (const T*)p.B;
  // K slice of this wavefront (multiple of 16 wide)
  const uint32_t kc = ((Kc + W - 1) / W + 15u) & ~15u;
  const uint32_t kb = (uint32_t)w * kc;
  const uint32_t ke = min(Kc, kb + kc);
  int32_t arow[FM];
  bool aok[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const uint32_t m = tc.m0 + 32 * i + r;
    aok[i] = m < p.M;
    arow[i] = tc.a_base + (aok[i] ? row_off(p, m, p.a_m1, p.a_m2) : 0);
  }
  int32_t bcol[FN];
  bool bok[FN];
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const uint32_t n = tc.n0 + 32 * j + r;
    bok[j] = n < p.N;
    bcol[j] = tc.b_base + (bok[j] ? (int32_t)n * p.b_n : 0);
  }
  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  float fa0[FM][U][8], fb0[FN][U][8], fa1[FM][U][8], fb1[FN][U][8];
  auto load = [&](float (&fa)[FM][U][8], float (&fb)[FN][U][8], uint32_t k0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t kg = k0 + 16u * u + 8u * h;  // first k of this lane group
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        if constexpr (AVK && !BF) {
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (aok[i] && kg + 4u * q < ke) v = *(const float4*)((const float*)A + arow[i] + (int32_t)(kg + 4u * q));
            fa[i][u][4 * q] = v.x; fa[i][u][4 * q + 1] = v.y; fa[i][u][4 * q + 2] = v.z; fa[i][u][4 * q + 3] = v.w;
          }
        } else if constexpr (AVK && BF) {
          uint4 v = make_uint4(0, 0, 0, 0);
          if (aok[i] && kg < ke) v = *(const uint4*)((const uint16_t*)A + arow[i] + (int32_t)kg);
          const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            fa[i][u][2 * q] = __uint_as_float(wv[q] << 16);
            fa[i][u][2 * q + 1] = __uint_as_float(wv[q] & 0xffff0000u);
          }
        } else {
#pragma unroll
          for (int s = 0; s < 8; ++s) {
            const uint32_t k = kg + s;
            fa[i][u][s] = (aok[i] && k < ke) ? Elem<T>::load(A, arow[i] + (int32_t)k * p.a_k) : 0.f;
          }
        }
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        if constexpr (BVK && !BF) {
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (bok[j] && kg + 4u * q < ke) v = *(const float4*)((const float*)B + bcol[j] + (int32_t)(kg + 4u * q));
            fb[j][u][4 * q] = v.x; fb[j][u][4 * q + 1] = v.y; fb[j][u][4 * q + 2] = v.z; fb[j][u][4 * q + 3] = v.w;
          }
        } else if constexpr (BVK && BF) {
          uint4 v = make_uint4(0, 0, 0, 0);
          if (bok[j] && kg < ke) v = *(const uint4*)((const uint16_t*)B + bcol[j] + (int32_t)kg);
          const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            fb[j][u][2 * q] = __uint_as_float(wv[q] << 16);
            fb[j][u][2 * q + 1] = __uint_as_float(wv[q] & 0xffff0000u);
          }
        } else {
#pragma unroll
          for (int s = 0; s < 8; ++s) {
            const uint32_t k = kg + s;
            fb[j][u][s] = (bok[j] && k < ke) ? Elem<T>::load(B, bcol[j] + (int32_t)k * p.b_k) : 0.f;
          }
        }
      }
    }
  };
  auto compute = [&](const float (&fa)[FM][U][8], const float (&fb)[FN][U][8]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if constexpr (BF) {
        bf16x8 av[FM], bv[FN];
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int s = 0; s < 8; ++s) av[i][s] = (__bf16)fa[i][u][s];
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int s = 0; s < 8; ++s) bv[j][s] = (__bf16)fb[j][u][s];
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
      } else {
#pragma unroll
        for (int s = 0; s < 8; ++s)
#pragma unroll
          for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[i][u][s], fb[j][u][s], acc[i][j], 0, 0, 0);
      }
    }
  };
  if (kb < ke) {
    load(fa0, fb0, kb);
    for (uint32_t k0 = kb;;) {
      if (k0 + KI < ke) load(fa1, fb1, k0 + KI);
      compute(fa0, fb0);
      k0 += KI;
      if (k0 >= ke) break;
      if (k0 + KI < ke) load(fa0, fb0, k0 + KI);
      compute(fa1, fb1);
      k0 += KI;
      if (k0 >= ke) break;
    }
  }
  // partial tiles -> LDS, then each thread sums W partials for its outputs
  float* mine = red + w * TM * RP;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = 32 * i + 8 * (v / 4) + 4 * h + (v % 4);
        mine[m * RP + 32 * j + r] = acc[i][j][v];
      }
  __syncthreads();
  const bool ncontig = p.c_n == 1;
  for (int e = tid; e < TM * TN; e += 64 * W) {
    const int ml = ncontig ? e / TN : e % TM;
    const int nl = ncontig ? e % TN : e / TM;
    const uint32_t m = tc.m0 + ml, n = tc.n0 + nl;
    if (m >= p.M || n >= p.N) continue;
    float sum = 0.f;
#pragma unroll
    for (int q = 0; q < W; ++q) sum += red[q * TM * RP + ml * RP + nl];
    sum = gemm_epi<RES>(p, tc.r_base, m, n, sum);
    Elem<T>::store(p.C, tc.c_base + row_off(p, m, p.c_m1, p.c_m2) + (int32_t)n * p.c_n, sum);
  }
}

namespace {

template <typename T, int FM, int FN, int W, int U>
hipError_t gemm_sk_go(const NodeKernel& k, hipStream_t s) {
  const GemmParams& p = k.gemm;
  const dim3 grid(p.tiles_m * p.tiles_n * p.G);
  const bool avk = k.amode == GM_K, bvk = k.bmode == GM_K;
#define FLUID_SK(AV, BV)                                                                         \
  do {                                                                                           \
    if (p.rop) hipLaunchKernelGGL((gemm_sk_kernel<T, FM, FN, W, U, AV, BV, true>), grid, dim3(64 * W), 0, s, p); \
    else hipLaunchKernelGGL((gemm_sk_kernel<T, FM, FN, W, U, AV, BV, false>), grid, dim3(64 * W), 0, s, p);      \
  } while (0)
  if (avk && bvk) FLUID_SK(true, true);
  else if (avk) FLUID_SK(true, false);
  else if (bvk) FLUID_SK(false, true);
  else FLUID_SK(false, false);
#undef FLUID_SK
  return hipGetLastError();
}

template <typename T>
hipError_t gemm_sk_dispatch(const NodeKernel& k, hipStream_t s) {
  switch (k.gemm_tile) {
    case 2: return gemm_sk_go<T, 1, 1, 4, 4>(k, s);
    case 3: return gemm_sk_go<T, 1, 1, 8, 4>(k, s);
    case 4: return gemm_sk_go<T, 2, 1, 4, 2>(k, s);
    default: return gemm_sk_go<T, 1, 1, 16, 2>(k, s);
  }
}


template <int T, int AM, int BMD>
hipError_t gemm_go(const NodeKernel& k, hipStream_t s) {
  const GemmParams& p = k.gemm;
  const dim3 grid(p.tiles_m * p.tiles_n * p.G);
  // the 128 x 128 tiles leave an Add / Mul to its own kernel (an instance
  // with it would lose a workgroup per SIMD)
  constexpr bool kRes = T != 128;
  if (p.rop && !kRes) return hipErrorInvalidValue;
  if (k.dtype == DT_BF16) {
    if (p.rop) hipLaunchKernelGGL((gemm_bf16_kernel<T, T, AM, BMD, kRes>), grid, dim3(256), 0, s, p);
    else hipLaunchKernelGGL((gemm_bf16_kernel<T, T, AM, BMD, false>), grid, dim3(256), 0, s, p);
  } else {
    if (p.rop) hipLaunchKernelGGL((gemm_f32_kernel<T, T, AM, BMD, kRes>), grid, dim3(256), 0, s, p);
    else hipLaunchKernelGGL((gemm_f32_kernel<T, T, AM, BMD, false>), grid, dim3(256), 0, s, p);
  }
  return hipGetLastError();
}

template <int T, int AM>
hipError_t gemm_b(const NodeKernel& k, hipStream_t s) {
  switch (k.bmode) {
    case GM_K: return gemm_go<T, AM, GM_K>(k, s);
    case GM_MN: return gemm_go<T, AM, GM_MN>(k, s);
    default: return gemm_go<T, AM, GM_GENERIC>(k, s);
  }
}

template <int T>
hipError_t gemm_a(const NodeKernel& k, hipStream_t s) {
  switch (k.amode) {
    case GM_K: return gemm_b<T, GM_K>(k, s);
    case GM_MN: return gemm_b<T, GM_MN>(k, s);
    default: return gemm_b<T, GM_GENERIC>(k, s);
  }
}

}  // namespace

hipError_t launch_gemm(const NodeKernel& k, hipStream_t s) {
  const GemmParams& p = k.gemm;
  if ((uint64_t)p.tiles_m * p.tiles_n * p.G >= (1ull << 31)) return hipErrorInvalidValue;
  if (k.gemm_tile >= 8 && k.dtype == DT_F32) return launch_gemm_f32_ring(k, s);
  if (k.gemm_tile >= 6) return k.dtype == DT_BF16 ? launch_gemm_bf16_pipe(k, s) : launch_gemm_f32_dl(k, s);
  if (k.gemm_tile >= 2) return k.dtype == DT_BF16 ? gemm_sk_dispatch<uint16_t>(k, s) : gemm_sk_dispatch<float>(k, s);
  return k.gemm_tile == 0 ? gemm_a<128>(k, s) : gemm_a<64>(k, s);
}

}  // namespace fluid
