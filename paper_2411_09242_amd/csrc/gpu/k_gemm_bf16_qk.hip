// bf16 GEMM for a short K (at most 128: the head dimension of Q K^T), where
// the product is bound by writing C (an S x S score matrix per head), not by
// the matrix cores.  A K-contiguous A and a K- or N-contiguous B, MFMA
// 32x32x16 bf16 with fp32 accumulate.
//
//  * Persistent workgroups, two per CU, each walking the 128 x 128 output
//    tiles t = blockIdx, blockIdx + gridDim, ...  The whole K range of a
//    tile's A and B fits in LDS (2 x 32 KiB).  The next tile's operands are
//    loaded into registers while the current tile is multiplied and written
//    out, and go to LDS once the current tile has left it, so the loads'
//    latency hides behind the previous tile's work and stores.
//  * Four wavefronts of 64 x 64 (2 x 2 blocks of 32 x 32).  K past the end
//    reads as zero, so every tile runs the same eight 16-k steps.
//  * The output tile leaves through LDS (the consumed A tile), each lane
//    writing 16 contiguous bytes, as in the other bf16 kernels.
//  * When a causal softmax is the only reader of C, only the tiles on or
//    below the diagonal are enumerated (row tm has tiles 0 .. tm), so the
//    work is evenly spread over the persistent workgroups.
//
// LDS rows are 256 bytes (128 bf16) = 16 chunks of 16 bytes.  A (and a
// K-contiguous B) row r stores logical chunk c at c ^ (r % 16): an MFMA
// operand read (16 consecutive rows, one chunk) then touches every bank
// once.  An N-contiguous B is stored [k][n] and read with ds_read_b64_tr_b16,
// row k storing chunk c at c ^ 4 (k % 4), as in the 256 x 128 kernel.
#include <math.h>

#include "gemm_common.h"
#include "launch.h"

namespace fluid {

namespace {

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __attribute__((address_space(3))) uint4 lds_uint4;

constexpr int QK_T = 128;                // tile rows = tile columns
constexpr int QK_KMAX = 128;             // K held whole in LDS
constexpr int QK_ROWB = QK_KMAX * 2;     // bytes per LDS row
constexpr int QK_OP = QK_T * QK_ROWB;    // 32 KiB per operand

}  // namespace

template <int BMD>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void gemm_bf16_qk_kernel(GemmParams p) {
  __shared__ __attribute__((aligned(1024))) uint8_t As[QK_OP];
  __shared__ __attribute__((aligned(1024))) uint8_t Bs[QK_OP];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 31, lh = lane >> 5;
  const Rsrc ra = make_rsrc(p.A, p.a_bytes);
  const Rsrc rb = make_rsrc(p.B, p.b_bytes);

  // tiles of one batch entry: all of them, or the lower triangle
  const bool tri = (p.causal & 1u) && p.tiles_m == p.tiles_n;
  const uint32_t per_g = tri ? p.tiles_m * (p.tiles_m + 1) / 2 : p.tiles_m * p.tiles_n;
  const uint32_t ntiles = per_g * p.G;
  auto coord = [&](uint32_t t) {
    const uint32_t g = t / per_g, j = t - g * per_g;
    uint32_t tm, tn;
    if (tri) {
      // row tm holds entries tm (tm + 1) / 2 .. (tm + 1) (tm + 2) / 2 - 1
      tm = (uint32_t)((sqrtf(8.f * (float)j + 1.f) - 1.f) * 0.5f);
      while ((tm + 1) * (tm + 2) / 2 <= j) ++tm;
      while (tm * (tm + 1) / 2 > j) --tm;
      tn = j - tm * (tm + 1) / 2;
    } else {
      tm = j / p.tiles_n;
      tn = j - tm * p.tiles_n;
    }
    const uint32_t g1 = fdiv(g, p.g2div), g2 = g - g1 * p.G2;
    TileCoord c;
    c.m0 = tm * QK_T;
    c.n0 = tn * QK_T;
    c.a_base = (int32_t)g1 * p.a_g1 + (int32_t)g2 * p.a_g2;
    c.b_base = (int32_t)g1 * p.b_g1 + (int32_t)g2 * p.b_g2;
    c.c_base = (int32_t)g1 * p.c_g1 + (int32_t)g2 * p.c_g2;
    c.r_base = 0;  // no Add / Mul epilogue here
    return c;
  };

  // One tile's operands: global -> registers (issued early), registers ->
  // LDS (once the LDS is free).  Piece q of wavefront w covers LDS rows
  // 32 w + 4 q .. +3; lane l carries row 32 w + 4 q + l / 16 at chunk
  // position l % 16.  Rows of A past M and of B past N are clamped onto
  // row / column 0 (they only feed outputs that are never stored); k past K
  // reads zero.
  struct Regs {
    uint4 a[8], b[8];
  };
  const int sub = lane >> 4, pc = lane & 15;
  auto gload = [&](Regs& R, const TileCoord& tc) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int row = 32 * wave + 4 * q + sub;
      const uint32_t k = 8u * (uint32_t)(pc ^ (row & 15));
      const uint32_t m = tc.m0 + row;
      const int32_t src = tc.a_base + (m < p.M ? row_off(p, m, p.a_m1, p.a_m2) : 0) + (int32_t)k;
      R.a[q] = bload16(ra, k < p.K ? 2u * (uint32_t)src : kOOB);
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int row = 32 * wave + 4 * q + sub;
      uint32_t off;
      if constexpr (BMD == GM_MN) {
        // row = k, 128 n per row; logical chunk c holds n0 + 8 c .. +7
        const uint32_t n = tc.n0 + 8u * (uint32_t)(pc ^ (4 * (row & 3)));
        const int32_t src = tc.b_base + (int32_t)row * p.b_k + (int32_t)(n < p.N ? n : 0);
        off = (uint32_t)row < p.K ? 2u * (uint32_t)src : kOOB;
      } else {
        // row = n, 128 k per row, like A
        const uint32_t k = 8u * (uint32_t)(pc ^ (row & 15));
        const uint32_t n = tc.n0 + row;
        const int32_t src = tc.b_base + (int32_t)(n < p.N ? n : 0) * p.b_n + (int32_t)k;
        off = k < p.K ? 2u * (uint32_t)src : kOOB;
      }
      R.b[q] = bload16(rb, off);
    }
  };
  auto lstore = [&](const Regs& R) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int row = 32 * wave + 4 * q + sub;
      *(uint4*)(As + row * QK_ROWB + pc * 16) = R.a[q];
      *(uint4*)(Bs + row * QK_ROWB + pc * 16) = R.b[q];
    }
  };

  // transpose-read addressing (N-contiguous B): lane l (group g = l / 16,
  // s = l % 16) points at row 16 kk + 8 (g / 2) + 4 h + s / 4, columns
  // c0 + 16 (g % 2) + 4 (s % 4) .. +3; the read returns column c0 + l % 32,
  // rows 16 kk + 8 (l / 32) + 4 h .. +3.
  const int tg = lane >> 4, ts = lane & 15;
  const int t_row = 8 * (tg >> 1) + (ts >> 2);
  const int t_col = 16 * (tg & 1) + 4 * (ts & 3);

  // Bare barrier: every wavefront's LDS accesses so far are done.  (A
  // workgroup fence would also wait for the output stores and the next
  // tile's loads; the loads are waited for where their registers are used.)
  auto lds_barrier = [&]() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  uint32_t t = blockIdx.x;
  if (t >= ntiles) return;
  TileCoord cur = coord(t);
  Regs R;
  gload(R, cur);
  lstore(R);
  __syncthreads();
  uint16_t* C = (uint16_t*)p.C;
  for (;;) {
    const uint32_t tnext = t + gridDim.x;
    const bool more = tnext < ntiles;
    TileCoord nxt = cur;
    if (more) {
      nxt = coord(tnext);
      gload(R, nxt);  // in flight while this tile is multiplied and stored
    }
    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
    // two 16-k steps per iteration: unrolling all eight would hoist every
    // operand read and leave too few registers for two workgroups per CU
#pragma unroll 2
    for (int kk = 0; kk < QK_KMAX / 16; ++kk) {
      bf16x8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int row = wm * 64 + 32 * i + lr;
        const int chunk = (2 * kk + lh) ^ (row & 15);
        a[i] = __builtin_bit_cast(bf16x8, *(const lds_uint4*)(As + row * QK_ROWB + chunk * 16));
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        if constexpr (BMD == GM_MN) {
          v4i16 h2[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int row = 16 * kk + 4 * h + t_row;  // row % 4 == ts / 4
            const int col = wn * 64 + 32 * j + t_col;
            const int chunk = (col >> 3) ^ (4 * (row & 3));
            h2[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(Bs + row * QK_ROWB + chunk * 16 + (col & 7) * 2));
          }
          b[j] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(h2[0], h2[1], 0, 1, 2, 3, 4, 5, 6, 7));
        } else {
          const int row = wn * 64 + 32 * j + lr;
          const int chunk = (2 * kk + lh) ^ (row & 15);
          b[j] = __builtin_bit_cast(bf16x8, *(const lds_uint4*)(Bs + row * QK_ROWB + chunk * 16));
        }
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }

#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        epi16<false, false>(p, cur.r_base, cur.m0 + wm * 64 + 32 * i + 4 * lh, cur.n0 + wn * 64 + 32 * j + lr, acc[i][j]);
    if (p.cmode == 1 || p.cmode == 2) {
      // every wavefront is done with the A tile: park the output there
      lds_barrier();
      uint16_t* cs = (uint16_t*)As;
      if (p.cmode == 1) {
        // row-major [128][128], chunk c of row r at c ^ (r % 16)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
              const int r = wm * 64 + 32 * i + 8 * (v / 4) + 4 * lh + (v % 4), c = wn * 64 + 32 * j + lr;
              cs[r * QK_T + (((c >> 3) ^ (r & 15)) << 3) + (c & 7)] = f32_to_bf16(acc[i][j][v]);
            }
        lds_barrier();
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int r = 32 * wave + 4 * u + (lane >> 4), ch = lane & 15;
          const uint4 val = *(const uint4*)&cs[r * QK_T + ((ch ^ (r & 15)) << 3)];
          const uint32_t m = cur.m0 + r, n0 = cur.n0 + 8 * ch;
          if (m >= p.M || n0 >= p.N) continue;
          uint16_t* dst = C + cur.c_base + row_off(p, m, p.c_m1, p.c_m2) + (int32_t)n0;
          if (n0 + 8 <= p.N && ((uintptr_t)dst & 15u) == 0) {
            *(uint4*)dst = val;
          } else {
            const uint32_t w[4] = {val.x, val.y, val.z, val.w};
            for (int e = 0; e < 8 && n0 + e < p.N; ++e) dst[e] = (uint16_t)(w[e / 2] >> (16 * (e & 1)));
          }
        }
      } else {
        // column-major [128][128] (rows contiguous), chunk c of column n at
        // c ^ (n % 16); a lane parks 4 consecutive rows (8 bytes)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int vg = 0; vg < 4; ++vg) {
              const int r0 = wm * 64 + 32 * i + 8 * vg + 4 * lh, c = wn * 64 + 32 * j + lr;
              const uint32_t lo = (uint32_t)f32_to_bf16(acc[i][j][4 * vg]) | ((uint32_t)f32_to_bf16(acc[i][j][4 * vg + 1]) << 16);
              const uint32_t hi = (uint32_t)f32_to_bf16(acc[i][j][4 * vg + 2]) | ((uint32_t)f32_to_bf16(acc[i][j][4 * vg + 3]) << 16);
              *(uint2*)&cs[c * QK_T + (((r0 >> 3) ^ (c & 15)) << 3) + (r0 & 7)] = make_uint2(lo, hi);
            }
        lds_barrier();
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int c = 32 * wave + 4 * u + (lane >> 4), ch = lane & 15;
          const uint4 val = *(const uint4*)&cs[c * QK_T + ((ch ^ (c & 15)) << 3)];
          const uint32_t n = cur.n0 + c, m0 = cur.m0 + 8 * ch;
          if (n >= p.N || m0 >= p.M) continue;
          const uint32_t m2 = m0 - fdiv(m0, p.m2div) * p.M2;  // position within the M2 run
          uint16_t* dst = C + cur.c_base + row_off(p, m0, p.c_m1, p.c_m2) + (int32_t)n * p.c_n;
          if (m0 + 8 <= p.M && m2 + 8 <= p.M2 && ((uintptr_t)dst & 15u) == 0) {
            *(uint4*)dst = val;
          } else {
            const uint32_t w[4] = {val.x, val.y, val.z, val.w};
            for (int e = 0; e < 8 && m0 + e < p.M; ++e)
              C[cur.c_base + row_off(p, m0 + e, p.c_m1, p.c_m2) + (int32_t)n * p.c_n] = (uint16_t)(w[e / 2] >> (16 * (e & 1)));
          }
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const uint32_t n = cur.n0 + wn * 64 + 32 * j + lr;
          if (n >= p.N) continue;
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const uint32_t m = cur.m0 + wm * 64 + 32 * i + 8 * (v / 4) + 4 * lh + (v % 4);
            if (m < p.M) C[cur.c_base + row_off(p, m, p.c_m1, p.c_m2) + (int32_t)n * p.c_n] = f32_to_bf16(acc[i][j][v]);
          }
        }
    }
    if (!more) break;
    // the tile (and its parked output) has left the LDS: the next tile's
    // operands go in
    lds_barrier();
    lstore(R);
    lds_barrier();
    t = tnext;
    cur = nxt;
  }
}

hipError_t launch_gemm_bf16_qk(const NodeKernel& k, hipStream_t s) {
  const GemmParams& p = k.gemm;
  if (k.dtype != DT_BF16 || k.amode != GM_K || (k.bmode != GM_MN && k.bmode != GM_K) || p.K > (uint32_t)QK_KMAX)
    return hipErrorInvalidValue;
  static int n_cu = 0;
  if (n_cu == 0) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n_cu <= 0)
      n_cu = 256;
  }
  const bool tri = (p.causal & 1u) && p.tiles_m == p.tiles_n;
  const uint64_t ntiles = (uint64_t)(tri ? p.tiles_m * (p.tiles_m + 1) / 2 : p.tiles_m * p.tiles_n) * p.G;
  const dim3 grid((uint32_t)std::min<uint64_t>(ntiles, 2 * (uint64_t)n_cu));
  if (grid.x == 0) return hipSuccess;
  // an epilogue of bias only (the register budget is spent)
  if (p.rop || p.act) return hipErrorInvalidValue;
  if (k.bmode == GM_MN) hipLaunchKernelGGL((gemm_bf16_qk_kernel<GM_MN>), grid, dim3(256), 0, s, p);
  else hipLaunchKernelGGL((gemm_bf16_qk_kernel<GM_K>), grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace fluid
