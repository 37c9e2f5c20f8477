// fp32 GEMM for a short K (at most 64: the head dimension of Q K^T) with a
// K-contiguous A and B, where the product is bound by writing C (an S x S
// score matrix per head) as much as by the matrix cores.  MFMA 32x32x2 f32
// (lane l: A[l%32][l/32], B[l/32][l%32]; accumulator v of lane l holds
// C[8(v/4) + 4(l/32) + v%4][l%32]).
//
//  * Persistent workgroups, two per CU, each walking the 128 x 128 output
//    tiles t = blockIdx, blockIdx + gridDim, ...  The whole K range of a
//    tile's A and B fits in LDS (2 x 32 KiB); the next tile's operands are
//    loaded into registers while the current tile is multiplied and written
//    out, and go to LDS once the current tile has left it.
//  * Four wavefronts of 64 x 64 (2 x 2 blocks of 32 x 32).  K past the end
//    reads as zero, so every tile runs the same 32 two-k steps.
//  * An N-contiguous C leaves through LDS (the consumed operand tiles, 64
//    KiB), each lane writing 16 contiguous bytes; other layouts of C are
//    written value by value from the accumulators.
//  * When a causal softmax is the only reader of C, only the tiles on or
//    below the diagonal are enumerated.
//
// LDS operand rows are 256 bytes (64 floats) = 16 chunks of 16 bytes; row r
// stores logical chunk c at c ^ (r % 16).  The parked output rows are 512
// bytes (128 floats) = 32 chunks; row r stores chunk c at c ^ (r % 32).
#include <math.h>

#include "gemm_common.h"
#include "launch.h"

namespace fluid {

namespace {

constexpr int QF_T = 128;               // tile rows = tile columns
constexpr int QF_KMAX = 64;             // K held whole in LDS
constexpr int QF_OP = QF_T * QF_KMAX;   // floats per operand tile (32 KiB)

}  // namespace

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void gemm_f32_qk_kernel(GemmParams p) {
  // A tile, then B tile; together they hold the parked output
  __shared__ __attribute__((aligned(1024))) float S[2 * QF_OP];
  float* As = S;
  float* Bs = S + QF_OP;
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
      // row tm of the triangle holds entries tm (tm + 1) / 2 .. +tm
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
    c.m0 = tm * QF_T;
    c.n0 = tn * QF_T;
    c.a_base = (int32_t)g1 * p.a_g1 + (int32_t)g2 * p.a_g2;
    c.b_base = (int32_t)g1 * p.b_g1 + (int32_t)g2 * p.b_g2;
    c.c_base = (int32_t)g1 * p.c_g1 + (int32_t)g2 * p.c_g2;
    c.r_base = 0;  // no Add / Mul epilogue here
    return c;
  };

  // One tile's operands: global -> registers (issued early), registers ->
  // LDS (once the LDS is free).  Piece q of wavefront w covers rows
  // 32 w + 4 q .. +3; lane l carries row 32 w + 4 q + l / 16 at chunk
  // position l % 16, which holds logical chunk (l % 16) ^ (row % 16), i.e.
  // k = 4 that .. +3.  Rows past M (of A) or N (of B) are clamped onto row
  // 0 (they only feed outputs that are never stored); k past K reads zero.
  struct Regs {
    uint4 a[8], b[8];
  };
  const int sub = lane >> 4, pc = lane & 15;
  auto gload = [&](Regs& R, const TileCoord& tc) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int row = 32 * wave + 4 * q + sub;
      const uint32_t k = 4u * (uint32_t)(pc ^ (row & 15));
      const uint32_t m = tc.m0 + row;
      const int32_t sa = tc.a_base + (m < p.M ? row_off(p, m, p.a_m1, p.a_m2) : 0) + (int32_t)k;
      R.a[q] = bload16(ra, k < p.K ? 4u * (uint32_t)sa : kOOB);
      const uint32_t n = tc.n0 + row;
      const int32_t sb = tc.b_base + (int32_t)(n < p.N ? n : 0) * p.b_n + (int32_t)k;
      R.b[q] = bload16(rb, k < p.K ? 4u * (uint32_t)sb : kOOB);
    }
  };
  auto lstore = [&](const Regs& R) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int row = 32 * wave + 4 * q + sub;
      *(uint4*)(As + row * QF_KMAX + pc * 4) = R.a[q];
      *(uint4*)(Bs + row * QF_KMAX + pc * 4) = R.b[q];
    }
  };
  // element k of operand row r in its LDS tile
  auto at = [](const float* T, int r, int k) { return T[r * QF_KMAX + (((k >> 2) ^ (r & 15)) << 2) + (k & 3)]; };

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
  float* C = (float*)p.C;
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
#pragma unroll 4
    for (int s = 0; s < QF_KMAX / 2; ++s) {
      const int k = 2 * s + lh;
      float a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = at(As, wm * 64 + 32 * i + lr, k);
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = at(Bs, wn * 64 + 32 * j + lr, k);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }

#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        epi16<false, false>(p, cur.r_base, cur.m0 + wm * 64 + 32 * i + 4 * lh, cur.n0 + wn * 64 + 32 * j + lr, acc[i][j]);
    if (p.cmode == 1) {
      // every wavefront is done with the operand tiles: park the output
      // there, row-major [128][128], chunk c of row r at c ^ (r % 32)
      lds_barrier();
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int r = wm * 64 + 32 * i + 8 * (v / 4) + 4 * lh + (v % 4), c = wn * 64 + 32 * j + lr;
            S[r * QF_T + (((c >> 2) ^ (r & 31)) << 2) + (c & 3)] = acc[i][j][v];
          }
      lds_barrier();
      // wavefront w writes rows 32 w .. +31, two rows of 32 chunks per step
#pragma unroll 4
      for (int u = 0; u < 16; ++u) {
        const int r = 32 * wave + 2 * u + (lane >> 5), ch = lane & 31;
        const uint4 val = *(const uint4*)&S[r * QF_T + ((ch ^ (r & 31)) << 2)];
        const uint32_t m = cur.m0 + r, n0 = cur.n0 + 4 * ch;
        if (m >= p.M || n0 >= p.N) continue;
        float* dst = C + cur.c_base + row_off(p, m, p.c_m1, p.c_m2) + (int32_t)n0;
        if (n0 + 4 <= p.N && ((uintptr_t)dst & 15u) == 0) {
          *(uint4*)dst = val;
        } else {
          const float w[4] = {__uint_as_float(val.x), __uint_as_float(val.y), __uint_as_float(val.z), __uint_as_float(val.w)};
          for (int e = 0; e < 4 && n0 + e < p.N; ++e) dst[e] = w[e];
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
            if (m < p.M) C[cur.c_base + row_off(p, m, p.c_m1, p.c_m2) + (int32_t)n * p.c_n] = acc[i][j][v];
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

hipError_t launch_gemm_f32_qk(const NodeKernel& k, hipStream_t s) {
  const GemmParams& p = k.gemm;
  if (k.dtype != DT_F32 || k.amode != GM_K || k.bmode != GM_K || p.K > (uint32_t)QF_KMAX) return hipErrorInvalidValue;
  // an epilogue of bias only
  if (p.rop || p.act) return hipErrorInvalidValue;
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
  hipLaunchKernelGGL(gemm_f32_qk_kernel, grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace fluid
