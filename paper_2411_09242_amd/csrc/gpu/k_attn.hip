// Attention of short sequences (keys T <= 128, head dim D <= 128) in one
// launch: the score product, the row softmax and the product with V that
// the graph holds as three nodes (a MatMul, a Softmax, a MatMul), for the
// executor to run together when the scores and probabilities have no other
// reader.  A workgroup owns 16 query rows of one head: K^T and V of the head
// go to LDS once, the 16 x T scores stay in LDS, and only O is written.  Both
// products are MFMA 16x16x4 f32 over LDS operands, each wavefront owning
// 16-column blocks of the result.  MFMA 16x16x4 f32 layout: lane l holds
// A[l % 16][k = l / 16], B[k = l / 16][l % 16] and result rows 4 (l / 16)
// .. +3 of column l % 16.
#include "gemm_common.h"
#include "launch.h"

namespace fluid {

namespace {

constexpr int AT_RB = 16;     // query rows per workgroup
constexpr int AT_MAX = 128;   // largest T and D

// A [R][C] tile of the source (element (r, c) at src[r sr + c sc]) bound
// for LDS at dst[r pitch + c], zero past nr rows / nc columns.  128 lanes
// walk the source's unit-stride dim (at most 128 long), the two halves of
// the workgroup alternate along the other.
struct Tile {
  float* dst;
  uint32_t pitch;
  const float* src;
  int32_t sr, sc;
  uint32_t R, C, nr, nc;
  __device__ bool c_fast() const { return sc == 1 || sr != 1; }
  __device__ uint32_t nf() const { return c_fast() ? C : R; }
  __device__ uint32_t ns() const { return c_fast() ? R : C; }
};

// Stages two tiles together: each lane keeps AT_BATCH loads of each in
// flight before writing them (a load-store chain per element, or one tile
// after the other, leaves the stage bound by memory latency).  The loads are
// buffer loads, so that the padding reads zero through the range check
// (offset kOOB) instead of a branch around each load, which would wait for
// every load before issuing the next.
constexpr int AT_BATCH = 8;
__device__ __forceinline__ float tile_load(Rsrc r, bool ok, int32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, ok ? 4u * (uint32_t)off : kOOB, 0, 0));
}
// A tile whose unit-stride dim has a multiple of 4 elements, with rows 16-byte
// aligned: 16-byte loads, lpr lanes per row (a power of two covering the
// row), 256 / lpr rows per step, AT_BATCH loads in flight per lane.
__device__ __forceinline__ bool vec_ok(const Tile& t) {
  const int32_t so = t.c_fast() ? t.sr : t.sc;  // stride of the other dim
  const uint32_t nfr = t.c_fast() ? t.nc : t.nr;
  return (t.c_fast() ? t.sc : t.sr) == 1 && nfr % 4 == 0 && so % 4 == 0 && ((uintptr_t)t.src & 15u) == 0;
}
// (not inlined: one copy of the code for the three tiles keeps the kernel
// small, and a one-pass kernel pays for every instruction-cache miss)
__device__ __attribute__((noinline)) void stage_vec(Tile t, int tid) {
  const bool cf = t.c_fast();
  const uint32_t nf = t.nf(), ns = t.ns(), nfr = cf ? t.nc : t.nr, nsr = cf ? t.nr : t.nc;
  uint32_t lpr = 1;
  while (4u * lpr < nf) lpr *= 2;
  const uint32_t f4 = 4u * (tid & (lpr - 1)), srow = tid / lpr, step = 256u / lpr;
  if (f4 >= nf) return;
  const Rsrc rs = make_rsrc(t.src, 0x7fffffffu);
  const int32_t so = cf ? t.sr : t.sc;
  for (uint32_t s0 = srow; s0 < ns; s0 += step * AT_BATCH) {
    uint4 v[AT_BATCH];
#pragma unroll
    for (int u = 0; u < AT_BATCH; ++u) {
      const uint32_t si = s0 + step * u;
      const bool ok = si < nsr && f4 < nfr;
      v[u] = bload16(rs, ok ? 4u * (uint32_t)((int32_t)si * so + (int32_t)f4) : kOOB);
    }
#pragma unroll
    for (int u = 0; u < AT_BATCH; ++u) {
      const uint32_t si = s0 + step * u;
      if (si >= ns) continue;
      if (cf) {
        *(uint4*)(t.dst + si * t.pitch + f4) = v[u];
      } else {
        const float e[4] = {__uint_as_float(v[u].x), __uint_as_float(v[u].y), __uint_as_float(v[u].z),
                            __uint_as_float(v[u].w)};
#pragma unroll
        for (int i = 0; i < 4; ++i) t.dst[(f4 + i) * t.pitch + si] = e[i];
      }
    }
  }
}

__device__ __attribute__((noinline)) void stage2(Tile a, Tile b, int tid) {
  const uint32_t fa = tid & 127;
  const uint32_t na = fa < a.nf() ? a.ns() : 0u, nb = fa < b.nf() ? b.ns() : 0u;
  const Rsrc ra = make_rsrc(a.src, 0x7fffffffu), rb = make_rsrc(b.src, 0x7fffffffu);
  for (uint32_t s0 = tid >> 7; s0 < max(na, nb); s0 += 2u * AT_BATCH) {
    float va[AT_BATCH], vb[AT_BATCH];
#pragma unroll
    for (int u = 0; u < AT_BATCH; ++u) {
      const uint32_t si = s0 + 2u * u;
      {
        const uint32_t r = a.c_fast() ? si : fa, c = a.c_fast() ? fa : si;
        va[u] = tile_load(ra, si < na && r < a.nr && c < a.nc, (int32_t)r * a.sr + (int32_t)c * a.sc);
      }
      {
        const uint32_t r = b.c_fast() ? si : fa, c = b.c_fast() ? fa : si;
        vb[u] = tile_load(rb, si < nb && r < b.nr && c < b.nc, (int32_t)r * b.sr + (int32_t)c * b.sc);
      }
    }
#pragma unroll
    for (int u = 0; u < AT_BATCH; ++u) {
      const uint32_t si = s0 + 2u * u;
      if (si < na) {
        const uint32_t r = a.c_fast() ? si : fa, c = a.c_fast() ? fa : si;
        a.dst[r * a.pitch + c] = va[u];
      }
      if (si < nb) {
        const uint32_t r = b.c_fast() ? si : fa, c = b.c_fast() ? fa : si;
        b.dst[r * b.pitch + c] = vb[u];
      }
    }
  }
}

}  // namespace

__global__ __launch_bounds__(256) void attn_small_kernel(AttnParams p) {
  extern __shared__ float4 smem4[];
  float* smem = (float*)smem4;
  // T and D padded to whole 16-column blocks
  const uint32_t TP = (p.T + 15u) & ~15u, DP = (p.D + 15u) & ~15u;
  const uint32_t kp = TP + 4u, vp = DP + 4u;  // row pitches
  float* Kt = smem;                  // [DP][kp]
  float* Vs = Kt + DP * kp;          // [TP][vp]
  float* Qs = Vs + TP * vp;          // [AT_RB][vp]
  float* Ps = Qs + AT_RB * vp;       // [AT_RB][kp]
  const uint32_t nblk = (p.S + AT_RB - 1u) / AT_RB;
  const uint32_t g = blockIdx.x / nblk, r0 = (blockIdx.x - g * nblk) * AT_RB;
  const uint32_t g1 = fdiv(g, p.g2div), g2 = g - g1 * p.G2;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lq = lane >> 4;
  const float* Q = p.Q + (int32_t)g1 * p.q_g1 + (int32_t)g2 * p.q_g2;
  const float* Kt_g = p.Kt + (int32_t)g1 * p.k_g1 + (int32_t)g2 * p.k_g2;
  const float* V = p.V + (int32_t)g1 * p.v_g1 + (int32_t)g2 * p.v_g2;
  float* O = p.O + (int32_t)g1 * p.o_g1 + (int32_t)g2 * p.o_g2;

  // operands -> LDS (zero padding past T, D and S)
  const Tile tk{Kt, kp, Kt_g, p.k_d, p.k_t, DP, TP, p.D, p.T};
  const Tile tv{Vs, vp, V, p.v_t, p.v_d, TP, DP, p.T, p.D};
  const Tile tq{Qs, vp, Q + (int32_t)r0 * p.q_s, p.q_s, p.q_d, AT_RB, DP, min((uint32_t)AT_RB, p.S - r0), p.D};
  const Tile none{nullptr, 0u, nullptr, 0, 1, 0u, 0u, 0u, 0u};
  const bool vk = vec_ok(tk), vv = vec_ok(tv), vq = vec_ok(tq);
  if (vk) stage_vec(tk, tid);
  if (vv) stage_vec(tv, tid);
  if (vq) stage_vec(tq, tid);
  stage2(vk ? none : tk, vv ? none : tv, tid);
  stage2(vq ? none : tq, none, tid);
  __syncthreads();

  // scores S = Q K^T: wavefront w owns the 16-column blocks w, w + 4, ...
  for (uint32_t j = w; j < TP / 16u; j += 4) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (uint32_t k = 0; k < DP; k += 4)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(Qs[lr * vp + k + lq], Kt[(k + lq) * kp + 16 * j + lr], acc, 0, 0,
                                                 0);
#pragma unroll
    for (int v = 0; v < 4; ++v) Ps[(4 * lq + v) * kp + 16 * j + lr] = acc[v];
  }
  __syncthreads();

  // row softmax of scale * scores: wavefront w takes rows 4 w .. 4 w + 3
  // (the four reductions interleaved), lane l the keys l and l + 64; masked
  // and padding keys end as exact 0
  {
    float v[4][2], m[4], sum[4];
    bool ok[4][2];
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const uint32_t r = 4 * w + rr, q = r0 + r;
      m[rr] = -INFINITY;
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const uint32_t t = lane + 64 * jj;
        ok[rr][jj] = t < p.T && !(p.causal && t > q);
        v[rr][jj] = ok[rr][jj] ? Ps[r * kp + t] * p.scale : 0.f;
        if (ok[rr][jj]) m[rr] = fmaxf(m[rr], v[rr][jj]);
      }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) m[rr] = fmaxf(m[rr], __shfl_xor(m[rr], o, 64));
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      sum[rr] = 0.f;
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        v[rr][jj] = ok[rr][jj] ? expf(v[rr][jj] - m[rr]) : 0.f;
        sum[rr] += v[rr][jj];
      }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) sum[rr] += __shfl_xor(sum[rr], o, 64);
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const float inv = 1.0f / sum[rr];
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const uint32_t t = lane + 64 * jj;
        if (t < TP) Ps[(4 * w + rr) * kp + t] = v[rr][jj] * inv;
      }
    }
  }
  __syncthreads();

  // O = P V: wavefront w owns the 16-column blocks w, w + 4, ... of O
  for (uint32_t j = w; j < DP / 16u; j += 4) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (uint32_t t = 0; t < TP; t += 4)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(Ps[lr * kp + t + lq], Vs[(t + lq) * vp + 16 * j + lr], acc, 0, 0,
                                                 0);
    const uint32_t d = 16 * j + lr;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const uint32_t srow = r0 + 4 * lq + v;
      if (srow < p.S && d < p.D) O[(int32_t)srow * p.o_s + (int32_t)d * p.o_d] = acc[v];
    }
  }
}

uint32_t attn_small_lds_bytes(const AttnParams& p) {
  const uint32_t TP = (p.T + 15u) & ~15u, DP = (p.D + 15u) & ~15u;
  return 4u * (DP * (TP + 4u) + TP * (DP + 4u) + AT_RB * (DP + 4u) + AT_RB * (TP + 4u));
}

hipError_t launch_attn_small(const AttnParams& p, hipStream_t s) {
  if (p.T == 0 || p.D == 0 || p.T > (uint32_t)AT_MAX || p.D > (uint32_t)AT_MAX || p.S == 0)
    return hipErrorInvalidValue;
  const uint32_t lds = attn_small_lds_bytes(p);
  // more than the default 64 KiB of dynamic LDS (at most 152 KiB here)
  if (lds > 64u * 1024u) {
    static const hipError_t attr = hipFuncSetAttribute((const void*)attn_small_kernel,
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (attr != hipSuccess) return attr;
  }
  const dim3 grid(p.G * ((p.S + AT_RB - 1u) / AT_RB));
  hipLaunchKernelGGL(attn_small_kernel, grid, dim3(256), lds, s, p);
  return hipGetLastError();
}

}  // namespace fluid
