// Layout-parameterised elementwise kernels: Add, Mul, GELU, SiLU and the
// relayout copy that a Transpose/Reshape needs when its layouts do not make
// it a view; plus RoPE.  All are HBM-bound: the streaming variant walks the
// output in its physical order (coalesced, 16-byte stores) and reads each
// input through its own strides (16-byte loads when that input is
// unit-stride along the same dim); the tiled variant stages 64x64 tiles in
// LDS so that both the read and the write are coalesced when the input's and
// the output's unit-stride dims differ.
#include "dev.h"
#include "launch.h"

namespace fluid {

template <int OP>
__device__ __forceinline__ float ew_apply(float a, float b) {
  if constexpr (OP == EW_ADD) return a + b;
  else if constexpr (OP == EW_MUL) return a * b;
  else if constexpr (OP == EW_GELU) return gelu_erf(a);
  else if constexpr (OP == EW_SILU) return silu(a);
  else if constexpr (OP == EW_RELU) return a < 0.f ? 0.f : a;   // a NaN stays NaN
  else return a;
}

template <typename T, int VEC>
__device__ __forceinline__ void load_vec(const void* p, int32_t off, float* v) {
  if constexpr (sizeof(T) == 4) {
    static_assert(VEC == 4, "f32 vector width");
    float4 q = *(const float4*)((const float*)p + off);
    v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
  } else {
    static_assert(VEC == 8, "bf16 vector width");
    uint4 q = *(const uint4*)((const uint16_t*)p + off);
    uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[2 * j] = __uint_as_float(w[j] << 16);
      v[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
    }
  }
}

template <typename T, int VEC>
__device__ __forceinline__ void store_vec(void* p, int32_t off, const float* v) {
  if constexpr (sizeof(T) == 4) {
    *(float4*)((float*)p + off) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
    uint4 q;
    q.x = (uint32_t)f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
    q.y = (uint32_t)f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16);
    q.z = (uint32_t)f32_to_bf16(v[4]) | ((uint32_t)f32_to_bf16(v[5]) << 16);
    q.w = (uint32_t)f32_to_bf16(v[6]) | ((uint32_t)f32_to_bf16(v[7]) << 16);
    *(uint4*)((uint16_t*)p + off) = q;
  }
}

template <typename T, int VEC, bool V0, bool V1, int OP>
__global__ __launch_bounds__(256) void ew_kernel(EwParams p) {
  constexpr bool BIN = OP == EW_ADD || OP == EW_MUL;
  const int R = p.rank;
  const uint32_t step = gridDim.x * 256u;
  const uint32_t inner_vecs = p.ext[R - 1] / VEC;
  for (uint32_t v = blockIdx.x * 256u + threadIdx.x; v < p.total; v += step) {
    uint32_t rest = fdiv(v, p.div[R - 1]);
    const uint32_t inner = (v - rest * inner_vecs) * VEC;
    int32_t oo = (int32_t)inner;
    int32_t o0 = (int32_t)inner * p.is0[R - 1];
    int32_t o1 = (int32_t)inner * p.is1[R - 1];
#pragma unroll
    for (int d = kMaxDims - 2; d >= 0; --d) {
      if (d < R - 1) {
        const uint32_t q = fdiv(rest, p.div[d]);
        const int32_t i = (int32_t)(rest - q * p.ext[d]);
        rest = q;
        oo += i * p.os[d];
        o0 += i * p.is0[d];
        o1 += i * p.is1[d];
      }
    }
    float a[VEC], b[VEC];
    if constexpr (V0) {
      load_vec<T, VEC>(p.x0, o0, a);
    } else {
#pragma unroll
      for (int j = 0; j < VEC; ++j) a[j] = Elem<T>::load(p.x0, o0 + j * p.is0[R - 1]);
    }
    if constexpr (BIN) {
      if constexpr (V1) {
        load_vec<T, VEC>(p.x1, o1, b);
      } else {
#pragma unroll
        for (int j = 0; j < VEC; ++j) b[j] = load_any(p.x1, o1 + j * p.is1[R - 1], p.in1_dtype);
      }
    }
    float r[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) r[j] = ew_apply<OP>(a[j], BIN ? b[j] : 0.f);
    if constexpr (VEC > 1) {
      store_vec<T, VEC>(p.y, oo, r);
    } else {
      Elem<T>::store(p.y, oo, r[0]);
    }
  }
}

template <typename T, int OP>
__global__ __launch_bounds__(256) void ew_tiled_kernel(EwParams p) {
  __shared__ float tile[64][65];
  const int R = p.rank, t = p.tdim;
  uint32_t b = blockIdx.x;
  uint32_t q = fdiv(b, p.div_ti);
  const uint32_t ti = b - q * p.tiles_inner;
  b = q;
  q = fdiv(b, p.div_tt);
  const uint32_t tt = b - q * p.tiles_t;
  b = q;
  int32_t bo = 0, bi = 0;
#pragma unroll
  for (int d = kMaxDims - 2; d >= 0; --d) {
    if (d < R - 1 && d != t) {
      const uint32_t qq = fdiv(b, p.div[d]);
      const int32_t i = (int32_t)(b - qq * p.ext[d]);
      b = qq;
      bo += i * p.os[d];
      bi += i * p.is0[d];
    }
  }
  const uint32_t ni = p.ext[R - 1], nk = p.ext[t];
  const uint32_t i0 = ti * 64u, k0 = tt * 64u;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int32_t si = p.is0[R - 1], sk = p.os[t];
  for (int r = ty; r < 64; r += 4) {  // read along the input's unit-stride dim
    const uint32_t ii = i0 + r, kk = k0 + tx;
    if (ii < ni && kk < nk) tile[r][tx] = Elem<T>::load(p.x0, bi + (int32_t)ii * si + (int32_t)kk);
  }
  __syncthreads();
  for (int r = ty; r < 64; r += 4) {  // write along the output's unit-stride dim
    const uint32_t kk = k0 + r, ii = i0 + tx;
    if (ii < ni && kk < nk) Elem<T>::store(p.y, bo + (int32_t)ii + (int32_t)kk * sk, ew_apply<OP>(tile[tx][r], 0.f));
  }
}

// VEC > 1: each thread rotates VEC consecutive pairs (D unit-stride in x and
// y; the host scaled the innermost extent and strides to pieces).
template <typename T, int VEC>
__global__ __launch_bounds__(256) void rope_vec_kernel(RopeParams p) {
  const uint32_t step = gridDim.x * 256u;
  for (uint32_t v = blockIdx.x * 256u + threadIdx.x; v < p.total; v += step) {
    uint32_t rest = v;
    int32_t xo = 0, yo = 0;
    uint32_t pos = 0, i = 0;
#pragma unroll
    for (int d = 3; d >= 0; --d) {
      const uint32_t q = fdiv(rest, p.div[d]);
      const uint32_t id = rest - q * p.ext[d];
      rest = q;
      xo += (int32_t)id * p.xs[d];
      yo += (int32_t)id * p.ys[d];
      if (d == p.pos_dim) pos = id;
      if (d == p.half_dim) i = id * VEC;
    }
    float c[VEC], s[VEC], x1[VEC], x2[VEC], y1[VEC], y2[VEC];
#pragma unroll
    for (int e = 0; e < VEC; e += 4) {
      const float4 cc = *(const float4*)(p.cos_t + pos * p.half + i + e);
      const float4 ss = *(const float4*)(p.sin_t + pos * p.half + i + e);
      c[e] = cc.x; c[e + 1] = cc.y; c[e + 2] = cc.z; c[e + 3] = cc.w;
      s[e] = ss.x; s[e + 1] = ss.y; s[e + 2] = ss.z; s[e + 3] = ss.w;
    }
    load_vec<T, VEC>(p.x, xo, x1);
    load_vec<T, VEC>(p.x, xo + p.x_half, x2);
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      y1[e] = x1[e] * c[e] - x2[e] * s[e];
      y2[e] = x2[e] * c[e] + x1[e] * s[e];
    }
    store_vec<T, VEC>(p.y, yo, y1);
    store_vec<T, VEC>(p.y, yo + p.y_half, y2);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void rope_kernel(RopeParams p) {
  const uint32_t step = gridDim.x * 256u;
  for (uint32_t v = blockIdx.x * 256u + threadIdx.x; v < p.total; v += step) {
    uint32_t rest = v;
    int32_t xo = 0, yo = 0;
    uint32_t pos = 0, i = 0;
#pragma unroll
    for (int d = 3; d >= 0; --d) {
      const uint32_t q = fdiv(rest, p.div[d]);
      const uint32_t id = rest - q * p.ext[d];
      rest = q;
      xo += (int32_t)id * p.xs[d];
      yo += (int32_t)id * p.ys[d];
      if (d == p.pos_dim) pos = id;
      if (d == p.half_dim) i = id;
    }
    const float c = p.cos_t[pos * p.half + i];
    const float s = p.sin_t[pos * p.half + i];
    const float x1 = Elem<T>::load(p.x, xo);
    const float x2 = Elem<T>::load(p.x, xo + p.x_half);
    Elem<T>::store(p.y, yo, x1 * c - x2 * s);
    Elem<T>::store(p.y, yo + p.y_half, x2 * c + x1 * s);
  }
}

namespace {

uint32_t grid_for(uint32_t work) {
  uint32_t b = (work + 255u) / 256u;
  return b < 1u ? 1u : (b > 16384u ? 16384u : b);
}

template <typename T, int VEC, int OP>
hipError_t ew_dispatch_vec(const NodeKernel& k, hipStream_t s) {
  const uint32_t g = grid_for(k.ew.total);
  constexpr bool BIN = OP == EW_ADD || OP == EW_MUL;
  if constexpr (VEC == 1) {
    hipLaunchKernelGGL((ew_kernel<T, 1, false, false, OP>), dim3(g), dim3(256), 0, s, k.ew);
  } else if constexpr (BIN) {
    if (k.vin0 && k.vin1) hipLaunchKernelGGL((ew_kernel<T, VEC, true, true, OP>), dim3(g), dim3(256), 0, s, k.ew);
    else if (k.vin0) hipLaunchKernelGGL((ew_kernel<T, VEC, true, false, OP>), dim3(g), dim3(256), 0, s, k.ew);
    else if (k.vin1) hipLaunchKernelGGL((ew_kernel<T, VEC, false, true, OP>), dim3(g), dim3(256), 0, s, k.ew);
    else hipLaunchKernelGGL((ew_kernel<T, VEC, false, false, OP>), dim3(g), dim3(256), 0, s, k.ew);
  } else {
    if (k.vin0) hipLaunchKernelGGL((ew_kernel<T, VEC, true, false, OP>), dim3(g), dim3(256), 0, s, k.ew);
    else hipLaunchKernelGGL((ew_kernel<T, VEC, false, false, OP>), dim3(g), dim3(256), 0, s, k.ew);
  }
  return hipGetLastError();
}

template <typename T, int OP>
hipError_t ew_dispatch_op(const NodeKernel& k, hipStream_t s) {
  constexpr int V = sizeof(T) == 4 ? 4 : 8;
  if (k.family == KF_EW_TILED) {
    hipLaunchKernelGGL((ew_tiled_kernel<T, OP>), dim3(k.ew.total), dim3(256), 0, s, k.ew);
    return hipGetLastError();
  }
  return k.vec > 1 ? ew_dispatch_vec<T, V, OP>(k, s) : ew_dispatch_vec<T, 1, OP>(k, s);
}

template <typename T>
hipError_t ew_dispatch(const NodeKernel& k, hipStream_t s) {
  switch (k.ew.op) {
    case EW_ADD: return ew_dispatch_op<T, EW_ADD>(k, s);
    case EW_MUL: return ew_dispatch_op<T, EW_MUL>(k, s);
    case EW_GELU: return ew_dispatch_op<T, EW_GELU>(k, s);
    case EW_SILU: return ew_dispatch_op<T, EW_SILU>(k, s);
    case EW_RELU: return ew_dispatch_op<T, EW_RELU>(k, s);
    default: return ew_dispatch_op<T, EW_COPY>(k, s);
  }
}

// Zero Pad and MaxPool: each thread produces output elements in the
// output's physical order (coalesced stores) and reads the input through its
// strides; out-of-range padding positions are zero; the pool maximum keeps a
// NaN (as a maximum over the window must).
template <typename T>
__global__ __launch_bounds__(256) void window_kernel(WinParams p) {
  const uint32_t step = gridDim.x * 256u;
  for (uint32_t idx = blockIdx.x * 256u + threadIdx.x; idx < p.total; idx += step) {
    uint32_t rem = idx;
    int32_t yo = 0, xo = 0, h = 0, w = 0;
#pragma unroll
    for (int d = 3; d >= 0; --d) {
      const uint32_t q = fdiv(rem, p.div[d]);
      const int32_t c = (int32_t)(rem - q * p.ext[d]);
      rem = q;
      yo += c * p.os[d];
      if (p.role[d] == 0) xo += c * p.is[d];
      else if (p.role[d] == 1) h = c;
      else w = c;
    }
    float v;
    if (p.op == 0) {
      const int32_t hi = h - p.k, wi = w - p.k;
      v = (hi >= 0 && hi < p.in_h && wi >= 0 && wi < p.in_w) ? Elem<T>::load(p.x, xo + hi * p.is_h + wi * p.is_w)
                                                             : 0.f;
    } else {
      v = -INFINITY;
      for (int32_t u = 0; u < p.k; ++u)
        for (int32_t t = 0; t < p.k; ++t) {
          const float a = Elem<T>::load(p.x, xo + (h * p.k + u) * p.is_h + (w * p.k + t) * p.is_w);
          v = (a > v || a != a) ? a : v;
        }
    }
    Elem<T>::store(p.y, yo, v);
  }
}

}  // namespace

hipError_t launch_elementwise(const NodeKernel& k, hipStream_t s) {
  return k.dtype == DT_BF16 ? ew_dispatch<uint16_t>(k, s) : ew_dispatch<float>(k, s);
}

hipError_t launch_window(const NodeKernel& k, hipStream_t s) {
  const uint32_t g = grid_for(k.win.total);
  if (k.dtype == DT_BF16) hipLaunchKernelGGL(window_kernel<uint16_t>, dim3(g), dim3(256), 0, s, k.win);
  else hipLaunchKernelGGL(window_kernel<float>, dim3(g), dim3(256), 0, s, k.win);
  return hipGetLastError();
}

hipError_t launch_rope(const NodeKernel& k, hipStream_t s) {
  const uint32_t g = grid_for(k.rope.total);
  if (k.vec > 1) {
    if (k.dtype == DT_BF16) hipLaunchKernelGGL((rope_vec_kernel<uint16_t, 8>), dim3(g), dim3(256), 0, s, k.rope);
    else hipLaunchKernelGGL((rope_vec_kernel<float, 4>), dim3(g), dim3(256), 0, s, k.rope);
  } else if (k.dtype == DT_BF16) {
    hipLaunchKernelGGL(rope_kernel<uint16_t>, dim3(g), dim3(256), 0, s, k.rope);
  } else {
    hipLaunchKernelGGL(rope_kernel<float>, dim3(g), dim3(256), 0, s, k.rope);
  }
  return hipGetLastError();
}

}  // namespace fluid
