// Row reductions over the last logical dim: Softmax (with fused scale and
// causal mask), LayerNorm and RMSNorm, in three variants.
//  * row (variant 0): one 64-lane wavefront per row; the row is held in
//    registers (up to 4096 values), reduced with cross-lane butterflies, and
//    written once -- one HBM read and one write per element.  Coalesced when
//    the reduced dim is unit-stride; when in addition rows start on 16-byte
//    boundaries, each lane moves 16-byte pieces (lane l takes pieces
//    l, l + 64, ...), so a wavefront load covers 1 KiB of contiguous row,
//    and a causal softmax skips the pieces that lie wholly past the mask.
//  * row, a workgroup per row (variant 2; 16-byte pieces only): four times
//    the wavefronts per row, a quarter of the pieces each, sums through LDS
//    -- for long rows and few of them; the cost table decides per shape.
//  * column (variant 1): one lane per row, consecutive lanes on consecutive
//    rows, so a layout whose unit-stride dim is a row dim still reads and
//    writes coalesced; the row is streamed twice (three times for
//    LayerNorm's exact two-pass variance).
// Causal softmax: keys k > q (q = index along the second-to-last logical
// dim) get probability exactly 0.  The RED_SUM_* norms read a second
// tensor x1 (own layout) and normalise x + x1, the sum formed on load (a
// residual Add performed in the normalisation's launch); given h, they also
// store the sum there, in y's layout, and normalise the stored (rounded)
// values.  All arithmetic is fp32.
#include <math.h>

#include "dev.h"
#include "launch.h"

namespace fluid {

// v rounded to the storage type T (a stored sum is normalised as stored)
template <typename T>
__device__ __forceinline__ float round_to(float v) {
  if constexpr (sizeof(T) == 2) return bf16_to_f32(f32_to_bf16(v));
  else return v;
}

__device__ __forceinline__ void row_offsets(const RedParams& p, uint32_t row, int32_t& io, int32_t& oo, int32_t& io1,
                                            uint32_t& qi) {
  io = 0; oo = 0; io1 = 0; qi = 0;
  uint32_t rest = row;
#pragma unroll
  for (int d = kMaxDims - 1; d >= 0; --d) {
    if (d < p.nrd) {
      const uint32_t q = fdiv(rest, p.rdiv[d]);
      const uint32_t i = rest - q * p.rext[d];
      rest = q;
      io += (int32_t)i * p.ris[d];
      oo += (int32_t)i * p.ros[d];
      io1 += (int32_t)i * p.ris1[d];
      if (d == p.qdim) qi = i;
    }
  }
}

template <typename T, int NPL, int OP>
__global__ __launch_bounds__(256) void red_row_kernel(RedParams p) {
  constexpr int BOP = red_base_op(OP);
  constexpr bool SUM = red_has_sum(OP);
  const uint32_t row = blockIdx.x * 4u + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= p.nrows) return;  // uniform per wavefront
  int32_t io, oo, io1;
  uint32_t qi;
  row_offsets(p, row, io, oo, io1, qi);
  const uint32_t R = p.R;
  const uint32_t valid = (OP == RED_SOFTMAX && p.causal) ? min(R, qi + 1u) : R;
  float v[NPL];
#pragma unroll
  for (int j = 0; j < NPL; ++j) {
    const uint32_t k = (uint32_t)lane + 64u * j;
    v[j] = k < valid ? Elem<T>::load(p.x, io + (int32_t)k * p.irs) : 0.f;
    if constexpr (SUM) v[j] += k < valid ? Elem<T>::load(p.x1, io1 + (int32_t)k * p.irs1) : 0.f;
  }
  if constexpr (SUM) {
    if (p.h) {
#pragma unroll
      for (int j = 0; j < NPL; ++j) {
        const uint32_t k = (uint32_t)lane + 64u * j;
        v[j] = round_to<T>(v[j]);
        if (k < R) Elem<T>::store(p.h, oo + (int32_t)k * p.ors, v[j]);
      }
    }
  }
  if constexpr (OP == RED_SOFTMAX) {
    float m = -INFINITY;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      const uint32_t k = (uint32_t)lane + 64u * j;
      v[j] *= p.attr;
      if (k < valid) m = fmaxf(m, v[j]);
    }
    m = wave_max(m);
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      const uint32_t k = (uint32_t)lane + 64u * j;
      v[j] = k < valid ? expf(v[j] - m) : 0.f;
      s += v[j];
    }
    s = wave_sum(s);
    const float inv = 1.0f / s;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      const uint32_t k = (uint32_t)lane + 64u * j;
      if (k < R) Elem<T>::store(p.y, oo + (int32_t)k * p.ors, v[j] * inv);
    }
  } else {
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NPL; ++j) s += (BOP == RED_LAYERNORM) ? v[j] : v[j] * v[j];
    s = wave_sum(s);
    const float invR = 1.0f / (float)R;
    float mean = 0.f, rstd;
    if constexpr (BOP == RED_LAYERNORM) {
      mean = s * invR;
      float q = 0.f;
#pragma unroll
      for (int j = 0; j < NPL; ++j) {
        const uint32_t k = (uint32_t)lane + 64u * j;
        const float d = v[j] - mean;
        q += k < R ? d * d : 0.f;
      }
      q = wave_sum(q);
      rstd = 1.0f / sqrtf(q * invR + p.attr);
    } else {
      rstd = 1.0f / sqrtf(s * invR + p.attr);
    }
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      const uint32_t k = (uint32_t)lane + 64u * j;
      if (k < R) {
        float y = (v[j] - mean) * rstd * Elem<T>::load(p.gamma, k);
        if constexpr (BOP == RED_LAYERNORM) y += Elem<T>::load(p.beta, k);
        Elem<T>::store(p.y, oo + (int32_t)k * p.ors, y);
      }
    }
  }
}

// 16-byte piece <-> VEC floats
template <typename T>
struct Piece;
template <>
struct Piece<float> {
  static constexpr int VEC = 4;
  __device__ static __forceinline__ void unpack(const uint4& u, float* f) {
    f[0] = __uint_as_float(u.x); f[1] = __uint_as_float(u.y); f[2] = __uint_as_float(u.z); f[3] = __uint_as_float(u.w);
  }
  __device__ static __forceinline__ uint4 pack(const float* f) {
    return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]), __float_as_uint(f[3]));
  }
};
template <>
struct Piece<uint16_t> {
  static constexpr int VEC = 8;
  __device__ static __forceinline__ void unpack(const uint4& u, float* f) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  __device__ static __forceinline__ uint4 pack(const float* f) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = (uint32_t)f32_to_bf16(f[2 * i]) | ((uint32_t)f32_to_bf16(f[2 * i + 1]) << 16);
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
};

// Row family with 16-byte pieces (unit-stride rows, 16-byte aligned): NC
// pieces per lane, piece c of lane l at l + 64 c.
template <typename T, int NC, int OP>
__global__ __launch_bounds__(256) void red_rowv_kernel(RedParams p) {
  constexpr int BOP = red_base_op(OP);
  constexpr bool SUM = red_has_sum(OP);
  constexpr int VEC = Piece<T>::VEC;
  const uint32_t row = blockIdx.x * 4u + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= p.nrows) return;  // uniform per wavefront
  int32_t io, oo, io1;
  uint32_t qi;
  row_offsets(p, row, io, oo, io1, qi);
  const uint32_t R = p.R;
  const uint32_t valid = (OP == RED_SOFTMAX && p.causal) ? min(R, qi + 1u) : R;
  const T* x = (const T*)p.x + io;
  const T* x1 = (const T*)p.x1 + io1;
  T* y = (T*)p.y + oo;
  float v[NC][VEC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const uint32_t e0 = (uint32_t)(lane + 64 * c) * VEC;
    uint4 u = make_uint4(0, 0, 0, 0);
    if (e0 < valid) u = *(const uint4*)(x + e0);
    Piece<T>::unpack(u, v[c]);
    if constexpr (SUM) {
      uint4 u1 = make_uint4(0, 0, 0, 0);
      if (e0 < valid) u1 = *(const uint4*)(x1 + e0);
      float w[VEC];
      Piece<T>::unpack(u1, w);
#pragma unroll
      for (int i = 0; i < VEC; ++i) v[c][i] += w[i];
    }
    if constexpr (SUM) {
      if (p.h && e0 < R) {
        const uint4 hs = Piece<T>::pack(v[c]);
        *(uint4*)((T*)p.h + oo + e0) = hs;
        Piece<T>::unpack(hs, v[c]);
      }
    }
  }
  // gamma / beta pieces are fetched with the row, not after the reduction,
  // so the row costs one memory round trip
  uint4 gq[OP == RED_SOFTMAX ? 1 : NC], bq[BOP == RED_LAYERNORM ? NC : 1];
  if constexpr (OP != RED_SOFTMAX) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const uint32_t e0 = (uint32_t)(lane + 64 * c) * VEC;
      gq[c] = e0 < R ? *(const uint4*)((const T*)p.gamma + e0) : make_uint4(0, 0, 0, 0);
      if constexpr (BOP == RED_LAYERNORM) bq[c] = e0 < R ? *(const uint4*)((const T*)p.beta + e0) : make_uint4(0, 0, 0, 0);
    }
  }
  if constexpr (OP == RED_SOFTMAX) {
    float m = -INFINITY;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        const uint32_t k = (uint32_t)(lane + 64 * c) * VEC + i;
        v[c][i] *= p.attr;
        if (k < valid) m = fmaxf(m, v[c][i]);
      }
    m = wave_max(m);
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        const uint32_t k = (uint32_t)(lane + 64 * c) * VEC + i;
        v[c][i] = k < valid ? expf(v[c][i] - m) : 0.f;
        s += v[c][i];
      }
    s = wave_sum(s);
    const float inv = 1.0f / s;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const uint32_t e0 = (uint32_t)(lane + 64 * c) * VEC;
      if (e0 < R) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[c][i] *= inv;
        *(uint4*)(y + e0) = Piece<T>::pack(v[c]);
      }
    }
  } else {
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int i = 0; i < VEC; ++i) s += (BOP == RED_LAYERNORM) ? v[c][i] : v[c][i] * v[c][i];
    s = wave_sum(s);
    const float invR = 1.0f / (float)R;
    float mean = 0.f, rstd;
    if constexpr (BOP == RED_LAYERNORM) {
      mean = s * invR;
      float q = 0.f;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const uint32_t e0 = (uint32_t)(lane + 64 * c) * VEC;
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
          const float d = v[c][i] - mean;
          q += e0 < R ? d * d : 0.f;
        }
      }
      q = wave_sum(q);
      rstd = 1.0f / sqrtf(q * invR + p.attr);
    } else {
      rstd = 1.0f / sqrtf(s * invR + p.attr);
    }
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const uint32_t e0 = (uint32_t)(lane + 64 * c) * VEC;
      if (e0 < R) {
        float g[VEC], b[VEC];
        Piece<T>::unpack(gq[c], g);
        if constexpr (BOP == RED_LAYERNORM) Piece<T>::unpack(bq[c], b);
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
          v[c][i] = (v[c][i] - mean) * rstd * g[i];
          if constexpr (BOP == RED_LAYERNORM) v[c][i] += b[i];
        }
        *(uint4*)(y + e0) = Piece<T>::pack(v[c]);
      }
    }
  }
}

// Row family with 16-byte pieces, one 256-thread workgroup per row
// (variant 2: four times the wavefronts of variant 0 per row, a quarter of
// the pieces each).  NC pieces per thread, piece c of thread t at t + 256 c;
// reductions through LDS.
template <typename T, int NC, int OP>
__global__ __launch_bounds__(256) void red_rowb_kernel(RedParams p) {
  constexpr int BOP = red_base_op(OP);
  constexpr bool SUM = red_has_sum(OP);
  constexpr int VEC = Piece<T>::VEC;
  __shared__ float part[4];
  const uint32_t row = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int32_t io, oo, io1;
  uint32_t qi;
  row_offsets(p, row, io, oo, io1, qi);
  const uint32_t R = p.R;
  const uint32_t valid = (OP == RED_SOFTMAX && p.causal) ? min(R, qi + 1u) : R;
  const T* x = (const T*)p.x + io;
  const T* x1 = (const T*)p.x1 + io1;
  T* y = (T*)p.y + oo;
  float v[NC][VEC];
  uint4 gq[OP == RED_SOFTMAX ? 1 : NC], bq[BOP == RED_LAYERNORM ? NC : 1];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const uint32_t e0 = (uint32_t)(tid + 256 * c) * VEC;
    uint4 u = make_uint4(0, 0, 0, 0);
    if (e0 < valid) u = *(const uint4*)(x + e0);
    Piece<T>::unpack(u, v[c]);
    if constexpr (SUM) {
      uint4 u1 = make_uint4(0, 0, 0, 0);
      if (e0 < valid) u1 = *(const uint4*)(x1 + e0);
      float w[VEC];
      Piece<T>::unpack(u1, w);
#pragma unroll
      for (int i = 0; i < VEC; ++i) v[c][i] += w[i];
    }
    if constexpr (SUM) {
      if (p.h && e0 < R) {
        const uint4 hs = Piece<T>::pack(v[c]);
        *(uint4*)((T*)p.h + oo + e0) = hs;
        Piece<T>::unpack(hs, v[c]);
      }
    }
    if constexpr (OP != RED_SOFTMAX) {
      gq[c] = e0 < R ? *(const uint4*)((const T*)p.gamma + e0) : make_uint4(0, 0, 0, 0);
      if constexpr (BOP == RED_LAYERNORM) bq[c] = e0 < R ? *(const uint4*)((const T*)p.beta + e0) : make_uint4(0, 0, 0, 0);
    }
  }
  // block-wide sum / max: wavefront butterflies, then the four partials
  auto block_sum = [&](float a) {
    a = wave_sum(a);
    if (lane == 0) part[wave] = a;
    __syncthreads();
    const float r = part[0] + part[1] + part[2] + part[3];
    __syncthreads();
    return r;
  };
  auto block_max = [&](float a) {
    a = wave_max(a);
    if (lane == 0) part[wave] = a;
    __syncthreads();
    const float r = fmaxf(fmaxf(part[0], part[1]), fmaxf(part[2], part[3]));
    __syncthreads();
    return r;
  };
  if constexpr (OP == RED_SOFTMAX) {
    float m = -INFINITY;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        const uint32_t k = (uint32_t)(tid + 256 * c) * VEC + i;
        v[c][i] *= p.attr;
        if (k < valid) m = fmaxf(m, v[c][i]);
      }
    m = block_max(m);
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        const uint32_t k = (uint32_t)(tid + 256 * c) * VEC + i;
        v[c][i] = k < valid ? expf(v[c][i] - m) : 0.f;
        s += v[c][i];
      }
    s = block_sum(s);
    const float inv = 1.0f / s;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const uint32_t e0 = (uint32_t)(tid + 256 * c) * VEC;
      if (e0 < R) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[c][i] *= inv;
        *(uint4*)(y + e0) = Piece<T>::pack(v[c]);
      }
    }
  } else {
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int i = 0; i < VEC; ++i) s += (BOP == RED_LAYERNORM) ? v[c][i] : v[c][i] * v[c][i];
    s = block_sum(s);
    const float invR = 1.0f / (float)R;
    float mean = 0.f, rstd;
    if constexpr (BOP == RED_LAYERNORM) {
      mean = s * invR;
      float q = 0.f;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const uint32_t e0 = (uint32_t)(tid + 256 * c) * VEC;
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
          const float d = v[c][i] - mean;
          q += e0 < R ? d * d : 0.f;
        }
      }
      q = block_sum(q);
      rstd = 1.0f / sqrtf(q * invR + p.attr);
    } else {
      rstd = 1.0f / sqrtf(s * invR + p.attr);
    }
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const uint32_t e0 = (uint32_t)(tid + 256 * c) * VEC;
      if (e0 < R) {
        float g[VEC], b[VEC];
        Piece<T>::unpack(gq[c], g);
        if constexpr (BOP == RED_LAYERNORM) Piece<T>::unpack(bq[c], b);
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
          v[c][i] = (v[c][i] - mean) * rstd * g[i];
          if constexpr (BOP == RED_LAYERNORM) v[c][i] += b[i];
        }
        *(uint4*)(y + e0) = Piece<T>::pack(v[c]);
      }
    }
  }
}

template <typename T, int OP>
__global__ __launch_bounds__(256) void red_col_kernel(RedParams p) {
  constexpr int BOP = red_base_op(OP);
  constexpr bool SUM = red_has_sum(OP);
  const uint32_t row = blockIdx.x * 256u + threadIdx.x;
  if (row >= p.nrows) return;
  int32_t io, oo, io1;
  uint32_t qi;
  row_offsets(p, row, io, oo, io1, qi);
  const uint32_t R = p.R;
  // element k of the row (of the sum for RED_SUM_*)
  auto ldx = [&](uint32_t k) {
    float a = Elem<T>::load(p.x, io + (int32_t)k * p.irs);
    if constexpr (SUM) {
      a += Elem<T>::load(p.x1, io1 + (int32_t)k * p.irs1);
      if (p.h) a = round_to<T>(a);
    }
    return a;
  };
  if constexpr (SUM) {
    if (p.h)
      for (uint32_t k = 0; k < R; ++k) Elem<T>::store(p.h, oo + (int32_t)k * p.ors, ldx(k));
  }
  if constexpr (OP == RED_SOFTMAX) {
    const uint32_t valid = p.causal ? min(R, qi + 1u) : R;
    float m = -INFINITY, s = 0.f;
    for (uint32_t k = 0; k < valid; ++k) {
      const float z = p.attr * ldx(k);
      if (z > m) {
        s = s * expf(m - z) + 1.f;
        m = z;
      } else {
        s += expf(z - m);
      }
    }
    const float inv = 1.0f / s;
    for (uint32_t k = 0; k < R; ++k) {
      float y = 0.f;
      if (k < valid) y = expf(p.attr * ldx(k) - m) * inv;
      Elem<T>::store(p.y, oo + (int32_t)k * p.ors, y);
    }
  } else {
    const float invR = 1.0f / (float)R;
    float mean = 0.f, rstd;
    if constexpr (BOP == RED_LAYERNORM) {
      float s = 0.f;
      for (uint32_t k = 0; k < R; ++k) s += ldx(k);
      mean = s * invR;
      float q = 0.f;
      for (uint32_t k = 0; k < R; ++k) {
        const float d = ldx(k) - mean;
        q += d * d;
      }
      rstd = 1.0f / sqrtf(q * invR + p.attr);
    } else {
      float q = 0.f;
      for (uint32_t k = 0; k < R; ++k) {
        const float x = ldx(k);
        q += x * x;
      }
      rstd = 1.0f / sqrtf(q * invR + p.attr);
    }
    for (uint32_t k = 0; k < R; ++k) {
      float y = (ldx(k) - mean) * rstd * Elem<T>::load(p.gamma, k);
      if constexpr (BOP == RED_LAYERNORM) y += Elem<T>::load(p.beta, k);
      Elem<T>::store(p.y, oo + (int32_t)k * p.ors, y);
    }
  }
}

// Column family with the row held in registers: a workgroup of 16
// wavefronts owns RT consecutive rows.  Lane l of a wavefront works on row
// RT b + l % RT at the k phase q = l / RT (one of KQ = 64 / RT), so one load
// by a wavefront reads KQ runs of RT neighbouring rows.  Wavefront w holds the
// k in [w KQ KPL, (w + 1) KQ KPL) with k = w KQ KPL + q + KQ j.  The input is
// read once; per-row sums and maxima are combined over the KQ phases with
// lane shuffles and over the 16 wavefronts through LDS, in a fixed order.
template <typename T, int RT, int KPL, int OP>
__global__ __launch_bounds__(1024) void red_colb_kernel(RedParams p) {
  constexpr int BOP = red_base_op(OP);
  constexpr bool SUM = red_has_sum(OP);
  constexpr int KQ = 64 / RT;
  __shared__ float part[16][RT];
  // the wavefront index is uniform: keep it in a scalar register
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane % RT, q = lane / RT;
  // Consecutive workgroups go to the 8 XCDs in turn.  A tile's run of RT
  // rows covers RT * sizeof(T) bytes, so G = 128 / (RT sizeof(T)) tiles share
  // one 128-byte line: place runs of G consecutive tiles on one XCD (tile t
  // on XCD (t / G) % 8), so that a line is fetched into, and written back
  // from, a single L2.
  constexpr uint32_t G = RT * sizeof(T) >= 128 ? 1u : 128u / (RT * (uint32_t)sizeof(T));
  uint32_t tile = blockIdx.x;
  if (G > 1 && gridDim.x % (8u * G) == 0) {
    const uint32_t x = tile & 7u, i = tile >> 3;
    tile = ((i / G) * 8u + x) * G + i % G;
  }
  const uint32_t row = tile * (uint32_t)RT + (uint32_t)r;
  // rows past the end compute on the last row and store nothing
  const bool live = row < p.nrows;
  int32_t io, oo, io1;
  uint32_t qi;
  row_offsets(p, live ? row : p.nrows - 1u, io, oo, io1, qi);
  const uint32_t R = p.R;
  const uint32_t valid = (OP == RED_SOFTMAX && p.causal) ? min(R, qi + 1u) : R;
  const uint32_t kb = (uint32_t)wave * (KQ * KPL);  // uniform
  const uint32_t kl = kb + (uint32_t)q;             // this lane's first k
  // Only a wavefront whose k range runs past R, or a causal softmax, masks
  // single loads and stores; the test is uniform across the wavefront.
  const bool masked = (OP == RED_SOFTMAX && p.causal) || kb + KQ * KPL > R;
  // Buffer loads and stores: the lane's row offset plus its phase is the one
  // per-lane address register, the uniform part of k a scalar offset.  Byte
  // offsets stay below 2^31 (the launcher checks), so a lane that must not
  // load or store points at offset 2^31, which the buffer range check turns
  // into a zero load or a dropped store.
  constexpr uint32_t ES = sizeof(T);
  constexpr uint32_t OOB = 0x80000000u;
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p.x), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t ry = __builtin_amdgcn_make_buffer_rsrc(p.y, 0, 0x7fffffff, 0x00020000);
  const uint32_t xstep = (uint32_t)p.irs * ES, ystep = (uint32_t)p.ors * ES;
  const uint32_t xo = (uint32_t)io * ES + (uint32_t)q * xstep;
  // the second summand (RED_SUM_*): its own resource, lane offset and step
  const __amdgpu_buffer_rsrc_t rx1 =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(SUM ? p.x1 : p.x), 0, 0x7fffffff, 0x00020000);
  const uint32_t xstep1 = (uint32_t)p.irs1 * ES;
  const uint32_t xo1 = (uint32_t)io1 * ES + (uint32_t)q * xstep1;
  const uint32_t yo = live ? (uint32_t)oo * ES + (uint32_t)q * ystep : OOB;
  auto ld1 = [&](const __amdgpu_buffer_rsrc_t& rs, uint32_t vo, uint32_t so) {
    if constexpr (ES == 4) return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, vo, so, 0));
    else return bf16_to_f32(__builtin_amdgcn_raw_buffer_load_b16(rs, vo, so, 0));
  };
  // element j of the lane (of the sum for RED_SUM_*); vo / vo1 the lane's
  // offsets, or OOB for a masked load
  auto ld = [&](int j, uint32_t vo, uint32_t vo1) {
    float a = ld1(rx, vo, (kb + (uint32_t)(KQ * j)) * xstep);
    if constexpr (SUM) a += ld1(rx1, vo1, (kb + (uint32_t)(KQ * j)) * xstep1);
    return a;
  };
  auto st1 = [&](int j, uint32_t vo, float y) {
    const uint32_t so = (kb + (uint32_t)(KQ * j)) * ystep;
    if constexpr (ES == 4) __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, y), ry, vo, so, 0);
    else __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16(y), ry, vo, so, 0);
  };
  float v[KPL];
  if (masked) {
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      const bool in = kl + KQ * j < valid;
      v[j] = ld(j, in ? xo : OOB, in ? xo1 : OOB);
    }
  } else {
#pragma unroll
    for (int j = 0; j < KPL; ++j) v[j] = ld(j, xo, xo1);
  }
  if constexpr (SUM) {
    if (p.h) {
      // the sum's own output: y's offsets, through its own resource
      const __amdgpu_buffer_rsrc_t rh = __builtin_amdgcn_make_buffer_rsrc(p.h, 0, 0x7fffffff, 0x00020000);
#pragma unroll
      for (int j = 0; j < KPL; ++j) {
        v[j] = round_to<T>(v[j]);
        const uint32_t vo = !masked || kl + KQ * j < R ? yo : OOB;
        const uint32_t so = (kb + (uint32_t)(KQ * j)) * ystep;
        if constexpr (ES == 4) __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v[j]), rh, vo, so, 0);
        else __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16(v[j]), rh, vo, so, 0);
      }
    }
  }
  // y[j] for every j, stored where k < R
  auto store_all = [&](auto&& yfun) {
    if (masked) {
#pragma unroll
      for (int j = 0; j < KPL; ++j) st1(j, kl + KQ * j < R ? yo : OOB, yfun(j));
    } else {
#pragma unroll
      for (int j = 0; j < KPL; ++j) st1(j, yo, yfun(j));
    }
  };
  auto combine = [&](float a, bool take_max) {
#pragma unroll
    for (int o = RT; o < 64; o <<= 1) {
      const float b = __shfl_xor(a, o, 64);
      a = take_max ? fmaxf(a, b) : a + b;
    }
    if (q == 0) part[wave][r] = a;
    __syncthreads();
    float t = part[0][r];
#pragma unroll
    for (int w = 1; w < 16; ++w) t = take_max ? fmaxf(t, part[w][r]) : t + part[w][r];
    __syncthreads();
    return t;
  };
  if constexpr (OP == RED_SOFTMAX) {
    float m = -INFINITY;
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      v[j] *= p.attr;
      if (kl + KQ * j < valid) m = fmaxf(m, v[j]);
    }
    m = combine(m, true);
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      v[j] = kl + KQ * j < valid ? expf(v[j] - m) : 0.f;
      sum += v[j];
    }
    sum = combine(sum, false);
    const float inv = 1.0f / sum;
    store_all([&](int j) { return v[j] * inv; });
  } else {
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < KPL; ++j) sum += (BOP == RED_LAYERNORM) ? v[j] : v[j] * v[j];
    sum = combine(sum, false);
    const float invR = 1.0f / (float)R;
    float mean = 0.f, rstd;
    if constexpr (BOP == RED_LAYERNORM) {
      mean = sum * invR;
      float qs = 0.f;
#pragma unroll
      for (int j = 0; j < KPL; ++j) {
        const float d = v[j] - mean;
        qs += kl + KQ * j < R ? d * d : 0.f;
      }
      qs = combine(qs, false);
      rstd = 1.0f / sqrtf(qs * invR + p.attr);
    } else {
      rstd = 1.0f / sqrtf(sum * invR + p.attr);
    }
    // gamma and beta are read at min(k, R - 1): in bounds for k past the row
    store_all([&](int j) {
      const uint32_t kc = min(kl + KQ * j, R - 1u);
      float y = (v[j] - mean) * rstd * Elem<T>::load(p.gamma, kc);
      if constexpr (BOP == RED_LAYERNORM) y += Elem<T>::load(p.beta, kc);
      return y;
    });
  }
}

namespace {

template <typename T, int OP>
hipError_t red_dispatch_op(const NodeKernel& k, hipStream_t s) {
  const RedParams& p = k.red;
  if (k.family == KF_RED_COL) {
    // register-resident variant: byte offsets below 2^31, at most 32 values
    // per lane; 64-row tiles where they still give 512 workgroups, else 16-
    // or (for rows longer than 2048) 8-row tiles
    const bool fits = (uint64_t)p.nrows * p.R * sizeof(T) < (uint64_t(1) << 31);
    const int rt = ((p.nrows + 63u) / 64u >= 512u && p.R <= 512u) ? 64 : p.R <= 2048u ? 16 : 8;
    const uint32_t kpl = (p.R + 16u * (64 / rt) - 1u) / (16u * (64 / rt));
#define FLUID_COLB(RTv, K) \
  hipLaunchKernelGGL((red_colb_kernel<T, RTv, K, OP>), dim3((p.nrows + RTv - 1u) / RTv), dim3(1024), 0, s, p)
#define FLUID_COLB_RT(RTv)                \
  if (kpl <= 1) FLUID_COLB(RTv, 1);       \
  else if (kpl <= 2) FLUID_COLB(RTv, 2);  \
  else if (kpl <= 4) FLUID_COLB(RTv, 4);  \
  else if (kpl <= 8) FLUID_COLB(RTv, 8);  \
  else if (kpl <= 16) FLUID_COLB(RTv, 16); \
  else FLUID_COLB(RTv, 32);
    if (!fits || kpl > 32) {
      hipLaunchKernelGGL((red_col_kernel<T, OP>), dim3((p.nrows + 255u) / 256u), dim3(256), 0, s, p);
    } else if (rt == 64) {
      FLUID_COLB_RT(64)
    } else if (rt == 16) {
      FLUID_COLB_RT(16)
    } else {
      FLUID_COLB_RT(8)
    }
#undef FLUID_COLB_RT
#undef FLUID_COLB
    return hipGetLastError();
  }
  const dim3 grid((p.nrows + 3u) / 4u);
  if (k.vec > 1) {
    const uint32_t pieces = p.R / Piece<T>::VEC;
    // variant 2: a workgroup per row (rows of at most 4096 values: at most
    // 4 pieces per thread)
    if (k.red_block) {
      const uint32_t ncb = (pieces + 255u) / 256u;
      const dim3 gb(p.nrows);
      if (ncb <= 1) hipLaunchKernelGGL((red_rowb_kernel<T, 1, OP>), gb, dim3(256), 0, s, p);
      else if (ncb <= 2) hipLaunchKernelGGL((red_rowb_kernel<T, 2, OP>), gb, dim3(256), 0, s, p);
      else if (ncb <= 4) hipLaunchKernelGGL((red_rowb_kernel<T, 4, OP>), gb, dim3(256), 0, s, p);
      else return hipErrorInvalidValue;
      return hipGetLastError();
    }
    const uint32_t nc = (pieces + 63u) / 64u;
    if (nc <= 1) hipLaunchKernelGGL((red_rowv_kernel<T, 1, OP>), grid, dim3(256), 0, s, p);
    else if (nc <= 2) hipLaunchKernelGGL((red_rowv_kernel<T, 2, OP>), grid, dim3(256), 0, s, p);
    else if (nc <= 4) hipLaunchKernelGGL((red_rowv_kernel<T, 4, OP>), grid, dim3(256), 0, s, p);
    else if (nc <= 8) hipLaunchKernelGGL((red_rowv_kernel<T, 8, OP>), grid, dim3(256), 0, s, p);
    else if (nc <= 16) hipLaunchKernelGGL((red_rowv_kernel<T, 16, OP>), grid, dim3(256), 0, s, p);
    else return hipErrorInvalidValue;
    return hipGetLastError();
  }
  const uint32_t npl = (p.R + 63u) / 64u;
  if (npl <= 1) hipLaunchKernelGGL((red_row_kernel<T, 1, OP>), grid, dim3(256), 0, s, p);
  else if (npl <= 2) hipLaunchKernelGGL((red_row_kernel<T, 2, OP>), grid, dim3(256), 0, s, p);
  else if (npl <= 4) hipLaunchKernelGGL((red_row_kernel<T, 4, OP>), grid, dim3(256), 0, s, p);
  else if (npl <= 8) hipLaunchKernelGGL((red_row_kernel<T, 8, OP>), grid, dim3(256), 0, s, p);
  else if (npl <= 16) hipLaunchKernelGGL((red_row_kernel<T, 16, OP>), grid, dim3(256), 0, s, p);
  else if (npl <= 32) hipLaunchKernelGGL((red_row_kernel<T, 32, OP>), grid, dim3(256), 0, s, p);
  else if (npl <= 64) hipLaunchKernelGGL((red_row_kernel<T, 64, OP>), grid, dim3(256), 0, s, p);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

template <typename T>
hipError_t red_dispatch(const NodeKernel& k, hipStream_t s) {
  switch (k.red.op) {
    case RED_SOFTMAX: return red_dispatch_op<T, RED_SOFTMAX>(k, s);
    case RED_LAYERNORM: return red_dispatch_op<T, RED_LAYERNORM>(k, s);
    case RED_RMSNORM: return red_dispatch_op<T, RED_RMSNORM>(k, s);
    case RED_SUM_LAYERNORM: return red_dispatch_op<T, RED_SUM_LAYERNORM>(k, s);
    case RED_SUM_RMSNORM: return red_dispatch_op<T, RED_SUM_RMSNORM>(k, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_reduce(const NodeKernel& k, hipStream_t s) {
  return k.dtype == DT_BF16 ? red_dispatch<uint16_t>(k, s) : red_dispatch<float>(k, s);
}

}  // namespace fluid
