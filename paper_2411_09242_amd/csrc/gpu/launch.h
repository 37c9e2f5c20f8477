// Kernel launchers (one per kernel family); each returns the launch status.
#pragma once

#include <hip/hip_runtime.h>

#include "../host/dispatch.h"

namespace fluid {

hipError_t launch_elementwise(const NodeKernel& k, hipStream_t s);
hipError_t launch_rope(const NodeKernel& k, hipStream_t s);
hipError_t launch_reduce(const NodeKernel& k, hipStream_t s);
hipError_t launch_gemm(const NodeKernel& k, hipStream_t s);
hipError_t launch_gemm_bf16_pipe(const NodeKernel& k, hipStream_t s);
hipError_t launch_gemm_bf16_dl(const NodeKernel& k, hipStream_t s);
hipError_t launch_gemm_bf16_qk(const NodeKernel& k, hipStream_t s);
hipError_t launch_gemm_f32_dl(const NodeKernel& k, hipStream_t s);
hipError_t launch_gemm_f32_ring(const NodeKernel& k, hipStream_t s);
// One launch for the G.n products of G, all of k's tile, operand modes and
// epilogue instance (fp32 tiles 6 and 7).
hipError_t launch_gemm_f32_dl_group(const NodeKernel& k, const GemmGroup& G, hipStream_t s);
hipError_t launch_fill(void* p, uint64_t bytes, uint32_t seed, hipStream_t s);
hipError_t launch_window(const NodeKernel& k, hipStream_t s);
hipError_t launch_conv(const NodeKernel& k, hipStream_t s);

inline hipError_t launch_node_kernel(const NodeKernel& k, hipStream_t s) {
  switch (k.family) {
    case KF_EW:
    case KF_EW_TILED: return launch_elementwise(k, s);
    case KF_ROPE: return launch_rope(k, s);
    case KF_RED_ROW:
    case KF_RED_COL: return launch_reduce(k, s);
    case KF_GEMM: return launch_gemm(k, s);
    case KF_WIN: return launch_window(k, s);
    case KF_CONV: return launch_conv(k, s);
    default: return hipSuccess;
  }
}

}  // namespace fluid
