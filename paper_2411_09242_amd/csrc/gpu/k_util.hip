// Scratch fill used before measuring kernels: every 16-bit half-word gets a
// bfloat16 value in [-1, 1), so the bytes read as fp32 or as bf16 are finite
// and of ordinary magnitude (no NaN/denormal paths while timing).
#include "dev.h"
#include "launch.h"

namespace fluid {

__global__ __launch_bounds__(256) void fill_kernel(uint32_t* p, uint64_t words, uint32_t seed) {
  const uint64_t step = (uint64_t)gridDim.x * 256u;
  for (uint64_t i = (uint64_t)blockIdx.x * 256u + threadIdx.x; i < words; i += step) {
    uint32_t h = (uint32_t)i * 2654435761u ^ seed;
    h ^= h >> 15;
    h *= 2246822519u;
    h ^= h >> 13;
    // exponent 125: magnitudes in [0.25, 0.5), random sign and mantissa
    const uint32_t lo = 0x3E80u | (h & 0x807Fu);
    const uint32_t hi = 0x3E80u | ((h >> 16) & 0x807Fu);
    p[i] = lo | (hi << 16);
  }
}

hipError_t launch_fill(void* p, uint64_t bytes, uint32_t seed, hipStream_t s) {
  const uint64_t words = bytes / 4;
  if (words == 0) return hipSuccess;
  uint64_t blocks = (words + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  hipLaunchKernelGGL(fill_kernel, dim3((uint32_t)blocks), dim3(256), 0, s, (uint32_t*)p, words, seed);
  return hipGetLastError();
}

}  // namespace fluid
