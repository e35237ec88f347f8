// GPU evaluation of the counter-based synthetic gradient values defined in
// workloads/rng.py (SplitMix64 streams; uniform (-1, 1) cell midpoints, or the
// Irwin-Hall sum of twelve 21-bit uniforms scaled by sigma).  Integer arithmetic
// plus one correctly rounded binary32 multiply, so the bits match the numpy
// definition exactly.  Input generation only: no part of the allreduce is here.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

__host__ __device__ __forceinline__ uint64_t mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// dist 0: uniform (-1, 1); dist 1: normal(0, sigma)
__global__ __launch_bounds__(256) void fill_kernel(float* dst, int64_t n, uint64_t seed, int64_t first, int dist,
                                                   float sigma) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n; e += stride) {
    const uint64_t i = (uint64_t)(first + e);
    const uint64_t base = seed + (4 * i + 1) * kGamma;
    float v;
    if (dist == 0) {
      const int64_t k = (int64_t)(mix(base) >> 40);
      v = (float)(int32_t)(2 * k + 1 - (1 << 24)) * 0x1p-24f;
    } else {
      int64_t total = 0;
      for (int j = 0; j < 4; ++j) {
        const uint64_t d = mix(base + (uint64_t)j * kGamma);
        total += (int64_t)(d & 0x1FFFFF) + (int64_t)((d >> 21) & 0x1FFFFF) + (int64_t)((d >> 42) & 0x1FFFFF);
      }
      const float z = (float)(int32_t)(total + 6 - 6 * (1 << 21)) * 0x1p-21f;
      v = z * sigma;
    }
    dst[e] = v;
  }
}

}  // namespace

extern "C" int wl_fill_f32(float* dst, int64_t n, uint64_t key, int64_t first_index, int dist, float sigma,
                           void* stream) {
  if (n < 0 || (n > 0 && !dst) || first_index < 0 || (dist != 0 && dist != 1)) return -1;
  if (n == 0) return 0;
  const uint64_t seed = mix(key + kGamma);  // the key's stream seed
  int64_t blocks = (n + 1023) / 1024;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, static_cast<hipStream_t>(stream), dst, n,
                     seed, first_index, dist, sigma);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}
