// Device implementation of the seeded weight generator (same definition as
// synth/__init__.py): SplitMix64 stream per (seed, tensor id), Box-Muller in
// fp64, rounded fp64 -> fp32 -> (bf16) with round-to-nearest-even. It only
// draws inputs; none of the denoising arithmetic lives here.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;

__host__ __device__ inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ inline uint16_t f32_to_bf16_bits(float f) {
  uint32_t b = __float_as_uint(f);
  return (uint16_t)((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

__global__ void fill_normal_kernel(void* dst, long n, int dtype, uint64_t key, long start,
                                   double stdv) {
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n;
       i += (long)gridDim.x * blockDim.x) {
    const uint64_t w = mix64(key + (uint64_t)(start + i + 1) * kGolden);
    const double u1 = ((double)(w >> 32) + 0.5) * (1.0 / 4294967296.0);
    const double u2 = ((double)(w & 0xFFFFFFFFull) + 0.5) * (1.0 / 4294967296.0);
    const double z = stdv * (sqrt(-2.0 * log(u1)) * cos(2.0 * 3.141592653589793 * u2));
    const float f = (float)z;
    if (dtype == 1)
      reinterpret_cast<uint16_t*>(dst)[i] = f32_to_bf16_bits(f);
    else
      reinterpret_cast<float*>(dst)[i] = f;
  }
}

__global__ void fill_const_kernel(float* dst, long n, float v) {
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n;
       i += (long)gridDim.x * blockDim.x)
    dst[i] = v;
}

}  // namespace

extern "C" {

// Fill n elements (dtype 0 = fp32, 1 = bf16) with elements start..start+n-1 of
// tensor `tid` under `seed`. Returns a hipError_t code.
int synth_fill_normal(void* dst, long n, int dtype, uint64_t seed, uint64_t tid, long start,
                      double stdv, void* stream) {
  if (n <= 0) return 0;
  const uint64_t key = mix64(mix64(seed) ^ tid);
  const long blocks = (n + 255) / 256 < 65536 ? (n + 255) / 256 : 65536;
  hipLaunchKernelGGL(fill_normal_kernel, dim3((unsigned)blocks), dim3(256), 0,
                     reinterpret_cast<hipStream_t>(stream), dst, n, dtype, key, start, stdv);
  return (int)hipGetLastError();
}

int synth_fill_const(float* dst, long n, float v, void* stream) {
  if (n <= 0) return 0;
  const long blocks = (n + 255) / 256 < 65536 ? (n + 255) / 256 : 65536;
  hipLaunchKernelGGL(fill_const_kernel, dim3((unsigned)blocks), dim3(256), 0,
                     reinterpret_cast<hipStream_t>(stream), dst, n, v);
  return (int)hipGetLastError();
}

}
