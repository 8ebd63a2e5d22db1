// Measured ceilings of the chip, for the roofline fractions the benchmark
// reports next to the datasheet peaks: a dependent-free loop of bf16 MFMAs
// (v_mfma_f32_16x16x32_bf16, the instruction of every bf16 GEMM and of the
// attention kernel) and a 16-byte-per-lane streaming copy.
#include "common.h"
#include "../../include/dlm.h"

namespace dlm {

constexpr int kCeilChains = 8;    // independent accumulators per wave

__global__ __launch_bounds__(256) void ceiling_mfma_kernel(int iters, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (bf16)(0.001f * (float)((lane + e) & 7));
    b[e] = (bf16)(0.001f * (float)((lane * 3 + e) & 7));
  }
  // every accumulator component seeded with a different run-time value, so
  // that no two chains or components are provably equal and the compiler
  // keeps eight independent accumulators in place
  auto seed = [&](int j) {
    const float x = (float)(lane * 32 + 4 * j) * 1e-30f;
    return f32x4{x, x + 1e-30f, x + 2e-30f, x + 3e-30f};
  };
  f32x4 c0 = seed(0), c1 = seed(1), c2 = seed(2), c3 = seed(3), c4 = seed(4), c5 = seed(5),
        c6 = seed(6), c7 = seed(7);
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {   // 32 MFMAs per trip: loop overhead off the MFMA pipe
      c0 = mfma16_bf16(a, b, c0);
      c1 = mfma16_bf16(a, b, c1);
      c2 = mfma16_bf16(a, b, c2);
      c3 = mfma16_bf16(a, b, c3);
      c4 = mfma16_bf16(a, b, c4);
      c5 = mfma16_bf16(a, b, c5);
      c6 = mfma16_bf16(a, b, c6);
      c7 = mfma16_bf16(a, b, c7);
    }
  }
  const f32x4 t = ((c0 + c1) + (c2 + c3)) + ((c4 + c5) + (c6 + c7));
  float s = t[0] + t[1] + t[2] + t[3];
  s = wave_sum(s);
  if (lane == 0) out[blockIdx.x * 4 + (threadIdx.x >> 6)] = s;
}

// four independent 16-byte loads in flight per lane before their stores
__global__ __launch_bounds__(256) void ceiling_copy_kernel(const u32x4* __restrict__ src,
                                                           u32x4* __restrict__ dst, size_t n) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < n; i += 4 * stride) {
    const u32x4 v0 = src[i], v1 = src[i + stride], v2 = src[i + 2 * stride], v3 = src[i + 3 * stride];
    dst[i] = v0;
    dst[i + stride] = v1;
    dst[i + 2 * stride] = v2;
    dst[i + 3 * stride] = v3;
  }
  for (; i < n; i += stride) dst[i] = src[i];
}

}  // namespace dlm

extern "C" dlm_status dlm_ceiling_mfma(int32_t n_blocks, int32_t iters, float* out,
                                       double* flop_out, void* stream) {
  if (n_blocks <= 0 || iters <= 0 || !out) return DLM_EINVAL;
  hipStream_t st = (hipStream_t)stream;
  hipLaunchKernelGGL(dlm::ceiling_mfma_kernel, dim3(n_blocks), dim3(256), 0, st, iters, out);
  if (hipGetLastError() != hipSuccess) return DLM_EHIP;
  if (flop_out)
    *flop_out = (double)n_blocks * 4 * iters * 4 * dlm::kCeilChains * (2.0 * 16 * 16 * 32);
  return DLM_OK;
}

extern "C" dlm_status dlm_ceiling_copy(const void* src, void* dst, size_t bytes, void* stream) {
  if (!src || !dst || bytes % 16 != 0 || ((uintptr_t)src | (uintptr_t)dst) % 16 != 0)
    return DLM_EINVAL;
  if (bytes == 0) return DLM_OK;
  hipStream_t st = (hipStream_t)stream;
  // 8 blocks of 256 lanes per CU, grid-stride over 16-byte elements
  hipLaunchKernelGGL(dlm::ceiling_copy_kernel, dim3(256 * 8), dim3(256), 0, st,
                     (const dlm::u32x4*)src, (dlm::u32x4*)dst, bytes / 16);
  return hipGetLastError() == hipSuccess ? DLM_OK : DLM_EHIP;
}
