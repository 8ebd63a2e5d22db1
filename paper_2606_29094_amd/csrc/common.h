// Shared device helpers for the gfx950 kernels: element types, bf16
// conversion, MFMA fragment types and wavefront reductions.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dlm {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
// fp32 -> bf16, round to nearest even (the compiler's conversion on gfx950)
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }

// ---- wavefront reductions (64 lanes) ----
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// ---- MFMA wrappers ----
// 16x16x32 bf16: lane l supplies A[row = l%16][k = 8*(l/16) .. +7] and
// B[col = l%16][k = 8*(l/16) .. +7]; D[row = 4*(l/16) + i][col = l%16] = acc[i].
__device__ __forceinline__ f32x4 mfma16_bf16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
// 32x32x16 bf16: lane l supplies A[row = l%32][k = 8*(l/32) .. +7] and
// B[col = l%32][k = 8*(l/32) .. +7]; D[row = 8*(i/4) + 4*(l/32) + i%4][col = l%32] = acc[i].
__device__ __forceinline__ f32x16 mfma32_bf16(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ int mf32_row(int i, int lane) { return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3); }
// 16x16x4 fp32: lane l supplies A[row = l%16][k = l/16], B[col = l%16][k = l/16].
__device__ __forceinline__ f32x4 mfma16_f32(float a, float b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__host__ __device__ constexpr int ceil_div(int a, int b) { return (a + b - 1) / b; }

// ---- kernel launches ----
// Timing hook of the library's profiler: when the host sets start/stop (one
// launch at a time), the next kernel launched through DLM_LAUNCH carries the
// two events in its own dispatch, so they time the kernel itself (no extra
// commands in the stream), and the hook is cleared.
struct LaunchTiming { hipEvent_t start = nullptr, stop = nullptr; };
extern thread_local LaunchTiming g_launch_timing;
#define DLM_LAUNCH(kernel, grid, block, shmem, stream, ...)                                     \
  do {                                                                                         \
    if (::dlm::g_launch_timing.start) {                                                        \
      const ::dlm::LaunchTiming lt_ = ::dlm::g_launch_timing;                                  \
      ::dlm::g_launch_timing = ::dlm::LaunchTiming{};                                          \
      hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, lt_.start, lt_.stop, 0,        \
                            __VA_ARGS__);                                                      \
    } else {                                                                                   \
      hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);                     \
    }                                                                                          \
  } while (0)

// XCDs the dispatcher spreads a launch's blocks over (block i to XCD i mod 8);
// each has its own L2
constexpr int kXcds = 8;

// ---- direct global -> LDS loads (global_load_lds_dwordx4) ----
// One wave instruction moves 1 KB: lane l reads 16 bytes at its own global
// address and writes them to LDS bytes [16 l, 16 l + 16) after the wave's
// destination base. Completion is counted by vmcnt like any global load.
typedef __attribute__((address_space(1))) const void* gptr_t;
typedef __attribute__((address_space(3))) void* lptr_t;

__device__ __forceinline__ void load_lds16(const void* src, void* lds_wave_base) {
  __builtin_amdgcn_global_load_lds((gptr_t)src, (lptr_t)lds_wave_base, 16, 0, 0);
}

// wait until at most N vector-memory operations of this wave are in flight
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // gfx9 s_waitcnt: vmcnt in [3:0] and [15:14]; expcnt (7) and lgkmcnt (15) not waited on
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

}  // namespace dlm
