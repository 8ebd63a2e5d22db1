// NT GEMM on the gfx950 matrix cores: C[m][n] = sum_k A[m][k] * B[n][k],
// A [M, K] and B [N, K] both K-contiguous (activations x weights^T), fp32
// accumulation, with the work after the contraction fused into a tile
// epilogue:
//   * store fp32 (split-K partial slices),
//   * add into an fp32 residual stream,
//   * SwiGLU: gate and up columns computed in the same tile, silu(g) * u stored,
//   * fused LM head: per row, the online (max, sum of exp, lowest argmax) of the
//     scaled logits over the tile's vocabulary columns; logits are never stored,
//   * scaled fp32 store (test hook).
//
// Tiling: 256 threads (4 waves), block tile BM x BN, k-tile of 128 bytes per
// row (64 bf16 or 32 fp32), double-buffered in LDS with 16-byte row padding so
// that 16 lanes reading 16 rows hit distinct banks; global loads are 16-byte
// vectors, prefetched into registers one k-tile ahead. bf16 uses
// v_mfma_f32_16x16x32_bf16, fp32 uses v_mfma_f32_16x16x4_f32 (four per 16-byte
// fragment, the k order is the same permutation for A and B).
#include "common.h"
#include "kernels.h"

namespace dlm {

template <typename T> struct MfmaTraits;
template <> struct MfmaTraits<bf16> {
  static constexpr int kVec = 8;
  __device__ __forceinline__ static f32x4 mma(const u32x4& a, const u32x4& b, f32x4 c) {
    return mfma16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c);
  }
};
template <> struct MfmaTraits<float> {
  static constexpr int kVec = 4;
  __device__ __forceinline__ static f32x4 mma(const u32x4& a, const u32x4& b, f32x4 c) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      c = mfma16_f32(__uint_as_float(a[j]), __uint_as_float(b[j]), c);
    return c;
  }
};

constexpr int kRowBytes = 128;          // k-tile bytes per row
constexpr int kLdsRow = kRowBytes + 16; // padded LDS row stride

// ------------------------------------------------------------ epilogues --
// Each epilogue sees the wave's accumulators: acc[fm][fn][i] is the value at
// row m0 + fm*16 + 4*(lane/16) + i, column n0 + fn*16 + lane%16.

struct EpiStore {
  float* C; int ldc; long split_stride; int M, N;
  __device__ int b_row(int n) const { return n; }
  template <int FM, int FN>
  __device__ void operator()(f32x4 (&acc)[FM][FN], int m0, int n0, int lane, int,
                             char*, int, int) const {
    float* Cz = C + (long)blockIdx.z * split_stride;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int m = m0 + fm * 16 + 4 * (lane >> 4) + i;
        if (m >= M) continue;
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
          int n = n0 + fn * 16 + (lane & 15);
          if (n < N) Cz[(long)m * ldc + n] = acc[fm][fn][i];
        }
      }
  }
};

struct EpiScaledStore {
  float* C; int ldc; int M, N; float scale;
  __device__ int b_row(int n) const { return n; }
  template <int FM, int FN>
  __device__ void operator()(f32x4 (&acc)[FM][FN], int m0, int n0, int lane, int,
                             char*, int, int) const {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int m = m0 + fm * 16 + 4 * (lane >> 4) + i;
        if (m >= M) continue;
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
          int n = n0 + fn * 16 + (lane & 15);
          if (n < N) C[(long)m * ldc + n] = acc[fm][fn][i] * scale;
        }
      }
  }
};

struct EpiAdd {
  float* C; int ldc; int M, N;
  __device__ int b_row(int n) const { return n; }
  template <int FM, int FN>
  __device__ void operator()(f32x4 (&acc)[FM][FN], int m0, int n0, int lane, int,
                             char*, int, int) const {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int m = m0 + fm * 16 + 4 * (lane >> 4) + i;
        if (m >= M) continue;
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
          int n = n0 + fn * 16 + (lane & 15);
          if (n < N) C[(long)m * ldc + n] += acc[fm][fn][i];
        }
      }
  }
};

// Gate/up interleave: output column block of 32 = 16 gate columns followed by
// the 16 up columns of the same ffn indices. GEMM column n maps to ffn index
// f = (n / 32) * 16 + n % 16, gate when (n / 16) is even.
template <typename T>
struct EpiSwiGLU {
  T* out; int ldo; int M; int F;   // F = d_ffn; GEMM N = 2F
  __device__ int b_row(int n) const {
    int f = (n >> 5) * 16 + (n & 15);
    return ((n >> 4) & 1) ? F + f : f;
  }
  template <int FM, int FN>
  __device__ void operator()(f32x4 (&acc)[FM][FN], int m0, int n0, int lane, int,
                             char*, int, int) const {
    static_assert(FN % 2 == 0, "gate/up pairs");
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int m = m0 + fm * 16 + 4 * (lane >> 4) + i;
        if (m >= M) continue;
#pragma unroll
        for (int fn = 0; fn < FN; fn += 2) {
          int n = n0 + fn * 16;               // multiple of 32
          int f = (n >> 5) * 16 + (lane & 15);
          if (f >= F) continue;
          float g = acc[fm][fn][i], u = acc[fm][fn + 1][i];
          float s = g / (1.0f + __expf(-g));
          out[(long)m * ldo + f] = from_f32<T>(s * u);
        }
      }
  }
};

// Online softmax statistics of one row over a set of columns.
struct RowStat { float m; float s; int i; };
__device__ __forceinline__ RowStat combine(RowStat a, RowStat b) {
  RowStat r;
  r.m = fmaxf(a.m, b.m);
  float sa = a.s == 0.f ? 0.f : a.s * __expf(a.m - r.m);
  float sb = b.s == 0.f ? 0.f : b.s * __expf(b.m - r.m);
  r.s = sa + sb;
  r.i = a.m > b.m ? a.i : (b.m > a.m ? b.i : min(a.i, b.i));
  return r;
}

// Fused LM head: per row and vocab tile, (max, sum exp(z - max), lowest argmax)
// of z = acc * inv_tau; written to part_[m|s|i][tile][row].
struct EpiLMHead {
  float* pm; float* ps; int* pi; int M; int V; float inv_tau; int ld;  // ld = rows stride
  __device__ int b_row(int n) const { return n; }
  template <int FM, int FN>
  __device__ void operator()(f32x4 (&acc)[FM][FN], int m0, int n0, int lane, int wave_n,
                             char* smem, int waves_n, int bm) const {
    // stats per (fm, i) row for this lane over its FN columns
    RowStat st[FM][4];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        RowStat r = {-INFINITY, 0.f, 0x7fffffff};
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
          int n = n0 + fn * 16 + (lane & 15);
          if (n < V) {
            float z = acc[fm][fn][i] * inv_tau;
            RowStat c = {z, 1.f, n};
            r = combine(r, c);
          }
        }
        // across the 16 lanes that hold the other columns of these rows
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
          RowStat x;
          x.m = __shfl_xor(r.m, o, 64);
          x.s = __shfl_xor(r.s, o, 64);
          x.i = __shfl_xor(r.i, o, 64);
          r = combine(r, x);
        }
        st[fm][i] = r;
      }
    // across the waves that share these rows (different column ranges): LDS
    RowStat* buf = reinterpret_cast<RowStat*>(smem);
    const int wave_m_row0 = m0 - blockIdx.y * bm;  // wave's row offset inside the block tile
    __syncthreads();
    if ((lane & 15) == 0) {
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          int r = wave_m_row0 + fm * 16 + 4 * (lane >> 4) + i;
          buf[r * waves_n + wave_n] = st[fm][i];
        }
    }
    __syncthreads();
    const int tile = blockIdx.x;
    for (int r = threadIdx.x; r < bm; r += blockDim.x) {
      int m = blockIdx.y * bm + r;
      if (m >= M) continue;
      RowStat acc_r = buf[r * waves_n];
      for (int w = 1; w < waves_n; ++w) acc_r = combine(acc_r, buf[r * waves_n + w]);
      pm[(long)tile * ld + m] = acc_r.m;
      ps[(long)tile * ld + m] = acc_r.s;
      pi[(long)tile * ld + m] = acc_r.i;
    }
  }
};

// ---------------------------------------------------------------- kernel --
template <typename T, int BM, int BN, int WAVES_M, int WAVES_N, class Epi>
__global__ __launch_bounds__(256) void gemm_nt_kernel(
    const T* __restrict__ A, int lda, const T* __restrict__ B, int ldb,
    int M, int N, int K, int k_per_split, Epi epi) {
  static_assert(WAVES_M * WAVES_N == 4, "4 waves");
  constexpr int TM = BM / WAVES_M, TN = BN / WAVES_N;
  constexpr int FM = TM / 16, FN = TN / 16;
  constexpr int kVec = MfmaTraits<T>::kVec;
  constexpr int BK = kRowBytes / sizeof(T);
  constexpr int CHUNKS = (BM + BN) * (kRowBytes / 16);
  static_assert(CHUNKS % 256 == 0, "chunk split");
  constexpr int PER = CHUNKS / 256;
  constexpr int STAGE = (BM + BN) * kLdsRow;
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int kbeg = blockIdx.z * k_per_split;
  const int kend = min(K, kbeg + k_per_split);
  const int nkt = kend > kbeg ? ceil_div(kend - kbeg, BK) : 0;

  // per-thread global source rows (fixed over k)
  const T* src[PER];
  bool row_ok[PER];
  int coff[PER];
#pragma unroll
  for (int p = 0; p < PER; ++p) {
    int c = tid + p * 256;
    int r = c >> 3;
    coff[p] = (c & 7) * kVec;
    if (r < BM) {
      int m = m0 + r;
      row_ok[p] = m < M;
      src[p] = A + (long)(row_ok[p] ? m : 0) * lda;
    } else {
      int n = n0 + r - BM;
      row_ok[p] = n < N;
      src[p] = B + (long)(row_ok[p] ? epi.b_row(n) : 0) * ldb;
    }
  }

  u32x4 reg[PER];
  auto gload = [&](int kt) {
    int kb = kbeg + kt * BK;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      int k = kb + coff[p];
      if (row_ok[p] && k < kend)
        reg[p] = *reinterpret_cast<const u32x4*>(src[p] + k);
      else
        reg[p] = u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto sstore = [&](int buf) {
    char* s = smem + buf * STAGE;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      int c = tid + p * 256;
      *reinterpret_cast<u32x4*>(s + (c >> 3) * kLdsRow + (c & 7) * 16) = reg[p];
    }
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int a = 0; a < FM; ++a)
#pragma unroll
    for (int b = 0; b < FN; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int arow = (wm * TM + (lane & 15)) * kLdsRow;
  const int brow = (BM + wn * TN + (lane & 15)) * kLdsRow;
  const int kq = (lane >> 4) * 16;

  if (nkt > 0) {
    gload(0);
    sstore(0);
  }
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nkt) gload(kt + 1);
    const char* s = smem + cur * STAGE;
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      u32x4 af[FM], bfr[FN];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
        af[fm] = *reinterpret_cast<const u32x4*>(s + arow + fm * 16 * kLdsRow + g * 64 + kq);
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        bfr[fn] = *reinterpret_cast<const u32x4*>(s + brow + fn * 16 * kLdsRow + g * 64 + kq);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
          acc[fm][fn] = MfmaTraits<T>::mma(af[fm], bfr[fn], acc[fm][fn]);
    }
    if (kt + 1 < nkt) sstore(cur ^ 1);
    __syncthreads();
  }
  epi(acc, m0 + wm * TM, n0 + wn * TN, lane, wn, smem, WAVES_N, BM);
}

// --------------------------------------------------------------- launch --
template <typename T, class Epi>
static hipError_t launch(const T* A, int lda, const T* B, int ldb, int M, int N, int K,
                         int splits, const Epi& epi, hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  constexpr int BK = kRowBytes / sizeof(T);
  // split-K slices must tile K exactly: the consumers sum every slice
  if (splits < 1 || (splits > 1 && K % (splits * BK) != 0)) return hipErrorInvalidValue;
  const int kps = splits == 1 ? ceil_div(K, BK) * BK : K / splits;
  if (M <= 32) {
    dim3 g(ceil_div(N, 128), ceil_div(M, 32), splits);
    hipLaunchKernelGGL((gemm_nt_kernel<T, 32, 128, 1, 4, Epi>), g, dim3(256), 0, st,
                       A, lda, B, ldb, M, N, K, kps, epi);
  } else if (M <= 64) {
    dim3 g(ceil_div(N, 128), ceil_div(M, 64), splits);
    hipLaunchKernelGGL((gemm_nt_kernel<T, 64, 128, 2, 2, Epi>), g, dim3(256), 0, st,
                       A, lda, B, ldb, M, N, K, kps, epi);
  } else {
    dim3 g(ceil_div(N, 128), ceil_div(M, 128), splits);
    hipLaunchKernelGGL((gemm_nt_kernel<T, 128, 128, 2, 2, Epi>), g, dim3(256), 0, st,
                       A, lda, B, ldb, M, N, K, kps, epi);
  }
  return hipGetLastError();
}

int gemm_split_count(int M, int N, int K, int num_cu) {
  // enough blocks to cover the chip about twice; K slices stay >= 512
  int bm = M <= 32 ? 32 : (M <= 64 ? 64 : 128);
  long tiles = (long)ceil_div(N, 128) * ceil_div(M, bm);
  int s = 1;
  while (tiles * s < 2L * num_cu && K % (s * 2 * 64) == 0 && K / (s * 2) >= 512 && s < 16)
    s *= 2;
  return s;
}

template <typename T>
hipError_t gemm_store_f32(const T* A, int lda, const T* B, int ldb, int M, int N, int K,
                          int splits, float* C, int ldc, hipStream_t st) {
  EpiStore e{C, ldc, (long)M * ldc, M, N};
  return launch<T>(A, lda, B, ldb, M, N, K, splits, e, st);
}

template <typename T>
hipError_t gemm_add_f32(const T* A, int lda, const T* B, int ldb, int M, int N, int K,
                        float* C, int ldc, hipStream_t st) {
  EpiAdd e{C, ldc, M, N};
  return launch<T>(A, lda, B, ldb, M, N, K, 1, e, st);
}

template <typename T>
hipError_t gemm_scaled_f32(const T* A, int lda, const T* B, int ldb, int M, int N, int K,
                           float scale, float* C, int ldc, hipStream_t st) {
  EpiScaledStore e{C, ldc, M, N, scale};
  return launch<T>(A, lda, B, ldb, M, N, K, 1, e, st);
}

template <typename T>
hipError_t gemm_swiglu(const T* A, int lda, const T* W, int ldw, int M, int F, int K,
                       T* out, int ldo, hipStream_t st) {
  EpiSwiGLU<T> e{out, ldo, M, F};
  return launch<T>(A, lda, W, ldw, M, 2 * F, K, 1, e, st);
}

int lm_head_tiles(int V) { return ceil_div(V, 128); }

template <typename T>
hipError_t gemm_lm_head(const T* U, int ldu, const T* W, int M, int V, int K, float inv_tau,
                        float* pm, float* ps, int* pi, int ld, hipStream_t st) {
  EpiLMHead e{pm, ps, pi, M, V, inv_tau, ld};
  return launch<T>(U, ldu, W, K, M, V, K, 1, e, st);
}

#define INST(T)                                                                          \
  template hipError_t gemm_store_f32<T>(const T*, int, const T*, int, int, int, int, int, \
                                        float*, int, hipStream_t);                        \
  template hipError_t gemm_add_f32<T>(const T*, int, const T*, int, int, int, int, float*, \
                                      int, hipStream_t);                                  \
  template hipError_t gemm_scaled_f32<T>(const T*, int, const T*, int, int, int, int,     \
                                         float, float*, int, hipStream_t);                \
  template hipError_t gemm_swiglu<T>(const T*, int, const T*, int, int, int, int, T*, int, \
                                     hipStream_t);                                        \
  template hipError_t gemm_lm_head<T>(const T*, int, const T*, int, int, int, float,      \
                                      float*, float*, int*, int, hipStream_t);
INST(bf16)
INST(float)

}  // namespace dlm
