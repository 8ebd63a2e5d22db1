// Shared pieces of the GEMM kernels: MFMA operand traits and the tile
// epilogues. Each epilogue sees a wave's accumulators: acc[fm][fn][i] is the
// value at row m0 + fm*16 + 4*(lane/16) + i, column n0 + fn*16 + lane%16.
#pragma once

#include "common.h"

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

// two adjacent outputs in one store (4 bytes for bf16, 8 for fp32)
__device__ __forceinline__ void store2(float* o, float a, float b) {
  *reinterpret_cast<float2*>(o) = make_float2(a, b);
}
__device__ __forceinline__ void store2(bf16* o, float a, float b) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 v;
  v[0] = (bf16)a;
  v[1] = (bf16)b;
  *reinterpret_cast<bf16x2*>(o) = v;
}

// ------------------------------------------------------------ epilogues --
// Each epilogue sees the wave's accumulators: acc[fm][fn][i] is the value at
// row m0 + fm*16 + 4*(lane/16) + i, column n0 + fn*16 + lane%16. The further
// arguments: wave column index, LDS scratch, waves per row, block rows, the
// block's first row, its column-tile index and its K-split index (the kernel's
// tile order decides these, not blockIdx).

struct EpiStore {
  float* C; int ldc; long split_stride; int M, N;
  static constexpr bool kRotateK = false;
  static constexpr bool kMf32 = true;
  static constexpr bool kTailSplit = true;   // last-round tiles may be split
  static constexpr bool kOddFragments = true;   // any number of 16-column fragments per wave
  __host__ __device__ void set_mfma(int) {}
  __device__ int b_row(int n) const { return n; }
  __device__ bool skip_tile(int) const { return false; }
  // 32x32 accumulators: lanes 0-31 hold 32 consecutive columns of a row
  template <int FM, int FN>
  __device__ void op32(f32x16 (&acc)[FM][FN], int m0, int n0, int lane, int split) const {
    float* Cz = C + (long)split * split_stride;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int m = m0 + fm * 32 + mf32_row(i, lane);
        if (m >= M) continue;
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
          const int n = n0 + fn * 32 + (lane & 31);
          if (n < N) Cz[(long)m * ldc + n] = acc[fm][fn][i];
        }
      }
  }
  template <int FM, int FN>
  __device__ void operator()(f32x4 (&acc)[FM][FN], int m0, int n0, int lane, int,
                             char*, int, int, int, int, int split) const {
    float* Cz = C + (long)split * split_stride;
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
  static constexpr bool kRotateK = false;
  static constexpr bool kMf32 = false;
  static constexpr bool kTailSplit = false;   // last-round tiles may be split
  static constexpr bool kOddFragments = true;   // any number of 16-column fragments per wave
  __host__ __device__ void set_mfma(int) {}
  template <int FM, int FN>
  __device__ void op32(f32x16 (&)[FM][FN], int, int, int, int) const {}
  __device__ int b_row(int n) const { return n; }
  __device__ bool skip_tile(int) const { return false; }
  template <int FM, int FN>
  __device__ void operator()(f32x4 (&acc)[FM][FN], int m0, int n0, int lane, int,
                             char*, int, int, int, int, int) const {
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

// C += acc (the residual update). The loads of one 16-row fragment row are all
// issued before its stores: element by element, each load would wait for the
// previous store (the compiler cannot tell that the addresses differ).
struct EpiAdd {
  float* C; int ldc; int M, N;
  static constexpr bool kRotateK = false;
  static constexpr bool kMf32 = true;
  static constexpr bool kTailSplit = true;   // last-round tiles may be split
  static constexpr bool kOddFragments = true;   // any number of 16-column fragments per wave
  __host__ __device__ void set_mfma(int) {}
  __device__ int b_row(int n) const { return n; }
  __device__ bool skip_tile(int) const { return false; }
  // 32x32 accumulators: per tile row group of 4 rows, the loads first
  template <int FM, int FN>
  __device__ void op32(f32x16 (&acc)[FM][FN], int m0, int n0, int lane, int) const {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i0 = 0; i0 < 16; i0 += 4) {
        float cv[4][FN];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + fm * 32 + mf32_row(i0 + i, lane);
#pragma unroll
          for (int fn = 0; fn < FN; ++fn) {
            const int n = n0 + fn * 32 + (lane & 31);
            cv[i][fn] = m < M && n < N ? C[(long)m * ldc + n] : 0.f;
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + fm * 32 + mf32_row(i0 + i, lane);
#pragma unroll
          for (int fn = 0; fn < FN; ++fn) {
            const int n = n0 + fn * 32 + (lane & 31);
            if (m < M && n < N) C[(long)m * ldc + n] = cv[i][fn] + acc[fm][fn][i0 + i];
          }
        }
      }
  }
  template <int FM, int FN>
  __device__ void operator()(f32x4 (&acc)[FM][FN], int m0, int n0, int lane, int,
                             char*, int, int, int, int, int) const {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      float cv[4][FN];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + fm * 16 + 4 * (lane >> 4) + i;
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
          const int n = n0 + fn * 16 + (lane & 15);
          cv[i][fn] = m < M && n < N ? C[(long)m * ldc + n] : 0.f;
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + fm * 16 + 4 * (lane >> 4) + i;
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
          const int n = n0 + fn * 16 + (lane & 15);
          if (m < M && n < N) C[(long)m * ldc + n] = cv[i][fn] + acc[fm][fn][i];
        }
      }
    }
  }
};

// Gate/up interleave: with w = 16 (16x16 MFMA tiles) or 32 (32x32 tiles), an
// output column block of 2w = w gate columns followed by the w up columns of
// the same ffn indices. GEMM column n maps to ffn index f = (n / 2w) w + n % w,
// gate when (n / w) is even. The loader reads weight row b_row(n).
template <typename T>
struct EpiSwiGLU {
  T* out; int ldo; int M; int F;   // F = d_ffn; GEMM N = 2F
  int wsh = 4;                     // log2 w
  __host__ __device__ void set_mfma(int mf) { wsh = mf == 32 ? 5 : 4; }
  __device__ int b_row(int n) const {
    const int f = ((n >> (wsh + 1)) << wsh) + (n & ((1 << wsh) - 1));
    return ((n >> wsh) & 1) ? F + f : f;
  }
  __device__ bool skip_tile(int) const { return false; }
  static constexpr bool kRotateK = false;
  static constexpr bool kMf32 = true;
  static constexpr bool kTailSplit = true;   // last-round tiles may be split
  static constexpr bool kOddFragments = false;  // fragments come in gate/up pairs
  // 32x32 accumulators: tiles fn (gate) and fn + 1 (up) hold the same ffn
  // indices in the same lanes; lanes 0-31 store 32 consecutive outputs of a row
  template <int FM, int FN>
  __device__ void op32(f32x16 (&acc)[FM][FN], int m0, int n0, int lane, int) const {
    static_assert(FN % 2 == 0, "gate/up pairs");
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int m = m0 + fm * 32 + mf32_row(i, lane);
#pragma unroll
        for (int fn = 0; fn < FN; fn += 2) {
          const float g = acc[fm][fn][i], u = acc[fm][fn + 1][i];
          const float y = g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
          const int f = ((n0 + fn * 32) >> 6) * 32 + (lane & 31);
          if (m < M && f < F) out[(long)m * ldo + f] = from_f32<T>(y);
        }
      }
  }
  // silu(g) * u with silu(g) = g / (1 + exp(-g)) through the hardware
  // reciprocal (about 1 ulp; the result is rounded to the storage type).
  // Outputs go out in pairs of adjacent columns: for rows i and i + 1 of a
  // fragment, lane 2k and lane 2k + 1 swap one value each, then lane 2k
  // stores columns (f, f + 1) of row i and lane 2k + 1 those of row i + 1.
  template <int FM, int FN>
  __device__ void operator()(f32x4 (&acc)[FM][FN], int m0, int n0, int lane, int,
                             char*, int, int, int, int, int) const {
    static_assert(FN % 2 == 0, "gate/up pairs");
    const bool odd = lane & 1;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i = 0; i < 4; i += 2) {
        const int m = m0 + fm * 16 + 4 * (lane >> 4) + i + (odd ? 1 : 0);   // row this lane stores
#pragma unroll
        for (int fn = 0; fn < FN; fn += 2) {
          float y[2];
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            const float g = acc[fm][fn][i + k], u = acc[fm][fn + 1][i + k];
            y[k] = g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
          }
          const float recv = __shfl_xor(odd ? y[0] : y[1], 1, 64);
          const int f = (((n0 + fn * 16) >> 5) * 16) + ((lane & 15) & ~1);   // even column
          if (m < M && f < F) {
            const float lo = odd ? recv : y[0], hi = odd ? y[1] : recv;
            store2(out + (long)m * ldo + f, lo, hi);
          }
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
// of z = acc * inv_tau; written to part_[m|s|i][tile][row]. When m_count is
// given (the device-side number of rows that need a prediction, packed first),
// row tiles at or beyond it are skipped.
struct EpiLMHead {
  float* pm; float* ps; int* pi; int M; int V; float inv_tau; int ld;  // ld = rows stride
  const int* m_count;
  static constexpr bool kRotateK = true;   // weight streaming: rotate the K walk per column tile
  static constexpr bool kMf32 = false;
  static constexpr bool kTailSplit = false;   // last-round tiles may be split
  static constexpr bool kOddFragments = true;   // any number of 16-column fragments per wave
  __host__ __device__ void set_mfma(int) {}
  template <int FM, int FN>
  __device__ void op32(f32x16 (&)[FM][FN], int, int, int, int) const {}
  __device__ int b_row(int n) const { return n; }
  __device__ bool skip_tile(int m0) const { return m_count && m0 >= *m_count; }
  template <int FM, int FN>
  __device__ void operator()(f32x4 (&acc)[FM][FN], int m0, int n0, int lane, int wave_n,
                             char* smem, int waves_n, int bm, int block_m0,
                             int tile_n, int) const {
    // per row (fm, i) over the wave's columns: each lane takes the max and its
    // lowest column over its FN columns; the 16 lanes that hold the row agree
    // on the row max, sum exp(z - max) with one exp per element, and take the
    // lowest column among the lanes that reached the max
    RowStat st[FM][4];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float mx = -INFINITY;
        int ix = 0x7fffffff;
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
          const int n = n0 + fn * 16 + (lane & 15);
          const float z = acc[fm][fn][i] * inv_tau;
          if (n < V && z > mx) { mx = z; ix = n; }   // columns ascend with fn: ties keep the lowest
        }
        float gm = mx;
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) gm = fmaxf(gm, __shfl_xor(gm, o, 64));
        float s = 0.f;
        if (gm != -INFINITY) {
#pragma unroll
          for (int fn = 0; fn < FN; ++fn) {
            const int n = n0 + fn * 16 + (lane & 15);
            if (n < V) s += __expf(acc[fm][fn][i] * inv_tau - gm);
          }
        }
        int gi = mx == gm ? ix : 0x7fffffff;
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
          s += __shfl_xor(s, o, 64);
          gi = min(gi, __shfl_xor(gi, o, 64));
        }
        st[fm][i] = RowStat{gm, s, gi};
      }
    // across the waves that share these rows (different column ranges): LDS
    RowStat* buf = reinterpret_cast<RowStat*>(smem);
    const int wave_m_row0 = m0 - block_m0;  // wave's row offset inside the block tile
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
    const int tile = tile_n;
    for (int r = threadIdx.x; r < bm; r += blockDim.x) {
      int m = block_m0 + r;
      if (m >= M) continue;
      RowStat acc_r = buf[r * waves_n];
      for (int w = 1; w < waves_n; ++w) acc_r = combine(acc_r, buf[r * waves_n + w]);
      pm[(long)tile * ld + m] = acc_r.m;
      ps[(long)tile * ld + m] = acc_r.s;
      pi[(long)tile * ld + m] = acc_r.i;
    }
  }
};

}  // namespace dlm
