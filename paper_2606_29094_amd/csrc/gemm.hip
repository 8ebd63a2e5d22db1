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
#include <algorithm>

#include "common.h"
#include "gemm_common.h"
#include "kernels.h"

namespace dlm {

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
  if (epi.skip_tile(m0)) return;   // uniform over the block
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
  epi(acc, m0 + wm * TM, n0 + wn * TN, lane, wn, smem, WAVES_N, BM, m0, (int)blockIdx.x,
      (int)blockIdx.z);
}

// --------------------------------------------------------------- launch --

// Register-staged kernel: any K that is a multiple of 16 bytes, fp32 or bf16.
template <typename T, class Epi>
static hipError_t launch_rs(const T* A, int lda, const T* B, int ldb, int M, int N, int K,
                            int splits, const Epi& epi, hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  constexpr int BK = kRowBytes / sizeof(T);
  // split-K slices must tile K exactly: the consumers sum every slice
  if (splits < 1 || (splits > 1 && K % (splits * BK) != 0)) return hipErrorInvalidValue;
  const int kps = splits == 1 ? ceil_div(K, BK) * BK : K / splits;
  if (M <= 32) {
    dim3 g(ceil_div(N, 128), ceil_div(M, 32), splits);
    DLM_LAUNCH((gemm_nt_kernel<T, 32, 128, 1, 4, Epi>), g, dim3(256), 0, st,
                       A, lda, B, ldb, M, N, K, kps, epi);
  } else if (M <= 64) {
    dim3 g(ceil_div(N, 128), ceil_div(M, 64), splits);
    DLM_LAUNCH((gemm_nt_kernel<T, 64, 128, 2, 2, Epi>), g, dim3(256), 0, st,
                       A, lda, B, ldb, M, N, K, kps, epi);
  } else {
    dim3 g(ceil_div(N, 128), ceil_div(M, 128), splits);
    DLM_LAUNCH((gemm_nt_kernel<T, 128, 128, 2, 2, Epi>), g, dim3(256), 0, st,
                       A, lda, B, ldb, M, N, K, kps, epi);
  }
  return hipGetLastError();
}

template <typename T, class Epi>
static hipError_t launch(const GemmPlan& p, const T* A, int lda, const T* B, int ldb, int M,
                         int N, int K, const Epi& epi, hipStream_t st) {
  if constexpr (sizeof(T) == 2) {
    if (p.cfg >= 0)
      return gemm_dl_launch<Epi>(p.cfg, A, lda, B, ldb, M, N, K, p.splits, p.group_m,
                                 Epi::kTailSplit ? p.sub : 0, p.n_tail, epi, st);
  }
  return launch_rs<T, Epi>(A, lda, B, ldb, M, N, K, p.splits, epi, st);
}

// Tile/split choice. bf16 with K a multiple of 64 uses the direct-load kernel.
// A configuration keeps `occ` blocks per CU resident. Its time is rounds x
// (time of one round at the block's k-tile count), the per-round times being
// medians of 757 launches measured on MI355X (the projection shapes of both
// model shapes at M = 256 .. 8192, every split, weights streamed from HBM),
// interpolated linearly in k-tiles (proportionally outside the measured range);
// a last, partly filled round of a multi-block configuration costs
// max(0.7, fill) of a full one. A last round that fills at most a quarter
// (half) of the CUs of a one-block-per-CU configuration may run its tiles as
// quarter (half) tiles, where the configuration has them: it then costs
// 0.55 (0.75) of a full round. These two factors minimise the summed measured
// time of the chosen plans over 56 projection shapes (both model shapes,
// 256 .. 7936 rows, every configuration with and without the split; 1.6 %
// below the plans without sub-tiles, within 0.1 % of the best measured plan
// of every shape; e.g. GQA QKV at 4096 rows 143 -> 130 us, gate/up 921 -> 894
// us, output projection at 5056 rows 165 -> 146 us). When K is split, the extra fp32 slices add
// the consumer's reads of them (their writes are inside the measured round
// times; charging both picked worse plans, e.g. 62 vs 52 us for the 512-row
// MHA QKV projection). The cheapest
// (configuration, split) wins. 128x192 with two blocks per CU (cfg 22) runs
// without K splits only (its table holds unsplit launches); the small tiles
// only for few rows. The eight-wave configurations run the split-phase tile
// form with a three-stage weight ring (6, 21, 70) or three stages of both
// operands (29); their tables are the ones measured for their two-ring form,
// each entry scaled by the time ratios of the forms measured at that k-tile
// count (full rounds: 0.94-0.98 from the split-phase loop, about 0.98-0.99
// more from the third weight stage; the 256x192 tile 0.93, measured at 256 to
// 6400 rows with the weights streamed from HBM); the three-stage 256x128 tile
// (29) takes the mean of the estimates from the tables of the two-ring
// 256x128 tiles it replaces (3- and 4-stage weight rings, scaled by
// 0.87-0.94 and 0.90-0.97).
namespace {
struct RoundTable {
  int cfg, occ, max_m;
  bool unsplit_only;
  int n;
  float kt[15], us[15];
  int min_kt = 0;          // used only for at least this many k-tiles per block
};
const RoundTable kRoundTables[] = {
    {6, 1, 1 << 30, false, 15,
     {8, 14, 16, 24, 28, 32, 37, 48, 56, 64, 74, 96, 148, 192, 296},
     {23.9f, 28.5f, 33.9f, 48.5f, 45.5f, 55.0f, 70.8f, 81.0f, 84.3f, 100.1f, 122.4f, 141.7f, 213.1f, 263.3f, 398.9f}},
    {21, 1, 1 << 30, false, 15,
     {8, 14, 16, 24, 28, 32, 37, 48, 56, 64, 74, 96, 148, 192, 296},
     {18.2f, 23.6f, 26.3f, 38.7f, 37.9f, 43.6f, 56.3f, 64.7f, 67.5f, 80.5f, 95.1f, 118.5f, 175.2f, 223.3f, 343.0f}},
    {22, 2, 1 << 30, true, 4, {56, 64, 192, 296}, {81.9f, 93.1f, 282.1f, 435.5f}},
    {29, 1, 1 << 30, false, 15,
     {8, 14, 16, 24, 28, 32, 37, 48, 56, 64, 74, 96, 148, 192, 296},
     {15.2f, 17.6f, 21.0f, 28.5f, 27.5f, 33.1f, 42.6f, 49.1f, 51.6f, 63.0f, 74.3f, 89.6f, 131.7f, 168.7f, 249.4f}},
    {42, 1, 1 << 30, false, 15,
     {8, 14, 16, 24, 28, 32, 37, 48, 56, 64, 74, 96, 148, 192, 296},
     {14.6f, 18.1f, 20.7f, 29.2f, 27.6f, 32.4f, 41.1f, 47.7f, 47.8f, 56.8f, 70.6f, 80.0f, 124.7f, 154.4f, 232.9f}},
    {1, 2, 128, false, 15,
     {8, 14, 16, 24, 28, 32, 37, 48, 56, 64, 74, 96, 148, 192, 296},
     {17.1f, 22.4f, 25.6f, 37.3f, 33.5f, 40.8f, 51.1f, 65.7f, 65.8f, 71.1f, 90.8f, 119.1f, 171.0f, 214.9f, 335.1f}},
    {10, 3, 64, false, 1, {64}, {75.0f}},
    // 32x32x16 MFMA tiles: 256x128 with four 128x64-wave tiles, and 384x256
    // with eight 96x128-wave tiles (two waves per SIMD). Their round times
    // were measured against configurations 29 and 6 in the same runs (full
    // rounds, weights streamed from HBM) and scaled by those configurations'
    // tables above, so all tables share one measurement basis.
    {62, 1, 1 << 30, false, 15,
     {8, 14, 16, 24, 28, 32, 37, 48, 56, 64, 74, 96, 148, 192, 296},
     {17.3f, 20.0f, 24.6f, 35.1f, 33.5f, 40.8f, 50.3f, 61.1f, 61.9f, 79.5f, 87.3f, 110.3f, 158.0f, 211.6f, 330.7f}},
    {65, 1, 1 << 30, false, 15,
     {8, 14, 16, 24, 28, 32, 37, 48, 56, 64, 74, 96, 148, 192, 296},
     {37.4f, 46.5f, 57.2f, 79.0f, 73.6f, 88.7f, 118.5f, 131.5f, 126.5f, 156.3f, 204.0f, 238.4f, 360.9f, 430.0f, 679.5f},
     148},   // measured ahead only with long K walks (the GQA down projection); the
             // table overrates it at 56 k-tiles (4096-row output projection 145 vs 112 us)
    // 256x224: measured against configuration 6 in the same runs (one and two
    // full rounds per k-tile count) and scaled by that configuration's table;
    // a round takes 0.82-0.94 (mean 0.89) of a 256x256 round for 0.875 of its work
    {70, 1, 1 << 30, false, 15,
     {8, 14, 16, 24, 28, 32, 37, 48, 56, 64, 74, 96, 148, 192, 296},
     {22.5f, 25.7f, 31.3f, 45.6f, 42.3f, 51.5f, 64.1f, 71.1f, 70.6f, 94.1f, 111.6f, 126.1f, 192.8f, 234.0f, 374.4f}},
};

double round_us(const RoundTable& t, double kt) {
  if (kt <= t.kt[0]) return t.us[0] * kt / t.kt[0];
  for (int i = 1; i < t.n; ++i)
    if (kt <= t.kt[i]) {
      const double w = (kt - t.kt[i - 1]) / (t.kt[i] - t.kt[i - 1]);
      return t.us[i - 1] + w * (t.us[i] - t.us[i - 1]);
    }
  return t.us[t.n - 1] * kt / t.kt[t.n - 1];
}
}  // namespace

GemmPlan gemm_plan(int es, int M, int N, int K, bool splittable, int num_cu, bool allow_mf32,
                   bool allow_tail, bool allow_odd) {
  GemmPlan best{-1, 1, 0};
  if (M <= 0 || N <= 0) return best;
  if (es != 2 || K % 64 != 0) {
    if (splittable) {
      int bm = M <= 32 ? 32 : (M <= 64 ? 64 : 128);
      long tiles = (long)ceil_div(N, 128) * ceil_div(M, bm);
      int s = 1;
      while (tiles * s < 2L * num_cu && K % (s * 2 * 64) == 0 && K / (s * 2) >= 512 && s < 8)
        s *= 2;
      best.splits = s;
    }
    return best;
  }
  double best_t = 1e30;
  for (const RoundTable& c : kRoundTables) {
    if (M > c.max_m) continue;
    if (!allow_mf32 && gemm_dl_mfma(c.cfg) == 32) continue;
    if (!allow_odd && gemm_dl_odd(c.cfg)) continue;
    int bm, bn, th;
    gemm_dl_tile(c.cfg, &bm, &bn, &th);
    for (int s = 1; s <= 8; s *= 2) {
      if (s > 1 && (c.unsplit_only || !splittable || (K / 64) % s != 0 || K / s < 512)) continue;
      if (K / 64 / s < c.min_kt) continue;
      const long units = (long)ceil_div(M, bm) * ceil_div(N, bn) * s;
      const long slots = (long)num_cu * c.occ;
      const long full = units / slots;
      const long rem = units - full * slots;
      const double fill = (double)rem / slots;
      const int subs = allow_tail && c.occ == 1 ? gemm_dl_subs(c.cfg) : 0;
      double rounds = (double)full;
      int sub = 0;
      if (rem > 0) {
        if (c.occ > 1) {
          rounds += std::max(0.7, fill);
        } else if ((subs & 4) && 4 * rem <= slots) {
          rounds += 0.55;
          sub = 4;
        } else if ((subs & 2) && 2 * rem <= slots) {
          rounds += 0.75;
          sub = 2;
        } else {
          rounds += 1.0;
        }
      }
      double t = rounds * round_us(c, (double)(K / s) / 64.0);
      if (s > 1) t += (double)M * N * 4.0 * (s - 1) / 5.0e12 * 1e6;
      if (t < best_t * 0.999) {
        best_t = t;
        best = GemmPlan{c.cfg, s, 0, sub, sub ? (int)rem : 0};
      }
    }
  }
  // weights larger than the last-level cache (256 MB Infinity Cache) stream
  // from HBM once per row tile in plain order: use the grouped XCD order
  int bm, bn, th;
  if (best.cfg >= 0 && gemm_dl_tile(best.cfg, &bm, &bn, &th) && ceil_div(M, bm) > 1 &&
      (double)N * K * es > 256e6)
    best.group_m = 8;
  return best;
}

// The LM head at <= 64 rows streams the vocab matrix once and is bound by HBM,
// not by the round-time tables: measured with the rotated K walk, a weight row
// pitch that is a multiple of 8 KB (the 4096-wide MHA head) runs best with the
// 3-stage 64x128 tiles (two weight tiles in flight per block, 5.9 TB/s), other
// pitches (the 3584-wide GQA head) with the 2-stage ones (three blocks per CU,
// 5.8 TB/s).
GemmPlan lm_head_plan(int es, int M, int V, int K, int num_cu) {
  // the head's epilogue is 16x16 and keeps whole tiles (its partial results are per column tile)
  GemmPlan p = gemm_plan(es, M, V, K, false, num_cu, false, false, false);
  if (p.cfg >= 0 && M <= 64) p = GemmPlan{((long)K * es) % 8192 == 0 ? 11 : 10, 1, 0};
  // The head is planned for its largest row count and skips, on the device,
  // the row tiles beyond the rows that need a prediction. The grouped order
  // must then span every row tile in one group: with several groups, the
  // XCDs that receive the later groups' ranges would only hold skipped tiles
  // (half the XCDs idle with two groups).
  int bm, bn, th;
  if (p.group_m > 0 && gemm_dl_tile(p.cfg, &bm, &bn, &th)) p.group_m = ceil_div(M, bm);
  // over several row tiles, walk only the tiles of the rows that need a prediction
  if (p.cfg >= 0 && gemm_dl_tile(p.cfg, &bm, &bn, &th) && ceil_div(M, bm) > 1)
    p.active_cus = num_cu;
  return p;
}

template <typename T>
hipError_t gemm_store_f32(const GemmPlan& p, const T* A, int lda, const T* B, int ldb, int M,
                          int N, int K, float* C, int ldc, hipStream_t st) {
  EpiStore e{C, ldc, (long)M * ldc, M, N};
  return launch<T>(p, A, lda, B, ldb, M, N, K, e, st);
}

template <typename T>
hipError_t gemm_add_f32(const GemmPlan& p, const T* A, int lda, const T* B, int ldb, int M, int N,
                        int K, float* C, int ldc, hipStream_t st) {
  if (p.splits != 1) return hipErrorInvalidValue;
  EpiAdd e{C, ldc, M, N};
  return launch<T>(p, A, lda, B, ldb, M, N, K, e, st);
}

template <typename T>
hipError_t gemm_scaled_f32(const GemmPlan& p, const T* A, int lda, const T* B, int ldb, int M,
                           int N, int K, float scale, float* C, int ldc, hipStream_t st) {
  if (p.splits != 1) return hipErrorInvalidValue;
  EpiScaledStore e{C, ldc, M, N, scale};
  return launch<T>(p, A, lda, B, ldb, M, N, K, e, st);
}

template <typename T>
hipError_t gemm_swiglu(const GemmPlan& p, const T* A, int lda, const T* W, int ldw, int M, int F,
                       int K, T* out, int ldo, hipStream_t st) {
  if (p.splits != 1) return hipErrorInvalidValue;
  // 32x32 tiles interleave gate and up columns in groups of 32
  if (p.cfg >= 0 && gemm_dl_mfma(p.cfg) == 32 && F % 32 != 0) return hipErrorInvalidValue;
  EpiSwiGLU<T> e{out, ldo, M, F};
  return launch<T>(p, A, lda, W, ldw, M, 2 * F, K, e, st);
}

hipError_t gemm_debug_launch(int cfg, int epilogue, int sub, int n_tail, int group_m,
                             int splits, const bf16* A, const bf16* B, void* C, int M, int N,
                             int K, hipStream_t st) {
  if (epilogue == 0) {
    EpiStore e{reinterpret_cast<float*>(C), N, (long)M * N, M, N};
    return gemm_dl_launch<EpiStore>(cfg, A, K, B, K, M, N, K, splits, group_m, sub, n_tail, e,
                                    st);
  }
  if (splits != 1) return hipErrorInvalidValue;
  if (epilogue == 1) {
    EpiSwiGLU<bf16> e{reinterpret_cast<bf16*>(C), N / 2, M, N / 2};
    return gemm_dl_launch<EpiSwiGLU<bf16>>(cfg, A, K, B, K, M, N, K, 1, group_m, sub, n_tail, e,
                                           st);
  }
  if (epilogue == 2) {
    EpiAdd e{reinterpret_cast<float*>(C), N, M, N};
    return gemm_dl_launch<EpiAdd>(cfg, A, K, B, K, M, N, K, 1, group_m, sub, n_tail, e, st);
  }
  return hipErrorInvalidValue;
}

int lm_head_tiles(const GemmPlan& p, int V) {
  int bm = 128, bn = 128, th = 256;
  if (p.cfg >= 0) gemm_dl_tile(p.cfg, &bm, &bn, &th);
  return ceil_div(V, bn);
}

template <typename T>
hipError_t gemm_lm_head(const GemmPlan& p, const T* U, int ldu, const T* W, int M, int V, int K,
                        float inv_tau, float* pm, float* ps, int* pi, int ld,
                        const int* m_count, hipStream_t st) {
  if (p.splits != 1) return hipErrorInvalidValue;
  EpiLMHead e{pm, ps, pi, M, V, inv_tau, ld, m_count};
  if constexpr (sizeof(T) == 2) {
    if (p.cfg >= 0 && p.active_cus > 0)
      return gemm_dl_head_launch(p.cfg, U, ldu, W, K, M, V, K, p.active_cus, e, st);
  }
  return launch<T>(p, U, ldu, W, K, M, V, K, e, st);
}

#define INST(T)                                                                                \
  template hipError_t gemm_store_f32<T>(const GemmPlan&, const T*, int, const T*, int, int, int, \
                                        int, float*, int, hipStream_t);                         \
  template hipError_t gemm_add_f32<T>(const GemmPlan&, const T*, int, const T*, int, int, int,   \
                                      int, float*, int, hipStream_t);                           \
  template hipError_t gemm_scaled_f32<T>(const GemmPlan&, const T*, int, const T*, int, int,     \
                                         int, int, float, float*, int, hipStream_t);            \
  template hipError_t gemm_swiglu<T>(const GemmPlan&, const T*, int, const T*, int, int, int,    \
                                     int, T*, int, hipStream_t);                                \
  template hipError_t gemm_lm_head<T>(const GemmPlan&, const T*, int, const T*, int, int, int,   \
                                      float, float*, float*, int*, int, const int*, hipStream_t);
INST(bf16)
INST(float)

}  // namespace dlm
