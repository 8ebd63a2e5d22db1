// Row-wise kernels of the denoising step: embedding gather, RMSNorm, RoPE and
// the key/value cache writes, split-K reduction into the residual stream, the
// selection of the rows that need a prediction, the final norm, the combine of
// the per-vocab-tile softmax statistics and the threshold/compaction step.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace dlm {

// ------------------------------------------------------------ embedding --
// h[n] = E[mask ? mask_id : token] for every recompute row n (fp32 residual).
// Token ids outside [0, vocab) are read as [MASK].
template <typename T>
__global__ void embed_kernel(StepPlan p, const T* __restrict__ E, int d, int vocab, int mask_id,
                             const int32_t* __restrict__ tokens, const uint8_t* __restrict__ mask,
                             float* __restrict__ h) {
  const int n = blockIdx.x;
  const int r = plan_req_of_row(p, n);
  const ReqPlan& q = p.r[r];
  const int pos = q.pos0 + (n - q.row0);
  const long ti = (long)q.tok_off + pos;
  const int tk = tokens[ti];
  const int id = (mask[ti] || tk < 0 || tk >= vocab) ? mask_id : tk;
  const T* src = E + (long)id * d;
  float* dst = h + (long)n * d;
  for (int j = threadIdx.x; j < d; j += blockDim.x) dst[j] = to_f32(src[j]);
}

template <typename T>
hipError_t embed_rows(const StepPlan& p, const T* E, int d, int vocab, int mask_id,
                      const int32_t* tokens, const uint8_t* mask, float* h, hipStream_t st) {
  if (p.n_rows == 0) return hipSuccess;
  DLM_LAUNCH(embed_kernel<T>, dim3(p.n_rows), dim3(256), 0, st, p, E, d, vocab, mask_id,
                     tokens, mask, h);
  return hipGetLastError();
}

// -------------------------------------------------------------- rmsnorm --
__device__ __forceinline__ float block_sum_256(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = red[0] + red[1] + red[2] + red[3];
  __syncthreads();
  return t;
}

// out[n] = h[n] / sqrt(mean(h[n]^2) + eps) * g, fp32 math, stored as T.
// With split-K slices (part != null), the row is first updated in place,
// h[n] += sum_s part[s][n] (slices in order), so the residual update of the
// previous projection and this norm take one pass over h. out may be null
// (update only). rows/count select and bound the rows (final-norm gather).
// four consecutive outputs in one 16-byte (fp32) or 8-byte (bf16) store
__device__ __forceinline__ void store4(float* o, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(o) = make_float4(a, b, c, d);
}
__device__ __forceinline__ void store4(bf16* o, float a, float b, float c, float d) {
  bf16x4 v;
  v[0] = (bf16)a; v[1] = (bf16)b; v[2] = (bf16)c; v[3] = (bf16)d;
  *reinterpret_cast<bf16x4*>(o) = v;
}

// S > 0: exactly S split-K slices, all of a row's slice loads issued before
// the first add (the row's partials are in flight at once instead of one
// slice per memory round trip); S == 0: `splits` slices, one at a time.
// Either way the sum is h + slice 0 + slice 1 + ... in that order.
template <typename T, int S>
__global__ __launch_bounds__(256) void rmsnorm_kernel(float* __restrict__ h,
                                                      const float* __restrict__ part, int splits,
                                                      long stride, const float* __restrict__ g,
                                                      int d, float eps, T* __restrict__ out,
                                                      const int* __restrict__ rows,
                                                      const int* __restrict__ count) {
  __shared__ float red[4];
  const int i = blockIdx.x;
  if (count && i >= *count) return;
  const int src_row = rows ? rows[i] : i;
  float* x = h + (long)src_row * d;
  float ss = 0.f;
  if (d <= 4096) {
    // rows of up to 4096: the thread's (at most) four float4 stay in registers
    // between the update and the normalisation; all loads of a slice are issued
    // together
    float4 v[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int j = threadIdx.x * 4 + c * 1024;
      if (j < d) v[c] = *reinterpret_cast<const float4*>(x + j);
    }
    if (part) {
      if constexpr (S > 0) {
        float4 pv[S][4];
#pragma unroll
        for (int sl = 0; sl < S; ++sl) {
          const float* ps = part + sl * stride + (long)src_row * d;
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int j = threadIdx.x * 4 + c * 1024;
            if (j < d) pv[sl][c] = *reinterpret_cast<const float4*>(ps + j);
          }
        }
#pragma unroll
        for (int sl = 0; sl < S; ++sl)
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int j = threadIdx.x * 4 + c * 1024;
            if (j < d) {
              v[c].x += pv[sl][c].x; v[c].y += pv[sl][c].y;
              v[c].z += pv[sl][c].z; v[c].w += pv[sl][c].w;
            }
          }
      } else {
        for (int sl = 0; sl < splits; ++sl) {
          const float* ps = part + sl * stride + (long)src_row * d;
          float4 pv[4];
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int j = threadIdx.x * 4 + c * 1024;
            if (j < d) pv[c] = *reinterpret_cast<const float4*>(ps + j);
          }
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int j = threadIdx.x * 4 + c * 1024;
            if (j < d) {
              v[c].x += pv[c].x; v[c].y += pv[c].y; v[c].z += pv[c].z; v[c].w += pv[c].w;
            }
          }
        }
      }
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int j = threadIdx.x * 4 + c * 1024;
        if (j < d) *reinterpret_cast<float4*>(x + j) = v[c];
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int j = threadIdx.x * 4 + c * 1024;
      if (j < d) ss += v[c].x * v[c].x + v[c].y * v[c].y + v[c].z * v[c].z + v[c].w * v[c].w;
    }
    if (!out) return;
    const float inv = 1.0f / sqrtf(block_sum_256(ss, red) / (float)d + eps);
    T* o = out + (long)i * d;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int j = threadIdx.x * 4 + c * 1024;
      if (j < d) {
        const float4 gg = *reinterpret_cast<const float4*>(g + j);
        store4(o + j, v[c].x * inv * gg.x, v[c].y * inv * gg.y, v[c].z * inv * gg.z,
               v[c].w * inv * gg.w);
      }
    }
    return;
  }
  for (int j = threadIdx.x * 4; j < d; j += 1024) {
    float4 v = *reinterpret_cast<const float4*>(x + j);
    if (part) {
      for (int s = 0; s < splits; ++s) {
        const float4 p = *reinterpret_cast<const float4*>(part + s * stride + (long)src_row * d + j);
        v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
      }
      *reinterpret_cast<float4*>(x + j) = v;
    }
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  if (!out) return;
  const float inv = 1.0f / sqrtf(block_sum_256(ss, red) / (float)d + eps);
  T* o = out + (long)i * d;
  for (int j = threadIdx.x * 4; j < d; j += 1024) {
    float4 v = *reinterpret_cast<const float4*>(x + j);
    float4 gg = *reinterpret_cast<const float4*>(g + j);
    o[j + 0] = from_f32<T>(v.x * inv * gg.x);
    o[j + 1] = from_f32<T>(v.y * inv * gg.y);
    o[j + 2] = from_f32<T>(v.z * inv * gg.z);
    o[j + 3] = from_f32<T>(v.w * inv * gg.w);
  }
}

template <typename T>
hipError_t add_rmsnorm_rows(float* h, const float* part, int splits, long stride, const float* g,
                            int n, int d, float eps, T* out, hipStream_t st) {
  if (n == 0) return hipSuccess;
#define ADD_NORM(S_)                                                                         \
  DLM_LAUNCH((rmsnorm_kernel<T, S_>), dim3(n), dim3(256), 0, st, h, part, splits, stride, g, \
             d, eps, out, (const int*)nullptr, (const int*)nullptr)
  switch (d <= 4096 ? splits : 0) {
    case 1: ADD_NORM(1); break;
    case 2: ADD_NORM(2); break;
    case 4: ADD_NORM(4); break;
    case 8: ADD_NORM(8); break;
    default: ADD_NORM(0); break;
  }
#undef ADD_NORM
  return hipGetLastError();
}

template <typename T>
hipError_t rmsnorm_rows(const float* h, const float* g, int n, int d, float eps, T* out,
                        hipStream_t st) {
  if (n == 0) return hipSuccess;
  DLM_LAUNCH((rmsnorm_kernel<T, 0>), dim3(n), dim3(256), 0, st, const_cast<float*>(h),
                     (const float*)nullptr, 0, 0L, g, d, eps, out, (const int*)nullptr,
                     (const int*)nullptr);
  return hipGetLastError();
}

template <typename T>
hipError_t final_norm_gather(const float* h, const float* g, const int* lm_rows,
                             const int* lm_count, int m_max, int d, float eps, T* u,
                             hipStream_t st) {
  if (m_max == 0) return hipSuccess;
  DLM_LAUNCH((rmsnorm_kernel<T, 0>), dim3(m_max), dim3(256), 0, st, const_cast<float*>(h),
                     (const float*)nullptr, 0, 0L, g, d, eps, u, lm_rows, lm_count);
  return hipGetLastError();
}

// ----------------------------------------------------------------- RoPE --
// cs[n][i] = (cos, sin) of pos(n) * theta^(-2i/dh), angle and trig in fp64.
__global__ void rope_table_kernel(StepPlan p, int half, double log_theta, float2* cs) {
  const int n = blockIdx.x;
  const int r = plan_req_of_row(p, n);
  const double pos = (double)(p.r[r].pos0 + (n - p.r[r].row0));
  for (int i = threadIdx.x; i < half; i += blockDim.x) {
    const double freq = exp(-log_theta * (double)(2 * i) / (double)(2 * half));
    double s, c;
    sincos(pos * freq, &s, &c);
    cs[(long)n * half + i] = make_float2((float)c, (float)s);
  }
}

hipError_t rope_table(const StepPlan& p, int head_dim, float theta, float2* cs, hipStream_t st) {
  if (p.n_rows == 0) return hipSuccess;
  DLM_LAUNCH(rope_table_kernel, dim3(p.n_rows), dim3(64), 0, st, p, head_dim / 2,
                     log((double)theta), cs);
  return hipGetLastError();
}

// One block = one 64-row tile of one request x one head slot:
//   y <  hq         : query head y   -> rotated, stored to q_out[n][y*dh..]
//   y >= hq         : kv head y - hq -> rotated key to K[slot][j][pos][:],
//                                       value (transposed in LDS) to V[slot][j][:][pos]
// The fp32 input is the sum of the split-K partial slices of the QKV GEMM.
// NTH threads per block: 1024 (one pass over the tile) when the launch has few
// blocks, so that each CU keeps more loads in flight; 256 (four quads per
// thread per pass) when it has many.
template <typename T, int DH, int NTH>
__global__ __launch_bounds__(NTH) void qkv_rope_scatter_kernel(
    StepPlan p, const float* __restrict__ qkv, int splits, long split_stride,
    const float2* __restrict__ cs, int hq, int hkv, T* __restrict__ q_out,
    T* __restrict__ kcache, T* __restrict__ vcache, int s_max) {
  constexpr int HALF = DH / 2;
  __shared__ T vt[DH][kQTile + 2];
  const int tile = blockIdx.x;
  // head slots in reverse dispatch order: the key/value blocks (rotation, value
  // transpose and two stores: the longest) start first instead of forming the
  // launch's last wave (GQA 64-request cache step 41 -> 35 us)
  const int y = (int)gridDim.y - 1 - (int)blockIdx.y;
  const int r = plan_req_of_tile(p, tile);
  const ReqPlan& q = p.r[r];
  const int lrow0 = (tile - q.tile0) * kQTile;           // first row within request
  const int nvalid = min(kQTile, q.nrows - lrow0);
  const int qkv_dim = (hq + 2 * hkv) * DH;
  const int row_base = q.row0 + lrow0;
  const int pos_base = q.pos0 + lrow0;


  // rotary pairs (i, i + HALF): each thread takes 4 consecutive i of one row,
  // UNR such quads per pass (a 64-row tile in one pass) with all their loads
  // issued before the stores
  auto rotate = [&](int col0, T* dst_base, long dst_row_stride, bool kv) {
    constexpr int QUADS = HALF / 4, UNR = (kQTile * QUADS + NTH - 1) / NTH;
    const int total = nvalid * QUADS;
    for (int base = threadIdx.x; base < total; base += UNR * blockDim.x) {
      float4 a[UNR], b[UNR], c01[UNR], c23[UNR];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int idx = base + u * blockDim.x;
        if (idx >= total) break;
        const int rr = idx / QUADS, i = (idx % QUADS) * 4;
        const int n = row_base + rr;
        const float* src = qkv + (long)n * qkv_dim + col0 + i;
        a[u] = *reinterpret_cast<const float4*>(src);
        b[u] = *reinterpret_cast<const float4*>(src + HALF);
        c01[u] = *reinterpret_cast<const float4*>(cs + (long)n * HALF + i);
        c23[u] = *reinterpret_cast<const float4*>(cs + (long)n * HALF + i + 2);
      }
      for (int sp = 1; sp < splits; ++sp) {
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
          const int idx = base + u * blockDim.x;
          if (idx >= total) break;
          const int rr = idx / QUADS, i = (idx % QUADS) * 4;
          const float* src = qkv + (long)(row_base + rr) * qkv_dim + col0 + i + sp * split_stride;
          const float4 a2 = *reinterpret_cast<const float4*>(src);
          const float4 b2 = *reinterpret_cast<const float4*>(src + HALF);
          a[u].x += a2.x; a[u].y += a2.y; a[u].z += a2.z; a[u].w += a2.w;
          b[u].x += b2.x; b[u].y += b2.y; b[u].z += b2.z; b[u].w += b2.w;
        }
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int idx = base + u * blockDim.x;
        if (idx >= total) break;
        const int rr = idx / QUADS, i = (idx % QUADS) * 4;
        const int n = row_base + rr;
        T* o = dst_base + (kv ? (long)(pos_base + rr) : (long)n) * dst_row_stride;
        store4(o + i, a[u].x * c01[u].x - b[u].x * c01[u].y, a[u].y * c01[u].z - b[u].y * c01[u].w,
               a[u].z * c23[u].x - b[u].z * c23[u].y, a[u].w * c23[u].z - b[u].w * c23[u].w);
        store4(o + i + HALF, b[u].x * c01[u].x + a[u].x * c01[u].y,
               b[u].y * c01[u].z + a[u].y * c01[u].w, b[u].z * c23[u].x + a[u].z * c23[u].y,
               b[u].w * c23[u].z + a[u].w * c23[u].w);
      }
    }
  };
  if (y < hq) {
    rotate(y * DH, q_out + y * DH, (long)hq * DH, false);
    return;
  }
  const int j = y - hq;
  T* kb = kcache + ((long)(q.slot * hkv + j) * s_max) * DH;
  T* vb = vcache + ((long)(q.slot * hkv + j) * DH) * s_max;
  const int kcol = hq * DH + j * DH;
  const int vcol = (hq + hkv) * DH + j * DH;
  rotate(kcol, kb, DH, true);
  {
    constexpr int UNR = (kQTile * (DH / 4) + NTH - 1) / NTH;
    const int total = nvalid * (DH / 4);
    for (int base = threadIdx.x; base < total; base += UNR * blockDim.x) {
      float4 v[UNR];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int idx = base + u * blockDim.x;
        if (idx >= total) break;
        const int rr = idx / (DH / 4), d = (idx % (DH / 4)) * 4;
        v[u] = *reinterpret_cast<const float4*>(qkv + (long)(row_base + rr) * qkv_dim + vcol + d);
      }
      for (int sp = 1; sp < splits; ++sp) {
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
          const int idx = base + u * blockDim.x;
          if (idx >= total) break;
          const int rr = idx / (DH / 4), d = (idx % (DH / 4)) * 4;
          const float4 v2 = *reinterpret_cast<const float4*>(
              qkv + (long)(row_base + rr) * qkv_dim + vcol + d + sp * split_stride);
          v[u].x += v2.x; v[u].y += v2.y; v[u].z += v2.z; v[u].w += v2.w;
        }
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int idx = base + u * blockDim.x;
        if (idx >= total) break;
        const int rr = idx / (DH / 4), d = (idx % (DH / 4)) * 4;
        vt[d + 0][rr] = from_f32<T>(v[u].x);
        vt[d + 1][rr] = from_f32<T>(v[u].y);
        vt[d + 2][rr] = from_f32<T>(v[u].z);
        vt[d + 3][rr] = from_f32<T>(v[u].w);
      }
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < nvalid * DH; idx += blockDim.x) {
    const int d = idx / nvalid, rr = idx % nvalid;
    vb[(long)d * s_max + pos_base + rr] = vt[d][rr];
  }
}

template <typename T>
hipError_t qkv_rope_scatter(const StepPlan& p, const float* qkv, int splits, long split_stride,
                            const float2* cs, int hq, int hkv, int dh, T* q_out,
                            T* kcache, T* vcache, int s_max, hipStream_t st) {
  if (p.n_tiles == 0) return hipSuccess;
  dim3 g(p.n_tiles, hq + hkv);
  const bool many = (long)p.n_tiles * (hq + hkv) >= 1024;   // four or more blocks per CU
#define ROPE_LAUNCH(DH_, NTH_)                                                                   \
  DLM_LAUNCH((qkv_rope_scatter_kernel<T, DH_, NTH_>), g, dim3(NTH_), 0, st, p, qkv,     \
                     splits, split_stride, cs, hq, hkv, q_out, kcache, vcache, s_max)
  if (dh == 128) {
    if (many) ROPE_LAUNCH(128, 256); else ROPE_LAUNCH(128, 1024);
  } else if (dh == 64) {
    if (many) ROPE_LAUNCH(64, 256); else ROPE_LAUNCH(64, 1024);
  } else {
    return hipErrorInvalidValue;
  }
#undef ROPE_LAUNCH
  return hipGetLastError();
}

// ----------------------------------------------------- LM row selection --
// Rows that get a prediction: the masked positions of each active block
// (all block positions when all_rows != 0), in request order, ascending
// position. One wave per request counts with a ballot; a single block then
// scans the counts in request order. Output indices are packed recompute rows.
__global__ __launch_bounds__(1024) void lm_select_kernel(StepPlan p, const uint8_t* __restrict__ mask,
                                                         int all_rows, int* __restrict__ lm_rows,
                                                         int* __restrict__ lm_count,
                                                         int* __restrict__ req_off,
                                                         int* __restrict__ req_cnt) {
  __shared__ unsigned long long bits[kMaxReq];
  __shared__ int offs[kMaxReq + 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int r = wave; r < p.n_req; r += nw) {
    const ReqPlan& q = p.r[r];
    bool m = false;
    if (lane < q.blk_len) m = all_rows || mask[(long)q.tok_off + q.blk_s + lane] != 0;
    unsigned long long b = __ballot(m);
    if (lane == 0) bits[r] = b;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int r = 0; r < p.n_req; ++r) {
      offs[r] = acc;
      acc += __popcll(bits[r]);
    }
    offs[p.n_req] = acc;
    *lm_count = acc;
  }
  __syncthreads();
  for (int r = wave; r < p.n_req; r += nw) {
    const ReqPlan& q = p.r[r];
    const unsigned long long b = bits[r];
    if (lane == 0) {
      req_off[r] = offs[r];
      req_cnt[r] = __popcll(b);
    }
    if (lane < q.blk_len && ((b >> lane) & 1ull)) {
      const int rank = __popcll(b & ((1ull << lane) - 1ull));
      const int pos = q.blk_s + lane;
      lm_rows[offs[r] + rank] = q.row0 + (pos - q.pos0);
    }
  }
}

hipError_t lm_select_rows(const StepPlan& p, const uint8_t* mask, int all_rows, int* lm_rows,
                          int* lm_count, int* req_lm_off, int* req_lm_cnt, hipStream_t st) {
  DLM_LAUNCH(lm_select_kernel, dim3(1), dim3(1024), 0, st, p, mask, all_rows, lm_rows,
                     lm_count, req_lm_off, req_lm_cnt);
  return hipGetLastError();
}

// --------------------------------------------------------- tile combine --
// conf = 1 / S, tok = lowest argmax, from the per-vocab-tile statistics; one
// wave per row, tiles strided over lanes, then a fixed xor tree: the result
// does not depend on scheduling.
struct Stat { float m; float s; int i; };
__device__ __forceinline__ Stat comb(Stat a, Stat b) {
  Stat r;
  r.m = fmaxf(a.m, b.m);
  float sa = a.s == 0.f ? 0.f : a.s * __expf(a.m - r.m);
  float sb = b.s == 0.f ? 0.f : b.s * __expf(b.m - r.m);
  r.s = sa + sb;
  r.i = a.m > b.m ? a.i : (b.m > a.m ? b.i : min(a.i, b.i));
  return r;
}

__global__ void lm_combine_kernel(const float* __restrict__ pm, const float* __restrict__ ps,
                                  const int* __restrict__ pi, int tiles, int ld,
                                  const int* __restrict__ lm_count, float* __restrict__ conf,
                                  int* __restrict__ tok) {
  const int row = blockIdx.x;
  if (row >= *lm_count) return;
  const int lane = threadIdx.x;
  Stat a = {-INFINITY, 0.f, 0x7fffffff};
  for (int t = lane; t < tiles; t += 64) {
    Stat b = {pm[(long)t * ld + row], ps[(long)t * ld + row], pi[(long)t * ld + row]};
    a = comb(a, b);
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    Stat b;
    b.m = __shfl_xor(a.m, o, 64);
    b.s = __shfl_xor(a.s, o, 64);
    b.i = __shfl_xor(a.i, o, 64);
    a = comb(a, b);
  }
  if (lane == 0) {
    conf[row] = 1.0f / a.s;
    tok[row] = a.i;
  }
}

hipError_t lm_combine(const float* pm, const float* ps, const int* pi, int tiles, int ld,
                      const int* lm_count, int m_max, float* conf, int* tok, hipStream_t st) {
  if (m_max == 0) return hipSuccess;
  DLM_LAUNCH(lm_combine_kernel, dim3(m_max), dim3(64), 0, st, pm, ps, pi, tiles, ld,
                     lm_count, conf, tok);
  return hipGetLastError();
}

// -------------------------------------------------- threshold / unmask --
// Wave 0 of the request's block, lane j = block position blk_s + j. Masked
// positions whose confidence exceeds gamma are unmasked; if none does, the
// most confident masked position (lowest position on ties) is unmasked alone.
// Unmasked (pos, tok, conf) are written in ascending position order.
// Optional statistics (paper, "Step Prediction"; appendix "Step Predictor
// Features"): count, min, quartiles, median, mean and max of the confidences of
// the request's unmasked output positions, and the unmasked count of the block.
constexpr int kUnmaskThreads = 256;
constexpr int kStatCap = 8192;          // largest sequence length: output positions per request

// One block per request. Wave 0 takes the unmask decision over the active
// block (one lane per position); with stats requested, the whole block then
// gathers the confidences of the request's unmasked output positions into
// LDS (order does not matter: they are sorted next), sorts them with a
// bitonic network and reads the order statistics off the sorted array.
__global__ __launch_bounds__(kUnmaskThreads) void unmask_kernel(
    StepPlan p, const float* __restrict__ conf, const int* __restrict__ tok,
    const int* __restrict__ req_lm_off, int32_t* __restrict__ tokens, uint8_t* __restrict__ mask,
    int32_t* __restrict__ n_unmasked, int32_t* __restrict__ out_pos, int32_t* __restrict__ out_tok,
    float* __restrict__ out_conf, float* __restrict__ blk_conf, int32_t* __restrict__ blk_tok,
    float* __restrict__ tok_conf, float* __restrict__ stats) {
  const int r = blockIdx.x;
  const ReqPlan& q = p.r[r];
  const int tid = threadIdx.x;
  if (tid < 64) {
    const int lane = tid;
    const long ti = (long)q.tok_off + q.blk_s + lane;
    const bool in_blk = lane < q.blk_len;
    const bool masked = in_blk && mask[ti] != 0;
    const unsigned long long mb = __ballot(masked);
    float c = -1.0f;
    int t = 0;
    if (masked) {
      const int idx = req_lm_off[r] + __popcll(mb & ((1ull << lane) - 1ull));
      c = conf[idx];
      t = tok[idx];
    }
    bool sel = masked && c > q.gamma;
    unsigned long long sb = __ballot(sel);
    if (sb == 0ull && mb != 0ull) {
      // wave argmax of c over masked lanes, lowest lane on ties
      float bc = masked ? c : -2.0f;
      int bl = masked ? lane : 64;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        float oc = __shfl_xor(bc, o, 64);
        int ol = __shfl_xor(bl, o, 64);
        if (oc > bc || (oc == bc && ol < bl)) { bc = oc; bl = ol; }
      }
      sel = lane == bl;
      sb = __ballot(sel);
    }
    if (blk_conf) blk_conf[r * kMaxBlock + lane] = masked ? c : -1.0f;
    if (blk_tok) blk_tok[r * kMaxBlock + lane] = masked ? t : -1;
    if (sel) {
      const int k = __popcll(sb & ((1ull << lane) - 1ull));
      out_pos[r * kMaxBlock + k] = q.blk_s + lane;
      out_tok[r * kMaxBlock + k] = t;
      out_conf[r * kMaxBlock + k] = c;
      tokens[ti] = t;
      mask[ti] = 0;
      if (tok_conf) tok_conf[ti] = c;
    }
    if (lane == 0) {
      n_unmasked[r] = __popcll(sb);
      if (stats) stats[r * kNStats + 7] = (float)(q.blk_len - __popcll(mb) + __popcll(sb));
    }
  }
  if (!stats) return;                         // uniform: a kernel argument
  __shared__ float sv[kStatCap];
  __shared__ int s_n;
  __shared__ float s_part[kUnmaskThreads / 64];
  if (tid == 0) s_n = 0;
  __syncthreads();                            // also publishes wave 0's mask / tok_conf writes
  // gather (LDS atomic slot: the order is irrelevant, the values are sorted)
  const long base = q.tok_off;
  for (int pos = q.prompt_len + tid; pos < q.seq_len; pos += kUnmaskThreads) {
    if (mask[base + pos] == 0) {
      const float v = tok_conf[base + pos];
      sv[atomicAdd(&s_n, 1)] = v;
    }
  }
  __syncthreads();
  const int n = s_n;
  int n2 = 1;
  while (n2 < n) n2 <<= 1;
  for (int i = n + tid; i < n2; i += kUnmaskThreads) sv[i] = INFINITY;
  __syncthreads();
  // bitonic sort, ascending
  for (int k = 2; k <= n2; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < n2; i += kUnmaskThreads) {
        const int ij = i ^ j;
        if (ij > i) {
          const float a = sv[i], b = sv[ij];
          if ((a > b) == ((i & k) == 0)) {
            sv[i] = b;
            sv[ij] = a;
          }
        }
      }
      __syncthreads();
    }
  }
  // mean over the sorted array (the gather order depends on scheduling):
  // per-thread strided sums, then a fixed-order reduction
  float lsum = 0.f;
  for (int i = tid; i < n; i += kUnmaskThreads) lsum += sv[i];
  lsum = wave_sum(lsum);
  if ((tid & 63) == 0) s_part[tid >> 6] = lsum;
  __syncthreads();
  if (tid == 0) {
    float* o = stats + r * kNStats;
    o[0] = (float)n;
    if (n == 0) {
      for (int i = 1; i < 7; ++i) o[i] = 0.f;
    } else {
      float tot = 0.f;
      for (int w = 0; w < kUnmaskThreads / 64; ++w) tot += s_part[w];
      auto quant = [&](int quarter) {     // p = quarter / 4: h = (n-1) p is exact in fp32
        const int hq = (n - 1) * quarter;
        const int j = hq / 4;
        const float f = (float)(hq % 4) * 0.25f;
        const float lo = sv[j], hi = j + 1 < n ? sv[j + 1] : sv[j];
        return fmaf(f, hi - lo, lo);
      };
      o[1] = sv[0];
      o[2] = quant(1);
      o[3] = quant(2);
      o[4] = tot / (float)n;
      o[5] = quant(3);
      o[6] = sv[n - 1];
    }
  }
}

hipError_t unmask_select(const StepPlan& p, const float* conf, const int* tok,
                         const int* req_lm_off, int32_t* tokens, uint8_t* mask,
                         int32_t* n_unmasked, int32_t* out_pos, int32_t* out_tok,
                         float* out_conf, float* blk_conf, int32_t* blk_tok, float* tok_conf,
                         float* stats, hipStream_t st) {
  DLM_LAUNCH(unmask_kernel, dim3(p.n_req), dim3(kUnmaskThreads), 0, st, p, conf, tok,
                     req_lm_off, tokens, mask, n_unmasked, out_pos, out_tok, out_conf, blk_conf,
                     blk_tok, tok_conf, stats);
  return hipGetLastError();
}

#define INST(T)                                                                                 \
  template hipError_t embed_rows<T>(const StepPlan&, const T*, int, int, int, const int32_t*,  \
                                    const uint8_t*, float*, hipStream_t);                      \
  template hipError_t rmsnorm_rows<T>(const float*, const float*, int, int, float, T*,         \
                                      hipStream_t);                                            \
  template hipError_t add_rmsnorm_rows<T>(float*, const float*, int, long, const float*, int,  \
                                          int, float, T*, hipStream_t);                        \
  template hipError_t final_norm_gather<T>(const float*, const float*, const int*, const int*, \
                                           int, int, float, T*, hipStream_t);                  \
  template hipError_t qkv_rope_scatter<T>(const StepPlan&, const float*, int, long,            \
                                          const float2*, int, int, int, T*, T*, T*, int,       \
                                          hipStream_t);
INST(bf16)
INST(float)

}  // namespace dlm
