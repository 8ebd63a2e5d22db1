// Bidirectional (non-causal) attention of the recomputed query rows over every
// cached key/value position of their request's slot: O = softmax(Q K^T /
// sqrt(dh)) V per query head; query head h reads key/value head h / (Hq/Hkv).
//
// bf16 path (matrix cores): one block = 64 query rows of one request x one
// query head, 4 waves of 16 rows. Key tiles of 64 positions are staged in LDS
// (keys row-major, values transposed, which is how the cache stores them).
// Each wave computes S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (keys as the A
// operand, its 16 query rows as B, held in registers), so that every lane
// ends up owning one query and 16 keys: the online softmax needs only two
// cross-lane steps, and the probabilities feed O^T = V^T P^T directly as the B
// operand (the key order inside the 32-wide k step is permuted identically in
// A and B, which leaves the sum unchanged). fp32 softmax, exp2 with the scale
// folded in; P enters the PV product as the sum of two bf16 terms (about 16
// significant bits), the output is rounded to bf16.
//
// fp32 path: a plain per-query-row kernel (one lane per query row) over LDS
// tiles; it serves the small fp32 model.
#include "common.h"
#include "kernels.h"

namespace dlm {

constexpr int kKeyTile = 64;

template <int DH>
__global__ __launch_bounds__(256) void attn_bf16_kernel(StepPlan p, const bf16* __restrict__ q,
                                                        const bf16* __restrict__ kc,
                                                        const bf16* __restrict__ vc, int s_max,
                                                        int hq, int hkv, bf16* __restrict__ out,
                                                        float scale_log2) {
  constexpr int KS = DH + 8;            // K tile row stride (elements)
  constexpr int VS = kKeyTile + 8;      // V^T tile row stride (elements)
  constexpr int NDB = DH / 16;          // output dh blocks
  constexpr int NKS = DH / 32;          // k steps of S
  __shared__ __attribute__((aligned(16))) bf16 ks[kKeyTile * KS];
  __shared__ __attribute__((aligned(16))) bf16 vs[DH * VS];

  // head-major grid: consecutive blocks (which the dispatcher spreads over the
  // XCDs round-robin) are different heads, so the query tiles of one head
  // (same K/V) land on the same XCD and share its L2
  const int h = blockIdx.x, tile = blockIdx.y;
  const int r = plan_req_of_tile(p, tile);
  const ReqPlan& rq = p.r[r];
  const int lrow0 = (tile - rq.tile0) * kQTile;
  const int nvalid = min(kQTile, rq.nrows - lrow0);
  const int L = rq.seq_len;
  const int kvh = h / (hq / hkv);
  const bf16* kb = kc + ((long)(rq.slot * hkv + kvh) * s_max) * DH;
  const bf16* vb = vc + ((long)(rq.slot * hkv + kvh) * DH) * s_max;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int qr = wave * 16 + (lane & 15);          // query row of this lane in the tile
  const bool q_ok = qr < nvalid;
  const long qrow = rq.row0 + lrow0 + qr;
  const int g = lane >> 4;

  // Q fragments (B operand): col = query lane&15, k = dh 32*s + 8*g .. +7
  u32x4 qf[NKS];
#pragma unroll
  for (int s = 0; s < NKS; ++s) {
    if (q_ok)
      qf[s] = *reinterpret_cast<const u32x4*>(q + qrow * hq * DH + h * DH + s * 32 + g * 8);
    else
      qf[s] = u32x4{0u, 0u, 0u, 0u};
  }

  f32x4 o[NDB];
#pragma unroll
  for (int i = 0; i < NDB; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  // K/V^T tiles go through registers: the next tile's global loads are issued
  // before the current tile's MFMAs and written to LDS after them.
  constexpr int KCH = kKeyTile * (DH / 8) / 256;   // 16-byte K chunks per thread
  constexpr int VCH = DH * (kKeyTile / 8) / 256;   // 16-byte V^T chunks per thread
  u32x4 kreg[KCH], vreg[VCH];
  auto load_tile = [&](int key0) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + i * 256;
      const int kk = c / (DH / 8), cc = c % (DH / 8);
      kreg[i] = key0 + kk < L
                    ? *reinterpret_cast<const u32x4*>(kb + (long)(key0 + kk) * DH + cc * 8)
                    : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
      const int c = tid + i * 256;
      const int d = c / (kKeyTile / 8), cc = c % (kKeyTile / 8);
      const int kk0 = key0 + cc * 8;
      const bf16* src = vb + (long)d * s_max + kk0;
      if (kk0 + 8 <= L) {
        vreg[i] = *reinterpret_cast<const u32x4*>(src);
      } else {
        bf16 tmp[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) tmp[e] = (kk0 + e < L) ? src[e] : (bf16)0.0f;
        vreg[i] = *reinterpret_cast<const u32x4*>(tmp);
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + i * 256;
      *reinterpret_cast<u32x4*>(ks + (c / (DH / 8)) * KS + (c % (DH / 8)) * 8) = kreg[i];
    }
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
      const int c = tid + i * 256;
      *reinterpret_cast<u32x4*>(vs + (c / (kKeyTile / 8)) * VS + (c % (kKeyTile / 8)) * 8) = vreg[i];
    }
  };

  const int ntiles = ceil_div(L, kKeyTile);
  load_tile(0);
  store_tile();
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int key0 = t * kKeyTile;
    if (t + 1 < ntiles) load_tile(key0 + kKeyTile);

    // S^T blocks: sblk[kb][i] = score(key = 16*kb + 4*g + i, query = lane&15)
    f32x4 sblk[4];
#pragma unroll
    for (int kbk = 0; kbk < 4; ++kbk) {
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NKS; ++s) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(ks + (kbk * 16 + (lane & 15)) * KS + s * 32 + g * 8);
        acc = mfma16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, qf[s]), acc);
      }
      sblk[kbk] = acc;
    }
    // scale (log2 domain) and mask keys beyond L
    float mt = -INFINITY;
#pragma unroll
    for (int kbk = 0; kbk < 4; ++kbk)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = key0 + kbk * 16 + 4 * g + i;
        float v = key < L ? sblk[kbk][i] * scale_log2 : -INFINITY;
        sblk[kbk][i] = v;
        mt = fmaxf(mt, v);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float m_new = fmaxf(m_run, mt);
    const float alpha = exp2f(m_run - m_new);     // m_run = -inf on the first tile -> 0
    float lsum = 0.f;
#pragma unroll
    for (int kbk = 0; kbk < 4; ++kbk)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float e = exp2f(sblk[kbk][i] - m_new);
        sblk[kbk][i] = e;
        lsum += e;
      }
    l_run = l_run * alpha + lsum;
    m_run = m_new;
#pragma unroll
    for (int i = 0; i < NDB; ++i) o[i] *= alpha;

    // O^T += V^T P^T over two 32-key steps; B operand slot 8g+e <-> key
    // 32*j + (e < 4 ? 4g + e : 16 + 4g + e - 4)
    // P = P_hi + P_lo with both terms bf16: the product with the bf16 values
    // keeps about 16 bits of P instead of 8 (two MFMAs per block).
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      bf16x8 ph, pl;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float pv = e < 4 ? sblk[2 * j][e] : sblk[2 * j + 1][e - 4];
        ph[e] = (bf16)pv;
        pl[e] = (bf16)(pv - (float)ph[e]);
      }
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const bf16* vrow = vs + (db * 16 + (lane & 15)) * VS + 32 * j + 4 * g;
        const u32x2 lo = *reinterpret_cast<const u32x2*>(vrow);
        const u32x2 hi = *reinterpret_cast<const u32x2*>(vrow + 16);
        const bf16x8 a = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
        o[db] = mfma16_bf16(a, ph, o[db]);
        o[db] = mfma16_bf16(a, pl, o[db]);
      }
    }
    if (t + 1 < ntiles) {
      __syncthreads();   // every wave is done with tile t
      store_tile();
      __syncthreads();
    }
  }
  // finish: l over the 4 lanes sharing the query, normalise, store
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_run;
  if (q_ok) {
    bf16* dst = out + qrow * hq * DH + h * DH;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      bf16x4 v;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = (bf16)(o[db][i] * inv);
      *reinterpret_cast<bf16x4*>(dst + db * 16 + 4 * g) = v;
    }
  }
}

// fp32: one lane per query row; K and V^T tiles staged in LDS.
template <int DH>
__global__ __launch_bounds__(64) void attn_f32_kernel(StepPlan p, const float* __restrict__ q,
                                                      const float* __restrict__ kc,
                                                      const float* __restrict__ vc, int s_max,
                                                      int hq, int hkv, float* __restrict__ out,
                                                      float scale) {
  __shared__ float ks[kKeyTile][DH + 1];
  __shared__ float vs[DH][kKeyTile + 1];
  const int tile = blockIdx.x, h = blockIdx.y;
  const int r = plan_req_of_tile(p, tile);
  const ReqPlan& rq = p.r[r];
  const int lrow0 = (tile - rq.tile0) * kQTile;
  const int nvalid = min(kQTile, rq.nrows - lrow0);
  const int L = rq.seq_len;
  const int kvh = h / (hq / hkv);
  const float* kb = kc + ((long)(rq.slot * hkv + kvh) * s_max) * DH;
  const float* vb = vc + ((long)(rq.slot * hkv + kvh) * DH) * s_max;
  const int lane = threadIdx.x;
  const bool q_ok = lane < nvalid;
  const long qrow = rq.row0 + lrow0 + lane;
  float qv[DH], acc[DH];
#pragma unroll
  for (int d = 0; d < DH; ++d) {
    qv[d] = q_ok ? q[qrow * hq * DH + h * DH + d] : 0.f;
    acc[d] = 0.f;
  }
  float m_run = -INFINITY, l_run = 0.f;
  for (int key0 = 0; key0 < L; key0 += kKeyTile) {
    __syncthreads();
    for (int c = lane; c < kKeyTile * DH; c += 64) {
      const int kk = c / DH, d = c % DH;
      ks[kk][d] = key0 + kk < L ? kb[(long)(key0 + kk) * DH + d] : 0.f;
    }
    for (int c = lane; c < kKeyTile * DH; c += 64) {
      const int d = c / kKeyTile, kk = c % kKeyTile;
      vs[d][kk] = key0 + kk < L ? vb[(long)d * s_max + key0 + kk] : 0.f;
    }
    __syncthreads();
    const int nk = min(kKeyTile, L - key0);
    for (int kk = 0; kk < nk; ++kk) {
      float s = 0.f;
#pragma unroll
      for (int d = 0; d < DH; ++d) s += qv[d] * ks[kk][d];
      s *= scale;
      const float m_new = fmaxf(m_run, s);
      const float alpha = expf(m_run - m_new);
      const float e = expf(s - m_new);
      l_run = l_run * alpha + e;
#pragma unroll
      for (int d = 0; d < DH; ++d) acc[d] = acc[d] * alpha + e * vs[d][kk];
      m_run = m_new;
    }
  }
  if (q_ok) {
    float* dst = out + qrow * hq * DH + h * DH;
    const float inv = 1.0f / l_run;
#pragma unroll
    for (int d = 0; d < DH; ++d) dst[d] = acc[d] * inv;
  }
}

template <>
hipError_t attention<bf16>(const StepPlan& p, const bf16* q, const bf16* kc, const bf16* vc,
                           int s_max, int hq, int hkv, int dh, bf16* out, hipStream_t st) {
  if (p.n_tiles == 0) return hipSuccess;
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)dh);
  dim3 g(hq, p.n_tiles);
  if (dh == 128)
    hipLaunchKernelGGL(attn_bf16_kernel<128>, g, dim3(256), 0, st, p, q, kc, vc, s_max, hq, hkv,
                       out, scale_log2);
  else if (dh == 64)
    hipLaunchKernelGGL(attn_bf16_kernel<64>, g, dim3(256), 0, st, p, q, kc, vc, s_max, hq, hkv,
                       out, scale_log2);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <>
hipError_t attention<float>(const StepPlan& p, const float* q, const float* kc, const float* vc,
                            int s_max, int hq, int hkv, int dh, float* out, hipStream_t st) {
  if (p.n_tiles == 0) return hipSuccess;
  const float scale = 1.0f / sqrtf((float)dh);
  dim3 g(p.n_tiles, hq);
  if (dh == 64)
    hipLaunchKernelGGL(attn_f32_kernel<64>, g, dim3(64), 0, st, p, q, kc, vc, s_max, hq, hkv,
                       out, scale);
  else if (dh == 128)
    hipLaunchKernelGGL(attn_f32_kernel<128>, g, dim3(64), 0, st, p, q, kc, vc, s_max, hq, hkv,
                       out, scale);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace dlm
