// Bidirectional (non-causal) attention of the recomputed query rows over every
// cached key/value position of their request's slot: O = softmax(Q K^T /
// sqrt(dh)) V per query head; query head h reads key/value head h / (Hq/Hkv).
//
// bf16 path (matrix cores), two kernels:
//  * attn_gqa_kernel: one block = all query heads that share a key/value head
//    (one for MHA) x 16-64 query rows of one request; 64-key tiles loaded
//    directly into a two-stage LDS ring. Used for grouped-query attention and
//    for MHA launches with at least two blocks per CU.
//  * attn_bf16_kernel: one block = 32 or 64 query rows of one request x one
//    query head; waves split the rows in groups of 16 and the keys in two
//    groups, tiles staged through registers. Used for MHA launches with few
//    blocks (one request's no-cache step, cache steps of short blocks).
// Key tiles are staged in LDS keys row-major and values transposed, which is
// how the cache stores them.
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

// P split into hi + lo bf16 terms (p = hi + lo to about 16 significant bits)
// for the eight probabilities a lane feeds one PV MFMA: lo = bf16(p - hi),
// converted two at a time (one packed conversion per pair for each term)
__device__ __forceinline__ void split_p8(const f32x4& a, const f32x4& b, bf16x8& ph, bf16x8& pl) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const f32x2_t v = e < 2 ? f32x2_t{a[2 * e], a[2 * e + 1]} : f32x2_t{b[2 * e - 4], b[2 * e - 3]};
    const bf16x2_t h = __builtin_convertvector(v, bf16x2_t);
    const bf16x2_t l = __builtin_convertvector(v - __builtin_convertvector(h, f32x2_t), bf16x2_t);
    ph[2 * e] = h[0];
    ph[2 * e + 1] = h[1];
    pl[2 * e] = l[0];
    pl[2 * e + 1] = l[1];
  }
}


constexpr int kKeyTile = 64;

// Wave layout: QG query groups of 16 rows x KG key groups. A block stages
// key tiles of 64 * KG positions; key group kg works on keys [64 kg, 64 kg +
// 64) of each tile. Each wave keeps its own online-softmax state; the key
// groups are merged in LDS at the end (rescaling by the group maxima), so the
// result is the same softmax over all keys.
//
// Softmax bookkeeping per query: m is a reference maximum of the raw scores,
// l and O^T are kept relative to 2^((s - m) c) with c = log2(e) / sqrt(dh).
// m is only moved (and l, O^T rescaled) when a tile's maximum exceeds it by
// more than 8 / c, so the weights stay below 2^8 and most tiles skip the
// rescale; the normalised result is the same.
// P is fed to the PV product as two bf16 terms (P = P_hi + P_lo, about
// 16 significant bits, two MFMAs per block) instead of one.
template <int DH, int QG, int KG>
__global__ __launch_bounds__(QG* KG * 64) void attn_bf16_kernel(StepPlan p, const bf16* __restrict__ q,
                                                               const bf16* __restrict__ kc,
                                                               const bf16* __restrict__ vc,
                                                               int s_max, int hq, int hkv,
                                                               bf16* __restrict__ out,
                                                               float scale_log2) {
  constexpr int NT = QG * KG * 64;
  constexpr int QT = 16 * QG;             // query rows per block
  constexpr int SK = 64 * KG;             // keys per staged tile
  constexpr int KS = DH + 8;              // K tile row stride (elements)
  constexpr int VS = SK + 8;              // V^T tile row stride (elements)
  constexpr int NDB = DH / 16;            // output dh blocks
  constexpr int NKS = DH / 32;            // k steps of S
  __shared__ __attribute__((aligned(16))) bf16 ks[SK * KS];
  __shared__ __attribute__((aligned(16))) bf16 vs[DH * VS];

  // head-major grid: consecutive blocks (spread over the XCDs round-robin) are
  // different heads, so the query tiles of one head share one XCD's L2
  const int h = blockIdx.x, tile = blockIdx.y;
  // request of this tile: tiles of QT rows are numbered request by request
  int r = 0, t0 = 0;
  for (; r + 1 < p.n_req; ++r) {
    const int nt = (p.r[r].nrows + QT - 1) / QT;
    if (tile < t0 + nt) break;
    t0 += nt;
  }
  const ReqPlan& rq = p.r[r];
  const int lrow0 = (tile - t0) * QT;
  const int nvalid = min(QT, rq.nrows - lrow0);
  const int L = rq.seq_len;
  const int kvh = h / (hq / hkv);
  const bf16* kb = kc + ((long)(rq.slot * hkv + kvh) * s_max) * DH;
  const bf16* vb = vc + ((long)(rq.slot * hkv + kvh) * DH) * s_max;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int qg = wave % QG, kg = wave / QG;
  const int qr = qg * 16 + (lane & 15);           // query row of this lane in the tile
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
  float m_ref = -INFINITY, l_run = 0.f;

  // K/V^T tiles go through registers: the next tile's global loads are issued
  // before the current tile's MFMAs and written to LDS after them.
  constexpr int KCH = SK * (DH / 8) / NT;   // 16-byte K chunks per thread
  constexpr int VCH = DH * (SK / 8) / NT;   // 16-byte V^T chunks per thread
  static_assert(KCH * NT == SK * (DH / 8) && VCH * NT == DH * (SK / 8), "tile split");
  u32x4 kreg[KCH], vreg[VCH];
  auto load_tile = [&](int key0) {
    if (key0 + SK <= L) {                       // whole tile inside the sequence
#pragma unroll
      for (int i = 0; i < KCH; ++i) {
        const int c = tid + i * NT;
        kreg[i] = *reinterpret_cast<const u32x4*>(kb + (long)(key0 + c / (DH / 8)) * DH +
                                                  (c % (DH / 8)) * 8);
      }
#pragma unroll
      for (int i = 0; i < VCH; ++i) {
        const int c = tid + i * NT;
        vreg[i] = *reinterpret_cast<const u32x4*>(vb + (long)(c / (SK / 8)) * s_max + key0 +
                                                  (c % (SK / 8)) * 8);
      }
    } else {
      // last tile: keys >= L read as zero. A V^T chunk starting below L lies
      // inside the slot (L <= s_max, both chunk start and s_max multiples of
      // 8); its values at keys >= L are cleared.
#pragma unroll
      for (int i = 0; i < KCH; ++i) {
        const int c = tid + i * NT;
        const int kk = key0 + c / (DH / 8);
        kreg[i] = kk < L ? *reinterpret_cast<const u32x4*>(kb + (long)kk * DH + (c % (DH / 8)) * 8)
                         : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int i = 0; i < VCH; ++i) {
        const int c = tid + i * NT;
        const int kk0 = key0 + (c % (SK / 8)) * 8;
        u32x4 v = u32x4{0u, 0u, 0u, 0u};
        if (kk0 < L) {
          v = *reinterpret_cast<const u32x4*>(vb + (long)(c / (SK / 8)) * s_max + kk0);
          const int n = L - kk0;                // valid keys in this chunk (> 0)
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const uint32_t keep = (2 * w < n ? 0x0000ffffu : 0u) | (2 * w + 1 < n ? 0xffff0000u : 0u);
            v[w] &= keep;
          }
        }
        vreg[i] = v;
      }
    }
  };
  // K rows are stored in the permuted key order of the shared-tile kernel:
  // inside each group of 32 keys, key 8 g + 4 h + i goes to row 16 h + 4 g + i
  // (h < 2, g < 4, i < 4), so the S^T values lane group g owns are the keys
  // 8 g .. 8 g + 7 of each 32-key group and V^T is read as one 16-byte chunk
  // per lane
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + i * NT;
      const int k = c / (DH / 8);
      const int row = (k & ~31) | (((k >> 2) & 1) << 4) | (((k >> 3) & 3) << 2) | (k & 3);
      *reinterpret_cast<u32x4*>(ks + row * KS + (c % (DH / 8)) * 8) = kreg[i];
    }
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
      const int c = tid + i * NT;
      *reinterpret_cast<u32x4*>(vs + (c / (SK / 8)) * VS + (c % (SK / 8)) * 8) = vreg[i];
    }
  };

  const int ntiles = ceil_div(L, SK);
  load_tile(0);
  store_tile();
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int key0 = t * SK + kg * 64;          // this wave's 64 keys
    if (t + 1 < ntiles) load_tile((t + 1) * SK);
    const bf16* ksg = ks + kg * 64 * KS;

    // S^T blocks: sblk[kb][i] = raw score(key = key0 + 32 (kb / 2) + 8 g + 4 (kb % 2) + i,
    // query = lane&15)
    f32x4 sblk[4];
#pragma unroll
    for (int kbk = 0; kbk < 4; ++kbk) {
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NKS; ++s) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(ksg + (kbk * 16 + (lane & 15)) * KS + s * 32 + g * 8);
        acc = mfma16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, qf[s]), acc);
      }
      sblk[kbk] = acc;
    }
    if (t == ntiles - 1) {                      // keys beyond L only in the last tile
#pragma unroll
      for (int kbk = 0; kbk < 4; ++kbk)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (key0 + 32 * (kbk >> 1) + 8 * g + 4 * (kbk & 1) + i >= L) sblk[kbk][i] = -INFINITY;
    }
    float mt = -INFINITY;
#pragma unroll
    for (int kbk = 0; kbk < 4; ++kbk)
#pragma unroll
      for (int i = 0; i < 4; ++i) mt = fmaxf(mt, sblk[kbk][i]);
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    // move the reference maximum only on a large increase (false while both
    // are -inf: a key group that has seen no key below L yet)
    const bool grow = (mt - m_ref) * scale_log2 > 8.0f;
    if (__builtin_amdgcn_ballot_w64(grow)) {
      const float alpha = grow ? __builtin_amdgcn_exp2f((m_ref - mt) * scale_log2) : 1.0f;
      if (grow) m_ref = mt;
      l_run *= alpha;
#pragma unroll
      for (int i = 0; i < NDB; ++i) o[i] *= alpha;
    }
    const float nm = m_ref == -INFINITY ? 0.0f : -m_ref * scale_log2;
    float lsum = 0.f;
#pragma unroll
    for (int kbk = 0; kbk < 4; ++kbk)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float e = __builtin_amdgcn_exp2f(fmaf(sblk[kbk][i], scale_log2, nm));
        sblk[kbk][i] = e;
        lsum += e;
      }
    l_run += lsum;

    // O^T += V^T P^T over two 32-key steps; B operand slot 8g+e <-> key
    // 32*j + 8g + e (sblk[2j] holds keys 8g..8g+3, sblk[2j+1] keys 8g+4..8g+7)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      bf16x8 ph, pl;
      split_p8(sblk[2 * j], sblk[2 * j + 1], ph, pl);
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const bf16* vrow = vs + (db * 16 + (lane & 15)) * VS + kg * 64 + 32 * j + 8 * g;
        const bf16x8 a = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(vrow));
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

  // merge the key groups: groups kg > 0 publish (m, partial l, O^T) in LDS,
  // group 0 of the same query group rescales and adds them
  if constexpr (KG > 1) {
    __syncthreads();                              // K/V tiles no longer needed
    float* xm = reinterpret_cast<float*>(ks);     // [KG-1][QG][64]
    float* xl = xm + (KG - 1) * QG * 64;          // [KG-1][QG][64]
    float* xo = reinterpret_cast<float*>(vs);     // [KG-1][QG][NDB*4][64]
    static_assert((KG - 1) * QG * 64 * 2 * 4 <= SK * KS * 2, "merge scratch (m, l)");
    static_assert((KG - 1) * QG * NDB * 4 * 64 * 4 <= DH * VS * 2, "merge scratch (O)");
    if (kg > 0) {
      const int slot = (kg - 1) * QG + qg;
      xm[slot * 64 + lane] = m_ref;
      xl[slot * 64 + lane] = l_run;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) xo[(slot * NDB * 4 + db * 4 + i) * 64 + lane] = o[db][i];
    }
    __syncthreads();
    if (kg > 0) return;
#pragma unroll
    for (int k = 1; k < KG; ++k) {
      const int slot = (k - 1) * QG + qg;
      const float m2 = xm[slot * 64 + lane];
      const float l2 = xl[slot * 64 + lane];
      const float mm = fmaxf(m_ref, m2);
      const float a1 = m_ref == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f((m_ref - mm) * scale_log2);
      const float a2 = m2 == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f((m2 - mm) * scale_log2);
      l_run = l_run * a1 + l2 * a2;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          o[db][i] = o[db][i] * a1 + xo[(slot * NDB * 4 + db * 4 + i) * 64 + lane] * a2;
      m_ref = mm;
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

// Shared-tile kernel (GH query heads per key/value head; GH = 1 for MHA):
// one block = the GH query heads of one key/value head x QG groups of 16
// query rows of one request, one wave per (query head, row group), so every
// staged K/V tile serves GH * QG * 16 query rows. Tiles of 64 keys are fetched with
// direct global->LDS loads into a two-stage ring: the next tile's loads run
// during the current tile's MFMAs and no registers hold tiles in flight,
// which keeps the register count low enough for two blocks per CU.
//
// LDS layout of a stage:
//   K: 64 rows of DH. Row rho holds key pi(rho) of the tile, where inside each
//      group of 32 keys pi(16 h + 4 g + i) = 8 g + 4 h + i (h < 2, g < 4,
//      i < 4). With this order the S^T values a lane of lane group g owns
//      are the keys 8 g .. 8 g + 7 of each 32-key group, which is the k slice
//      that lane group supplies to the PV MFMA, so V^T is read as one
//      16-byte chunk per lane and no shuffle is needed.
//   V^T: DH rows of 64 keys (128 bytes).
//   The 16-byte chunk c of row r is stored at chunk slot c ^ (r & 7): the
//   eight lanes of one LDS read phase (one chunk of eight consecutive rows)
//   hit distinct banks. Each lane of a load instruction fetches the global
//   chunk that belongs at its slot.
// Keys at or beyond L inside the last tile are read from the slot (a slot
// holds s_max positions, a multiple of 64) and then masked: their scores are
// set to -inf and their V^T entries cleared in LDS.
template <int DH, int GH, int QG>
__global__ __launch_bounds__(GH* QG * 64) void attn_gqa_kernel(StepPlan p, const bf16* __restrict__ q,
                                                             const bf16* __restrict__ kc,
                                                             const bf16* __restrict__ vc,
                                                             int s_max, int hq, int hkv, int n_tiles,
                                                             bf16* __restrict__ out,
                                                             float scale_log2) {
  constexpr int NW = GH * QG;              // waves
  constexpr int NT = NW * 64;
  constexpr int QT = 16 * QG;              // query rows per block
  constexpr int SK = 64;                   // keys per tile
  constexpr int KRB = DH * 2;              // K row bytes
  constexpr int KCPR = DH / 8;             // 16-byte chunks per K row
  constexpr int KRPI = 1024 / KRB;         // K rows per load instruction
  constexpr int NKI = SK / KRPI;           // K load instructions per tile
  constexpr int NVI = DH / 8;              // V^T load instructions per tile (8 rows each)
  constexpr int NI = NKI + NVI;
  constexpr int IPW = (NI + NW - 1) / NW;  // load instructions per wave (at most)
  constexpr int KBYTES = SK * KRB;
  constexpr int STAGE = KBYTES + DH * SK * 2;
  constexpr int NDB = DH / 16;             // output dh blocks
  constexpr int NKS = DH / 32;             // k steps of S
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

  // Block order: blocks are handed out in linear order round-robin over the
  // XCDs; the linear id is remapped so that each XCD receives one contiguous
  // range of (key/value head, query tile) with query tiles fastest, so the
  // row tiles of one request and key/value head run on one XCD at about the
  // same time and share its L2.
  int kvh, tile;
  {
    const int total = gridDim.x, id = blockIdx.x;
    const int xcd = id % kXcds, per = total / kXcds, rem = total % kXcds;
    const int lid = xcd * per + min(xcd, rem) + id / kXcds;
    kvh = lid / n_tiles;
    tile = lid - kvh * n_tiles;
  }
  // request of this tile: tiles of QT rows are numbered request by request
  int r = 0, t0 = 0;
  for (; r + 1 < p.n_req; ++r) {
    const int nt = (p.r[r].nrows + QT - 1) / QT;
    if (tile < t0 + nt) break;
    t0 += nt;
  }
  const ReqPlan& rq = p.r[r];
  const int lrow0 = (tile - t0) * QT;
  const int nvalid = min(QT, rq.nrows - lrow0);
  const int L = rq.seq_len;
  const bf16* kb = kc + ((long)(rq.slot * hkv + kvh) * s_max) * DH;
  const bf16* vb = vc + ((long)(rq.slot * hkv + kvh) * DH) * s_max;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int qg = wave % QG;                       // 16-row group
  const int h = kvh * GH + wave / QG;             // query head
  const int qr = qg * 16 + (lane & 15);           // query row of this lane in the tile
  const bool q_ok = qr < nvalid;
  const long qrow = rq.row0 + lrow0 + qr;
  const int g = lane >> 4;

  // this wave's load instructions: j = wave + NW m over the tile's NI
  // instructions (the first NKI fill K, the rest V^T); per instruction the
  // lane's source at key 0 of the slot and the LDS byte offset in the stage
  const bf16* src[IPW];
  int dst[IPW];
#pragma unroll
  for (int m = 0; m < IPW; ++m) {
    const int j = wave + NW * m;
    if (j < NKI) {
      const int rho = KRPI * j + lane / KCPR;
      const int c = (lane % KCPR) ^ (rho & 7);
      const int key = (rho & ~31) | (((rho >> 2) & 3) << 3) | (((rho >> 4) & 1) << 2) | (rho & 3);
      src[m] = kb + (long)key * DH + c * 8;
      dst[m] = j * 1024;
    } else {
      const int jv = min(j, NI - 1) - NKI;
      const int d = 8 * jv + lane / 8;
      const int c = (lane % 8) ^ (d & 7);
      src[m] = vb + (long)d * s_max + c * 8;
      dst[m] = KBYTES + jv * 1024;
    }
  }
  auto issue = [&](int stage, int key0) {
    char* base = smem + stage * STAGE;
#pragma unroll
    for (int m = 0; m < IPW; ++m) {
      const int j = wave + NW * m;
      if (j < NI)
        load_lds16(src[m] + (j < NKI ? (long)key0 * DH : (long)key0), base + dst[m]);
    }
  };

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
  float m_ref = -INFINITY, l_run = 0.f;
  const int sw = (lane & 7) << 4;                 // chunk-slot XOR of rows 16 b + (lane & 15)

  const int ntiles = ceil_div(L, SK);
  issue(0, 0);
  for (int t = 0; t < ntiles; ++t) {
    const int key0 = t * SK;
    wait_vmcnt<0>();
    __syncthreads();                              // tile t in LDS; stage (t + 1) & 1 free
    const char* kst = smem + (t & 1) * STAGE;
    const char* vst = kst + KBYTES;
    const bool tail = key0 + SK > L;
    if (tail) {                                   // clear V^T at keys >= L
      const int kl = L - key0;
      for (int idx = tid; idx < DH * 8; idx += NT) {
        const int d = idx >> 3, c = idx & 7;
        if (8 * c + 8 > kl) {
          u32x4* ptr = reinterpret_cast<u32x4*>(const_cast<char*>(vst) + d * 128 + ((c ^ (d & 7)) << 4));
          u32x4 v = *ptr;
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const uint32_t keep = (8 * c + 2 * w < kl ? 0x0000ffffu : 0u) |
                                  (8 * c + 2 * w + 1 < kl ? 0xffff0000u : 0u);
            v[w] &= keep;
          }
          *ptr = v;
        }
      }
      __syncthreads();
    }
    if (t + 1 < ntiles) issue((t + 1) & 1, key0 + SK);

    // S^T blocks: sblk[kb][i] = raw score(key = key0 + pi(16 kb + 4 g + i), query = lane & 15)
    f32x4 sblk[4];
#pragma unroll
    for (int kbk = 0; kbk < 4; ++kbk) {
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
      const char* krow = kst + (kbk * 16 + (lane & 15)) * KRB;
#pragma unroll
      for (int s = 0; s < NKS; ++s) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(krow + (((s * 4 + g) << 4) ^ sw));
        acc = mfma16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, qf[s]), acc);
      }
      sblk[kbk] = acc;
    }
    if (tail) {
#pragma unroll
      for (int kbk = 0; kbk < 4; ++kbk)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (key0 + 32 * (kbk >> 1) + 8 * g + 4 * (kbk & 1) + i >= L) sblk[kbk][i] = -INFINITY;
    }
    float mt = -INFINITY;
#pragma unroll
    for (int kbk = 0; kbk < 4; ++kbk)
#pragma unroll
      for (int i = 0; i < 4; ++i) mt = fmaxf(mt, sblk[kbk][i]);
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    // move the reference maximum only on a large increase
    const bool grow = (mt - m_ref) * scale_log2 > 8.0f;
    if (__builtin_amdgcn_ballot_w64(grow)) {
      const float alpha = grow ? __builtin_amdgcn_exp2f((m_ref - mt) * scale_log2) : 1.0f;
      if (grow) m_ref = mt;
      l_run *= alpha;
#pragma unroll
      for (int i = 0; i < NDB; ++i) o[i] *= alpha;
    }
    const float nm = m_ref == -INFINITY ? 0.0f : -m_ref * scale_log2;
    float lsum = 0.f;
#pragma unroll
    for (int kbk = 0; kbk < 4; ++kbk)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float e = __builtin_amdgcn_exp2f(fmaf(sblk[kbk][i], scale_log2, nm));
        sblk[kbk][i] = e;
        lsum += e;
      }
    l_run += lsum;

    // O^T += V^T P^T over two 32-key steps; B operand slot 8 g + e <-> key
    // 32 j + 8 g + e, which lane group g holds as sblk[2 j + e / 4][e % 4]
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      bf16x8 ph, pl;
      split_p8(sblk[2 * j], sblk[2 * j + 1], ph, pl);
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(vst + (db * 16 + (lane & 15)) * 128 +
                                                        (((4 * j + g) << 4) ^ sw));
        o[db] = mfma16_bf16(__builtin_bit_cast(bf16x8, a), ph, o[db]);
        o[db] = mfma16_bf16(__builtin_bit_cast(bf16x8, a), pl, o[db]);
      }
    }
  }

  // finish: l over the 4 lanes sharing the query, normalise, store
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_run;
  if (q_ok) {
    bf16* dstp = out + qrow * hq * DH + h * DH;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      bf16x4 v;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = (bf16)(o[db][i] * inv);
      *reinterpret_cast<bf16x4*>(dstp + db * 16 + 4 * g) = v;
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

template <int DH, int QG, int KG>
static hipError_t launch_attn(const StepPlan& p, const bf16* q, const bf16* kc, const bf16* vc,
                              int s_max, int hq, int hkv, bf16* out, float scale_log2,
                              hipStream_t st) {
  constexpr int QT = 16 * QG;
  int tiles = 0;
  for (int r = 0; r < p.n_req; ++r) tiles += (p.r[r].nrows + QT - 1) / QT;
  if (tiles == 0) return hipSuccess;
  DLM_LAUNCH((attn_bf16_kernel<DH, QG, KG>), dim3(hq, tiles), dim3(QG * KG * 64), 0, st,
                     p, q, kc, vc, s_max, hq, hkv, out, scale_log2);
  return hipGetLastError();
}

template <int DH, int GH, int QG>
static hipError_t launch_gqa(const StepPlan& p, const bf16* q, const bf16* kc, const bf16* vc,
                             int s_max, int hq, int hkv, bf16* out, float scale_log2,
                             hipStream_t st) {
  constexpr int QT = 16 * QG;
  int tiles = 0;
  for (int r = 0; r < p.n_req; ++r) tiles += (p.r[r].nrows + QT - 1) / QT;
  if (tiles == 0) return hipSuccess;
  DLM_LAUNCH((attn_gqa_kernel<DH, GH, QG>), dim3(hkv * tiles), dim3(GH * QG * 64), 0,
                     st, p, q, kc, vc, s_max, hq, hkv, tiles, out, scale_log2);
  return hipGetLastError();
}

// Grouped-query attention with 2, 4, 7 or 8 query heads per key/value head:
// the shared-tile kernel with 7 or 8 waves per block.
template <int DH>
static hipError_t attention_dh(const StepPlan& p, const bf16* q, const bf16* kc, const bf16* vc,
                               int s_max, int hq, int hkv, bf16* out, float scale_log2,
                               hipStream_t st) {
  switch (hkv > 0 && hq % hkv == 0 ? hq / hkv : 0) {
    case 2: return launch_gqa<DH, 2, 4>(p, q, kc, vc, s_max, hq, hkv, out, scale_log2, st);
    case 4: return launch_gqa<DH, 4, 2>(p, q, kc, vc, s_max, hq, hkv, out, scale_log2, st);
    case 7: return launch_gqa<DH, 7, 1>(p, q, kc, vc, s_max, hq, hkv, out, scale_log2, st);
    case 8: return launch_gqa<DH, 8, 1>(p, q, kc, vc, s_max, hq, hkv, out, scale_log2, st);
    default: break;
  }
  // MHA and other ratios. With at least two 64-row blocks per CU (256 CUs)
  // the shared-tile kernel with one head per block (4 waves) is used: its
  // blocks overlap each other's loads. Otherwise the per-head kernel with
  // two key groups per block (8 waves), on query tiles of 32 rows when no
  // request recomputes more than 32 rows (cache steps of blocks <= 32), else
  // 64.
  int max_rows = 0, tiles64 = 0;
  for (int r = 0; r < p.n_req; ++r) {
    max_rows = max(max_rows, p.r[r].nrows);
    tiles64 += (p.r[r].nrows + 63) / 64;
  }
  if (hq == hkv && max_rows > 32 && (long)hq * tiles64 >= 512)
    return launch_gqa<DH, 1, 4>(p, q, kc, vc, s_max, hq, hkv, out, scale_log2, st);
  return max_rows <= 32
             ? launch_attn<DH, 2, 2>(p, q, kc, vc, s_max, hq, hkv, out, scale_log2, st)
             : launch_attn<DH, 4, 2>(p, q, kc, vc, s_max, hq, hkv, out, scale_log2, st);
}

template <>
hipError_t attention<bf16>(const StepPlan& p, const bf16* q, const bf16* kc, const bf16* vc,
                           int s_max, int hq, int hkv, int dh, bf16* out, hipStream_t st) {
  if (p.n_rows == 0) return hipSuccess;
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)dh);
  if (dh == 128) return attention_dh<128>(p, q, kc, vc, s_max, hq, hkv, out, scale_log2, st);
  if (dh == 64) return attention_dh<64>(p, q, kc, vc, s_max, hq, hkv, out, scale_log2, st);
  return hipErrorInvalidValue;
}

template <>
hipError_t attention<float>(const StepPlan& p, const float* q, const float* kc, const float* vc,
                            int s_max, int hq, int hkv, int dh, float* out, hipStream_t st) {
  if (p.n_tiles == 0) return hipSuccess;
  const float scale = 1.0f / sqrtf((float)dh);
  dim3 g(p.n_tiles, hq);
  if (dh == 64)
    DLM_LAUNCH(attn_f32_kernel<64>, g, dim3(64), 0, st, p, q, kc, vc, s_max, hq, hkv,
                       out, scale);
  else if (dh == 128)
    DLM_LAUNCH(attn_f32_kernel<128>, g, dim3(64), 0, st, p, q, kc, vc, s_max, hq, hkv,
                       out, scale);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace dlm
