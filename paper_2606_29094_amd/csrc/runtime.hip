// Host runtime behind include/dlm.h: argument validation, the per-step row
// plan, KV-slot bookkeeping, workspace layout and the kernel sequence of one
// denoising step. Device memory is always the caller's.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdint>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "../../include/dlm.h"
#include "common.h"
#include "kernels.h"

using namespace dlm;

namespace dlm {
thread_local LaunchTiming g_launch_timing;
}

namespace {

thread_local std::string g_err;

dlm_status fail(dlm_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

#define HIPCHECK(expr)                                                               \
  do {                                                                               \
    hipError_t e_ = (expr);                                                          \
    if (e_ != hipSuccess)                                                            \
      return fail(DLM_EHIP, "%s failed: %s", #expr, hipGetErrorString(e_));          \
  } while (0)

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace

// Scratch of dlm_denoise_step_noalloc: one copy per device, in the library's
// code object. Host code never uses this name as an address: the device
// address of each GPU's copy comes from hipGetSymbolAddress (scratch_address).
static __device__ __align__(256) char scratch[DLM_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch, looked up once per device.
dlm_status scratch_address(void** out) {
  int dev = 0;
  HIPCHECK(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(DLM_EUNSUPPORTED, "device %d outside [0, %d)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HIPCHECK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p || reinterpret_cast<uintptr_t>(p) % 256 != 0)
      return fail(DLM_EHIP, "scratch of device %d is not 256-byte aligned", dev);
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return DLM_OK;
}

}  // namespace

// Enqueue one kernel class (`expr`, a launch returning hipError_t); when the
// model's profiler times this launch, its kernel
// carries a pair of events in its own dispatch (DLM_LAUNCH), so the measured
// time is the kernel's and the stream gets no extra commands. (A class that
// enqueues no kernel this time returns the events unused.)
#define LAUNCH(model, stream, name, expr)                                           \
  do {                                                                            \
    Profiler& pf_ = (model)->prof;                                                \
    hipEvent_t a_ = nullptr, b_ = nullptr;                                        \
    if (pf_.wants(name)) {                                                        \
      a_ = pf_.take();                                                            \
      b_ = pf_.take();                                                            \
      if (a_ && b_) g_launch_timing = LaunchTiming{a_, b_};                       \
    }                                                                             \
    const hipError_t le_ = (expr);                                                \
    const bool used_ = a_ && b_ && !g_launch_timing.start;                        \
    g_launch_timing = LaunchTiming{};                                             \
    if (used_) {                                                                  \
      pf_.pending.push_back({pf_.kind_of(name), a_, b_});                         \
    } else {                                                                      \
      if (a_) pf_.pool.push_back(a_);                                             \
      if (b_) pf_.pool.push_back(b_);                                             \
    }                                                                             \
    if (le_ != hipSuccess)                                                        \
      return fail(DLM_EHIP, "%s failed: %s", #expr, hipGetErrorString(le_));      \
  } while (0)

// Per-kernel-class event timing (dlm_profile_*).
struct Profiler {
  bool on = false;
  std::string only;        // empty: every class
  int every = 1;           // time one launch in `every` of each class
  std::vector<long> seen;  // launches of each class since enable / sample (sampling phase)
  std::vector<int> since_read;   // launches of each class since the last read
  bool wants(const char* n) {
    if (!on || !(only.empty() || only == n)) return false;
    const int k = kind_of(n);
    if ((int)seen.size() <= k) seen.resize(k + 1, 0);
    if ((int)since_read.size() <= k) since_read.resize(k + 1, 0);
    since_read[k] += 1;
    return seen[k]++ % every == 0;
  }
  struct Rec { int kind; hipEvent_t a, b; };
  std::vector<Rec> pending;
  std::vector<hipEvent_t> pool;
  std::vector<std::string> names;
  int kind_of(const char* n) {
    for (size_t i = 0; i < names.size(); ++i)
      if (names[i] == n) return (int)i;
    names.emplace_back(n);
    return (int)names.size() - 1;
  }
  hipEvent_t take() {
    if (pool.empty()) {
      hipEvent_t e;
      if (hipEventCreate(&e) != hipSuccess) return nullptr;
      return e;
    }
    hipEvent_t e = pool.back();
    pool.pop_back();
    return e;
  }
  ~Profiler() {
    for (auto& r : pending) { (void)hipEventDestroy(r.a); (void)hipEventDestroy(r.b); }
    for (auto e : pool) (void)hipEventDestroy(e);
  }
};

struct dlm_model {
  Profiler prof;
  dlm_config cfg;
  const void* embed;
  const void* lm_head;
  const float* final_norm;
  std::vector<dlm_layer_weights> layers;
  int num_cu;
  size_t es;   // element size
};

struct SlotState {
  bool valid = false;
  int block_start = -1;
  int seq_len = -1;
};

struct dlm_cache {
  const dlm_model* model;
  int n_slots;
  int s_max;          // positions per slot (multiple of 64)
  char* base;
  size_t region;      // bytes of one layer's K (or V) region
  std::vector<SlotState> slots;
  void* k_layer(int l) const { return base + (size_t)(2 * l) * region; }
  void* v_layer(int l) const { return base + (size_t)(2 * l + 1) * region; }
};

namespace {

// Workspace layout of a step with n recomputed rows and n_req requests.
struct Layout {
  size_t h, a, qkv, cs, q, ao, part, act, lm_rows, lm_count, req_off, req_cnt, u, pm, ps, pi,
      conf, tok, total;
  GemmPlan g_qkv, g_o, g_gu, g_down, g_lm, g_logits;
  int s_qkv, s_o, s_down, tiles, m_max;
};

Layout layout(const dlm_model* m, int n, int n_req) {
  const dlm_config& c = m->cfg;
  Layout L{};
  const int qkv_dim = (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  const int qd = c.n_q_heads * c.head_dim;
  const int es_i = (int)m->es;
  L.g_qkv = gemm_plan(es_i, n, qkv_dim, c.d_model, true, m->num_cu);
  L.g_o = gemm_plan(es_i, n, c.d_model, qd, true, m->num_cu);
  // the SwiGLU GEMM keeps 16x16 tiles: its 32x32 variants measured 5-6 %
  // slower on every gate/up shape
  L.g_gu = gemm_plan(es_i, n, 2 * c.d_ffn, c.d_model, false, m->num_cu, false, true, false);
  L.g_down = gemm_plan(es_i, n, c.d_model, c.d_ffn, true, m->num_cu);
  L.m_max = std::min(n, n_req * kMaxBlock);
  L.g_lm = lm_head_plan(es_i, L.m_max, c.vocab, c.d_model, m->num_cu);
  L.g_logits = L.g_lm;
  L.s_qkv = L.g_qkv.splits;
  L.s_o = L.g_o.splits;
  L.s_down = L.g_down.splits;
  L.tiles = lm_head_tiles(L.g_lm, c.vocab);
  const size_t es = m->es;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  L.h = take((size_t)n * c.d_model * 4);
  L.a = take((size_t)n * c.d_model * es);
  L.qkv = take((size_t)L.s_qkv * n * qkv_dim * 4);
  L.cs = take((size_t)n * (c.head_dim / 2) * 8);
  L.q = take((size_t)n * qd * es);
  L.ao = take((size_t)n * qd * es);
  L.part = take((size_t)std::max(L.s_o, L.s_down) * n * c.d_model * 4);
  L.act = take((size_t)n * c.d_ffn * es);
  L.lm_rows = take((size_t)std::max(L.m_max, 1) * 4);
  L.lm_count = take(4);
  L.req_off = take((size_t)kMaxReq * 4);
  L.req_cnt = take((size_t)kMaxReq * 4);
  L.u = take((size_t)std::max(L.m_max, 1) * c.d_model * es);
  L.pm = take((size_t)L.tiles * std::max(L.m_max, 1) * 4);
  L.ps = take((size_t)L.tiles * std::max(L.m_max, 1) * 4);
  L.pi = take((size_t)L.tiles * std::max(L.m_max, 1) * 4);
  L.conf = take((size_t)std::max(L.m_max, 1) * 4);
  L.tok = take((size_t)std::max(L.m_max, 1) * 4);
  L.total = off;
  return L;
}

dlm_status check_config(const dlm_config* c) {
  if (!c) return fail(DLM_EINVAL, "config is NULL");
  if (c->dtype != DLM_F32 && c->dtype != DLM_BF16)
    return fail(DLM_EINVAL, "dtype %d is not DLM_F32 or DLM_BF16", c->dtype);
  if (c->n_layers < 1 || c->d_model < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1 ||
      c->head_dim < 1 || c->d_ffn < 1 || c->vocab < 2)
    return fail(DLM_EINVAL, "non-positive model dimension");
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(DLM_EUNSUPPORTED, "head_dim %d (supported: 64, 128)", c->head_dim);
  if (c->n_q_heads % c->n_kv_heads != 0)
    return fail(DLM_EINVAL, "n_q_heads %d is not a multiple of n_kv_heads %d", c->n_q_heads,
                c->n_kv_heads);
  if (c->d_model % 64 != 0)
    return fail(DLM_EUNSUPPORTED, "d_model %d is not a multiple of 64", c->d_model);
  if (c->d_ffn % 16 != 0)
    return fail(DLM_EUNSUPPORTED, "d_ffn %d is not a multiple of 16", c->d_ffn);
  if (c->mask_id < 0 || c->mask_id >= c->vocab)
    return fail(DLM_EINVAL, "mask_id %d outside [0, vocab)", c->mask_id);
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f) || !std::isfinite(c->inv_tau) ||
      !(c->inv_tau > 0.f))
    return fail(DLM_EINVAL, "rms_eps, rope_theta or inv_tau out of range");
  return DLM_OK;
}

// Row plan of one step; returns the error status (nothing enqueued yet).
dlm_status make_plan(const dlm_model* m, const dlm_cache* c, const dlm_batch* b,
                     const float* thr, bool force_refresh, StepPlan* p) {
  if (!b) return fail(DLM_EINVAL, "batch is NULL");
  if (b->n_req < 1 || b->n_req > kMaxReq)
    return fail(DLM_EINVAL, "n_req %d outside [1, %d]", b->n_req, kMaxReq);
  if (!b->reqs || !b->tokens || !b->mask) return fail(DLM_EINVAL, "batch pointer is NULL");
  if (b->mode < DLM_CACHE_NONE || b->mode > DLM_CACHE_DUAL)
    return fail(DLM_EINVAL, "cache mode %d", b->mode);
  std::vector<char> used(c->n_slots, 0);
  int row = 0, tile = 0, blk = 0;
  p->n_req = b->n_req;
  for (int r = 0; r < b->n_req; ++r) {
    const dlm_req& q = b->reqs[r];
    if (q.slot < 0 || q.slot >= c->n_slots)
      return fail(DLM_EINVAL, "request %d: slot %d outside [0, %d)", r, q.slot, c->n_slots);
    if (used[q.slot]) return fail(DLM_EINVAL, "request %d: slot %d used twice", r, q.slot);
    used[q.slot] = 1;
    if (q.seq_len < 1 || q.seq_len > c->s_max)
      return fail(DLM_ESIZE, "request %d: seq_len %d outside [1, %d]", r, q.seq_len, c->s_max);
    if (q.prompt_len < 0 || q.prompt_len > q.block_start)
      return fail(DLM_EINVAL, "request %d: prompt_len %d vs block_start %d", r, q.prompt_len,
                  q.block_start);
    if (q.block_len < 1 || q.block_len > kMaxBlock || q.block_start + q.block_len > q.seq_len)
      return fail(DLM_EINVAL, "request %d: block [%d, %d) invalid for seq_len %d", r,
                  q.block_start, q.block_start + q.block_len, q.seq_len);
    if (q.tok_offset < 0) return fail(DLM_EINVAL, "request %d: negative tok_offset", r);
    if (q.flags & ~DLM_REQ_REFRESH) return fail(DLM_EINVAL, "request %d: unknown flags", r);
    float g = 0.f;
    if (thr) {
      g = thr[r];
      if (!(g >= 0.f && g <= 1.f))
        return fail(DLM_EINVAL, "request %d: threshold outside [0, 1]", r);
    }
    const bool refresh = force_refresh || b->mode == DLM_CACHE_NONE || (q.flags & DLM_REQ_REFRESH);
    int r0, r1;
    if (refresh) {
      r0 = 0; r1 = q.seq_len;
    } else {
      const SlotState& s = c->slots[q.slot];
      if (!s.valid || s.block_start != q.block_start || s.seq_len != q.seq_len)
        return fail(DLM_ESTATE,
                    "request %d: cache step on slot %d whose cache is not current (refreshed at "
                    "block %d, seq_len %d; step at block %d, seq_len %d)",
                    r, q.slot, s.valid ? s.block_start : -1, s.valid ? s.seq_len : -1,
                    q.block_start, q.seq_len);
      r0 = q.block_start;
      r1 = b->mode == DLM_CACHE_DUAL ? q.block_start + q.block_len : q.seq_len;
    }
    ReqPlan& rp = p->r[r];
    rp.row0 = row;
    rp.nrows = r1 - r0;
    rp.pos0 = r0;
    rp.seq_len = q.seq_len;
    rp.prompt_len = q.prompt_len;
    rp.slot = q.slot;
    rp.tok_off = q.tok_offset;
    rp.blk_s = q.block_start;
    rp.blk_len = q.block_len;
    rp.tile0 = tile;
    rp.blk0 = blk;
    rp.gamma = g;
    row += rp.nrows;
    tile += ceil_div(rp.nrows, kQTile);
    blk += q.block_len;
  }
  // the requests' packed token ranges must be disjoint (each step updates its
  // request's tokens and mask in place)
  std::vector<std::pair<long, long>> ranges(b->n_req);
  for (int r = 0; r < b->n_req; ++r)
    ranges[r] = {(long)b->reqs[r].tok_offset, (long)b->reqs[r].tok_offset + b->reqs[r].seq_len};
  std::sort(ranges.begin(), ranges.end());
  for (int r = 1; r < b->n_req; ++r)
    if (ranges[r].first < ranges[r - 1].second)
      return fail(DLM_EINVAL, "token ranges [%ld, %ld) and [%ld, %ld) overlap", ranges[r - 1].first,
                  ranges[r - 1].second, ranges[r].first, ranges[r].second);
  if (ranges.back().second > INT32_MAX)
    return fail(DLM_EINVAL, "token range end %ld exceeds the int32 index range", ranges.back().second);
  p->n_rows = row;
  p->n_tiles = tile;
  p->n_blk = blk;
  (void)m;
  return DLM_OK;
}

dlm_status check_ws(const dlm_model* m, const StepPlan& p, void* ws, size_t ws_bytes,
                    Layout* L) {
  *L = layout(m, p.n_rows, p.n_req);
  if (!ws) return fail(DLM_EINVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % 256 != 0)
    return fail(DLM_EINVAL, "workspace is not 256-byte aligned");
  if (ws_bytes < L->total)
    return fail(DLM_ESIZE, "workspace of %zu bytes; this step needs %zu (%d rows)", ws_bytes,
                L->total, p.n_rows);
  return DLM_OK;
}

enum class Tail { Unmask, Logits, None };

// Device-to-device copy of a recorded intermediate (dlm_debug_trace); a NULL
// destination records nothing.
#define TRACE_COPY(dst, src, bytes)                                                    \
  do {                                                                                 \
    if (dst) HIPCHECK(hipMemcpyAsync((dst), (src), (bytes), hipMemcpyDeviceToDevice, st)); \
  } while (0)

template <typename T>
dlm_status run_forward(dlm_model* m, dlm_cache* c, const dlm_batch* b, const StepPlan& p,
                       const Layout& L, char* ws, const dlm_trace* tr, hipStream_t st) {
  const dlm_config& cf = m->cfg;
  const int d = cf.d_model, hq = cf.n_q_heads, hkv = cf.n_kv_heads, dh = cf.head_dim;
  const int qkv_dim = (hq + 2 * hkv) * dh, qd = hq * dh, n = p.n_rows;
  float* h = reinterpret_cast<float*>(ws + L.h);
  T* a = reinterpret_cast<T*>(ws + L.a);
  float* qkv = reinterpret_cast<float*>(ws + L.qkv);
  float2* cs = reinterpret_cast<float2*>(ws + L.cs);
  T* q = reinterpret_cast<T*>(ws + L.q);
  T* ao = reinterpret_cast<T*>(ws + L.ao);
  float* part = reinterpret_cast<float*>(ws + L.part);
  T* act = reinterpret_cast<T*>(ws + L.act);

  LAUNCH(m, st, "rope_table", rope_table(p, dh, cf.rope_theta, cs, st));
  LAUNCH(m, st, "embed", embed_rows<T>(p, reinterpret_cast<const T*>(m->embed), d, cf.vocab, cf.mask_id,
                         b->tokens, b->mask, h, st));
  LAUNCH(m, st, "rmsnorm", rmsnorm_rows<T>(h, m->layers[0].attn_norm, n, d, cf.rms_eps, a, st));
  const size_t es = sizeof(T);
  for (int l = 0; l < cf.n_layers; ++l) {
    const dlm_layer_weights& w = m->layers[l];
    T* kc = reinterpret_cast<T*>(c->k_layer(l));
    T* vc = reinterpret_cast<T*>(c->v_layer(l));
    const dlm_trace* t = tr && tr->layer == l ? tr : nullptr;
    if (t) {
      TRACE_COPY(t->h_in, h, (size_t)n * d * 4);
      TRACE_COPY(t->a_attn, a, (size_t)n * d * es);
    }
    LAUNCH(m, st, "gemm_qkv", gemm_store_f32<T>(L.g_qkv, a, d, reinterpret_cast<const T*>(w.w_qkv), d, n,
                                                      qkv_dim, d, qkv, qkv_dim, st));
    if (t) TRACE_COPY(t->qkv, qkv, (size_t)L.s_qkv * n * qkv_dim * 4);
    LAUNCH(m, st, "rope_kv_write", qkv_rope_scatter<T>(p, qkv, L.s_qkv, (long)n * qkv_dim, cs, hq, hkv, dh, q, kc, vc,
                                 c->s_max, st));
    if (t) TRACE_COPY(t->q, q, (size_t)n * qd * es);
    LAUNCH(m, st, "attention", attention<T>(p, q, kc, vc, c->s_max, hq, hkv, dh, ao, st));
    if (t) TRACE_COPY(t->attn_out, ao, (size_t)n * qd * es);
    // O projection; its residual update is fused into the FFN norm when K is split
    if (L.s_o == 1) {
      LAUNCH(m, st, "gemm_o", gemm_add_f32<T>(L.g_o, ao, qd, reinterpret_cast<const T*>(w.w_o), qd, n, d,
                                                  qd, h, d, st));
      LAUNCH(m, st, "rmsnorm", rmsnorm_rows<T>(h, w.ffn_norm, n, d, cf.rms_eps, a, st));
    } else {
      LAUNCH(m, st, "gemm_o", gemm_store_f32<T>(L.g_o, ao, qd, reinterpret_cast<const T*>(w.w_o), qd, n, d,
                                                    qd, part, d, st));
      LAUNCH(m, st, "residual_rmsnorm", add_rmsnorm_rows<T>(h, part, L.s_o, (long)n * d, w.ffn_norm, n, d,
                                                                cf.rms_eps, a, st));
    }
    if (t) {
      TRACE_COPY(t->h_mid, h, (size_t)n * d * 4);
      TRACE_COPY(t->a_ffn, a, (size_t)n * d * es);
    }
    LAUNCH(m, st, "gemm_gate_up_swiglu", gemm_swiglu<T>(L.g_gu, a, d, reinterpret_cast<const T*>(w.w_gate_up), d, n, cf.d_ffn, d, act,
                            cf.d_ffn, st));
    if (t) TRACE_COPY(t->act, act, (size_t)n * cf.d_ffn * es);
    // down projection; its residual update is fused into the next layer's norm
    const float* next_norm = l + 1 < cf.n_layers ? m->layers[l + 1].attn_norm : nullptr;
    T* next_a = l + 1 < cf.n_layers ? a : nullptr;
    if (L.s_down == 1) {
      LAUNCH(m, st, "gemm_down", gemm_add_f32<T>(L.g_down, act, cf.d_ffn, reinterpret_cast<const T*>(w.w_down), cf.d_ffn, n, d,
                               cf.d_ffn, h, d, st));
      if (next_a) LAUNCH(m, st, "rmsnorm", rmsnorm_rows<T>(h, next_norm, n, d, cf.rms_eps, a, st));
    } else {
      LAUNCH(m, st, "gemm_down", gemm_store_f32<T>(L.g_down, act, cf.d_ffn, reinterpret_cast<const T*>(w.w_down),
                                                       cf.d_ffn, n, d, cf.d_ffn, part, d, st));
      LAUNCH(m, st, "residual_rmsnorm", add_rmsnorm_rows<T>(h, part, L.s_down, (long)n * d, next_norm, n, d,
                                                                cf.rms_eps, next_a, st));
    }
    if (t) TRACE_COPY(t->h_out, h, (size_t)n * d * 4);
  }
  return DLM_OK;
}

template <typename T>
dlm_status run_step(dlm_model* m, dlm_cache* c, const dlm_batch* b, const StepPlan& p,
                    const Layout& L, char* ws, Tail tail, const dlm_step_out* out,
                    float* logits, const dlm_trace* tr, hipStream_t st) {
  dlm_status s = run_forward<T>(m, c, b, p, L, ws, tr, st);
  if (s != DLM_OK || tail == Tail::None) return s;
  const dlm_config& cf = m->cfg;
  const int d = cf.d_model;
  float* h = reinterpret_cast<float*>(ws + L.h);
  int* lm_rows = reinterpret_cast<int*>(ws + L.lm_rows);
  int* lm_count = reinterpret_cast<int*>(ws + L.lm_count);
  int* req_off = reinterpret_cast<int*>(ws + L.req_off);
  int* req_cnt = reinterpret_cast<int*>(ws + L.req_cnt);
  T* u = reinterpret_cast<T*>(ws + L.u);
  const int m_max = p.n_blk;
  LAUNCH(m, st, "lm_select", lm_select_rows(p, b->mask, tail == Tail::Logits ? 1 : 0, lm_rows, lm_count, req_off,
                          req_cnt, st));
  LAUNCH(m, st, "final_norm", final_norm_gather<T>(h, m->final_norm, lm_rows, lm_count, m_max, d, cf.rms_eps, u, st));
  if (tr && tail == Tail::Logits) TRACE_COPY(tr->u, u, (size_t)m_max * d * sizeof(T));
  if (tail == Tail::Logits) {
    LAUNCH(m, st, "gemm_logits", gemm_scaled_f32<T>(L.g_logits, u, d, reinterpret_cast<const T*>(m->lm_head), d, m_max, cf.vocab,
                                d, cf.inv_tau, logits, cf.vocab, st));
    return DLM_OK;
  }
  float* pm = reinterpret_cast<float*>(ws + L.pm);
  float* ps = reinterpret_cast<float*>(ws + L.ps);
  int* pi = reinterpret_cast<int*>(ws + L.pi);
  float* conf = reinterpret_cast<float*>(ws + L.conf);
  int* tok = reinterpret_cast<int*>(ws + L.tok);
  LAUNCH(m, st, "lm_head", gemm_lm_head<T>(L.g_lm, u, d, reinterpret_cast<const T*>(m->lm_head), m_max, cf.vocab, d,
                           cf.inv_tau, pm, ps, pi, L.m_max, lm_count, st));
  LAUNCH(m, st, "lm_combine", lm_combine(pm, ps, pi, L.tiles, L.m_max, lm_count, m_max, conf, tok, st));
  LAUNCH(m, st, "unmask", unmask_select(p, conf, tok, req_off, b->tokens, b->mask, out->n_unmasked, out->pos,
                         out->tok, out->conf, out->block_conf, out->block_tok, b->tok_conf,
                         out->stats, st));
  return DLM_OK;
}

void mark_refreshed(dlm_cache* c, const dlm_batch* b, bool force_refresh) {
  for (int r = 0; r < b->n_req; ++r) {
    const dlm_req& q = b->reqs[r];
    if (force_refresh || b->mode == DLM_CACHE_NONE || (q.flags & DLM_REQ_REFRESH)) {
      SlotState& s = c->slots[q.slot];
      s.valid = true;
      s.block_start = q.block_start;
      s.seq_len = q.seq_len;
    }
  }
}

dlm_status dispatch(dlm_model* m, dlm_cache* c, const dlm_batch* b, const StepPlan& p,
                    const Layout& L, void* ws, Tail tail, const dlm_step_out* out,
                    float* logits, void* stream, const dlm_trace* tr = nullptr) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  char* w = reinterpret_cast<char*>(ws);
  if (m->cfg.dtype == DLM_BF16) return run_step<bf16>(m, c, b, p, L, w, tail, out, logits, tr, st);
  return run_step<float>(m, c, b, p, L, w, tail, out, logits, tr, st);
}

dlm_status check_handles(dlm_model* m, dlm_cache* c) {
  if (!m) return fail(DLM_EINVAL, "model is NULL");
  if (!c) return fail(DLM_EINVAL, "cache is NULL");
  if (c->model != m) return fail(DLM_EINVAL, "cache was allocated for another model");
  return DLM_OK;
}

__global__ void fill_i32_kernel(int* p, int v) { *p = v; }

}  // namespace

extern "C" {

const char* dlm_last_error(void) { return g_err.c_str(); }

dlm_status dlm_load_weights(const dlm_config* cfg, const dlm_weights* w, dlm_model** out) {
  g_err.clear();
  if (!out) return fail(DLM_EINVAL, "out is NULL");
  *out = nullptr;
  dlm_status s = check_config(cfg);
  if (s != DLM_OK) return s;
  if (!w || !w->embed || !w->lm_head || !w->final_norm || !w->layers)
    return fail(DLM_EINVAL, "weights pointer is NULL");
  for (int l = 0; l < cfg->n_layers; ++l) {
    const dlm_layer_weights& lw = w->layers[l];
    if (!lw.attn_norm || !lw.w_qkv || !lw.w_o || !lw.ffn_norm || !lw.w_gate_up || !lw.w_down)
      return fail(DLM_EINVAL, "layer %d: weight pointer is NULL", l);
  }
  dlm_model* m = new dlm_model();
  m->cfg = *cfg;
  m->embed = w->embed;
  m->lm_head = w->lm_head;
  m->final_norm = w->final_norm;
  m->layers.assign(w->layers, w->layers + cfg->n_layers);
  m->es = cfg->dtype == DLM_BF16 ? 2 : 4;
  int dev = 0, cu = 0;
  if (hipGetDevice(&dev) == hipSuccess &&
      hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cu > 0)
    m->num_cu = cu;
  else
    m->num_cu = 256;
  (void)hipGetLastError();
  *out = m;
  return DLM_OK;
}

void dlm_model_destroy(dlm_model* m) { delete m; }

dlm_status dlm_profile_enable(dlm_model* m, int32_t on, const char* only_class) {
  g_err.clear();
  if (!m) return fail(DLM_EINVAL, "model is NULL");
  m->prof.on = on != 0;
  m->prof.only = only_class ? only_class : "";
  m->prof.seen.clear();
  return DLM_OK;
}

dlm_status dlm_profile_sample(dlm_model* m, int32_t every) {
  g_err.clear();
  if (!m) return fail(DLM_EINVAL, "model is NULL");
  if (every < 1) return fail(DLM_EINVAL, "every %d < 1", every);
  m->prof.every = every;
  m->prof.seen.clear();
  return DLM_OK;
}

dlm_status dlm_profile_read(dlm_model* m, dlm_profile_entry* out, int32_t cap, int32_t* n_out) {
  g_err.clear();
  if (!m || !n_out || cap < 0 || (cap > 0 && !out)) return fail(DLM_EINVAL, "NULL argument or cap < 0");
  Profiler& pf = m->prof;
  std::vector<int> calls(pf.names.size(), 0);
  std::vector<double> ms(pf.names.size(), 0.0);
  dlm_status st = DLM_OK;
  for (auto& r : pf.pending) {
    float t = 0.f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&t, r.a, r.b);
    if (e != hipSuccess && st == DLM_OK)
      st = fail(DLM_EHIP, "profile event: %s", hipGetErrorString(e));
    calls[r.kind] += 1;
    ms[r.kind] += t;
    pf.pool.push_back(r.a);
    pf.pool.push_back(r.b);
  }
  pf.pending.clear();
  int n = 0;
  for (size_t k = 0; k < pf.names.size(); ++k) {
    const int launches = k < pf.since_read.size() ? pf.since_read[k] : 0;
    if (calls[k] == 0 && launches == 0) continue;
    if (n < cap) {
      snprintf(out[n].name, sizeof out[n].name, "%s", pf.names[k].c_str());
      out[n].calls = calls[k];
      out[n].total_ms = ms[k];
      out[n].launches = launches;
    }
    ++n;
  }
  pf.since_read.assign(pf.since_read.size(), 0);
  *n_out = n < cap ? n : cap;
  return st;
}

dlm_status dlm_workspace_bytes(const dlm_model* m, int32_t max_rows, int32_t max_reqs,
                               size_t* out_bytes) {
  g_err.clear();
  if (!m || !out_bytes) return fail(DLM_EINVAL, "NULL argument");
  if (max_rows < 1 || max_reqs < 1 || max_reqs > kMaxReq)
    return fail(DLM_EINVAL, "max_rows %d / max_reqs %d out of range", max_rows, max_reqs);
  // the planner's split-K factors (and with them the slice buffers) depend on
  // the row count and are not monotonic in it: take the largest layout over
  // every row count up to max_rows
  size_t best = 0;
  for (int n = 1; n <= max_rows; ++n) best = std::max(best, layout(m, n, max_reqs).total);
  *out_bytes = best;
  return DLM_OK;
}

dlm_status dlm_kv_cache_alloc(const dlm_model* m, int32_t n_slots, int32_t max_seq_len,
                              void* dev_buf, size_t buf_bytes, size_t* required_bytes,
                              dlm_cache** out) {
  g_err.clear();
  if (!m) return fail(DLM_EINVAL, "model is NULL");
  if (n_slots < 1) return fail(DLM_EINVAL, "n_slots %d < 1", n_slots);
  if (max_seq_len < 1 || max_seq_len > DLM_MAX_SEQ)
    return fail(DLM_ESIZE, "max_seq_len %d outside [1, %d]", max_seq_len, DLM_MAX_SEQ);
  const dlm_config& c = m->cfg;
  const int s_max = (int)align_up(max_seq_len, 64);
  const size_t region = (size_t)n_slots * c.n_kv_heads * s_max * c.head_dim * m->es;
  const size_t need = region * 2 * c.n_layers;
  if (required_bytes) *required_bytes = need;
  if (!dev_buf) {
    if (out) *out = nullptr;
    return DLM_OK;
  }
  if (!out) return fail(DLM_EINVAL, "out is NULL");
  *out = nullptr;
  if (buf_bytes < need) return fail(DLM_ESIZE, "cache buffer %zu bytes < %zu", buf_bytes, need);
  if (reinterpret_cast<uintptr_t>(dev_buf) % 256 != 0)
    return fail(DLM_EINVAL, "cache buffer is not 256-byte aligned");
  dlm_cache* k = new dlm_cache();
  k->model = m;
  k->n_slots = n_slots;
  k->s_max = s_max;
  k->base = reinterpret_cast<char*>(dev_buf);
  k->region = region;
  k->slots.assign(n_slots, SlotState{});
  *out = k;
  return DLM_OK;
}

void dlm_cache_destroy(dlm_cache* c) { delete c; }

dlm_status dlm_cache_invalidate(dlm_cache* c, int32_t slot) {
  g_err.clear();
  if (!c) return fail(DLM_EINVAL, "cache is NULL");
  if (slot < 0 || slot >= c->n_slots) return fail(DLM_EINVAL, "slot %d out of range", slot);
  c->slots[slot] = SlotState{};
  return DLM_OK;
}

dlm_status dlm_denoise_step(dlm_model* m, dlm_cache* c, const dlm_batch* b,
                            const float* thresholds, const dlm_step_out* out, void* workspace,
                            size_t ws_bytes, void* stream) {
  g_err.clear();
  dlm_status s = check_handles(m, c);
  if (s != DLM_OK) return s;
  if (!thresholds) return fail(DLM_EINVAL, "thresholds is NULL");
  if (!out || !out->n_unmasked || !out->pos || !out->tok || !out->conf)
    return fail(DLM_EINVAL, "step output pointer is NULL");
  if (out->stats && (!b || !b->tok_conf))
    return fail(DLM_EINVAL, "confidence statistics need batch.tok_conf");
  StepPlan p;
  s = make_plan(m, c, b, thresholds, false, &p);
  if (s != DLM_OK) return s;
  Layout L;
  s = check_ws(m, p, workspace, ws_bytes, &L);
  if (s != DLM_OK) return s;
  s = dispatch(m, c, b, p, L, workspace, Tail::Unmask, out, nullptr, stream);
  if (s == DLM_OK) mark_refreshed(c, b, false);
  return s;
}

dlm_status dlm_denoise_step_noalloc(dlm_model* m, dlm_cache* c, const dlm_batch* b,
                                    const float* thresholds, const dlm_step_out* out,
                                    void* stream) {
  g_err.clear();
  dlm_status s = check_handles(m, c);
  if (s != DLM_OK) return s;
  if (!thresholds) return fail(DLM_EINVAL, "thresholds is NULL");
  if (!out || !out->n_unmasked || !out->pos || !out->tok || !out->conf)
    return fail(DLM_EINVAL, "step output pointer is NULL");
  if (out->stats && (!b || !b->tok_conf))
    return fail(DLM_EINVAL, "confidence statistics need batch.tok_conf");
  StepPlan p;
  s = make_plan(m, c, b, thresholds, false, &p);
  if (s != DLM_OK) return s;
  const size_t need = layout(m, p.n_rows, p.n_req).total;
  if (need > (size_t)DLM_SCRATCH_BYTES)
    return fail(DLM_ESIZE, "this step needs %zu bytes of scratch (%d rows); the fixed scratch "
                "holds %zu", need, p.n_rows, (size_t)DLM_SCRATCH_BYTES);
  void* ws = nullptr;
  s = scratch_address(&ws);
  if (s != DLM_OK) return s;
  Layout L;
  s = check_ws(m, p, ws, (size_t)DLM_SCRATCH_BYTES, &L);
  if (s != DLM_OK) return s;
  // no kernel timing here (its events would be created on first use)
  const bool prof_on = m->prof.on;
  m->prof.on = false;
  s = dispatch(m, c, b, p, L, ws, Tail::Unmask, out, nullptr, stream);
  m->prof.on = prof_on;
  if (s == DLM_OK) mark_refreshed(c, b, false);
  return s;
}

dlm_status dlm_cache_refresh(dlm_model* m, dlm_cache* c, const dlm_batch* b, void* workspace,
                             size_t ws_bytes, void* stream) {
  g_err.clear();
  dlm_status s = check_handles(m, c);
  if (s != DLM_OK) return s;
  StepPlan p;
  s = make_plan(m, c, b, nullptr, true, &p);
  if (s != DLM_OK) return s;
  Layout L;
  s = check_ws(m, p, workspace, ws_bytes, &L);
  if (s != DLM_OK) return s;
  s = dispatch(m, c, b, p, L, workspace, Tail::None, nullptr, nullptr, stream);
  if (s == DLM_OK) mark_refreshed(c, b, true);
  return s;
}

dlm_status dlm_debug_logits(dlm_model* m, dlm_cache* c, const dlm_batch* b, float* logits_out,
                            void* workspace, size_t ws_bytes, void* stream) {
  g_err.clear();
  dlm_status s = check_handles(m, c);
  if (s != DLM_OK) return s;
  if (!logits_out) return fail(DLM_EINVAL, "logits_out is NULL");
  StepPlan p;
  s = make_plan(m, c, b, nullptr, false, &p);
  if (s != DLM_OK) return s;
  Layout L;
  s = check_ws(m, p, workspace, ws_bytes, &L);
  if (s != DLM_OK) return s;
  s = dispatch(m, c, b, p, L, workspace, Tail::Logits, nullptr, logits_out, stream);
  if (s == DLM_OK) mark_refreshed(c, b, false);
  return s;
}

dlm_status dlm_debug_trace(dlm_model* m, dlm_cache* c, const dlm_batch* b, dlm_trace* tr,
                           void* workspace, size_t ws_bytes, void* stream) {
  g_err.clear();
  dlm_status s = check_handles(m, c);
  if (s != DLM_OK) return s;
  if (!tr) return fail(DLM_EINVAL, "trace is NULL");
  if (tr->layer < 0 || tr->layer >= m->cfg.n_layers)
    return fail(DLM_EINVAL, "trace layer %d outside [0, %d)", tr->layer, m->cfg.n_layers);
  if (tr->u && !tr->logits) return fail(DLM_EINVAL, "trace.u needs trace.logits");
  StepPlan p;
  s = make_plan(m, c, b, nullptr, false, &p);
  if (s != DLM_OK) return s;
  Layout L;
  s = check_ws(m, p, workspace, ws_bytes, &L);
  if (s != DLM_OK) return s;
  if (tr->qkv && tr->qkv_cap < L.s_qkv)
    return fail(DLM_ESIZE, "trace.qkv holds %d K-split slices; this step writes %d", tr->qkv_cap,
                L.s_qkv);
  tr->qkv_splits = L.s_qkv;
  s = dispatch(m, c, b, p, L, workspace, tr->logits ? Tail::Logits : Tail::None, nullptr,
               tr->logits, stream, tr);
  if (s == DLM_OK) mark_refreshed(c, b, false);
  return s;
}

dlm_status dlm_head_confidence(dlm_model* m, const void* u_rows, int32_t m_rows, float* conf,
                               int32_t* tok, void* workspace, size_t ws_bytes, void* stream) {
  g_err.clear();
  if (!m) return fail(DLM_EINVAL, "model is NULL");
  if (!u_rows || !conf || !tok) return fail(DLM_EINVAL, "NULL buffer");
  if (m_rows < 1) return fail(DLM_EINVAL, "m_rows %d < 1", m_rows);
  if (!workspace) return fail(DLM_EINVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
    return fail(DLM_EINVAL, "workspace is not 256-byte aligned");
  const GemmPlan gp = lm_head_plan((int)m->es, m_rows, m->cfg.vocab, m->cfg.d_model, m->num_cu);
  const int tiles = lm_head_tiles(gp, m->cfg.vocab);
  const size_t stat = align_up((size_t)tiles * m_rows * 4, 256);
  const size_t need = 3 * stat + 256;
  if (ws_bytes < need) return fail(DLM_ESIZE, "workspace of %zu bytes; needs %zu", ws_bytes, need);
  char* w = reinterpret_cast<char*>(workspace);
  float* pm = reinterpret_cast<float*>(w);
  float* ps = reinterpret_cast<float*>(w + stat);
  int* pi = reinterpret_cast<int*>(w + 2 * stat);
  int* cnt = reinterpret_cast<int*>(w + 3 * stat);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(1), 0, st, cnt, (int)m_rows);
  HIPCHECK(hipGetLastError());
  const dlm_config& cf = m->cfg;
  if (cf.dtype == DLM_BF16) {
    HIPCHECK(gemm_lm_head<bf16>(gp, reinterpret_cast<const bf16*>(u_rows), cf.d_model,
                                reinterpret_cast<const bf16*>(m->lm_head), m_rows, cf.vocab,
                                cf.d_model, cf.inv_tau, pm, ps, pi, m_rows, cnt, st));
  } else {
    HIPCHECK(gemm_lm_head<float>(gp, reinterpret_cast<const float*>(u_rows), cf.d_model,
                                 reinterpret_cast<const float*>(m->lm_head), m_rows, cf.vocab,
                                 cf.d_model, cf.inv_tau, pm, ps, pi, m_rows, cnt, st));
  }
  HIPCHECK(lm_combine(pm, ps, pi, tiles, m_rows, cnt, m_rows, conf, tok, st));
  return DLM_OK;
}

dlm_status dlm_debug_gemm_info(int32_t cfg, int32_t* bm, int32_t* bn, int32_t* subs) {
  g_err.clear();
  int tm = 0, tn = 0, th = 0;
  if (!gemm_dl_tile(cfg, &tm, &tn, &th)) return fail(DLM_EINVAL, "no GEMM configuration %d", cfg);
  if (bm) *bm = tm;
  if (bn) *bn = tn;
  if (subs) *subs = gemm_dl_subs(cfg) | (gemm_dl_odd(cfg) ? 8 : 0);
  return DLM_OK;
}

dlm_status dlm_debug_gemm(int32_t cfg, int32_t epilogue, int32_t sub, int32_t n_tail,
                          int32_t group_m, int32_t splits, const void* a, const void* b, void* c,
                          int32_t M, int32_t N, int32_t K, void* stream) {
  g_err.clear();
  if (!a || !b || !c) return fail(DLM_EINVAL, "NULL buffer");
  if (M < 1 || N < 1 || K < 1 || K % 64 != 0)
    return fail(DLM_EINVAL, "sizes M %d N %d K %d (K a positive multiple of 64)", M, N, K);
  if (epilogue < 0 || epilogue > 2) return fail(DLM_EINVAL, "epilogue %d", epilogue);
  if (epilogue == 1 && N % 2 != 0) return fail(DLM_EINVAL, "odd N %d for the SwiGLU epilogue", N);
  if (group_m < 0 || n_tail < 0) return fail(DLM_EINVAL, "negative group_m or n_tail");
  if (splits < 1 || (splits > 1 && epilogue != 0) || (K / 64) % splits != 0)
    return fail(DLM_EINVAL, "splits %d (K slices of the plain store only, dividing the %d k-tiles)",
                splits, K / 64);
  int tm = 0, tn = 0, th = 0;
  if (!gemm_dl_tile(cfg, &tm, &tn, &th)) return fail(DLM_EINVAL, "no GEMM configuration %d", cfg);
  // the gate/up interleave pairs columns in groups of the MFMA tile width
  const int pair = gemm_dl_mfma(cfg) == 32 ? 32 : 16;
  if (epilogue == 1 && (N / 2) % pair != 0)
    return fail(DLM_EINVAL, "SwiGLU width %d is not a multiple of %d", N / 2, pair);
  if (epilogue == 1 && gemm_dl_odd(cfg))
    return fail(DLM_EINVAL, "configuration %d has no SwiGLU epilogue (odd fragment count)", cfg);
  if (sub != 0 && ((sub != 2 && sub != 4) || !(gemm_dl_subs(cfg) & sub)))
    return fail(DLM_EINVAL, "configuration %d has no %d-way sub-tiles", cfg, sub);
  if (sub != 0 && (long)n_tail > (long)ceil_div(M, tm) * ceil_div(N, tn) * splits)
    return fail(DLM_EINVAL, "n_tail %d beyond the tile count", n_tail);
  const hipError_t e = gemm_debug_launch(cfg, epilogue, sub, n_tail, group_m, splits,
                                         reinterpret_cast<const bf16*>(a),
                                         reinterpret_cast<const bf16*>(b), c, M, N, K,
                                         reinterpret_cast<hipStream_t>(stream));
  if (e == hipErrorInvalidValue)
    return fail(DLM_EINVAL, "GEMM configuration %d rejects this launch", cfg);
  if (e != hipSuccess) return fail(DLM_EHIP, "GEMM launch: %s", hipGetErrorString(e));
  return DLM_OK;
}

}  // extern "C"
