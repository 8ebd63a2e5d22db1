// Launch functions of the denoising-step kernels (internal to libdlm.so).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dlm {

constexpr int kMaxReq = 64;
constexpr int kMaxBlock = 64;
constexpr int kNStats = 8;      // confidence statistics per request
constexpr int kQTile = 64;      // query rows per attention block / rows per RoPE tile

// Per-request plan of one step, passed by value as a kernel argument.
struct ReqPlan {
  int row0;      // first packed recompute row
  int nrows;     // recompute rows
  int pos0;      // position of the first recompute row
  int seq_len;   // keys attended (all positions of the slot)
  int prompt_len;
  int slot;
  int tok_off;   // offset of position 0 in tokens/mask
  int blk_s;     // active block [blk_s, blk_s + blk_len)
  int blk_len;
  int tile0;     // first 64-row tile of this request (attention / RoPE grids)
  int blk0;      // offset of this request's block rows in the packed block-row order
  float gamma;   // threshold
};
struct StepPlan {
  int n_req;
  int n_rows;    // total recompute rows N
  int n_tiles;   // total 64-row tiles
  int n_blk;     // total block rows
  ReqPlan r[kMaxReq];
};

// Row -> request lookup (requests are few; plan rows are ascending).
__device__ __forceinline__ int plan_req_of_row(const StepPlan& p, int row) {
  int r = 0;
  while (r + 1 < p.n_req && p.r[r + 1].row0 <= row) ++r;
  return r;
}
__device__ __forceinline__ int plan_req_of_tile(const StepPlan& p, int tile) {
  int r = 0;
  while (r + 1 < p.n_req && p.r[r + 1].tile0 <= tile) ++r;
  return r;
}

// ---- GEMM family (gemm.hip, gemm_dl.hip) ----
// cfg >= 0: a direct-load tile configuration (bf16); cfg < 0: register-staged
// kernel. splits: number of K slices (fp32 partial slices, summed by the consumer).
// group_m: tile order (0 = plain); sub, n_tail: the last n_tail tiles of the
// order are each run as `sub` (2 or 4) sub-tiles (0: none); active_cus > 0
// (LM head over several row tiles only): one launch of blocks on that many
// CUs that walk the tiles of the rows needing a prediction (see
// gemm_dl_head_launch) instead of one block per tile
struct GemmPlan { int cfg; int splits; int group_m; int sub = 0; int n_tail = 0; int active_cus = 0; };
// allow_mf32: configurations with 32x32x16 MFMA tiles may be chosen (their
// epilogues exist for the plain, residual-add and SwiGLU stores; SwiGLU needs
// d_ffn % 32 == 0)
// direct-load bf16 kernel: one launch of configuration cfg; its output tile,
// MFMA shape and the sub-tile splits it allows (bit 1: halves, bit 2: quarters)
template <class Epi>
hipError_t gemm_dl_launch(int cfg, const bf16* A, int lda, const bf16* B, int ldb, int M, int N,
                          int K, int splits, int group_m, int sub, int n_tail, const Epi& epi,
                          hipStream_t st);
struct EpiLMHead;
// LM head whose row count is known only on the device (epi.m_count): as many
// blocks as fit on num_cu CUs, each XCD's blocks walking the tiles of its
// contiguous range of column tiles whose rows lie below the count
hipError_t gemm_dl_head_launch(int cfg, const bf16* A, int lda, const bf16* B, int ldb, int M,
                               int N, int K, int num_cu, const EpiLMHead& epi, hipStream_t st);
int gemm_dl_tile(int cfg, int* bm, int* bn, int* threads);
int gemm_dl_mfma(int cfg);
int gemm_dl_subs(int cfg);
int gemm_dl_odd(int cfg);
// one launch of configuration cfg with epilogue 0 (fp32 store of `splits` K
// slices), 1 (SwiGLU to bf16, N = 2 F) or 2 (fp32 add), A [M, K], B [N, K],
// C row-major (test hook)
hipError_t gemm_debug_launch(int cfg, int epilogue, int sub, int n_tail, int group_m,
                             int splits, const bf16* A, const bf16* B, void* C, int M, int N,
                             int K, hipStream_t st);
// allow_tail: the last round may be split into sub-tiles (epilogues that allow it)
// allow_odd: configurations whose wave tiles hold an odd number of column
// fragments may be chosen (every epilogue but SwiGLU)
GemmPlan gemm_plan(int elem_bytes, int M, int N, int K, bool splittable, int num_cu,
                   bool allow_mf32 = true, bool allow_tail = true, bool allow_odd = true);
// plan of the LM-head GEMM (M rows x V vocab entries)
GemmPlan lm_head_plan(int elem_bytes, int M, int V, int K, int num_cu);
template <typename T>
hipError_t gemm_store_f32(const GemmPlan& p, const T* A, int lda, const T* B, int ldb, int M,
                          int N, int K, float* C, int ldc, hipStream_t st);
template <typename T>
hipError_t gemm_add_f32(const GemmPlan& p, const T* A, int lda, const T* B, int ldb, int M, int N,
                        int K, float* C, int ldc, hipStream_t st);
template <typename T>
hipError_t gemm_scaled_f32(const GemmPlan& p, const T* A, int lda, const T* B, int ldb, int M,
                           int N, int K, float scale, float* C, int ldc, hipStream_t st);
template <typename T>
hipError_t gemm_swiglu(const GemmPlan& p, const T* A, int lda, const T* W, int ldw, int M, int F,
                       int K, T* out, int ldo, hipStream_t st);
int lm_head_tiles(const GemmPlan& p, int V);
template <typename T>
hipError_t gemm_lm_head(const GemmPlan& p, const T* U, int ldu, const T* W, int M, int V, int K,
                        float inv_tau, float* pm, float* ps, int* pi, int ld,
                        const int* m_count, hipStream_t st);

// ---- per-row kernels (rowwise.hip) ----
template <typename T>
hipError_t embed_rows(const StepPlan& p, const T* E, int d, int vocab, int mask_id,
                      const int32_t* tokens, const uint8_t* mask, float* h, hipStream_t st);
template <typename T>
hipError_t rmsnorm_rows(const float* h, const float* g, int n, int d, float eps, T* out,
                        hipStream_t st);
// h[n] += sum of split-K slices (part may be null), then out = rmsnorm(h) (out may be null)
template <typename T>
hipError_t add_rmsnorm_rows(float* h, const float* part, int splits, long stride, const float* g,
                            int n, int d, float eps, T* out, hipStream_t st);
hipError_t rope_table(const StepPlan& p, int head_dim, float theta, float2* cs, hipStream_t st);
template <typename T>
hipError_t qkv_rope_scatter(const StepPlan& p, const float* qkv, int splits, long split_stride,
                            const float2* cs, int hq, int hkv, int dh, T* q_out,
                            T* kcache, T* vcache, int s_max, hipStream_t st);
hipError_t lm_select_rows(const StepPlan& p, const uint8_t* mask, int all_rows, int* lm_rows,
                          int* lm_count, int* req_lm_off, int* req_lm_cnt, hipStream_t st);
template <typename T>
hipError_t final_norm_gather(const float* h, const float* g, const int* lm_rows,
                             const int* lm_count, int m_max, int d, float eps, T* u,
                             hipStream_t st);
hipError_t lm_combine(const float* pm, const float* ps, const int* pi, int tiles, int ld,
                      const int* lm_count, int m_max, float* conf, int* tok, hipStream_t st);
hipError_t unmask_select(const StepPlan& p, const float* conf, const int* tok,
                         const int* req_lm_off, int32_t* tokens, uint8_t* mask,
                         int32_t* n_unmasked, int32_t* out_pos, int32_t* out_tok,
                         float* out_conf, float* blk_conf, int32_t* blk_tok, float* tok_conf,
                         float* stats, hipStream_t st);

// ---- attention (attention.hip) ----
template <typename T>
hipError_t attention(const StepPlan& p, const T* q, const T* kcache, const T* vcache,
                     int s_max, int hq, int hkv, int dh, T* out, hipStream_t st);

}  // namespace dlm
