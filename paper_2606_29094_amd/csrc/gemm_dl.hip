// bf16 NT GEMM with direct global->LDS loads (gfx950 global_load_lds_dwordx4).
//
// Each k-tile is 64 bf16 (128 bytes) of BM rows of A and BN rows of B. A wave
// instruction moves 8 rows (1 KB): lane l writes LDS bytes [16 l, 16 l + 16)
// of that kilobyte, and it fetches the global 16-byte chunk that belongs
// there under an XOR swizzle (LDS chunk slot = global chunk ^ swz(row)), so
// that the lanes that later read consecutive rows of one chunk hit distinct
// banks. The weight operand B goes SB-1 k-tiles ahead through a ring of SB LDS
// stages and the activation operand A one k-tile ahead through two (A is
// re-read by every column tile and mostly served from cache; B streams from
// HBM and needs the deeper prefetch); no registers hold tiles in flight.
// Waves multiply with v_mfma_f32_16x16x32_bf16 (MF = 16) or
// v_mfma_f32_32x32x16_bf16 (MF = 32); the 16x16 epilogues are the same as the
// register-staged kernel's, the 32x32 ones (plain, residual-add and SwiGLU
// stores) follow the 32x32 accumulator layout.
#include <type_traits>

#include "common.h"
#include "gemm_common.h"
#include "kernels.h"

namespace dlm {

// One BM x BN output tile at rows m0.., columns n0.., K range [kbeg, kend),
// with the block's LDS at smem. tn and tz (column tile, K slice) are passed
// to the K order and the epilogue. (Two-ring form; the split-phase form of
// the eight-wave tiles follows.)
template <int BM, int BN, int WAVES_M, int WAVES_N, int SA, int SB, int RB, int MF, class Epi>
__device__ __forceinline__ void dl_tile(char* smem, const bf16* __restrict__ A, int lda,
                                        const bf16* __restrict__ B, int ldb, int M, int N,
                                        int m0, int n0, int tn, int tz, int kbeg, int kend,
                                        const Epi& epi) {
  static_assert(RB == 64 || RB == 128, "k-tile row bytes");
  static_assert(SA >= 2 && SA <= 3 && SB >= SA && SB <= 4, "A and B stages");
  static_assert(MF == 16 || MF == 32, "MFMA tile");
  constexpr int DA = SA - 1, DB = SB - 1;  // prefetch distances (k-tiles ahead)
  constexpr int NW = WAVES_M * WAVES_N;
  constexpr int TM = BM / WAVES_M, TN = BN / WAVES_N;
  constexpr int FM = TM / MF, FN = TN / MF;
  static_assert(FM * MF == TM && FN * MF == TN, "wave tile");
  constexpr int BK = RB / 2;              // bf16 per row per k-tile
  constexpr int CPR = RB / 16;            // 16-byte chunks per row
  constexpr int RPI = 1024 / RB;          // rows per 1 KB wave instruction
  constexpr int KG = RB / 64;             // 32-wide k groups per k-tile
  constexpr int STAGE_A = BM * RB, STAGE_B = BN * RB;
  // 1 KB instructions per stage, and per wave: an equal share when the count
  // divides by the waves (wave w takes a contiguous run), else wave w takes
  // instructions w, w + NW, ... (the first NI % NW waves one more than the rest)
  constexpr int NI_A = BM / RPI, NI_B = BN / RPI;
  static_assert(NI_A * RPI == BM && NI_B * RPI == BN, "rows per instruction");
  constexpr bool EVEN_A = NI_A % NW == 0, EVEN_B = NI_B % NW == 0;
  constexpr int PERW_A = (NI_A + NW - 1) / NW, PERW_B = (NI_B + NW - 1) / NW;
  constexpr int MINW_A = NI_A / NW, MINW_B = NI_B / NW;
  // loads of a wave that may stay in flight at the top of an iteration: those
  // issued after A(kt) in the steady issue order (see the pipeline below),
  // counted for the waves with the fewest (a wave with more then waits for
  // one or two of the next k-tile's loads too, which is safe)
  constexpr int INFLIGHT = DB > DA ? DA * MINW_B + (DA - 1) * MINW_A : (DA - 1) * (MINW_A + MINW_B);
  static_assert(INFLIGHT < 64, "vmcnt range");
  char* const smem_b = smem + SA * STAGE_A;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const int nkt = kend > kbeg ? (kend - kbeg) / BK : 0;
  // K order: epilogues that ask for it (the LM head, which streams a large
  // weight matrix with a 2^n-byte row pitch) start each column tile's K walk
  // at a different k-tile (column tile mod k-tiles), so that the blocks in
  // flight read different column offsets of their weight rows at any moment
  // and spread over the HBM channels (MHA vocab head with 32 rows: 4.5 -> 5.9
  // TB/s); the others walk K from the start.
  const int krot = Epi::kRotateK && nkt > 0 ? tn % nkt : 0;
  auto ktile = [&](int kt) { const int k = kt + krot; return k >= nkt ? k - nkt : k; };

  // LDS chunk slot of global chunk c in row r: c ^ swz(r). With 16x16x32
  // fragments (16 consecutive rows of one chunk per 16 lanes) 8 consecutive
  // rows map to distinct banks (two per 128-byte bank line for 64-byte rows);
  // with 32x32x16 fragments (32 consecutive rows of one chunk per 32 lanes)
  // the slot follows row / 2, which keeps those reads free of bank conflicts
  // (row & 7 gives ~4 conflict cycles per read, measured with
  // SQ_LDS_BANK_CONFLICT). Both are invariant under row offsets that are
  // multiples of the fragment height.
  auto swz = [](int r) {
    return CPR == 8 ? (MF == 32 ? ((r >> 1) & 7) : (r & 7)) : ((r >> 1) & 3);
  };
  // source of this lane for each of its wave's instructions (fixed over k),
  // as 32-bit element offsets from the matrix base (operands hold fewer than
  // 2^31 elements; half the registers of 64-bit pointers)
  // stage instruction of this wave's j-th load, and whether the wave has one
  auto inst_a = [&](int j) { return EVEN_A ? wave * PERW_A + j : wave + j * NW; };
  auto inst_b = [&](int j) { return EVEN_B ? wave * PERW_B + j : wave + j * NW; };
  auto has_a = [&](int j) { return j < MINW_A || inst_a(j) < NI_A; };
  auto has_b = [&](int j) { return j < MINW_B || inst_b(j) < NI_B; };
  uint32_t srcA[PERW_A];
  uint32_t srcB[PERW_B];
#pragma unroll
  for (int j = 0; j < PERW_A; ++j) {
    const int row = RPI * inst_a(j) + lane / CPR;
    const int cc = (lane % CPR) ^ swz(row);
    srcA[j] = (uint32_t)min(m0 + row, M - 1) * (uint32_t)lda + kbeg + cc * 8;
  }
#pragma unroll
  for (int j = 0; j < PERW_B; ++j) {
    const int row = RPI * inst_b(j) + lane / CPR;
    const int cc = (lane % CPR) ^ swz(row);
    srcB[j] = (uint32_t)epi.b_row(min(n0 + row, N - 1)) * (uint32_t)ldb + kbeg + cc * 8;
  }
  auto issue_a = [&](int stage, int kt) {
    char* dst = smem + stage * STAGE_A;
    const bf16* base = A + kt * BK;
#pragma unroll
    for (int j = 0; j < PERW_A; ++j)
      if (has_a(j))
        __builtin_amdgcn_global_load_lds((gptr_t)(base + srcA[j]),
                                         (lptr_t)(dst + inst_a(j) * 1024), 16, 0, 0);
  };
  auto issue_b = [&](int stage, int kt) {
    char* dst = smem_b + stage * STAGE_B;
    const bf16* base = B + kt * BK;
#pragma unroll
    for (int j = 0; j < PERW_B; ++j)
      if (has_b(j))
        __builtin_amdgcn_global_load_lds((gptr_t)(base + srcB[j]),
                                         (lptr_t)(dst + inst_b(j) * 1024), 16, 0, 0);
  };

  // accumulators: 16x16 tiles (4 values per lane) or 32x32 tiles (16 per lane)
  typedef typename std::conditional<MF == 32, f32x16, f32x4>::type Acc;
  Acc acc[FM][FN];
#pragma unroll
  for (int a = 0; a < FM; ++a)
#pragma unroll
    for (int b = 0; b < FN; ++b) acc[a][b] = Acc{};

  // fragment offsets. 16x16x32: row R = base + (lane & 15) with base a
  // multiple of 16, chunk c = 4 g + lane / 16 (g: 32-wide k group), stored at
  // slot c ^ swz(R) = c ^ swz(lane & 15). 32x32x16: row R = base + (lane & 31)
  // with base a multiple of 32, chunk c = 2 s + lane / 32 (s: 16-wide k step),
  // slot c ^ swz(lane & 31).
  constexpr int LR = MF == 32 ? 31 : 15;
  constexpr int NCO = MF == 32 ? RB / 32 : KG;
  const int a_row = (wm * TM + (lane & LR)) * RB;
  const int b_row = (wn * TN + (lane & LR)) * RB;
  int co[NCO];
#pragma unroll
  for (int g = 0; g < NCO; ++g)
    co[g] = (MF == 32 ? ((2 * g + (lane >> 5)) ^ swz(lane & 31))
                      : ((g * 4 + (lane >> 4)) ^ swz(lane & 15))) << 4;

  // 32x32x16 tiles: per 16-wide k step, FM A and FN B fragments (one 16-byte
  // LDS read each) feed FM x FN MFMAs; the next step's fragments are read
  // while the current step's MFMAs run (two register buffers)
  auto compute32 = [&](int sa, int sb) {
    if constexpr (MF == 32) {
      const char* pa = smem + sa * STAGE_A + a_row;
      const char* pb = smem_b + sb * STAGE_B + b_row;
      constexpr int KS = RB / 32;
      u32x4 af[2][FM], bq[2][FN];
      auto rd = [&](int buf, int st) {
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
          af[buf][fm] = *reinterpret_cast<const u32x4*>(pa + fm * 32 * RB + co[st]);
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
          bq[buf][fn] = *reinterpret_cast<const u32x4*>(pb + fn * 32 * RB + co[st]);
      };
      // two fragment buffers unless the accumulators leave too few registers
      // for them (then each step reads, then multiplies)
      constexpr bool kTwoBuf = FM * FN * 16 + 8 * (FM + FN) <= 224;
      if constexpr (!kTwoBuf) {
#pragma unroll
        for (int st = 0; st < KS; ++st) {
          rd(0, st);
#pragma unroll
          for (int fm = 0; fm < FM; ++fm)
#pragma unroll
            for (int fn = 0; fn < FN; ++fn)
              acc[fm][fn] = mfma32_bf16(__builtin_bit_cast(bf16x8, af[0][fm]),
                                        __builtin_bit_cast(bf16x8, bq[0][fn]), acc[fm][fn]);
        }
        return;
      }
      rd(0, 0);
#pragma unroll
      for (int st = 0; st < KS; ++st) {
        if (st + 1 < KS) rd((st + 1) & 1, st + 1);
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
          for (int fn = 0; fn < FN; ++fn)
            acc[fm][fn] = mfma32_bf16(__builtin_bit_cast(bf16x8, af[st & 1][fm]),
                                      __builtin_bit_cast(bf16x8, bq[st & 1][fn]), acc[fm][fn]);
      }
      // schedule (mask 0x100: LDS reads, 0x008: MFMA): the first step's reads,
      // then each step's MFMAs with the next step's reads spread among them
      // (left to itself the compiler reuses one fragment register and waits
      // on every read)
      constexpr int NR = FM + FN, NM = FM * FN;
      __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);
#pragma unroll
      for (int st = 0; st < KS; ++st) {
        if (st + 1 < KS) {
#pragma unroll
          for (int i = 0; i < NR; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, NM / NR, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          __builtin_amdgcn_sched_group_barrier(0x008, NM - (NM / NR) * NR, 0);
        } else {
          __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
        }
      }
    }
  };

  auto compute = [&](int sa, int sb) {
    const char* pa = smem + sa * STAGE_A;
    const char* pb = smem_b + sb * STAGE_B;
    if constexpr (MF == 32) {
      (void)pa; (void)pb;
    } else if constexpr (KG == 2) {
      // Both k groups' fragments, then the MFMAs of group 0 with the reads of
      // group 1 spread among them, then the MFMAs of group 1: the LDS latency
      // of group 1 hides behind group 0's MFMAs (left to itself the compiler
      // issues each read right before its first use and waits on it).
      u32x4 af0[FM], bf0[FN], af1[FM], bf1[FN];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
        af0[fm] = *reinterpret_cast<const u32x4*>(pa + a_row + fm * 16 * RB + co[0]);
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        bf0[fn] = *reinterpret_cast<const u32x4*>(pb + b_row + fn * 16 * RB + co[0]);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
        af1[fm] = *reinterpret_cast<const u32x4*>(pa + a_row + fm * 16 * RB + co[1]);
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        bf1[fn] = *reinterpret_cast<const u32x4*>(pb + b_row + fn * 16 * RB + co[1]);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
          acc[fm][fn] = mfma16_bf16(__builtin_bit_cast(bf16x8, af0[fm]),
                                    __builtin_bit_cast(bf16x8, bf0[fn]), acc[fm][fn]);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
          acc[fm][fn] = mfma16_bf16(__builtin_bit_cast(bf16x8, af1[fm]),
                                    __builtin_bit_cast(bf16x8, bf1[fn]), acc[fm][fn]);
      // scheduling groups (mask 0x100: LDS reads, 0x008: MFMA)
      constexpr int NR = FM + FN, NM = FM * FN;
      __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);
#pragma unroll
      for (int i = 0; i < NR; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, NM / NR, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, NM - (NM / NR) * NR, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
    } else {
#pragma unroll
      for (int g = 0; g < KG; ++g) {
        u32x4 af[FM], bfr[FN];
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
          af[fm] = *reinterpret_cast<const u32x4*>(pa + a_row + fm * 16 * RB + co[g]);
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
          bfr[fn] = *reinterpret_cast<const u32x4*>(pb + b_row + fn * 16 * RB + co[g]);
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
          for (int fn = 0; fn < FN; ++fn)
            acc[fm][fn] = mfma16_bf16(__builtin_bit_cast(bf16x8, af[fm]),
                                      __builtin_bit_cast(bf16x8, bfr[fn]), acc[fm][fn]);
      }
    }
  };

  // Pipeline: activations (A, mostly cache-resident) run DA = SA - 1 k-tiles
  // ahead through an SA-stage ring, weights (B, streamed from HBM) DB = SB - 1
  // ahead through an SB-stage ring. Iteration j issues A(j + DA) then
  // B(j + DB); the prologue issues the same sequence for j = -DB .. -1. vmcnt
  // counts a wave's loads in issue order, so at the top of iteration kt the
  // loads that may stay in flight while A(kt) and B(kt) must have landed are
  // exactly those issued after A(kt): INFLIGHT of them (everything issued
  // before A(kt) has landed by then, which is why a deeper B ring needs A
  // issued further ahead as well). Near the end, where fewer loads were
  // issued, the wait drains everything.
#pragma unroll
  for (int j = -DB; j < 0; ++j) {
    if (j + DA >= 0 && j + DA < nkt) issue_a((j + DA) % SA, ktile(j + DA));
    if (j + DB < nkt) issue_b((j + DB) % SB, ktile(j + DB));
  }

  for (int kt = 0; kt < nkt; ++kt) {
    if (INFLIGHT > 0 && kt + DB - 1 < nkt) wait_vmcnt<INFLIGHT>(); else wait_vmcnt<0>();
    // Every wave has its own loads of tile kt in LDS and has finished reading
    // the stages about to be refilled (read at kt - 1). A bare s_barrier:
    // __syncthreads() would add a fence that drains every load in flight.
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    if (kt + DA < nkt) issue_a((kt + DA) % SA, ktile(kt + DA));
    if (kt + DB < nkt) issue_b((kt + DB) % SB, ktile(kt + DB));
    if constexpr (MF == 32) compute32(kt % SA, kt % SB);
    else compute(kt % SA, kt % SB);
  }
  __syncthreads();
  if constexpr (MF == 32)
    epi.op32(acc, m0 + wm * TM, n0 + wn * TN, lane, tz);
  else
    epi(acc, m0 + wm * TM, n0 + wn * TN, lane, wn, smem, WAVES_N, BM, m0, tn, tz);
}

// wait until at most N vector-memory operations and no LDS operation of this
// wave are in flight (gfx9 s_waitcnt: vmcnt in [3:0] and [15:14], lgkmcnt 0,
// expcnt (7) not waited on)
template <int N>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

// Scheduling groups of a pipelined phase (masks 0x008: MFMA, 0x020: global
// loads, 0x100: LDS reads): group I < NV + NR is one MFMA (while any of the
// phase's P remain) followed by load I (I < NV) or fragment read I - NV; the
// remaining MFMAs follow.
template <int I, int NV, int NR, int P>
__device__ __forceinline__ void sched_pipe() {
  if constexpr (I < NV + NR) {
    __builtin_amdgcn_sched_group_barrier(0x008, I < P ? 1 : 0, 0);
    __builtin_amdgcn_sched_group_barrier(I < NV ? 0x020 : 0x100, 1, 0);
    sched_pipe<I + 1, NV, NR, P>();
  } else {
    __builtin_amdgcn_sched_group_barrier(0x008, P > NV + NR ? P - NV - NR : 0, 0);
  }
}

// Split-phase form for 64-deep k-tiles (128 bytes per row, 16x16x32 MFMAs,
// two 32-wide k groups per k-tile), with an SA-stage activation ring and an
// SB-stage weight ring (SB >= SA). The two-ring form above starts every
// k-tile by reading the first group's fragments right after the barrier and
// waiting for them; here the barrier sits in the middle of a k-tile instead:
// the MFMAs of group 0 run while group 1's fragments are read, then (once
// this wave's loads of k-tile kt + 1 have landed and it has read all of
// k-tile kt; the barrier makes that hold for every wave) the barrier, the
// loads of A(kt + SA) and B(kt + SB) into k-tile kt's stages, and the MFMAs
// of group 1 while group 0 of k-tile kt + 1 is read. Both sides of the
// barrier have MFMAs ready in registers. Same k order, same results bit for
// bit.
template <int BM, int BN, int WAVES_M, int WAVES_N, int SA, int SB, class Epi>
__device__ __forceinline__ void dls_tile(char* smem, const bf16* __restrict__ A, int lda,
                                         const bf16* __restrict__ B, int ldb, int M, int N,
                                         int m0, int n0, int tn, int tz, int kbeg, int kend,
                                         const Epi& epi) {
  static_assert(SA >= 2 && SB >= SA && SB <= 4, "stages");
  constexpr int RB = 128, BK = 64, CPR = 8, RPI = 8;
  constexpr int NW = WAVES_M * WAVES_N;
  constexpr int TM = BM / WAVES_M, TN = BN / WAVES_N;
  constexpr int FM = TM / 16, FN = TN / 16;
  static_assert(FM * 16 == TM && FN * 16 == TN, "wave tile");
  constexpr int STAGE_A = BM * RB, STAGE_B = BN * RB;
  constexpr int NI_A = BM / RPI, NI_B = BN / RPI;
  static_assert(NI_A * RPI == BM && NI_B * RPI == BN, "rows per instruction");
  constexpr bool EVEN_A = NI_A % NW == 0, EVEN_B = NI_B % NW == 0;
  constexpr int PERW_A = (NI_A + NW - 1) / NW, PERW_B = (NI_B + NW - 1) / NW;
  constexpr int MINW_A = NI_A / NW, MINW_B = NI_B / NW;
  // Issue order: the prologue loads A0 B0 A1 B1 .. A(SA-1) B(SA-1), then
  // B(SA) .. B(SB-1); iteration j loads A(j + SA) then B(j + SB). At the
  // barrier of iteration kt the loads that may stay in flight are those
  // issued after the later of A(kt + 1) and B(kt + 1), counted for the waves
  // with the fewest loads (a wave with more then also waits for a load or
  // two of a later k-tile, which is safe).
  constexpr int INFLIGHT = SA < SB ? MINW_B + (SA - 2) * (MINW_A + MINW_B)
                                   : (SA - 2) * (MINW_A + MINW_B);
  constexpr int PROLOGUE = (SA - 1) * MINW_A + (SB - 1) * MINW_B;   // after A0, B0
  static_assert(PROLOGUE < 64, "vmcnt range");
  char* const smem_b = smem + SA * STAGE_A;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const int nkt = kend > kbeg ? (kend - kbeg) / BK : 0;
  const int krot = Epi::kRotateK && nkt > 0 ? tn % nkt : 0;
  auto ktile = [&](int kt) { const int k = kt + krot; return k >= nkt ? k - nkt : k; };
  auto swz = [](int r) { return r & 7; };
  auto inst_a = [&](int j) { return EVEN_A ? wave * PERW_A + j : wave + j * NW; };
  auto inst_b = [&](int j) { return EVEN_B ? wave * PERW_B + j : wave + j * NW; };
  auto has_a = [&](int j) { return j < MINW_A || inst_a(j) < NI_A; };
  auto has_b = [&](int j) { return j < MINW_B || inst_b(j) < NI_B; };
  uint32_t srcA[PERW_A];
  uint32_t srcB[PERW_B];
#pragma unroll
  for (int j = 0; j < PERW_A; ++j) {
    const int row = RPI * inst_a(j) + lane / CPR;
    const int cc = (lane % CPR) ^ swz(row);
    srcA[j] = (uint32_t)min(m0 + row, M - 1) * (uint32_t)lda + kbeg + cc * 8;
  }
#pragma unroll
  for (int j = 0; j < PERW_B; ++j) {
    const int row = RPI * inst_b(j) + lane / CPR;
    const int cc = (lane % CPR) ^ swz(row);
    srcB[j] = (uint32_t)epi.b_row(min(n0 + row, N - 1)) * (uint32_t)ldb + kbeg + cc * 8;
  }
  auto issue_a = [&](int stage, int kt) {
    char* dst = smem + stage * STAGE_A;
    const bf16* a = A + kt * BK;
#pragma unroll
    for (int j = 0; j < PERW_A; ++j)
      if (has_a(j))
        __builtin_amdgcn_global_load_lds((gptr_t)(a + srcA[j]),
                                         (lptr_t)(dst + inst_a(j) * 1024), 16, 0, 0);
  };
  auto issue_b = [&](int stage, int kt) {
    char* dst = smem_b + stage * STAGE_B;
    const bf16* b = B + kt * BK;
#pragma unroll
    for (int j = 0; j < PERW_B; ++j)
      if (has_b(j))
        __builtin_amdgcn_global_load_lds((gptr_t)(b + srcB[j]),
                                         (lptr_t)(dst + inst_b(j) * 1024), 16, 0, 0);
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int a = 0; a < FM; ++a)
#pragma unroll
    for (int b = 0; b < FN; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  // fragment rows: base + (lane & 15); group g's chunk 4 g + lane / 16 at slot chunk ^ (row & 7)
  const int co0 = ((lane >> 4) ^ swz(lane & 15)) << 4;
  const int co1 = ((4 + (lane >> 4)) ^ swz(lane & 15)) << 4;
  const int a_off = (wm * TM + (lane & 15)) * RB;
  const int b_off = (wn * TN + (lane & 15)) * RB;
  u32x4 g0a[FM], g0b[FN], g1a[FM], g1b[FN];
  auto read0 = [&](int sa, int sb) {
    const char* pa = smem + sa * STAGE_A;
    const char* pb = smem_b + sb * STAGE_B;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
      g0a[fm] = *reinterpret_cast<const u32x4*>(pa + a_off + fm * 16 * RB + co0);
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
      g0b[fn] = *reinterpret_cast<const u32x4*>(pb + b_off + fn * 16 * RB + co0);
  };
  auto read1 = [&](int sa, int sb) {
    const char* pa = smem + sa * STAGE_A;
    const char* pb = smem_b + sb * STAGE_B;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
      g1a[fm] = *reinterpret_cast<const u32x4*>(pa + a_off + fm * 16 * RB + co1);
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
      g1b[fn] = *reinterpret_cast<const u32x4*>(pb + b_off + fn * 16 * RB + co1);
  };
  constexpr int NM = FM * FN, NR = FM + FN, NV = PERW_A + PERW_B;
  auto mma0 = [&]() {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        acc[fm][fn] = mfma16_bf16(__builtin_bit_cast(bf16x8, g0a[fm]),
                                  __builtin_bit_cast(bf16x8, g0b[fn]), acc[fm][fn]);
  };
  auto mma1 = [&]() {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        acc[fm][fn] = mfma16_bf16(__builtin_bit_cast(bf16x8, g1a[fm]),
                                  __builtin_bit_cast(bf16x8, g1b[fn]), acc[fm][fn]);
  };

#pragma unroll
  for (int j = 0; j < SB; ++j) {
    if (j < SA && j < nkt) issue_a(j, ktile(j));
    if (j < nkt) issue_b(j, ktile(j));
  }
  if (nkt > 0) {
    if (nkt >= SB) wait_vmcnt<PROLOGUE>(); else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    read0(0, 0);
  }
  // group 0 of k-tile kt with the reads of its group 1
  auto phase0 = [&](int kt) {
    read1(kt % SA, kt % SB);
    mma0();
    sched_pipe<0, 0, NR, NM>();
    __builtin_amdgcn_sched_barrier(0);
  };
  // steady state: the loads of k-tiles kt + SA (A) and kt + SB (B) go out
  // with the MFMAs of group 1
  int kt = 0;
  for (; kt + SB < nkt; ++kt) {
    phase0(kt);
    wait_vmcnt_lgkm0<INFLIGHT>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    issue_a(kt % SA, ktile(kt + SA));
    issue_b(kt % SB, ktile(kt + SB));
    // group 1 of k-tile kt with the reads of group 0 of k-tile kt + 1
    read0((kt + 1) % SA, (kt + 1) % SB);
    mma1();
    sched_pipe<0, NV, NR, NM>();
    __builtin_amdgcn_sched_barrier(0);
  }
  // the last k-tiles: the remaining activation loads, everything issued is
  // waited for
  for (; kt + 1 < nkt; ++kt) {
    phase0(kt);
    wait_vmcnt_lgkm0<0>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    if (kt + SA < nkt) issue_a(kt % SA, ktile(kt + SA));
    read0((kt + 1) % SA, (kt + 1) % SB);
    mma1();
    sched_pipe<0, 0, NR, NM>();
    __builtin_amdgcn_sched_barrier(0);
  }
  if (kt < nkt) {   // the last k-tile
    phase0(kt);
    mma1();
  }
  __syncthreads();
  epi(acc, m0 + wm * TM, n0 + wn * TN, lane, wn, smem, WAVES_N, BM, m0, tn, tz);
}

// The tile form of a configuration: SP = 1 the split-phase form, SP = 0 the
// two-ring form (both with SA activation and SB weight stages).
template <int BM, int BN, int WAVES_M, int WAVES_N, int SA, int SB, int RB, int MF, int SP,
          class Epi>
__device__ __forceinline__ void any_tile(char* smem, const bf16* __restrict__ A, int lda,
                                         const bf16* __restrict__ B, int ldb, int M, int N,
                                         int m0, int n0, int tn, int tz, int kbeg, int kend,
                                         const Epi& epi) {
  if constexpr (SP) {
    static_assert(MF == 16 && RB == 128, "split-phase form: 16x16x32 tiles, 128-byte rows");
    dls_tile<BM, BN, WAVES_M, WAVES_N, SA, SB, Epi>(smem, A, lda, B, ldb, M, N, m0, n0, tn, tz,
                                                    kbeg, kend, epi);
  } else {
    dl_tile<BM, BN, WAVES_M, WAVES_N, SA, SB, RB, MF, Epi>(smem, A, lda, B, ldb, M, N, m0, n0, tn,
                                                            tz, kbeg, kend, epi);
  }
}

// Sub-tiles of the last round: tile shapes a BM x BN tile splits into with the
// same waves (halves: two (BM/2) x BN tiles; quarters: four (BM/2) x (BN/2)).
template <int BM, int BN, int WAVES_M, int WAVES_N, int RB, int MF>
struct SubTiles {
  static constexpr int NW = WAVES_M * WAVES_N, RPI = 1024 / RB;
  static constexpr bool fits(int bm, int bn) {
    return bm % (RPI * NW) == 0 && bn % (RPI * NW) == 0 && (bm / WAVES_M) % MF == 0 &&
           (bn / WAVES_N) % (2 * MF) == 0;
  }
  static constexpr bool kHalf = fits(BM / 2, BN);
  static constexpr bool kQuarter = fits(BM / 2, BN / 2);
};

// Grid: one block per tile of the logical order (a 3-D grid of column tiles x
// row tiles x K slices), except that the last n_tail tiles of that order may
// each be split into `sub` (2 or 4) sub-tiles, one block each, launched after
// all whole tiles (then a 1-D grid): when the tile count leaves a last round
// that fills at most half of the CUs, its tiles then finish in a fraction of a
// whole tile's time. Sub-tiles accumulate every output element over the same
// k order as whole tiles, so the results are the same bit for bit.
template <int BM, int BN, int WAVES_M, int WAVES_N, int SA, int SB, int RB, int MF, int SP,
          bool TAIL, class Epi>
__global__ __launch_bounds__(WAVES_M* WAVES_N * 64) void gemm_dl_kernel(
    const bf16* __restrict__ A, int lda, const bf16* __restrict__ B, int ldb, int M, int N,
    int K, int k_per_split, int n_n, int n_m, int group_m, int n_tail, int sub, Epi epi) {
  __shared__ __attribute__((aligned(1024))) char smem[(SA * BM + SB * BN) * RB];
  // Tile order. The logical order enumerates (K slice, row tile, column tile)
  // with the column tile fastest (group_m == 0), or, for weight matrices
  // larger than the last-level cache (group_m > 0), goes down a group of
  // group_m row tiles before moving to the next column tile, so that each
  // weight column tile is fetched from HBM about once per group of row tiles
  // instead of once per row tile. The dispatcher hands out blocks in linear
  // order round-robin over the 8 XCDs (block i to XCD i mod 8), each with its
  // own L2; with group_m > 0 the whole tiles are remapped so that each XCD
  // receives one contiguous range of the logical order (blocks sharing a
  // weight column tile run on the same XCD at about the same time).
  // (TAIL: the instance for launches with sub-tiles, a 1-D grid; the other
  // one has whole tiles only and a 3-D grid)
  // logical tile lid -> (K slice, row tile, column tile)
  auto logical = [&](int lid, int& tz, int& tm, int& tn) {
    const int plane = n_n * n_m;
    tz = lid / plane;
    const int l = lid - tz * plane;
    if (group_m > 0) {
      const int per_group = group_m * n_n;
      const int gi = l / per_group;
      const int first = gi * group_m;
      const int gsz = min(n_m - first, group_m);
      const int r = l - gi * per_group;
      tm = first + r % gsz;
      tn = r / gsz;
    } else {
      tm = l / n_n;
      tn = l - tm * n_n;
    }
  };
  // linear dispatch id -> logical tile: each XCD a contiguous range of nb tiles
  auto xcd_range = [](int id, int nb) {
    const int xcd = id % kXcds, per = nb / kXcds, rem = nb % kXcds;
    return xcd * per + min(xcd, rem) + id / kXcds;
  };
  int tz, tm, tn, part = 0;
  bool is_sub = false;
  if constexpr (!TAIL) {
    tm = blockIdx.y;
    tn = blockIdx.x;
    tz = blockIdx.z;
    if (group_m > 0) {
      const int id = (blockIdx.z * n_m + blockIdx.y) * n_n + blockIdx.x;
      logical(xcd_range(id, n_n * n_m * (int)gridDim.z), tz, tm, tn);
    }
  } else {
    const int n_main = n_n * n_m * (K / k_per_split) - n_tail;
    const int id = blockIdx.x;
    if (id < n_main) {
      logical(group_m > 0 ? xcd_range(id, n_main) : id, tz, tm, tn);
    } else {
      is_sub = true;
      part = (id - n_main) % sub;
      logical(n_main + (id - n_main) / sub, tz, tm, tn);
    }
  }
  const int m0 = tm * BM, n0 = tn * BN;
  if (epi.skip_tile(m0)) return;   // uniform over the block
  const int kbeg = tz * k_per_split;
  const int kend = min(K, kbeg + k_per_split);
  typedef SubTiles<BM, BN, WAVES_M, WAVES_N, RB, MF> Sub;
  if (is_sub) {
    if constexpr (TAIL && Epi::kTailSplit && Sub::kQuarter) {
      if (sub == 4) {
        any_tile<BM / 2, BN / 2, WAVES_M, WAVES_N, SA, SB, RB, MF, SP, Epi>(
            smem, A, lda, B, ldb, M, N, m0 + (part >> 1) * (BM / 2), n0 + (part & 1) * (BN / 2),
            tn, tz, kbeg, kend, epi);
        return;
      }
    }
    if constexpr (TAIL && Epi::kTailSplit && Sub::kHalf) {
      if (sub == 2) {
        any_tile<BM / 2, BN, WAVES_M, WAVES_N, SA, SB, RB, MF, SP, Epi>(
            smem, A, lda, B, ldb, M, N, m0 + part * (BM / 2), n0, tn, tz, kbeg, kend, epi);
        return;
      }
    }
    return;   // not reached: the launcher only splits where the shapes allow
  }
  any_tile<BM, BN, WAVES_M, WAVES_N, SA, SB, RB, MF, SP, Epi>(smem, A, lda, B, ldb, M, N, m0, n0, tn,
                                                          tz, kbeg, kend, epi);
}

// LM head over the rows that need a prediction only. The head is planned for
// its largest row count and the count of rows that need a prediction is
// known on the device only; one block per tile would dispatch every tile and
// let those beyond the count exit, and in the grouped order such skipped
// blocks come in runs between the active ones of each column tile (18-23 %
// of the launch at ~1400 of 4096 rows). Here each XCD's blocks (linear block
// i runs on XCD i mod 8) walk the active tiles of the XCD's contiguous range
// of column tiles, the rows of one column tile on consecutive blocks, so
// those share the column's weight tile in L2 at about the same time, as in
// the grouped order. No block waits on another.
template <int BM, int BN, int WAVES_M, int WAVES_N, int SA, int SB, int RB, int MF, int SP>
__global__ __launch_bounds__(WAVES_M* WAVES_N * 64) void gemm_dl_head_kernel(
    const bf16* __restrict__ A, int lda, const bf16* __restrict__ B, int ldb, int M, int N,
    int K, int n_n, EpiLMHead epi) {
  __shared__ __attribute__((aligned(1024))) char smem[(SA * BM + SB * BN) * RB];
  const int rows = epi.m_count ? min(*epi.m_count, M) : M;
  const int act = rows > 0 ? (rows + BM - 1) / BM : 0;     // active row tiles
  const int xcd = blockIdx.x % kXcds, k = blockIdx.x / kXcds;
  const int nbx = ((int)gridDim.x - xcd + kXcds - 1) / kXcds;   // blocks on this XCD
  const int c0 = (int)((long)n_n * xcd / kXcds), c1 = (int)((long)n_n * (xcd + 1) / kXcds);
  const int total = (c1 - c0) * act;
  for (int a = k; a < total; a += nbx) {
    const int c = a / act;
    const int tn = c0 + c, tm = a - c * act;
    any_tile<BM, BN, WAVES_M, WAVES_N, SA, SB, RB, MF, SP, EpiLMHead>(
        smem, A, lda, B, ldb, M, N, tm * BM, tn * BN, tn, 0, 0, K, epi);
    __syncthreads();   // the epilogue's LDS reads before the next tile's loads
  }
}

// Tile configurations (BM, BN, waves M x N, activation stages, weight stages,
// k-tile row bytes, MFMA tile 16x16x32 or 32x32x16, split-phase form). The
// split-phase form serves the eight-wave tiles (two waves per SIMD: 3-10 %
// faster than the two-ring form of the same tile at every k-tile count; the
// four-wave tiles, one wave per SIMD, run slower in it and keep the two-ring
// form). 256x224 (wave tiles of 64x112, seven column
// fragments) covers a 3584-wide output in 16 column tiles, so that 4096 rows
// make exactly one round of 256 tiles.
#define DL_CONFIGS(X)                      \
  X(1, 128, 128, 2, 2, 2, 2, 128, 16, 0)   \
  X(6, 256, 256, 2, 4, 2, 3, 128, 16, 1)   \
  X(10, 64, 128, 2, 2, 2, 2, 128, 16, 0)   \
  X(11, 64, 128, 2, 2, 2, 3, 128, 16, 0)   \
  X(21, 256, 192, 4, 2, 2, 3, 128, 16, 1)  \
  X(22, 128, 192, 2, 2, 2, 2, 128, 16, 0)  \
  X(29, 256, 128, 4, 2, 3, 3, 128, 16, 1)  \
  X(42, 128, 192, 2, 2, 2, 3, 128, 16, 0)  \
  X(62, 256, 128, 2, 2, 2, 2, 128, 32, 0)  \
  X(65, 384, 256, 4, 2, 2, 2, 128, 32, 0)  \
  X(70, 256, 224, 4, 2, 2, 3, 128, 16, 1)

int gemm_dl_tile(int cfg, int* bm, int* bn, int* threads) {
  switch (cfg) {
#define X(id, BM_, BN_, WM_, WN_, SA_, S_, RB_, MF_, SP_) \
  case id: *bm = BM_; *bn = BN_; *threads = WM_ * WN_ * 64; return 1;
    DL_CONFIGS(X)
#undef X
  }
  return 0;
}

int gemm_dl_mfma(int cfg) {
  switch (cfg) {
#define X(id, BM_, BN_, WM_, WN_, SA_, S_, RB_, MF_, SP_) \
  case id: return MF_;
    DL_CONFIGS(X)
#undef X
  }
  return 0;
}

// Whether a wave's tile holds an odd number of MFMA column fragments (the
// SwiGLU epilogue, which stores gate/up fragment pairs, cannot run it).
int gemm_dl_odd(int cfg) {
  switch (cfg) {
#define X(id, BM_, BN_, WM_, WN_, SA_, S_, RB_, MF_, SP_) \
  case id: return (BN_ / WN_ / MF_) % 2;
    DL_CONFIGS(X)
#undef X
  }
  return 0;
}

// Sub-tile splits a configuration allows for the last round (bit 1: halves,
// bit 2: quarters).
int gemm_dl_subs(int cfg) {
  switch (cfg) {
#define X(id, BM_, BN_, WM_, WN_, SA_, S_, RB_, MF_, SP_)                          \
  case id: {                                                                \
    typedef SubTiles<BM_, BN_, WM_, WN_, RB_, MF_> S;                       \
    return (S::kHalf ? 2 : 0) | (S::kQuarter ? 4 : 0);                      \
  }
    DL_CONFIGS(X)
#undef X
  }
  return 0;
}

template <class Epi>
hipError_t gemm_dl_launch(int cfg, const bf16* A, int lda, const bf16* B, int ldb, int M, int N,
                          int K, int splits, int group_m, int sub, int n_tail, const Epi& epi,
                          hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (K % 64 != 0 || splits < 1 || (K / 64) % splits != 0) return hipErrorInvalidValue;
  // the kernel addresses operands with 32-bit element offsets
  if ((double)(M - 1) * lda + K >= 4294967296.0 || (double)(N - 1) * ldb + K >= 4294967296.0)
    return hipErrorInvalidValue;
  const int kps = K / splits;
  if (sub == 0) n_tail = 0;
  if (n_tail < 0 || (sub != 0 && (!Epi::kTailSplit || !(gemm_dl_subs(cfg) & sub))))
    return hipErrorInvalidValue;
  switch (cfg) {
#define X(id, BM_, BN_, WM_, WN_, SA_, S_, RB_, MF_, SP_)                                        \
  case id: {                                                                             \
    if constexpr ((MF_ == 32 && !Epi::kMf32) ||                                          \
                  (!Epi::kOddFragments && (BN_ / WN_ / MF_) % 2 != 0))                   \
      return hipErrorInvalidValue;                                                       \
    else {                                                                               \
      const int n_n = ceil_div(N, BN_), n_m = ceil_div(M, BM_);                          \
      const long total = (long)n_n * n_m * splits;                                       \
      if (n_tail > total) return hipErrorInvalidValue;                                   \
      const long blocks = total - n_tail + (long)sub * n_tail;                           \
      if (blocks >= (1L << 31)) return hipErrorInvalidValue;                             \
      Epi e = epi;                                                                       \
      e.set_mfma(MF_);                                                                   \
      if (n_tail == 0) {                                                                 \
        DLM_LAUNCH((gemm_dl_kernel<BM_, BN_, WM_, WN_, SA_, S_, RB_, MF_, SP_, false, Epi>),   \
                   dim3(n_n, n_m, splits), dim3(WM_ * WN_ * 64), 0, st, A, lda, B, ldb, M, \
                   N, K, kps, n_n, n_m, group_m, 0, 0, e);                               \
      } else if constexpr (Epi::kTailSplit) {                                            \
        DLM_LAUNCH((gemm_dl_kernel<BM_, BN_, WM_, WN_, SA_, S_, RB_, MF_, SP_, true, Epi>),    \
                   dim3((unsigned)blocks), dim3(WM_ * WN_ * 64), 0, st, A, lda, B, ldb, M, \
                   N, K, kps, n_n, n_m, group_m, n_tail, sub, e);                        \
      }                                                                                  \
      return hipGetLastError();                                                          \
    }                                                                                    \
  }
    DL_CONFIGS(X)
#undef X
  }
  return hipErrorInvalidValue;
}

hipError_t gemm_dl_head_launch(int cfg, const bf16* A, int lda, const bf16* B, int ldb, int M,
                               int N, int K, int num_cu, const EpiLMHead& epi, hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (K % 64 != 0 || num_cu < kXcds) return hipErrorInvalidValue;
  if ((double)(M - 1) * lda + K >= 4294967296.0 || (double)(N - 1) * ldb + K >= 4294967296.0)
    return hipErrorInvalidValue;
  switch (cfg) {
#define X(id, BM_, BN_, WM_, WN_, SA_, S_, RB_, MF_, SP_)                                         \
  case id: {                                                                              \
    if constexpr (MF_ == 32) return hipErrorInvalidValue;                                 \
    else {                                                                                \
      /* blocks per CU: bounded by the LDS (160 KB) and by 32 waves per CU */              \
      constexpr int kLds = (SA_ * BM_ + S_ * BN_) * RB_, kWaves = WM_ * WN_;                     \
      constexpr int kOcc = 163840 / kLds < 32 / kWaves ? 163840 / kLds : 32 / kWaves;     \
      EpiLMHead e = epi;                                                                  \
      e.set_mfma(MF_);                                                                    \
      DLM_LAUNCH((gemm_dl_head_kernel<BM_, BN_, WM_, WN_, SA_, S_, RB_, MF_, SP_>),            \
                 dim3(num_cu * (kOcc > 0 ? kOcc : 1)), dim3(kWaves * 64), 0, st, A, lda, B, \
                 ldb, M, N, K, ceil_div(N, BN_), e);                                      \
      return hipGetLastError();                                                           \
    }                                                                                     \
  }
    DL_CONFIGS(X)
#undef X
  }
  return hipErrorInvalidValue;
}

template hipError_t gemm_dl_launch<EpiStore>(int, const bf16*, int, const bf16*, int, int, int,
    int, int, int, int, int, const EpiStore&, hipStream_t);
template hipError_t gemm_dl_launch<EpiAdd>(int, const bf16*, int, const bf16*, int, int, int,
    int, int, int, int, int, const EpiAdd&, hipStream_t);
template hipError_t gemm_dl_launch<EpiScaledStore>(int, const bf16*, int, const bf16*, int, int, int,
    int, int, int, int, int, const EpiScaledStore&, hipStream_t);
template hipError_t gemm_dl_launch<EpiSwiGLU<bf16>>(int, const bf16*, int, const bf16*, int, int, int,
    int, int, int, int, int, const EpiSwiGLU<bf16>&, hipStream_t);
template hipError_t gemm_dl_launch<EpiLMHead>(int, const bf16*, int, const bf16*, int, int, int,
    int, int, int, int, int, const EpiLMHead&, hipStream_t);

}  // namespace dlm
