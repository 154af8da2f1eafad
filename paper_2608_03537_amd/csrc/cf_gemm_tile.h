// GEMM + row-subgraph kernel template for gfx950 (instantiated in cf_gemm_inst_*.hip).
//
// One tiled MFMA GEMM template whose epilogue runs the Stage-Stream stage
// chain (Sec. III) on the accumulator tile while it is still in registers:
//   stage 1 (elementwise): x = alpha * acc + bias + residual
//   stage 2 (reduction):   LayerNorm / RMSNorm row statistics, then the
//                          normalising PostOp on the same register values
//                          (the bypass path of Sec. III-B: x is not recomputed)
//   stage 3 (elementwise): activation, store
//   stage 4 (reduction):   row amax -> scale -> E4M3 codes
//
// Transposed product.  The MFMA computes D^T = W^T . X^T: the A operand is a
// slab of W^T (rows n), the B operand a slab of X (rows m).  In the 32x32
// accumulator block a lane then holds ONE output row m (column of D^T) and 16
// of its columns n, so a row reduction is mostly lane-local (16 values per
// block), then one exchange with lane l^32, then an LDS combine across the
// waves that share the row (reduce levels 1 and 2 of Sec. III-A).
//
// Level 3 (across workgroups sharing a row block, Sec. III-A) has two forms:
//   ROWS_CLUSTER: the cn workgroups of a row block are co-resident (persistent
//     grid no larger than the resident capacity) and exchange per-row partial
//     (mean, M2) / amax through a small workspace with an arrival counter,
//     peer to peer: each workgroup merges all partials itself in a fixed
//     order, so every workgroup gets bit-identical statistics.
//   ROWS_SPLIT: each workgroup writes fp32 x and its partial (mean, M2); a
//     light finish pass merges them (Chan et al.'s pairwise update) and runs
//     stages 2..4.
#pragma once

#include <type_traits>

#include "cf_device.h"
#include "cf_internal.h"

namespace cf {

template <typename TIn, int BM_, int BN_, int WM_, int WN_, int TKB_, int STAGES_ = 0>
struct TileShape {
  using T = TIn;
  // STAGES > 0 selects the direct-to-LDS pipeline (mainloop_v2) for K a
  // multiple of the 128-byte stage (bf16 weights in either layout, fp32 ones
  // stored N x K); the register-staged loop (mainloop) serves the rest.
  static constexpr int STAGES = STAGES_;
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr int NW = WM * WN, NT = 64 * NW;
  static constexpr int WTM = 32 * BM, WTN = 32 * BN;     // wave tile (m, n)
  static constexpr int TM = WTM * WM, TN = WTN * WN;     // workgroup tile
  static constexpr int EPC = 16 / (int)sizeof(T);        // elements per 16 B
  static constexpr int TKB = TKB_;                        // k bytes per stage
  static constexpr int TK = TKB / (int)sizeof(T);
  static constexpr int KSTEP = 2 * EPC;                   // k per MFMA step
  static constexpr int CPR = TK / EPC;                    // chunks per row
  static constexpr int ROWB = TKB + 16;                   // padded LDS row
  static constexpr int A_BYTES = TN * ROWB, B_BYTES = TM * ROWB;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int V2_ROWB = 128;                    // bytes of k per row per stage
  static constexpr int V2_TK = V2_ROWB / (int)sizeof(T);
  static constexpr int V2_STAGE = (TM + TN) * V2_ROWB;
  static constexpr int V2_INSTR = (TM + TN) / 8;          // 8 rows per wave-wide load
  static constexpr int V2_PER_WAVE = V2_INSTR / NW;
  static constexpr int LDS_V1 = 2 * STAGE;
  static constexpr int LDS_V2 = STAGES * V2_STAGE;
  static_assert(STAGES == 0 || (V2_INSTR % NW == 0 && STAGES >= 2), "v2 pipeline shape");
  static_assert(STAGES == 0 || V2_PER_WAVE * (STAGES - 2) < 64, "vmcnt range");
  static constexpr int A_CHUNKS = TN * CPR, B_CHUNKS = TM * CPR;
  static constexpr int A_PT = (A_CHUNKS + NT - 1) / NT;
  static constexpr int B_PT = (B_CHUNKS + NT - 1) / NT;
  static constexpr int LDS_STORE = TM * (TN * 4 + 16);   // staged output tile (fp32 worst case)
  // Row-reduction scratch sits at the end of LDS, past the staged output tile.
  // (count, mean, M2) per row and wave column, then the row-cluster round tag
  static constexpr int RED_BYTES = 3 * WN * TM * 4, TAIL_BYTES = RED_BYTES + 16;
  static constexpr int SMEM_V1 = LDS_V1 > LDS_STORE + TAIL_BYTES ? LDS_V1 : LDS_STORE + TAIL_BYTES;
  static constexpr int SMEM_V2 = LDS_V2 > LDS_STORE + TAIL_BYTES ? LDS_V2 : LDS_STORE + TAIL_BYTES;
  static_assert(SMEM_V1 <= 160 * 1024 && SMEM_V2 <= 160 * 1024, "LDS budget");
  // Epilogue operands of the bf16 direct-to-LDS loop (residual tile and the
  // per-column vectors) are loaded by the last main-loop iterations into the
  // two ring slots that free up first (slots 0 and 1): residual rows [0, RA)
  // and the four 1 KB vector regions in slot 0, rows [RA, TM) in slot 1.  A
  // vector region holds 256 fp32 columns (one 16-byte load per lane).
  static constexpr bool STG = STAGES >= 3 && sizeof(T) == 2 && TN <= 256;
  static constexpr int STG_VEC = 4096;
  static constexpr int STG_RA0 = STAGES ? (V2_STAGE - STG_VEC) / (TN * 2) / 32 * 32 : 0;
  static constexpr int STG_RA = STG_RA0 < TM ? STG_RA0 : TM;
  static constexpr int STG_RB = TM - STG_RA;
  static constexpr int STG_CPR = TN * 2 / 16;                      // 16-byte chunks per residual row
  static constexpr int STG_IA = STG_RA * STG_CPR / (64 * NW);      // wave-wide loads per wave, rows [0, RA)
  static constexpr int STG_IB = STG_RB * STG_CPR / (64 * NW);      // rows [RA, TM)
  static_assert(!STG || ((STG_RA * STG_CPR) % (64 * NW) == 0 && (STG_RB * STG_CPR) % (64 * NW) == 0 &&
                         STG_RB * TN * 2 <= V2_STAGE && STG_RA > 0), "epilogue staging split");
  static_assert(!STG || V2_PER_WAVE * (STAGES - 2) + STG_IA + 1 + STG_IB < 64, "vmcnt range (staging)");
  static_assert(TK % KSTEP == 0, "stage must hold whole MFMA steps");
};

// ---------------------------------------------------------------------------
// Accumulator start value.  When the epilogue adds the bias unscaled
// (alpha = 1), the accumulators start from the bias of their columns, so
// x = acc + bias comes out of the MFMA chain and stage 1 loses one add per
// element.  Columns past N start at 0.  The loads are issued before any
// main-loop load, so the first wait of the main loop covers them.
// ---------------------------------------------------------------------------
// PERM: the main loop loads the W^T rows of every 32-row block with bits 2
// and 3 of the row index swapped (perm23), so accumulator elements 4g..4g+3
// of lane half lg hold columns 16 (g / 2) + 8 lg + 4 (g % 2) + 0..3 of the block.
__device__ __forceinline__ int perm23(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }

template <class S, bool PERM = false>
__device__ __forceinline__ void acc_init(f32x16_t (&acc)[S::BM][S::BN], const GemmRowsParams& p, int n0, int lane,
                                         int wn, bool fold_bias) {
  const int lg = lane >> 5;
#pragma unroll
  for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int n = n0 + wn * S::WTN + bn * 32 + (PERM ? 16 * (g >> 1) + 8 * lg + 4 * (g & 1) : 8 * g + 4 * lg);
      f32x4_t b = {0.0f, 0.0f, 0.0f, 0.0f};
      if (fold_bias && n < p.N) b = *reinterpret_cast<const f32x4_t*>(p.epi.bias + n);
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[bm][bn][4 * g + q] = b[q];
    }
  __builtin_amdgcn_sched_barrier(0);
}

// ---------------------------------------------------------------------------
// Main loop: global -> registers -> LDS (double buffered) -> MFMA.
// ---------------------------------------------------------------------------
template <class S>
__device__ __forceinline__ void mainloop(f32x16_t (&acc)[S::BM][S::BN],
                                         const typename S::T* __restrict__ X,
                                         const typename S::T* __restrict__ W,
                                         const GemmRowsParams& p, int m0, int n0,
                                         char* smem, int tid, int lane, int wm, int wn, bool fold_bias) {
  using T = typename S::T;
  acc_init<S>(acc, p, n0, lane, wn, fold_bias);

  const int M = p.M, N = p.N, K = p.K;
  const int KT = (K + S::TK - 1) / S::TK;
  const bool nk = p.w_nk != 0;
  u32x4_t ra[S::A_PT], rb[S::B_PT];
  const u32x4_t zero = {0u, 0u, 0u, 0u};

  auto gload = [&](int kt) {
    const int k0 = kt * S::TK;
#pragma unroll
    for (int j = 0; j < S::A_PT; ++j) {
      const int ch = tid + j * S::NT;
      ra[j] = zero;
      if (ch < S::A_CHUNKS) {
        if (nk) {           // W stored N x K: chunk = 8 (4) consecutive k of row n
          const int row = ch / S::CPR, col = ch % S::CPR;
          const int n = n0 + row, k = k0 + col * S::EPC;
          if (n < N && k < K) ra[j] = gload16(W + (int64_t)n * p.ldw + k);
        } else {            // W stored K x N: chunk = 8 (4) consecutive n of row k
          const int cpn = S::TN / S::EPC;
          const int kr = ch / cpn, nc = ch % cpn;
          const int n = n0 + nc * S::EPC, k = k0 + kr;
          if (n < N && k < K) ra[j] = gload16(W + (int64_t)k * p.ldw + n);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < S::B_PT; ++j) {
      const int ch = tid + j * S::NT;
      rb[j] = zero;
      if (ch < S::B_CHUNKS) {
        const int row = ch / S::CPR, col = ch % S::CPR;
        const int m = m0 + row, k = k0 + col * S::EPC;
        if (m < M && k < K) rb[j] = gload16(X + (int64_t)m * p.ldx + k);
      }
    }
  };

  auto lstore = [&](int buf) {
    char* sA = smem + buf * S::STAGE;
    char* sB = sA + S::A_BYTES;
#pragma unroll
    for (int j = 0; j < S::A_PT; ++j) {
      const int ch = tid + j * S::NT;
      if (ch < S::A_CHUNKS) {
        if (nk) {
          const int row = ch / S::CPR, col = ch % S::CPR;
          lds_write16(sA + row * S::ROWB + col * 16, ra[j]);
        } else {
          // Transpose on the way in: element e of the chunk is W[k][n+e],
          // stored at LDS row n+e, column k.
          const int cpn = S::TN / S::EPC;
          const int kr = ch / cpn, nc = ch % cpn;
          char* dst = sA + (nc * S::EPC) * S::ROWB + kr * (int)sizeof(T);
          if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const uint32_t w = ra[j][e >> 1];
              *reinterpret_cast<uint16_t*>(dst + e * S::ROWB) =
                  (uint16_t)((e & 1) ? (w >> 16) : (w & 0xFFFFu));
            }
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              *reinterpret_cast<uint32_t*>(dst + e * S::ROWB) = ra[j][e];
          }
        }
      }
    }
#pragma unroll
    for (int j = 0; j < S::B_PT; ++j) {
      const int ch = tid + j * S::NT;
      if (ch < S::B_CHUNKS) {
        const int row = ch / S::CPR, col = ch % S::CPR;
        lds_write16(sB + row * S::ROWB + col * 16, rb[j]);
      }
    }
  };

  const int lr = lane & 31, lg = lane >> 5;
  auto compute = [&](int buf) {
    const char* sA = smem + buf * S::STAGE;
    const char* sB = sA + S::A_BYTES;
#pragma unroll
    for (int ks = 0; ks < S::TK / S::KSTEP; ++ks) {
      const int koff = (ks * S::KSTEP + lg * S::EPC) * (int)sizeof(T);
      u32x4_t a[S::BN], b[S::BM];
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
        a[bn] = lds_read16(sA + (wn * S::WTN + bn * 32 + lr) * S::ROWB + koff);
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm)
        b[bm] = lds_read16(sB + (wm * S::WTM + bm * 32 + lr) * S::ROWB + koff);
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
        for (int bn = 0; bn < S::BN; ++bn) Mma<T>::run(acc[bm][bn], a[bn], b[bm]);
    }
  };

  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const bool more = kt + 1 < KT;
    if (more) gload(kt + 1);
    compute(kt & 1);
    if (more) lstore((kt + 1) & 1);
    __syncthreads();
  }
}

// 16-byte global -> LDS copy for the whole wave: lane i's 16 bytes land at
// LDS address lds + 16 * i (lds must be wave-uniform).
template <int AUX = 0>
__device__ __forceinline__ void dma16(const void* gptr, char* lds) {
  __builtin_amdgcn_global_load_lds(gptr, (__attribute__((address_space(3))) void*)lds, 16, 0, AUX);
}
// Workgroup barrier without the implicit wait for outstanding memory
// operations (callers wait explicitly); also a compiler reordering fence.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Wait until at most N vector-memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // gfx9 s_waitcnt: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] at [15:14]
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// ---------------------------------------------------------------------------
// Main loop v2: direct global -> LDS loads (global_load_lds_dwordx4), a ring
// of S::STAGES stages, no register staging.  A stage holds 128 bytes of k for
// the TN rows of W^T followed by the TM rows of X.  Needs K / V2_TK >= STAGES-1
// (the host plans the register-staged loop otherwise).
//
// LDS layout: within a row the eight 16-byte chunks are XOR-swizzled by
// ((row >> 1) & 7).  gfx950 serves a 64-lane ds_read_b128 in 16-lane groups
// over 64 four-byte banks; the 16 lanes of a group read one chunk column of 16
// consecutive rows, and this swizzle puts them on 16 distinct 16-byte bank
// groups (rows 2j and 2j+1 differ by 128 bytes, the pairs by the swizzle).
// A wave-wide load writes 1 KB of consecutive LDS = 8 rows, lane i filling
// row i/8 at chunk position i%8.
//
// Schedule of one stage (KS MFMA steps).  All fragments of a stage live in
// registers.  Iteration kt first reads the fragments of its last step, then
// issues the MFMAs of steps 0..KS-2 with this wave's share of the loads of
// stage kt+S-1 spread between them.  It then waits until stage kt+1 has landed
// (vmcnt) and all of this wave's LDS reads are done (lgkmcnt), meets the other
// waves at a barrier, and reads the fragments of steps 0..KS-2 of stage kt+1
// while the MFMAs of its last step run.  So LDS latency is hidden behind MFMAs
// and the one barrier per stage also frees the ring slot that the next
// iteration's loads overwrite (its last reader finished before the barrier).
// The last S-1 iterations issue no loads; their waits shrink accordingly.
//
// Rows past M (or N) are clamped to the last valid row: they only feed output
// rows/columns that the epilogue masks.
//
// KN (bf16, W stored K x N, N a multiple of 8, TN a multiple of 128): the W
// part of a stage holds the 64 k-rows of the tile as they lie in memory, TN
// columns each, the 64-byte blocks of row k XOR-swizzled by (k & 3).  The A
// fragment (8 consecutive k of one column) comes from two transposing reads
// (ds_read_b64_tr_b16): in each group of 16 lanes, lane r points at 4
// consecutive columns of k-row r / 4, and lane i gets the 4 k-values of
// column i.  The 32 lanes served together read 4 k-rows x 64 bytes, which the
// swizzle places on 4 distinct 64-byte bank groups.  Columns past N are
// clamped to the last 8-column chunk.
// ---------------------------------------------------------------------------
// Ring geometry shared by the main loop and the early issue of its first
// stages: this wave's global source of each of its PW 1 KB loads at stage 0,
// the bytes between consecutive stages, and the slot rotation.
template <class S, bool PERM, bool KN>
struct RingSrc {
  const char* src[S::V2_PER_WAVE];
  int64_t w_step;
  int rot;
  __device__ __forceinline__ RingSrc(const typename S::T* __restrict__ X, const typename S::T* __restrict__ W,
                                     const GemmRowsParams& p, int m0, int n0, int lane, int wave) {
    using T = typename S::T;
    constexpr int NS = S::STAGES, PW = S::V2_PER_WAVE;
    static_assert(!KN || (sizeof(T) == 2 && S::TN % 128 == 0 && !PERM), "K x N ring: bf16, TN % 128 == 0");
    constexpr int KN_RW = S::TN * 2;               // bytes of one k-row of the W part (KN)
    // Ring slot of stage st: rotated so that the last stage lands in slot
    // NS-1 and the slots freed during the last iterations are 0, 1, ...
    rot = (NS - (p.K / S::V2_TK) % NS) % NS;
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      const int row = (wave + j * S::NW) * 8 + (lane >> 3);
      const int c = (lane & 7) ^ ((row >> 1) & 7);
      if (row < S::TN) {
        if constexpr (KN) {
          const int o = (wave + j * S::NW) * 1024 + lane * 16;   // byte within the W part
          const int k = o / KN_RW, gc = ((o % KN_RW) >> 4) ^ ((k & 3) << 2);
          const int n = min(n0 + gc * 8, p.N - 8);
          src[j] = reinterpret_cast<const char*>(W + (int64_t)k * p.ldw + n);
        } else {
          const int n = min(n0 + (PERM ? perm23(row) : row), p.N - 1);
          src[j] = reinterpret_cast<const char*>(W + (int64_t)n * p.ldw) + c * 16;
        }
      } else {
        const int m = min(m0 + row - S::TN, p.M - 1);
        src[j] = reinterpret_cast<const char*>(X + (int64_t)m * p.ldx) + c * 16;
      }
    }
    // Bytes between consecutive stages of a load: 128 along k, or (KN W
    // part) 64 k-rows of W.
    w_step = KN ? (int64_t)S::V2_TK * p.ldw * (int64_t)sizeof(T) : S::V2_ROWB;
  }
  __device__ __forceinline__ char* slot(char* smem, int st) const {
    return smem + ((st + rot) % S::STAGES) * S::V2_STAGE;
  }
  // Load j (of PW) of stage st into its ring slot.
  __device__ __forceinline__ void issue(char* smem, int wave, int j, int st) const {
    const bool wpart = (wave + j * S::NW) * 8 < S::TN;
    dma16(src[j] + (int64_t)st * (wpart ? w_step : (int64_t)S::V2_ROWB), slot(smem, st) + (wave + j * S::NW) * 1024);
  }
  // Stages 0 .. NS-2 (the ring's prologue).
  __device__ __forceinline__ void prologue(char* smem, int wave) const {
#pragma unroll
    for (int st = 0; st < S::STAGES - 1; ++st)
#pragma unroll
      for (int j = 0; j < S::V2_PER_WAVE; ++j) issue(smem, wave, j, st);
  }
};

template <class S, bool STG, bool PERM = false, bool KN = false>
__device__ __forceinline__ void mainloop_v2(f32x16_t (&acc)[S::BM][S::BN],
                                            const typename S::T* __restrict__ X,
                                            const typename S::T* __restrict__ W,
                                            const GemmRowsParams& p, int m0, int n0, int bz,
                                            char* smem, int lane, int wave, int wm, int wn, bool fold_bias) {
  using T = typename S::T;
  acc_init<S, PERM>(acc, p, n0, lane, wn, fold_bias);

  constexpr int NS = S::STAGES, PW = S::V2_PER_WAVE;
  const int KT = p.K / S::V2_TK;
  constexpr int KN_RW = S::TN * 2;                 // bytes of one k-row of the W part (KN)
  const RingSrc<S, PERM, KN> ring(X, W, p, m0, n0, lane, wave);
  auto slot = [&](int st) { return ring.slot(smem, st); };
  auto dma = [&](int j, int st) { ring.issue(smem, wave, j, st); };
  // Epilogue staging loads: residual rows (part 0: rows [0, RA) into slot 0,
  // part 1: rows [RA, TM) into slot 1) with the 16-byte chunk of column group
  // c of row r stored at chunk position c ^ (r & 7); and one vector region per
  // wave (bias, gamma, beta, unused).  Absent operands load a valid dummy so
  // every wave issues the same number of loads.
  auto stage_dma = [&](int part, int i) {
    if constexpr (STG) {
      const RowEpi& e = p.epi;
      const int q = (wave * (part ? S::STG_IB : S::STG_IA) + i) * 64 + lane;
      const int rr = (part ? S::STG_RA : 0) + q / S::STG_CPR;
      const int c = (q % S::STG_CPR) ^ (rr & 7);
      const char* g = reinterpret_cast<const char*>(X);
      if (e.R) {
        const int m = min(m0 + rr, p.M - 1), n = min(n0 + c * 8, p.N - 8);
        g = reinterpret_cast<const char*>(reinterpret_cast<const T*>(e.R) + (int64_t)bz * e.sr +
                                          (int64_t)m * e.ldr + n);
      }
      dma16<2>(g, smem + part * S::V2_STAGE + (wave * (part ? S::STG_IB : S::STG_IA) + i) * 1024);
    }
  };
  auto vec_dma = [&]() {
    if constexpr (STG) {
      const RowEpi& e = p.epi;
      const float* v = wave == 0 ? e.bias : wave == 1 ? e.gamma : wave == 2 ? e.beta : nullptr;
      const char* g = reinterpret_cast<const char*>(X);
      if (v) g = reinterpret_cast<const char*>(v + min(n0 + 4 * lane, p.N - 4));
      dma16(g, smem + S::STG_RA * S::TN * 2 + wave * 1024);
    }
  };

  constexpr int KS = S::V2_TK / S::KSTEP;          // MFMA steps per stage
  constexpr int NMF = S::BN * S::BM;               // MFMAs per step
  const int lr = lane & 31, lg = lane >> 5, sw = (lr >> 1) & 7;
  u32x4_t fa[KS][S::BN], fb[KS][S::BM];
  // Fragment `idx` of MFMA step ks of stage st: idx < BN -> W^T block idx, else X block idx-BN.
  auto frag1 = [&](int st, int ks, int idx) {
    const int off = ((2 * ks + lg) ^ sw) << 4;
    if (idx < S::BN) {
      if constexpr (KN) {
        typedef short v4i16 __attribute__((ext_vector_type(4)));
        const int r = lane & 15;
        const int k = 16 * ks + 8 * lg + (r >> 2);
        const int nb = (wn * S::WTN + idx * 32 + (lane & 16) + 4 * (r & 3)) * 2;
        const char* a = slot(st) + k * KN_RW + (nb ^ ((r >> 2) << 6));
        const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)(a));
        const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) v4i16*)(a + 4 * KN_RW));
        const u32x2_t l2 = __builtin_bit_cast(u32x2_t, lo), h2 = __builtin_bit_cast(u32x2_t, hi);
        fa[ks][idx] = u32x4_t{l2[0], l2[1], h2[0], h2[1]};
      } else {
        fa[ks][idx] = lds_read16(slot(st) + (wn * S::WTN + idx * 32 + lr) * S::V2_ROWB + off);
      }
    } else
      fb[ks][idx - S::BN] = lds_read16(slot(st) + (S::TN + wm * S::WTM + (idx - S::BN) * 32 + lr) * S::V2_ROWB + off);
  };
  constexpr int NFR = S::BN + S::BM;               // fragments per step

  ring.prologue(smem, wave);
  wait_vmcnt<PW * (NS - 2)>();
  lds_barrier();
#pragma unroll
  for (int ks = 0; ks < KS - 1; ++ks)
#pragma unroll
    for (int f = 0; f < NFR; ++f) frag1(0, ks, f);

  // One iteration.  J < 0: steady state (loads stage kt+NS-1).  J = 0..NS-2:
  // the last NS-1 iterations (kt = KT-NS+1+J), which load the epilogue
  // operands instead (J = 0: residual part 0 and vectors, J = 1: part 1).
  // The instruction order is pinned (sched_barrier) because MFMAs, being pure
  // register operations, would otherwise drift across the LDS barrier.
  auto body = [&](int kt, auto j_t) {
    constexpr int J = decltype(j_t)::value;
    constexpr bool MORE = J < NS - 2;              // stage kt+1 exists
    constexpr int NL = J < 0 ? PW : !STG ? 0 : J == 0 ? S::STG_IA + 1 : J == 1 ? S::STG_IB : 0;
    // Loads this wave issued after stage kt+1's (the wait below allows them).
    constexpr int AFTER = J < 0 ? PW * (NS - 2)
                                : PW * (NS - 3 - J) + (!STG ? 0 : J == 0 ? S::STG_IA + 1 : S::STG_IA + 1 + S::STG_IB);
    constexpr int LPS = (NL + (KS - 1) * NMF - 1) / ((KS - 1) * NMF);   // loads per MFMA slot
    const int nxt = kt + NS - 1;
    auto load = [&](int l) {
      if constexpr (J < 0) dma(l, nxt);
      else if constexpr (J == 0) { if (l < S::STG_IA) stage_dma(0, l); else vec_dma(); }
      else stage_dma(1, l);
    };
    // Steps 0..KS-2; behind each of the first MFMAs one fragment read of the
    // last step (issued after an MFMA so that the MFMA's operands, read during
    // the previous iteration, need no wait on these) and LPS loads.
    constexpr int RPF = (NFR + NMF - 1) / NMF;               // last-step reads per MFMA slot
#pragma unroll
    for (int ks = 0; ks < KS - 1; ++ks)
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
        for (int bn = 0; bn < S::BN; ++bn) {
          Mma<T>::run(acc[bm][bn], fa[ks][bn], fb[ks][bm]);
          __builtin_amdgcn_sched_barrier(0);
          const int i = (ks * S::BM + bm) * S::BN + bn;
#pragma unroll
          for (int r = 0; r < RPF; ++r)
            if (i * RPF + r < NFR) frag1(kt, KS - 1, i * RPF + r);
#pragma unroll
          for (int r = 0; r < LPS; ++r)
            if (i * LPS + r < NL) load(i * LPS + r);
          __builtin_amdgcn_sched_barrier(0);
        }
    if constexpr (MORE) {
      static_assert(AFTER >= 0 && AFTER < 64, "vmcnt range");
      wait_vmcnt<AFTER>();
      __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (3 << 14));   // lgkmcnt(0); vmcnt, expcnt unconstrained
      lds_barrier();
      __builtin_amdgcn_sched_barrier(0);
    }
    // Last step; its MFMAs interleaved with the next stage's fragment reads.
    constexpr int RPM = ((KS - 1) * NFR + NMF - 1) / NMF;   // reads per MFMA
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn) {
        Mma<T>::run(acc[bm][bn], fa[KS - 1][bn], fb[KS - 1][bm]);
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (MORE) {
          const int i = bm * S::BN + bn;
#pragma unroll
          for (int r = 0; r < RPM; ++r) {
            const int fr = i * RPM + r;
            if (fr < (KS - 1) * NFR) frag1(kt + 1, fr / NFR, fr % NFR);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
  };
  int kt = 0;
  for (; kt < KT - (NS - 1); ++kt) body(kt, std::integral_constant<int, -1>{});
  static_assert(NS <= 5, "tail unrolled for at most 4 iterations");
  body(kt, std::integral_constant<int, 0>{});
  if constexpr (NS > 2) body(kt + 1, std::integral_constant<int, 1>{});
  if constexpr (NS > 3) body(kt + 2, std::integral_constant<int, 2>{});
  if constexpr (NS > 4) body(kt + 3, std::integral_constant<int, 3>{});
  wait_vmcnt<0>();
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Row reductions over the values a workgroup holds (levels 1 and 2).
// v[bm] is this lane's partial for row (wm*WTM + bm*32 + lane%32).
// ---------------------------------------------------------------------------
template <class S, bool MAX>
__device__ __forceinline__ void wg_row_reduce(float (&v)[S::BM], float* red, int lane,
                                              int wm, int wn) {
#pragma unroll
  for (int bm = 0; bm < S::BM; ++bm) {
    const float o = __shfl_xor(v[bm], 32);
    v[bm] = MAX ? fmaxf(v[bm], o) : v[bm] + o;
  }
  if constexpr (S::WN > 1) {
    const int lr = lane & 31;
    if (lane < 32) {
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) red[wn * S::TM + wm * S::WTM + bm * 32 + lr] = v[bm];
    }
    __syncthreads();
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      const int idx = wm * S::WTM + bm * 32 + lr;
      float t = red[idx];
#pragma unroll
      for (int w = 1; w < S::WN; ++w) t = MAX ? fmaxf(t, red[w * S::TM + idx]) : t + red[w * S::TM + idx];
      v[bm] = t;
    }
    __syncthreads();
  }
}

// Pairwise update of (count, mean, M2) of two disjoint sets (Chan, Golub and
// LeVeque): d = mean_b - mean_a, mean = mean_a + d n_b / n, M2 = M2_a + M2_b
// + d^2 n_a n_b / n.  An empty side leaves the other unchanged.
__device__ __forceinline__ void chan_merge(float& n, float& mean, float& m2, float nb, float mb, float m2b) {
  const float nn = n + nb;
  if (nn > 0.0f) {
    const float f = nb * __builtin_amdgcn_rcpf(nn), d = mb - mean;
    mean = fmaf(d, f, mean);
    m2 = m2 + m2b + d * d * (n * f);
    n = nn;
  }
}

// Levels 1 and 2 of the statistics reduction for (count, mean, M2) per row:
// each lane holds its own row's partial statistics; the two lanes of a row
// (l, l ^ 32) merge, then the WN waves sharing the row merge through LDS.
// Every merge takes the parts in a fixed order (lane half 0 first, then wave
// columns 0, 1, ...), so every lane of the row ends with identical values.
template <class S>
__device__ __forceinline__ void wg_stat_reduce(float (&n)[S::BM], float (&mean)[S::BM], float (&m2)[S::BM],
                                               float* red, int lane, int wm, int wn) {
  const int lg = lane >> 5;
#pragma unroll
  for (int bm = 0; bm < S::BM; ++bm) {
    const float on = __shfl_xor(n[bm], 32), om = __shfl_xor(mean[bm], 32), o2 = __shfl_xor(m2[bm], 32);
    float an = lg ? on : n[bm], am = lg ? om : mean[bm], a2 = lg ? o2 : m2[bm];
    chan_merge(an, am, a2, lg ? n[bm] : on, lg ? mean[bm] : om, lg ? m2[bm] : o2);
    n[bm] = an;
    mean[bm] = am;
    m2[bm] = a2;
  }
  if constexpr (S::WN > 1) {
    const int lr = lane & 31;
    if (lane < 32) {
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) {
        float* d = red + (wn * S::TM + wm * S::WTM + bm * 32 + lr) * 3;
        d[0] = n[bm];
        d[1] = mean[bm];
        d[2] = m2[bm];
      }
    }
    __syncthreads();
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      const int idx = wm * S::WTM + bm * 32 + lr;
      float an = red[idx * 3], am = red[idx * 3 + 1], a2 = red[idx * 3 + 2];
#pragma unroll
      for (int w = 1; w < S::WN; ++w) {
        const float* q = red + (w * S::TM + idx) * 3;
        chan_merge(an, am, a2, q[0], q[1], q[2]);
      }
      n[bm] = an;
      mean[bm] = am;
      m2[bm] = a2;
    }
    __syncthreads();
  }
}

// Level 3, ROWS_CLUSTER: the cn workgroups of a row block exchange per-row
// partials through records in the workspace header.
//
// Rounds.  One wave of every workgroup adds kArriveUnit / cn to its peer
// group's counter once per tile (round_begin), so a round adds exactly
// kArriveUnit and old / kArriveUnit numbers the round, identically in every
// workgroup of the group.  The add goes out after the main loop (the loop's
// waits count memory operations in issue order); the adding wave waits for
// its return and leaves the round number in LDS before the workgroup's first
// epilogue barrier (the other waves read it after that barrier).  So all adds
// of a round have landed before any record of the round can be seen, and the
// next round's adds see the next round number.  One add per workgroup rather
// than per wave: adds to one address are serialised, and sixteen of them per
// round were measured at about 2 us.
//
// Records.  record(stage, parity, slot, peer, row) holds one or two 64-bit
// words, each a 32-bit value with the round number + 1 in its upper half.  A
// word is written and read with single 64-bit device-coherent atomics
// (relaxed, agent scope; on gfx950 these bypass the non-coherent caches), so
// a reader that sees the current round in a word also sees that round's
// value: no fence, no completion wait on the writer and no separate arrival
// flag.  Only this path writes the records and a slot's round numbers only
// grow, so a stale or zero-filled record never carries the current tag.
// Rounds of odd and even number use separate record sets, so a peer that
// runs one round ahead never overwrites a record another peer still waits
// for.  Agent-scope release / acquire fences are avoided on purpose: on
// gfx950 they write back and invalidate the whole L2, evicting the operands
// of every workgroup sharing it.
//
// Failure.  A wait that exceeds p.spin_limit polls sets the sticky error word
// and moves on; every later wait sees the word and gives up at once, so a
// broken launch ends quickly.  The host reads and clears the word
// (cf_workspace_check); results of a call that set it are invalid.
// The group's add for this workgroup (lane 0 of wave 0; 0 elsewhere).
__device__ __forceinline__ unsigned long long round_begin(const GemmRowsParams& p, int slot, int lane, int wave) {
  unsigned long long old = 0;
  if (wave == 0 && lane == 0)
    old = __hip_atomic_fetch_add(p.ws_arrive + slot, kArriveUnit / (unsigned long long)p.cn, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
  return old;
}

// Tag of the round whose counter value `old` the adding lane received.
__device__ __forceinline__ unsigned round_tag(unsigned long long old) {
  return (unsigned)(old / kArriveUnit) + 1u;
}

__device__ __forceinline__ unsigned long long rec_word(float v, unsigned tag) {
  return ((unsigned long long)tag << 32) | __float_as_uint(v);
}

// How cluster_exchange merges the peers' per-row values.
enum MergeKind {
  MERGE_CHAN = 0,      // (a, b) = (mean, M2) of TN columns: pairwise update (Chan, Golub, LeVeque)
  MERGE_MAX = 1,       // a = max over peers
  MERGE_SOFTMAX = 2    // (a, b) = (max, sum of exp(x - max)): b rescaled to the common max
};

// Publishes (a, b) (MERGE_MAX: a only) of this workgroup's rows, then reads
// every peer's records of the lane's rows, peer 0 first, until all carry
// `tag`, and merges them in that order.  Every workgroup merges in the same
// order, so all get bit-identical values.  With p.leader (many peers, the
// dual-mode aggregation of Sec. III-A) only peer 0 reads and merges all
// records; it publishes the merged values in record kRecLead, which the
// other peers read instead.
template <class S, int MERGE>
__device__ __forceinline__ void cluster_exchange(const GemmRowsParams& p, int stage, int slot, int c, unsigned tag,
                                                 float (&a)[S::BM], float (&b)[S::BM], int lane, int wm, int wn) {
  static_assert(S::TM <= kRecRows, "records hold kRecRows rows per peer");
  constexpr bool MAX = MERGE == MERGE_MAX;
  constexpr int NV = MAX ? 1 : 2;
  constexpr int PB = 4;   // peers read per batch
  unsigned long long* rec = reinterpret_cast<unsigned long long*>(p.ws_part) + stage * kRecStageWords +
                            (tag & 1u) * kRecSetWords + (size_t)slot * kRecPeers * kRecRows * 2;
  const int lr = lane & 31;
  if (wn == 0 && lane < 32) {
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      unsigned long long* w = rec + ((size_t)c * kRecRows + wm * S::WTM + bm * 32 + lr) * 2;
      __hip_atomic_store(w, rec_word(a[bm], tag), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      if (!MAX) __hip_atomic_store(w + 1, rec_word(b[bm], tag), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
  }
  const int cn = p.cn;
  if (p.leader && c != 0) {
    // Leader-follower (for many peers): peer 0 merges every record and
    // publishes the result; the others read that one record only.
    unsigned long long w[S::BM][NV];
    for (int spins = 0;; ++spins) {
      const unsigned err = __hip_atomic_load(p.ws_err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      bool ok = true;
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) {
        const unsigned long long* r = rec + ((size_t)kRecLead * kRecRows + wm * S::WTM + bm * 32 + lr) * 2;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          w[bm][v] = __builtin_nontemporal_load(r + v);
          ok = ok && (unsigned)(w[bm][v] >> 32) == tag;
        }
      }
      if (__all(ok)) break;
      if (__builtin_amdgcn_readfirstlane(err) != 0u) break;
      if (spins >= p.spin_limit) {
        __hip_atomic_store(p.ws_err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      a[bm] = __uint_as_float((unsigned)w[bm][0]);
      if (!MAX) b[bm] = __uint_as_float((unsigned)w[bm][NV - 1]);
    }
    return;
  }
  float n_acc[S::BM], mu[S::BM], sq[S::BM];
#pragma unroll
  for (int bm = 0; bm < S::BM; ++bm) {
    n_acc[bm] = mu[bm] = sq[bm] = 0.0f;
    if (MERGE == MERGE_SOFTMAX) mu[bm] = -INFINITY;
  }
  for (int c0 = 0; c0 < cn; c0 += PB) {
    unsigned long long w[S::BM][PB][NV];
    for (int spins = 0;; ++spins) {
      // the sticky error word rides along with every poll
      const unsigned err = __hip_atomic_load(p.ws_err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      bool ok = true;
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
        for (int j = 0; j < PB; ++j) {
          const int cc = c0 + j < cn ? c0 + j : cn - 1;
          const unsigned long long* r = rec + ((size_t)cc * kRecRows + wm * S::WTM + bm * 32 + lr) * 2;
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            w[bm][j][v] = __builtin_nontemporal_load(r + v);
            ok = ok && (unsigned)(w[bm][j][v] >> 32) == tag;
          }
        }
      if (__all(ok)) break;
      if (__builtin_amdgcn_readfirstlane(err) != 0u) break;   // an earlier wait failed: give up now
      if (spins >= p.spin_limit) {
        __hip_atomic_store(p.ws_err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
      for (int j = 0; j < PB; ++j) {
        if (c0 + j >= cn) break;
        const float va = __uint_as_float((unsigned)w[bm][j][0]);
        if constexpr (MAX) {
          mu[bm] = fmaxf(mu[bm], va);
        } else if constexpr (MERGE == MERGE_SOFTMAX) {
          // sum_c s_c exp(m_c - m) with m the running maximum; exp2 of a
          // non-positive argument (exp2(-inf) = 0 for the first record)
          const float vb = __uint_as_float((unsigned)w[bm][j][NV - 1]);
          const float mn = fmaxf(mu[bm], va);
          sq[bm] = sq[bm] * __builtin_amdgcn_exp2f((mu[bm] - mn) * 1.4426950408889634f) +
                   vb * __builtin_amdgcn_exp2f((va - mn) * 1.4426950408889634f);
          mu[bm] = mn;
        } else {
          // every peer holds TN columns: merging peer k (k peers merged
          // before) weighs its mean by 1 / (k + 1) and the squared
          // difference by TN k / (k + 1)
          const float vb = __uint_as_float((unsigned)w[bm][j][NV - 1]);
          const float k = n_acc[bm], f = __builtin_amdgcn_rcpf(k + 1.0f);
          const float d = va - mu[bm];
          mu[bm] = fmaf(d, f, mu[bm]);
          sq[bm] += vb + d * d * ((float)S::TN * k * f);
          n_acc[bm] = k + 1.0f;
        }
      }
  }
#pragma unroll
  for (int bm = 0; bm < S::BM; ++bm) {
    a[bm] = mu[bm];
    if (!MAX) b[bm] = sq[bm];
  }
  if (p.leader && wn == 0 && lane < 32) {   // the leader broadcasts the merged values
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      unsigned long long* w = rec + ((size_t)kRecLead * kRecRows + wm * S::WTM + bm * 32 + lr) * 2;
      __hip_atomic_store(w, rec_word(a[bm], tag), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      if (!MAX) __hip_atomic_store(w + 1, rec_word(b[bm], tag), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
  }
}

// ---------------------------------------------------------------------------
// Output tile store through LDS.  The accumulator layout gives each lane 4
// consecutive columns of 32 different rows, which as direct global stores
// leaves 16-byte pieces in many cache lines (and roughly doubles HBM write
// traffic for bf16).  Instead the tile is written to LDS in row-major order
// (row pitch padded by 8 or 16 bytes so the 32 rows of one write hit
// different banks), then stored as coalesced 16-byte chunks, consecutive
// lanes covering consecutive bytes of a row.  Columns >= N and rows >= M are
// not stored.  Needs TM * (TN * esz + pad) bytes of LDS; callers reach it
// after the main loop's final barrier.
// ---------------------------------------------------------------------------
template <class S, int ESZ>
__device__ __forceinline__ void store_tile_staged_t(const f32x16_t (&x)[S::BM][S::BN], void* Ybase, int64_t ldy,
                                                    int M, int N, int m0, int n0, char* smem, int tid, int lane,
                                                    int wm, int wn) {
  const int lr = lane & 31, lg = lane >> 5;
  constexpr int PITCH = S::TN * ESZ + (ESZ == 4 ? 16 : 8);
#pragma unroll
  for (int bm = 0; bm < S::BM; ++bm) {
    const int r = wm * S::WTM + bm * 32 + lr;
#pragma unroll
    for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int cidx = wn * S::WTN + bn * 32 + 8 * g + 4 * lg;
        char* dst = smem + r * PITCH + cidx * ESZ;
        if constexpr (ESZ == 4) {
          f32x4_t o = {x[bm][bn][4 * g], x[bm][bn][4 * g + 1], x[bm][bn][4 * g + 2], x[bm][bn][4 * g + 3]};
          *reinterpret_cast<f32x4_t*>(dst) = o;
        } else {
          u32x2_t o = {pack_bf16x2(x[bm][bn][4 * g], x[bm][bn][4 * g + 1]),
                       pack_bf16x2(x[bm][bn][4 * g + 2], x[bm][bn][4 * g + 3])};
          *reinterpret_cast<u32x2_t*>(dst) = o;
        }
      }
  }
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (3 << 14));   // lgkmcnt(0): this wave's LDS writes are done
  lds_barrier();
  constexpr int CPR = S::TN * ESZ / 16;   // 16-byte chunks per tile row
  constexpr int EPC = 16 / ESZ;           // elements per chunk
  constexpr int TOTAL = S::TM * CPR;
  constexpr int ITER = (TOTAL + S::NT - 1) / S::NT;
  constexpr int BATCH = ITER < 8 ? ITER : 8;   // LDS reads in flight before their stores
  // Addresses are 32-bit offsets from the tile origin (the host keeps
  // TM * ldy * ESZ below 2^31).
  char* yb = reinterpret_cast<char*>(Ybase) + ((int64_t)m0 * ldy + n0) * ESZ;
  const int ldyb = (int)ldy * ESZ;
  const bool full = m0 + S::TM <= M && n0 + S::TN <= N;
  const int rows = M - m0, cols = N - n0;
#pragma unroll
  for (int j0 = 0; j0 < ITER; j0 += BATCH) {
    u32x4_t v[BATCH];
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      const int id = tid + (j0 + j) * S::NT;
      if (j0 + j < ITER && (TOTAL % S::NT == 0 || id < TOTAL))
        v[j] = *reinterpret_cast<const u32x4_t*>(smem + (id / CPR) * PITCH + (id % CPR) * 16);
    }
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      const int id = tid + (j0 + j) * S::NT;
      const int r = id / CPR, cc = id % CPR;
      if (j0 + j < ITER && (TOTAL % S::NT == 0 || id < TOTAL) && (full || (r < rows && cc * EPC < cols)))
        __builtin_nontemporal_store(v[j], reinterpret_cast<u32x4_t*>(yb + (unsigned)(r * ldyb + cc * 16)));
    }
  }
  // The staging area is reused by the next reduction: every lane has read
  // its chunks (the stores consumed them), so a bare barrier suffices and the
  // global stores drain while the workgroup goes on.
  lds_barrier();
}

template <class S>
__device__ __forceinline__ void store_tile_staged(const f32x16_t (&x)[S::BM][S::BN], void* Ybase, int64_t ldy,
                                                  int y_f32, int M, int N, int m0, int n0, char* smem,
                                                  int tid, int lane, int wm, int wn) {
  if (y_f32) store_tile_staged_t<S, 4>(x, Ybase, ldy, M, N, m0, n0, smem, tid, lane, wm, wn);
  else store_tile_staged_t<S, 2>(x, Ybase, ldy, M, N, m0, n0, smem, tid, lane, wm, wn);
}

// ---------------------------------------------------------------------------
// Epilogue operands fetched BEFORE the main loop: the residual tile (in the
// accumulator layout) and the bias.  Their load latency then overlaps the
// pipeline fill instead of stalling the epilogue (the bypass operands of the
// Stage-Stream chain are ready when the accumulator tile is).
// ---------------------------------------------------------------------------
template <class S>
struct EpiPrefetch {
  using RVec = typename std::conditional<sizeof(typename S::T) == 2, u32x2_t, u32x4_t>::type;
  // The residual is prefetched when its registers fit (bf16, or small fp32 tiles).
  static constexpr bool PF_R = sizeof(typename S::T) == 2 || S::BM * S::BN <= 4;
  RVec r[PF_R ? S::BM : 1][PF_R ? S::BN : 1][4];   // 4 consecutive residual elements per (bm, bn, g)
  f32x4_t b[S::BN][4];                             // bias for the 4 columns of (bn, g)
};

template <class S>
__device__ __forceinline__ void epi_prefetch(EpiPrefetch<S>& pf, const GemmRowsParams& p, int m0, int n0,
                                             int bz, int lane, int wm, int wn) {
  using T = typename S::T;
  using RVec = typename EpiPrefetch<S>::RVec;
  const RowEpi& e = p.epi;
  const int lr = lane & 31, lg = lane >> 5;
  const T* R = reinterpret_cast<const T*>(e.R) + (int64_t)bz * e.sr;
#pragma unroll
  for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int n = n0 + wn * S::WTN + bn * 32 + 8 * g + 4 * lg;
      const bool nv = n < p.N;
      pf.b[bn][g] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
      if (e.bias && e.alpha != 1.0f && nv) pf.b[bn][g] = *reinterpret_cast<const f32x4_t*>(e.bias + n);
      if constexpr (EpiPrefetch<S>::PF_R) {
#pragma unroll
        for (int bm = 0; bm < S::BM; ++bm) {
          const int m = m0 + wm * S::WTM + bm * 32 + lr;
          pf.r[bm][bn][g] = RVec{};
          if (e.R && nv && m < p.M) pf.r[bm][bn][g] = *reinterpret_cast<const RVec*>(R + (int64_t)m * e.ldr + n);
        }
      }
    }
}

// ---------------------------------------------------------------------------
// Epilogue on the register tile.
// ---------------------------------------------------------------------------
// STG: the residual tile and the vectors were staged in LDS by the main loop
// (slots 0 and 1); otherwise they come from `pf` or straight from memory.
// SPLIT: the split-N GEMM pass; stage 1, then publish fp32 x and the tile's
// (mean, M2) for the finish pass (nothing else is compiled in).
template <class S, bool STG, bool SPLIT>
__device__ __forceinline__ void epilogue(f32x16_t (&x)[S::BM][S::BN], const EpiPrefetch<S>& pf,
                                         const GemmRowsParams& p, int m0, int n0, int slot, int c,
                                         unsigned long long round_old, int bz, char* smem, float* red, int tid,
                                         int lane, int wm, int wn) {
  using T = typename S::T;
  const RowEpi& e = p.epi;
  const int M = p.M, N = p.N;
  const int lr = lane & 31, lg = lane >> 5;
  // The round tag (row clusters): the adding lane leaves it in LDS before the
  // workgroup's first barrier (the round protocol needs the add returned by
  // then; the work before that barrier covers its round trip), and every wave
  // reads it after that barrier.
  unsigned* tag_lds = reinterpret_cast<unsigned*>(red) + S::RED_BYTES / 4;
  bool tag_sent = false;
  auto send_tag = [&] {
    if (!tag_sent) {
      if (wm == 0 && wn == 0 && lane == 0) *tag_lds = round_tag(round_old);
      tag_sent = true;
    }
  };
  auto tag = [&] { return __builtin_amdgcn_readfirstlane(*tag_lds); };
  // Staged vector v (0 bias, 1 gamma, 2 beta) at tile column cl.
  auto vec_lds = [&](int v, int cl) {
    return *reinterpret_cast<const f32x4_t*>(smem + S::STG_RA * S::TN * 2 + v * 1024 + cl * 4);
  };
  auto col_l = [&](int bn, int g) { return wn * S::WTN + bn * 32 + 8 * g + 4 * lg; };

  int mrow[S::BM];
  bool mval[S::BM];
#pragma unroll
  for (int bm = 0; bm < S::BM; ++bm) {
    mrow[bm] = m0 + wm * S::WTM + bm * 32 + lr;
    mval[bm] = mrow[bm] < M;
  }
  auto ncol = [&](int bn, int g) { return n0 + wn * S::WTN + bn * 32 + 8 * g + 4 * lg; };

  // ---- stage 1: x = alpha * acc + bias + R (columns >= N stay exactly 0)
  const float alpha = e.alpha;
  if (alpha != 1.0f) {
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int i = 0; i < 16; ++i) x[bm][bn][i] *= alpha;
  }
  // LDS operands are read a block at a time, all reads issued before the
  // first use (sched_barrier), so their latencies overlap.
  // Only given terms are added (x + 0 would turn -0 into +0).  With alpha = 1
  // the accumulators started from the bias.
  if (e.bias && alpha != 1.0f) {
#pragma unroll
    for (int bn = 0; bn < S::BN; ++bn) {
      f32x4_t bv[4];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        if constexpr (STG) bv[g] = vec_lds(0, col_l(bn, g));
        else bv[g] = pf.b[bn][g];
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
          for (int q = 0; q < 4; ++q) x[bm][bn][4 * g + q] += bv[g][q];
    }
  }
  if constexpr (STG) if (e.R) {
    // The residual by two MFMAs per 32 x 32 block with an identity operand:
    // D[n][m] += sum_k I[n][k] R[m][16h + k] adds R[m][n] for n in
    // [16h, 16h + 16) exactly (one non-zero product, rounded once into the
    // accumulator like a VALU add).  Lane l supplies the identity row n = l % 32
    // at k = 8 (l / 32) .. + 7 and, as the B operand, 8 consecutive residual
    // values of its row: the 16-byte chunk 2h + l / 32 of the block's 32
    // columns, which the staged layout keeps at chunk position c ^ (r & 7).
    u32x4_t eye[2];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int e0 = lr - 16 * h - 8 * lg - 2 * w;   // one-hot position relative to this dword
        eye[h][w] = (e0 == 0 ? 0x3F80u : 0u) | (e0 == 1 ? 0x3F800000u : 0u);
      }
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      const int r = wm * S::WTM + bm * 32 + lr;
      const char* rowp = r < S::STG_RA ? smem + r * S::TN * 2 : smem + S::V2_STAGE + (r - S::STG_RA) * S::TN * 2;
      u32x4_t rv[S::BN][2];
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int cc = (wn * S::WTN + bn * 32) / 8 + 2 * h + lg;
          rv[bn][h] = lds_read16(rowp + ((cc ^ (r & 7)) << 4));
        }
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int h = 0; h < 2; ++h) Mma<T>::run(x[bm][bn], eye[h], rv[bn][h]);
    }
  }
  if (!STG && e.R && !EpiPrefetch<S>::PF_R) {
    const T* R = reinterpret_cast<const T*>(e.R) + (int64_t)bz * e.sr;
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      if (!mval[bm]) continue;
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = ncol(bn, g);
          if (n < N) {
            float r[4];
            load4<T>(R + (int64_t)mrow[bm] * e.ldr + n, r);
#pragma unroll
            for (int q = 0; q < 4; ++q) x[bm][bn][4 * g + q] += r[q];
          }
        }
    }
  }
  if constexpr (!STG && EpiPrefetch<S>::PF_R) if (e.R) {
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          if constexpr (sizeof(T) == 2) {
            const u32x2_t u = pf.r[bm][bn][g];
            x[bm][bn][4 * g + 0] += bf16_to_f32(u[0] & 0xFFFFu);
            x[bm][bn][4 * g + 1] += bf16_to_f32(u[0] >> 16);
            x[bm][bn][4 * g + 2] += bf16_to_f32(u[1] & 0xFFFFu);
            x[bm][bn][4 * g + 3] += bf16_to_f32(u[1] >> 16);
          } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) x[bm][bn][4 * g + q] += __uint_as_float(pf.r[bm][bn][g][q]);
          }
        }
  }

  if (n0 + S::TN > N) {   // clamped or zero-filled columns past N contribute nothing
#pragma unroll
    for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        if (ncol(bn, g) >= N)
#pragma unroll
          for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
            for (int q = 0; q < 4; ++q) x[bm][bn][4 * g + q] = 0.0f;
  }

  bool exchanged = false;

  // ---- stage 2: row statistics and the normalising PostOp
  if (SPLIT || e.norm == NORM_LAYER) {
    // Per lane, two passes over its values of each row (sum, then squared
    // deviations from the lane's own mean), then the merges of
    // wg_stat_reduce: (mean, M2) of the tile's valid columns of every row.
    float cnt[S::BM], mean[S::BM], m2[S::BM];
    auto lane_stats = [&](auto ragged_t) {
      constexpr bool RAGGED = decltype(ragged_t)::value;
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) {
        float t = 0.0f, nl = 0.0f;
#pragma unroll
        for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            if (RAGGED && ncol(bn, g) >= N) continue;
            nl += 4.0f;
#pragma unroll
            for (int q = 0; q < 4; ++q) t += x[bm][bn][4 * g + q];
          }
        const float mu = RAGGED ? (nl > 0.0f ? t / nl : 0.0f) : t * (1.0f / (16 * S::BN));
        float d2 = 0.0f;
#pragma unroll
        for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            if (RAGGED && ncol(bn, g) >= N) continue;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const float d = x[bm][bn][4 * g + q] - mu;
              d2 = fmaf(d, d, d2);
            }
          }
        cnt[bm] = RAGGED ? nl : (float)(16 * S::BN);
        mean[bm] = mu;
        m2[bm] = d2;
      }
    };
    if (n0 + S::TN <= N) lane_stats(std::false_type{});
    else lane_stats(std::true_type{});
    send_tag();
    wg_stat_reduce<S>(cnt, mean, m2, red, lane, wm, wn);

    if constexpr (SPLIT) {
      // Publish the tile's (mean, M2) and fp32 x (coalesced through LDS); the
      // finish pass does the rest.
      if (wn == 0 && lane < 32) {
#pragma unroll
        for (int bm = 0; bm < S::BM; ++bm)
          if (mval[bm])
            reinterpret_cast<float2*>(p.ws_part)[(int64_t)mrow[bm] * p.cn + c] = make_float2(mean[bm], m2[bm]);
      }
      store_tile_staged<S>(x, p.ws_x, N, 1, M, N, m0, n0, smem, tid, lane, wm, wn);
      return;
    }

    if (p.mode == ROWS_CLUSTER && p.cn > 1) {
      cluster_exchange<S, MERGE_CHAN>(p, 0, slot, c, tag(), mean, m2, lane, wm, wn);
      exchanged = true;
    }

    if (e.norm == NORM_LAYER) {
      const float invN = 1.0f / (float)N;
      // y = (x - mean) * rstd (a constant row gives exactly 0), then
      // y * gamma + beta when either is given.
      float rstd[S::BM];
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) rstd[bm] = rsqrtf(m2[bm] * invN + e.eps);
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
        for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
          for (int i = 0; i < 16; ++i) x[bm][bn][i] = (x[bm][bn][i] - mean[bm]) * rstd[bm];
      if (e.gamma || e.beta) {
#pragma unroll
        for (int bn = 0; bn < S::BN; ++bn) {
          f32x4_t ga[4], be[4];
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int n = min(ncol(bn, g), N - 4);   // padding columns are never stored
            ga[g] = f32x4_t{1.0f, 1.0f, 1.0f, 1.0f};
            be[g] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
            if constexpr (STG) {
              if (e.gamma) ga[g] = vec_lds(1, col_l(bn, g));
              if (e.beta) be[g] = vec_lds(2, col_l(bn, g));
            } else {
              if (e.gamma) ga[g] = *reinterpret_cast<const f32x4_t*>(e.gamma + n);
              if (e.beta) be[g] = *reinterpret_cast<const f32x4_t*>(e.beta + n);
            }
          }
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
              for (int q = 0; q < 4; ++q)
                x[bm][bn][4 * g + q] = fmaf(x[bm][bn][4 * g + q], ga[g][q], be[g][q]);
        }
      }
    }
  } else if (e.norm == NORM_RMS) {
    float s[S::BM];
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      float t = 0.0f;
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int i = 0; i < 16; ++i) t += x[bm][bn][i] * x[bm][bn][i];
      s[bm] = t;
    }
    send_tag();
    wg_row_reduce<S, false>(s, red, lane, wm, wn);
    if (p.mode == ROWS_CLUSTER && p.cn > 1) {
      // sum of squares: a merge of (mean, M2) pairs (0, s) keeps M2 = sum of s
      float z[S::BM];
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) z[bm] = 0.0f;
      cluster_exchange<S, MERGE_CHAN>(p, 0, slot, c, tag(), z, s, lane, wm, wn);
      exchanged = true;
    }
    const float invN = 1.0f / (float)N;
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) s[bm] = rsqrtf(s[bm] * invN + e.eps);
#pragma unroll
    for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = ncol(bn, g);
        f32x4_t ga = {1.0f, 1.0f, 1.0f, 1.0f};
        if (n < N && e.gamma) ga = STG ? vec_lds(1, col_l(bn, g)) : *reinterpret_cast<const f32x4_t*>(e.gamma + n);
#pragma unroll
        for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
          for (int q = 0; q < 4; ++q) x[bm][bn][4 * g + q] = x[bm][bn][4 * g + q] * s[bm] * ga[q];
      }
  }

  // ---- stage 3: activation and store
  // One straight loop per activation kind (the kind is uniform): a per-element
  // switch would put every kind's code on the path of every element.
  auto act_all = [&](auto f) {   // one 16-value block at a time (bounds the live temporaries)
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn) {
#pragma unroll
        for (int i = 0; i < 16; ++i) x[bm][bn][i] = f(x[bm][bn][i]);
        __builtin_amdgcn_sched_barrier(0);
      }
  };
  switch (e.act) {
    case ACT_GELU: act_all([](float v) { return gelu_erf(v); }); break;
    case ACT_GELU_TANH: act_all([](float v) { return gelu_tanh(v); }); break;
    case ACT_RELU: act_all([](float v) { return v > 0.0f ? v : 0.0f; }); break;
    case ACT_SOFTCAP: {
      const float cap = e.softcap, inv = 1.0f / cap;
      act_all([=](float v) { return cap * tanh_exp(v * inv); });
      break;
    }
    default: break;
  }
  // ---- stage 3b: row softmax.  Local row maximum, e = exp(x - max_local) and
  // its sum; across workgroups the (max, sum) pairs merge with the sums
  // rescaled to the common maximum (one exchange); then x = e * exp(max_local
  // - max) / sum.  Padding columns of a ragged tile take no part.
  if (e.softmax) {
    const bool full_n = n0 + S::TN <= N;
    float mx[S::BM], sm[S::BM];
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      float t = -INFINITY;
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int g = 0; g < 4; ++g)
          if (full_n || ncol(bn, g) < N)
#pragma unroll
            for (int q = 0; q < 4; ++q) t = fmaxf(t, x[bm][bn][4 * g + q]);
      mx[bm] = t;
    }
    send_tag();
    wg_row_reduce<S, true>(mx, red, lane, wm, wn);
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      const float nl = -mx[bm] * 1.4426950408889634f;
      float t = 0.0f;
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const bool v = full_n || ncol(bn, g) < N;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float ev = v ? __builtin_amdgcn_exp2f(fmaf(x[bm][bn][4 * g + q], 1.4426950408889634f, nl)) : 0.0f;
            x[bm][bn][4 * g + q] = ev;
            t += ev;
          }
        }
      sm[bm] = t;
    }
    wg_row_reduce<S, false>(sm, red, lane, wm, wn);
    float f[S::BM];
    if (p.mode == ROWS_CLUSTER && p.cn > 1) {
      float mg[S::BM];
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) mg[bm] = mx[bm];
      cluster_exchange<S, MERGE_SOFTMAX>(p, 0, slot, c, tag(), mg, sm, lane, wm, wn);
      exchanged = true;
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm)
        f[bm] = __builtin_amdgcn_exp2f((mx[bm] - mg[bm]) * 1.4426950408889634f) / sm[bm];
    } else {
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) f[bm] = 1.0f / sm[bm];
    }
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int i = 0; i < 16; ++i) x[bm][bn][i] *= f[bm];
  }
  if (e.Y) {
    char* Yb = reinterpret_cast<char*>(e.Y) + (int64_t)bz * e.sy * (e.y_f32 ? 4 : 2);
    send_tag();
    if constexpr (STG) __syncthreads();   // staged vectors are no longer read
    store_tile_staged<S>(x, Yb, e.ldy, e.y_f32, M, N, m0, n0, smem, tid, lane, wm, wn);
  }

  // ---- stage 4: row amax -> scale -> E4M3 codes
  if (e.quant) {
    float a[S::BM];
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      float t = 0.0f;
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int g = 0; g < 4; ++g)
          if (ncol(bn, g) < N)   // padding columns of a ragged tile are not zero after the PostOps
#pragma unroll
            for (int q = 0; q < 4; ++q) t = fmaxf(t, fabsf(x[bm][bn][4 * g + q]));
      a[bm] = t;
    }
    send_tag();
    wg_row_reduce<S, true>(a, red, lane, wm, wn);
    if (p.mode == ROWS_CLUSTER && p.cn > 1) {
      cluster_exchange<S, MERGE_MAX>(p, exchanged ? 1 : 0, slot, c, tag(), a, a, lane, wm, wn);
      exchanged = true;
    }
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      if (!mval[bm]) continue;
      const float sc = a[bm] / e.qmax;
      if (c == 0 && wn == 0 && lane < 32 && e.s_out) e.s_out[mrow[bm]] = sc;
      if (e.q_out) {
        // codes of fl32(z / s); a zero row (s = 0) gives codes 0
        const bool nz = sc > 0.0f;
        const float sd = nz ? sc : 1.0f, inv = nz ? 1.0f / sc : 1.0f;
#pragma unroll
        for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int n = ncol(bn, g);
            if (n < N) {
              const uint32_t w =
                  e4m3x4(div_rn(x[bm][bn][4 * g], sd, inv), div_rn(x[bm][bn][4 * g + 1], sd, inv),
                         div_rn(x[bm][bn][4 * g + 2], sd, inv), div_rn(x[bm][bn][4 * g + 3], sd, inv));
              *reinterpret_cast<uint32_t*>(e.q_out + (int64_t)mrow[bm] * e.ldq + n) = nz ? w : 0u;
            }
          }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Plain epilogue: C = alpha * acc + bias, stored (bf16 or fp32).
// ---------------------------------------------------------------------------
template <class S>
__device__ __forceinline__ void epilogue_plain(f32x16_t (&x)[S::BM][S::BN], const GemmRowsParams& p,
                                               int m0, int n0, int bz, char* smem, int tid, int lane,
                                               int wm, int wn) {
  const RowEpi& e = p.epi;
  const int lg = lane >> 5;
  if (e.alpha != 1.0f) {
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int i = 0; i < 16; ++i) x[bm][bn][i] *= e.alpha;
  }
  // only a given bias is added (x + 0 would turn -0 into +0); with alpha = 1
  // the accumulators started from it
  if (e.bias && e.alpha != 1.0f) {
#pragma unroll
    for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n0 + wn * S::WTN + bn * 32 + 8 * g + 4 * lg;
        if (n >= p.N) continue;
        const f32x4_t b = *reinterpret_cast<const f32x4_t*>(e.bias + n);
#pragma unroll
        for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
          for (int q = 0; q < 4; ++q) x[bm][bn][4 * g + q] += b[q];
      }
  }
  char* Yb = reinterpret_cast<char*>(e.Y) + (int64_t)bz * e.sy * (e.y_f32 ? 4 : 2);
  store_tile_staged<S>(x, Yb, e.ldy, e.y_f32, p.M, p.N, m0, n0, smem, tid, lane, wm, wn);
}

// LOOP: 0 = register-staged main loop (any layout, ragged K),
//       1 = direct-to-LDS pipeline (W stored N x K, K a multiple of the stage),
//       2 = the same pipeline for bf16 W stored K x N (N a multiple of 8).
// EPI:  0 = plain epilogue (alpha, bias, store), 1 = row-subgraph epilogue
//       (whole rows or row clusters), 2 = the split-N GEMM pass.
// PERSIST: workgroups loop over row-block slots (the row-cluster path when
//       the co-resident grid is smaller than the tile count).  Otherwise each
//       workgroup runs one tile and there is no tile loop, so the compiler
//       has no loop to hoist the epilogue's setup out of: hoisted, that setup
//       ran before the first operand load and was parked in AGPRs and spilled
//       SGPR lanes until the epilogue (measured at the BERT-base post-norm
//       shape: 22.3 us with the loop against 21.0 us without).
template <class S, int LOOP, int EPI, bool PERSIST = false>
__global__ __launch_bounds__(S::NT, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gemm_rows_kernel(GemmRowsParams p) {
  using T = typename S::T;
  constexpr int SMEM = LOOP ? S::SMEM_V2 : S::SMEM_V1;
  constexpr bool STG = LOOP >= 1 && EPI >= 1 && S::STG;   // epilogue operands staged by the main loop
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  float* red = reinterpret_cast<float*>(smem + SMEM - S::TAIL_BYTES);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / S::WN, wn = wave % S::WN;
  const int bz = blockIdx.y;
  const T* X = reinterpret_cast<const T*>(p.X) + (int64_t)bz * p.sx;
  const T* W = reinterpret_cast<const T*>(p.W) + (int64_t)bz * p.sw;
  // blockIdx.x -> (XCD, slot, peer).  Consecutive block ids go round-robin
  // over the 8 XCDs, so the cn peers of a row block share one XCD and its L2.
  // Row block rb runs on XCD rb % 8.  Without peer groups (one tile per
  // workgroup) an XCD's tiles go in the grouped order of kTileGroupRows.
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const bool grouped = p.mode != ROWS_CLUSTER;
  const int q = local / p.cn;
  // Tile (row block rb, column tile c) of iteration it; false when done.
  auto tile_at = [&](int it, int& rb, int& c) {
    if (grouped) {
      const int R = (p.num_rb - xcd + 7) / 8;            // row blocks of this XCD
      if (it > 0 || local >= R * p.cn) return false;
      const int span = kTileGroupRows * p.cn;
      const int g0 = local / span * kTileGroupRows, gsz = min(R - g0, kTileGroupRows), w = local % span;
      rb = (g0 + w % gsz) * 8 + xcd;
      c = w / gsz;
    } else {
      rb = (it * p.slots + q) * 8 + xcd;
      if (rb >= p.num_rb) return false;
      c = local % p.cn;
    }
    return true;
  };
  for (int it = 0; PERSIST || it < 1; ++it) {
    int rb, c;
    if (!tile_at(it, rb, c)) break;
    int m0 = rb * S::TM, n0 = c * S::TN;
    // Opaque copies of the tile origin and lane ids for this iteration: the
    // epilogue's addresses and column masks would otherwise be hoisted out of
    // the tile loop and kept live (spilled) across the whole main loop.
    int lane_t = lane, tid_t = tid;
    asm volatile("" : "+s"(n0), "+s"(m0));
    asm volatile("" : "+v"(lane_t), "+v"(tid_t));
    f32x16_t acc[S::BM][S::BN];
    EpiPrefetch<S> pf;
    const bool cluster = EPI == 1 && p.mode == ROWS_CLUSTER && p.cn > 1;
    unsigned long long round_old = 0;
    if constexpr (EPI >= 1 && !STG) epi_prefetch<S>(pf, p, m0, n0, bz, lane, wm, wn);
    // The bias enters the accumulators unless alpha scales the product.
    const bool fold_bias = p.epi.bias != nullptr && p.epi.alpha == 1.0f;
    if constexpr (LOOP >= 1) mainloop_v2<S, STG, false, LOOP == 2>(acc, X, W, p, m0, n0, bz, smem, lane, wave, wm, wn, fold_bias);
    else mainloop<S>(acc, X, W, p, m0, n0, smem, tid, lane, wm, wn, fold_bias);
    // The round counter's add goes out after the main loop (see cluster_exchange).
    if (cluster) round_old = round_begin(p, q * 8 + xcd, lane, wave);
    if constexpr (EPI >= 1)
      epilogue<S, STG, EPI == 2>(acc, pf, p, m0, n0, q * 8 + xcd, c, round_old, bz, smem, red, tid_t, lane_t, wm, wn);
    else epilogue_plain<S>(acc, p, m0, n0, bz, smem, tid_t, lane_t, wm, wn);
    __syncthreads();
  }
}

// The persistent form of an instantiation: only 128-row tiles with the row
// subgraph run the row-cluster path; every other entry runs one tile per
// workgroup and names its one-tile kernel again.
template <class S, int LOOP, int EPI>
inline const void* gemm_persist_fn() {
  if constexpr (EPI == 1 && S::TM == 128) return reinterpret_cast<const void*>(&gemm_rows_kernel<S, LOOP, EPI, true>);
  else return reinterpret_cast<const void*>(&gemm_rows_kernel<S, LOOP, EPI, false>);
}

// Registry entry of one instantiation: <tile shape S, main loop, epilogue>.
#define CF_GEMM_ENTRY(S, LOOP, EPI)                                                                  \
  GemmKernel {                                                                                       \
    S::TM, S::TN, std::is_same<typename S::T, float>::value ? 1 : 0, LOOP, EPI, S::NT, S::STAGES,    \
        reinterpret_cast<const void*>(&gemm_rows_kernel<S, LOOP, EPI, false>),                       \
        gemm_persist_fn<S, LOOP, EPI>()                                                              \
  }

}  // namespace cf
