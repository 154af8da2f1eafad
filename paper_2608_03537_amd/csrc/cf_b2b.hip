// Back-to-back GEMM kernels for gfx950 (Sec. IV, Eq. 2: P = X W1, S = F(P),
// O = S W2) with the intermediate S kept in registers.
//
// Register hand-off between the two products.  GEMM 1 is computed in the
// transposed form P^T = W1^T X^T, so in each 32x32 accumulator block a lane
// holds one row m of P and 16 of its columns n1: rows 8*(i/4) + 4*g + i%4
// of the block for element i, g = lane/32.  GEMM 2 (O^T = W2^T S^T) consumes
// S^T as its B operand, where lane group g supplies 8 values of the
// contraction index per MFMA step.  The k order inside a step is free as long
// as both operands use the same one, so step s of block b is DEFINED to use
//     n1(s, g, j) = 32 b + 16 s + 8 (j/4) + 4 g + j%4,   j = 0..7,
// which is exactly accumulator elements 8s .. 8s+7 of the lane.  S therefore
// never leaves the registers of the wave that produced it (the register-
// resident S_tile of Sec. IV-A); only the W2 operand is read from LDS, as two
// 8-byte pieces per lane in that same order.
//
// Each wave owns 32 complete rows (all N1 columns of P, all N2 columns of O),
// so the FFN's LayerNorm and the attention's softmax statistics need only
// the lane pair (l, l^32) — no cross-wave or cross-workgroup exchange.
#include "cf_gemm_tile.h"
#include "comfuse.h"

namespace cf {

// Byte offset of 16-byte chunk c of LDS row `row` (128-byte rows, chunk
// position XOR-swizzled by (row >> 1) & 7; see mainloop_v2).
__device__ __forceinline__ int swz_off(int row, int c) { return row * 128 + ((c ^ ((row >> 1) & 7)) << 4); }

__device__ __forceinline__ u32x2_t lds_read8(const char* p) { return *reinterpret_cast<const u32x2_t*>(p); }

// A-operand fragment in the permuted k order of step (bl, s) for LDS row
// `row` of a 128-byte stage row (64 bf16 of the contraction index).
__device__ __forceinline__ u32x4_t frag_perm(const char* base, int row, int bl, int s, int lg) {
  const int c0 = 4 * bl + 2 * s;
  const u32x2_t lo = lds_read8(base + swz_off(row, c0) + 8 * lg);
  const u32x2_t hi = lds_read8(base + swz_off(row, c0 + 1) + 8 * lg);
  return u32x4_t{lo[0], lo[1], hi[0], hi[1]};
}

// Accumulator elements 8s .. 8s+7 of a block, as 8 packed bf16.
__device__ __forceinline__ u32x4_t pack_step(const f32x16_t& v, int s) {
  return u32x4_t{pack_bf16x2(v[8 * s + 0], v[8 * s + 1]), pack_bf16x2(v[8 * s + 2], v[8 * s + 3]),
                 pack_bf16x2(v[8 * s + 4], v[8 * s + 5]), pack_bf16x2(v[8 * s + 6], v[8 * s + 7])};
}

__device__ __forceinline__ float lane_pair_sum(float v) { return v + __shfl_xor(v, 32); }
__device__ __forceinline__ float lane_pair_max(float v) { return fmaxf(v, __shfl_xor(v, 32)); }

// ===========================================================================
// FFN:  O = GELU(X W1 + b1) W2 (+ b2 + R, LayerNorm)
// 4 waves x 32 rows = 128 rows per workgroup.  The hidden dimension N1 is
// processed in passes of NP columns: a pass computes P^T for its NP columns,
// packs S, and adds its share S^(c) W2^(c) to the output accumulator — the
// partial-sum identity O = sum_c S^(c) W2^(c) of Sec. IV-A, here accumulated
// in registers by one wave instead of across co-scheduled workgroups.  With
// NP = 256 a wave holds 128 accumulator registers for P, 128 for O and 64 for
// S, which fits the register file without spilling.
// One LDS ring of two stages serves both products (the unified circular
// buffer of Sec. IV-B): GEMM-1 stages hold 64 k of the NP rows of W1^T and
// the 128 rows of X, GEMM-2 stages 64 n1 of the N2 rows of W2^T.  Stage t+1 is
// loaded while stage t is consumed, across pass and phase boundaries
// (ML1 -> Epi1 -> ML2 -> Epi2 of Sec. IV-C).
// ===========================================================================
template <int N1, int N2>
struct FfnShape {
  static constexpr int TM = 128, NT = 256;
  static constexpr int NP = N1 < 256 ? N1 : 256;    // hidden columns per pass
  static constexpr int NPASS = N1 / NP;
  static constexpr int ROWS1 = NP + TM, ROWS2 = N2;
  static constexpr int STAGE = (ROWS1 > ROWS2 ? ROWS1 : ROWS2) * 128;
  static constexpr int LDS_RING = 2 * STAGE;
  static constexpr int LDS_STORE = TM * (N2 * 2 + 8);
  static constexpr int LDS = LDS_RING > LDS_STORE ? LDS_RING : LDS_STORE;
  static constexpr int BP = NP / 32, B2 = N2 / 32;   // accumulator blocks of P (per pass) and O
  static constexpr int KT2 = NP / 64;                 // GEMM-2 stages per pass
  static_assert(N1 % NP == 0 && NP % 64 == 0 && N2 % 32 == 0, "shape");
  static_assert(LDS <= 160 * 1024, "LDS budget");
  using Out = TileShape<bf16_t, 1, B2, 4, 1, 128, 0>;   // for the staged store (128 x N2)
};

template <int N1, int N2>
__global__ __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
void b2b_ffn_kernel(B2BParams p) {
  using F = FfnShape<N1, N2>;
  __shared__ __attribute__((aligned(16))) char smem[F::LDS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lg = lane >> 5, sw = (lr >> 1) & 7;
  const int bz = blockIdx.y;
  const int m0 = blockIdx.x * F::TM;
  const bf16_t* X = p.X + (int64_t)bz * p.sx;
  const bf16_t* W1 = p.W1 + (int64_t)bz * p.sw1;
  const bf16_t* W2 = p.W2 + (int64_t)bz * p.sw2;
  const int KT1 = p.K / 64;
  const int TP = KT1 + F::KT2;              // stages per pass
  const int T = F::NPASS * TP;

  // Wave-wide loads of global stage t: 8 rows per instruction, chunk (lane&7)
  // of the LDS row is fed from logical chunk (lane&7) ^ ((row>>1)&7).
  auto issue = [&](int t) {
    if (t >= T) return;
    char* dst = smem + (t & 1) * F::STAGE;
    const int pass = t / TP, r = t % TP;
    const bool g1 = r < KT1;
    const int rows = g1 ? F::ROWS1 : F::ROWS2;
    for (int ins = wave; ins < rows / 8; ins += 4) {
      const int row = ins * 8 + (lane >> 3);
      const int c = (lane & 7) ^ ((row >> 1) & 7);
      const bf16_t* src;
      if (g1) {
        src = row < F::NP ? W1 + (int64_t)(pass * F::NP + row) * p.ldw1
                          : X + (int64_t)min(m0 + row - F::NP, p.M - 1) * p.ldx;
        src += r * 64;
      } else {
        src = W2 + (int64_t)row * p.ldw2 + pass * F::NP + (r - KT1) * 64;
      }
      dma16(reinterpret_cast<const char*>(src) + c * 16, dst + ins * 1024);
    }
  };

  f32x16_t Oa[F::B2];
#pragma unroll
  for (int b = 0; b < F::B2; ++b)
#pragma unroll
    for (int i = 0; i < 16; ++i) Oa[b][i] = 0.0f;

  issue(0);
#pragma unroll
  for (int pass = 0; pass < F::NPASS; ++pass) {
    f32x16_t P[F::BP];
#pragma unroll
    for (int b = 0; b < F::BP; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) P[b][i] = 0.0f;

    // ML1: P^T += W1^T(stage) X^T(stage) for this pass's NP columns.
    for (int r = 0; r < KT1; ++r) {
      const int t = pass * TP + r;
      wait_vmcnt<0>();
      lds_barrier();
      issue(t + 1);
      const char* st = smem + (t & 1) * F::STAGE;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int c = 2 * ks + lg;
        const u32x4_t xb = lds_read16(st + (F::NP + wave * 32 + lr) * 128 + ((c ^ sw) << 4));
#pragma unroll
        for (int b = 0; b < F::BP; ++b) {
          const u32x4_t wa = lds_read16(st + (b * 32 + lr) * 128 + ((c ^ sw) << 4));
          Mma<bf16_t>::run(P[b], wa, xb);
        }
      }
    }

    // Epi1: S = GELU(P + b1), packed as GEMM-2 B fragments (in registers).
    u32x4_t S[F::BP][2];
#pragma unroll
    for (int b = 0; b < F::BP; ++b) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4_t bb = {0.0f, 0.0f, 0.0f, 0.0f};
        if (p.b1) bb = *reinterpret_cast<const f32x4_t*>(p.b1 + pass * F::NP + b * 32 + 8 * g + 4 * lg);
#pragma unroll
        for (int q = 0; q < 4; ++q) P[b][4 * g + q] = gelu_erf(P[b][4 * g + q] + bb[q]);
      }
      S[b][0] = pack_step(P[b], 0);
      S[b][1] = pack_step(P[b], 1);
    }

    // ML2: O^T += W2^T(stage) S^T over this pass's NP hidden columns.
#pragma unroll
    for (int tl = 0; tl < F::KT2; ++tl) {
      const int t = pass * TP + KT1 + tl;
      wait_vmcnt<0>();
      lds_barrier();
      issue(t + 1);
      const char* st = smem + (t & 1) * F::STAGE;
#pragma unroll
      for (int bl = 0; bl < 2; ++bl)
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          const u32x4_t sb = S[2 * tl + bl][s];
#pragma unroll
          for (int b = 0; b < F::B2; ++b) Mma<bf16_t>::run(Oa[b], frag_perm(st, b * 32 + lr, bl, s, lg), sb);
        }
    }
  }
  __syncthreads();

  // Epi2: x = O + b2 + R, LayerNorm over the row (lane pair holds it all).
  const int m = m0 + wave * 32 + lr;
  const bool mv = m < p.M;
#pragma unroll
  for (int b = 0; b < F::B2; ++b)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int n = b * 32 + 8 * g + 4 * lg;
      if (p.b2) {
        const f32x4_t bb = *reinterpret_cast<const f32x4_t*>(p.b2 + n);
#pragma unroll
        for (int q = 0; q < 4; ++q) Oa[b][4 * g + q] += bb[q];
      }
      if (p.R && mv) {
        float r[4];
        load4<bf16_t>(p.R + (int64_t)bz * p.sr + (int64_t)m * p.ldr + n, r);
#pragma unroll
        for (int q = 0; q < 4; ++q) Oa[b][4 * g + q] += r[q];
      }
    }
  if (p.out_ln) {
    float s = 0.0f;
#pragma unroll
    for (int b = 0; b < F::B2; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) s += Oa[b][i];
    const float mean = lane_pair_sum(s) * (1.0f / N2);
    float q2 = 0.0f;
#pragma unroll
    for (int b = 0; b < F::B2; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float d = Oa[b][i] - mean;
        q2 += d * d;
      }
    const float rstd = rsqrtf(lane_pair_sum(q2) * (1.0f / N2) + p.eps);
#pragma unroll
    for (int b = 0; b < F::B2; ++b)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = b * 32 + 8 * g + 4 * lg;
        f32x4_t ga = {1.0f, 1.0f, 1.0f, 1.0f}, be = {0.0f, 0.0f, 0.0f, 0.0f};
        if (p.gamma) ga = *reinterpret_cast<const f32x4_t*>(p.gamma + n);
        if (p.beta) be = *reinterpret_cast<const f32x4_t*>(p.beta + n);
#pragma unroll
        for (int q = 0; q < 4; ++q) Oa[b][4 * g + q] = (Oa[b][4 * g + q] - mean) * rstd * ga[q] + be[q];
      }
  }
  store_tile_staged<typename F::Out>(reinterpret_cast<f32x16_t(&)[1][F::B2]>(Oa), p.O + (int64_t)bz * p.so, p.ldo, 0, p.M, N2, m0, 0, smem, tid, lane,
                                     wave, 0);
}

// ===========================================================================
// Attention: O = softmax(scale * Q K^T) V per (batch*head), online softmax.
// 4 waves x 32 queries = 128 queries per workgroup; key/value blocks of 64.
// Q fragments stay in registers for the whole sweep.  Per block:
//   S^T = K Q^T (K rows from LDS), lane-local row max / sum over its 32
//   values + the lane pair, P = exp2(S*scale*log2e - m), O = O*corr + P V
//   with P fed from registers and V^T rows from LDS.
// K blocks arrive by wave-wide direct loads; V is transposed on its way into
// LDS (rows d, 64 keys contiguous) through registers.
// ===========================================================================
template <int D>
struct AttnShape {
  static constexpr int TM = 128, TN = 64, NT = 256;
  static constexpr int KB = TN * D * 2;           // K block bytes (TN rows of D*2 bytes)
  static constexpr int VB = D * TN * 2;           // V^T block bytes (D rows of 128 bytes)
  static constexpr int STAGE = KB + VB;
  static constexpr int LDS_RING = 2 * STAGE;
  static constexpr int LDS_STORE = TM * (D * 2 + 8);
  static constexpr int LDS = LDS_RING > LDS_STORE ? LDS_RING : LDS_STORE;
  static constexpr int DK = D / 16;               // MFMA k steps over d
  static constexpr int BD = D / 32;               // output blocks over d
  static constexpr int KROW = D * 2;              // bytes per K row
  static constexpr int KCH = KROW / 16;           // 16-byte chunks per K row
  static constexpr int VCH = TN * D / 8 / NT;     // V chunks (8 d of one key) per thread
  using Out = TileShape<bf16_t, 1, BD, 4, 1, 128, 0>;
  static_assert(D % 32 == 0 && D <= 128, "head dim");
};

template <int D>
__global__ __launch_bounds__(256, 2) void b2b_attention_kernel(B2BParams p) {
  using A = AttnShape<D>;
  __shared__ __attribute__((aligned(16))) char smem[A::LDS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lg = lane >> 5;
  const int bz = blockIdx.y;
  const int m0 = blockIdx.x * A::TM;
  const int Lk = p.N1;
  const bf16_t* Q = p.X + (int64_t)bz * p.sx;
  const bf16_t* Kp = p.W1 + (int64_t)bz * p.sw1;
  const bf16_t* Vp = p.W2 + (int64_t)bz * p.sw2;
  const float sl2 = p.mid_scale * 1.4426950408889634f;   // scale * log2(e)
  const int NB = (Lk + A::TN - 1) / A::TN;

  // Q fragments (B operand of S^T = K Q^T): row m, 8 d per lane per step.
  const int m = m0 + wave * 32 + lr;
  const int mc = min(m, p.M - 1);
  u32x4_t qf[A::DK];
#pragma unroll
  for (int ks = 0; ks < A::DK; ++ks) qf[ks] = gload16(Q + (int64_t)mc * p.ldx + ks * 16 + lg * 8);

  // K block rows: swizzled 16-byte chunks inside D*2-byte rows (D/8 chunks;
  // the XOR uses only chunk bits that exist).  Rows past Lk are clamped and
  // masked to -inf in the scores.
  // 256-byte rows (d = 128) all start on bank 0, so 16 consecutive rows need
  // 16 distinct chunk positions: XOR with (row & 15).  128-byte rows (d = 64)
  // pair up within 256 bytes: XOR with ((row >> 1) & 7).
  auto kswz = [](int row) { return A::KCH == 16 ? (row & 15) : ((row >> 1) & 7); };
  auto koff = [&](int row, int c) { return row * A::KROW + ((c ^ kswz(row)) << 4); };
  u32x4_t vreg[A::VCH];
  auto issue_k = [&](int j) {
    char* dst = smem + (j & 1) * A::STAGE;
    constexpr int LPR = A::KCH;                 // lanes per row in one wave-wide load
    constexpr int RPI = 64 / LPR;               // rows per instruction
    for (int ins = wave; ins < A::TN / RPI; ins += 4) {
      const int row = ins * RPI + lane / LPR;
      const int pos = lane % LPR;
      const int c = pos ^ kswz(row);
      const int key = min(j * A::TN + row, Lk - 1);
      dma16(reinterpret_cast<const char*>(Kp + (int64_t)key * p.ldw1) + c * 16, dst + ins * 1024);
    }
  };
  auto load_v = [&](int j) {
#pragma unroll
    for (int i = 0; i < A::VCH; ++i) {
      const int ch = tid + i * A::NT;            // chunk = 8 d of one key
      const int key = ch / (D / 8), dc = ch % (D / 8);
      const int kk = min(j * A::TN + key, Lk - 1);
      vreg[i] = gload16(Vp + (int64_t)kk * p.ldw2 + dc * 8);
    }
  };
  auto store_v = [&](int j) {
    char* vt = smem + (j & 1) * A::STAGE + A::KB;
#pragma unroll
    for (int i = 0; i < A::VCH; ++i) {
      const int ch = tid + i * A::NT;
      const int key = ch / (D / 8), dc = ch % (D / 8);
      // V^T row d, key column: 16-byte chunk key/8 of the 128-byte row.
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = dc * 8 + e;
        const uint32_t w = vreg[i][e >> 1];
        *reinterpret_cast<uint16_t*>(vt + swz_off(d, key >> 3) + (key & 7) * 2) =
            (uint16_t)((e & 1) ? (w >> 16) : (w & 0xFFFFu));
      }
    }
  };

  f32x16_t Oa[A::BD];
#pragma unroll
  for (int b = 0; b < A::BD; ++b)
#pragma unroll
    for (int i = 0; i < 16; ++i) Oa[b][i] = 0.0f;
  float mrun = -INFINITY, lrun = 0.0f;

  issue_k(0);
  load_v(0);
  store_v(0);
  for (int j = 0; j < NB; ++j) {
    wait_vmcnt<0>();
    __syncthreads();
    if (j + 1 < NB) {
      issue_k(j + 1);
      load_v(j + 1);
    }
    const char* kb = smem + (j & 1) * A::STAGE;
    const char* vt = kb + A::KB;
    // S^T block (64 keys x 32 queries) = K Q^T
    f32x16_t Sb[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
#pragma unroll
      for (int i = 0; i < 16; ++i) Sb[b][i] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < A::DK; ++ks)
        Mma<bf16_t>::run(Sb[b], lds_read16(kb + koff(b * 32 + lr, 2 * ks + lg)), qf[ks]);
    }
    // Online softmax for this lane's query row.
    float bmax = -INFINITY;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = j * A::TN + b * 32 + acc_row(i, lane);
        const float sv = key < Lk ? Sb[b][i] * sl2 : -INFINITY;
        Sb[b][i] = sv;
        bmax = fmaxf(bmax, sv);
      }
    const float mnew = fmaxf(mrun, lane_pair_max(bmax));
    const float corr = exp2f(mrun - mnew);
    float bsum = 0.0f;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float pv = exp2f(Sb[b][i] - mnew);
        Sb[b][i] = pv;
        bsum += pv;
      }
    lrun = lrun * corr + lane_pair_sum(bsum);
    mrun = mnew;
#pragma unroll
    for (int b = 0; b < A::BD; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) Oa[b][i] *= corr;
    // O^T += V^T P^T, P from registers in the permuted k order.
#pragma unroll
    for (int bl = 0; bl < 2; ++bl)
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const u32x4_t pb = pack_step(Sb[bl], s);
#pragma unroll
        for (int b = 0; b < A::BD; ++b) Mma<bf16_t>::run(Oa[b], frag_perm(vt, b * 32 + lr, bl, s, lg), pb);
      }
    // Buffer (j+1)&1 was last read in iteration j-1, which every wave left
    // at this iteration's first barrier; the next barrier publishes it.
    if (j + 1 < NB) store_v(j + 1);
  }
  __syncthreads();
  const float inv = 1.0f / lrun;
#pragma unroll
  for (int b = 0; b < A::BD; ++b)
#pragma unroll
    for (int i = 0; i < 16; ++i) Oa[b][i] *= inv;
  store_tile_staged<typename A::Out>(reinterpret_cast<f32x16_t(&)[1][A::BD]>(Oa), p.O + (int64_t)bz * p.so, p.ldo, 0, p.M, D, m0, 0, smem, tid, lane,
                                     wave, 0);
}

// ---------------------------------------------------------------------------
bool b2b_ffn_supported(int N1, int N2) {
  return (N1 == 512 && N2 == 256) || (N1 == 256 && N2 == 128) || (N1 == 128 && N2 == 64) ||
         (N1 == 256 && N2 == 256);
}
bool b2b_attention_supported(int d) { return d == 64 || d == 128; }

hipError_t launch_b2b_ffn(const B2BParams& p, hipStream_t st) {
  const dim3 grid((unsigned)((p.M + 127) / 128), (unsigned)p.batch), block(256);
  if (p.N1 == 512 && p.N2 == 256) hipLaunchKernelGGL((b2b_ffn_kernel<512, 256>), grid, block, 0, st, p);
  else if (p.N1 == 256 && p.N2 == 256) hipLaunchKernelGGL((b2b_ffn_kernel<256, 256>), grid, block, 0, st, p);
  else if (p.N1 == 256 && p.N2 == 128) hipLaunchKernelGGL((b2b_ffn_kernel<256, 128>), grid, block, 0, st, p);
  else if (p.N1 == 128 && p.N2 == 64) hipLaunchKernelGGL((b2b_ffn_kernel<128, 64>), grid, block, 0, st, p);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_b2b_attention(const B2BParams& p, hipStream_t st) {
  const dim3 grid((unsigned)((p.M + 127) / 128), (unsigned)p.batch), block(256);
  if (p.K == 128) hipLaunchKernelGGL((b2b_attention_kernel<128>), grid, block, 0, st, p);
  else if (p.K == 64) hipLaunchKernelGGL((b2b_attention_kernel<64>), grid, block, 0, st, p);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace cf
