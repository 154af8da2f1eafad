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
// FFN:  O = GELU(X W1 + b1) W2 (+ b2 + R, LayerNorm), K = N2 = D.
// 4 waves x 32 rows = 128 rows per workgroup.  The hidden dimension is swept
// in chunks of HC = 32 columns; for chunk k a wave computes its 32 x 32 block
// of P^T = W1^T X^T (the X^T fragments of its rows stay in registers for the
// whole sweep), adds b1, applies GELU, packs S as the second product's B
// fragment and accumulates O^T += W2^T S^T (the partial-sum identity
// O = sum_k S^(k) W2^(k) of Sec. IV-A, accumulated in registers).  S never
// leaves the registers of the wave that produced it.
// Three-stage software pipeline (the PingPong of Sec. III-C inside one wave):
// iteration c issues the MFMAs of chunk c+1's first product and of chunk
// c-1's second product, and between consecutive MFMAs one stage of chunk c's
// GELU for four independent elements (gelu_stage), so the matrix pipe and the
// vector ALU work together without dependency stalls.  W1^T chunks (32 rows,
// all K) and W2^T chunks (D rows, 32 hidden) stream through two two-slot LDS
// rings (Sec. IV-B) one chunk ahead.  The residual, when it is X itself, is
// taken from the X fragments through the lane pair.
// ===========================================================================
template <int N1, int D>
struct FfnShape {
  static constexpr int TM = 128, NT = 256, HC = 32;
  static constexpr int NC = N1 / HC;                 // hidden chunks
  static constexpr int KS1 = D / 16;                 // MFMA steps of GEMM 1 (= X fragments)
  static constexpr int B2 = D / 32;                  // output blocks
  static constexpr int RB1 = D * 2;                  // bytes of one W1^T row (all of K)
  static constexpr int CPR1 = RB1 / 16;              // 16-byte chunks per W1^T row
  static constexpr int W1C = HC * RB1, W2C = D * HC * 2;
  static constexpr int RING1 = 2 * W1C, RING = RING1 + 2 * W2C;
  static constexpr int VEC = (N1 + 3 * D) * 4;       // b1, b2, gamma, beta
  static constexpr int LDS_STORE = TM * (D * 2 + 8);
  static constexpr int LDS = (RING > LDS_STORE ? RING : LDS_STORE) + VEC;
  static constexpr int I1 = W1C / 4096, I2 = W2C / 4096;   // wave-wide loads per wave per chunk
  static constexpr int NM1 = KS1, NM2 = 2 * B2;      // MFMAs per chunk of GEMM 1 / GEMM 2
  static constexpr int GSLOTS = 32;                  // GELU work: 4 groups x 8 stages
  static_assert(N1 % HC == 0 && D % 64 == 0 && W1C % 4096 == 0 && W2C % 4096 == 0, "shape");
  static_assert(LDS <= 160 * 1024, "LDS budget");
  using Out = TileShape<bf16_t, 1, B2, 4, 1, 128, 0>;   // for the staged store (128 x D)
};

// Position of 16-byte chunk c of W1^T row r inside its LDS row: 16 consecutive
// rows read one chunk column, so the position is XOR-swizzled by the row
// (by (r >> 1) & 7 for 128-byte rows, as the GEMM stages).
template <int CPR>
__device__ __forceinline__ int w1_pos(int r, int c) {
  if constexpr (CPR == 8) return c ^ ((r >> 1) & 7);
  else return c ^ (r & 15);
}
// W2^T chunk rows are 64 bytes (32 hidden): chunk c of row r sits at
// position c ^ ((r >> 2) & 3), which spreads 16 consecutive rows over all
// 64 banks.
__device__ __forceinline__ int w2_pos(int r, int c) { return c ^ ((r >> 2) & 3); }

// GEMM-2 A fragment of W2^T row `row` for step s, in the permuted k order of
// pack_step (hidden 16 s + 4 lg + 0..3, then 16 s + 8 + 4 lg + 0..3).
__device__ __forceinline__ u32x4_t frag_perm64(const char* base, int row, int s, int lg) {
  const char* r = base + row * 64 + 8 * lg;
  const u32x2_t lo = lds_read8(r + (w2_pos(row, 2 * s) << 4));
  const u32x2_t hi = lds_read8(r + (w2_pos(row, 2 * s + 1) << 4));
  return u32x4_t{lo[0], lo[1], hi[0], hi[1]};
}

// GELU(x) = x/2 (1 + erf(x / sqrt 2)) with the erf of erf_as (Abramowitz and
// Stegun 7.1.26), split into 8 stages of about two operations so that four
// independent elements can advance one stage between two MFMAs.
struct GeluPipe {
  float h[4], u[4], t[4], y[4], e[4];
};
__device__ __forceinline__ void gelu_stage(GeluPipe& g, float* x, int st) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    switch (st) {
      case 0: g.h[j] = 0.5f * x[j]; g.u[j] = x[j] * 0.70710678118654752f;
              g.t[j] = fmaf(0.3275911f, fabsf(g.u[j]), 1.0f); break;
      case 1: g.t[j] = __builtin_amdgcn_rcpf(g.t[j]); g.e[j] = -(g.u[j] * g.u[j]) * 1.4426950408889634f; break;
      case 2: g.y[j] = fmaf(1.061405429f, g.t[j], -1.453152027f); g.e[j] = __builtin_amdgcn_exp2f(g.e[j]); break;
      case 3: g.y[j] = fmaf(g.y[j], g.t[j], 1.421413741f); break;
      case 4: g.y[j] = fmaf(g.y[j], g.t[j], -0.284496736f); break;
      case 5: g.y[j] = fmaf(g.y[j], g.t[j], 0.254829592f) * g.t[j]; break;
      case 6: g.y[j] = copysignf(fmaf(-g.y[j], g.e[j], 1.0f), g.u[j]); break;
      default: x[j] = fmaf(g.h[j], g.y[j], g.h[j]); break;
    }
  }
}

template <int N1, int D>
__global__ __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
void b2b_ffn_kernel(B2BParams p) {
  using F = FfnShape<N1, D>;
  __shared__ __attribute__((aligned(16))) char smem[F::LDS];
  float* vec = reinterpret_cast<float*>(smem + F::LDS - F::VEC);   // b1[N1] b2[D] gamma[D] beta[D]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lg = lane >> 5;
  const int bz = blockIdx.y;
  const int m0 = blockIdx.x * F::TM;
  const bf16_t* X = p.X + (int64_t)bz * p.sx;
  const bf16_t* W1 = p.W1 + (int64_t)bz * p.sw1;
  const bf16_t* W2 = p.W2 + (int64_t)bz * p.sw2;

  // Per-column vectors into LDS (absent ones as 0 / 1 / 0).
  for (int i = tid; i < N1 + 3 * D; i += F::NT) {
    float v;
    if (i < N1) v = p.b1 ? p.b1[i] : 0.0f;
    else if (i < N1 + D) v = p.b2 ? p.b2[i - N1] : 0.0f;
    else if (i < N1 + 2 * D) v = p.gamma ? p.gamma[i - N1 - D] : 1.0f;
    else v = p.beta ? p.beta[i - N1 - 2 * D] : 0.0f;
    vec[i] = v;
  }

  // Wave-wide loads of hidden chunk k: W1^T rows 32k .. +31 (all K) into
  // ring-1 slot k & 1; W2^T rows 0 .. D-1, hidden 32k .. +31, into ring 2.
  auto issue1 = [&](int k) {
    char* slot = smem + (k & 1) * F::W1C;
#pragma unroll
    for (int j = 0; j < F::I1; ++j) {
      const int q = (wave * F::I1 + j) * 64 + lane;
      const int r = q / F::CPR1, c = w1_pos<F::CPR1>(r, q % F::CPR1);
      dma16(W1 + (int64_t)(k * F::HC + r) * p.ldw1 + c * 8, slot + (wave * F::I1 + j) * 1024);
    }
  };
  auto issue2 = [&](int k) {
    char* slot = smem + F::RING1 + (k & 1) * F::W2C;
#pragma unroll
    for (int j = 0; j < F::I2; ++j) {
      const int q = (wave * F::I2 + j) * 64 + lane;
      const int r = q >> 2, c = w2_pos(r, q & 3);
      dma16(W2 + (int64_t)r * p.ldw2 + k * F::HC + c * 8, slot + (wave * F::I2 + j) * 1024);
    }
  };
  issue1(0);

  // X^T fragments of this wave's 32 rows: xf[ks] = X[m][16 ks + 8 lg .. +8].
  const int m = m0 + wave * 32 + lr;
  const bf16_t* xrow = X + (int64_t)min(m, p.M - 1) * p.ldx + 8 * lg;
  u32x4_t xf[F::KS1];
#pragma unroll
  for (int ks = 0; ks < F::KS1; ++ks) xf[ks] = gload16(xrow + 16 * ks);

  f32x16_t Oa[F::B2];
#pragma unroll
  for (int b = 0; b < F::B2; ++b)
#pragma unroll
    for (int i = 0; i < 16; ++i) Oa[b][i] = 0.0f;

  // One pipeline iteration c: GEMM 1 of chunk c+1 (into Pn, if ONE), GEMM 2
  // of chunk c-1 (with Sp, if TWO) and the GELU of chunk c (on Pc, if GEL).
  // Slot i issues MFMA i (if any), the A-fragment read for MFMA i+2, and GELU
  // stage i % 8 of elements 4 (i / 8) .. +3; the order is pinned.
  f32x16_t Pc, Pn;
  u32x4_t Sp[2];
  auto iter = [&](int c, auto one_t, auto two_t, auto gel_t) {
    constexpr bool ONE = decltype(one_t)::value, TWO = decltype(two_t)::value, GEL = decltype(gel_t)::value;
    constexpr int NM = (ONE ? F::NM1 : 0) + (TWO ? F::NM2 : 0);
    constexpr int NS = GEL ? (NM > F::GSLOTS ? NM : F::GSLOTS) : NM;   // slots
    static_assert(!GEL || NS == F::GSLOTS, "one GELU stage per slot");
    const char* s1 = smem + ((c + 1) & 1) * F::W1C;
    const char* s2 = smem + F::RING1 + ((c - 1) & 1) * F::W2C;
    auto afrag = [&](int i) -> u32x4_t {
      if (ONE && i < F::NM1) return lds_read16(s1 + lr * F::RB1 + (w1_pos<F::CPR1>(lr, 2 * i + lg) << 4));
      const int j = i - (ONE ? F::NM1 : 0);
      return frag_perm64(s2, (j % F::B2) * 32 + lr, j / F::B2, lg);
    };
    if constexpr (ONE) {
#pragma unroll
      for (int i = 0; i < 16; ++i) Pn[i] = 0.0f;
    }
    u32x4_t fr[3];
    GeluPipe gp;
    if constexpr (NM > 0) fr[0] = afrag(0);
    if constexpr (NM > 1) fr[1] = afrag(1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      if (i < NM) {
        if (ONE && i < F::NM1) {
          Mma<bf16_t>::run(Pn, fr[i % 3], xf[i]);
        } else {
          const int j = i - (ONE ? F::NM1 : 0);
          Mma<bf16_t>::run(Oa[j % F::B2], fr[i % 3], Sp[j / F::B2]);
        }
        if (i + 2 < NM) fr[(i + 2) % 3] = afrag(i + 2);
      }
      if constexpr (GEL) {
        const int gi = i;   // GELU stage gi & 7 of elements 4 (gi >> 3) .. +3
        {
          float x4[4] = {Pc[(gi >> 3) * 4], Pc[(gi >> 3) * 4 + 1], Pc[(gi >> 3) * 4 + 2], Pc[(gi >> 3) * 4 + 3]};
          gelu_stage(gp, x4, gi & 7);
          if ((gi & 7) == 7) {
#pragma unroll
            for (int q = 0; q < 4; ++q) Pc[(gi >> 3) * 4 + q] = x4[q];
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // P += b1 of chunk k (right after its GEMM 1; the GELU work then touches registers only).
  auto add_b1 = [&](int k, f32x16_t& P) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4_t bb = *reinterpret_cast<const f32x4_t*>(vec + k * F::HC + 8 * g + 4 * lg);
#pragma unroll
      for (int q = 0; q < 4; ++q) P[4 * g + q] += bb[q];
    }
  };
  using T_ = std::true_type;
  using F_ = std::false_type;
  // Iteration c: W1^T(c+1) and W2^T(c-1) have landed; every wave is done with
  // the slots the next loads overwrite (W1^T(c), W2^T(c-2)).
  auto top = [&](int c) {
    wait_vmcnt<0>();
    __syncthreads();
    if (c + 2 < F::NC) issue1(c + 2);
    if (c < F::NC) issue2(c);
  };
  auto rotate = [&](int c) {   // after iteration c: S of chunk c, P of chunk c+1
    Sp[0] = pack_step(Pc, 0);
    Sp[1] = pack_step(Pc, 1);
    if (c + 1 < F::NC) {
      add_b1(c + 1, Pn);
      Pc = Pn;
    }
  };

  // Prologue: GEMM 1 of chunk 0, then iteration 0 (no GEMM 2 yet).
  wait_vmcnt<0>();
  __syncthreads();
  if (F::NC > 1) issue1(1);
  iter(-1, T_{}, F_{}, F_{});
  add_b1(0, Pn);
  Pc = Pn;
  top(0);
  if constexpr (F::NC > 1) iter(0, T_{}, F_{}, T_{});
  else iter(0, F_{}, F_{}, T_{});
  rotate(0);
  // Steady state: one body, so every accumulator keeps its registers.
  for (int c = 1; c + 1 < F::NC; ++c) {
    top(c);
    iter(c, T_{}, T_{}, T_{});
    rotate(c);
  }
  if constexpr (F::NC > 1) {
    top(F::NC - 1);
    iter(F::NC - 1, F_{}, T_{}, T_{});
    rotate(F::NC - 1);
  }
  top(F::NC);
  iter(F::NC, F_{}, T_{}, F_{});
  __syncthreads();

  // Epi2: x = O + b2 + R, LayerNorm over the row (the lane pair holds it all).
  const bool mv = m < p.M;
  const bool r_is_x = p.R == p.X && p.ldr == p.ldx && (p.batch == 1 || p.sr == p.sx);
#pragma unroll
  for (int b = 0; b < F::B2; ++b)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int n = b * 32 + 8 * g + 4 * lg;
      const f32x4_t bb = *reinterpret_cast<const f32x4_t*>(vec + N1 + n);
#pragma unroll
      for (int q = 0; q < 4; ++q) Oa[b][4 * g + q] += bb[q];
    }
  if (p.R && r_is_x) {
    // X[m][32 b + 8 g + 4 lg + q] lives in xf[2 b + g / 2] of lane half g % 2:
    // each lane keeps one half of a fragment and takes the other from its pair.
#pragma unroll
    for (int ks = 0; ks < F::KS1; ++ks) {
      const uint32_t s0 = lg ? xf[ks][0] : xf[ks][2], s1 = lg ? xf[ks][1] : xf[ks][3];
      const uint32_t r0 = __shfl_xor(s0, 32), r1 = __shfl_xor(s1, 32);
      const uint32_t e0 = lg ? r0 : xf[ks][0], e1 = lg ? r1 : xf[ks][1];   // columns of g even
      const uint32_t o0 = lg ? xf[ks][2] : r0, o1 = lg ? xf[ks][3] : r1;   // columns of g odd
      const int b = ks >> 1, ge = 2 * (ks & 1);
      Oa[b][4 * ge + 0] += bf16_to_f32(e0 & 0xFFFFu);
      Oa[b][4 * ge + 1] += bf16_to_f32(e0 >> 16);
      Oa[b][4 * ge + 2] += bf16_to_f32(e1 & 0xFFFFu);
      Oa[b][4 * ge + 3] += bf16_to_f32(e1 >> 16);
      Oa[b][4 * ge + 4] += bf16_to_f32(o0 & 0xFFFFu);
      Oa[b][4 * ge + 5] += bf16_to_f32(o0 >> 16);
      Oa[b][4 * ge + 6] += bf16_to_f32(o1 & 0xFFFFu);
      Oa[b][4 * ge + 7] += bf16_to_f32(o1 >> 16);
    }
  } else if (p.R && mv) {
#pragma unroll
    for (int b = 0; b < F::B2; ++b)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float r[4];
        load4<bf16_t>(p.R + (int64_t)bz * p.sr + (int64_t)m * p.ldr + b * 32 + 8 * g + 4 * lg, r);
#pragma unroll
        for (int q = 0; q < 4; ++q) Oa[b][4 * g + q] += r[q];
      }
  }
  if (p.out_ln) {
    float s4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int b = 0; b < F::B2; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) s4[i & 3] += Oa[b][i];
    const float mean = lane_pair_sum((s4[0] + s4[1]) + (s4[2] + s4[3])) * (1.0f / D);
    float q4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int b = 0; b < F::B2; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float d = Oa[b][i] - mean;
        q4[i & 3] += d * d;
      }
    const float rstd = rsqrtf(lane_pair_sum((q4[0] + q4[1]) + (q4[2] + q4[3])) * (1.0f / D) + p.eps);
#pragma unroll
    for (int b = 0; b < F::B2; ++b)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = b * 32 + 8 * g + 4 * lg;
        const f32x4_t ga = *reinterpret_cast<const f32x4_t*>(vec + N1 + D + n);
        const f32x4_t be = *reinterpret_cast<const f32x4_t*>(vec + N1 + 2 * D + n);
#pragma unroll
        for (int q = 0; q < 4; ++q) Oa[b][4 * g + q] = (Oa[b][4 * g + q] - mean) * rstd * ga[q] + be[q];
      }
  }
  store_tile_staged<typename F::Out>(reinterpret_cast<f32x16_t(&)[1][F::B2]>(Oa), p.O + (int64_t)bz * p.so, p.ldo, 0,
                                     p.M, D, m0, 0, smem, tid, lane, wave, 0);
}

// ===========================================================================
// Attention: O = softmax(scale * Q K^T) V per (batch*head), online softmax.
// 4 waves x 32 queries = 128 queries per workgroup; key/value blocks of 64.
// Q fragments stay in registers for the whole sweep.  Per block j:
//   S^T = K Q^T (K rows from LDS); lane-local row max / sum over its 32
//   values + the lane pair; P = exp2(S*scale*log2e - m); O = O*corr + P V
//   with P fed from registers and V^T rows from LDS.
// Software pipeline inside each wave (the PingPong of Sec. III-C): the 16
// MFMAs of block j+1's S^T are issued one per slot, and between them the
// softmax of block j runs in 16 VALU chunks; then block j's P V MFMAs.
// The running maximum is raised lazily: O and the row sum are rescaled only
// when a block's maximum exceeds the one in use by more than 2^8, so
// exp2(s - m) <= 256 and the common case skips the rescale; the final O / l
// uses the same maximum throughout, so the result is unchanged.
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
  static constexpr int NSA = 2 * DK;              // MFMAs of one S^T block (two 32-key halves)
  static constexpr int NSB = 4 * BD;              // MFMAs of one P V block
  using Out = TileShape<bf16_t, 1, BD, 4, 1, 128, 0>;
  static_assert(D % 32 == 0 && D <= 128, "head dim");
  static_assert(16 % NSA == 0 || NSA % 16 == 0, "softmax chunks per slot");
};

// Softmax state of one block for one lane (query row lane % 32).
struct SoftmaxStep {
  float bmax, bsum, corr;
  bool need;
  u32x4_t P[2][2];   // bf16 P^T fragments: [32-key half][MFMA step]
};

template <int D>
__global__ __launch_bounds__(256, 1) void b2b_attention_kernel(B2BParams p) {
  using A = AttnShape<D>;
  __shared__ __attribute__((aligned(16))) char smem[A::LDS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lg = lane >> 5;
  // XCD-aware order: workgroups go round-robin over the 8 XCDs by linear id,
  // so linear id L runs on XCD L % 8.  Give each XCD a contiguous range of
  // (head, query block) pairs: the query blocks of one head then share that
  // XCD's L2 copy of the head's K and V instead of fetching it on all eight.
  const int nq = gridDim.x, T = gridDim.x * gridDim.y;
  const int L = blockIdx.x + nq * blockIdx.y;
  const int g = (T & 7) == 0 ? (L & 7) * (T >> 3) + (L >> 3) : L;
  const int bz = g / nq;
  const int m0 = (g % nq) * A::TM;
  const int Lk = p.N1;
  const bf16_t* Q = p.X + (int64_t)bz * p.sx;
  const bf16_t* Kp = p.W1 + (int64_t)bz * p.sw1;
  const bf16_t* Vp = p.W2 + (int64_t)bz * p.sw2;
  const float sl2 = p.mid_scale * 1.4426950408889634f;   // scale * log2(e), > 0
  const int NB = (Lk + A::TN - 1) / A::TN;
  constexpr float kLazy = 8.0f;                           // rescale threshold (log2 units)

  // Q fragments (B operand of S^T = K Q^T): row m, 8 d per lane per step.
  const int m = m0 + wave * 32 + lr;
  const int mc = min(m, p.M - 1);
  u32x4_t qf[A::DK];
#pragma unroll
  for (int ks = 0; ks < A::DK; ++ks) qf[ks] = gload16(Q + (int64_t)mc * p.ldx + ks * 16 + lg * 8);

  // K block rows: swizzled 16-byte chunks inside D*2-byte rows (D/8 chunks;
  // the XOR uses only chunk bits that exist).  Rows past Lk are clamped and
  // masked out of P in the last block.
  // 256-byte rows (d = 128) all start on bank 0, so 16 consecutive rows need
  // 16 distinct chunk positions: XOR with (row & 15).  128-byte rows (d = 64)
  // pair up within 256 bytes: XOR with ((row >> 1) & 7).
  auto kswz = [](int row) { return A::KCH == 16 ? (row & 15) : ((row >> 1) & 7); };
  auto koff = [&](int row, int c) { return row * A::KROW + ((c ^ kswz(row)) << 4); };
  // V^T in LDS: rows d of 64 keys (128 bytes), 16-byte chunk c of row d at
  // position c ^ vswz(d).  vswz mixes d >> 3 into the row-pair swizzle so the
  // transposing writes (16 rows d = 8 dc + e at a time) spread over the banks
  // while 32 consecutive rows still read conflict-free.
  auto vt_off = [](int d, int c) { return d * 128 + ((c ^ (((d >> 1) ^ (d >> 3)) & 7)) << 4); };
  // Thread t moves keys 4 kg .. 4 kg + 3 of d chunk dc (8 d): four 16-byte
  // global loads, an in-register 4 x 8 transpose, eight 8-byte LDS writes.
  constexpr int DC = D / 8;
  const int vkg = tid / DC, vdc = tid % DC;
  const bool vact = tid < (A::TN / 4) * DC;
  u32x4_t vreg[4];
  auto issue_k = [&](int j) {
    char* dst = smem + (j & 1) * A::STAGE;
    constexpr int LPR = A::KCH;                 // lanes per row in one wave-wide load
    constexpr int RPI = 64 / LPR;               // rows per instruction
#pragma unroll
    for (int ins = 0; ins < A::TN / RPI / 4; ++ins) {
      const int in = wave + 4 * ins;
      const int row = in * RPI + lane / LPR;
      const int pos = lane % LPR;
      const int c = pos ^ kswz(row);
      const int key = min(j * A::TN + row, Lk - 1);
      dma16(reinterpret_cast<const char*>(Kp + (int64_t)key * p.ldw1) + c * 16, dst + in * 1024);
    }
  };
  auto load_v = [&](int j) {
    if (vact) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int kk = min(j * A::TN + 4 * vkg + k, Lk - 1);
        vreg[k] = gload16(Vp + (int64_t)kk * p.ldw2 + vdc * 8);
      }
    }
  };
  auto store_v = [&](int j) {
    if (vact) {
      char* vt = smem + (j & 1) * A::STAGE + A::KB;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // keys 0..3 of d = 8 vdc + e: low (e even) or high halves of word e / 2
        const unsigned sel = (e & 1) ? 0x07060302u : 0x05040100u;
        const u32x2_t w = {__builtin_amdgcn_perm(vreg[1][e >> 1], vreg[0][e >> 1], sel),
                           __builtin_amdgcn_perm(vreg[3][e >> 1], vreg[2][e >> 1], sel)};
        *reinterpret_cast<u32x2_t*>(vt + vt_off(8 * vdc + e, vkg >> 1) + (vkg & 1) * 8) = w;
      }
    }
  };
  auto lds_sync = [] {   // this wave's LDS accesses are done, then a workgroup barrier
    __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (3 << 14));
    lds_barrier();
  };

  f32x16_t Oa[A::BD];
#pragma unroll
  for (int b = 0; b < A::BD; ++b)
#pragma unroll
    for (int i = 0; i < 16; ++i) Oa[b][i] = 0.0f;
  float m_used = -INFINITY, lrun = 0.0f;

  // MFMA i of an S^T block (half i / DK, d step i % DK); its K fragment is
  // read two slots ahead.
  auto kfrag = [&](const char* kb, int i) {
    return lds_read16(kb + koff((i / A::DK) * 32 + lr, 2 * (i % A::DK) + lg));
  };
  auto mma_s = [&](f32x16_t (&S)[2], int i, u32x4_t kf) {
    const int b = i / A::DK, ks = i % A::DK;
    const f32x16_t zero = {};
    S[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, kf),
                                                   __builtin_bit_cast(bf16x8_t, qf[ks]), ks == 0 ? zero : S[b],
                                                   0, 0, 0);
  };
  // Softmax of block j in 16 chunks (S is this lane's 32 scores, raw).
  auto sm_chunk = [&](f32x16_t (&S)[2], int c, SoftmaxStep& st, int j, auto mask_t) {
    constexpr bool MASK = decltype(mask_t)::value;
    if (c < 4) {   // block maximum of the raw scores (scale > 0)
      float t = c == 0 ? -INFINITY : st.bmax;
#pragma unroll
      for (int q = 0; q < 8; ++q) t = fmaxf(t, S[c >> 1][(c & 1) * 8 + q]);
      st.bmax = t;
    } else if (c == 4) {
      st.bmax = lane_pair_max(st.bmax) * sl2;
    } else if (c == 5) {
      const float mnew = fmaxf(m_used, st.bmax);
      st.need = mnew > m_used + kLazy;
      const float m_eff = st.need ? mnew : m_used;
      st.corr = __builtin_amdgcn_exp2f(m_used - m_eff);   // exactly 1 when the maximum in use stays
      m_used = m_eff;
      st.bsum = 0.0f;
    } else if (c < 14) {   // P = exp2(s * scale * log2e - m), 4 values per chunk
      const float nm = -m_used;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = (c - 6) * 4 + q;
        float pv = __builtin_amdgcn_exp2f(fmaf(S[e >> 4][e & 15], sl2, nm));
        if constexpr (MASK) {
          const int key = j * A::TN + (e >> 4) * 32 + acc_row(e & 15, lane);
          pv = key < Lk ? pv : 0.0f;
        }
        S[e >> 4][e & 15] = pv;
        st.bsum += pv;
      }
    } else if (c == 14) {
      st.P[0][0] = pack_step(S[0], 0);
      st.P[0][1] = pack_step(S[0], 1);
      st.bsum = lane_pair_sum(st.bsum);
    } else {
      st.P[1][0] = pack_step(S[1], 0);
      st.P[1][1] = pack_step(S[1], 1);
      lrun = lrun * st.corr + st.bsum;
    }
  };
  auto rescale = [&](const SoftmaxStep& st) {
    if (__any(st.need)) {
#pragma unroll
      for (int b = 0; b < A::BD; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) Oa[b][i] *= st.corr;
    }
  };
  // O^T += V^T P^T for block j (V^T fragments two MFMAs ahead).
  auto pv_block = [&](int j, const SoftmaxStep& st) {
    const char* vt = smem + (j & 1) * A::STAGE + A::KB;
    auto vfrag = [&](int i) {   // i = (bl * 2 + s) * BD + b; permuted k order of pack_step
      const int b = i % A::BD, s = (i / A::BD) & 1, bl = i / (2 * A::BD);
      const int row = b * 32 + lr, c0 = 4 * bl + 2 * s;
      const u32x2_t lo = lds_read8(vt + vt_off(row, c0) + 8 * lg);
      const u32x2_t hi = lds_read8(vt + vt_off(row, c0 + 1) + 8 * lg);
      return u32x4_t{lo[0], lo[1], hi[0], hi[1]};
    };
    u32x4_t vf[3];
    vf[0] = vfrag(0);
    if (A::NSB > 1) vf[1] = vfrag(1);
#pragma unroll
    for (int i = 0; i < A::NSB; ++i) {
      if (i + 2 < A::NSB) vf[(i + 2) % 3] = vfrag(i + 2);
      const int b = i % A::BD, s = (i / A::BD) & 1, bl = i / (2 * A::BD);
      Mma<bf16_t>::run(Oa[b], vf[i % 3], st.P[bl][s]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // One pipelined step: S^T of block j+1 (into Sn) under the softmax of block j (Sc).
  auto s_and_softmax = [&](f32x16_t (&Sn)[2], f32x16_t (&Sc)[2], int j, SoftmaxStep& st, auto mask_t) {
    const char* kb = smem + ((j + 1) & 1) * A::STAGE;
    u32x4_t kf[3];
    kf[0] = kfrag(kb, 0);
    kf[1] = kfrag(kb, 1);
    constexpr int CPS = A::NSA >= 16 ? 1 : 16 / A::NSA;   // softmax chunks per MFMA slot
#pragma unroll
    for (int i = 0; i < A::NSA; ++i) {
      if (i + 2 < A::NSA) kf[(i + 2) % 3] = kfrag(kb, i + 2);
      mma_s(Sn, i, kf[i % 3]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < CPS; ++q)
        if (i * CPS + q < 16) sm_chunk(Sc, i * CPS + q, st, j, mask_t);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  auto softmax_only = [&](f32x16_t (&Sc)[2], int j, SoftmaxStep& st, auto mask_t) {
#pragma unroll
    for (int c = 0; c < 16; ++c) sm_chunk(Sc, c, st, j, mask_t);
  };

  f32x16_t Sa[2], Sb[2];
  SoftmaxStep st;
  // Prologue: K, V of block 0 (V transposed into LDS), K, V of block 1 in
  // flight, S^T of block 0.
  issue_k(0);
  load_v(0);
  wait_vmcnt<0>();
  store_v(0);
  if (NB > 1) {
    issue_k(1);
    load_v(1);
  }
  lds_sync();
  {
    const char* kb = smem;
#pragma unroll
    for (int i = 0; i < A::NSA; ++i) mma_s(Sa, i, kfrag(kb, i));
  }
  // Steady step j (blocks j and j+1 exist): K, V of block j+1 landed; V of
  // block j+1 goes to LDS; K, V of block j+2 are issued; then the pipelined
  // S^T(j+1) / softmax(j), the rescale and P V of block j.
  auto step = [&](int j, f32x16_t (&Sc)[2], f32x16_t (&Sn)[2]) {
    wait_vmcnt<0>();
    lds_sync();   // V(j) and K(j+1) visible; buffers of blocks j-1 (V) and j (K) are free
    store_v(j + 1);
    if (j + 2 < NB) {
      issue_k(j + 2);
      load_v(j + 2);
    }
    s_and_softmax(Sn, Sc, j, st, std::false_type{});
    rescale(st);
    pv_block(j, st);
  };
  // Last block (NB-1): masked softmax, rescale, P V.
  auto last = [&](f32x16_t (&Sl)[2]) {
    lds_sync();   // V(NB-1), stored after the previous barrier, is visible
    softmax_only(Sl, NB - 1, st, std::true_type{});
    rescale(st);
    pv_block(NB - 1, st);
  };
  int j = 0;
  for (; j + 2 < NB; j += 2) {
    step(j, Sa, Sb);
    step(j + 1, Sb, Sa);
  }
  if (j + 1 < NB) {
    step(j, Sa, Sb);
    last(Sb);
  } else {
    last(Sa);
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
