// Back-to-back FFN for gfx950 (Sec. IV, Eq. 2 with F = +b1, GELU; Sec. IV-A):
//   O = GELU(X W1 + b1) W2 (+ b2 + R, LayerNorm),   K = N2 = D,
// with the intermediate S kept on chip.
//
// Work split.  A workgroup owns 128 rows and runs 8 waves, two per SIMD: a
// single wave issues vector instructions at about half the SIMD's rate, and
// the GELU between the two products is vector work.  Waves w and w + 4 form
// a pair that shares 32 rows (row group pr = w & 3); half h = w >> 2 of the
// pair owns output columns [h D/2, (h+1) D/2) and the hidden chunks c with
// c % 2 == h (chunks are HC = 32 hidden units).  Round t covers chunks 2t and
// 2t+1: each half computes the first product and the GELU of its own chunk,
// hands the bf16 S of that chunk to its partner through LDS, and accumulates
// the second product of both chunks into its own half of O (the partial-sum
// identity O = sum_k S^(k) W2^(k) of Sec. IV-A).
//
// Register hand-off.  The first product is computed transposed,
// P^T = W1^T X^T, so in a 32x32 accumulator block lane (lr, g = lane / 32)
// holds row m = lr of P and element i sits in block row 8 (i/4) + 4 g + i%4.
// The rows of each W1^T chunk are loaded in a permuted order
// (ffn_hidden_row), so that accumulator elements 8 s .. 8 s + 7 hold hidden
// units 16 s + 8 g + 0..7.  Packed to bf16 they are exactly the B operand of
// step s of the second product O^T = W2^T S^T, whose A operand is then one
// contiguous 16-byte piece of a W2^T row.
//
// Weight loads.  Every wave-wide direct load (global_load_lds) brings 8 whole
// 128-byte lines: 8 rows x 128 bytes of one operand, which lands as 8
// consecutive 128-byte LDS rows whose 16-byte chunks are XOR-swizzled by
// (row >> 1) & 7.  A fragment read (16 consecutive rows, one chunk column per
// 16 lanes) is then conflict-free.  Loads that gather 32-byte pieces of 32
// rows instead touch four times as many lines per byte, and the weights'
// L2-to-LDS stream ran at about a quarter of this rate.  Layout (bytes):
//   ring 1: 2 stages x W1^T rows of chunks 2t, 2t+1: [k block D/64][row 64][128 B]
//   ring 2: 2 stages x W2^T columns of chunks 2t, 2t+1: [row D][128 B]
//   S exchange: 2 stages x [row group 4][half 2][lane 64][32 B]
#include "cf_gemm_tile.h"
#include "comfuse.h"

namespace cf {

template <int N1, int D>
struct FfnShape {
  static constexpr int TM = 128, NW = 8, NT = 64 * NW, HC = 32;
  static constexpr int NC = N1 / HC;            // hidden chunks
  static constexpr int NR = NC / 2;             // rounds (one chunk per half)
  static constexpr int KS1 = D / 16;            // MFMA steps of the first product (= X fragments)
  static constexpr int B2 = D / 32, B2H = B2 / 2;   // output blocks: all, per half
  static constexpr int NM1 = KS1;               // first-product MFMAs per round (own chunk)
  static constexpr int NM2 = 2 * 2 * B2H;       // second-product MFMAs per round (2 chunks x B2H x 2 steps)
  static constexpr int W1C = KS1 * 1024;        // one W1^T chunk (32 x D bf16)
  static constexpr int W2C = 2 * B2 * 1024;     // one W2^T chunk (D x 32 bf16)
  static constexpr int W1S = 2 * W1C, W2S = 2 * W2C;
  static constexpr int OFF_W2 = 2 * W1S;
  static constexpr int OFF_X = OFF_W2 + 2 * W2S;
  static constexpr int XCH = 4 * 2 * 64 * 32;   // one exchange stage
  static constexpr int LDS = OFF_X + 2 * XCH;
  static constexpr int LDS_STORE = TM * (D * 2 + 8);
  static constexpr int DMA_W = (2 * KS1 + 2 * 2 * B2) / NW;   // wave-wide loads per wave per round
  static constexpr int GSLOTS = 32;             // GELU work per round: 4 groups x 8 stages
  static constexpr int FG = 4;                  // A-fragment reads per group
  static_assert(N1 % (2 * HC) == 0 && D % 64 == 0, "shape");
  static_assert(NM1 == NM2, "the two products alternate MFMA by MFMA");
  static_assert((2 * KS1 + 4 * B2) % NW == 0, "loads per wave");
  static_assert(LDS <= 160 * 1024 && LDS_STORE <= OFF_X, "LDS budget");
  using Out = TileShape<bf16_t, 1, B2H, 4, 2, 128, 0>;   // staged store: 128 x D, wave tile 32 x D/2
};

// Hidden unit (within its chunk) held by row r of a W1^T chunk in LDS: bits
// 2 and 3 of r swapped (see the register hand-off above).
__device__ __forceinline__ int ffn_hidden_row(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }

// Accumulator elements 8 s .. 8 s + 7 as 8 packed bf16 (B operand of step s).
__device__ __forceinline__ u32x4_t ffn_pack_step(const f32x16_t& v, int s) {
  return u32x4_t{pack_bf16x2(v[8 * s + 0], v[8 * s + 1]), pack_bf16x2(v[8 * s + 2], v[8 * s + 3]),
                 pack_bf16x2(v[8 * s + 4], v[8 * s + 5]), pack_bf16x2(v[8 * s + 6], v[8 * s + 7])};
}

// GELU(x) = x/2 (1 + erf(x / sqrt 2)) with the erf of Abramowitz and Stegun
// 7.1.26 (as erf_as), in the form
//   GELU(x) = max(x, 0) - |x| y(t) exp(-x^2 / 2) / 2,
//   t = 1 / (1 + p |x| / sqrt 2),  y(t) = a1 t + ... + a5 t^5,
// which follows from erf(z) = 1 - y(t) exp(-z^2) for z >= 0 and the odd
// extension (for x >= 0 the two halves x/2 + x/2 erf give x - x y e / 2; for
// x < 0 they give x y e / 2).  Eleven vector operations and two
// transcendentals per element, split into 8 stages so that four independent
// elements advance one stage between two MFMAs.  The input x stays in place
// until the last stage.
struct GeluPipe {
  float t[4], y[4], e[4];
};
__device__ __forceinline__ void gelu_stage(GeluPipe& g, const float* x, float* out, int st) {
  constexpr float kP = 0.3275911f * 0.70710678118654752f;   // p / sqrt 2
  constexpr float kNegHalfLog2e = -0.72134752044448170f;    // -log2(e) / 2
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    switch (st) {
      case 0: g.t[j] = fmaf(kP, fabsf(x[j]), 1.0f); break;
      case 1: g.t[j] = __builtin_amdgcn_rcpf(g.t[j]); g.e[j] = x[j] * kNegHalfLog2e; break;
      // 2^(-x^2 log2(e) / 2 - 1) = exp(-x^2 / 2) / 2
      case 2: g.e[j] = __builtin_amdgcn_exp2f(fmaf(x[j], g.e[j], -1.0f)); break;
      case 3: g.y[j] = fmaf(1.061405429f, g.t[j], -1.453152027f); break;
      case 4: g.y[j] = fmaf(g.y[j], g.t[j], 1.421413741f); break;
      case 5: g.y[j] = fmaf(g.y[j], g.t[j], -0.284496736f); break;
      case 6: g.y[j] = fmaf(g.y[j], g.t[j], 0.254829592f); g.e[j] = fabsf(x[j]) * g.e[j]; break;
      default: {
        // max(x, 0) as one v_max_f32 (fmaxf adds a canonicalising max in front)
        float r;
        asm("v_max_f32_e32 %0, 0, %1" : "=v"(r) : "v"(x[j]));
        out[j] = fmaf(-g.e[j], g.y[j] * g.t[j], r);
      } break;
    }
  }
}

template <int N1, int D>
__global__ __launch_bounds__(512, 1) __attribute__((amdgpu_waves_per_eu(2, 2)))
void b2b_ffn_kernel(B2BParams p) {
  using F = FfnShape<N1, D>;
  __shared__ __attribute__((aligned(16))) char smem[F::LDS];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int lr = lane & 31, lg = lane >> 5;
  const int pr = wave & 3, h = wave >> 2;       // row group, half
  const int bz = blockIdx.y;
  const int m0 = blockIdx.x * F::TM;
  const int m = m0 + pr * 32 + lr;
  const bf16_t* X = p.X + (int64_t)bz * p.sx;
  const bf16_t* W1 = p.W1 + (int64_t)bz * p.sw1;
  const bf16_t* W2 = p.W2 + (int64_t)bz * p.sw2;
  const int nb0 = h * F::B2H;                   // first output block of this half

  // Wave-wide loads of one round.  Waves 0-3 load the W1^T rows of chunks 2r
  // and 2r+1: load q in [0, D/8) covers k block q / 8 (64 k) of LDS rows
  // 8 (q % 8) .. +7, and LDS row i holds hidden unit
  // 32 (2r + i / 32) + ffn_hidden_row(i % 32).  Waves 4-7 load the W2^T
  // columns of both chunks (hidden 64r .. 64r+63, 128 bytes of each of the D
  // rows): load q covers rows 8q .. 8q+7.
  // A load's address is a wave-uniform part (q, round) plus one of two lane
  // offsets: the lane's row within the 8-row group (W1: its bits of the hidden
  // unit) and its swizzled chunk, which depends on q only through q % 2
  // (bit 2 of the swizzle term).
  const bool w1part = wave < 4;
  const int lrow = lane >> 3, lch = lane & 7;
  const char* gbase = w1part ? reinterpret_cast<const char*>(W1) : reinterpret_cast<const char*>(W2);
  const int64_t pitch = 2 * (w1part ? p.ldw1 : p.ldw2);
  const int lrow_h = w1part ? ((lrow & 3) | ((lrow & 4) << 1)) : lrow;
  uint32_t loff[2];
#pragma unroll
  for (int v = 0; v < 2; ++v) loff[v] = (uint32_t)(lrow_h * pitch + 16 * (lch ^ (lrow >> 1) ^ (v << 2)));
  auto issue = [&](int r1, bool do1, int r2, bool do2) {
    if (w1part ? !do1 : !do2) return;
    const int r = w1part ? r1 : r2;
#pragma unroll
    for (int j = 0; j < F::DMA_W; ++j) {
      const int q = (wave & 3) * F::DMA_W + j;
      int64_t goff;
      int soff;
      if (w1part) {
        const int i8 = q & 7;   // 8-row group of LDS rows 8 i8 .. +7
        const int hid = 64 * r + 32 * (i8 >> 2) + 16 * ((i8 >> 1) & 1) + 4 * (i8 & 1);
        goff = hid * pitch + 128 * (q >> 3);
        soff = (r & 1) * F::W1S + q * 1024;
      } else {
        goff = 8 * q * pitch + 128 * r;
        soff = F::OFF_W2 + (r & 1) * F::W2S + q * 1024;
      }
      dma16(gbase + goff + loff[q & 1], smem + soff);
    }
  };
  // Lane offsets of the fragment reads.  First product, step ks: LDS row
  // 32 h + lr of k block ks / 4, chunk 2 (ks % 4) + lg.  Second product,
  // output block b, step s of chunk 2t + e: row 32 (nb0 + b) + lr, chunk
  // 4 e + 2 s + lg.  The swizzle term (row >> 1) & 7 is (lr >> 1) & 7 for both.
  const int sw = (lr >> 1) & 7;
  auto o1 = [&](int u) { return (32 * h + lr) * 128 + ((((u << 1) | lg) ^ sw) << 4); };
  auto o2 = [&](int e, int s2) { return lr * 128 + (((4 * e + 2 * s2 + lg) ^ sw) << 4); };

  // The X tile goes to LDS first, through the second product's weight ring
  // (free until round 0's W2^T loads, issued after every wave has read its
  // fragments): whole rows by wave-wide direct loads, so every 128-byte line
  // of X is fetched once, in full.  Row r, 16-byte chunk c sits at chunk
  // position c ^ (r & XSW) of its 2D-byte LDS row; one load fills 1 KB =
  // 1024 / (2D) rows, lane i the position i % (D / 8) of row i / (D / 8).
  constexpr int XCPR = D / 8;                       // 16-byte chunks per X row
  constexpr int XSW = (XCPR < 16 ? XCPR : 16) - 1;  // swizzle mask
  constexpr int XLOADS = F::TM * XCPR / 64 / F::NW; // wave-wide loads per wave
  static_assert(F::TM * 2 * D == 2 * F::W2S && (F::TM * XCPR) % (64 * F::NW) == 0, "X staging");
#pragma unroll
  for (int j = 0; j < XLOADS; ++j) {
    const int ld = wave * XLOADS + j;
    const int r = (ld * 64 + lane) / XCPR, cp = lane % XCPR;
    const int c = cp ^ (r & XSW);
    dma16(X + (int64_t)min(m0 + r, p.M - 1) * p.ldx + 8 * c, smem + F::OFF_W2 + ld * 1024);
  }
  u32x4_t xf[F::KS1];   // X^T fragments, read from LDS in the prologue below

  // O accumulators start at b2 (element i of block b: column 32 b + 8 (i/4) + 4 lg + i%4).
  f32x16_t Oa[F::B2H];
  if (p.b2) {
    const float* b2l = p.b2 + nb0 * 32 + 4 * lg;
#pragma unroll
    for (int b = 0; b < F::B2H; ++b)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4_t bb = *reinterpret_cast<const f32x4_t*>(b2l + b * 32 + 8 * g);
#pragma unroll
        for (int q = 0; q < 4; ++q) Oa[b][4 * g + q] = bb[q];
      }
  } else {
#pragma unroll
    for (int b = 0; b < F::B2H; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) Oa[b][i] = 0.0f;
  }
  // b1 enters the first product as one more MFMA step: A holds b1 of the
  // lane's hidden row split into two bf16 (hi = bf16(b1), lo = bf16(b1 - hi))
  // at k = 0, 1 and B holds ones there, so P^T starts at hi + lo (within about
  // 2^-16 |b1| of b1) and needs no zeroing or vector add.  bq[r] holds the
  // pair for the chunk of round r (lanes of group lg = 1 hold 0), shifted one
  // place per round.
  uint32_t bq[F::NR];
#pragma unroll
  for (int r = 0; r < F::NR; ++r) {
    const float v = p.b1 ? p.b1[32 * (2 * r + h) + ffn_hidden_row(lr)] : 0.0f;
    const float hi = __uint_as_float(pack_bf16x2(v, 0.0f) << 16);
    bq[r] = lg == 0 ? pack_bf16x2(hi, v - hi) : 0u;
  }
  const u32x4_t ones = {lg == 0 ? 0x3F803F80u : 0u, 0u, 0u, 0u};
  auto first_step = [&](f32x16_t& P) {
    const u32x4_t a = {bq[0], 0u, 0u, 0u};
    P = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, ones),
                                                f32x16_t{}, 0, 0, 0);
#pragma unroll
    for (int r = 0; r + 1 < F::NR; ++r) bq[r] = bq[r + 1];
  };

  issue(0, true, 0, false);

  // One pipeline round t: the first product of this half's chunk of round
  // t+1 (into Pn, if ONE), the second product of both chunks of round t-1
  // (own S from Sp, the partner's from Sx, if TWO) and the GELU of this
  // half's chunk of round t (on Pc, if GEL).  MFMAs of the two products
  // alternate; slot i issues MFMA i (if any) and GELU stage i % 8 of
  // elements 4 (i / 8) .. +3.  A fragments are read in groups of FG, each
  // group right after the first MFMA of the previous group.
  f32x16_t Pc, Pn;
  u32x4_t Sp[2], Sx[2];
  auto iter = [&](int t, auto one_t, auto two_t, auto gel_t) {
    constexpr bool ONE = decltype(one_t)::value, TWO = decltype(two_t)::value, GEL = decltype(gel_t)::value;
    constexpr int NM = (ONE ? F::NM1 : 0) + (TWO ? F::NM2 : 0);
    constexpr int NS = GEL ? (NM > F::GSLOTS ? NM : F::GSLOTS) : NM;
    constexpr int FG = F::FG;
    static_assert(!GEL || NS == F::GSLOTS, "one GELU stage per slot");
    const char* a1 = smem + ((t + 1) & 1) * F::W1S;
    const char* a2 = smem + F::OFF_W2 + ((t - 1) & 1) * F::W2S + nb0 * 32 * 128;
    auto is1 = [&](int i) { return ONE && (TWO ? (i & 1) == 0 : true); };
    auto idx = [&](int i) { return ONE && TWO ? i >> 1 : i; };
    // second-product op j: block nb0 + j % B2H, step j / (2 B2H), with this
    // half's chunk of round t-1 (S in Sp) if (j / B2H) is even, else the
    // partner's chunk (S in Sx)
    auto afrag = [&](int i) -> u32x4_t {
      const int j = idx(i);
      if (is1(i)) return lds_read16(a1 + o1(j & 3) + (j >> 2) * 64 * 128);
      const int b = j % F::B2H, own = ((j / F::B2H) & 1) == 0, s = j / (2 * F::B2H);
      return lds_read16(a2 + o2(own ? h : 1 - h, s) + b * 32 * 128);
    };
    if constexpr (ONE) first_step(Pn);
    u32x4_t fr[2][FG];
    GeluPipe gp;
#pragma unroll
    for (int k = 0; k < FG; ++k)
      if (k < NM) fr[0][k] = afrag(k);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      if (i < NM) {
        const u32x4_t& a = fr[(i / FG) & 1][i % FG];
        const int j = idx(i);
        if (is1(i)) {
          Mma<bf16_t>::run(Pn, a, xf[j]);
        } else {
          const bool own = ((j / F::B2H) & 1) == 0;
          const int s = j / (2 * F::B2H);
          Mma<bf16_t>::run(Oa[j % F::B2H], a, own ? Sp[s] : Sx[s]);
        }
        if (i % FG == 0) {
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int k = 0; k < FG; ++k) {
            const int nx = (i / FG + 1) * FG + k;
            if (nx < NM) fr[(i / FG + 1) & 1][k] = afrag(nx);
          }
        }
      }
      if constexpr (GEL) {
        const float x4[4] = {Pc[(i >> 3) * 4], Pc[(i >> 3) * 4 + 1], Pc[(i >> 3) * 4 + 2], Pc[(i >> 3) * 4 + 3]};
        float o4[4];
        gelu_stage(gp, x4, o4, i & 7);
        if ((i & 7) == 7) {
#pragma unroll
          for (int q = 0; q < 4; ++q) Pc[(i >> 3) * 4 + q] = o4[q];
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  char* xch_own = smem + F::OFF_X + ((pr * 2 + h) * 64 + lane) * 32;
  char* xch_par = smem + F::OFF_X + ((pr * 2 + (1 - h)) * 64 + lane) * 32;
  using T_ = std::true_type;
  using F_ = std::false_type;
  // Top of round t: W1^T of round t+1 and W2^T of round t-1 have landed and
  // every wave is done with the slots the next loads overwrite (W1^T of
  // round t, W2^T of round t-2); the partner's S of round t-1 is visible.
  auto top = [&](int t) {
    wait_vmcnt<0>();
    __syncthreads();
    issue(t + 2, t + 2 < F::NR, t, t < F::NR);
    if (t >= 1) {
      const char* src = xch_par + ((t - 1) & 1) * F::XCH;
      Sx[0] = lds_read16(src);
      Sx[1] = lds_read16(src + 16);
    }
  };
  // After round t: S of round t to registers and to the exchange; P of round t+1.
  auto rotate = [&](int t) {
    Sp[0] = ffn_pack_step(Pc, 0);
    Sp[1] = ffn_pack_step(Pc, 1);
    char* dst = xch_own + (t & 1) * F::XCH;
    lds_write16(dst, Sp[0]);
    lds_write16(dst + 16, Sp[1]);
    if (t + 1 < F::NR) Pc = Pn;
  };

  // Prologue: the first product of round 0, then round 0 (no second product yet).
  wait_vmcnt<0>();
  __syncthreads();
  // X^T fragments of this pair's 32 rows: xf[ks] = X[m][16 ks + 8 lg .. +8].
  {
    const int r = pr * 32 + lr;
    const char* xr = smem + F::OFF_W2 + r * 2 * D;
#pragma unroll
    for (int ks = 0; ks < F::KS1; ++ks) xf[ks] = lds_read16(xr + (((2 * ks + lg) ^ (r & XSW)) << 4));
  }
  // Residual R = X: O^T += I X^T, one MFMA per (block, k step) with an
  // identity fragment as A (exact: the products are x * 1 and x * 0).
  const bool r_is_x = p.R == p.X && p.ldr == p.ldx && (p.batch == 1 || p.sr == p.sx);
  if (p.R && r_is_x) {
    u32x4_t id[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int j = lr - 16 * e - 8 * lg;   // position of the 1 in this lane's 8 k values
#pragma unroll
      for (int w = 0; w < 4; ++w)
        id[e][w] = (j == 2 * w ? 0x3F80u : 0u) | (j == 2 * w + 1 ? 0x3F800000u : 0u);
    }
#pragma unroll
    for (int b = 0; b < F::B2H; ++b) {   // block nb0 + b takes X fragments 2 (nb0 + b) and 2 (nb0 + b) + 1
      Mma<bf16_t>::run(Oa[b], id[0], h ? xf[2 * (F::B2H + b)] : xf[2 * b]);
      Mma<bf16_t>::run(Oa[b], id[1], h ? xf[2 * (F::B2H + b) + 1] : xf[2 * b + 1]);
    }
  }

  if (F::NR > 1) issue(1, true, 0, false);
  iter(-1, T_{}, F_{}, F_{});
  Pc = Pn;
  top(0);
  if constexpr (F::NR > 1) iter(0, T_{}, F_{}, T_{});
  else iter(0, F_{}, F_{}, T_{});
  rotate(0);
#pragma unroll 1
  for (int t = 1; t + 1 < F::NR; ++t) {
    top(t);
    iter(t, T_{}, T_{}, T_{});
    rotate(t);
  }
  if constexpr (F::NR > 1) {
    top(F::NR - 1);
    iter(F::NR - 1, F_{}, T_{}, T_{});
    rotate(F::NR - 1);
  }
  top(F::NR);
  iter(F::NR, F_{}, T_{}, F_{});
  __syncthreads();

  // Epi2: residual (general R), then LayerNorm over the row, whose D values
  // sit in lanes (lr, lr + 32) of both halves of the pair.
  const bool mv = m < p.M;
  if (p.R && !r_is_x && mv) {
#pragma unroll
    for (int b = 0; b < F::B2H; ++b)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float r[4];
        load4_once<bf16_t>(p.R + (int64_t)bz * p.sr + (int64_t)m * p.ldr + (nb0 + b) * 32 + 8 * g + 4 * lg, r);
#pragma unroll
        for (int q = 0; q < 4; ++q) Oa[b][4 * g + q] += r[q];
      }
  }
  if (p.out_ln) {
    float* red = reinterpret_cast<float*>(smem + F::OFF_X);   // [stat 2][row group 4][half 2][row 32]
    auto pair_total = [&](float v, int stat) {
      v += __shfl_xor(v, 32);
      if (lg == 0) red[((stat * 4 + pr) * 2 + h) * 32 + lr] = v;
      __syncthreads();
      return red[((stat * 4 + pr) * 2 + 0) * 32 + lr] + red[((stat * 4 + pr) * 2 + 1) * 32 + lr];
    };
    float s4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int b = 0; b < F::B2H; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) s4[i & 3] += Oa[b][i];
    const float mean = pair_total((s4[0] + s4[1]) + (s4[2] + s4[3]), 0) * (1.0f / D);
    float q4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int b = 0; b < F::B2H; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        Oa[b][i] -= mean;
        q4[i & 3] = fmaf(Oa[b][i], Oa[b][i], q4[i & 3]);
      }
    const float rstd = rsqrtf(pair_total((q4[0] + q4[1]) + (q4[2] + q4[3]), 1) * (1.0f / D) + p.eps);
#pragma unroll
    for (int b = 0; b < F::B2H; ++b)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = (nb0 + b) * 32 + 8 * g + 4 * lg;
        f32x4_t ga = {1.0f, 1.0f, 1.0f, 1.0f}, be = {0.0f, 0.0f, 0.0f, 0.0f};
        if (p.gamma) ga = *reinterpret_cast<const f32x4_t*>(p.gamma + n);
        if (p.beta) be = *reinterpret_cast<const f32x4_t*>(p.beta + n);
#pragma unroll
        for (int q = 0; q < 4; ++q) Oa[b][4 * g + q] = fmaf(Oa[b][4 * g + q] * rstd, ga[q], be[q]);
      }
  }
  store_tile_staged<typename F::Out>(reinterpret_cast<f32x16_t(&)[1][F::B2H]>(Oa), p.O + (int64_t)bz * p.so, p.ldo, 0,
                                     p.M, D, m0, 0, smem, tid, lane, pr, h);
}

bool b2b_ffn_supported(int N1, int N2) {
  return (N1 == 512 && N2 == 256) || (N1 == 256 && N2 == 128) || (N1 == 128 && N2 == 64) ||
         (N1 == 256 && N2 == 256);
}

template <int N1, int D>
static hipError_t launch_ffn(const B2BParams& p, hipStream_t st) {
  using F = FfnShape<N1, D>;
  const dim3 grid((unsigned)((p.M + F::TM - 1) / F::TM), (unsigned)p.batch), block(F::NT);
  hipLaunchKernelGGL((b2b_ffn_kernel<N1, D>), grid, block, 0, st, p);
  return hipGetLastError();
}

hipError_t launch_b2b_ffn(const B2BParams& p, hipStream_t st) {
  if (p.N1 == 512 && p.N2 == 256) return launch_ffn<512, 256>(p, st);
  if (p.N1 == 256 && p.N2 == 256) return launch_ffn<256, 256>(p, st);
  if (p.N1 == 256 && p.N2 == 128) return launch_ffn<256, 128>(p, st);
  if (p.N1 == 128 && p.N2 == 64) return launch_ffn<128, 64>(p, st);
  return hipErrorInvalidValue;
}

}  // namespace cf
