// Back-to-back attention kernel for gfx950 (Sec. IV, Eq. 2 with F = scaled
// softmax: P = softmax(scale Q K^T), O = P V) with the intermediate P kept in
// registers.
//
// Register hand-off between the two products.  The first product is computed
// in the transposed form S^T = K Q^T, so in each 32x32 accumulator block a
// lane holds one query row m and 16 of its key columns: rows
// 8*(i/4) + 4*g + i%4 of the block for element i, g = lane/32.  The second
// product (O^T = V^T P^T) consumes P^T as its B operand, where lane group g
// supplies 8 values of the contraction index per MFMA step; step s takes
// accumulator elements 8s .. 8s+7 of the lane, so P never leaves the
// registers of the wave that produced it (the register-resident S_tile of
// Sec. IV-A).  The k order inside a step is free as long as both operands use
// the same one: step s of block b is DEFINED to use
//     n1(s, g, j) = 32 b + 16 s + 8 (j/4) + 4 g + j%4,   j = 0..7,
// and the V operand is read from LDS as two 8-byte pieces per lane in that
// same order.
//
// Each wave owns 32 complete query rows, so the softmax statistics need only
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
// Attention: O = softmax(scale * Q K^T) V per (batch*head), online softmax.
// 4 waves x 32 queries = 128 queries per workgroup; key/value blocks of 64.
// Q fragments stay in registers for the whole sweep.  Per block j:
//   S^T = K Q^T (K rows from LDS); lane-local row max / sum over its 32
//   values + the lane pair; P = exp2(S*scale*log2e - m); O = O*corr + P V
//   with P fed from registers and V^T rows from LDS.
// Two workgroups share a CU (at most 256 VGPRs per wave), so each SIMD runs
// two waves of different workgroups, which no barrier holds in step: one
// wave's softmax overlaps the other's MFMAs (the PingPong of Sec. III-C across
// waves rather than inside one).
// The running maximum is raised lazily: O and the row sum are rescaled only
// when a block's maximum exceeds the one in use by more than 2^8, so
// exp2(s - m) <= 256 and the common case skips the rescale; the final O / l
// uses the same maximum throughout, so the result is unchanged.
// K and V blocks arrive by wave-wide direct loads, both key-major; the
// second product reads V^T fragments with transposing LDS reads.
// ===========================================================================
template <int D>
struct AttnShape {
  static constexpr int TM = 128, TN = 64, NT = 256;
  static constexpr int KB = TN * D * 2;           // K block bytes (TN rows of D*2 bytes)
  static constexpr int VB = TN * D * 2;           // V block bytes (TN rows of D*2 bytes)
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
  float bmax, corr;
  bool need;
  u32x4_t P[2][2];   // bf16 P^T fragments: [32-key half][MFMA step]
};

template <int D>
__global__ __launch_bounds__(256, 2) void b2b_attention_kernel(B2BParams p) {
  using A = AttnShape<D>;
  __shared__ __attribute__((aligned(16))) char smem[A::LDS];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
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
  // V rows in LDS as they are in memory (key-major, D*2 bytes), 16-byte chunk
  // c of key row k at position c ^ vswz(k).  The second product reads V^T
  // fragments with transposing LDS reads (see vfrag), and this swizzle keeps
  // each 32-lane half of such a read on distinct banks.
  auto vswz = [](int k) { return A::KCH == 16 ? 4 * (k & 3) : 4 * ((k >> 1) & 1); };
  constexpr int LPR = A::KCH;                   // lanes per row in one wave-wide load
  constexpr int RPI = 64 / LPR;                 // rows per instruction
  // Wave-wide direct loads of key block j (K, or V when v_t is true) into a
  // ring stage.  Load ins of a wave covers rows in * RPI .. + RPI - 1, in =
  // wave + 4 ins; both swizzles depend on the row only through
  // (row & 15) = (4 wave + lane / LPR) & 15 (d = 128) or the row pair
  // ((row >> 1) & 7, d = 64), which does not change with ins, so the lane's
  // byte offset inside its rows is fixed and the rest is wave-uniform.  Rows
  // past Lk (the last block only) are clamped, and masked out of P.
  const int row0 = wave * RPI + lane / LPR;     // this lane's row in load 0
  const uint32_t kl_off = (uint32_t)((lane / LPR) * p.ldw1 * 2 + (((lane % LPR) ^ kswz(row0)) << 4));
  const uint32_t vl_off = (uint32_t)((lane / LPR) * p.ldw2 * 2 + (((lane % LPR) ^ vswz(row0)) << 4));
  auto issue_rows = [&](int j, auto stage_t, auto v_t) {
    constexpr bool VS = decltype(v_t)::value;
    char* dst = smem + decltype(stage_t)::value * A::STAGE + (VS ? A::KB : 0);
    const bf16_t* src = VS ? Vp : Kp;
    const int64_t ld = VS ? p.ldw2 : p.ldw1;
    if ((j + 1) * A::TN <= Lk) {
#pragma unroll
      for (int ins = 0; ins < A::TN / RPI / 4; ++ins) {
        const int in = wave + 4 * ins;
        const char* base = reinterpret_cast<const char*>(src + (int64_t)(j * A::TN + in * RPI) * ld);
        dma16(base + (VS ? vl_off : kl_off), dst + in * 1024);
      }
    } else {
#pragma unroll
      for (int ins = 0; ins < A::TN / RPI / 4; ++ins) {
        const int in = wave + 4 * ins;
        const int row = in * RPI + lane / LPR;
        const int c = (lane % LPR) ^ (VS ? vswz(row) : kswz(row));
        const int key = min(j * A::TN + row, Lk - 1);
        dma16(reinterpret_cast<const char*>(src + (int64_t)key * ld) + c * 16, dst + in * 1024);
      }
    }
  };
  auto issue_kv = [&](int j, auto stage_t) {
    issue_rows(j, stage_t, std::false_type{});
    issue_rows(j, stage_t, std::true_type{});
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
  float m_used = -INFINITY;
  // Row sums l of P, accumulated by MFMAs with an all-ones A operand (every
  // row of the block holds l of query lr), from the same bf16 P as O.
  f32x16_t Lacc = {};

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
      }
    } else if (c == 14) {
      st.P[0][0] = pack_step(S[0], 0);
      st.P[0][1] = pack_step(S[0], 1);
    } else {
      st.P[1][0] = pack_step(S[1], 0);
      st.P[1][1] = pack_step(S[1], 1);
    }
  };
  auto rescale = [&](const SoftmaxStep& st) {
    if (__any(st.need)) {
#pragma unroll
      for (int b = 0; b < A::BD; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) Oa[b][i] *= st.corr;
#pragma unroll
      for (int i = 0; i < 16; ++i) Lacc[i] *= st.corr;
    }
  };
  // O^T += V^T P^T for block j (V^T fragments two MFMAs ahead).  Fragment
  // (b, s, bl) gives lane (lr, lg) V[k0 + 0..3][32 b + lr] and
  // V[k0 + 8 + 0..3][32 b + lr], k0 = 32 bl + 16 s + 4 lg: the permuted k order
  // of pack_step.  Each half comes from one ds_read_b64_tr_b16: in a group of
  // 16 lanes, lane r names 4 consecutive d of key k0 + r / 4 (d offset
  // 4 (r % 4)), and lane i receives the 4 keys of d offset i.
  auto pv_block = [&](auto stage_t, const SoftmaxStep& st) {
    const char* vt = smem + decltype(stage_t)::value * A::STAGE + A::KB;
    const int r = lane & 15;
    const int dcol = (lane & 16) + 4 * (r & 3);       // d within the 32-block named by this lane
    const int hb = 8 * (r & 1);
    auto tr_read = [&](int key, int d) {
      typedef short v4i16 __attribute__((ext_vector_type(4)));
      const char* a = vt + key * A::KROW + (((d >> 3) ^ vswz(key)) << 4) + hb;
      const v4i16 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) v4i16*)(a));
      return __builtin_bit_cast(u32x2_t, v);
    };
    auto vfrag = [&](int i) {   // i = (bl * 2 + s) * BD + b
      const int b = i % A::BD, s = (i / A::BD) & 1, bl = i / (2 * A::BD);
      const int k0 = 32 * bl + 16 * s + 4 * lg + (r >> 2);
      const u32x2_t lo = tr_read(k0, 32 * b + dcol);
      const u32x2_t hi = tr_read(k0 + 8, 32 * b + dcol);
      return u32x4_t{lo[0], lo[1], hi[0], hi[1]};
    };
    u32x4_t vf[3];
    vf[0] = vfrag(0);
    vf[1] = vfrag(1);
#pragma unroll
    for (int i = 0; i < A::NSB; ++i) {
      if (i + 2 < A::NSB) vf[(i + 2) % 3] = vfrag(i + 2);
      const int b = i % A::BD, s = (i / A::BD) & 1, bl = i / (2 * A::BD);
      Mma<bf16_t>::run(Oa[b], vf[i % 3], st.P[bl][s]);
      __builtin_amdgcn_sched_barrier(0);
    }
    const u32x4_t ones = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};   // bf16 1.0 x 8
#pragma unroll
    for (int q = 0; q < 4; ++q) Mma<bf16_t>::run(Lacc, ones, st.P[q >> 1][q & 1]);
  };
  // S^T of block j from its K rows in LDS (K fragments two MFMAs ahead).
  auto s_block = [&](f32x16_t (&S)[2], auto stage_t) {
    const char* kb = smem + decltype(stage_t)::value * A::STAGE;
    u32x4_t kf[3];
    kf[0] = kfrag(kb, 0);
    kf[1] = kfrag(kb, 1);
#pragma unroll
    for (int i = 0; i < A::NSA; ++i) {
      if (i + 2 < A::NSA) kf[(i + 2) % 3] = kfrag(kb, i + 2);
      mma_s(S, i, kf[i % 3]);
    }
  };
  auto softmax_all = [&](f32x16_t (&Sc)[2], int j, SoftmaxStep& st, auto mask_t) {
#pragma unroll
    for (int c = 0; c < 16; ++c) sm_chunk(Sc, c, st, j, mask_t);
  };

  f32x16_t S[2];
  SoftmaxStep st;
  // Prologue: K and V of block 0 on their way into LDS stage 0.
  using S0_ = std::integral_constant<int, 0>;
  using S1_ = std::integral_constant<int, 1>;
  issue_kv(0, S0_{});
  // Step j: K(j) and V(j) are in stage j & 1 once every wave has passed the
  // barrier, and every wave is then done with block j-1, so stage (j+1) & 1
  // takes K(j+1) and V(j+1) (direct loads).  Then S^T(j), softmax, rescale
  // and the P V of block j.  Two workgroups share a
  // CU, so while one wave of a SIMD runs the softmax the other (from the other
  // workgroup) can issue MFMAs.  The loop runs two blocks per trip so that the
  // stage, and with it every LDS offset, is a compile-time constant.
  auto step = [&](int j, auto stage_t, auto next_t) {
    wait_vmcnt<0>();
    lds_sync();
    if (j + 1 < NB) issue_kv(j + 1, next_t);
    s_block(S, stage_t);
    if (j + 1 < NB) softmax_all(S, j, st, std::false_type{});
    else softmax_all(S, j, st, std::true_type{});
    rescale(st);
    pv_block(stage_t, st);
  };
  for (int j = 0; j < NB; j += 2) {
    step(j, S0_{}, S1_{});
    if (j + 1 < NB) step(j + 1, S1_{}, S0_{});
  }

  __syncthreads();
  const float inv = 1.0f / Lacc[0];
#pragma unroll
  for (int b = 0; b < A::BD; ++b)
#pragma unroll
    for (int i = 0; i < 16; ++i) Oa[b][i] *= inv;
  store_tile_staged<typename A::Out>(reinterpret_cast<f32x16_t(&)[1][A::BD]>(Oa), p.O + (int64_t)bz * p.so, p.ldo, 0, p.M, D, m0, 0, smem, tid, lane,
                                     wave, 0);
}

// ---------------------------------------------------------------------------
bool b2b_attention_supported(int d) { return d == 64 || d == 128; }

hipError_t launch_b2b_attention(const B2BParams& p, hipStream_t st) {
  const dim3 grid((unsigned)((p.M + 127) / 128), (unsigned)p.batch), block(256);
  if (p.K == 128) hipLaunchKernelGGL((b2b_attention_kernel<128>), grid, block, 0, st, p);
  else if (p.K == 64) hipLaunchKernelGGL((b2b_attention_kernel<64>), grid, block, 0, st, p);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace cf
