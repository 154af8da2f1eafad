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

// Accumulator elements 8s .. 8s+7 of a block, as 8 packed bf16.
__device__ __forceinline__ u32x4_t pack_step(const f32x16_t& v, int s) {
  return u32x4_t{pack_bf16x2(v[8 * s + 0], v[8 * s + 1]), pack_bf16x2(v[8 * s + 2], v[8 * s + 3]),
                 pack_bf16x2(v[8 * s + 4], v[8 * s + 5]), pack_bf16x2(v[8 * s + 6], v[8 * s + 7])};
}

// Transposing 8-byte LDS read (ds_read_b64_tr_b16) at LDS byte address
// addr + OFF, written as inline assembly.  The compiler builtin carries no
// memory operand, so the compiler's wait insertion assumes it may read bytes
// that an outstanding direct-to-LDS load is still writing and puts a wait for
// every such load (vmcnt(0)) in front of it.  The caller knows the stage it
// reads is not the one being loaded; it waits for the result itself
// (lgkm_wait), since the compiler does not know this instruction loads.
template <int OFF>
__device__ __forceinline__ u32x2_t ds_read_tr_b64(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset field");
  u32x2_t v;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
  return v;
}
// 16-byte LDS read at byte address addr + OFF as inline assembly, for the
// same reason (K rows sit in a stage that direct loads also write); the
// caller waits for the result.
template <int OFF>
__device__ __forceinline__ u32x4_t ds_read_b128_at(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset field");
  u32x4_t v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
  return v;
}
// Wait until at most N LDS operations of this wave are outstanding; v is tied
// to the wait so that its uses cannot move above it.  The count is exact only
// while no scalar memory load is in flight (they share the counter and return
// out of order): the kernel's loop issues none, and each step begins with a
// full wait (lds_sync).
template <int N>
__device__ __forceinline__ void lgkm_wait(u32x4_t& v) {
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(v) : "i"(N));
}
// Calls f(std::integral_constant<int, I>) for I = B .. E-1 in order.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
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
  constexpr int NINS = A::TN / RPI / 4;   // direct loads per wave for one K or V block
  // Load ins of this wave for key block j (K, or V when v_t is true) into a
  // ring stage; `full` (block j lies inside Lk) selects the wave-uniform form.
  auto issue_one = [&](int j, auto stage_t, auto v_t, int ins, bool full) {
    constexpr bool VS = decltype(v_t)::value;
    char* dst = smem + decltype(stage_t)::value * A::STAGE + (VS ? A::KB : 0);
    const bf16_t* src = VS ? Vp : Kp;
    const int64_t ld = VS ? p.ldw2 : p.ldw1;
    const int in = wave + 4 * ins;
    if (full) {
      const char* base = reinterpret_cast<const char*>(src + (int64_t)(j * A::TN + in * RPI) * ld);
      dma16(base + (VS ? vl_off : kl_off), dst + in * 1024);
    } else {
      const int row = in * RPI + lane / LPR;
      const int c = (lane % LPR) ^ (VS ? vswz(row) : kswz(row));
      const int key = min(j * A::TN + row, Lk - 1);
      dma16(reinterpret_cast<const char*>(src + (int64_t)key * ld) + c * 16, dst + in * 1024);
    }
  };
  auto issue_kv = [&](int j, auto stage_t) {
    const bool full = (j + 1) * A::TN <= Lk;
#pragma unroll
    for (int ins = 0; ins < NINS; ++ins) issue_one(j, stage_t, std::false_type{}, ins, full);
#pragma unroll
    for (int ins = 0; ins < NINS; ++ins) issue_one(j, stage_t, std::true_type{}, ins, full);
  };
  auto lds_sync = [] {   // this wave's LDS accesses are done, then a workgroup barrier
    __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (3 << 14));
    lds_barrier();
  };

  // LDS byte address of K-fragment reads for d step ks (lane row lr of a
  // 32-key half; the half and the stage are compile-time offsets).  The
  // swizzle of row 32 h + lr equals that of row lr.
  uint32_t kbase[A::DK];
  // LDS byte address of the V^T fragment reads of output block b, less the
  // stage and key offsets (compile-time constants at each read).  In a group
  // of 16 lanes, lane r names 4 consecutive d (offset 4 (r % 4)) of key
  // k0 + r / 4, where k0 = 32 bl + 16 s + 4 lg is a multiple of 4, so the V
  // swizzle of that key depends on r only.
  uint32_t vbase[A::BD];
  {
    const int r = lane & 15;
    const int dcol = (lane & 16) + 4 * (r & 3);
    const int krow = 4 * lg + (r >> 2);
    const uint32_t s0 = (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) char*)smem);
#pragma unroll
    for (int ks = 0; ks < A::DK; ++ks) kbase[ks] = s0 + koff(lr, 2 * ks + lg);
#pragma unroll
    for (int b = 0; b < A::BD; ++b)
      vbase[b] = s0 + krow * A::KROW + ((((32 * b + dcol) >> 3) ^ vswz(krow)) << 4) + 8 * (r & 1);
  }

  f32x16_t Oa[A::BD];
#pragma unroll
  for (int b = 0; b < A::BD; ++b)
#pragma unroll
    for (int i = 0; i < 16; ++i) Oa[b][i] = 0.0f;
  float m_used = -INFINITY;
  // This lane's part of the row sum l of P (its 32 of each block's keys),
  // summed from the same bf16 P as the numerator by dot products with
  // (1, 1); the lane pair's parts are added at the end.
  float lsum = 0.0f;

  // One MFMA of an S^T block: 32-key half b, d step ks.
  auto mma_s = [&](f32x16_t (&S)[2], int b, int ks, u32x4_t kf) {
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
      lsum *= st.corr;
    }
  };
  // O^T += V^T P^T for block j (V^T fragments two MFMAs ahead).  Fragment
  // (b, s, bl) gives lane (lr, lg) V[k0 + 0..3][32 b + lr] and
  // V[k0 + 8 + 0..3][32 b + lr], k0 = 32 bl + 16 s + 4 lg: the permuted k order
  // of pack_step.  Each half comes from one ds_read_b64_tr_b16: in a group of
  // 16 lanes, lane r names 4 consecutive d of key k0 + r / 4 (d offset
  // 4 (r % 4)), and lane i receives the 4 keys of d offset i.
  auto pv_block = [&](auto stage_t, const SoftmaxStep& st) {
    constexpr int VT = decltype(stage_t)::value * A::STAGE + A::KB;   // this stage's V rows
    auto vfrag = [&](auto i_t) {   // i = (bl * 2 + s) * BD + b
      constexpr int i = decltype(i_t)::value;
      constexpr int b = i % A::BD, s = (i / A::BD) & 1, bl = i / (2 * A::BD);
      constexpr int off = VT + (32 * bl + 16 * s) * A::KROW;
      const u32x2_t lo = ds_read_tr_b64<off>(vbase[b]);
      const u32x2_t hi = ds_read_tr_b64<off + 8 * A::KROW>(vbase[b]);
      return u32x4_t{lo[0], lo[1], hi[0], hi[1]};
    };
    u32x4_t vf[3];
    vf[0] = vfrag(std::integral_constant<int, 0>{});
    vf[1] = vfrag(std::integral_constant<int, 1>{});
    static_for<0, A::NSB>([&](auto i_t) {
      constexpr int i = decltype(i_t)::value;
      constexpr int b = i % A::BD, s = (i / A::BD) & 1, bl = i / (2 * A::BD);
      // Two reads per fragment and no other LDS operation in between, so
      // fragment i is complete once at most fragment i + 1's two reads are
      // outstanding.  Fragment i + 2 is read after MFMA i, into the registers
      // MFMA i - 1 read.
      lgkm_wait<(i + 1 < A::NSB ? 2 : 0)>(vf[i % 3]);
      Mma<bf16_t>::run(Oa[b], vf[i % 3], st.P[bl][s]);
      if constexpr (i + 2 < A::NSB) vf[(i + 2) % 3] = vfrag(std::integral_constant<int, i + 2>{});
      __builtin_amdgcn_sched_barrier(0);
    });
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const bf16x2_t one2 = __builtin_bit_cast(bf16x2_t, 0x3F803F80u);   // bf16 (1.0, 1.0)
    // Each packed pair goes through a 32-bit value of its own: with the
    // vector element written inside the call, the compiler passed the
    // fragment's first register for all four pairs.
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t x = st.P[q >> 1][q & 1][e];
        lsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, x), one2, lsum, false);
      }
  };
  // S^T of block j from its K rows in LDS: one 16-byte read per MFMA, KLA
  // reads ahead; MFMA i takes half i % 2 and d step i / 2, so the two
  // halves' accumulation chains alternate.  No other LDS operation is issued
  // in between, so read i is complete once at most the KLA - 1 later ones
  // are outstanding.
  auto s_block = [&](f32x16_t (&S)[2], auto stage_t, auto&& after_mma) {
    constexpr int KST = decltype(stage_t)::value * A::STAGE;
    constexpr int KLA = 4;
    auto kread = [&](auto i_t) {
      constexpr int i = decltype(i_t)::value;
      constexpr int h = i % 2, ks = i / 2;
      return ds_read_b128_at<KST + h * 32 * A::KROW>(kbase[ks]);
    };
    u32x4_t kf[KLA];
    static_for<0, KLA>([&](auto i_t) { kf[decltype(i_t)::value] = kread(i_t); });
    static_for<0, A::NSA>([&](auto i_t) {
      constexpr int i = decltype(i_t)::value;
      constexpr int rest = A::NSA - 1 - i;
      lgkm_wait<(rest < KLA - 1 ? rest : KLA - 1)>(kf[i % KLA]);
      mma_s(S, i % 2, i / 2, kf[i % KLA]);
      if constexpr (i + KLA < A::NSA) kf[(i + KLA) % KLA] = kread(std::integral_constant<int, i + KLA>{});
      after_mma(i_t);
      __builtin_amdgcn_sched_barrier(0);
    });
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
  // and the P V of block j.  Two workgroups share a CU, so while one wave of
  // a SIMD runs the softmax the other (from the other workgroup) can issue
  // MFMAs.  The loop runs two blocks per trip so that the stage, and with it
  // every LDS offset, is a compile-time constant.
  // The next block's loads go one after every second MFMA of S^T(j): a
  // wave's load issue waits while the CU's load path takes earlier loads,
  // and MFMAs already issued keep the matrix core busy meanwhile (eight
  // loads in a row at the barrier cost a quarter of the step).
  static_assert(2 * NINS <= A::NSA / 2, "loads per S^T block");
  auto step = [&](int j, auto stage_t, auto next_t) {
    wait_vmcnt<0>();
    lds_sync();
    // Load q of the next block (K for q < NINS, then V) after MFMA 2 q + 1.
    auto loads = [&](auto full_t) {
      using FT = decltype(full_t);
      return [&](auto i_t) {
        constexpr int i = decltype(i_t)::value;
        if constexpr (i % 2 == 1 && i / 2 < 2 * NINS) {
          constexpr bool VS = i / 2 >= NINS;
          issue_one(j + 1, next_t, std::integral_constant<bool, VS>{}, VS ? i / 2 - NINS : i / 2, FT::value);
        }
      };
    };
    // The three cases are separate code paths so that the common one (the
    // next block lies inside Lk) keeps its wave-uniform addressing.
    if (j + 2 < NB || (j + 2 == NB && (j + 2) * A::TN <= Lk)) s_block(S, stage_t, loads(std::true_type{}));
    else if (j + 1 < NB) s_block(S, stage_t, loads(std::false_type{}));
    else s_block(S, stage_t, [](auto) {});
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
  const float inv = 1.0f / lane_pair_sum(lsum);
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
