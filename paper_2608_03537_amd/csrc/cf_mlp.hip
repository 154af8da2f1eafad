// Back-to-back MLP for gfx950 (Sec. IV, Eq. 2 with F = ReLU(. + b1);
// Sec. IV-A): O = ReLU(X W1 + b1) W2 + b2, optionally ReLU(O) -- the DLRM
// bottom-MLP pattern of Table 2 (1024 -> 512 -> 128).
//
// Work split (the cross-workgroup dataflow of Sec. IV-A).  The hidden
// dimension N1 is split into chunks of 256 units; the cn = N1 / 256
// workgroups of a 128-row block each own one chunk c:
//   ML1   P_c^T = W1_c^T X^T on the direct-to-LDS ring of the GEMM kernels
//         (the accumulators start from b1, so they hold P_c + b1_c);
//   Epi1  S_c = ReLU(.) packed to bf16 in registers;
//   ML2   O_c = S_c W2_c, the partial second product over the chunk, with
//         the W2^T chunk staged in LDS;
//   Epi2  O = sum_c O_c + b2 (the partial-sum identity of Sec. IV-A), summed
//         at commit: each workgroup publishes O_c, the last one of its row
//         block to arrive adds the partials in the fixed order c = 0, 1, ...
//         and stores O.  No workgroup waits for another, so no co-residency
//         is needed, and the result does not depend on the arrival order.
//
// Register hand-off.  The rows of each 32-row block of W1_c^T are loaded with
// bits 2 and 3 of the row index swapped (perm23), so accumulator elements
// 8s .. 8s+7 of lane half g hold hidden units 16s + 8g + 0..7 of the block.
// Packed to bf16 they are the B operand of one MFMA step of the second
// product O^T = W2^T S^T, whose A operand is then one contiguous 16-byte piece
// of a W2^T row (k order inside an MFMA step is free as long as both operands
// use the same one).
//
// Commit visibility.  Partials are written with agent-scope stores, the
// writer waits for their completion before its arrival add (agent scope), and
// the last arriver reads them with agent-scope loads issued after its add
// returned: every access involved is device-coherent, so no cache flush is
// needed.  The arrival counter of a row block goes back to 0 at the end of
// the call (the last arriver resets it), so a zero-filled counter area stays
// valid for every later call.
#include "cf_gemm_tile.h"
#include "comfuse.h"

namespace cf {

using MlpS = TileShape<bf16_t, 2, 4, 2, 2, 128, 3>;   // 128 rows x 256 hidden units, 4 waves (2 x 2)
static_assert(MlpS::TM == kMlpRows && MlpS::TN == kMlpHidden, "MLP tile");

template <int N2>
struct MlpLayout {
  static constexpr int NB2 = N2 / 32;                 // output column blocks
  static constexpr int W2_ROWB = kMlpHidden * 2;      // bytes of one W2^T chunk row
  static constexpr int W2_BYTES = N2 * W2_ROWB;       // W2^T chunk in LDS
  static constexpr int OFF_RED = W2_BYTES;            // partial sums of the wn = 1 waves
  static constexpr int RED_WAVE = 64 * N2 * 4;        // one wave's 64 rows x N2 fp32
  static constexpr int W2_LOADS = W2_BYTES / 1024;    // wave-wide 1 KB loads
  static constexpr int PT_ROWB = N2 * 4;              // row-major fp32 partial tile (over the W2 chunk)
  static constexpr int OFF_FLAG = OFF_RED + 2 * RED_WAVE;   // "this workgroup commits" flag
  static_assert(OFF_FLAG + 16 <= MlpS::SMEM_V2, "flag in LDS");
  static_assert(kMlpRows * PT_ROWB <= OFF_RED, "partial tile fits the W2 region");
  static_assert(OFF_RED + 2 * RED_WAVE <= MlpS::SMEM_V2, "LDS budget");
  static_assert(W2_LOADS % MlpS::NW == 0, "W2 loads per wave");
};

template <int N2>
__global__ __launch_bounds__(MlpS::NT, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
void b2b_mlp_kernel(B2BParams p) {
  using S = MlpS;
  using L = MlpLayout<N2>;
  constexpr int NB2 = L::NB2;
  // One LDS array only: a second __shared__ object makes the compiler wait
  // for every outstanding direct-to-LDS load before each LDS read of the main
  // loop (it can no longer tell the loads' targets apart).
  __shared__ __attribute__((aligned(16))) char smem[S::SMEM_V2];
  int& last_flag = *reinterpret_cast<int*>(smem + L::OFF_FLAG);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / S::WN, wn = wave % S::WN;
  const int lr = lane & 31, lg = lane >> 5;
  const int cn = p.cn;
  // XCD-aware order: linear id L runs on XCD L % 8.  In full groups of 8 row
  // blocks, the cn workgroups of row block 8 i + x are L = 8 (cn i + c) + x:
  // they share XCD x and run at about the same time, so the row block's X
  // comes from HBM into that XCD's L2 once for all its chunks.  The rows past
  // the last full group go in plain order.
  int c, rb;
  {
    const int L = blockIdx.x, full = (int)(gridDim.x / cn) / 8 * 8 * cn;
    if (L < full) {
      c = (L >> 3) % cn;
      rb = (L >> 3) / cn * 8 + (L & 7);
    } else {
      c = (L - full) % cn;
      rb = full / cn + (L - full) / cn;
    }
  }
  const int m0 = rb * S::TM, h0 = c * kMlpHidden;
  const int bz = blockIdx.y;
  const bf16_t* X = p.X + (int64_t)bz * p.sx;
  const bf16_t* W1 = p.W1 + (int64_t)bz * p.sw1;
  const bf16_t* W2 = p.W2 + (int64_t)bz * p.sw2;

  // ---- ML1 (+ b1): P_c^T on the ring, hidden rows in perm23 order
  GemmRowsParams g{};
  g.batch = 1;
  g.M = p.M;
  g.N = p.N1;
  g.K = p.K;
  g.X = X;
  g.ldx = p.ldx;
  g.W = W1;
  g.ldw = p.ldw1;
  g.w_nk = 1;
  g.epi.alpha = 1.0f;
  g.epi.bias = p.b1;
  f32x16_t acc[S::BM][S::BN];
  mainloop_v2<S, false, true>(acc, X, W1, g, m0, h0, 0, smem, lane, wave, wm, wn, p.b1 != nullptr);

  // ---- W2^T chunk (N2 rows x 256 hidden) to LDS; 16-byte chunk q of row r
  // at position q ^ (r & 15), so the 16 rows a 16-lane group reads spread over
  // all banks.  The ring is free after the main loop's final barrier.
#pragma unroll
  for (int j = 0; j < L::W2_LOADS / S::NW; ++j) {
    const int ld = wave + j * S::NW;                  // one load = two W2^T rows
    const int r = 2 * ld + (lane >> 5);
    const int q = (lane & 31) ^ (r & 15);
    dma16(W2 + (int64_t)r * p.ldw2 + h0 + q * 8, smem + ld * 1024);
  }

  // ---- Epi1: S = ReLU(P + b1), packed bf16, the B operands of ML2
  u32x4_t sf[S::BM][S::BN][2];
#pragma unroll
  for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
    for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int w = 0; w < 4; ++w)
          sf[bm][bn][s][w] = pack_bf16x2(fmaxf(acc[bm][bn][8 * s + 2 * w], 0.0f),
                                         fmaxf(acc[bm][bn][8 * s + 2 * w + 1], 0.0f));
  wait_vmcnt<0>();
  __syncthreads();

  // ---- ML2: O_c partial over this wave's 128 hidden units (wave column wn)
  f32x16_t o[S::BM][NB2];
#pragma unroll
  for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
    for (int b2 = 0; b2 < NB2; ++b2)
#pragma unroll
      for (int i = 0; i < 16; ++i) o[bm][b2][i] = 0.0f;
#pragma unroll
  for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int q = (wn * S::WTN + bn * 32 + 16 * s + 8 * lg) / 8;
      u32x4_t a[NB2];
#pragma unroll
      for (int b2 = 0; b2 < NB2; ++b2) {
        const int r = b2 * 32 + lr;
        a[b2] = lds_read16(smem + r * L::W2_ROWB + ((q ^ (r & 15)) << 4));
      }
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
        for (int b2 = 0; b2 < NB2; ++b2) Mma<bf16_t>::run(o[bm][b2], a[b2], sf[bm][bn][s]);
    }

  // ---- the two wave columns of a row group add their halves (wn = 0 keeps the sum)
  char* red = smem + L::OFF_RED + wm * L::RED_WAVE;
  auto red_at = [&](int bm, int b2, int gq) { return red + (((bm * NB2 + b2) * 4 + gq) * 64 + lane) * 16; };
  if (wn == 1) {
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
      for (int b2 = 0; b2 < NB2; ++b2)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq)
          *reinterpret_cast<f32x4_t*>(red_at(bm, b2, gq)) =
              f32x4_t{o[bm][b2][4 * gq], o[bm][b2][4 * gq + 1], o[bm][b2][4 * gq + 2], o[bm][b2][4 * gq + 3]};
  }
  __syncthreads();
  if (wn == 0) {
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
      for (int b2 = 0; b2 < NB2; ++b2)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
          const f32x4_t v = *reinterpret_cast<const f32x4_t*>(red_at(bm, b2, gq));
#pragma unroll
          for (int e = 0; e < 4; ++e) o[bm][b2][4 * gq + e] += v[e];
        }
  }

  // ---- the workgroup's partial O_c (128 rows x N2 fp32) to LDS, row-major
  // with 16-byte chunk q of row r at position q ^ (r & 31) (the W2 chunk
  // region is free: every wave passed the barrier above after its last read).
  // Accumulator element 4 gq + e of block (bm, b2): row wm 64 + bm 32 + lr,
  // column b2 32 + 8 gq + 4 lg + e.
  auto pt_at = [&](int r, int q) { return smem + r * L::PT_ROWB + ((q ^ (r & 31)) << 4); };
  if (wn == 0) {
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
      for (int b2 = 0; b2 < NB2; ++b2)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq)
          *reinterpret_cast<f32x4_t*>(pt_at(wm * S::WTM + bm * 32 + lr, b2 * 8 + 2 * gq + lg)) =
              f32x4_t{o[bm][b2][4 * gq], o[bm][b2][4 * gq + 1], o[bm][b2][4 * gq + 2], o[bm][b2][4 * gq + 3]};
  }
  __syncthreads();

  // ---- Epi2 (commit) over the row-major tile: thread t handles the column
  // quad (t + 256 j) % QPR of row (t + 256 j) / QPR, so every wave-wide
  // access covers two whole rows: 1 KB of partials, 512 bytes of O.
  // The partials go through memory with device-coherent 16-byte accesses
  // (sc1): the workgroups of a row block need not share an XCD, and the
  // reader reads only after the writer's stores completed (arrival count).
  constexpr int QPR = N2 / 4;                          // column quads per row
  constexpr int QUADS = S::TM * QPR / S::NT;           // quads per thread
  static_assert(S::NT % QPR == 0, "a thread's column quad is the same in every step");
  constexpr int kSc1 = 16;                             // cache policy: device-coherent
  const int q4 = tid % QPR;
  auto quad_lds = [&](int j) { return *reinterpret_cast<const f32x4_t*>(pt_at((tid + j * S::NT) / QPR, q4)); };
  float* part = p.ws_part + (int64_t)bz * cn * p.M * N2;
  const int rows = min(S::TM, p.M - m0);
  // Buffer resource over chunk k's partial rows [m0, m0 + rows): raw 32-bit
  // data; accesses past its end are dropped (stores) or read as 0 (loads).
  auto part_rsrc = [&](int k) {
    return __builtin_amdgcn_make_buffer_rsrc(part + ((int64_t)k * p.M + m0) * N2, 0, rows * N2 * 4, 0x00020000);
  };
  if (cn > 1) {
    // publish O_c, then count this workgroup's arrival
    const auto mine = part_rsrc(c);
#pragma unroll 8
    for (int j = 0; j < QUADS; ++j) {
      const int r = (tid + j * S::NT) / QPR;
      if (r < rows)
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, quad_lds(j)), mine, (r * QPR + q4) * 16, 0,
                                               kSc1);
    }
    wait_vmcnt<0>();          // this wave's partial stores have completed
    __syncthreads();          // ... and every wave's
    if (tid == 0) {
      unsigned* cnt = p.ws_count + (int64_t)bz * (gridDim.x / cn) + rb;
      const unsigned old = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int last = old == (unsigned)(cn - 1);
      if (last) __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);   // ready for the next call
      last_flag = last;
    }
    __syncthreads();
    if (!last_flag) return;   // the last workgroup of the row block commits
  }

  // O = O_0 + O_1 + ... (chunk order, whichever workgroup finished last; its
  // own partial comes from LDS, equal to what it stored) + b2, output ReLU,
  // bf16 rows.  A thread's column quad is the same in every step, so b2 is
  // read once; the other chunks' partials are loaded for all steps before
  // any is used, so their latencies overlap.
  uint16_t* O = p.O + (int64_t)bz * p.so;
  f32x4_t bb = {0.0f, 0.0f, 0.0f, 0.0f};
  if (p.b2) bb = *reinterpret_cast<const f32x4_t*>(p.b2 + 4 * q4);
  f32x4_t t[QUADS];
#pragma unroll
  for (int j = 0; j < QUADS; ++j) t[j] = quad_lds(j);
  if (cn > 1) {
    f32x4_t acc2[QUADS];
    for (int k = 0; k < cn; ++k) {
      if (k == c) {
#pragma unroll
        for (int j = 0; j < QUADS; ++j) acc2[j] = k == 0 ? t[j] : acc2[j] + t[j];
        continue;
      }
      const auto src = part_rsrc(k);
      u32x4_t w[QUADS];
#pragma unroll
      for (int j = 0; j < QUADS; ++j) {
        const int r = min((tid + j * S::NT) / QPR, rows - 1);
        w[j] = __builtin_amdgcn_raw_buffer_load_b128(src, (r * QPR + q4) * 16, 0, kSc1);
      }
#pragma unroll
      for (int j = 0; j < QUADS; ++j) {
        const f32x4_t v = __builtin_bit_cast(f32x4_t, w[j]);
        acc2[j] = k == 0 ? v : acc2[j] + v;
      }
    }
#pragma unroll
    for (int j = 0; j < QUADS; ++j) t[j] = acc2[j];
  }
#pragma unroll
  for (int j = 0; j < QUADS; ++j) {
    const int m = m0 + (tid + j * S::NT) / QPR;
    if (m >= p.M) continue;
    f32x4_t y = t[j];
    if (p.b2) y += bb;
    if (p.out_relu)
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = fmaxf(y[e], 0.0f);
    const u32x2_t o2 = {pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3])};
    __builtin_nontemporal_store(o2, reinterpret_cast<u32x2_t*>(O + (int64_t)m * p.ldo + 4 * q4));
  }
}

// Whole-row-block form: one workgroup per 128-row block runs the N1 / 256
// chunks in turn and accumulates the partial second products O_c in
// registers, in chunk order, so nothing goes through memory.  For the second
// product a wave takes its 64 rows and half of the N2 output columns over all
// 256 hidden units of the chunk: its own S half from registers, its wave-
// column partner's half from LDS.  So each output element has one owner (no
// reduction across waves), and a wave keeps 64 accumulator registers live
// across the next chunk's first product.  It needs as many row blocks as
// the split form has workgroups to fill the chip; the host takes it when the
// row blocks alone fill every CU.
template <int N2>
__global__ __launch_bounds__(MlpS::NT, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
void b2b_mlp_whole_kernel(B2BParams p) {
  using S = MlpS;
  using L = MlpLayout<N2>;
  constexpr int NB2 = L::NB2, HB2 = NB2 / 2;        // output blocks: all, per wave column
  constexpr int OFF_XS = L::W2_BYTES;               // S exchange: [wave 4][bm][bn][s][lane 64][16 B]
  constexpr int XS_WAVE = S::BM * S::BN * 2 * 1024;
  static_assert(OFF_XS + 4 * XS_WAVE <= S::SMEM_V2 && S::TM * L::PT_ROWB <= S::SMEM_V2, "LDS budget");
  __shared__ __attribute__((aligned(16))) char smem[S::SMEM_V2];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / S::WN, wn = wave % S::WN;
  const int lr = lane & 31, lg = lane >> 5;
  const int rb = blockIdx.x, m0 = rb * S::TM;
  const int bz = blockIdx.y;
  const bf16_t* X = p.X + (int64_t)bz * p.sx;
  const bf16_t* W1 = p.W1 + (int64_t)bz * p.sw1;
  const bf16_t* W2 = p.W2 + (int64_t)bz * p.sw2;
  GemmRowsParams g{};
  g.batch = 1;
  g.M = p.M;
  g.N = p.N1;
  g.K = p.K;
  g.X = X;
  g.ldx = p.ldx;
  g.W = W1;
  g.ldw = p.ldw1;
  g.w_nk = 1;
  g.epi.alpha = 1.0f;
  g.epi.bias = p.b1;

  // O^T blocks (bm, h): rows wm 64 + bm 32 + lr, output columns (wn HB2 + h) 32 + ...
  f32x16_t o[S::BM][HB2];
#pragma unroll
  for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
    for (int h = 0; h < HB2; ++h)
#pragma unroll
      for (int i = 0; i < 16; ++i) o[bm][h][i] = 0.0f;
  char* xs_own = smem + OFF_XS + wave * XS_WAVE + lane * 16;
  const char* xs_par = smem + OFF_XS + (wm * S::WN + (1 - wn)) * XS_WAVE + lane * 16;
  const int cn = p.N1 / kMlpHidden;
  for (int c = 0; c < cn; ++c) {
    const int h0 = c * kMlpHidden;
    // ML1 (+ b1) of chunk c.  Its ring prologue writes LDS at once: the
    // barrier that ends the previous chunk keeps it behind every wave's
    // reads of that chunk's W2^T and S exchange.  The row offset is opaque
    // to the compiler here, so the ring's X addresses are formed per chunk
    // instead of being hoisted and kept live (spilled) across the loop.
    int m0c = m0;
    asm volatile("" : "+s"(m0c));
    f32x16_t acc[S::BM][S::BN];
    mainloop_v2<S, false, true>(acc, X, W1, g, m0c, h0, 0, smem, lane, wave, wm, wn, p.b1 != nullptr);
    // W2^T chunk to LDS (layout as in the split form)
#pragma unroll
    for (int j = 0; j < L::W2_LOADS / S::NW; ++j) {
      const int ld = wave + j * S::NW;
      const int r = 2 * ld + (lane >> 5);
      const int q = (lane & 31) ^ (r & 15);
      dma16(W2 + (int64_t)r * p.ldw2 + h0 + q * 8, smem + ld * 1024);
    }
    // Epi1: S = ReLU(P + b1), packed bf16 (hidden units wn 128 + bn 32 +
    // 16 s + 8 lg + 0..7 of the chunk), and to the partner through LDS
    u32x4_t sf[S::BM][S::BN][2];
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int s = 0; s < 2; ++s) {
#pragma unroll
          for (int w = 0; w < 4; ++w)
            sf[bm][bn][s][w] = pack_bf16x2(fmaxf(acc[bm][bn][8 * s + 2 * w], 0.0f),
                                           fmaxf(acc[bm][bn][8 * s + 2 * w + 1], 0.0f));
          lds_write16(xs_own + ((bm * S::BN + bn) * 2 + s) * 1024, sf[bm][bn][s]);
        }
    wait_vmcnt<0>();
    __syncthreads();
    // ML2: O += S_c W2_c over all 256 hidden units of the chunk, half e of
    // them (e = wn: own registers, else the partner's LDS copy)
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          const int q = (e * S::WTN + bn * 32 + 16 * s + 8 * lg) / 8;
          u32x4_t a[HB2], b[S::BM];
#pragma unroll
          for (int h = 0; h < HB2; ++h) {
            const int r = (wn * HB2 + h) * 32 + lr;
            a[h] = lds_read16(smem + r * L::W2_ROWB + ((q ^ (r & 15)) << 4));
          }
#pragma unroll
          for (int bm = 0; bm < S::BM; ++bm)
            b[bm] = e == wn ? sf[bm][bn][s] : lds_read16(xs_par + ((bm * S::BN + bn) * 2 + s) * 1024);
#pragma unroll
          for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
            for (int h = 0; h < HB2; ++h) Mma<bf16_t>::run(o[bm][h], a[h], b[bm]);
        }
    __syncthreads();   // every wave is done with the W2^T chunk and the S exchange
  }

  // O to LDS, row-major fp32 with 16-byte chunk q of row r at position
  // q ^ (r & 31); element 4 gq + e of block (bm, h): row wm 64 + bm 32 + lr,
  // column (wn HB2 + h) 32 + 8 gq + 4 lg + e.
  auto pt_at = [&](int r, int q) { return smem + r * L::PT_ROWB + ((q ^ (r & 31)) << 4); };
#pragma unroll
  for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
    for (int h = 0; h < HB2; ++h)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq)
        *reinterpret_cast<f32x4_t*>(pt_at(wm * S::WTM + bm * 32 + lr, (wn * HB2 + h) * 8 + 2 * gq + lg)) =
            f32x4_t{o[bm][h][4 * gq], o[bm][h][4 * gq + 1], o[bm][h][4 * gq + 2], o[bm][h][4 * gq + 3]};
  __syncthreads();
  // O + b2 (ReLU) as bf16 rows: thread t takes column quad t % QPR of rows
  // (t + 256 j) / QPR, so every wave-wide store covers two whole rows.
  constexpr int QPR = N2 / 4;
  constexpr int QUADS = S::TM * QPR / S::NT;
  static_assert(S::NT % QPR == 0, "a thread's column quad is the same in every step");
  const int q4 = tid % QPR;
  uint16_t* O = p.O + (int64_t)bz * p.so;
  f32x4_t bb = {0.0f, 0.0f, 0.0f, 0.0f};
  if (p.b2) bb = *reinterpret_cast<const f32x4_t*>(p.b2 + 4 * q4);
#pragma unroll
  for (int j = 0; j < QUADS; ++j) {
    const int r = (tid + j * S::NT) / QPR, m = m0 + r;
    if (m >= p.M) continue;
    f32x4_t y = *reinterpret_cast<const f32x4_t*>(pt_at(r, q4));
    if (p.b2) y += bb;
    if (p.out_relu)
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = fmaxf(y[e], 0.0f);
    const u32x2_t o2 = {pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3])};
    __builtin_nontemporal_store(o2, reinterpret_cast<u32x2_t*>(O + (int64_t)m * p.ldo + 4 * q4));
  }
}

bool b2b_mlp_supported(int K, int N1, int N2) {
  return N2 == 128 && N1 % kMlpHidden == 0 && N1 > 0 && K % 64 == 0 && K / 64 >= MlpS::STAGES - 1;
}

hipError_t launch_b2b_mlp(const B2BParams& p, hipStream_t st) {
  if (!b2b_mlp_supported(p.K, p.N1, p.N2) || (p.cn != 1 && p.cn != p.N1 / kMlpHidden)) return hipErrorInvalidValue;
  const unsigned rbs = (unsigned)((p.M + kMlpRows - 1) / kMlpRows);
  const dim3 grid(rbs * (unsigned)p.cn, (unsigned)p.batch), block(MlpS::NT);
  if (p.cn == 1) hipLaunchKernelGGL((b2b_mlp_whole_kernel<128>), grid, block, 0, st, p);
  else hipLaunchKernelGGL((b2b_mlp_kernel<128>), grid, block, 0, st, p);
  return hipGetLastError();
}

}  // namespace cf
