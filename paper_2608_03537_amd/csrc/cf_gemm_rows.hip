// GEMM + row-subgraph kernels for gfx950.
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
#include "cf_device.h"
#include "cf_internal.h"

namespace cf {

constexpr int kSpinLimit = 1 << 22;   // bounded wait for peers (~1 s)

template <typename TIn, int BM_, int BN_, int WM_, int WN_, int TKB_>
struct TileShape {
  using T = TIn;
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
  static constexpr int LDS = 2 * STAGE;
  static constexpr int A_CHUNKS = TN * CPR, B_CHUNKS = TM * CPR;
  static constexpr int A_PT = (A_CHUNKS + NT - 1) / NT;
  static constexpr int B_PT = (B_CHUNKS + NT - 1) / NT;
  static_assert(LDS <= 160 * 1024, "LDS budget");
  static_assert(TK % KSTEP == 0, "stage must hold whole MFMA steps");
};

// ---------------------------------------------------------------------------
// Main loop: global -> registers -> LDS (double buffered) -> MFMA.
// ---------------------------------------------------------------------------
template <class S>
__device__ __forceinline__ void mainloop(f32x16_t (&acc)[S::BM][S::BN],
                                         const typename S::T* __restrict__ X,
                                         const typename S::T* __restrict__ W,
                                         const GemmRowsParams& p, int m0, int n0,
                                         char* smem, int tid, int lane, int wm, int wn) {
  using T = typename S::T;
#pragma unroll
  for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
    for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[bm][bn][i] = 0.0f;

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

// Level 3, ROWS_CLUSTER: publish one float2 per row, wait for the cn peers of
// this row block, gather all cn partials (in peer order) into out[bm][c].
// Arrival: each peer adds kArriveUnit / cn to its group's counter; the group
// is complete when the counter reaches the next multiple of kArriveUnit.
template <class S, int CNMAX>
__device__ __forceinline__ void cluster_exchange(const GemmRowsParams& p, int stage, int slot, int c,
                                                 int m0, const float2 (&val)[S::BM],
                                                 float2 (&out)[S::BM][CNMAX], int tid,
                                                 int lane, int wm, int wn) {
  const int M = p.M, cn = p.cn;
  unsigned long long* part = reinterpret_cast<unsigned long long*>(p.ws_part) + (int64_t)stage * M * cn;
  const int lr = lane & 31;
  if (wn == 0) {
    if (lane < 32) {
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) {
        const int m = m0 + wm * S::WTM + bm * 32 + lr;
        if (m < M)
          __hip_atomic_store(part + (int64_t)m * cn + c, __builtin_bit_cast(unsigned long long, val[bm]),
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    __threadfence();
  }
  __syncthreads();
  if (tid == 0) {
    unsigned long long* ctr = p.ws_arrive + slot;
    const unsigned long long old =
        __hip_atomic_fetch_add(ctr, kArriveUnit / (unsigned long long)cn, __ATOMIC_RELEASE,
                               __HIP_MEMORY_SCOPE_AGENT);
    const unsigned long long target = (old / kArriveUnit + 1ull) * kArriveUnit;
    int spins = 0;
    while (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      if (++spins > kSpinLimit) {
        __hip_atomic_store(p.ws_err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      __builtin_amdgcn_s_sleep(4);
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
  __syncthreads();
#pragma unroll
  for (int bm = 0; bm < S::BM; ++bm) {
    const int m = m0 + wm * S::WTM + bm * 32 + lr;
    const int mm = m < M ? m : M - 1;
#pragma unroll
    for (int cc = 0; cc < CNMAX; ++cc) {
      if (cc < cn) {
        const unsigned long long u = __hip_atomic_load(part + (int64_t)mm * cn + cc, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT);
        out[bm][cc] = __builtin_bit_cast(float2, u);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Epilogue on the register tile.
// ---------------------------------------------------------------------------
template <class S>
__device__ __forceinline__ void epilogue(f32x16_t (&x)[S::BM][S::BN], const GemmRowsParams& p,
                                         int m0, int n0, int slot, int c, int bz, char* smem,
                                         int tid, int lane, int wm, int wn) {
  using T = typename S::T;
  constexpr int CNMAX = 16;
  const RowEpi& e = p.epi;
  const int M = p.M, N = p.N;
  const int lr = lane & 31, lg = lane >> 5;
  float* red = reinterpret_cast<float*>(smem);

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
#pragma unroll
  for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
    for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
      for (int i = 0; i < 16; ++i) x[bm][bn][i] *= alpha;
  if (e.bias) {
#pragma unroll
    for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = ncol(bn, g);
        if (n < N) {
          const f32x4_t b = *reinterpret_cast<const f32x4_t*>(e.bias + n);
#pragma unroll
          for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
            for (int q = 0; q < 4; ++q) x[bm][bn][4 * g + q] += b[q];
        }
      }
  }
  if (e.R) {
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

  bool exchanged = false;
  const int cnt_c = min(S::TN, N - n0);   // valid columns in this tile

  // ---- stage 2: row statistics and the normalising PostOp
  if (e.norm == NORM_LAYER || p.mode == ROWS_SPLIT) {
    float s[S::BM];
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      float t = 0.0f;
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int i = 0; i < 16; ++i) t += x[bm][bn][i];
      s[bm] = t;
    }
    wg_row_reduce<S, false>(s, red, lane, wm, wn);
    const float inv_c = 1.0f / (float)cnt_c;
    float mean[S::BM], m2[S::BM];
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      mean[bm] = s[bm] * inv_c;
      float t = 0.0f;
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          if (ncol(bn, g) < N) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const float d = x[bm][bn][4 * g + q] - mean[bm];
              t += d * d;
            }
          }
        }
      m2[bm] = t;
    }
    wg_row_reduce<S, false>(m2, red, lane, wm, wn);

    if (p.mode == ROWS_SPLIT) {
      // Publish fp32 x and the tile's (mean, M2); the finish pass does the rest.
      float* xb = p.ws_x;
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) {
        if (!mval[bm]) continue;
#pragma unroll
        for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int n = ncol(bn, g);
            if (n < N) {
              float v[4] = {x[bm][bn][4 * g], x[bm][bn][4 * g + 1], x[bm][bn][4 * g + 2], x[bm][bn][4 * g + 3]};
              store4(xb, (int64_t)mrow[bm] * N + n, 1, v);
            }
          }
        if (wn == 0 && lane < 32)
          reinterpret_cast<float2*>(p.ws_part)[(int64_t)mrow[bm] * p.cn + c] = make_float2(mean[bm], m2[bm]);
      }
      return;
    }

    if (p.mode == ROWS_CLUSTER && p.cn > 1) {
      float2 val[S::BM];
      float2 all[S::BM][CNMAX];
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) val[bm] = make_float2(mean[bm], m2[bm]);
      cluster_exchange<S, CNMAX>(p, 0, slot, c, m0, val, all, tid, lane, wm, wn);
      exchanged = true;
      // Equal-count merge (every peer holds S::TN columns):
      //   mean = avg(mean_c);  M2 = sum(M2_c) + TN * sum((mean_c - mean)^2)
      const float inv_cn = 1.0f / (float)p.cn;
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) {
        float t = 0.0f;
#pragma unroll
        for (int cc = 0; cc < CNMAX; ++cc)
          if (cc < p.cn) t += all[bm][cc].x;
        const float mu = t * inv_cn;
        float a = 0.0f, b = 0.0f;
#pragma unroll
        for (int cc = 0; cc < CNMAX; ++cc)
          if (cc < p.cn) {
            a += all[bm][cc].y;
            const float d = all[bm][cc].x - mu;
            b += d * d;
          }
        mean[bm] = mu;
        m2[bm] = a + (float)S::TN * b;
      }
    }

    if (e.norm == NORM_LAYER) {
      const float invN = 1.0f / (float)N;
      float rstd[S::BM];
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) rstd[bm] = rsqrtf(m2[bm] * invN + e.eps);
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = ncol(bn, g);
          f32x4_t ga = {1.0f, 1.0f, 1.0f, 1.0f}, be = {0.0f, 0.0f, 0.0f, 0.0f};
          if (n < N) {
            if (e.gamma) ga = *reinterpret_cast<const f32x4_t*>(e.gamma + n);
            if (e.beta) be = *reinterpret_cast<const f32x4_t*>(e.beta + n);
          }
#pragma unroll
          for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
            for (int q = 0; q < 4; ++q)
              x[bm][bn][4 * g + q] = (x[bm][bn][4 * g + q] - mean[bm]) * rstd[bm] * ga[q] + be[q];
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
    wg_row_reduce<S, false>(s, red, lane, wm, wn);
    if (p.mode == ROWS_CLUSTER && p.cn > 1) {
      float2 val[S::BM];
      float2 all[S::BM][CNMAX];
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) val[bm] = make_float2(s[bm], 0.0f);
      cluster_exchange<S, CNMAX>(p, 0, slot, c, m0, val, all, tid, lane, wm, wn);
      exchanged = true;
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) {
        float t = 0.0f;
#pragma unroll
        for (int cc = 0; cc < CNMAX; ++cc)
          if (cc < p.cn) t += all[bm][cc].x;
        s[bm] = t;
      }
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
        if (n < N && e.gamma) ga = *reinterpret_cast<const f32x4_t*>(e.gamma + n);
#pragma unroll
        for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
          for (int q = 0; q < 4; ++q) x[bm][bn][4 * g + q] = x[bm][bn][4 * g + q] * s[bm] * ga[q];
      }
  }

  // ---- stage 3: activation and store
  if (e.act != ACT_NONE) {
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm)
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int i = 0; i < 16; ++i) x[bm][bn][i] = apply_act(e.act, x[bm][bn][i]);
  }
  if (e.Y) {
    char* Yb = reinterpret_cast<char*>(e.Y) + (int64_t)bz * e.sy * (e.y_f32 ? 4 : 2);
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      if (!mval[bm]) continue;
#pragma unroll
      for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = ncol(bn, g);
          if (n < N) {
            float v[4] = {x[bm][bn][4 * g], x[bm][bn][4 * g + 1], x[bm][bn][4 * g + 2], x[bm][bn][4 * g + 3]};
            store4(Yb, (int64_t)mrow[bm] * e.ldy + n, e.y_f32, v);
          }
        }
    }
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
        for (int i = 0; i < 16; ++i) t = fmaxf(t, fabsf(x[bm][bn][i]));
      a[bm] = t;
    }
    wg_row_reduce<S, true>(a, red, lane, wm, wn);
    if (p.mode == ROWS_CLUSTER && p.cn > 1) {
      float2 val[S::BM];
      float2 all[S::BM][CNMAX];
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) val[bm] = make_float2(a[bm], 0.0f);
      cluster_exchange<S, CNMAX>(p, exchanged ? 1 : 0, slot, c, m0, val, all, tid, lane, wm, wn);
      exchanged = true;
#pragma unroll
      for (int bm = 0; bm < S::BM; ++bm) {
        float t = 0.0f;
#pragma unroll
        for (int cc = 0; cc < CNMAX; ++cc)
          if (cc < p.cn) t = fmaxf(t, all[bm][cc].x);
        a[bm] = t;
      }
    }
#pragma unroll
    for (int bm = 0; bm < S::BM; ++bm) {
      if (!mval[bm]) continue;
      const float sc = a[bm] / e.qmax;
      if (c == 0 && wn == 0 && lane < 32 && e.s_out) e.s_out[mrow[bm]] = sc;
      if (e.q_out) {
#pragma unroll
        for (int bn = 0; bn < S::BN; ++bn)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int n = ncol(bn, g);
            if (n < N) {
              uint32_t w = 0;
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const uint32_t code = sc > 0.0f ? f32_to_e4m3(x[bm][bn][4 * g + q] / sc) : 0u;
                w |= code << (8 * q);
              }
              *reinterpret_cast<uint32_t*>(e.q_out + (int64_t)mrow[bm] * e.ldq + n) = w;
            }
          }
      }
    }
  }
}

template <class S>
__global__ __launch_bounds__(S::NT, 1) void gemm_rows_kernel(GemmRowsParams p) {
  using T = typename S::T;
  __shared__ __attribute__((aligned(16))) char smem[S::LDS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / S::WN, wn = wave % S::WN;
  const int bz = blockIdx.y;
  const T* X = reinterpret_cast<const T*>(p.X) + (int64_t)bz * p.sx;
  const T* W = reinterpret_cast<const T*>(p.W) + (int64_t)bz * p.sw;
  // blockIdx.x -> (XCD, slot, peer).  Consecutive block ids go round-robin
  // over the 8 XCDs, so the cn peers of a row block share one XCD and its L2.
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int c = local % p.cn, q = local / p.cn;
  for (int it = 0;; ++it) {
    const int rb = (it * p.slots + q) * 8 + xcd;
    if (rb >= p.num_rb) break;
    const int m0 = rb * S::TM, n0 = c * S::TN;
    f32x16_t acc[S::BM][S::BN];
    mainloop<S>(acc, X, W, p, m0, n0, smem, tid, lane, wm, wn);
    epilogue<S>(acc, p, m0, n0, q * 8 + xcd, c, bz, smem, tid, lane, wm, wn);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Configurations.  Whole-row tiles (TM = 32, TN up to 768 for bf16) keep the
// full row in one workgroup; 128-row tiles serve the cluster and split paths
// and the plain GEMM.
// ---------------------------------------------------------------------------
#define CF_TILE_LIST(X)                                       \
  X(0, bf16_t, 1, 1, 1, 4, 64)  /* TM 32,  TN 128 */          \
  X(1, bf16_t, 1, 2, 1, 4, 64)  /* TM 32,  TN 256 */          \
  X(2, bf16_t, 1, 3, 1, 4, 64)  /* TM 32,  TN 384 */          \
  X(3, bf16_t, 1, 4, 1, 4, 64)  /* TM 32,  TN 512 */          \
  X(4, bf16_t, 1, 6, 1, 4, 64)  /* TM 32,  TN 768 */          \
  X(5, bf16_t, 2, 2, 2, 2, 128) /* TM 128, TN 128 */          \
  X(6, bf16_t, 2, 3, 2, 2, 128) /* TM 128, TN 192 */          \
  X(7, bf16_t, 2, 4, 2, 2, 128) /* TM 128, TN 256 */          \
  X(8, float, 1, 1, 1, 4, 64)   /* TM 32,  TN 128 */          \
  X(9, float, 1, 2, 1, 4, 64)   /* TM 32,  TN 256 */          \
  X(10, float, 1, 3, 1, 4, 64)  /* TM 32,  TN 384 */          \
  X(11, float, 1, 4, 1, 4, 64)  /* TM 32,  TN 512 */          \
  X(12, float, 1, 6, 1, 4, 64)  /* TM 32,  TN 768 */          \
  X(13, float, 2, 2, 2, 2, 128) /* TM 128, TN 128 */          \
  X(14, float, 2, 4, 2, 2, 128) /* TM 128, TN 256 */

#define CF_TILE_SHAPE(id, T, BM, BN, WM, WN, TKB) TileShape<T, BM, BN, WM, WN, TKB>

static const TileCfg kTiles[] = {
#define X(id, T, BM, BN, WM, WN, TKB) \
  {id, CF_TILE_SHAPE(id, T, BM, BN, WM, WN, TKB)::TM, CF_TILE_SHAPE(id, T, BM, BN, WM, WN, TKB)::TN, \
   sizeof(T) == 4, CF_TILE_SHAPE(id, T, BM, BN, WM, WN, TKB)::NT},
    CF_TILE_LIST(X)
#undef X
};

int tile_cfg_count() { return (int)(sizeof(kTiles) / sizeof(kTiles[0])); }
const TileCfg& tile_cfg(int i) { return kTiles[i]; }

static const void* kernel_ptr(int cfg) {
  switch (cfg) {
#define X(id, T, BM, BN, WM, WN, TKB) \
    case id: return reinterpret_cast<const void*>(&gemm_rows_kernel<CF_TILE_SHAPE(id, T, BM, BN, WM, WN, TKB)>);
    CF_TILE_LIST(X)
#undef X
    default: return nullptr;
  }
}

int resident_wgs(int cfg) {
  static int cache[64] = {0};
  if (cfg < 0 || cfg >= tile_cfg_count()) return 0;
  if (cache[cfg]) return cache[cfg];
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel_ptr(cfg), kTiles[cfg].threads, 0) !=
      hipSuccess)
    return 0;
  cache[cfg] = cus * per_cu;
  return cache[cfg];
}

hipError_t launch_gemm_rows(const GemmRowsParams& p, int in_f32, int cfg, hipStream_t st) {
  (void)in_f32;
  const void* fn = kernel_ptr(cfg);
  if (!fn) return hipErrorInvalidValue;
  dim3 grid((unsigned)(8 * p.slots * p.cn), (unsigned)p.batch), block((unsigned)kTiles[cfg].threads);
  switch (cfg) {
#define X(id, T, BM, BN, WM, WN, TKB) \
    case id: hipLaunchKernelGGL((gemm_rows_kernel<CF_TILE_SHAPE(id, T, BM, BN, WM, WN, TKB)>), grid, block, 0, st, p); break;
    CF_TILE_LIST(X)
#undef X
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace cf
