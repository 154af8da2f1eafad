// Row kernels for gfx950.
//
// row_kernel: one 64-lane wave owns one row: its values stay in registers
// from load to store, every reduction is a wave-wide butterfly (no LDS, no
// barrier), and the row is read from HBM exactly once.  wide_row_kernel:
// the same for rows wider than 1024, with a 256-thread workgroup per row.
// Two users:
//   * the finish pass of the split-N path: the GEMM has written fp32 x and a
//     partial (mean, M2) per (row, N tile); the wave merges the partials with
//     the k-way form of the pairwise update of Chan, Golub and LeVeque, then
//     runs stages 2..4;
//   * the unfused row operator (the materialising baseline): stages 1..4, or
//     a softmax, on a matrix that a plain GEMM wrote to global memory.
#include "cf_device.h"
#include "cf_internal.h"

namespace cf {

// Element offset of row m of the input (rows of a batch of matrices with
// stride sp, or one matrix when sp = 0).
__device__ __forceinline__ int64_t prow(const RowKernelParams& p, int m) {
  if (p.sp == 0) return (int64_t)m * p.ldp;
  const int b = m / p.rows_per_batch;
  return (int64_t)b * p.sp + (int64_t)(m - b * p.rows_per_batch) * p.ldp;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// Row statistics from the split GEMM pass's per-tile partials (mean_c, M2_c)
// of cn tiles of width tn (the last one N - (cn - 1) tn wide), in the k-way
// form of the pairwise update of Chan, Golub and LeVeque:
//   mean = sum_c n_c mean_c / N,   M2 = sum_c (M2_c + n_c (mean_c - mean)^2).
// Lane c (< cn <= 64) holds tile c's pair; both sums are butterflies, whose
// pairwise additions commute exactly, so every lane gets the same values.
__device__ __forceinline__ void merge_partials(const float2* part, int cn, int tn, int N, int lane, float& mean,
                                               float& m2) {
  const bool has = lane < cn;
  const float2 pc = has ? part[lane] : make_float2(0.0f, 0.0f);
  const float nc = has ? (float)min(tn, N - lane * tn) : 0.0f;
  mean = wave_sum(nc * pc.x) / (float)N;
  const float d = pc.x - mean;
  m2 = wave_sum(has ? fmaf(nc * d, d, pc.y) : 0.0f);
}

// VPL = groups of 4 consecutive columns per lane; a row of up to 256*VPL.
// Lane l holds columns 256*j + 4*l + (0..3), j < VPL: each j is one fully
// coalesced 1 KB (fp32) or 512 B (bf16) access by the wave.  SM: the node
// list has a SOFTMAX stage (compiled separately: its exp chain would raise
// the register use of every other list).
template <int VPL, bool SM>
__global__ __launch_bounds__(256) void row_kernel(RowKernelParams p) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= p.M) return;
  const int N = p.N;
  const RowEpi& e = p.epi;
  float v[VPL][4];
  bool val[VPL];

  // ---- load (and stage 1 for the row operator)
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const int n = 256 * j + 4 * lane;
    val[j] = n < N;
    if (val[j]) {
      if (p.p_f32) load4_once<float>(reinterpret_cast<const float*>(p.P) + prow(p, m) + n, v[j]);
      else load4_once<bf16_t>(reinterpret_cast<const bf16_t*>(p.P) + prow(p, m) + n, v[j]);
    } else {
      v[j][0] = v[j][1] = v[j][2] = v[j][3] = 0.0f;
    }
  }

  if (p.softmax) {
    // softmax(scale * P) over the row: max, exp(x - max), sum, divide.
    const float sc = p.softmax_scale;
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < VPL; ++j)
      if (val[j])
#pragma unroll
        for (int q = 0; q < 4; ++q) mx = fmaxf(mx, v[j][q] * sc);
    mx = wave_max(mx);
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < VPL; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float t = val[j] ? __expf(v[j][q] * sc - mx) : 0.0f;
        v[j][q] = t;
        s += t;
      }
    const float inv = 1.0f / wave_sum(s);
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      if (!val[j]) continue;
      float o[4] = {v[j][0] * inv, v[j][1] * inv, v[j][2] * inv, v[j][3] * inv};
      store4(e.Y, (int64_t)m * e.ldy + 256 * j + 4 * lane, e.y_f32, o);
    }
    return;
  }

  if (!p.finish) {
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      if (!val[j]) continue;
      const int n = 256 * j + 4 * lane;
      // Only the terms that are given are added (x + 0 would turn -0 into +0).
#pragma unroll
      for (int q = 0; q < 4; ++q) v[j][q] *= e.alpha;
      if (e.bias) {
        float b[4];
        load4<float>(e.bias + n, b);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[j][q] += b[q];
      }
      if (e.R) {
        float r[4];
        if (e.r_f32) load4_once<float>(reinterpret_cast<const float*>(e.R) + (int64_t)m * e.ldr + n, r);
        else load4_once<bf16_t>(reinterpret_cast<const bf16_t*>(e.R) + (int64_t)m * e.ldr + n, r);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[j][q] += r[q];
      }
    }
  }

  // ---- stage 2: statistics and normalisation
  if (e.norm != NORM_NONE) {
    float mean, m2;
    if (p.finish) {
      merge_partials(reinterpret_cast<const float2*>(p.part) + (int64_t)m * p.cn, p.cn, p.tn, N, lane, mean, m2);
    } else {
      float s = 0.0f;
#pragma unroll
      for (int j = 0; j < VPL; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) s += v[j][q];
      mean = wave_sum(s) / (float)N;
      float t = 0.0f;
#pragma unroll
      for (int j = 0; j < VPL; ++j)
        if (val[j])
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float d = v[j][q] - mean;
            t += d * d;
          }
      m2 = wave_sum(t);
    }
    const float invN = 1.0f / (float)N;
    if (e.norm == NORM_LAYER) {
      const float rstd = rsqrtf(m2 * invN + e.eps);
#pragma unroll
      for (int j = 0; j < VPL; ++j) {
        if (!val[j]) continue;
        const int n = 256 * j + 4 * lane;
        float g[4] = {1.0f, 1.0f, 1.0f, 1.0f}, b[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        if (e.gamma) load4<float>(e.gamma + n, g);
        if (e.beta) load4<float>(e.beta + n, b);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[j][q] = (v[j][q] - mean) * rstd * g[q] + b[q];
      }
    } else {
      // RMSNorm: mean of squares = M2/N + mean^2.
      const float rstd = rsqrtf(m2 * invN + mean * mean + e.eps);
#pragma unroll
      for (int j = 0; j < VPL; ++j) {
        if (!val[j]) continue;
        const int n = 256 * j + 4 * lane;
        float g[4] = {1.0f, 1.0f, 1.0f, 1.0f};
        if (e.gamma) load4<float>(e.gamma + n, g);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[j][q] = v[j][q] * rstd * g[q];
      }
    }
  }

  // ---- stage 3: activation and store
  // The kind is switched per element here: one loop per kind would keep
  // every kind's temporaries of all 4 * VPL values live at once (74 against
  // 48 VGPRs for VPL = 4, and two fewer resident waves per SIMD).
  if (e.act != ACT_NONE) {
#pragma unroll
    for (int j = 0; j < VPL; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float x = v[j][q];
        switch (e.act) {
          case ACT_GELU: v[j][q] = gelu_erf(x); break;
          case ACT_GELU_TANH: v[j][q] = gelu_tanh(x); break;
          case ACT_RELU: v[j][q] = x > 0.0f ? x : 0.0f; break;
          case ACT_SOFTCAP: v[j][q] = e.softcap * tanh_exp(x / e.softcap); break;
          default: break;
        }
      }
  }
  if (SM) {   // row softmax of the (activated) values
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < VPL; ++j)
      if (val[j])
#pragma unroll
        for (int q = 0; q < 4; ++q) mx = fmaxf(mx, v[j][q]);
    mx = wave_max(mx);
    const float nl = -mx * 1.4426950408889634f;
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < VPL; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float t = val[j] ? __builtin_amdgcn_exp2f(fmaf(v[j][q], 1.4426950408889634f, nl)) : 0.0f;
        v[j][q] = t;
        s += t;
      }
    const float inv = 1.0f / wave_sum(s);
#pragma unroll
    for (int j = 0; j < VPL; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) v[j][q] *= inv;
  }
  if (e.Y) {
#pragma unroll
    for (int j = 0; j < VPL; ++j)
      if (val[j]) store4(e.Y, (int64_t)m * e.ldy + 256 * j + 4 * lane, e.y_f32, v[j]);
  }

  // ---- stage 4: row amax -> scale -> E4M3 codes
  if (e.quant) {
    float a = 0.0f;
#pragma unroll
    for (int j = 0; j < VPL; ++j)
      if (val[j])
#pragma unroll
        for (int q = 0; q < 4; ++q) a = fmaxf(a, fabsf(v[j][q]));
    a = wave_max(a);
    const float sc = a / e.qmax;
    if (lane == 0 && e.s_out) e.s_out[m] = sc;
    if (e.q_out) {
      // codes of fl32(z / s); a zero row (s = 0, uniform over the wave) gives codes 0
      const bool nz = sc > 0.0f;
      const float sd = nz ? sc : 1.0f, inv = nz ? 1.0f / sc : 1.0f;
#pragma unroll
      for (int j = 0; j < VPL; ++j) {
        if (!val[j]) continue;
        const uint32_t w = e4m3x4(div_rn(v[j][0], sd, inv), div_rn(v[j][1], sd, inv), div_rn(v[j][2], sd, inv),
                                  div_rn(v[j][3], sd, inv));
        __builtin_nontemporal_store(nz ? w : 0u, reinterpret_cast<uint32_t*>(e.q_out + (int64_t)m * e.ldq + 256 * j + 4 * lane));
      }
    }
  }
}

// Rows wider than 1024 (split-N finish pass and the unfused row operator,
// softmax lists excepted): one 256-thread workgroup per row, so a lane holds
// 4 * VPW values (not 4 * N / 256) and a CU keeps enough waves resident to
// overlap the row reads with the element work.  Lane l of wave w holds
// columns 1024 j + 256 w + 4 l + (0..3), j < VPW (each j one coalesced read
// per wave).  Row sums and the amax are combined across the four waves
// through LDS in a fixed order, so every wave gets the same values; the
// finish pass merges the partial statistics in every wave.  FULL: N = 1024
// VPW, no column guards.
template <int VPW, bool FULL>
__global__ __launch_bounds__(256) void wide_row_kernel(RowKernelParams p) {
  __shared__ float red[3][4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m = blockIdx.x;
  const int N = p.N;
  const RowEpi& e = p.epi;
  auto col = [&](int j) { return 1024 * j + 256 * wave + 4 * lane; };
  // sum over the workgroup of one value per lane (reduction slot r)
  auto block_sum = [&](float t, int r) {
    t = wave_sum(t);
    if (lane == 0) red[r][wave] = t;
    __syncthreads();
    return (red[r][0] + red[r][1]) + (red[r][2] + red[r][3]);
  };
  float v[VPW][4];
  bool val[VPW];
#pragma unroll
  for (int j = 0; j < VPW; ++j) {
    val[j] = FULL || col(j) < N;
    if (val[j]) {
      if (p.p_f32) load4_once<float>(reinterpret_cast<const float*>(p.P) + prow(p, m) + col(j), v[j]);
      else load4_once<bf16_t>(reinterpret_cast<const bf16_t*>(p.P) + prow(p, m) + col(j), v[j]);
    } else {
      v[j][0] = v[j][1] = v[j][2] = v[j][3] = 0.0f;
    }
  }
  if (!p.finish) {
    // stage 1; only the terms that are given are added (x + 0 would turn -0 into +0)
#pragma unroll
    for (int j = 0; j < VPW; ++j) {
      if (!val[j]) continue;
#pragma unroll
      for (int q = 0; q < 4; ++q) v[j][q] *= e.alpha;
      if (e.bias) {
        float b[4];
        load4<float>(e.bias + col(j), b);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[j][q] += b[q];
      }
      if (e.R) {
        float r[4];
        if (e.r_f32) load4_once<float>(reinterpret_cast<const float*>(e.R) + (int64_t)m * e.ldr + col(j), r);
        else load4_once<bf16_t>(reinterpret_cast<const bf16_t*>(e.R) + (int64_t)m * e.ldr + col(j), r);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[j][q] += r[q];
      }
    }
  }
  if (e.norm == NORM_LAYER || e.norm == NORM_RMS) {
    float mean, m2;
    if (p.finish) {
      merge_partials(reinterpret_cast<const float2*>(p.part) + (int64_t)m * p.cn, p.cn, p.tn, N, lane, mean, m2);
    } else {
      // two passes: mean, then the sum of squared deviations (padding columns skipped)
      float t = 0.0f;
#pragma unroll
      for (int j = 0; j < VPW; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) t += v[j][q];
      mean = block_sum(t, 0) / (float)N;
      t = 0.0f;
#pragma unroll
      for (int j = 0; j < VPW; ++j)
        if (val[j])
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float d = v[j][q] - mean;
            t = fmaf(d, d, t);
          }
      m2 = block_sum(t, 1);
    }
    const float invN = 1.0f / (float)N;
    // LayerNorm: (x - mean) rstd; RMSNorm: x rstd with mean of squares M2/N + mean^2
    const bool ln = e.norm == NORM_LAYER;
    const float rstd = ln ? rsqrtf(m2 * invN + e.eps) : rsqrtf(m2 * invN + mean * mean + e.eps);
    const float sh = ln ? mean : 0.0f;
#pragma unroll
    for (int j = 0; j < VPW; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) v[j][q] = (v[j][q] - sh) * rstd;
    if (e.gamma || (ln && e.beta)) {
#pragma unroll
      for (int j = 0; j < VPW; ++j) {
        if (!val[j]) continue;
        float g[4] = {1.0f, 1.0f, 1.0f, 1.0f}, b[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        if (e.gamma) load4<float>(e.gamma + col(j), g);
        if (ln && e.beta) load4<float>(e.beta + col(j), b);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[j][q] = fmaf(v[j][q], g[q], b[q]);
      }
    }
  }
  auto act_all = [&](auto f) {
#pragma unroll
    for (int j = 0; j < VPW; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) v[j][q] = f(v[j][q]);
  };
  switch (e.act) {
    case ACT_GELU: act_all([](float t) { return gelu_erf(t); }); break;
    case ACT_GELU_TANH: act_all([](float t) { return gelu_tanh(t); }); break;
    case ACT_RELU: act_all([](float t) { return t > 0.0f ? t : 0.0f; }); break;
    case ACT_SOFTCAP: {
      const float cap = e.softcap;
      act_all([cap](float t) { return cap * tanh_exp(t / cap); });
      break;
    }
    default: break;
  }
  if (e.Y) {
#pragma unroll
    for (int j = 0; j < VPW; ++j)
      if (val[j]) store4(e.Y, (int64_t)m * e.ldy + col(j), e.y_f32, v[j]);
  }
  if (e.quant) {
    float a = 0.0f;
#pragma unroll
    for (int j = 0; j < VPW; ++j)
      if (val[j])
#pragma unroll
        for (int q = 0; q < 4; ++q) a = fmaxf(a, fabsf(v[j][q]));
    a = wave_max(a);
    if (lane == 0) red[2][wave] = a;
    __syncthreads();
    a = fmaxf(fmaxf(red[2][0], red[2][1]), fmaxf(red[2][2], red[2][3]));
    const float sc = a / e.qmax;
    if (threadIdx.x == 0 && e.s_out) e.s_out[m] = sc;
    if (e.q_out) {
      // codes of fl32(z / s); a zero row (s = 0) gives codes 0
      const bool nz = sc > 0.0f;
      const float sd = nz ? sc : 1.0f, inv = nz ? 1.0f / sc : 1.0f;
#pragma unroll
      for (int j = 0; j < VPW; ++j) {
        if (!val[j]) continue;
        const uint32_t w = e4m3x4(div_rn(v[j][0], sd, inv), div_rn(v[j][1], sd, inv), div_rn(v[j][2], sd, inv),
                                  div_rn(v[j][3], sd, inv));
        __builtin_nontemporal_store(nz ? w : 0u, reinterpret_cast<uint32_t*>(e.q_out + (int64_t)m * e.ldq + col(j)));
      }
    }
  }
}

hipError_t launch_row_kernel(const RowKernelParams& p, hipStream_t st) {
  if (p.M <= 0) return hipSuccess;
  if (!p.epi.softmax && !p.softmax && p.N > 1024) {
    const dim3 grid((unsigned)p.M), block(256);
#define CF_FIN_LAUNCH(V)                                                                    \
  do {                                                                                      \
    if (p.N == 1024 * (V)) hipLaunchKernelGGL((wide_row_kernel<V, true>), grid, block, 0, st, p); \
    else hipLaunchKernelGGL((wide_row_kernel<V, false>), grid, block, 0, st, p);            \
  } while (0)
    const int vpw = (p.N + 1023) / 1024;
    if (vpw <= 2) CF_FIN_LAUNCH(2);
    else if (vpw <= 4) CF_FIN_LAUNCH(4);
    else if (vpw <= 8) CF_FIN_LAUNCH(8);
    else return hipErrorInvalidValue;
#undef CF_FIN_LAUNCH
    return hipGetLastError();
  }
  const dim3 grid((unsigned)((p.M + 3) / 4)), block(256);
  const int vpl = (p.N + 255) / 256;
  const bool sm = p.epi.softmax != 0;
#define CF_ROW_LAUNCH(V)                                                                    \
  do {                                                                                      \
    if (sm) hipLaunchKernelGGL((row_kernel<V, true>), grid, block, 0, st, p);               \
    else hipLaunchKernelGGL((row_kernel<V, false>), grid, block, 0, st, p);                 \
  } while (0)
  if (vpl <= 1) CF_ROW_LAUNCH(1);
  else if (vpl <= 2) CF_ROW_LAUNCH(2);
  else if (vpl <= 4) CF_ROW_LAUNCH(4);
  else if (vpl <= 8) CF_ROW_LAUNCH(8);
  else if (vpl <= 16) CF_ROW_LAUNCH(16);
  else if (vpl <= 32) CF_ROW_LAUNCH(32);
  else return hipErrorInvalidValue;
#undef CF_ROW_LAUNCH
  return hipGetLastError();
}

}  // namespace cf
