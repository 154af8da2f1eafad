// Wave-per-row kernels for gfx950.
//
// One 64-lane wave owns one row: its values stay in registers from load to
// store, every reduction is a wave-wide butterfly (no LDS, no barrier), and
// the row is read from HBM exactly once.  Two users:
//   * the finish pass of the split-N path: the GEMM has written fp32 x and a
//     partial (mean, M2) per (row, N tile); the wave merges the partials with
//     the pairwise update of Chan, Golub and LeVeque, then runs stages 2..4;
//   * the unfused row operator (the materialising baseline): stages 1..4, or
//     a softmax, on a matrix that a plain GEMM wrote to global memory.
#include "cf_device.h"
#include "cf_internal.h"

namespace cf {

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
      if (p.p_f32) load4<float>(reinterpret_cast<const float*>(p.P) + (int64_t)m * p.ldp + n, v[j]);
      else load4<bf16_t>(reinterpret_cast<const bf16_t*>(p.P) + (int64_t)m * p.ldp + n, v[j]);
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
        if (e.r_f32) load4<float>(reinterpret_cast<const float*>(e.R) + (int64_t)m * e.ldr + n, r);
        else load4<bf16_t>(reinterpret_cast<const bf16_t*>(e.R) + (int64_t)m * e.ldr + n, r);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[j][q] += r[q];
      }
    }
  }

  // ---- stage 2: statistics and normalisation
  if (e.norm != NORM_NONE) {
    float mean, m2;
    if (p.finish) {
      // Pairwise merge of (count, mean, M2) over the row's tiles, in order.
      const float2* part = reinterpret_cast<const float2*>(p.part) + (int64_t)m * p.cn;
      float n_acc = 0.0f;
      mean = 0.0f;
      m2 = 0.0f;
      for (int c = 0; c < p.cn; ++c) {
        const float nb = (float)min(p.tn, N - c * p.tn);
        const float2 pb = part[c];
        const float nn = n_acc + nb;
        const float delta = pb.x - mean;
        mean += delta * (nb / nn);
        m2 += pb.y + delta * delta * (n_acc * nb / nn);
        n_acc = nn;
      }
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
  if (e.act != ACT_NONE) {
#pragma unroll
    for (int j = 0; j < VPL; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) v[j][q] = apply_act(e.act, v[j][q], e.softcap);
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
#pragma unroll
      for (int j = 0; j < VPL; ++j) {
        if (!val[j]) continue;
        uint32_t w = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) w |= (sc > 0.0f ? f32_to_e4m3(v[j][q] / sc) : 0u) << (8 * q);
        *reinterpret_cast<uint32_t*>(e.q_out + (int64_t)m * e.ldq + 256 * j + 4 * lane) = w;
      }
    }
  }
}

hipError_t launch_row_kernel(const RowKernelParams& p, hipStream_t st) {
  if (p.M <= 0) return hipSuccess;
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
