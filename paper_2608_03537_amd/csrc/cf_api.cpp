// C ABI of libcomfuse: argument validation, path planning, workspace sizing
// and kernel dispatch.  Every check runs before the first launch, so an
// invalid call enqueues nothing; no exception leaves this file.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>

#include "comfuse.h"
#include "cf_internal.h"

using namespace cf;

// Split-MLP arrival counters: a fixed region at the start of the workspace,
// one word per (batch entry, row block); the partials start after it.
static constexpr size_t kMlpCounterBytes = size_t(1) << 20;
static constexpr int64_t kMlpMaxRowBlocks = int64_t(kMlpCounterBytes / 4);

static_assert(kWsHeaderBytes == CF_WS_HEADER_BYTES, "row-cluster workspace header size in the header file");
static_assert(kMlpCounterBytes == CF_B2B_WS_HEADER_BYTES, "split-MLP counter region size in the header file");

namespace {

thread_local std::string g_last_error;

cf_status fail(cf_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
cf_status fail(cf_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

size_t dsize(cf_dtype t) { return t == CF_F32 ? 4 : t == CF_BF16 ? 2 : 1; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

constexpr int64_t kMaxRowPitch = int64_t(1) << 23;   // bytes per row; 256 rows stay below 2^31

cf_status check_matrix(const char* name, const void* p, int64_t rows, int64_t cols, int64_t ld,
                       cf_dtype t, bool required) {
  if (!p) {
    // An empty matrix (rows == 0) may come with a NULL pointer.
    if (required && rows > 0) return fail(CF_ERR_NULL, "%s is NULL", name);
    return CF_OK;
  }
  if (rows > 0 && ld < cols) return fail(CF_ERR_LD, "%s: leading dimension %lld < %lld", name, (long long)ld,
                                         (long long)cols);
  if (!aligned16(p)) return fail(CF_ERR_ALIGN, "%s is not 16-byte aligned", name);
  if ((ld * (int64_t)dsize(t)) % 16 != 0)
    return fail(CF_ERR_ALIGN, "%s: leading dimension %lld is not a multiple of 16 bytes", name, (long long)ld);
  // Kernels address a tile's rows with 32-bit byte offsets.
  if (ld * (int64_t)dsize(t) >= kMaxRowPitch)
    return fail(CF_ERR_LD, "%s: leading dimension %lld is %lld bytes or more", name, (long long)ld,
                (long long)kMaxRowPitch);
  return CF_OK;
}

cf_status check_vec(const char* name, const float* p) {
  if (p && !aligned16(p)) return fail(CF_ERR_ALIGN, "%s is not 16-byte aligned", name);
  return CF_OK;
}

cf_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return CF_OK;
  return fail(CF_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// ---------------------------------------------------------------------------
// Planning of the GEMM + row-subgraph launch.
// ---------------------------------------------------------------------------
enum Path { PATH_AUTO = 0, PATH_WHOLE_ROW = 1, PATH_CLUSTER = 2, PATH_SPLIT = 3 };

constexpr int kWholeRowMaxN = 768;
constexpr int kClusterMaxPeers = 16;
constexpr int kAutoClusterPeers = 8;

struct Plan {
  int kidx = -1, mode = ROWS_LOCAL, cn = 1, num_rb = 0, slots = 0, tm = 0, tn = 0;
  size_t ws = 0;
  size_t off_part = 0, off_x = 0;
};

constexpr int kAssumedCUs = 256;   // MI355X; used only to rank tile widths

// Every non-empty workspace starts with the fixed header (error word, round
// counters and exchange records; only the cluster path writes it), which is
// all the cluster path needs.  The split path keeps part[M][cn] float2 and
// x[M][N] after it.
// The allocation-free entry point never runs the cluster path and keeps no
// header (header = false): its split buffers start at the scratch base.
void size_workspace(Plan& pl, int64_t M, int64_t N, bool header) {
  if (pl.mode == ROWS_CLUSTER) {
    pl.off_part = kWsCounterBytes;
    pl.ws = kWsHeaderBytes;
  } else if (pl.mode == ROWS_SPLIT) {
    pl.off_part = header ? kWsHeaderBytes : 0;
    pl.off_x = pl.off_part + round_up((size_t)M * pl.cn * 8, 256);
    pl.ws = pl.off_x + round_up((size_t)M * N * 4, 256);
  } else {
    pl.ws = 0;
  }
}

// Picks the 128-row tile width: the one whose workgroups, laid out in waves
// of one workgroup per CU, give the least work per CU (rounds x width).
// `divides` restricts to widths that split N exactly into <= max_cn peers.
int pick_tile(int64_t M, int64_t N, int64_t K, int in_f32, int loop, int epi, bool divides, int max_cn) {
  int best = -1;
  double best_cost = 1e300;
  for (int tn : {256, 192, 128}) {
    const int idx = find_gemm_kernel(in_f32, 128, tn, loop, epi);
    if (idx < 0) continue;
    // the direct-to-LDS ring is filled with stages-1 stages before the first MFMA
    if (loop >= 1 && K / (in_f32 ? 32 : 64) < gemm_kernel(idx).stages - 1) continue;
    const int64_t cn = (N + tn - 1) / tn;
    if (divides && (N % tn != 0 || cn > max_cn)) continue;
    const int64_t wgs = ((M + 127) / 128) * cn;
    const double cost = (double)((wgs + kAssumedCUs - 1) / kAssumedCUs) * tn - 1e-3 * tn;
    if (cost < best_cost) { best_cost = cost; best = idx; }
  }
  return best;
}

// Chooses kernel and row path for a GEMM (+ row subgraph).  `epi` selects the
// epilogue: 0 = plain (alpha, bias, store), 1 = row subgraph.  `need_rows` is
// true when the subgraph has a row reduction (then rows must be completed
// across tiles); without one any tiling is valid.
cf_status plan_rows(int64_t M, int64_t N, int64_t K, int in_f32, bool w_nk, int path, int epi, bool need_rows,
                    bool probe_device, Plan& pl, bool allow_cluster = true) {
  pl = Plan();
  if (!allow_cluster && need_rows) {
    if (path == PATH_CLUSTER)
      return fail(CF_ERR_UNSUPPORTED, "the allocation-free entry point has no row-cluster path");
    if (path == PATH_AUTO) path = N <= kWholeRowMaxN ? PATH_WHOLE_ROW : PATH_SPLIT;
  }
  const int tk = in_f32 ? 32 : 64;                     // k per 128-byte stage
  // Direct-to-LDS ring when K fills whole stages: W stored N x K (loop 1), or
  // bf16 W stored K x N with N a multiple of 8 (loop 2, transposing reads).
  const int loop = K % tk != 0 ? 0 : w_nk ? 1 : (!in_f32 && N % 8 == 0) ? 2 : 0;
  if (!need_rows) {
    pl.kidx = pick_tile(M, N, K, in_f32, loop, epi, false, 0);
    if (pl.kidx < 0) pl.kidx = pick_tile(M, N, K, in_f32, 0, epi, false, 0);
    pl.mode = ROWS_LOCAL;
  } else {
    if (path == PATH_AUTO) {
      // Row clusters when N splits into <= kAutoClusterPeers tiles; whole rows
      // instead when N is narrow and they give more workgroups (small M);
      // else split-N.  Every tile's exchange waits for the slowest of its
      // peers, and with 16 peers that wait costs more than split-N's fp32
      // round trip of x, so wide rows go to split-N unless a caller asks
      // for the cluster path.
      path = PATH_SPLIT;
      int ck = pick_tile(M, N, K, in_f32, loop, 1, true, kAutoClusterPeers);
      if (ck < 0) ck = pick_tile(M, N, K, in_f32, 0, 1, true, kAutoClusterPeers);
      if (ck >= 0) {
        path = PATH_CLUSTER;
        const GemmKernel& t = gemm_kernel(ck);
        const int64_t cluster_wgs = ((M + t.tm - 1) / t.tm) * ((N + t.tn - 1) / t.tn);
        if (N <= kWholeRowMaxN && (M + 31) / 32 > cluster_wgs) path = PATH_WHOLE_ROW;
      } else if (N <= kWholeRowMaxN) {
        path = PATH_WHOLE_ROW;
      }
    }
    if (path == PATH_WHOLE_ROW) {
      if (N > kWholeRowMaxN)
        return fail(CF_ERR_UNSUPPORTED, "whole-row path needs N <= %d (N = %lld)", kWholeRowMaxN, (long long)N);
      for (int tn : {128, 256, 384, 512, 768})
        if (tn >= N) {
          // the direct-to-LDS ring where compiled and K fills its prologue
          const int v2 = loop >= 1 ? find_gemm_kernel(in_f32, 32, tn, loop, 1) : -1;
          if (v2 >= 0 && K / tk >= gemm_kernel(v2).stages - 1) pl.kidx = v2;
          else pl.kidx = find_gemm_kernel(in_f32, 32, tn, 0, 1);
          break;
        }
      pl.mode = ROWS_LOCAL;
    } else if (path == PATH_CLUSTER) {
      pl.kidx = pick_tile(M, N, K, in_f32, loop, 1, true, kClusterMaxPeers);
      if (pl.kidx < 0) pl.kidx = pick_tile(M, N, K, in_f32, 0, 1, true, kClusterMaxPeers);
      if (pl.kidx < 0)
        return fail(CF_ERR_UNSUPPORTED, "cluster path: no tile width divides N = %lld into <= %d peers",
                    (long long)N, kClusterMaxPeers);
      pl.mode = ROWS_CLUSTER;
    } else if (path == PATH_SPLIT) {
      pl.kidx = pick_tile(M, N, K, in_f32, loop, 2, false, 0);
      if (pl.kidx < 0) pl.kidx = pick_tile(M, N, K, in_f32, 0, 2, false, 0);
      pl.mode = ROWS_SPLIT;
    } else {
      return fail(CF_ERR_UNSUPPORTED, "unknown path %d", path);
    }
  }
  if (pl.kidx < 0) return fail(CF_ERR_UNSUPPORTED, "no compiled tile for this shape");
  const GemmKernel& t = gemm_kernel(pl.kidx);
  pl.tm = t.tm;
  pl.tn = t.tn;
  pl.cn = (int)((N + t.tn - 1) / t.tn);
  pl.num_rb = (int)((M + t.tm - 1) / t.tm);
  pl.slots = (pl.num_rb + 7) / 8;
  if (pl.mode == ROWS_CLUSTER && probe_device) {
    // Every peer group must be resident at once: cap the persistent grid.
    const int cap = resident_wgs(pl.kidx);
    const int slots = cap / (8 * pl.cn);
    if (slots < 1) return fail(CF_ERR_UNSUPPORTED, "cluster path: %d peers do not fit the device", pl.cn);
    pl.slots = std::min(pl.slots, std::min(slots, kMaxSlots / 8));
  }
  // the finish pass reads a row's partials one per lane of a 64-lane wave
  if (pl.mode == ROWS_SPLIT && pl.cn > 64)
    return fail(CF_ERR_UNSUPPORTED, "split path: %d tiles per row exceed 64", pl.cn);
  if (pl.mode == ROWS_CLUSTER && (pl.tm > kRecRows || pl.cn > kRecPeers))
    return fail(CF_ERR_UNSUPPORTED, "cluster path: tile of %d rows x %d peers exceeds the exchange records",
                pl.tm, pl.cn);
  size_workspace(pl, M, N, allow_cluster);
  return CF_OK;
}

void bind_workspace(const Plan& pl, void* ws, GemmRowsParams& p) {
  char* b = reinterpret_cast<char*>(ws);
  if (pl.mode == ROWS_CLUSTER) {
    p.ws_err = reinterpret_cast<unsigned*>(b);
    p.ws_arrive = reinterpret_cast<unsigned long long*>(b + 256);
    static_assert(kWsCounterBytes % 256 == 0, "records alignment");
    p.ws_part = reinterpret_cast<float*>(b + pl.off_part);
    p.spin_limit = kSpinLimitDefault;
    p.leader = pl.cn >= kLeaderFollowerPeers;
  } else if (pl.mode == ROWS_SPLIT) {
    p.ws_part = reinterpret_cast<float*>(b + pl.off_part);
    p.ws_x = reinterpret_cast<float*>(b + pl.off_x);
  }
}

// Runs a planned GEMM + row subgraph (and the finish pass of the split path).
cf_status run_rows(const Plan& pl, GemmRowsParams p, void* ws, hipStream_t st) {
  p.mode = pl.mode;
  p.cn = pl.cn;
  p.num_rb = pl.num_rb;
  p.slots = pl.slots;
  bind_workspace(pl, ws, p);
  if (pl.mode == ROWS_SPLIT) {
    RowEpi full = p.epi;
    // The GEMM runs stage 1 only and publishes x and partial statistics.
    p.epi.norm = NORM_NONE;
    p.epi.act = ACT_NONE;
    p.epi.softmax = 0;
    p.epi.Y = nullptr;
    p.epi.quant = 0;
    cf_status s = hip_status(launch_gemm_rows(p, pl.kidx, st), "GEMM launch");
    if (s != CF_OK) return s;
    RowKernelParams f{};
    f.M = p.M;
    f.N = p.N;
    f.P = p.ws_x;
    f.ldp = p.N;
    f.p_f32 = 1;
    f.finish = 1;
    f.cn = pl.cn;
    f.tn = pl.tn;
    f.part = p.ws_part;
    f.epi = full;
    f.epi.alpha = 1.0f;
    f.epi.bias = nullptr;
    f.epi.R = nullptr;
    return hip_status(launch_row_kernel(f, st), "finish launch");
  }
  return hip_status(launch_gemm_rows(p, pl.kidx, st), "GEMM launch");
}

// ---------------------------------------------------------------------------
// Node lists -> RowEpi (the fixed stage grammar).
// ---------------------------------------------------------------------------
cf_status parse_nodes(const cf_node* nodes, int n, int64_t M, int64_t N, cf_dtype in, RowEpi& e,
                      bool allow_softmax, int* softmax, float* softmax_scale) {
  e = RowEpi{};
  e.alpha = 1.0f;
  e.qmax = 448.0f;
  if (softmax) *softmax = 0;
  if (!nodes || n <= 0) return fail(CF_ERR_NULL, "empty node list");
  if (n == 1 && nodes[0].kind == CF_N_SOFTMAX) {
    if (!allow_softmax) return fail(CF_ERR_UNSUPPORTED, "SOFTMAX is available in cf_rowop only");
    const cf_node& d = nodes[0];
    if (d.dtype != CF_F32 && d.dtype != CF_BF16) return fail(CF_ERR_DTYPE, "SOFTMAX output dtype");
    cf_status s = check_matrix("SOFTMAX out", d.out, M, N, d.ld, d.dtype, true);
    if (s != CF_OK) return s;
    e.Y = d.out;
    e.ldy = d.ld;
    e.y_f32 = d.dtype == CF_F32;
    *softmax = 1;
    *softmax_scale = d.f0;
    return CF_OK;
  }
  // Grammar position of each kind; positions must strictly increase.
  auto rank = [](cf_node_kind k) -> int {
    switch (k) {
      case CF_N_SCALE: return 0;
      case CF_N_BIAS: return 1;
      case CF_N_RESIDUAL: return 2;
      case CF_N_LAYERNORM: case CF_N_RMSNORM: return 3;
      case CF_N_GELU: case CF_N_GELU_TANH: case CF_N_RELU: case CF_N_SOFTCAP: return 4;
      case CF_N_SOFTMAX: return 5;
      case CF_N_STORE: return 6;
      case CF_N_ROWAMAX_QUANT: return 7;
      default: return -1;
    }
  };
  int last = -1;
  for (int i = 0; i < n; ++i) {
    const cf_node& d = nodes[i];
    const int r = rank(d.kind);
    if (r < 0) return fail(CF_ERR_UNSUPPORTED, "node %d: kind %d is not in the fused vocabulary", i, (int)d.kind);
    if (r <= last)
      return fail(CF_ERR_UNSUPPORTED,
                  "node %d: kind %d out of order (grammar: SCALE BIAS RESIDUAL NORM ACT SOFTMAX STORE QUANT)", i,
                  (int)d.kind);
    last = r;
    cf_status s = CF_OK;
    switch (d.kind) {
      case CF_N_SCALE: e.alpha = d.f0; break;
      case CF_N_BIAS:
        if (!d.v0) return fail(CF_ERR_NULL, "BIAS vector is NULL");
        if ((s = check_vec("BIAS", d.v0)) != CF_OK) return s;
        e.bias = d.v0;
        break;
      case CF_N_RESIDUAL:
        if (d.dtype != CF_F32 && d.dtype != CF_BF16) return fail(CF_ERR_DTYPE, "RESIDUAL dtype must be F32 or BF16");
        if (!allow_softmax && d.dtype != in)
          return fail(CF_ERR_DTYPE, "RESIDUAL dtype must equal the GEMM input dtype");
        if ((s = check_matrix("RESIDUAL", d.in, M, N, d.ld, d.dtype, true)) != CF_OK) return s;
        e.R = d.in;
        e.ldr = d.ld;
        e.r_f32 = d.dtype == CF_F32;
        break;
      case CF_N_LAYERNORM: case CF_N_RMSNORM:
        if ((s = check_vec("gamma", d.v0)) != CF_OK || (s = check_vec("beta", d.v1)) != CF_OK) return s;
        if (!(d.f0 >= 0.0f)) return fail(CF_ERR_SHAPE, "eps must be >= 0");
        e.norm = d.kind == CF_N_LAYERNORM ? NORM_LAYER : NORM_RMS;
        e.gamma = d.v0;
        e.beta = d.kind == CF_N_LAYERNORM ? d.v1 : nullptr;
        e.eps = d.f0;
        break;
      case CF_N_GELU: e.act = ACT_GELU; break;
      case CF_N_GELU_TANH: e.act = ACT_GELU_TANH; break;
      case CF_N_RELU: e.act = ACT_RELU; break;
      case CF_N_SOFTCAP:
        if (!(d.f0 > 0.0f) || !std::isfinite(d.f0)) return fail(CF_ERR_SHAPE, "SOFTCAP cap must be finite and > 0");
        e.act = ACT_SOFTCAP;
        e.softcap = d.f0;
        break;
      case CF_N_SOFTMAX:
        if (e.norm != NORM_NONE) return fail(CF_ERR_UNSUPPORTED, "SOFTMAX after a NORM is not in the fused vocabulary");
        e.softmax = 1;
        break;
      case CF_N_STORE:
        if (d.dtype != CF_F32 && d.dtype != CF_BF16) return fail(CF_ERR_DTYPE, "STORE dtype must be F32 or BF16");
        if ((s = check_matrix("STORE", d.out, M, N, d.ld, d.dtype, true)) != CF_OK) return s;
        e.Y = d.out;
        e.ldy = d.ld;
        e.y_f32 = d.dtype == CF_F32;
        break;
      case CF_N_ROWAMAX_QUANT:
        if (!d.out) return fail(CF_ERR_NULL, "ROWAMAX_QUANT scale output is NULL");
        if (!(d.f0 > 0.0f)) return fail(CF_ERR_SHAPE, "ROWAMAX_QUANT qmax must be > 0");
        if (d.out2) {
          if (!aligned16(d.out2) || d.ld % 16 != 0)
            return fail(CF_ERR_ALIGN, "ROWAMAX_QUANT codes: 16-byte alignment and ld %% 16 == 0 required");
          if (M > 0 && d.ld < N) return fail(CF_ERR_LD, "ROWAMAX_QUANT codes: ld < N");
        }
        e.quant = 1;
        e.qmax = d.f0;
        e.s_out = reinterpret_cast<float*>(d.out);
        e.q_out = reinterpret_cast<uint8_t*>(d.out2);
        e.ldq = d.ld;
        break;
      default: break;
    }
  }
  if (!e.Y && !e.quant) return fail(CF_ERR_UNSUPPORTED, "node list has no output (STORE or ROWAMAX_QUANT)");
  return CF_OK;
}

cf_status check_gemm_shape(int64_t M, int64_t N, int64_t K) {
  if (M < 0 || N <= 0 || K <= 0) return fail(CF_ERR_SHAPE, "need M >= 0, N > 0, K > 0");
  if (N % 32 != 0) return fail(CF_ERR_SHAPE, "N = %lld must be a multiple of 32", (long long)N);
  if (K % 16 != 0) return fail(CF_ERR_SHAPE, "K = %lld must be a multiple of 16", (long long)K);
  if (N > 8192) return fail(CF_ERR_SHAPE, "N = %lld exceeds 8192", (long long)N);
  if (M > (int64_t)1 << 30 || K > (int64_t)1 << 30) return fail(CF_ERR_SHAPE, "size exceeds 2^30");
  return CF_OK;
}

bool outputs_alias(const void* out, std::initializer_list<const void*> ins) {
  if (!out) return false;
  for (const void* p : ins)
    if (p && p == out) return true;
  return false;
}

// Shared body of cf_gemm_postnorm / cf_gemm_subgraph.
// scratch = true: ws is the library's own allocation-free scratch (no
// header, no cluster path; a plan needing more than ws_bytes is refused).
cf_status rows_common(int64_t M, int64_t N, int64_t K, cf_dtype in, const void* X, int64_t ldx,
                      const void* W, int64_t ldw, cf_layout wl, const RowEpi& epi, int path,
                      void* ws, size_t ws_bytes, void* stream, bool size_only, size_t* ws_out,
                      bool scratch = false) {
  cf_status s = check_gemm_shape(M, N, K);
  if (s != CF_OK) return s;
  if (in != CF_F32 && in != CF_BF16) return fail(CF_ERR_DTYPE, "input dtype must be F32 or BF16");
  if (wl != CF_LAYOUT_KN && wl != CF_LAYOUT_NK) return fail(CF_ERR_UNSUPPORTED, "unknown weight layout");
  if ((s = check_matrix("X", X, M, K, ldx, in, true)) != CF_OK) return s;
  if ((s = check_matrix("W", W, 1, wl == CF_LAYOUT_NK ? K : N, ldw, in, true)) != CF_OK) return s;
  const bool need_rows = epi.norm != NORM_NONE || epi.quant || epi.softmax;
  // The plain epilogue only applies alpha and bias; anything else runs the
  // row-subgraph epilogue.
  const int epi_kind = (need_rows || epi.R || epi.act != ACT_NONE) ? 1 : 0;
  Plan pl;
  // Validation and sizing never touch the device; residency is queried only
  // right before a launch.
  if ((s = plan_rows(M, N, K, in == CF_F32, wl == CF_LAYOUT_NK, path, epi_kind, need_rows, false, pl,
                     !scratch)) != CF_OK)
    return s;
  if (size_only) {
    *ws_out = pl.ws;
    return CF_OK;
  }
  for (const void* out : {(const void*)epi.Y, (const void*)epi.s_out, (const void*)epi.q_out})
    if (outputs_alias(out, {X, W, epi.R, (const void*)epi.bias, (const void*)epi.gamma, (const void*)epi.beta}))
      return fail(CF_ERR_ALIAS, "an output aliases an input");
  if (M == 0) return CF_OK;   // nothing to compute: no workspace needed
  if (scratch && pl.ws > ws_bytes)
    return fail(CF_ERR_WORKSPACE, "this shape needs %zu bytes of scratch; the allocation-free entry point holds %zu",
                pl.ws, ws_bytes);
  if (pl.ws > 0) {
    if (!ws) return fail(CF_ERR_WORKSPACE, "workspace of %zu bytes required", pl.ws);
    if (ws_bytes < pl.ws) return fail(CF_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, pl.ws);
    if (!aligned16(ws)) return fail(CF_ERR_ALIGN, "workspace is not 16-byte aligned");
  }
  if (M == 0) return CF_OK;
  if (pl.mode == ROWS_CLUSTER &&
      (s = plan_rows(M, N, K, in == CF_F32, wl == CF_LAYOUT_NK, path, epi_kind, need_rows, true, pl)) != CF_OK)
    return s;
  GemmRowsParams p{};
  p.batch = 1;
  p.M = (int)M;
  p.N = (int)N;
  p.K = (int)K;
  p.X = X;
  p.ldx = ldx;
  p.W = W;
  p.ldw = ldw;
  p.w_nk = wl == CF_LAYOUT_NK;
  p.epi = epi;
  return run_rows(pl, p, ws, reinterpret_cast<hipStream_t>(stream));
}

cf_status postnorm_epi(const cf_postnorm_args* a, RowEpi& e) {
  if (!a) return fail(CF_ERR_NULL, "args is NULL");
  if (a->struct_size != sizeof(cf_postnorm_args))
    return fail(CF_ERR_STRUCT, "struct_size %zu != %zu", a->struct_size, sizeof(cf_postnorm_args));
  if (a->in_dtype != CF_F32 && a->in_dtype != CF_BF16) return fail(CF_ERR_DTYPE, "in_dtype must be F32 or BF16");
  if (a->out_dtype != CF_F32 && a->out_dtype != CF_BF16) return fail(CF_ERR_DTYPE, "out_dtype must be F32 or BF16");
  if (a->in_dtype == CF_F32 && a->out_dtype != CF_F32) return fail(CF_ERR_DTYPE, "F32 input needs F32 output");
  if (!(a->eps >= 0.0f)) return fail(CF_ERR_SHAPE, "eps must be >= 0");
  cf_status s;
  if ((s = check_matrix("Y", a->Y, a->M, a->N, a->ldy, a->out_dtype, true)) != CF_OK) return s;
  if ((s = check_matrix("R", a->R, a->M, a->N, a->ldr, a->in_dtype, false)) != CF_OK) return s;
  if ((s = check_vec("bias", a->bias)) != CF_OK || (s = check_vec("gamma", a->gamma)) != CF_OK ||
      (s = check_vec("beta", a->beta)) != CF_OK)
    return s;
  e = RowEpi{};
  e.alpha = a->alpha;
  e.bias = a->bias;
  e.R = a->R;
  e.ldr = a->ldr;
  e.r_f32 = a->in_dtype == CF_F32;
  e.norm = NORM_LAYER;
  e.gamma = a->gamma;
  e.beta = a->beta;
  e.eps = a->eps;
  e.Y = a->Y;
  e.ldy = a->ldy;
  e.y_f32 = a->out_dtype == CF_F32;
  e.qmax = 448.0f;
  return CF_OK;
}

cf_status subgraph_epi(const cf_subgraph_args* a, RowEpi& e) {
  if (!a) return fail(CF_ERR_NULL, "args is NULL");
  if (a->struct_size != sizeof(cf_subgraph_args))
    return fail(CF_ERR_STRUCT, "struct_size %zu != %zu", a->struct_size, sizeof(cf_subgraph_args));
  if (a->in_dtype != CF_F32 && a->in_dtype != CF_BF16) return fail(CF_ERR_DTYPE, "in_dtype must be F32 or BF16");
  return parse_nodes(a->nodes, a->n_nodes, a->M, a->N, a->in_dtype, e, false, nullptr, nullptr);
}

}  // namespace

namespace cf {
// cf_gemm_subgraph through a given scratch buffer (the allocation-free entry
// point's device array): validation as cf_gemm_subgraph, then a plan without
// the row-cluster path whose buffers must fit in scratch_bytes.
// validate_only: check the arguments and that the plan fits scratch_bytes,
// touch nothing on the device; *empty tells whether the call is a no-op.
cf_status gemm_subgraph_scratch(const cf_subgraph_args* a, void* scratch, size_t scratch_bytes, void* hip_stream,
                                bool validate_only, bool* empty) {
  try {
    RowEpi e;
    cf_status s = subgraph_epi(a, e);
    if (s != CF_OK) return s;
    if (validate_only) {
      size_t need = 0;
      if ((s = rows_common(a->M, a->N, a->K, a->in_dtype, a->X, a->ldx, a->W, a->ldw, a->w_layout, e, a->path,
                           nullptr, 0, nullptr, true, &need, true)) != CF_OK)
        return s;
      if (need > scratch_bytes)
        return fail(CF_ERR_WORKSPACE,
                    "this shape needs %zu bytes of scratch; the allocation-free entry point holds %zu", need,
                    scratch_bytes);
      if (empty) *empty = a->M == 0;
      return CF_OK;
    }
    return rows_common(a->M, a->N, a->K, a->in_dtype, a->X, a->ldx, a->W, a->ldw, a->w_layout, e, a->path,
                       scratch, scratch_bytes, hip_stream, false, nullptr, true);
  } catch (...) {
    return fail(CF_ERR_HIP, "internal error");
  }
}

cf_status record_error(cf_status s, const char* what) { return fail(s, "%s", what); }
}  // namespace cf

extern "C" {

int cf_version(void) { return CF_VERSION; }

const char* cf_last_error(void) { return g_last_error.c_str(); }

const char* cf_status_string(cf_status s) {
  switch (s) {
    case CF_OK: return "CF_OK";
    case CF_ERR_NULL: return "CF_ERR_NULL: a required pointer is NULL";
    case CF_ERR_SHAPE: return "CF_ERR_SHAPE: invalid size";
    case CF_ERR_LD: return "CF_ERR_LD: leading dimension too small";
    case CF_ERR_ALIGN: return "CF_ERR_ALIGN: misaligned pointer or leading dimension";
    case CF_ERR_DTYPE: return "CF_ERR_DTYPE: unsupported dtype";
    case CF_ERR_WORKSPACE: return "CF_ERR_WORKSPACE: workspace missing or too small";
    case CF_ERR_UNSUPPORTED: return "CF_ERR_UNSUPPORTED: outside the compiled vocabulary";
    case CF_ERR_ALIAS: return "CF_ERR_ALIAS: an output aliases an input";
    case CF_ERR_HIP: return "CF_ERR_HIP: HIP runtime error";
    case CF_ERR_STRUCT: return "CF_ERR_STRUCT: struct_size mismatch";
    case CF_ERR_PEER_TIMEOUT: return "CF_ERR_PEER_TIMEOUT: a wait for peer workgroups gave up";
  }
  return "unknown cf_status";
}

size_t cf_gemm_postnorm_workspace(const cf_postnorm_args* a) {
  try {
    RowEpi e;
    if (postnorm_epi(a, e) != CF_OK) return 0;
    size_t ws = 0;
    if (rows_common(a->M, a->N, a->K, a->in_dtype, a->X, a->ldx, a->W, a->ldw, a->w_layout, e, a->path,
                    nullptr, 0, nullptr, true, &ws) != CF_OK)
      return 0;
    return ws;
  } catch (...) {
    return 0;
  }
}

cf_status cf_gemm_postnorm(const cf_postnorm_args* a, void* workspace, size_t ws_bytes, void* hip_stream) {
  try {
    RowEpi e;
    cf_status s = postnorm_epi(a, e);
    if (s != CF_OK) return s;
    return rows_common(a->M, a->N, a->K, a->in_dtype, a->X, a->ldx, a->W, a->ldw, a->w_layout, e, a->path,
                       workspace, ws_bytes, hip_stream, false, nullptr);
  } catch (...) {
    return fail(CF_ERR_HIP, "internal error");
  }
}

size_t cf_gemm_subgraph_workspace(const cf_subgraph_args* a) {
  try {
    RowEpi e;
    if (subgraph_epi(a, e) != CF_OK) return 0;
    size_t ws = 0;
    if (rows_common(a->M, a->N, a->K, a->in_dtype, a->X, a->ldx, a->W, a->ldw, a->w_layout, e, a->path,
                    nullptr, 0, nullptr, true, &ws) != CF_OK)
      return 0;
    return ws;
  } catch (...) {
    return 0;
  }
}

cf_status cf_gemm_subgraph(const cf_subgraph_args* a, void* workspace, size_t ws_bytes, void* hip_stream) {
  try {
    RowEpi e;
    cf_status s = subgraph_epi(a, e);
    if (s != CF_OK) return s;
    return rows_common(a->M, a->N, a->K, a->in_dtype, a->X, a->ldx, a->W, a->ldw, a->w_layout, e, a->path,
                       workspace, ws_bytes, hip_stream, false, nullptr);
  } catch (...) {
    return fail(CF_ERR_HIP, "internal error");
  }
}

cf_status cf_gemm(int64_t batch, int64_t M, int64_t N, int64_t K, cf_dtype in, cf_dtype out, const void* A,
                  int64_t lda, int64_t sa, const void* B, int64_t ldb, int64_t sb, cf_layout b_layout,
                  const float* bias, float alpha, void* C, int64_t ldc, int64_t sc, void* hip_stream) {
  try {
    cf_status s = check_gemm_shape(M, N, K);
    if (s != CF_OK) return s;
    if (batch < 0 || batch > 65535) return fail(CF_ERR_SHAPE, "batch must be in [0, 65535]");
    if (in != CF_F32 && in != CF_BF16) return fail(CF_ERR_DTYPE, "input dtype must be F32 or BF16");
    if (out != CF_F32 && out != CF_BF16) return fail(CF_ERR_DTYPE, "output dtype must be F32 or BF16");
    if (b_layout != CF_LAYOUT_KN && b_layout != CF_LAYOUT_NK) return fail(CF_ERR_UNSUPPORTED, "unknown layout");
    if ((s = check_matrix("A", A, M, K, lda, in, true)) != CF_OK) return s;
    if ((s = check_matrix("B", B, 1, b_layout == CF_LAYOUT_NK ? K : N, ldb, in, true)) != CF_OK) return s;
    if ((s = check_matrix("C", C, M, N, ldc, out, true)) != CF_OK) return s;
    if ((s = check_vec("bias", bias)) != CF_OK) return s;
    if (batch > 1 && (sa % 8 != 0 || sb % 8 != 0 || sc % 8 != 0 || sa < 0 || sb < 0 || sc < 0))
      return fail(CF_ERR_ALIGN, "batch strides must be non-negative multiples of 8 elements");
    if (outputs_alias(C, {A, B, (const void*)bias})) return fail(CF_ERR_ALIAS, "C aliases an input");
    if (M == 0 || batch == 0) return CF_OK;
    Plan pl;
    if ((s = plan_rows(M, N, K, in == CF_F32, b_layout == CF_LAYOUT_NK, PATH_AUTO, 0, false, false, pl)) != CF_OK)
      return s;
    GemmRowsParams p{};
    p.batch = (int)batch;
    p.M = (int)M;
    p.N = (int)N;
    p.K = (int)K;
    p.X = A;
    p.ldx = lda;
    p.sx = sa;
    p.W = B;
    p.ldw = ldb;
    p.sw = sb;
    p.w_nk = b_layout == CF_LAYOUT_NK;
    p.epi.alpha = alpha;
    p.epi.bias = bias;
    p.epi.Y = C;
    p.epi.ldy = ldc;
    p.epi.sy = sc;
    p.epi.y_f32 = out == CF_F32;
    p.epi.qmax = 448.0f;
    return run_rows(pl, p, nullptr, reinterpret_cast<hipStream_t>(hip_stream));
  } catch (...) {
    return fail(CF_ERR_HIP, "internal error");
  }
}

cf_status cf_rowop(int64_t batch, int64_t M, int64_t N, cf_dtype in, const void* P, int64_t ldp, int64_t sp,
                   const cf_node* nodes, int n_nodes, void* hip_stream) {
  try {
    if (M < 0 || N <= 0 || N % 4 != 0 || N > 8192) return fail(CF_ERR_SHAPE, "need M >= 0, 0 < N <= 8192, N %% 4 == 0");
    if (batch < 0 || batch > 65535) return fail(CF_ERR_SHAPE, "batch must be in [0, 65535]");
    if (batch * M > ((int64_t)1 << 31) - 1) return fail(CF_ERR_SHAPE, "batch * M exceeds 2^31 - 1 rows");
    if (in != CF_F32 && in != CF_BF16) return fail(CF_ERR_DTYPE, "input dtype must be F32 or BF16");
    cf_status s = check_matrix("P", P, batch > 0 ? M : 0, N, ldp, in, true);
    if (s != CF_OK) return s;
    if (batch > 1 && (sp < 0 || (sp * (int64_t)dsize(in)) % 16 != 0))
      return fail(CF_ERR_ALIGN, "batch stride of P must be a non-negative multiple of 16 bytes");
    const int64_t rows = batch * M;   // node matrices and s hold batch * M consecutive rows
    RowKernelParams r{};
    if ((s = parse_nodes(nodes, n_nodes, rows, N, in, r.epi, true, &r.softmax, &r.softmax_scale)) != CF_OK) return s;
    for (const void* out : {(const void*)r.epi.Y, (const void*)r.epi.s_out, (const void*)r.epi.q_out})
      if (outputs_alias(out, {P, r.epi.R, (const void*)r.epi.bias}))
        return fail(CF_ERR_ALIAS, "an output aliases an input");
    if (rows == 0) return CF_OK;
    r.M = (int)rows;
    r.N = (int)N;
    r.P = P;
    r.ldp = ldp;
    r.rows_per_batch = (int)M;
    r.sp = batch > 1 ? sp : 0;
    r.p_f32 = in == CF_F32;
    return hip_status(launch_row_kernel(r, reinterpret_cast<hipStream_t>(hip_stream)), "row kernel launch");
  } catch (...) {
    return fail(CF_ERR_HIP, "internal error");
  }
}

cf_status cf_workspace_check(void* workspace, size_t ws_bytes, void* hip_stream) {
  try {
    if (!workspace) return CF_OK;   // no workspace: no cluster exchange ran
    if (ws_bytes < sizeof(unsigned)) return fail(CF_ERR_WORKSPACE, "workspace smaller than its error word");
    if (!aligned16(workspace)) return fail(CF_ERR_ALIGN, "workspace is not 16-byte aligned");
    hipStream_t st = reinterpret_cast<hipStream_t>(hip_stream);
    cf_status s = hip_status(hipStreamSynchronize(st), "stream synchronize");
    if (s != CF_OK) return s;
    unsigned err = 0;
    if ((s = hip_status(hipMemcpy(&err, workspace, sizeof(err), hipMemcpyDeviceToHost), "read error word")) != CF_OK)
      return s;
    if (err == 0) return CF_OK;
    const unsigned zero = 0;
    if ((s = hip_status(hipMemcpy(workspace, &zero, sizeof(zero), hipMemcpyHostToDevice), "clear error word")) != CF_OK)
      return s;
    return fail(CF_ERR_PEER_TIMEOUT,
                "a row-cluster wait for peer workgroups exceeded its bound; results written through this "
                "workspace since the last check are invalid (the word is now cleared)");
  } catch (...) {
    return fail(CF_ERR_HIP, "internal error");
  }
}

// MLP form.  The hidden chunks are split over workgroups (their partial
// products meeting in the workspace) when the split grid fits one generation
// of a 256-CU device, one workgroup per CU; otherwise one workgroup per row
// block runs all chunks and needs no workspace.  Measured at K = 1024,
// N1 = 512: split 28-32 us against 37-39 us at 96-128 row blocks, whole
// 42-53 us against 51-62 us at 160-255.  The rule depends on the arguments
// only.
static constexpr int64_t kMlpSplitMaxWorkgroups = 256;
static bool mlp_split(const cf_b2b_args* a) {
  return a->N1 > kMlpHidden &&
         a->batch * ((a->M + kMlpRows - 1) / kMlpRows) * (a->N1 / kMlpHidden) <= kMlpSplitMaxWorkgroups;
}

// Workspace of the split MLP: the fixed counter region (words [batch][row
// blocks] at its start), then fp32 partials [batch][cn][M][N2].  The counter
// region does not depend on the shape, so partials of one call never land
// where a later call of another shape expects zeroed counters.  Other B2B
// forms need none.
static size_t mlp_workspace(const cf_b2b_args* a) {
  if (!a || a->struct_size != sizeof(cf_b2b_args) || a->mid != CF_MID_RELU_BIAS || a->M <= 0 || a->batch <= 0 ||
      !mlp_split(a))
    return 0;
  const int64_t cn = a->N1 / kMlpHidden;
  return kMlpCounterBytes + (size_t)(a->batch * cn * a->M * a->N2 * 4);
}
static_assert(kMlpSplitMaxWorkgroups <= kMlpMaxRowBlocks, "split MLP counters");

size_t cf_b2bgemm_workspace(const cf_b2b_args* a) {
  try {
    return mlp_workspace(a);
  } catch (...) {
    return 0;
  }
}

cf_status cf_b2bgemm(const cf_b2b_args* a, void* workspace, size_t ws_bytes, void* hip_stream) {
  try {
    if (!a) return fail(CF_ERR_NULL, "args is NULL");
    if (a->struct_size != sizeof(cf_b2b_args))
      return fail(CF_ERR_STRUCT, "struct_size %zu != %zu", a->struct_size, sizeof(cf_b2b_args));
    if (a->dtype != CF_BF16) return fail(CF_ERR_DTYPE, "cf_b2bgemm computes in bf16 only");
    if (a->batch < 0 || a->batch > 65535 || a->M < 0 || a->K <= 0 || a->N1 <= 0 || a->N2 <= 0)
      return fail(CF_ERR_SHAPE, "need 0 <= batch <= 65535, M >= 0, K, N1, N2 > 0");
    if (a->M > (int64_t)1 << 30 || a->N1 > (int64_t)1 << 30) return fail(CF_ERR_SHAPE, "size exceeds 2^30");
    const bool ffn = a->mid == CF_MID_GELU_BIAS, mlp = a->mid == CF_MID_RELU_BIAS;
    if (!ffn && !mlp && a->mid != CF_MID_SOFTMAX) return fail(CF_ERR_UNSUPPORTED, "unknown mid op");
    if (a->out != CF_OUT_STORE && a->out != CF_OUT_BIAS_RESIDUAL_LN && a->out != CF_OUT_BIAS_RELU)
      return fail(CF_ERR_UNSUPPORTED, "unknown out op");
    if (a->out == CF_OUT_BIAS_RELU && !mlp) return fail(CF_ERR_UNSUPPORTED, "the output ReLU belongs to the MLP form");
    cf_status s;
    if (mlp) {
      if (a->w1_layout != CF_LAYOUT_NK || a->w2_layout != CF_LAYOUT_NK)
        return fail(CF_ERR_UNSUPPORTED, "MLP weights must be stored N x K (W1^T: N1 x K, W2^T: N2 x N1)");
      if (!b2b_mlp_supported((int)std::min<int64_t>(a->K, 1 << 30), (int)a->N1, (int)a->N2))
        return fail(CF_ERR_UNSUPPORTED, "MLP needs N2 = 128, N1 a multiple of %d, K a multiple of 64 and >= 128 "
                    "(K = %lld, N1 = %lld, N2 = %lld)", kMlpHidden, (long long)a->K, (long long)a->N1, (long long)a->N2);
      if (a->out == CF_OUT_BIAS_RESIDUAL_LN || a->R || a->gamma || a->beta)
        return fail(CF_ERR_UNSUPPORTED, "the MLP form stores O + b2 or ReLU(O + b2) only");
      if ((s = check_vec("b1", a->b1)) != CF_OK) return s;
      if (a->M > 0 && a->batch > 0) {
        const size_t need = mlp_workspace(a);
        if (need > 0) {
          if (!workspace) return fail(CF_ERR_WORKSPACE, "workspace of %zu bytes required (N1 split over workgroups)", need);
          if (ws_bytes < need) return fail(CF_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
          if (!aligned16(workspace)) return fail(CF_ERR_ALIGN, "workspace is not 16-byte aligned");
        }
      }
    } else if (ffn) {
      if (a->w1_layout != CF_LAYOUT_NK || a->w2_layout != CF_LAYOUT_NK)
        return fail(CF_ERR_UNSUPPORTED, "FFN weights must be stored N x K (W1^T: N1 x K, W2^T: N2 x N1)");
      if (a->K != a->N2) return fail(CF_ERR_UNSUPPORTED, "FFN needs K == N2 = d (K = %lld, N2 = %lld)", (long long)a->K, (long long)a->N2);
      if (!b2b_ffn_supported((int)a->N1, (int)a->N2))
        return fail(CF_ERR_UNSUPPORTED, "FFN (N1, N2) = (%lld, %lld) not compiled", (long long)a->N1,
                    (long long)a->N2);
      if ((s = check_vec("b1", a->b1)) != CF_OK) return s;
    } else {
      if (a->w1_layout != CF_LAYOUT_NK || a->w2_layout != CF_LAYOUT_KN)
        return fail(CF_ERR_UNSUPPORTED, "attention: keys stored Lk x d (NK), values Lk x d (KN)");
      if (a->K != a->N2 || !b2b_attention_supported((int)a->K))
        return fail(CF_ERR_UNSUPPORTED, "attention head dim %lld not compiled (64, 128)", (long long)a->K);
      if (a->out != CF_OUT_STORE || a->b2 || a->R || a->b1)
        return fail(CF_ERR_UNSUPPORTED, "attention supports the plain store of O only");
      if (!std::isfinite(a->mid_scale) || !(a->mid_scale > 0.0f))
        return fail(CF_ERR_SHAPE, "mid_scale must be finite and > 0");
    }
    const bool empty = a->M == 0 || a->batch == 0;
    const int64_t w1_rows = a->N1, w1_cols = a->K;
    const int64_t w2_rows = (ffn || mlp) ? a->N2 : a->N1, w2_cols = (ffn || mlp) ? a->N1 : a->N2;
    if ((s = check_matrix("X", a->X, empty ? 0 : a->M, a->K, a->ldx, CF_BF16, true)) != CF_OK) return s;
    if ((s = check_matrix("W1", a->W1, empty ? 0 : w1_rows, w1_cols, a->ldw1, CF_BF16, true)) != CF_OK) return s;
    if ((s = check_matrix("W2", a->W2, empty ? 0 : w2_rows, w2_cols, a->ldw2, CF_BF16, true)) != CF_OK) return s;
    if ((s = check_matrix("O", a->O, empty ? 0 : a->M, a->N2, a->ldo, CF_BF16, true)) != CF_OK) return s;
    if ((s = check_matrix("R", a->R, empty ? 0 : a->M, a->N2, a->ldr, CF_BF16, false)) != CF_OK) return s;
    if ((s = check_vec("b2", a->b2)) != CF_OK || (s = check_vec("gamma", a->gamma)) != CF_OK ||
        (s = check_vec("beta", a->beta)) != CF_OK)
      return s;
    if (a->batch > 1)
      for (int64_t st : {a->sx, a->sw1, a->sw2, a->so, a->R ? a->sr : (int64_t)0})
        if (st < 0 || st % 8 != 0) return fail(CF_ERR_ALIGN, "batch strides must be non-negative multiples of 8");
    if (outputs_alias(a->O, {a->X, a->W1, a->W2, a->R})) return fail(CF_ERR_ALIAS, "O aliases an input");
    if (!(a->eps >= 0.0f)) return fail(CF_ERR_SHAPE, "eps must be >= 0");
    if (empty) return CF_OK;
    B2BParams p{};
    p.batch = (int)a->batch;
    p.M = (int)a->M;
    p.K = (int)a->K;
    p.N1 = (int)a->N1;
    p.N2 = (int)a->N2;
    p.X = reinterpret_cast<const uint16_t*>(a->X);
    p.ldx = a->ldx;
    p.sx = a->sx;
    p.W1 = reinterpret_cast<const uint16_t*>(a->W1);
    p.ldw1 = a->ldw1;
    p.sw1 = a->sw1;
    p.b1 = a->b1;
    p.mid_scale = a->mid_scale;
    p.W2 = reinterpret_cast<const uint16_t*>(a->W2);
    p.ldw2 = a->ldw2;
    p.sw2 = a->sw2;
    p.out_ln = a->out == CF_OUT_BIAS_RESIDUAL_LN;
    p.b2 = a->b2;
    p.R = reinterpret_cast<const uint16_t*>(a->R);
    p.ldr = a->ldr;
    p.sr = a->sr;
    p.gamma = a->gamma;
    p.beta = a->beta;
    p.eps = a->eps;
    p.O = reinterpret_cast<uint16_t*>(a->O);
    p.ldo = a->ldo;
    p.so = a->so;
    hipStream_t st = reinterpret_cast<hipStream_t>(hip_stream);
    if (mlp) {
      p.out_relu = a->out == CF_OUT_BIAS_RELU;
      p.cn = mlp_split(a) ? (int)(a->N1 / kMlpHidden) : 1;
      if (p.cn > 1) {
        char* b = reinterpret_cast<char*>(workspace);
        p.ws_count = reinterpret_cast<unsigned*>(b);
        p.ws_part = reinterpret_cast<float*>(b + kMlpCounterBytes);
      }
      return hip_status(launch_b2b_mlp(p, st), "B2B MLP launch");
    }
    return hip_status(ffn ? launch_b2b_ffn(p, st) : launch_b2b_attention(p, st), "B2B launch");
  } catch (...) {
    return fail(CF_ERR_HIP, "internal error");
  }
}

}  // extern "C"
