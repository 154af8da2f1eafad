// Internal host <-> kernel interface of libcomfuse (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cf {

enum NormKind { NORM_NONE = 0, NORM_LAYER = 1, NORM_RMS = 2 };
enum ActKind { ACT_NONE = 0, ACT_GELU = 1, ACT_GELU_TANH = 2, ACT_RELU = 3, ACT_SOFTCAP = 4 };

// Epilogue "program": the stage chain of the Stage-Stream model in a fixed
// order.  Every field is uniform across the launch, so the kernel branches on
// it with scalar branches.
//   stage 1: x = alpha * acc + bias[n] + R[m, n]
//   stage 2: optional row reduction (LayerNorm / RMSNorm) and its PostOp
//   stage 3: optional activation, then optional row softmax (a reduction:
//            row max and the sum of exp(x - max))
//   store  : Y[m, n] = x (bf16 or fp32)
//   stage 4: optional row amax -> s[m] = amax / qmax, Q[m, n] = e4m3(x / s)
struct RowEpi {
  float alpha;
  const float* bias;
  const void* R; int64_t ldr; int64_t sr;   // residual
  int r_f32;                                // row kernel: residual is fp32
  int norm;
  const float* gamma; const float* beta; float eps;
  int act; float softcap;                   // ACT_SOFTCAP: cap
  int softmax;
  void* Y; int64_t ldy; int64_t sy; int y_f32;
  int quant; float qmax; float* s_out; uint8_t* q_out; int64_t ldq;
};

// Where the row statistics of one row block are finished.
enum RowMode {
  ROWS_LOCAL = 0,    // the workgroup holds whole rows (or no reduction)
  ROWS_CLUSTER = 1,  // cn co-resident workgroups exchange partials on chip
  ROWS_SPLIT = 2     // write fp32 x and partial (mean, M2) for a finish pass
};

struct GemmRowsParams {
  int batch, M, N, K;
  const void* X; int64_t ldx; int64_t sx;
  const void* W; int64_t ldw; int64_t sw; int w_nk;   // w_nk: W stored N x K
  RowEpi epi;
  int mode;            // RowMode
  int cn;              // workgroups along N per row block
  int num_rb;          // row blocks = ceil(M / TM)
  int slots;           // row-block slots per XCD processed concurrently
  // Workspace views.  Every workspace starts with a fixed header that only
  // the cluster path writes: an error word, one 64-bit round counter per
  // concurrent peer group ("slot") and the exchange records.  Counters only
  // ever grow by whole multiples of kArriveUnit and every record carries the
  // round it belongs to, so a zero-filled header stays valid across calls of
  // any shape and path without a reset.
  unsigned* ws_err;              // sticky flag: a peer wait exceeded its spin limit
  unsigned long long* ws_arrive; // [kMaxSlots] round counters
  float* ws_part;                // CLUSTER: records (kRecStageWords u64 per stage);
                                 // SPLIT: [M][cn] float2
  float* ws_x;                   // SPLIT: [M][N] fp32 pre-norm x
  int spin_limit;                // polls before a peer wait gives up (sets ws_err)
  int leader;                    // CLUSTER: leader-follower exchange (peer 0 merges and broadcasts)
};

// Each of the NW waves of the cn workgroups of a peer group adds
// kArriveUnit / (cn * NW) to the group's counter once per tile, so a round
// adds exactly kArriveUnit.  lcm(1..16) * 8 is divisible by cn * NW for every
// cn <= 16 and NW in {1, 2, 4, 8}.
constexpr unsigned long long kArriveUnit = 720720ull * 8ull;
constexpr int kMaxSlots = 64;                        // concurrent peer groups
// Exchange records: [stage 2][round parity 2][slot kMaxSlots][peer kRecPeers]
// [row kRecRows] x 2 words (peer kRecLead: the leader's merged values).  A record's position depends only on (slot,
// peer), never on the launch's peer count: round numbers grow per slot, so a
// record left by an earlier call in a position only ever carries an older
// round of the same slot (a position shared by different slots could hold
// another slot's equal round number).  The parity of the round selects one
// of two record sets: a fast peer that has finished round r and publishes
// round r + 1 writes the other set, so a slow peer still reading round r
// never finds its value overwritten.  (It cannot get two rounds ahead: round
// r + 1 completes only with every peer's round r + 1 record, written after
// that peer finished round r.)
constexpr int kRecPeers = 17, kRecRows = 128;        // peers 0..15, then the leader's broadcast
constexpr int kRecLead = 16;                         // record of the merged values (leader-follower)
constexpr int kLeaderFollowerPeers = 16;             // peer counts from which the leader merges for all
constexpr size_t kRecSetWords = (size_t)kMaxSlots * kRecPeers * kRecRows * 2;   // one parity of one stage
constexpr size_t kRecStageWords = 2 * kRecSetWords;
constexpr size_t kWsCounterBytes = 4096;             // err word, then the counters
constexpr size_t kWsHeaderBytes = kWsCounterBytes + 2 * kRecStageWords * 8;
static_assert(256 + 8 * kMaxSlots <= kWsCounterBytes, "counter area");
constexpr int kSpinLimitDefault = 1 << 20;           // ~1 s of device-scope polls
// Tile order of launches without peer groups: each XCD's tiles run in groups
// of kTileGroupRows row blocks by every column tile, column by column, so the
// about 32 tiles an XCD runs at once cover 8 row blocks x 4 column tiles and
// share their operands in its L2 (2 row blocks x 16 column tiles fetch about
// twice as many bytes per k-step at N = 4096).
constexpr int kTileGroupRows = 8;

// Wave-per-row kernel: the finish pass of the split path (merge the partial
// (mean, M2) of each row's tiles, then stages 2..4 on the fp32 x the GEMM
// wrote) and the unfused row operator (stages 1..4, or softmax, on a
// materialised matrix).
struct RowKernelParams {
  int M, N;                               // M counts the rows of every batch
  const void* P; int64_t ldp; int p_f32;  // input rows (finish: fp32 x)
  int rows_per_batch; int64_t sp;         // row r of P: (r / rows_per_batch) * sp + (r % rows_per_batch) * ldp
  int finish;                             // 1: statistics from partials
  int cn, tn;                             // finish: tiles per row, tile width
  const float* part;                      // finish: [M][cn] (mean, M2)
  int softmax; float softmax_scale;       // softmax(scale * P) instead
  RowEpi epi;
};


// Compiled GEMM kernels (instantiations of gemm_rows_kernel<S, LOOP, EPI>).
struct GemmKernel {
  int tm, tn, in_f32, loop, epi, threads;
  int stages;   // direct-to-LDS ring depth (needs K / k_per_stage >= stages - 1); 0 for other loops
  const void* fn;           // one tile per workgroup
  const void* fn_persist;   // workgroups loop over row-block slots (row-cluster path with a capped grid)
};
const GemmKernel* gemm_kernels_v2(int* n);     // direct-to-LDS pipeline
const GemmKernel* gemm_kernels_v1(int* n);     // register-staged, any layout
const GemmKernel* gemm_kernels_wr(int* n);     // whole-row tiles (register-staged)
const GemmKernel* gemm_kernels_split(int* n);  // split-N GEMM pass (both main loops)
const GemmKernel* gemm_kernels_kn(int* n);     // direct-to-LDS pipeline, bf16 W stored K x N
int find_gemm_kernel(int in_f32, int tm, int tn, int loop, int epi);   // -1 if none
const GemmKernel& gemm_kernel(int idx);
int resident_wgs(int idx);   // co-resident workgroups of this kernel on the device

// Back-to-back GEMM (Sec. IV, Eq. 2).  All matrices bf16; weights stored as
// the transposed operand (rows = output features, contiguous along the
// contraction).  Batched over blockIdx.y with element strides.
struct B2BParams {
  int batch, M, K, N1, N2;
  const uint16_t* X; int64_t ldx, sx;     // M x K
  const uint16_t* W1; int64_t ldw1, sw1;  // N1 x K (FFN W1^T; attention keys Lk x d)
  const float* b1;                         // [N1] (FFN) or NULL
  float mid_scale;                         // attention: scale of Q.K^T
  const uint16_t* W2; int64_t ldw2, sw2;  // FFN: N2 x N1 (W2^T); attention: values Lk x d
  int out_ln;                              // 1: Y = LN(O + b2 + R) * gamma + beta
  const float* b2;                         // [N2] or NULL
  const uint16_t* R; int64_t ldr, sr;     // residual M x N2 or NULL
  const float* gamma; const float* beta; float eps;
  uint16_t* O; int64_t ldo, so;           // M x N2 output (bf16)
  // MLP (S = ReLU(P + b1)): output ReLU, and the split of N1 over cn
  // workgroups whose partial second products are summed at commit
  int out_relu;
  int cn;                                  // workgroups per row block: N1 / 256 (split), or 1 (whole)
  unsigned* ws_count;                      // [batch][row blocks] arrival counters (zero between calls)
  float* ws_part;                          // [batch][cn][M][N2] fp32 partial products
};

// Launchers (return hipSuccess or the launch error).
hipError_t launch_gemm_rows(const GemmRowsParams& p, int idx, hipStream_t st);
hipError_t launch_row_kernel(const RowKernelParams& p, hipStream_t st);
hipError_t launch_b2b_ffn(const B2BParams& p, hipStream_t st);        // -> hipErrorInvalidValue if N1/N2 not compiled
hipError_t launch_b2b_attention(const B2BParams& p, hipStream_t st);  // -> hipErrorInvalidValue if d not compiled
hipError_t launch_b2b_mlp(const B2BParams& p, hipStream_t st);        // -> hipErrorInvalidValue if N2 not compiled
bool b2b_ffn_supported(int N1, int N2);
bool b2b_mlp_supported(int K, int N1, int N2);
constexpr int kMlpRows = 128, kMlpHidden = 256;   // rows and hidden units of one MLP workgroup
bool b2b_attention_supported(int d);

}  // namespace cf
