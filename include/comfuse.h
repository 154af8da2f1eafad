/*
 * libcomfuse — fused GEMM + row-subgraph operators for AMD Instinct MI355X
 * (gfx950), after "ComFuse: Fusing Complex Memory-Intensive Subgraphs with
 * Compute-Intensive Kernels" (arXiv 2608.03537).
 *
 * A GEMM keeps its output tile on chip while a dependent elementwise /
 * reduction subgraph consumes it (the paper's joint compute-memory operator
 * fusion, Sec. I and Sec. III); two GEMMs joined by such a subgraph keep the
 * intermediate on chip as well (B2BGEMM, Sec. IV, Eq. 2).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Ownership   Every data pointer is a DEVICE pointer owned by the caller.
 *             The library never allocates or frees device memory, never
 *             synchronises, and enqueues work only on the given HIP stream
 *             (NULL = the null stream).  Host descriptors and node arrays are
 *             read during the call only.  Buffers must stay alive until the
 *             enqueued work completes.
 * Layout      Matrices are row-major with an explicit leading dimension (in
 *             elements).  A weight that plays the mathematical role W (K x N)
 *             may be stored K x N (CF_LAYOUT_KN) or N x K (CF_LAYOUT_NK, the
 *             torch.nn.Linear layout; the fast path).  Per-column vectors
 *             (bias, gamma, beta) are fp32.
 * Errors      All validation happens before the first launch; on failure
 *             nothing is enqueued and a non-zero cf_status is returned, with a
 *             detail string from cf_last_error().  A launch failure returns
 *             CF_ERR_HIP.  Faults inside a kernel surface at the caller's next
 *             synchronisation.  No C++ exception crosses this interface.
 * Domain      Shapes or node lists outside the compiled vocabulary return
 *             CF_ERR_UNSUPPORTED (never a silent slow path), mirroring the
 *             restricted domain of the paper's frontend (Sec. V, frontend
 *             mapping).  M = 0 (or batch = 0) is a no-op returning CF_OK.
 * Alignment   Base pointers of matrices must be 16-byte aligned and leading
 *             dimensions multiples of 16 bytes (CF_ERR_ALIGN otherwise);
 *             a row pitch of 2^23 bytes or more returns CF_ERR_LD.
 * Aliasing    An output equal to an input pointer returns CF_ERR_ALIAS;
 *             partial overlap is undefined.
 * Determinism Results are bitwise reproducible run to run: no floating-point
 *             atomics, fixed merge orders.
 * Threads     The library is stateless apart from an immutable device-info
 *             cache filled once; calls from several host threads are safe.
 *             Two calls that share one workspace must not overlap in time.
 */
#ifndef COMFUSE_H
#define COMFUSE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CF_VERSION 1
#define CF_WS_HEADER_BYTES 8916992  /* 4096 + 2 stages * 2 parities * 64 slots * 17 records * 128 rows * 16 */
#define CF_B2B_WS_HEADER_BYTES 1048576  /* split-MLP arrival counters: 262144 words of 4 bytes */

typedef enum {
  CF_F32 = 0,       /* IEEE binary32 */
  CF_BF16 = 1,      /* bfloat16 */
  CF_FP8_E4M3 = 2   /* OCP E4M3FN: bias 7, max 448, no infinities */
} cf_dtype;

typedef enum {
  CF_LAYOUT_KN = 0, /* weight stored K x N row-major (ld >= N) */
  CF_LAYOUT_NK = 1  /* weight stored N x K row-major (ld >= K) */
} cf_layout;

typedef enum {
  CF_OK = 0,
  CF_ERR_NULL = 1,        /* a required pointer is NULL */
  CF_ERR_SHAPE = 2,       /* a size is negative or violates the shape rules */
  CF_ERR_LD = 3,          /* a leading dimension is smaller than the row */
  CF_ERR_ALIGN = 4,       /* pointer or leading dimension misaligned */
  CF_ERR_DTYPE = 5,       /* unsupported dtype combination */
  CF_ERR_WORKSPACE = 6,   /* workspace missing or smaller than required */
  CF_ERR_UNSUPPORTED = 7, /* outside the compiled vocabulary */
  CF_ERR_ALIAS = 8,       /* an output aliases an input */
  CF_ERR_HIP = 9,         /* the HIP runtime reported an error */
  CF_ERR_STRUCT = 10,     /* struct_size does not match this library */
  CF_ERR_PEER_TIMEOUT = 11 /* cf_workspace_check: a row-cluster wait gave up */
} cf_status;

/* ------------------------------------------------------------------------
 * cf_gemm_postnorm — post-norm GEMM epilogue (Sec. III; the MatMul +
 * LayerNorm illustration and the bypass example x = alpha*Acc + Bias of
 * Sec. III-B):
 *
 *     x = alpha * (X . W) + bias + R
 *     Y = (x - mean_row(x)) / sqrt(var_row(x) + eps) * gamma + beta
 *
 * mean/var over each row of N, biased variance.  X is M x K (in_dtype), W
 * plays K x N (in_dtype, layout w_layout), R is M x N (in_dtype) or NULL,
 * bias/gamma/beta are fp32 [N] or NULL (= 0 / 1 / 0), Y is M x N (out_dtype).
 * dtypes: in {F32, BF16} with out == in, or in = BF16 with out = F32.
 * Shape rules: N % 32 == 0, K % 16 == 0, 32 <= N <= 8192.
 * Workspace: cf_gemm_postnorm_workspace() bytes (0 on the whole-row path),
 * 16-byte aligned.  Every non-empty workspace begins with CF_WS_HEADER_BYTES
 * of library state (an error word, the round counters and the exchange
 * records of the row-cluster path): zero-fill that header once before first
 * use and do not modify it afterwards; every call leaves it valid for any
 * later call, whatever its shape or path.  A non-zero first 32-bit word means
 * a wait for peer workgroups exceeded its bound: results written through the
 * workspace since it was last cleared are invalid.  cf_workspace_check reads
 * and clears it.
 * ------------------------------------------------------------------------ */
typedef struct {
  size_t struct_size;            /* = sizeof(cf_postnorm_args) */
  int64_t M, N, K;
  cf_dtype in_dtype, out_dtype;
  const void* X; int64_t ldx;
  const void* W; int64_t ldw; cf_layout w_layout;
  const float* bias;
  const void* R; int64_t ldr;
  const float* gamma;
  const float* beta;
  float alpha, eps;
  void* Y; int64_t ldy;
  int path;                      /* 0 = auto, 1 = whole-row, 2 = row cluster
                                    (on-chip statistics exchange), 3 = split-N
                                    through the workspace */
} cf_postnorm_args;

size_t    cf_gemm_postnorm_workspace(const cf_postnorm_args* a);
cf_status cf_gemm_postnorm(const cf_postnorm_args* a, void* workspace,
                           size_t ws_bytes, void* hip_stream);

/* ------------------------------------------------------------------------
 * cf_gemm_subgraph — GEMM followed by an elementwise/reduction node list
 * executed on the on-chip tile (the Stage-Stream execution model, Sec. III;
 * reductions are stage boundaries, Sec. III-B).  The list is read in order
 * and must match this grammar (anything else is CF_ERR_UNSUPPORTED):
 *
 *     [SCALE] [BIAS] [RESIDUAL] [LAYERNORM | RMSNORM]
 *     [GELU | GELU_TANH | RELU | SOFTCAP] [SOFTMAX] STORE [ROWAMAX_QUANT]
 *
 * (a NORM and SOFTMAX do not appear in one list).
 *
 * SCALE       x *= f0                    (alpha)
 * BIAS        x += v0[n]                 (fp32 [N])
 * RESIDUAL    x += in[m, n]   (dtype: the GEMM input dtype here; F32 or
 *             BF16 in cf_rowop; ld)
 * LAYERNORM   x = (x-mean)/sqrt(var+f0) * v0 + v1   (v0/v1 may be NULL)
 * RMSNORM     x = x/sqrt(mean(x^2)+f0) * v0         (v0 may be NULL)
 * GELU        x = x * Phi(x) (erf form); GELU_TANH the tanh approximation
 * SOFTCAP     x = f0 * tanh(x / f0)       (f0 = cap > 0, finite)
 * SOFTMAX     x = exp(x - max_row(x)) / sum_row(exp(x - max_row(x)))
 *             (a scale goes in SCALE; f0 is unused here.  A list holding
 *             only SOFTMAX is cf_rowop's standalone form below.)
 * STORE       out[m, n] = x  (dtype: F32 or BF16; ld)
 * ROWAMAX_QUANT  s[m] = max_n |x| / f0 (f0 = qmax, 448 for E4M3) into out
 *             (fp32 [M]); out2[m, n] = e4m3(x / s[m]) (ld, may be NULL).
 *             A row with amax 0 gets s = 0 and zero codes.  The amax is
 *             taken over the fp32 value before the STORE rounding.
 * ------------------------------------------------------------------------ */
typedef enum {
  CF_N_SCALE = 0, CF_N_BIAS = 1, CF_N_RESIDUAL = 2, CF_N_LAYERNORM = 3,
  CF_N_RMSNORM = 4, CF_N_GELU = 5, CF_N_GELU_TANH = 6, CF_N_RELU = 7,
  CF_N_STORE = 8, CF_N_ROWAMAX_QUANT = 9, CF_N_SOFTMAX = 10, CF_N_SOFTCAP = 11
} cf_node_kind;

typedef struct {
  cf_node_kind kind;
  const void* in;     /* RESIDUAL: matrix */
  void* out;          /* STORE: matrix; ROWAMAX_QUANT: s (fp32 [M]) */
  void* out2;         /* ROWAMAX_QUANT: codes (uint8 M x N) or NULL */
  int64_t ld;         /* leading dimension of in / out (STORE) / out2 */
  cf_dtype dtype;     /* STORE output dtype */
  const float* v0;    /* BIAS: bias; LAYERNORM/RMSNORM: gamma */
  const float* v1;    /* LAYERNORM: beta */
  float f0;           /* SCALE: alpha; *NORM: eps; ROWAMAX_QUANT: qmax; SOFTCAP: cap */
} cf_node;

typedef struct {
  size_t struct_size;            /* = sizeof(cf_subgraph_args) */
  int64_t M, N, K;
  cf_dtype in_dtype;
  const void* X; int64_t ldx;
  const void* W; int64_t ldw; cf_layout w_layout;
  const cf_node* nodes; int n_nodes;
  int path;                      /* as cf_postnorm_args.path */
} cf_subgraph_args;

size_t    cf_gemm_subgraph_workspace(const cf_subgraph_args* a);
cf_status cf_gemm_subgraph(const cf_subgraph_args* a, void* workspace,
                           size_t ws_bytes, void* hip_stream);

/* ------------------------------------------------------------------------
 * cf_gemm_subgraph_noalloc — cf_gemm_subgraph for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): same arguments, same results, no
 * workspace argument, and no allocation of any kind.
 *
 * The split-N path's scratch (per-tile partial statistics and the fp32
 * pre-norm rows) lives in a 32 MiB device array inside the library, one per
 * GPU, held until the process ends; a shape whose split path needs more
 * (about M * N * 4 bytes) returns CF_ERR_WORKSPACE.  The row-cluster path is
 * not used (it keeps state between calls): path 0 (auto) takes whole rows for
 * N <= 768 and split-N above; path 2 returns CF_ERR_UNSUPPORTED.
 * Every call on one GPU shares that GPU's array: calls that overlap in time
 * on one GPU (several streams or threads) race and must be serialised by the
 * caller.  Validation happens first, as for cf_gemm_subgraph.
 * ------------------------------------------------------------------------ */
cf_status cf_gemm_subgraph_noalloc(const cf_subgraph_args* a, void* hip_stream);

/* ------------------------------------------------------------------------
 * cf_b2bgemm — back-to-back GEMM with the intermediate kept on chip
 * (Sec. IV, Eq. 2: P = X W1, S = F(P), O = S W2), batched over `batch`
 * independent problems (strides sx, sw1, ... in elements).
 *
 *   mid = CF_MID_GELU_BIAS : S = GELU(P + b1)                       (FFN)
 *   mid = CF_MID_RELU_BIAS : S = ReLU(P + b1)        (MLP, the DLRM bottom
 *                            MLP of Table 2)
 *   mid = CF_MID_SOFTMAX   : S = softmax_row(mid_scale * P), computed
 *                            online over blocks of N1 (running row max and
 *                            sum in fp32), so O = S W2 is exact softmax   (attention);
 *                            mid_scale must be finite and > 0 (CF_ERR_SHAPE)
 *   out = CF_OUT_STORE     : Y = O (+ b2 if given)
 *   out = CF_OUT_BIAS_RESIDUAL_LN : Y = LN(O + b2 + R) * gamma + beta
 *   out = CF_OUT_BIAS_RELU : Y = ReLU(O + b2)                     (MLP only)
 *
 * FFN: W1 is given as W1^T (N1 x K, CF_LAYOUT_NK), W2 as W2^T (N2 x N1,
 * CF_LAYOUT_NK); the model width d = K = N2 (CF_ERR_UNSUPPORTED otherwise);
 * (N1, d) in {(512, 256), (256, 256), (256, 128), (128, 64)}; b1 [N1] fp32
 * or NULL; R (M x d) or NULL; the FFN block Y = LN(GELU(X W1 + b1) W2 + b2
 * + X) passes R = X.
 * Attention: batch = B*H, M = Lq, K = N2 = d in {64, 128}, N1 = Lk >= 1,
 * W1 = keys stored Lk x d (CF_LAYOUT_NK, i.e. Q.K^T), W2 = values stored
 * Lk x d (CF_LAYOUT_KN); out = CF_OUT_STORE, b1 = b2 = R = NULL.
 * All matrices bf16 (dtype = CF_BF16), 16-byte aligned, leading dimensions
 * and batch strides multiples of 8 elements.  Output O is M x N2 bf16.
 * MLP: W1 given as W1^T (N1 x K, CF_LAYOUT_NK), W2 as W2^T (N2 x N1,
 * CF_LAYOUT_NK); N2 = 128, N1 a multiple of 256, K a multiple of 64 and
 * >= 128; b1 [N1] / b2 [N2] fp32 or NULL; out = CF_OUT_STORE or
 * CF_OUT_BIAS_RELU; R, gamma, beta NULL.  N1 is cut into chunks of 256
 * hidden units and the partial second products of the chunks are summed in
 * chunk order (the partial-sum identity of Sec. IV-A).  When
 * batch * ceil(M / 128) * N1 / 256 <= 256 (and N1 > 256), the chunks are
 * split over workgroups, one per chunk and 128-row block (the cross-CTA
 * dataflow of Sec. IV-A), and the last workgroup of a row block to finish
 * sums their partials at commit.  Otherwise one workgroup per row block runs
 * all chunks and keeps the sum in registers.
 * Workspace: 0 bytes for the FFN, attention, and the MLP unless it splits
 * the chunks; then cf_b2bgemm_workspace() bytes, 16-byte aligned:
 * CF_B2B_WS_HEADER_BYTES of arrival counters (one 32-bit word per batch
 * entry and 128-row block), then the fp32 partial products.  Zero-fill the
 * header once before the first MLP call; every call leaves it all zero
 * again and the partials never reach into it, so later calls of any shape
 * find it valid.  Do not share the workspace with calls of another kind,
 * and do not let calls that share it overlap in time.
 * ------------------------------------------------------------------------ */
typedef enum { CF_MID_GELU_BIAS = 0, CF_MID_SOFTMAX = 1, CF_MID_RELU_BIAS = 2 } cf_mid_op;
typedef enum { CF_OUT_STORE = 0, CF_OUT_BIAS_RESIDUAL_LN = 1, CF_OUT_BIAS_RELU = 2 } cf_out_op;

typedef struct {
  size_t struct_size;            /* = sizeof(cf_b2b_args) */
  int64_t batch, M, K, N1, N2;
  cf_dtype dtype;
  const void* X;  int64_t ldx, sx;
  const void* W1; int64_t ldw1, sw1; cf_layout w1_layout; const float* b1;
  cf_mid_op mid; float mid_scale;
  const void* W2; int64_t ldw2, sw2; cf_layout w2_layout;
  cf_out_op out; const float* b2;
  const void* R; int64_t ldr, sr;
  const float* gamma; const float* beta; float eps;
  void* O; int64_t ldo, so;
} cf_b2b_args;

size_t    cf_b2bgemm_workspace(const cf_b2b_args* a);
cf_status cf_b2bgemm(const cf_b2b_args* a, void* workspace, size_t ws_bytes,
                     void* hip_stream);

/* ------------------------------------------------------------------------
 * Unfused comparator (the materialising baseline the paper's introduction
 * describes): a plain GEMM whose result goes to global memory, then a
 * row-operator kernel that reloads it.
 *
 * cf_gemm:  C[b] = alpha * A[b] . B[b] (+ bias), A M x K, B K x N (layout),
 *           C M x N in out dtype (F32 or BF16).  in: F32 or BF16.
 *           Shape rules: N % 32 == 0, K % 16 == 0.
 * cf_rowop: runs a node list (same grammar as cf_gemm_subgraph, or a single
 *           SOFTMAX node, f0 = scale, writing out) over each row of the
 *           materialised P: batch matrices of M x N (dtype in, leading
 *           dimension ldp), matrix b at P + b * sp elements (sp a multiple
 *           of 16 bytes; ignored when batch <= 1).  The node list's matrices
 *           and s hold the batch * M rows one after another (row b * M + m),
 *           with their own leading dimensions.
 * ------------------------------------------------------------------------ */
cf_status cf_gemm(int64_t batch, int64_t M, int64_t N, int64_t K,
                  cf_dtype in, cf_dtype out,
                  const void* A, int64_t lda, int64_t sa,
                  const void* B, int64_t ldb, int64_t sb, cf_layout b_layout,
                  const float* bias, float alpha,
                  void* C, int64_t ldc, int64_t sc, void* hip_stream);

cf_status cf_rowop(int64_t batch, int64_t M, int64_t N, cf_dtype in,
                   const void* P, int64_t ldp, int64_t sp,
                   const cf_node* nodes, int n_nodes, void* hip_stream);

/* ------------------------------------------------------------------------
 * cf_workspace_check — reads and clears the error word of a workspace used by
 * cf_gemm_postnorm / cf_gemm_subgraph.  The row-cluster path (the paper's
 * inter-CTA reduction, Sec. III-A) waits for its co-resident peers with a
 * bounded spin; if a wait gives up (peers not resident, for example because
 * other work holds the compute units), the kernel sets that word, every later
 * wait gives up at once, and the outputs are invalid.  This call
 * SYNCHRONISES hip_stream, then returns CF_ERR_PEER_TIMEOUT (and clears the
 * word) if it was set since the last check, else CF_OK.  workspace may be
 * NULL (CF_OK).  Not callable during stream capture.
 * ------------------------------------------------------------------------ */
cf_status cf_workspace_check(void* workspace, size_t ws_bytes, void* hip_stream);

/* ------------------------------------------------------------------------
 * Diagnostics
 * ------------------------------------------------------------------------ */
const char* cf_status_string(cf_status s);
const char* cf_last_error(void);   /* thread-local detail of the last error */
int         cf_version(void);

#ifdef __cplusplus
}
#endif
#endif /* COMFUSE_H */
