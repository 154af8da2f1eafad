"""Seeded synthetic operands for the fused GEMM + row-subgraph workloads.

This module only draws random numbers and rounds them to their storage type.
It performs none of the fused method's arithmetic (no product, no
normalisation, no activation), so the HIP path and the fp64 CPU oracle can
both consume exactly the same operand values without sharing any method code.

Conventions
-----------
* Every tensor comes from its own stream:
  ``numpy.random.default_rng([seed, workload_id, tensor_id])``.  Tensors are
  drawn in a fixed order, so adding a tensor never changes the others.
* Each draw is made in fp64, scaled by the tensor's standard deviation, then
  cast to fp32.  For bf16 workloads the matrices are then rounded to the
  nearest bf16, ties to even.  The returned arrays are float32 whose values are
  exactly representable in the storage type, so an upcast to fp64 (oracle) or
  a cast to ``torch.bfloat16`` (device) is exact.
* Per-column vectors (bias, gamma, beta) are always stored fp32.
* The weight of a linear layer is drawn as the mathematical ``W`` with shape
  K x N.  ``lay_out_weight`` gives the storage order the caller asks for:
  K x N row-major ("kn") or N x K row-major ("nk", the nn.Linear layout).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

# Workload identifiers used in the seed tuple.
WL_POSTNORM_TINY = 1
WL_BERT_POSTNORM = 2
WL_LN_GELU_AMAX = 3
WL_FFN_B2B = 4
WL_ATTENTION = 5
WL_MSTS = 6
WL_SELF_ATTN_T2 = 7
WL_TARGET_ATTN_T2 = 8
WL_DLRM_MLP = 9
WL_CUSTOM = 99


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even), returned as fp32.

    bf16 keeps the upper 16 bits of the fp32 pattern.  Adding 0x7FFF plus the
    lowest kept bit and truncating implements round-to-nearest-even.  Inputs
    here are finite Gaussian draws, so NaN/Inf handling is not needed.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    rounded = ((bits + 0x7FFF + lsb) >> 16) << 16
    return rounded.astype(np.uint32).view(np.float32)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Upper 16 bits of bf16-exact fp32 values, as uint16."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)


def _normal(seed, wl, tid, shape, std, dtype):
    rng = np.random.default_rng([seed, wl, tid])
    v = (rng.standard_normal(shape) * std).astype(np.float32)
    return round_to_bf16(v) if dtype == "bf16" else v


def _uniform(seed, wl, tid, shape, lo, hi):
    rng = np.random.default_rng([seed, wl, tid])
    return rng.uniform(lo, hi, shape).astype(np.float32)


def lay_out_weight(w_kn: np.ndarray, layout: str) -> np.ndarray:
    """Storage order of a K x N weight: 'kn' (as drawn) or 'nk' (transposed)."""
    if layout == "kn":
        return np.ascontiguousarray(w_kn)
    if layout == "nk":
        return np.ascontiguousarray(w_kn.T)
    raise ValueError(f"unknown weight layout {layout!r}")


@dataclass
class PostnormInputs:
    """Operands of Y = LN(alpha * X.W + bias + R) * gamma + beta."""
    M: int
    K: int
    N: int
    dtype: str                 # "f32" or "bf16" (matrices); vectors are fp32
    X: np.ndarray              # M x K
    W: np.ndarray              # K x N (mathematical orientation)
    bias: np.ndarray | None    # N
    R: np.ndarray | None       # M x N
    gamma: np.ndarray | None   # N
    beta: np.ndarray | None    # N
    alpha: float = 1.0
    eps: float = 1e-5
    meta: dict = field(default_factory=dict)


def postnorm_inputs(M, K, N, dtype="bf16", seed=0, workload=WL_CUSTOM, *,
                    x_std=1.0, r_std=1.0, w_std=None, bias_std=0.02,
                    gamma="normal", gamma_std=0.02, beta_std=0.02,
                    with_bias=True, with_residual=True, with_affine=True,
                    eps=1e-5, alpha=1.0) -> PostnormInputs:
    """Draw the operands of a GEMM + bias + residual + LayerNorm problem.

    ``w_std`` defaults to 1/sqrt(K), i.e. variance 1/K, which keeps X.W at
    unit variance.  ``gamma`` is "normal" (1 + N(0, gamma_std^2)),
    "uniform" (U(0.5, 1.5)) or "ones".
    """
    if w_std is None:
        w_std = 1.0 / np.sqrt(K)
    X = _normal(seed, workload, 0, (M, K), x_std, dtype)
    W = _normal(seed, workload, 1, (K, N), w_std, dtype)
    bias = _normal(seed, workload, 2, (N,), bias_std, "f32") if with_bias else None
    R = _normal(seed, workload, 3, (M, N), r_std, dtype) if with_residual else None
    gam = bet = None
    if with_affine:
        if gamma == "normal":
            gam = (1.0 + _normal(seed, workload, 4, (N,), gamma_std, "f32")).astype(np.float32)
        elif gamma == "uniform":
            gam = _uniform(seed, workload, 4, (N,), 0.5, 1.5)
        elif gamma == "ones":
            gam = None
        else:
            raise ValueError(gamma)
        bet = _normal(seed, workload, 5, (N,), beta_std, "f32") if beta_std else None
    return PostnormInputs(M, K, N, dtype, X, W, bias, R, gam, bet, alpha, eps)


def postnorm_tiny_fp32(seed=0) -> PostnormInputs:
    """fp32 post-norm, M=128, K=N=256: X, R, b ~ N(0,1); W ~ N(0,1)/16;
    gamma ~ U(0.5,1.5); beta ~ N(0, 0.1^2); eps 1e-5."""
    return postnorm_inputs(128, 256, 256, "f32", seed, WL_POSTNORM_TINY,
                           w_std=1.0 / 16.0, bias_std=1.0, gamma="uniform",
                           beta_std=0.1)


def bert_base_postnorm(seed=0, M=8192) -> PostnormInputs:
    """BERT-base attention-output post-norm, bf16: M=8192 (16 x 512 tokens),
    K=N=768; X, R ~ N(0,1); W ~ N(0, 1/768); b ~ N(0, 0.02^2);
    gamma = 1 + N(0, 0.02^2); beta ~ N(0, 0.02^2); eps 1e-5."""
    return postnorm_inputs(M, 768, 768, "bf16", seed, WL_BERT_POSTNORM)


def ln_gelu_amax_inputs(seed=0, M=16384, K=4096, N=4096) -> PostnormInputs:
    """LN -> GELU -> row-amax -> e4m3 chain, bf16: X, R ~ N(0,1);
    W ~ N(0, 1/K); b ~ N(0, 0.02^2); gamma = 1, beta = 0 (not passed)."""
    return postnorm_inputs(M, K, N, "bf16", seed, WL_LN_GELU_AMAX,
                           with_affine=False)


def msts_inputs(seed=0, M=16384, K=768, N=1024, dtype="bf16", alpha=8.0, cap=10.0) -> PostnormInputs:
    """Scale -> tanh softcap -> softmax on a GEMM output: X ~ N(0,1);
    W ~ N(0, 1/K); b ~ N(0, 0.02^2); alpha = 8 spreads the logits to about
    +-30 so that the softcap (cap 10) saturates part of them."""
    inp = postnorm_inputs(M, K, N, dtype, seed, WL_MSTS, with_residual=False, with_affine=False, alpha=alpha)
    inp.meta["cap"] = cap
    return inp


@dataclass
class FFNInputs:
    """Operands of Y = LN(GELU(X.W1 + b1).W2 + b2 + X) (gamma=1, beta=0)."""
    M: int
    d: int
    N1: int
    X: np.ndarray    # M x d (also the residual)
    W1: np.ndarray   # d x N1
    b1: np.ndarray   # N1
    W2: np.ndarray   # N1 x d
    b2: np.ndarray   # d
    eps: float = 1e-5


def ffn_inputs(seed=0, M=65536, d=256, N1=512, workload=WL_FFN_B2B) -> FFNInputs:
    """FFN B2B, bf16: X ~ N(0,1); W1 ~ N(0, 1/d); W2 ~ N(0, 1/N1);
    b1, b2 ~ N(0, 0.02^2)."""
    X = _normal(seed, workload, 0, (M, d), 1.0, "bf16")
    W1 = _normal(seed, workload, 1, (d, N1), 1.0 / np.sqrt(d), "bf16")
    b1 = _normal(seed, workload, 2, (N1,), 0.02, "f32")
    W2 = _normal(seed, workload, 3, (N1, d), 1.0 / np.sqrt(N1), "bf16")
    b2 = _normal(seed, workload, 4, (d,), 0.02, "f32")
    return FFNInputs(M, d, N1, X, W1, b1, W2, b2)


@dataclass
class AttentionInputs:
    """Q, K, V of shape [B, H, L, d], bf16-exact fp32; no mask."""
    B: int
    H: int
    Lq: int
    Lk: int
    d: int
    Q: np.ndarray
    K: np.ndarray
    V: np.ndarray


def attention_inputs(seed=0, B=4, H=16, Lq=2048, Lk=2048, d=128,
                     workload=WL_ATTENTION) -> AttentionInputs:
    """Attention B2B, bf16: Q, K, V ~ N(0,1), layout [B, H, L, d]."""
    Q = _normal(seed, workload, 0, (B, H, Lq, d), 1.0, "bf16")
    K = _normal(seed, workload, 1, (B, H, Lk, d), 1.0, "bf16")
    V = _normal(seed, workload, 2, (B, H, Lk, d), 1.0, "bf16")
    return AttentionInputs(B, H, Lq, Lk, d, Q, K, V)


def self_attention_table2(seed=0, B=16, H=16) -> AttentionInputs:
    """Self-Attention of Table 2: sequence length 512, head dimension 128.
    The paper gives no batch or head count; B = H = 16 gives 1024 workgroups."""
    return attention_inputs(seed, B, H, 512, 512, 128, WL_SELF_ATTN_T2)


def target_attention_table2(seed=0, B=4, H=16, d=128) -> AttentionInputs:
    """Target-Attention of Table 2: 4096 target (query) rows against 256 source
    (key/value) rows.  The paper gives no head dimension, batch or head count;
    d = 128 as in its Self-Attention row, B = 4, H = 16 (2048 workgroups)."""
    return attention_inputs(seed, B, H, 4096, 256, d, WL_TARGET_ATTN_T2)


@dataclass
class MlpInputs:
    """Operands of O = ReLU(X.W1 + b1).W2 + b2 (optionally ReLU(O))."""
    M: int
    K: int
    N1: int
    N2: int
    X: np.ndarray    # M x K
    W1: np.ndarray   # K x N1
    b1: np.ndarray   # N1
    W2: np.ndarray   # N1 x N2
    b2: np.ndarray   # N2


def dlrm_mlp_inputs(seed=0, M=65536, K=1024, N1=512, N2=128, workload=WL_DLRM_MLP) -> MlpInputs:
    """The DLRM bottom-MLP shape of Table 2 (1024 -> 512 -> 128), bf16: X ~ N(0,1);
    W1 ~ N(0, 1/K); W2 ~ N(0, 1/N1); b1, b2 ~ N(0, 0.02^2).  Table 2 gives no
    batch; 65536 rows are used (the FFN workload's row count)."""
    X = _normal(seed, workload, 0, (M, K), 1.0, "bf16")
    W1 = _normal(seed, workload, 1, (K, N1), 1.0 / np.sqrt(K), "bf16")
    b1 = _normal(seed, workload, 2, (N1,), 0.02, "f32")
    W2 = _normal(seed, workload, 3, (N1, N2), 1.0 / np.sqrt(N1), "bf16")
    b2 = _normal(seed, workload, 4, (N2,), 0.02, "f32")
    return MlpInputs(M, K, N1, N2, X, W1, b1, W2, b2)
