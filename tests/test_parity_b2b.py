"""GPU parity of cf_b2bgemm (back-to-back GEMM with the intermediate in
registers) against the fp64 oracle.

FFN:  Y = LN(GELU(X W1 + b1) W2 + b2 + X), bf16, max-abs 2e-2 and rel-RMS
5e-3 (the on-chip intermediate S is rounded to bf16 as the second product's
operand; the oracle keeps it exact).  Full size M=65536, d=256, N1=512 is
compared over every element.
Attention: O = softmax(Q K^T / sqrt(d)) V per head, online softmax; rel-RMS
5e-3 is the binding check (|O| is small, so max-abs 2e-2 is loose), plus the
invariants V = 1 -> O = 1 and Q = 0 -> O = mean_j V_j.
"""
import numpy as np
import pytest

from oracle import comfuse_oracle as O
from paper_2608_03537_amd import inputs as I
from tests.helpers import assert_close_bf16, dev, host, max_abs, rel_rms

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2608_03537_amd import comfuse as cf  # noqa: E402


def run_ffn(inp, layernorm=True, residual=True):
    X = dev(inp.X)
    W1t = dev(I.lay_out_weight(inp.W1, "nk"))
    W2t = dev(I.lay_out_weight(inp.W2, "nk"))
    Y = cf.b2b_ffn(X, W1t, dev(inp.b1, "f32"), W2t, dev(inp.b2, "f32"), X if residual else None,
                   eps=inp.eps, layernorm=layernorm)
    torch.cuda.synchronize()
    return host(Y)


@pytest.mark.parametrize("M,d,N1", [(300, 64, 128), (129, 128, 256), (257, 256, 256), (200, 256, 512)])
def test_ffn_small(M, d, N1):
    inp = I.ffn_inputs(seed=2, M=M, d=d, N1=N1)
    ref = O.ffn_b2b(inp.X, inp.W1, inp.b1, inp.W2, inp.b2, eps=inp.eps)
    assert_close_bf16(run_ffn(inp), ref, f"FFN {M}x{d}x{N1}")


def test_ffn_without_layernorm():
    inp = I.ffn_inputs(seed=3, M=160, d=128, N1=256)
    got = run_ffn(inp, layernorm=False, residual=False)
    S = O.gelu_erf(O.bias_residual(O.matmul(inp.X, inp.W1), inp.b1))
    ref = O.bias_residual(O.matmul(S, inp.W2), inp.b2)
    assert rel_rms(got, ref) < 5e-3 and max_abs(got, ref) < 2e-2


@pytest.mark.parametrize("M,d,N1", [(190, 128, 256), (257, 256, 512)])
def test_ffn_other_residual_gamma_beta(M, d, N1):
    """Residual R != X (read from memory) and a LayerNorm with gamma/beta."""
    inp = I.ffn_inputs(seed=5, M=M, d=d, N1=N1)
    rng = np.random.default_rng(7)
    R = I.round_to_bf16(rng.standard_normal((M, d)).astype(np.float32))
    gamma = (1.0 + 0.1 * rng.standard_normal(d)).astype(np.float32)
    beta = (0.1 * rng.standard_normal(d)).astype(np.float32)
    X = dev(inp.X)
    Y = cf.b2b_ffn(X, dev(I.lay_out_weight(inp.W1, "nk")), dev(inp.b1, "f32"), dev(I.lay_out_weight(inp.W2, "nk")),
                   dev(inp.b2, "f32"), dev(R), dev(gamma, "f32"), dev(beta, "f32"), eps=inp.eps)
    torch.cuda.synchronize()
    S = O.gelu_erf(O.bias_residual(O.matmul(inp.X, inp.W1), inp.b1))
    ref = O.layernorm(O.bias_residual(O.matmul(S, inp.W2), inp.b2, R), gamma, beta, inp.eps)
    assert_close_bf16(host(Y), ref, f"FFN R != X {M}x{d}x{N1}")


def test_ffn_zero_second_weight_is_layernorm_of_input():
    inp = I.ffn_inputs(seed=4, M=256, d=256, N1=512)
    inp.W2[:] = 0.0
    inp.b2[:] = 0.0
    got = run_ffn(inp)
    assert_close_bf16(got, O.layernorm(inp.X), "W2 = 0")


def test_ffn_full_size():
    inp = I.ffn_inputs()
    ref = O.ffn_b2b(inp.X, inp.W1, inp.b1, inp.W2, inp.b2, eps=inp.eps)
    assert_close_bf16(run_ffn(inp), ref, "FFN 65536x256x512")


@pytest.mark.parametrize("residual", ["x", "other"])
def test_ffn_batched(residual):
    """batch = 3 entries of 257 rows, d = 256, N1 = 512: X, R, O [3, M, d];
    W1 shared (2-D), W2 per entry (3-D); b1, b2, gamma, beta shared.  R = X
    takes the kernel's residual-from-the-X-tile path, another R the load."""
    Bn, M, d, N1 = 3, 257, 256, 512
    ins = [I.ffn_inputs(seed=30 + b, M=M, d=d, N1=N1) for b in range(Bn)]
    X = dev(np.stack([t.X for t in ins]))
    Rh = np.stack([t.X for t in ins]) if residual == "x" else \
        I.round_to_bf16(np.random.default_rng(9).standard_normal((Bn, M, d)).astype(np.float32))
    R = X if residual == "x" else dev(Rh)
    W1t = dev(I.lay_out_weight(ins[0].W1, "nk"))
    W2t = dev(np.stack([I.lay_out_weight(t.W2, "nk") for t in ins]))
    Y = cf.b2b_ffn(X, W1t, dev(ins[0].b1, "f32"), W2t, dev(ins[0].b2, "f32"), R, eps=ins[0].eps)
    torch.cuda.synchronize()
    got = host(Y)
    for b in range(Bn):
        S = O.gelu_erf(O.bias_residual(O.matmul(ins[b].X, ins[0].W1), ins[0].b1))
        ref = O.layernorm(O.bias_residual(O.matmul(S, ins[b].W2), ins[0].b2, Rh[b]), eps=ins[0].eps)
        assert_close_bf16(got[b], ref, f"FFN batch entry {b} residual={residual}")


def run_attn(Q, K, V, scale=None):
    o = cf.b2b_attention(dev(Q), dev(K), dev(V), scale)
    torch.cuda.synchronize()
    return host(o)


# Ragged Lk puts the partial last key block in either ring stage: with an odd
# block count (300, 289 keys) it is loaded from stage 1's step, with an even
# one (333, 350) from stage 0's, for both head dimensions.
@pytest.mark.parametrize("B,H,Lq,Lk,d", [(1, 2, 200, 300, 64), (2, 1, 129, 64, 128), (1, 3, 64, 1, 128),
                                         (1, 1, 256, 333, 128), (1, 2, 130, 289, 128), (1, 1, 100, 350, 64)])
def test_attention_small(B, H, Lq, Lk, d):
    a = I.attention_inputs(seed=5, B=B, H=H, Lq=Lq, Lk=Lk, d=d)
    got = run_attn(a.Q, a.K, a.V)
    ref = O.attention(a.Q, a.K, a.V)
    assert rel_rms(got, ref) < 5e-3, rel_rms(got, ref)
    assert max_abs(got, ref) < 2e-2


@pytest.mark.parametrize("which", ["self", "target"])
def test_attention_table2_shapes(which):
    """Table 2 shapes (one batch, two heads), every element against the oracle:
    Self-Attention (512 x 512, d 128) and Target-Attention (4096 target rows,
    256 source rows, d 128)."""
    a = I.self_attention_table2(seed=3, B=1, H=2) if which == "self" else I.target_attention_table2(seed=3, B=1, H=2)
    got = run_attn(a.Q, a.K, a.V)
    ref = O.attention(a.Q, a.K, a.V)
    assert rel_rms(got, ref) < 5e-3 and max_abs(got, ref) < 2e-2, (rel_rms(got, ref), max_abs(got, ref))


def test_attention_invariants():
    a = I.attention_inputs(seed=6, B=1, H=2, Lq=128, Lk=200, d=128)
    # V = 1: the row sums l and the numerator add the same bf16 P (in fp32,
    # in different orders), so O / l is within a few fp32 ulps of 1 and every
    # bf16 output is exactly 1
    ones = run_attn(a.Q, a.K, np.ones_like(a.V))
    assert np.array_equal(ones, np.ones_like(ones)), np.max(np.abs(ones - 1.0))
    zq = run_attn(np.zeros_like(a.Q), a.K, a.V)
    mean_v = a.V.astype(np.float64).mean(axis=2, keepdims=True)
    assert max_abs(zq, np.broadcast_to(mean_v, zq.shape)) < 4e-3


def test_attention_full_size_sampled_rows():
    # one query row in every 128-query block of every (batch, head), at a
    # position that moves from block to block and head to head
    a = I.attention_inputs()
    got = run_attn(a.Q, a.K, a.V)
    nblk = (a.Lq + 127) // 128
    for b in range(a.B):
        for h in range(a.H):
            off = (np.arange(nblk) * 37 + 11 * (b * a.H + h)) % 128
            rows = np.minimum(np.arange(nblk) * 128 + off, a.Lq - 1)
            ref = O.attention(a.Q[b, h][rows], a.K[b, h], a.V[b, h])
            g = got[b, h][rows]
            assert rel_rms(g, ref) < 5e-3, (b, h, rel_rms(g, ref))
            assert max_abs(g, ref) < 2e-2, (b, h, max_abs(g, ref))
