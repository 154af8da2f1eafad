"""GPU parity of the unfused comparator pieces: cf_gemm (batched, both B
layouts, fp32/bf16) and cf_rowop softmax, against the fp64 oracle."""
import numpy as np
import pytest

from oracle import comfuse_oracle as O
from paper_2608_03537_amd import inputs as I
from tests.helpers import assert_close_bf16, assert_close_f32, dev, host, rel_rms

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2608_03537_amd import comfuse as cf  # noqa: E402


def _rand(shape, seed, dtype, std=1.0):
    v = (np.random.default_rng(seed).standard_normal(shape) * std).astype(np.float32)
    return I.round_to_bf16(v) if dtype == "bf16" else v


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("layout", ["nk", "kn"])
@pytest.mark.parametrize("M,K,N", [(100, 64, 96), (257, 160, 320), (64, 32, 512)])
def test_gemm(M, K, N, layout, dtype):
    A = _rand((M, K), 1, dtype)
    Bm = _rand((K, N), 2, dtype, 1 / np.sqrt(K))
    bias = _rand((N,), 3, "f32")
    Cg = cf.gemm(dev(A, dtype), dev(I.lay_out_weight(Bm, layout), dtype),
                 b_layout=cf.CF_LAYOUT_NK if layout == "nk" else cf.CF_LAYOUT_KN,
                 bias=dev(bias, "f32"), alpha=0.5, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref = 0.5 * O.matmul(A, Bm) + bias
    got = host(Cg)
    assert_close_f32(got, ref, "gemm") if dtype == "f32" else None
    assert rel_rms(got, ref) < 1e-6


# bf16 B stored K x N with K a multiple of 64 (>= 192) takes the direct-to-LDS
# ring with transposing LDS reads: ragged M, N not a multiple of the tile
# width (clamped columns), batched operands.
@pytest.mark.parametrize("M,K,N,nb", [(300, 256, 224, 1), (129, 192, 288, 1), (64, 512, 1024, 2),
                                      (257, 256, 96, 1), (33, 2048, 128, 3)])
def test_gemm_kn_ring(M, K, N, nb):
    A = np.stack([_rand((M, K), 11 + i, "bf16") for i in range(nb)])
    Bm = np.stack([_rand((K, N), 21 + i, "bf16", 1 / np.sqrt(K)) for i in range(nb)])
    Cg = cf.gemm(dev(A), dev(Bm), b_layout=cf.CF_LAYOUT_KN, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref = np.stack([O.matmul(A[i], Bm[i]) for i in range(nb)])
    got = host(Cg)
    assert got.shape == ref.shape
    assert rel_rms(got, ref) < 1e-6
    assert np.max(np.abs(got - ref)) < 1e-4 * np.max(np.abs(ref))


def test_gemm_kn_attention_pv_full_length():
    """P.V of two heads at the attention workload's length (2048 keys, d = 128):
    the unfused comparator's second product, B stored K x N."""
    nb, L, d = 2, 2048, 128
    rng = np.random.default_rng(31)
    Pb = I.round_to_bf16((rng.random((nb, L, L)) / L * 2).astype(np.float32))
    V = np.stack([_rand((L, d), 32 + i, "bf16") for i in range(nb)])
    O2 = cf.gemm(dev(Pb), dev(V), b_layout=cf.CF_LAYOUT_KN, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref = np.stack([O.matmul(Pb[i], V[i]) for i in range(nb)])
    assert rel_rms(host(O2), ref) < 1e-6


def test_gemm_batched_attention_shapes():
    B, L, d = 3, 160, 64
    Q, K, V = (_rand((B, L, d), s, "bf16") for s in (4, 5, 6))
    S = cf.gemm(dev(Q), dev(K), b_layout=cf.CF_LAYOUT_NK, alpha=1 / 8, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref = np.stack([O.matmul(Q[i], K[i].T) / 8 for i in range(B)])
    assert rel_rms(host(S), ref) < 1e-6
    Pm = (np.random.default_rng(7).random((B, L, L)) / L).astype(np.float32)
    Pb = I.round_to_bf16(Pm)
    O2 = cf.gemm(dev(Pb), dev(V), b_layout=cf.CF_LAYOUT_KN, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref2 = np.stack([O.matmul(Pb[i], V[i]) for i in range(B)])
    assert rel_rms(host(O2), ref2) < 1e-6


def test_rowop_softmax():
    S = _rand((50, 1024), 8, "f32", 3.0)
    Y = torch.empty((50, 1024), dtype=torch.float32, device="cuda")
    cf.rowop(dev(S, "f32"), [dict(kind=cf.CF_N_SOFTMAX, out=Y, ld=1024, dtype=cf.CF_F32, f0=0.25)])
    torch.cuda.synchronize()
    got = host(Y)
    ref = O.softmax_rows(0.25 * S.astype(np.float64))
    np.testing.assert_allclose(got.sum(axis=1), 1.0, atol=1e-5)
    assert np.max(np.abs(got - ref)) < 1e-6
