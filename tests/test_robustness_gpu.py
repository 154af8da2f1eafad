"""GPU tests of the failure handling and the batched row operator.

The row-cluster path waits for co-resident peer workgroups with a bounded
spin and reports a wait that gave up through a sticky error word in the
workspace.  The failure is forced from the host (the word is set before the
call), so every wait gives up at its first poll and every kernel exits
normally; the call must then be reported, and a clean call afterwards must
be correct.
"""
import numpy as np
import pytest

from oracle import comfuse_oracle as O
from paper_2608_03537_amd import inputs as I
from tests.helpers import assert_close_bf16, assert_close_f32, dev, host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2608_03537_amd import comfuse as cf  # noqa: E402


def _postnorm_operands(inp):
    X, W, R = dev(inp.X), dev(I.lay_out_weight(inp.W, "nk")), dev(inp.R)
    b, g, be = dev(inp.bias, "f32"), dev(inp.gamma, "f32"), dev(inp.beta, "f32")
    return X, W, b, R, g, be


def test_peer_wait_failure_is_reported_then_cleared():
    inp = I.postnorm_inputs(512, 128, 768, "bf16", seed=41)
    X, W, b, R, g, be = _postnorm_operands(inp)
    Y = torch.empty((inp.M, inp.N), dtype=torch.bfloat16, device="cuda")
    need = cf.cf_gemm_postnorm_workspace(cf.postnorm_args(X, W, b, R, g, be, Y, path=cf.PATH_CLUSTER))
    assert need > 0
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    ws.view(torch.int32)[0] = 1            # as if an earlier wait had given up
    cf.gemm_postnorm(X, W, b, R, g, be, eps=inp.eps, path=cf.PATH_CLUSTER, out=Y, ws=ws, check=False)
    with pytest.raises(cf.CfError, match="PEER_TIMEOUT"):
        cf.check_workspace(ws)
    assert int(ws.view(torch.int32)[0].item()) == 0   # the check cleared the word
    cf.check_workspace(ws)                             # nothing new: no error
    # a clean call through the same workspace is checked and correct
    cf.gemm_postnorm(X, W, b, R, g, be, eps=inp.eps, path=cf.PATH_CLUSTER, out=Y, ws=ws)
    torch.cuda.synchronize()
    ref = O.postnorm(inp.X, inp.W, inp.bias, inp.R, inp.gamma, inp.beta, 1.0, inp.eps)
    assert_close_bf16(host(Y), ref, "cluster after a reported failure")


def test_helper_raises_on_failure():
    inp = I.postnorm_inputs(256, 128, 512, "bf16", seed=42, with_affine=False)
    X, W, b, R, _, _ = _postnorm_operands(inp)
    Z = torch.empty((inp.M, inp.N), dtype=torch.bfloat16, device="cuda")
    spec = [dict(kind=cf.CF_N_BIAS, v0=b), dict(kind=cf.CF_N_RESIDUAL, **{"in": R}, ld=inp.N, dtype=cf.CF_BF16),
            dict(kind=cf.CF_N_LAYERNORM, f0=inp.eps), dict(kind=cf.CF_N_STORE, out=Z, ld=inp.N, dtype=cf.CF_BF16)]
    need = cf.cf_gemm_subgraph_workspace(cf.subgraph_args(X, W, cf.make_nodes(spec), path=cf.PATH_CLUSTER))
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    ws.view(torch.int32)[0] = 1
    with pytest.raises(cf.CfError, match="PEER_TIMEOUT"):
        cf.gemm_subgraph(X, W, spec, path=cf.PATH_CLUSTER, ws=ws)   # check=True by default
    cf.gemm_subgraph(X, W, spec, path=cf.PATH_CLUSTER, ws=ws)
    torch.cuda.synchronize()
    ref = O.layernorm(O.bias_residual(O.matmul(inp.X, inp.W), inp.bias, inp.R), eps=inp.eps)
    assert_close_bf16(host(Z), ref, "subgraph after a reported failure")


def test_workspace_cache_is_per_stream():
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    a = cf.workspace(4096, "cuda", s1)
    b = cf.workspace(4096, "cuda", s2)
    assert a.data_ptr() != b.data_ptr()
    assert cf.workspace(4096, "cuda", s1).data_ptr() == a.data_ptr()


def test_rowop_batched_strided():
    # three 100 x 256 matrices inside a [3, 120, 256] buffer (batch stride
    # 120 rows): bias, LayerNorm, store of the 300 rows one after another
    rng = np.random.default_rng(43)
    full = rng.standard_normal((3, 120, 256)).astype(np.float32) * 2 + 0.5
    P = dev(full, "f32")[:, :100]
    b = rng.standard_normal(256).astype(np.float32) * 0.1
    Y = torch.empty((300, 256), dtype=torch.float32, device="cuda")
    cf.rowop(P, [dict(kind=cf.CF_N_BIAS, v0=dev(b, "f32")), dict(kind=cf.CF_N_LAYERNORM, f0=1e-5),
                 dict(kind=cf.CF_N_STORE, out=Y, ld=256, dtype=cf.CF_F32)])
    torch.cuda.synchronize()
    rows = full[:, :100].reshape(300, 256).astype(np.float64)
    assert_close_f32(host(Y), O.layernorm(O.bias_residual(rows, b), eps=1e-5), "batched rowop")


def test_rowop_batched_softmax_matches_flat():
    rng = np.random.default_rng(44)
    S = dev(rng.standard_normal((4, 64, 512)).astype(np.float32) * 3, "f32")
    A = torch.empty((256, 512), dtype=torch.float32, device="cuda")
    B = torch.empty((256, 512), dtype=torch.float32, device="cuda")
    cf.rowop(S, [dict(kind=cf.CF_N_SOFTMAX, out=A, ld=512, dtype=cf.CF_F32, f0=0.5)])
    cf.rowop(S.reshape(256, 512), [dict(kind=cf.CF_N_SOFTMAX, out=B, ld=512, dtype=cf.CF_F32, f0=0.5)])
    torch.cuda.synchronize()
    assert torch.equal(A, B)
    assert_close_f32(host(A), O.softmax_rows(0.5 * host(S).reshape(256, 512)), "batched softmax")


def test_cluster_calls_of_different_widths_share_a_workspace():
    # Row-cluster calls with 4, 8 and 16 peers per row block and one to three
    # rounds per peer group, all through one fresh workspace: each call's
    # exchange must only ever accept its own round's records, whatever earlier
    # calls of another width left in the header.
    ws = torch.zeros(64 << 20, dtype=torch.uint8, device="cuda")
    for M, N in [(2048, 1024), (4096, 2048), (1024, 4096), (6144, 1024), (2048, 2048), (3072, 1024)]:
        inp = I.postnorm_inputs(M, 64, N, "f32", seed=45 + N // 1024, with_residual=False)
        X, W = dev(inp.X, "f32"), dev(I.lay_out_weight(inp.W, "nk"), "f32")
        b, g, be = dev(inp.bias, "f32"), dev(inp.gamma, "f32"), dev(inp.beta, "f32")
        Y = torch.empty((M, N), dtype=torch.float32, device="cuda")
        spec = [dict(kind=cf.CF_N_BIAS, v0=b), dict(kind=cf.CF_N_LAYERNORM, v0=g, v1=be, f0=1e-5),
                dict(kind=cf.CF_N_STORE, out=Y, ld=N, dtype=cf.CF_F32)]
        cf.gemm_subgraph(X, W, spec, path=cf.PATH_CLUSTER, ws=ws)
        torch.cuda.synchronize()
        ref = O.postnorm(inp.X, inp.W, inp.bias, None, inp.gamma, inp.beta, 1.0, 1e-5)
        assert_close_f32(host(Y), ref, f"cluster {M}x{N} after other widths")
