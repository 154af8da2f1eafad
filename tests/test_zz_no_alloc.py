"""The allocation-free entry point cf_gemm_subgraph_noalloc, called through
the C ABI, against the workspace-taking cf_gemm_subgraph on the same inputs
and path (same kernels: bit-identical outputs) and against the fp64 oracle.
Two calls in a row per path, the second with a smaller input, so the second
reuses the per-GPU scratch array the first one left behind."""
import numpy as np
import pytest

from oracle import comfuse_oracle as O
from paper_2608_03537_amd import inputs as I
from tests.helpers import assert_close_bf16, dev, host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2608_03537_amd import comfuse as cf  # noqa: E402


def _chain(M, K, N, seed, path_noalloc, path_ws):
    inp = I.postnorm_inputs(M, K, N, "bf16", seed=seed, with_affine=False)
    X, W = dev(inp.X), dev(I.lay_out_weight(inp.W, "nk"))
    b, R = dev(inp.bias, "f32"), dev(inp.R)
    outs = []
    for _ in range(2):
        Z = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
        s = torch.full((M,), float("nan"), dtype=torch.float32, device="cuda")
        Q = torch.zeros((M, N), dtype=torch.uint8, device="cuda")
        spec = [dict(kind=cf.CF_N_BIAS, v0=b), dict(kind=cf.CF_N_RESIDUAL, **{"in": R}, ld=N, dtype=cf.CF_BF16),
                dict(kind=cf.CF_N_LAYERNORM, f0=inp.eps), dict(kind=cf.CF_N_GELU),
                dict(kind=cf.CF_N_STORE, out=Z, ld=N, dtype=cf.CF_BF16),
                dict(kind=cf.CF_N_ROWAMAX_QUANT, out=s, out2=Q, ld=N, f0=448.0)]
        outs.append((Z, s, Q, spec))
    # the allocation-free call, straight through the C ABI
    nodes = cf.make_nodes(outs[0][3])
    a = cf.subgraph_args(X, W, nodes, path=path_noalloc)
    st = cf.cf_gemm_subgraph_noalloc(a, torch.cuda.current_stream().cuda_stream)
    assert st == 0, (cf.STATUS.get(st), cf.cf_last_error())
    # the workspace-taking entry point on the same inputs, with the plan the
    # allocation-free call takes (its auto choice never is the cluster path)
    cf.gemm_subgraph(X, W, outs[1][3], path=path_ws)
    torch.cuda.synchronize()
    return inp, outs


@pytest.mark.parametrize("path,first,second", [
    (cf.PATH_SPLIT, (1000, 128, 2048), (300, 64, 1024)),     # split: scratch reused, smaller
    (cf.PATH_AUTO, (700, 128, 1536), (129, 128, 1280)),      # auto -> split above N = 768
    (cf.PATH_AUTO, (513, 128, 768), (70, 64, 512)),          # auto -> whole rows (no scratch)
])
def test_noalloc_matches_workspace_entry_point(path, first, second):
    for i, (M, K, N) in enumerate((first, second)):
        ws_path = path if path != cf.PATH_AUTO else (cf.PATH_WHOLE_ROW if N <= 768 else cf.PATH_SPLIT)
        inp, ((Za, sa, Qa, _), (Zb, sb, Qb, _)) = _chain(M, K, N, 60 + i, path, ws_path)
        assert torch.equal(Za.view(torch.int16), Zb.view(torch.int16)), (M, N)
        assert torch.equal(sa, sb) and torch.equal(Qa, Qb), (M, N)
        z, s, q = O.ln_gelu_amax(inp.X, inp.W, inp.bias, inp.R, eps=inp.eps)
        assert_close_bf16(host(Za), z, f"no-alloc {M}x{K}x{N}")
        np.testing.assert_allclose(sa.cpu().numpy(), s, rtol=1e-3)
        assert np.mean(Qa.cpu().numpy() == q) >= 0.9999


def test_noalloc_rejects_oversize_and_cluster():
    X = torch.zeros((4096, 64), dtype=torch.bfloat16, device="cuda")
    W = torch.zeros((4096, 64), dtype=torch.bfloat16, device="cuda")
    Z = torch.empty((4096, 4096), dtype=torch.bfloat16, device="cuda")
    spec = [dict(kind=cf.CF_N_LAYERNORM, f0=1e-5), dict(kind=cf.CF_N_STORE, out=Z, ld=4096, dtype=cf.CF_BF16)]
    with pytest.raises(cf.CfError, match="WORKSPACE"):
        cf.gemm_subgraph_noalloc(X, W, spec)
    with pytest.raises(cf.CfError, match="UNSUPPORTED"):
        cf.gemm_subgraph_noalloc(X[:256], W[:1024], spec[:1] + [dict(kind=cf.CF_N_STORE, out=Z, ld=4096,
                                                                      dtype=cf.CF_BF16)], path=cf.PATH_CLUSTER)
