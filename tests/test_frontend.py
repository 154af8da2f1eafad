"""The Python frontend (Sec. V): capture -> Fusion Spec IR (Phi) -> node list.

CPU tests pin the lowering two ways: the node kinds and parameters each
function must produce, and the semantics — the lowered node list evaluated
with the oracle's fp64 primitives equals the original function evaluated in
fp64 by PyTorch on the same inputs.  Functions outside the domain must be
reported (never silently lowered).  The GPU test runs lowered epilogues through
cf_gemm_subgraph against the fp64 oracle.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
import torch.nn.functional as F  # noqa: E402

from oracle import comfuse_oracle as O  # noqa: E402
from paper_2608_03537_amd import comfuse as cf  # noqa: E402
from paper_2608_03537_amd import frontend as fe  # noqa: E402

M, K, N = 6, 32, 64
KIND = {v: k[5:] for k, v in vars(cf).items() if k.startswith("CF_N_")}


def _args(kinds, seed=0, dtype=torch.float64):
    g = torch.Generator().manual_seed(seed)
    shapes = {"X": (M, K), "W": (N, K), "Wk": (K, N), "b": (N,), "r": (M, N), "g": (N,), "be": (N,)}
    out = []
    for k in kinds:
        t = torch.randn(*shapes[k], generator=g, dtype=dtype)
        if k == "g":
            t = 1.0 + 0.1 * t
        out.append(t)
    return tuple(out)


def _ln_manual(X, W, r):
    x = r + X @ W.t()
    mu = x.mean(-1, keepdim=True)
    var = ((x - mu) ** 2).mean(-1, keepdim=True)
    return (x - mu) / torch.sqrt(var + 1e-6)


def _rms_manual(X, W, g):
    x = X @ W.t()
    return x * torch.rsqrt(x.pow(2).mean(-1, keepdim=True) + 1e-6) * g


def _ln(x, *a):
    return F.layer_norm(x, x.shape[-1:], *a)


def _rms(x, *a):
    return F.rms_norm(x, x.shape[-1:], *a)


# name -> (fn, argument kinds, expected node kinds without the STORE)
CASES = {
    "postnorm": (lambda X, W, b, r, g, be: _ln(X @ W.t() + b + r, g, be, 1e-5),
                 "X W b r g be", ["BIAS", "RESIDUAL", "LAYERNORM"]),
    "postnorm_residual_first": (lambda X, W, b, r, g, be: _ln(r + (X @ W.t() + b), g, be, 1e-5),
                                "X W b r g be", ["BIAS", "RESIDUAL", "LAYERNORM"]),
    "linear_layernorm": (lambda X, W, b, g, be: _ln(F.linear(X, W, b), g, be, 1e-5),
                         "X W b g be", ["BIAS", "LAYERNORM"]),
    "layernorm_by_hand": (_ln_manual, "X W r", ["RESIDUAL", "LAYERNORM"]),
    "rmsnorm": (lambda X, W, g: _rms(X @ W.t(), g, 1e-6), "X W g", ["RMSNORM"]),
    "rmsnorm_by_hand": (_rms_manual, "X W g", ["RMSNORM"]),
    "mbr": (lambda X, W, b, g: _rms(X @ W.t() + b, g, 1e-6), "X W b g", ["BIAS", "RMSNORM"]),
    "mblr": (lambda X, W, b, g, be: torch.relu(_ln(X @ W.t() + b, g, be)), "X W b g be",
             ["BIAS", "LAYERNORM", "RELU"]),
    "msts": (lambda X, W: torch.softmax(10.0 * torch.tanh((X @ W.t()) * 0.5 / 10.0), dim=-1), "X W",
             ["SCALE", "SOFTCAP", "SOFTMAX"]),
    "ln_gelu": (lambda X, W, b, r: F.gelu(_ln(X @ W.t() + b + r)), "X W b r",
                ["BIAS", "RESIDUAL", "LAYERNORM", "GELU"]),
    "gelu_tanh_kn": (lambda X, Wk, b: F.gelu(X @ Wk + b, approximate="tanh"), "X Wk b", ["BIAS", "GELU_TANH"]),
    "scaled_softmax": (lambda X, W: torch.softmax((X @ W.t()) / 8.0, -1), "X W", ["SCALE", "SOFTMAX"]),
    "fp32_then_relu": (lambda X, W, b: torch.relu((X @ W.t()).float() + b), "X W b", ["BIAS", "RELU"]),
}


def _compile(name):
    fn, kinds, _ = CASES[name]
    args = _args(kinds.split(), dtype=torch.float32)
    return fe.compile_epilogue(fn, args)


def _eval_oracle(P, ep, args):
    """The lowered node list evaluated with the oracle's fp64 primitives."""
    names = {n: args[p].numpy() for n, (_, p) in ep.spec.params.items()}
    x = np.asarray(P, dtype=np.float64)
    for t in ep.templates:
        k = KIND[t.kind]
        if k == "SCALE":
            x = x * t.f0
        elif k == "BIAS":
            x = O.bias_residual(x, names[t.v0])
        elif k == "RESIDUAL":
            x = O.bias_residual(x, None, names[t.inp])
        elif k == "LAYERNORM":
            x = O.layernorm(x, names.get(t.v0), names.get(t.v1), t.f0)
        elif k == "RMSNORM":
            x = O.rmsnorm(x, names.get(t.v0), t.f0)
        elif k == "GELU":
            x = O.gelu_erf(x)
        elif k == "GELU_TANH":
            x = O.gelu_tanh(x)
        elif k == "RELU":
            x = O.relu(x)
        elif k == "SOFTCAP":
            x = O.tanh_softcap(x, t.f0)
        elif k == "SOFTMAX":
            x = O.softmax_rows(x)
        else:
            raise AssertionError(k)
    return x


@pytest.mark.parametrize("name", sorted(CASES))
def test_lowered_node_kinds(name):
    ep = _compile(name)
    assert ep.fused
    assert [KIND[k] for k in ep.node_kinds()] == CASES[name][2] + ["STORE"]


@pytest.mark.parametrize("name", sorted(CASES))
def test_lowering_preserves_semantics(name):
    """Oracle evaluation of the lowered list == the function itself, in fp64."""
    fn, kinds, _ = CASES[name]
    ep = _compile(name)
    args = _args(kinds.split(), seed=1)
    want = fn(*args).numpy()
    X, W = args[ep.spec.x_arg].numpy(), args[ep.spec.w_arg].numpy()
    P = O.matmul(X, W.T if ep.spec.w_layout == cf.CF_LAYOUT_NK else W)
    got = _eval_oracle(P, ep, args)
    # the oracle's erf / tanh GELU vs torch's; an explicit fp32 cast in the
    # function rounds once more than the fused path (fp32 math, one rounding)
    tol = 2e-6 if "GELU" in CASES[name][2] else 1e-5 if "fp32" in name else 1e-10
    assert np.max(np.abs(got - want)) < tol


def test_parameters_and_constants():
    ep = _compile("postnorm")
    roles = {n: r for n, (r, _) in ep.spec.params.items()}
    assert sorted(roles.values()) == ["row", "row", "row", "tile"]
    ln = ep.templates[-1]
    assert KIND[ln.kind] == "LAYERNORM" and ln.f0 == pytest.approx(1e-5)
    assert roles[ln.v0] == "row" and roles[ln.v1] == "row"
    ep = _compile("msts")
    assert [t.f0 for t in ep.templates] == [pytest.approx(0.5), pytest.approx(10.0), 0.0]


def test_fusion_spec_five_tuple():
    """<N, E, tau, A, C>: topological order, consistent edges, the terminal,
    the parameter table and one nested spec per reduction, entered through
    its statistic and the tensor it reduced."""
    ep = _compile("postnorm")
    s = ep.spec
    assert all(i < sn.idx for sn in s.nodes for i in sn.inputs)
    assert sorted(s.edges) == sorted((i, sn.idx) for sn in s.nodes for i in sn.inputs)
    assert s.terminal == len(s.nodes) - 1
    assert [sn.kind for sn in s.nodes].count("acc") == 1
    assert len(s.nested) == 1
    c = s.nested[0]
    red = s.nodes[c["reduce"]]
    assert red.kind == "reduce" and red.op == "var_mean"
    assert c["passthrough"] == red.inputs[0]
    assert s.terminal in c["nodes"]
    # the reduced tensor is bias + residual + product, which the normalisation reuses
    assert s.nodes[c["passthrough"]].op == "add"
    ep = _compile("msts")
    assert sorted(s2["reduce"] for s2 in ep.spec.nested) == sorted(
        sn.idx for sn in ep.spec.nodes if sn.kind == "reduce")
    assert {ep.spec.nodes[c["reduce"]].op for c in ep.spec.nested} == {"amax", "sum"}


UNSUPPORTED = {
    "sigmoid": (lambda X, W: torch.sigmoid(X @ W.t()), "X W", "sigmoid"),
    "scale_after_bias": (lambda X, W, b: (X @ W.t() + b) * 2.0, "X W b", "no rule"),
    "norm_then_softmax": (lambda X, W: torch.softmax(_ln(X @ W.t()), -1), "X W", "softmax"),
    "column_reduction": (lambda X, W: (lambda x: x - x.mean(0, keepdim=True))(X @ W.t()), "X W", "last dimension"),
    "two_products": (lambda X, W: (X @ W.t()) @ W, "X W", "one matrix product"),
    "unbiased_variance": (lambda X, W: (lambda x: (x - x.mean(-1, keepdim=True)) /
                                        torch.sqrt(x.var(-1, keepdim=True) + 1e-5))(X @ W.t()), "X W", "outside the pattern set"),
    "row_scale_without_norm": (lambda X, W, g: (X @ W.t()) * g, "X W g", "no rule"),
}


@pytest.mark.parametrize("name", sorted(UNSUPPORTED))
def test_outside_the_domain_is_reported(name):
    fn, kinds, why = UNSUPPORTED[name]
    args = _args(kinds.split(), dtype=torch.float32)
    with pytest.raises(fe.UnsupportedEpilogue, match=why):
        fe.compile_epilogue(fn, args)
    with pytest.warns(RuntimeWarning, match="not fused"):
        ep = fe.compile_epilogue(fn, args, fallback=True)
    assert not ep.fused and ep.reason
    assert torch.equal(ep(*args), fn(*args))


@pytest.mark.gpu
@pytest.mark.parametrize("name", ["postnorm", "mblr", "msts", "mbr", "ln_gelu", "gelu_tanh_kn"])
def test_lowered_epilogue_on_gpu(name):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fn, kinds, _ = CASES[name]
    ks = kinds.split()
    small = tuple(a.cuda() for a in _args(ks, dtype=torch.float32))
    ep = fe.compile_epilogue(fn, small)
    assert ep.fused
    # real size: 300 rows (ragged), K = N = 256, bf16 matrices, fp32 vectors
    shapes = {"X": (300, 256), "W": (256, 256), "Wk": (256, 256), "b": (256,), "r": (300, 256), "g": (256,),
              "be": (256,)}
    g = torch.Generator().manual_seed(5)
    args = []
    for k in ks:
        t = torch.randn(*shapes[k], generator=g)
        if k in ("W", "Wk"):
            t = t / 16.0
        if k == "g":
            t = 1.0 + 0.1 * t
        args.append(t.to(torch.bfloat16).cuda() if k in ("X", "W", "Wk", "r") else t.cuda())
    got = ep(*args).float().cpu().numpy().astype(np.float64)
    torch.cuda.synchronize()
    # the fp64 oracle on the same (bf16 / fp32) values: the product, then the
    # lowered node list evaluated with the oracle's primitives (whose
    # agreement with the function itself is pinned on the CPU above)
    host = tuple(a.float().cpu().double() for a in args)
    X, W = host[ep.spec.x_arg].numpy(), host[ep.spec.w_arg].numpy()
    P = O.matmul(X, W.T if ep.spec.w_layout == cf.CF_LAYOUT_NK else W)
    ref = _eval_oracle(P, ep, host)
    err = float(np.max(np.abs(got - ref)))
    rel = float(np.sqrt(np.sum((got - ref) ** 2) / np.sum(ref ** 2)))
    assert err < 2e-2 and rel < 5e-3, (err, rel)


# -- the row quantisation tail (ROWAMAX_QUANT): extra results beside z
FP8 = torch.float8_e4m3fn


def _chain_div(X, W, b, r):
    z = F.gelu(_ln(X @ W.t() + b + r))
    s = z.abs().amax(dim=-1, keepdim=True) / 448.0
    return z, s, (z / s).to(FP8)


def _chain_rcp_reordered(X, W, b, r):
    z = F.gelu(_ln(X @ W.t() + b + r))
    s = z.abs().amax(dim=-1, keepdim=True) * (1.0 / 448.0)
    return (z * torch.reciprocal(s)).to(FP8), z, s


def _chain_scale_only(X, W, b, r):
    z = F.gelu(_ln(X @ W.t() + b + r))
    return z, z.abs().amax(dim=-1, keepdim=True) / 448.0


QUANT = {"div": (_chain_div, ["z", "s", "q"]), "rcp_reordered": (_chain_rcp_reordered, ["q", "z", "s"]),
         "scale_only": (_chain_scale_only, ["z", "s"])}


@pytest.mark.parametrize("name", sorted(QUANT))
def test_quant_tail_lowering(name):
    fn, roles = QUANT[name]
    ep = fe.compile_epilogue(fn, _args("X W b r".split(), dtype=torch.float32))
    assert ep.fused and ep.roles == roles
    assert [KIND[k] for k in ep.node_kinds()] == ["BIAS", "RESIDUAL", "LAYERNORM", "GELU", "STORE", "ROWAMAX_QUANT"]
    assert ep.templates[-1].f0 == pytest.approx(448.0)


def test_quant_tail_semantics():
    """Oracle evaluation of the lowered list (main part, then the oracle's
    row-amax quantiser) == the function evaluated by PyTorch in fp64."""
    args = _args("X W b r".split(), seed=2)
    z_t, s_t, q_t = _chain_div(*args)
    ep = fe.compile_epilogue(_chain_div, tuple(a.float() for a in args))
    X, W = args[ep.spec.x_arg].numpy(), args[ep.spec.w_arg].numpy()
    main = fe.FusedGemmEpilogue(ep.spec, ep.templates[:-1])
    z = _eval_oracle(O.matmul(X, W.T), main, args)
    s, q = O.rowamax_quant(z, ep.templates[-1].f0)
    assert np.max(np.abs(z - z_t.numpy())) < 2e-6          # the oracle's erf vs torch's
    np.testing.assert_allclose(s, s_t.numpy()[:, 0], rtol=1e-5)
    codes_t = q_t.view(torch.uint8).numpy()
    assert np.mean(codes_t == q) >= 0.99
    assert np.max(np.abs(O.e4m3_decode(codes_t) - O.e4m3_decode(q)) / s[:, None]) <= 32.0


UNSUPPORTED_TAIL = {
    "amax_without_abs": lambda X, W: (lambda z: (z, z.amax(-1, keepdim=True) / 448.0))(F.gelu(X @ W.t())),
    "codes_of_another_scale": lambda X, W: (lambda z: (z, (z / 2.0).to(FP8)))(F.gelu(X @ W.t())),
    "two_stored_tensors": lambda X, W: (lambda z: (z, z * 2.0))(F.gelu(X @ W.t())),
}


@pytest.mark.parametrize("name", sorted(UNSUPPORTED_TAIL))
def test_quant_tail_outside_the_domain(name):
    with pytest.raises(fe.UnsupportedEpilogue):
        fe.compile_epilogue(UNSUPPORTED_TAIL[name], _args("X W".split(), dtype=torch.float32))


@pytest.mark.gpu
def test_lowered_quant_tail_on_gpu():
    """The LN -> GELU -> amax -> E4M3 chain written in PyTorch, lowered and run
    fused (fp32 z out, so the codes can be recomputed exactly from it), against
    the fp64 oracle (ragged 300 rows, K = N = 256)."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    small = tuple(a.cuda() for a in _args("X W b r".split(), dtype=torch.float32))
    ep = fe.compile_epilogue(_chain_div, small, out_dtype=torch.float32)
    g = torch.Generator().manual_seed(9)
    X = torch.randn(300, 256, generator=g).to(torch.bfloat16)
    W = (torch.randn(256, 256, generator=g) / 16.0).to(torch.bfloat16)
    b = 0.02 * torch.randn(256, generator=g)
    r = torch.randn(300, 256, generator=g).to(torch.bfloat16)
    z, s, q = ep(X.cuda(), W.cuda(), b.cuda(), r.cuda())
    torch.cuda.synchronize()
    assert q.dtype == FP8 and s.shape == (300, 1)
    zg, sg, qg = z.cpu().numpy(), s.cpu().numpy()[:, 0], q.view(torch.uint8).cpu().numpy()
    zr, sr, qr = O.ln_gelu_amax(X.double().numpy(), W.double().numpy().T, b.double().numpy(), r.double().numpy())
    assert np.max(np.abs(zg - zr)) < 1e-4
    np.testing.assert_allclose(sg, sr, rtol=1e-3)
    s32, q32 = O.rowamax_quant_f32(zg)
    np.testing.assert_array_equal(sg, s32)
    np.testing.assert_array_equal(qg, q32)
    assert np.mean(qg == qr) >= 0.9999
