"""GPU parity of cf_gemm_subgraph / cf_rowop (the Stage-Stream node lists)
against the fp64 oracle.

The LN -> GELU -> row-amax -> E4M3 chain: Z (bf16) within max-abs 2e-2 /
rel-RMS 5e-3, s within relative 1e-3, codes equal to the oracle's for at least
99.99 % of elements with every mismatch one code step away (Z differs from
the exact value by bf16 GEMM rounding, so codes at rounding boundaries can
move by one step).  With Z stored in fp32 the quantisation stage is checked
bit-exactly against the kernel's own z, deciding in fp32 on both sides.
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


def signed_code_index(q):
    q = np.asarray(q, np.int64)
    return np.where(q & 0x80, -(q & 0x7F), q & 0x7F)


def check_codes(q_gpu, q_ref, min_equal=0.9999):
    eq = np.mean(q_gpu == q_ref)
    step = np.abs(signed_code_index(q_gpu) - signed_code_index(q_ref))
    assert eq >= min_equal, f"codes equal {eq:.6f}"
    assert step.max() <= 1, f"max code step {step.max()}"
    return eq


def run_chain(inp, path=0, z_f32=False, layout="nk", gelu=cf.CF_N_GELU):
    X = dev(inp.X, inp.dtype)
    W = dev(I.lay_out_weight(inp.W, layout), inp.dtype)
    R = dev(inp.R, inp.dtype) if inp.R is not None else None
    b = dev(inp.bias, "f32") if inp.bias is not None else None
    Z, s, Q = cf.ln_gelu_amax(X, W, b, R, eps=inp.eps, z_dtype=torch.float32 if z_f32 else None,
                              w_layout=cf.CF_LAYOUT_NK if layout == "nk" else cf.CF_LAYOUT_KN, path=path,
                              gelu=gelu)
    torch.cuda.synchronize()
    return host(Z), s.cpu().numpy(), Q.cpu().numpy()


@pytest.mark.parametrize("path", [1, 2, 3])
@pytest.mark.parametrize("N", [256, 768, 1024])
def test_chain_small(N, path):
    if path == 1 and N > 768:
        pytest.skip("whole-row path covers N <= 768")
    inp = I.postnorm_inputs(150, 128, N, "bf16", seed=11, with_affine=False)
    z, s, q = O.ln_gelu_amax(inp.X, inp.W, inp.bias, inp.R, eps=inp.eps)
    Zg, sg, Qg = run_chain(inp, path)
    assert_close_bf16(Zg, z, f"Z N={N} path {path}")
    np.testing.assert_allclose(sg, s, rtol=1e-3)
    check_codes(Qg, q)


@pytest.mark.parametrize("N", [160, 320])
def test_chain_ragged_tile_whole_row(N):
    # N = 160 / 320 leave 96 / 64 padding columns in the 256 / 384-wide tile;
    # after LayerNorm they hold -mean/std, and must not enter the row amax.
    # A residual shifted by -10 makes that about +7, above every real |z|.
    inp = I.postnorm_inputs(70, 128, N, "bf16", seed=21, with_affine=False)
    inp.R = I.round_to_bf16(inp.R - 10.0)
    z, s, q = O.ln_gelu_amax(inp.X, inp.W, inp.bias, inp.R, eps=inp.eps)
    Zg, sg, Qg = run_chain(inp, 1)
    assert_close_bf16(Zg, z, f"Z N={N} whole-row")
    np.testing.assert_allclose(sg, s, rtol=1e-3)
    check_codes(Qg, q)


@pytest.mark.parametrize("path", [1, 2, 3])
def test_chain_quant_exact_against_own_z(path):
    inp = I.postnorm_inputs(97, 64, 512, "f32", seed=12, with_affine=False)
    Zg, sg, Qg = run_chain(inp, path, z_f32=True)
    s32, q32 = O.rowamax_quant_f32(Zg.astype(np.float32))
    assert np.array_equal(sg, s32)
    assert np.array_equal(Qg, q32)
    z, _, _ = O.ln_gelu_amax(inp.X, inp.W, inp.bias, inp.R, eps=inp.eps)
    assert_close_f32(Zg, z, "fp32 chain")


@pytest.mark.parametrize("N", [1280, 2048, 3072, 4160])
def test_chain_split_wide_rows(N):
    # Split-N rows wider than 1024 finish in one workgroup per row: whole
    # multiples of 1024 (2048) and ragged widths, where whole column groups
    # of the last waves (3072: the fourth group of every wave) hold no data.
    inp = I.postnorm_inputs(70, 64, N, "bf16", seed=31, with_affine=False)
    z, s, q = O.ln_gelu_amax(inp.X, inp.W, inp.bias, inp.R, eps=inp.eps)
    Zg, sg, Qg = run_chain(inp, 3)
    assert_close_bf16(Zg, z, f"Z N={N} split")
    np.testing.assert_allclose(sg, s, rtol=1e-3)
    check_codes(Qg, q)


def test_chain_split_wide_quant_exact_against_own_z():
    # fp32 Z from the wide-row finish pass: its scale and codes equal the
    # fp32 scale chain applied to that Z, exactly.
    inp = I.postnorm_inputs(33, 64, 2112, "f32", seed=32, with_affine=False)
    Zg, sg, Qg = run_chain(inp, 3, z_f32=True)
    s32, q32 = O.rowamax_quant_f32(Zg.astype(np.float32))
    assert np.array_equal(sg, s32)
    assert np.array_equal(Qg, q32)


@pytest.mark.parametrize("norm,N", [("rms", 2560), ("ln", 3136)])
def test_split_wide_rows_affine(norm, N):
    # RMSNorm (gamma) and LayerNorm (gamma, beta) on the wide-row finish pass.
    inp = I.postnorm_inputs(40, 64, N, "f32", seed=33, with_residual=False)
    X, W = dev(inp.X, "f32"), dev(I.lay_out_weight(inp.W, "nk"), "f32")
    b, g, be = dev(inp.bias, "f32"), dev(inp.gamma, "f32"), dev(inp.beta, "f32")
    Y = torch.empty((inp.M, inp.N), dtype=torch.float32, device="cuda")
    if norm == "rms":
        spec = [dict(kind=cf.CF_N_BIAS, v0=b), dict(kind=cf.CF_N_RMSNORM, v0=g, f0=1e-5),
                dict(kind=cf.CF_N_STORE, out=Y, ld=inp.N, dtype=cf.CF_F32)]
        r = O.rmsnorm(O.bias_residual(O.matmul(inp.X, inp.W), inp.bias), inp.gamma, 1e-5)
    else:
        spec = [dict(kind=cf.CF_N_BIAS, v0=b), dict(kind=cf.CF_N_LAYERNORM, v0=g, v1=be, f0=1e-5),
                dict(kind=cf.CF_N_STORE, out=Y, ld=inp.N, dtype=cf.CF_F32)]
        r = O.postnorm(inp.X, inp.W, inp.bias, None, inp.gamma, inp.beta, 1.0, 1e-5)
    cf.gemm_subgraph(X, W, spec, path=3)
    torch.cuda.synchronize()
    assert_close_f32(host(Y), r, f"{norm} N={N} split")


def test_gelu_tanh_variant_is_the_tanh_one():
    inp = I.postnorm_inputs(64, 64, 256, "f32", seed=13, with_affine=False)
    Zg, _, _ = run_chain(inp, 1, z_f32=True, gelu=cf.CF_N_GELU_TANH)
    y = O.postnorm(inp.X, inp.W, inp.bias, inp.R, eps=inp.eps)
    assert_close_f32(Zg, O.gelu_tanh(y), "tanh GELU")
    assert np.max(np.abs(Zg - O.gelu_erf(y))) > 2e-4


def block_rows(M, block=128, seed=0):
    """One row in every block of `block` rows (at a position that moves from
    block to block, so every slot of a tile is hit somewhere), plus the
    first, last and tile-edge rows."""
    nb = (M + block - 1) // block
    off = (np.arange(nb) * 37 + seed) % block
    rows = np.minimum(np.arange(nb) * block + off, M - 1)
    return np.unique(np.concatenate([rows, [0, 1, block - 1, block, M - 1]]))


@pytest.mark.parametrize("path", [0, 2])
def test_chain_full_size_sampled_rows(path):
    inp = I.ln_gelu_amax_inputs()
    Zg, sg, Qg = run_chain(inp, path)
    rows = block_rows(inp.M)
    assert len(rows) >= inp.M // 128
    z, s, q = O.ln_gelu_amax(inp.X[rows], inp.W, inp.bias, inp.R[rows], eps=inp.eps)
    assert_close_bf16(Zg[rows], z, f"cfg3 Z path {path}")
    np.testing.assert_allclose(sg[rows], s, rtol=1e-3)
    check_codes(Qg[rows], q)
    # every compared row's largest code is +-448 (s = amax / 448 by construction)
    assert np.all(np.max(np.abs(O.e4m3_decode(Qg[rows])), axis=1) == 448.0)
    # and the same on every 97th row of the whole output (a property at any size)
    assert np.all(np.max(np.abs(O.e4m3_decode(Qg[::97])), axis=1) == 448.0)


def test_chain_cluster_capped_grid_uneven_rounds():
    """Row clusters of 16 peers (N = 4096 in 256-wide tiles) at M = 3072: 24 row
    blocks, but only 2 slots per XCD fit the device, so the workgroups loop
    (the persistent kernel form) and the slots of an XCD run different numbers
    of rounds (row blocks 0..15 in the first, 16..23 in the second).  Every
    row is compared."""
    inp = I.postnorm_inputs(3072, 128, 4096, "bf16", seed=21, with_affine=False)
    Zg, sg, Qg = run_chain(inp, path=2)
    z, s, q = O.ln_gelu_amax(inp.X, inp.W, inp.bias, inp.R, eps=inp.eps)
    assert_close_bf16(Zg, z, "cluster 3072x4096 capped grid")
    np.testing.assert_allclose(sg, s, rtol=1e-3)
    check_codes(Qg, q)


@pytest.mark.parametrize("norm", ["rms", "ln_relu"])
def test_other_stage_stream_patterns(norm):
    # MatMul-BiasAdd-RMSNorm and MatMul-BiasAdd-LayerNorm-ReLU (Sec. VI).
    inp = I.postnorm_inputs(130, 96, 512, "f32", seed=14, with_residual=False)
    X, W = dev(inp.X, "f32"), dev(I.lay_out_weight(inp.W, "nk"), "f32")
    b, g, be = dev(inp.bias, "f32"), dev(inp.gamma, "f32"), dev(inp.beta, "f32")
    for path in (1, 2, 3):
        Y = torch.empty((inp.M, inp.N), dtype=torch.float32, device="cuda")
        if norm == "rms":
            spec = [dict(kind=cf.CF_N_BIAS, v0=b), dict(kind=cf.CF_N_RMSNORM, v0=g, f0=1e-5),
                    dict(kind=cf.CF_N_STORE, out=Y, ld=inp.N, dtype=cf.CF_F32)]
            r = O.rmsnorm(O.bias_residual(O.matmul(inp.X, inp.W), inp.bias), inp.gamma, 1e-5)
        else:
            spec = [dict(kind=cf.CF_N_BIAS, v0=b), dict(kind=cf.CF_N_LAYERNORM, v0=g, v1=be, f0=1e-5),
                    dict(kind=cf.CF_N_RELU), dict(kind=cf.CF_N_STORE, out=Y, ld=inp.N, dtype=cf.CF_F32)]
            r = O.relu(O.postnorm(inp.X, inp.W, inp.bias, None, inp.gamma, inp.beta, 1.0, 1e-5))
        cf.gemm_subgraph(X, W, spec, path=path)
        torch.cuda.synchronize()
        assert_close_f32(host(Y), r, f"{norm} path {path}")


def test_rowop_quant_encoder_exact():
    # Rows built so that z/s hits every E4M3 value, every midpoint between
    # neighbours, and values just either side of each midpoint.
    vals = O.e4m3_decode(np.arange(0, 0x7F)).astype(np.float64)
    mids = (vals[:-1] + vals[1:]) / 2
    pts = np.concatenate([vals, mids, np.nextafter(mids.astype(np.float32), np.float32(0)),
                          np.nextafter(mids.astype(np.float32), np.float32(1e9))]).astype(np.float32)
    pts = np.concatenate([pts, -pts])
    n = ((len(pts) + 255) // 256) * 256
    row = np.zeros(n, np.float32)
    row[:len(pts)] = pts
    # Scales that are not powers of two put z/s next to the midpoints, where
    # only a correctly rounded fp32 quotient gives the reference code.
    P = np.stack([row, row * np.float32(0.5), row * np.float32(1e-3), np.zeros(n, np.float32),
                  row * np.float32(0.37), row * np.float32(0.033), row * np.float32(7.1)])
    Pd = dev(P, "f32")
    s = torch.empty(len(P), dtype=torch.float32, device="cuda")
    Q = torch.empty((len(P), n), dtype=torch.uint8, device="cuda")
    cf.rowop(Pd, [dict(kind=cf.CF_N_ROWAMAX_QUANT, out=s, out2=Q, ld=n, f0=448.0)])
    torch.cuda.synchronize()
    s32, q32 = O.rowamax_quant_f32(P)
    assert np.array_equal(s.cpu().numpy(), s32)
    qg = Q.cpu().numpy()
    bad = np.argwhere(qg != q32)
    assert len(bad) == 0, [(int(i), int(j), float(P[i, j]), hex(qg[i, j]), hex(q32[i, j])) for i, j in bad[:8]]


@pytest.mark.parametrize("N,p_dtype", [(3072, torch.bfloat16), (4160, torch.float32)])
def test_rowop_wide_rows_chain(N, p_dtype):
    # The unfused row operator on rows wider than 1024 (one workgroup per
    # row): bias, residual, LayerNorm, GELU, store, row amax and E4M3 codes
    # over a materialised product (bf16 or fp32), against the oracle.
    inp = I.postnorm_inputs(45, 64, N, "bf16", seed=34, with_affine=False)
    X, W = dev(inp.X), dev(I.lay_out_weight(inp.W, "nk"))
    b, R = dev(inp.bias, "f32"), dev(inp.R)
    P = cf.gemm(X, W, out_dtype=p_dtype)
    Z = torch.empty((inp.M, N), dtype=torch.bfloat16, device="cuda")
    s = torch.empty(inp.M, dtype=torch.float32, device="cuda")
    Q = torch.empty((inp.M, N), dtype=torch.uint8, device="cuda")
    cf.rowop(P, [dict(kind=cf.CF_N_BIAS, v0=b), dict(kind=cf.CF_N_RESIDUAL, **{"in": R}, ld=N, dtype=cf.CF_BF16),
                 dict(kind=cf.CF_N_LAYERNORM, f0=1e-5), dict(kind=cf.CF_N_GELU),
                 dict(kind=cf.CF_N_STORE, out=Z, ld=N, dtype=cf.CF_BF16),
                 dict(kind=cf.CF_N_ROWAMAX_QUANT, out=s, out2=Q, ld=N, f0=448.0)])
    torch.cuda.synchronize()
    if p_dtype == torch.bfloat16:
        # the oracle runs on the same bf16-rounded product the row pass reads
        Pr = host(P).astype(np.float64)
        z = O.gelu_erf(O.layernorm(O.bias_residual(Pr, inp.bias, inp.R), eps=1e-5))
        sr, q = O.rowamax_quant(z)
    else:
        z, sr, q = O.ln_gelu_amax(inp.X, inp.W, inp.bias, inp.R, eps=1e-5)
    assert_close_bf16(host(Z), z, f"unfused wide chain N={N}")
    np.testing.assert_allclose(s.cpu().numpy(), sr, rtol=1e-3)
    check_codes(Q.cpu().numpy(), q)


def test_rowop_wide_rows_rms():
    inp = I.postnorm_inputs(37, 64, 2560, "f32", seed=35, with_residual=False)
    X, W = dev(inp.X, "f32"), dev(I.lay_out_weight(inp.W, "nk"), "f32")
    b, g = dev(inp.bias, "f32"), dev(inp.gamma, "f32")
    P = cf.gemm(X, W, out_dtype=torch.float32)
    Y = torch.empty((inp.M, inp.N), dtype=torch.float32, device="cuda")
    cf.rowop(P, [dict(kind=cf.CF_N_BIAS, v0=b), dict(kind=cf.CF_N_RMSNORM, v0=g, f0=1e-5),
                 dict(kind=cf.CF_N_STORE, out=Y, ld=inp.N, dtype=cf.CF_F32)])
    torch.cuda.synchronize()
    r = O.rmsnorm(O.bias_residual(O.matmul(inp.X, inp.W), inp.bias), inp.gamma, 1e-5)
    assert_close_f32(host(Y), r, "unfused wide RMSNorm")


def test_rowop_matches_fused_chain():
    inp = I.postnorm_inputs(70, 64, 384, "bf16", seed=15, with_affine=False)
    X, W = dev(inp.X), dev(I.lay_out_weight(inp.W, "nk"))
    b, R = dev(inp.bias, "f32"), dev(inp.R)
    P = cf.gemm(X, W, out_dtype=torch.float32)
    Z = torch.empty((70, 384), dtype=torch.bfloat16, device="cuda")
    s = torch.empty(70, dtype=torch.float32, device="cuda")
    Q = torch.empty((70, 384), dtype=torch.uint8, device="cuda")
    cf.rowop(P, [dict(kind=cf.CF_N_BIAS, v0=b), dict(kind=cf.CF_N_RESIDUAL, **{"in": R}, ld=384, dtype=cf.CF_BF16),
                 dict(kind=cf.CF_N_LAYERNORM, f0=1e-5), dict(kind=cf.CF_N_GELU),
                 dict(kind=cf.CF_N_STORE, out=Z, ld=384, dtype=cf.CF_BF16),
                 dict(kind=cf.CF_N_ROWAMAX_QUANT, out=s, out2=Q, ld=384, f0=448.0)])
    torch.cuda.synchronize()
    z, sr, q = O.ln_gelu_amax(inp.X, inp.W, inp.bias, inp.R, eps=1e-5)
    assert_close_bf16(host(Z), z, "unfused chain")
    np.testing.assert_allclose(s.cpu().numpy(), sr, rtol=1e-3)
    check_codes(Q.cpu().numpy(), q)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("act", ["none", "gelu", "relu"])
def test_subgraph_without_reduction(act, dtype):
    # Residual / activation without a row reduction: any tiling, row epilogue.
    inp = I.postnorm_inputs(150, 64, 320, dtype, seed=16, with_affine=False, bias_std=0.3)
    X, W = dev(inp.X, dtype), dev(I.lay_out_weight(inp.W, "nk"), dtype)
    b, R = dev(inp.bias, "f32"), dev(inp.R, dtype)
    Y = torch.empty((inp.M, inp.N), dtype=torch.float32, device="cuda")
    spec = [dict(kind=cf.CF_N_SCALE, f0=0.5), dict(kind=cf.CF_N_BIAS, v0=b),
            dict(kind=cf.CF_N_RESIDUAL, **{"in": R}, ld=inp.N, dtype=cf._dt(R))]
    if act == "gelu":
        spec.append(dict(kind=cf.CF_N_GELU))
    if act == "relu":
        spec.append(dict(kind=cf.CF_N_RELU))
    spec.append(dict(kind=cf.CF_N_STORE, out=Y, ld=inp.N, dtype=cf.CF_F32))
    cf.gemm_subgraph(X, W, spec)
    torch.cuda.synchronize()
    x = O.bias_residual(O.matmul(inp.X, inp.W), inp.bias, inp.R, alpha=0.5)
    ref = {"none": x, "gelu": O.gelu_erf(x), "relu": O.relu(x)}[act]
    assert_close_f32(host(Y), ref, f"no-reduction {act} {dtype}")


# ---------------------------------------------------------------- MSTS: scale -> softcap -> softmax
def run_msts(inp, path=0, out_f32=False, layout="nk"):
    X = dev(inp.X, inp.dtype)
    W = dev(I.lay_out_weight(inp.W, layout), inp.dtype)
    Y = torch.empty((inp.M, inp.N), dtype=torch.float32 if out_f32 else torch.bfloat16, device="cuda")
    spec = [dict(kind=cf.CF_N_SCALE, f0=inp.alpha)]
    if inp.bias is not None:
        spec.append(dict(kind=cf.CF_N_BIAS, v0=dev(inp.bias, "f32")))
    spec += [dict(kind=cf.CF_N_SOFTCAP, f0=inp.meta["cap"]), dict(kind=cf.CF_N_SOFTMAX),
             dict(kind=cf.CF_N_STORE, out=Y, ld=inp.N, dtype=cf.CF_F32 if out_f32 else cf.CF_BF16)]
    cf.gemm_subgraph(X, W, spec, w_layout=cf.CF_LAYOUT_NK if layout == "nk" else cf.CF_LAYOUT_KN, path=path)
    torch.cuda.synchronize()
    return host(Y)


def msts_ref(inp):
    return O.msts(inp.X, inp.W, inp.alpha, inp.bias, inp.meta["cap"])


@pytest.mark.parametrize("path", [1, 2, 3])
@pytest.mark.parametrize("M,K,N", [(200, 128, 512), (77, 192, 384), (130, 64, 320), (64, 256, 1024)])
def test_msts_small(M, K, N, path):
    inp = I.msts_inputs(seed=12, M=M, K=K, N=N)
    if path == 1 and N > 768:
        pytest.skip("whole-row path covers N <= 768")
    if path == 2 and not any(N % t == 0 for t in (256, 192, 128)):
        with pytest.raises(cf.CfError, match="UNSUPPORTED"):
            run_msts(inp, path)
        return
    ref = msts_ref(inp)
    got = run_msts(inp, path)
    assert_close_bf16(got, ref, f"MSTS {M}x{K}x{N} path {path}")
    np.testing.assert_allclose(got.astype(np.float64).sum(axis=1), 1.0, atol=0.02)


@pytest.mark.parametrize("path", [0, 3])
def test_msts_fp32_out_and_kn_layout(path):
    inp = I.msts_inputs(seed=13, M=150, K=128, N=512, dtype="f32")
    ref = msts_ref(inp)
    assert_close_f32(run_msts(inp, path, out_f32=True, layout="kn"), ref, f"MSTS fp32 kn path {path}")


def test_msts_full_size_sampled_rows():
    inp = I.msts_inputs()
    got = run_msts(inp)
    rows = np.unique(np.concatenate([[0, 1, 127, 128, inp.M - 1],
                                     np.random.default_rng(1).choice(inp.M, 27, replace=False)]))
    ref = O.msts(inp.X[rows], inp.W, inp.alpha, inp.bias, inp.meta["cap"])
    assert_close_bf16(got[rows], ref, "MSTS full size")


def test_rowop_msts_grammar():
    # the unfused row operator runs the same node list on a materialised P
    inp = I.msts_inputs(seed=14, M=96, K=128, N=640, dtype="f32")
    P = dev(O.matmul(inp.X, inp.W), "f32")
    Y = torch.empty((inp.M, inp.N), dtype=torch.float32, device="cuda")
    spec = [dict(kind=cf.CF_N_SCALE, f0=inp.alpha), dict(kind=cf.CF_N_BIAS, v0=dev(inp.bias, "f32")),
            dict(kind=cf.CF_N_SOFTCAP, f0=inp.meta["cap"]), dict(kind=cf.CF_N_SOFTMAX),
            dict(kind=cf.CF_N_STORE, out=Y, ld=inp.N, dtype=cf.CF_F32)]
    cf.rowop(P, spec)
    torch.cuda.synchronize()
    assert_close_f32(host(Y), msts_ref(inp), "rowop MSTS")
