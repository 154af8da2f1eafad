"""GPU parity of the back-to-back MLP (cf_b2bgemm with S = ReLU(X W1 + b1),
the DLRM bottom-MLP pattern of Table 2) against the fp64 oracle.

O is bf16: max-abs 2e-2 and rel-RMS 5e-3 (the intermediate S is rounded to
bf16 as the second product's operand; the oracle keeps it exact).  The hidden
dimension comes in chunks of 256 units whose partial second products are
summed in chunk order.  While batch x 128-row blocks x chunks fits 256
workgroups the chunks are split over workgroups and the last workgroup of
each row block to finish sums their partials at commit, so the result is
the same whichever finishes last; beyond that one workgroup per row block
runs every chunk.
"""
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


def run_mlp(inp, out_relu=False, with_b2=True, ws=None):
    Y = cf.b2b_mlp(dev(inp.X), dev(I.lay_out_weight(inp.W1, "nk")), dev(inp.b1, "f32"),
                   dev(I.lay_out_weight(inp.W2, "nk")), dev(inp.b2, "f32") if with_b2 else None,
                   out_relu=out_relu, ws=ws)
    torch.cuda.synchronize()
    return Y


@pytest.mark.parametrize("M,K,N1", [(300, 128, 256), (257, 256, 512), (129, 192, 768), (77, 1024, 512)])
@pytest.mark.parametrize("out_relu", [False, True])
def test_mlp_small(M, K, N1, out_relu):
    inp = I.dlrm_mlp_inputs(seed=3, M=M, K=K, N1=N1)
    got = host(run_mlp(inp, out_relu))
    ref = O.mlp_b2b(inp.X, inp.W1, inp.b1, inp.W2, inp.b2, out_relu=out_relu)
    assert_close_bf16(got, ref, f"MLP {M}x{K}x{N1} relu={out_relu}")


def test_mlp_without_b2_and_all_negative_hidden():
    inp = I.dlrm_mlp_inputs(seed=4, M=200, K=256, N1=512)
    got = host(run_mlp(inp, with_b2=False))
    assert_close_bf16(got, O.mlp_b2b(inp.X, inp.W1, inp.b1, inp.W2, None), "MLP without b2")
    # every pre-activation negative: S = 0 and O = b2 exactly
    inp.b1[:] = -100.0
    got = host(run_mlp(inp))
    assert np.array_equal(got, np.broadcast_to(I.round_to_bf16(inp.b2.astype(np.float32)).astype(np.float64),
                                                got.shape))


def test_mlp_split_is_deterministic_and_leaves_counters_at_zero():
    inp = I.dlrm_mlp_inputs(seed=5, M=4096, K=512, N1=1024)
    X, W1, W2 = dev(inp.X), dev(I.lay_out_weight(inp.W1, "nk")), dev(I.lay_out_weight(inp.W2, "nk"))
    b1, b2 = dev(inp.b1, "f32"), dev(inp.b2, "f32")
    ws = torch.zeros(64 << 20, dtype=torch.uint8, device="cuda")
    outs = [cf.b2b_mlp(X, W1, b1, W2, b2, ws=ws) for _ in range(3)]
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o.view(torch.int16), outs[0].view(torch.int16))
    assert int(ws[:cf.CF_B2B_WS_HEADER_BYTES].view(torch.int32).abs().sum().item()) == 0
    assert_close_bf16(host(outs[0]), O.mlp_b2b(inp.X, inp.W1, inp.b1, inp.W2, inp.b2), "MLP 4096x512x1024")


def test_mlp_dlrm_full_size_block_rows():
    # the Table 2 widths 1024 -> 512 -> 128 at 65536 rows: one row in every
    # 128-row block (both workgroups of the block and their commit) against
    # the oracle, and the ReLU output's exact zero count against the oracle's
    inp = I.dlrm_mlp_inputs()
    Y = host(run_mlp(inp, out_relu=True))
    nb = inp.M // 128
    rows = np.arange(nb) * 128 + (np.arange(nb) * 37) % 128
    ref = O.mlp_b2b(inp.X[rows], inp.W1, inp.b1, inp.W2, inp.b2, out_relu=True)
    assert_close_bf16(Y[rows], ref, "DLRM MLP 65536x1024x512x128")
    assert np.all(Y >= 0.0)


def _block_rows(M, seed):
    # one row in every 128-row block, and every row of the last block
    nb = (M + 127) // 128
    rows = np.arange(nb) * 128 + (np.arange(nb) * seed) % 128
    rows = rows[rows < M]
    return np.unique(np.concatenate([rows, np.arange((nb - 1) * 128, M)]))


def test_mlp_whole_row_block_form():
    # 257 row blocks (the last one ragged) x 3 chunks: the whole-row-block
    # form, one workgroup runs all 3 chunks of its rows; no workspace
    inp = I.dlrm_mlp_inputs(seed=8, M=256 * 128 + 77, K=256, N1=768)
    assert cf.cf_b2bgemm_workspace(cf._b2b_args(batch=1, M=inp.M, K=256, N1=768, N2=128, dtype=cf.CF_BF16,
                                                mid=cf.CF_MID_RELU_BIAS, out=cf.CF_OUT_STORE)) == 0
    Y = host(run_mlp(inp, out_relu=True))
    rows = _block_rows(inp.M, 41)
    ref = O.mlp_b2b(inp.X[rows], inp.W1, inp.b1, inp.W2, inp.b2, out_relu=True)
    assert_close_bf16(Y[rows], ref, "MLP whole form 32845x256x768")


def test_mlp_whole_row_block_form_is_deterministic():
    # the chunks' partial products are summed in registers in chunk order:
    # repeated calls give the same bits
    inp = I.dlrm_mlp_inputs(seed=9, M=200 * 128 + 3, K=128, N1=512)
    X, W1, W2 = dev(inp.X), dev(I.lay_out_weight(inp.W1, "nk")), dev(I.lay_out_weight(inp.W2, "nk"))
    b1, b2 = dev(inp.b1, "f32"), dev(inp.b2, "f32")
    outs = [cf.b2b_mlp(X, W1, b1, W2, b2, out_relu=True) for _ in range(3)]
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o.view(torch.int16), outs[0].view(torch.int16))
    rows = _block_rows(inp.M, 17)
    ref = O.mlp_b2b(inp.X[rows], inp.W1, inp.b1, inp.W2, inp.b2, out_relu=True)
    assert_close_bf16(host(outs[0])[rows], ref, "MLP whole form 25603x128x512")


def test_mlp_whole_row_block_form_batched():
    # 2 entries x 129 row blocks x 2 chunks: the whole form over a batch, W1
    # shared, W2 per entry
    Bn, M, K, N1 = 2, 128 * 128 + 5, 128, 512
    ins = [I.dlrm_mlp_inputs(seed=30 + b, M=M, K=K, N1=N1) for b in range(Bn)]
    X = dev(np.stack([t.X for t in ins]))
    W1t = dev(I.lay_out_weight(ins[0].W1, "nk"))
    W2t = dev(np.stack([I.lay_out_weight(t.W2, "nk") for t in ins]))
    Y = cf.b2b_mlp(X, W1t, dev(ins[0].b1, "f32"), W2t, dev(ins[0].b2, "f32"))
    torch.cuda.synchronize()
    got = host(Y)
    rows = _block_rows(M, 23)
    for b in range(Bn):
        ref = O.mlp_b2b(ins[b].X[rows], ins[0].W1, ins[0].b1, ins[b].W2, ins[0].b2)
        assert_close_bf16(got[b][rows], ref, f"MLP whole form batch entry {b}")


def test_mlp_shape_change_on_one_workspace():
    """Calls of different shapes share a workspace (all three take the split
    form): the second call has more row blocks (more arrival counters) than
    the first, and the first call's partials must not be read as the second
    call's counters."""
    ws = torch.zeros(96 << 20, dtype=torch.uint8, device="cuda")
    for M, K, N1 in [(8192, 128, 1024), (16000, 128, 512), (300, 256, 768)]:
        inp = I.dlrm_mlp_inputs(seed=6, M=M, K=K, N1=N1)
        got = host(run_mlp(inp, ws=ws))
        assert_close_bf16(got, O.mlp_b2b(inp.X, inp.W1, inp.b1, inp.W2, inp.b2), f"MLP {M}x{K}x{N1} after another shape")
        assert int(ws[:cf.CF_B2B_WS_HEADER_BYTES].view(torch.int32).abs().sum().item()) == 0


@pytest.mark.parametrize("shared_w1,shared_w2", [(False, True), (True, False), (False, False)])
def test_mlp_batched(shared_w1, shared_w2):
    """batch = 3 entries of 300 rows: X and O [3, M, .], each weight per entry
    (3-D, batch stride) or shared (2-D, stride 0); biases shared."""
    Bn, M, K, N1 = 3, 300, 256, 512
    ins = [I.dlrm_mlp_inputs(seed=20 + b, M=M, K=K, N1=N1) for b in range(Bn)]
    w1 = [ins[0 if shared_w1 else b].W1 for b in range(Bn)]
    w2 = [ins[0 if shared_w2 else b].W2 for b in range(Bn)]
    X = dev(np.stack([t.X for t in ins]))
    W1t = dev(I.lay_out_weight(w1[0], "nk")) if shared_w1 else dev(np.stack([I.lay_out_weight(w, "nk") for w in w1]))
    W2t = dev(I.lay_out_weight(w2[0], "nk")) if shared_w2 else dev(np.stack([I.lay_out_weight(w, "nk") for w in w2]))
    Y = cf.b2b_mlp(X, W1t, dev(ins[0].b1, "f32"), W2t, dev(ins[0].b2, "f32"), out_relu=True)
    torch.cuda.synchronize()
    assert tuple(Y.shape) == (Bn, M, 128)
    got = host(Y)
    for b in range(Bn):
        ref = O.mlp_b2b(ins[b].X, w1[b], ins[0].b1, w2[b], ins[0].b2, out_relu=True)
        assert_close_bf16(got[b], ref, f"MLP batch entry {b}")

