"""Pins for the fp64 oracle: each check compares it against something other
than itself — exact rational arithmetic, mpmath at 40 digits, closed forms,
textbook tables, invariants the mathematics fixes, or a library routine that
is not the one the oracle calls.  Chosen so that a dropped term, a sign or
index slip, or a transposed operand in the oracle fails at least one of them.
"""
import math
import os
from fractions import Fraction

import mpmath
import numpy as np
import pytest
import torch

from oracle import comfuse_oracle as O
from paper_2608_03537_amd import inputs as I

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
mpmath.mp.dps = 40


def _fr(a):
    return [[Fraction(float(v)) for v in row] for row in np.asarray(a, np.float64)]


def _mm_exact(A, B):
    A, B = _fr(A), _fr(B)
    M, K, N = len(A), len(B), len(B[0])
    return [[sum(A[i][k] * B[k][j] for k in range(K)) for j in range(N)] for i in range(M)]


def _small(shape, seed, tid, std=1.0):
    rng = np.random.default_rng([seed, 7777, tid])
    return I.round_to_bf16((rng.standard_normal(shape) * std).astype(np.float32))


# ---------------------------------------------------------------- matmul
@pytest.mark.parametrize("M,K,N", [(4, 4, 4), (4, 8, 4), (3, 5, 7)])
def test_matmul_exact_rational(M, K, N):
    A, B = _small((M, K), 1, 0), _small((K, N), 1, 1)
    ref = _mm_exact(A, B)
    got = O.matmul(A, B)
    for i in range(M):
        for j in range(N):
            # bf16 x bf16 products are exact in fp64; only the K-term sum rounds.
            assert abs(Fraction(float(got[i, j])) - ref[i][j]) <= Fraction(K) * Fraction(2) ** -52 * (
                abs(ref[i][j]) + 1)


def test_matmul_orientation():
    # A 2x3 times 3x2 with a hand-computed result: catches a transposed operand.
    A = np.array([[1.0, 2.0, 3.0], [4.0, 5.0, 6.0]])
    B = np.array([[7.0, 8.0], [9.0, 10.0], [11.0, 12.0]])
    assert np.array_equal(O.matmul(A, B), np.array([[58.0, 64.0], [139.0, 154.0]]))


# ---------------------------------------------------------------- bias / residual
def test_bias_residual_exact():
    P, R = _small((4, 4), 2, 0), _small((4, 4), 2, 1)
    b = _small((4,), 2, 2)
    got = O.bias_residual(P, b, R, alpha=0.5)
    for i in range(4):
        for j in range(4):
            ref = Fraction(1, 2) * Fraction(float(P[i, j])) + Fraction(float(b[j])) + Fraction(float(R[i, j]))
            assert Fraction(float(got[i, j])) == ref  # small bf16 sums are exact in fp64


# ---------------------------------------------------------------- LayerNorm
def _ln_mp(row, gamma, beta, eps):
    fr = [v if isinstance(v, Fraction) else Fraction(float(v)) for v in row]
    n = len(fr)
    mu = sum(fr) / n
    var = sum((v - mu) ** 2 for v in fr) / n
    rstd = 1 / mpmath.sqrt(mpmath.mpf(var.numerator) / var.denominator + mpmath.mpf(eps))
    out = []
    for j, v in enumerate(fr):
        d = mpmath.mpf((v - mu).numerator) / (v - mu).denominator
        out.append(d * rstd * mpmath.mpf(float(gamma[j])) + mpmath.mpf(float(beta[j])))
    return mu, var, out


def test_layernorm_exact_stats_4x4():
    x = _small((4, 4), 3, 0, std=3.0)
    g = 1.0 + _small((4,), 3, 1, std=0.3)
    b = _small((4,), 3, 2, std=0.3)
    y = O.layernorm(x, g, b, 1e-5)
    mu = O.row_mean(x)
    var = O.row_var(x, mu)
    for i in range(4):
        mu_r, var_r, y_r = _ln_mp(x[i], g, b, 1e-5)
        assert abs(Fraction(float(mu[i])) - mu_r) <= abs(mu_r) * Fraction(1, 10 ** 15) + Fraction(1, 10 ** 300)
        assert abs(Fraction(float(var[i])) - var_r) <= var_r * Fraction(1, 10 ** 14)
        for j in range(4):
            assert abs(float(y[i, j]) - float(y_r[j])) <= 1e-14 * (1 + abs(float(y_r[j])))


def test_layernorm_constant_row_gives_beta():
    x = np.full((3, 64), 1.75)
    beta = _small((64,), 4, 0)
    gamma = 1.0 + _small((64,), 4, 1)
    y = O.layernorm(x, gamma, beta, 1e-5)
    assert np.array_equal(y, np.broadcast_to(beta.astype(np.float64), y.shape))


@pytest.mark.parametrize("a,b,eps", [(3.0, -1.0, 1e-5), (0.125, 0.5, 1e-5), (2.0, 7.0, 0.0)])
def test_layernorm_two_element_closed_form(a, b, eps):
    h = (a - b) / 2.0
    expect = h / math.sqrt(h * h + eps)
    y = O.layernorm(np.array([[a, b]]), np.array([2.0, 2.0]), np.array([3.0, -3.0]), eps)
    assert y[0, 0] == pytest.approx(2.0 * expect + 3.0, rel=1e-15, abs=1e-15)
    assert y[0, 1] == pytest.approx(-2.0 * expect - 3.0, rel=1e-15, abs=1e-15)


def test_layernorm_invariants_identity_affine():
    x = np.random.default_rng(5).standard_normal((64, 768)) * 2.5 + 0.7
    eps = 1e-5
    y = O.layernorm(x, None, None, eps)
    var = x.var(axis=1)  # numpy's own variance routine, not the oracle's
    assert np.max(np.abs(y.mean(axis=1))) <= 1e-12 * np.max(np.abs(y))
    np.testing.assert_allclose((y * y).mean(axis=1), var / (var + eps), rtol=1e-12)
    y0 = O.layernorm(x, None, None, 0.0)
    np.testing.assert_allclose((y0 * y0).mean(axis=1), 1.0, rtol=1e-12)


def test_rmsnorm_closed_form():
    y = O.rmsnorm(np.array([[3.0, 4.0]]), None, 0.0)  # rms = 5/sqrt(2)
    np.testing.assert_allclose(y, [[3.0 * math.sqrt(2) / 5.0, 4.0 * math.sqrt(2) / 5.0]], rtol=1e-15)


@pytest.mark.parametrize("eps", [0.5, 1e-5])
def test_rmsnorm_eps_and_gamma_closed_form(eps):
    # [3, 4]: mean square 12.5, so y = x / sqrt(12.5 + eps) * gamma.  eps = 0.5
    # gives sqrt(13) exactly: eps outside the root (sqrt(12.5) + 0.5), eps
    # added to the sum of squares instead of the mean, or a dropped gamma all
    # move the values by far more than the tolerance.
    g = np.array([2.0, -0.5])
    y = O.rmsnorm(np.array([[3.0, 4.0]]), g, eps)
    r = math.sqrt(12.5 + eps)
    np.testing.assert_allclose(y, [[3.0 / r * 2.0, 4.0 / r * -0.5]], rtol=1e-15)


def _rms_mp(row, gamma, eps):
    fr = [Fraction(float(v)) for v in row]
    ms = sum(v * v for v in fr) / len(fr)   # exact mean square
    r = mpmath.sqrt(mpmath.mpf(ms.numerator) / ms.denominator + mpmath.mpf(eps))
    return [mpmath.mpf(v.numerator) / v.denominator / r * mpmath.mpf(float(gamma[j])) for j, v in enumerate(fr)]


def test_rmsnorm_exact_4x5_with_gamma():
    x = _small((4, 5), 31, 0, std=2.0)
    g = 1.0 + _small((5,), 31, 1, std=0.3)
    y = O.rmsnorm(x, g, 1e-3)
    for i in range(4):
        want = _rms_mp(x[i], g, 1e-3)
        for j in range(5):
            assert abs(float(y[i, j]) - float(want[j])) <= 1e-14 * (1 + abs(float(want[j])))


def test_rmsnorm_invariant_mean_square():
    # gamma = 1: the mean of y^2 is ms / (ms + eps), with ms from numpy's own mean
    x = np.random.default_rng(32).standard_normal((32, 640)) * 1.7
    ms = np.mean(np.square(x), axis=1)
    y = O.rmsnorm(x, None, 0.25)
    np.testing.assert_allclose(np.mean(y * y, axis=1), ms / (ms + 0.25), rtol=1e-13)


# ---------------------------------------------------------------- ReLU
def test_relu_definition_points_and_identities():
    x = np.array([-3.5, -1e-300, -0.0, 0.0, 5e-324, 2.25, 1e300])
    y = O.relu(x)
    assert list(y) == [0.0, 0.0, 0.0, 0.0, 5e-324, 2.25, 1e300]
    assert not np.any(np.signbit(y))            # no negative zero comes out
    v = np.random.default_rng(33).standard_normal(5000) * 10
    np.testing.assert_array_equal(O.relu(v) - O.relu(-v), v)       # odd part is the identity
    np.testing.assert_array_equal(O.relu(v) + O.relu(-v), np.abs(v))


def test_mblr_brute_force():
    # MatMul - BiasAdd - LayerNorm - ReLU (Sec. VI) on 3 x 5, exact product and
    # 40-digit LayerNorm, then max(., 0) by comparison
    X, W = _small((3, 7), 34, 0), _small((7, 5), 34, 1)
    b, g, be = _small((5,), 34, 2, 0.3), 1 + _small((5,), 34, 3, 0.2), _small((5,), 34, 4, 0.2)
    got = O.relu(O.layernorm(O.bias_residual(O.matmul(X, W), b), g, be, 1e-5))
    Pm = _mm_exact(X, W)
    for i in range(3):
        x = [Pm[i][j] + Fraction(float(b[j])) for j in range(5)]
        _, _, y = _ln_mp(x, g, be, 1e-5)
        want = [float(v) if v > 0 else 0.0 for v in y]
        np.testing.assert_allclose(got[i], want, rtol=1e-13, atol=1e-14)


# ---------------------------------------------------------------- GELU
def _golden_cdf():
    rows = []
    with open(os.path.join(GOLDEN, "normal_cdf.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                x, p = line.split()[:2]
                rows.append((float(x), float(p)))
    return rows


def test_gelu_textbook_values():
    for x, phi in _golden_cdf():
        assert O.gelu_erf(np.array([x]))[0] == pytest.approx(x * phi, rel=1e-15, abs=1e-17)


def test_gelu_identities_and_library():
    from scipy.special import ndtr
    x = np.linspace(-8, 8, 4001)
    g = O.gelu_erf(x)
    np.testing.assert_allclose(g - O.gelu_erf(-x), x, rtol=0, atol=1e-14)
    np.testing.assert_allclose(g, x * ndtr(x), rtol=1e-15, atol=1e-15)
    assert O.gelu_erf(np.array([0.0]))[0] == 0.0


def test_gelu_tanh_variant():
    x = np.linspace(-6, 6, 2001)
    gt = O.gelu_tanh(x)
    np.testing.assert_allclose(gt - O.gelu_tanh(-x), x, atol=1e-14)
    c = mpmath.sqrt(2 / mpmath.pi)
    ref = float(mpmath.mpf(0.5) * (1 + mpmath.tanh(c * (1 + mpmath.mpf("0.044715")))))
    assert O.gelu_tanh(np.array([1.0]))[0] == pytest.approx(ref, rel=1e-15)
    diff = np.max(np.abs(gt - O.gelu_erf(x)))
    assert 1e-4 < diff < 1e-3  # the two variants differ by ~5e-4: a swap is visible


# ---------------------------------------------------------------- e4m3
def _golden_e4m3():
    rows = []
    with open(os.path.join(GOLDEN, "e4m3_spec_points.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                c, v = line.split()[:2]
                rows.append((int(c, 16), float(v)))
    return rows


def test_e4m3_decode_spec_points():
    for code, val in _golden_e4m3():
        got = O.e4m3_decode(code)
        if math.isnan(val):
            assert np.isnan(got)
        else:
            assert float(got) == val and math.copysign(1, float(got)) == math.copysign(1, val)


def test_e4m3_decode_exhaustive_vs_torch():
    codes = np.arange(256, dtype=np.uint8)
    ours = O.e4m3_decode(codes)
    theirs = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    nan = np.isnan(theirs)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], theirs[~nan])


def test_e4m3_roundtrip_midpoints_saturation():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    assert np.array_equal(O.e4m3_encode(O.e4m3_decode(codes)), codes)
    pos = O.e4m3_decode(np.arange(0x00, 0x7F))
    mids = (pos[:-1] + pos[1:]) / 2
    enc = O.e4m3_encode(mids).astype(int)
    lo = np.arange(0x00, 0x7E)
    assert np.all(enc == np.where(lo % 2 == 0, lo, lo + 1))   # ties to even mantissa
    assert np.all(O.e4m3_encode(np.array([448.0, 449.0, 464.0, 1e6])) == 0x7E)
    assert np.all(O.e4m3_encode(np.array([-448.0, -1e6])) == 0xFE)
    assert O.e4m3_encode(np.array([np.nan]))[0] == 0x7F


def test_e4m3_encode_vs_torch_in_range():
    x = (np.random.default_rng(9).standard_normal(200000) * 60).astype(np.float32)
    x = np.clip(x, -448, 448)
    x[:1000] *= 1e-3  # subnormal range
    theirs = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(O.e4m3_encode(x), theirs)


# ---------------------------------------------------------------- amax / quant
def test_rowamax_quant_properties():
    z = np.random.default_rng(11).standard_normal((32, 300)) * np.linspace(0.1, 9, 32)[:, None]
    z[5] = 0.0
    s, q = O.rowamax_quant(z)
    dq = O.e4m3_decode(q)
    nz = np.arange(32) != 5
    assert np.all(np.max(np.abs(dq[nz]), axis=1) == 448.0)
    assert s[5] == 0.0 and np.all(q[5] == 0)
    np.testing.assert_allclose(s[nz], np.max(np.abs(z[nz]), axis=1) / 448.0, rtol=0)
    s2, q2 = O.rowamax_quant(-z)
    assert np.array_equal(s2, s)
    assert np.array_equal(q2[nz], q[nz] ^ 0x80)             # sign bit flips, magnitude kept
    s4, q4 = O.rowamax_quant(z * 4.0)          # power-of-two scale: codes unchanged
    assert np.array_equal(q4, q) and np.array_equal(s4, s * 4.0)


# ---------------------------------------------------------------- softmax / attention
def test_softmax_rows_sum_and_shift():
    s = np.random.default_rng(12).standard_normal((16, 333)) * 4
    p = O.softmax_rows(s)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-14)
    np.testing.assert_allclose(O.softmax_rows(s + 123.25), p, rtol=1e-12, atol=1e-300)


# ---------------------------------------------------------------- softcap / MSTS
def test_tanh_softcap_closed_forms():
    cap = 7.5
    # tanh(atanh(1/2)) = 1/2 (math.atanh, not the oracle's np.tanh)
    np.testing.assert_allclose(O.tanh_softcap(np.array([cap * math.atanh(0.5)]), cap), [cap / 2], rtol=1e-15)
    # tanh(1) = (e^2 - 1) / (e^2 + 1)
    e2 = math.exp(2.0)
    np.testing.assert_allclose(O.tanh_softcap(np.array([cap]), cap), [cap * (e2 - 1) / (e2 + 1)], rtol=1e-15)
    x = np.random.default_rng(21).standard_normal(1000) * 40
    y = O.tanh_softcap(x, cap)
    np.testing.assert_array_equal(O.tanh_softcap(-x, cap), -y)                   # odd
    assert np.all(np.abs(y) <= cap) and np.all(np.abs(y) <= np.abs(x))            # bounded, contracting
    z = x * 1e-3 / cap                                                            # |x| << cap: tanh series
    series = z - z ** 3 / 3 + 2 * z ** 5 / 15 - 17 * z ** 7 / 315 + 62 * z ** 9 / 2835
    np.testing.assert_allclose(O.tanh_softcap(z * cap, cap), cap * series, rtol=5e-14, atol=1e-300)


def test_msts_by_hand_and_limits():
    # 2 x 3 logits by hand: x = alpha X.W + b, y = cap tanh(x / cap), softmax of each row
    X = np.array([[1.0, -2.0], [0.5, 0.25]])
    W = np.array([[1.0, 0.0, 2.0], [0.5, -1.0, 0.0]])
    b = np.array([0.1, -0.2, 0.3])
    alpha, cap = 3.0, 2.5
    want = []
    for i in range(2):
        logits = [alpha * (X[i, 0] * W[0, j] + X[i, 1] * W[1, j]) + b[j] for j in range(3)]
        y = [cap * math.tanh(v / cap) for v in logits]
        m = max(y)
        e = [math.exp(v - m) for v in y]
        want.append([v / math.fsum(e) for v in e])
    np.testing.assert_allclose(O.msts(X, W, alpha, b, cap), np.array(want), rtol=1e-14)
    # rows sum to 1; a very large cap leaves the plain softmax of the logits
    rng = np.random.default_rng(22)
    X, W = rng.standard_normal((8, 16)), rng.standard_normal((16, 40)) / 4
    p = O.msts(X, W, 2.0, None, 1e6)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-14)
    np.testing.assert_allclose(p, O.softmax_rows(2.0 * (X @ W)), rtol=1e-9)


def _attn_mp(Q, K, V, scale):
    Lq, Lk, dv = Q.shape[0], K.shape[0], V.shape[1]
    out = np.zeros((Lq, dv))
    for i in range(Lq):
        sc = [mpmath.fsum(mpmath.mpf(float(Q[i, k])) * mpmath.mpf(float(K[j, k])) for k in range(Q.shape[1]))
              * mpmath.mpf(scale) for j in range(Lk)]
        m = max(sc)
        e = [mpmath.exp(v - m) for v in sc]
        l = mpmath.fsum(e)
        for d in range(dv):
            out[i, d] = float(mpmath.fsum(e[j] * mpmath.mpf(float(V[j, d])) for j in range(Lk)) / l)
    return out


def test_attention_brute_force_asymmetric():
    Q, K, V = _small((4, 3), 13, 0), _small((5, 3), 13, 1), _small((5, 2), 13, 2)
    ref = _attn_mp(Q, K, V, 0.7)
    got = O.attention(Q[None], K[None], V[None], 0.7)[0]
    np.testing.assert_allclose(got, ref, rtol=1e-14, atol=1e-15)


def test_attention_special_cases():
    rng = np.random.default_rng(14)
    Q, K, V = rng.standard_normal((2, 8, 16)), rng.standard_normal((2, 12, 16)), rng.standard_normal((2, 12, 16))
    ones = O.attention(Q, K, np.ones_like(V))
    np.testing.assert_allclose(ones, 1.0, rtol=1e-14)
    zq = O.attention(np.zeros_like(Q), K, V)
    np.testing.assert_allclose(zq, np.broadcast_to(V.mean(axis=1, keepdims=True), zq.shape), rtol=1e-13, atol=1e-15)
    one = O.attention(Q, K[:, :1], V[:, :1])
    np.testing.assert_allclose(one, np.broadcast_to(V[:, :1], one.shape), rtol=1e-15)


# ---------------------------------------------------------------- composites
def test_postnorm_end_to_end_brute_force():
    X, W, R = _small((4, 6), 15, 0), _small((6, 4), 15, 1), _small((4, 4), 15, 2)
    b, g, be = _small((4,), 15, 3), 1 + _small((4,), 15, 4, 0.2), _small((4,), 15, 5, 0.2)
    Pm = _mm_exact(X, W)
    got = O.postnorm(X, W, b, R, g, be, 1.0, 1e-5)
    for i in range(4):
        x = [Pm[i][j] + Fraction(float(b[j])) + Fraction(float(R[i, j])) for j in range(4)]
        _, _, y = _ln_mp(x, g, be, 1e-5)
        np.testing.assert_allclose(got[i], [float(v) for v in y], rtol=1e-13, atol=1e-14)


def test_ln_gelu_amax_brute_force():
    X, W, R = _small((3, 8), 16, 0), _small((8, 5), 16, 1), _small((3, 5), 16, 2)
    b = _small((5,), 16, 3, 0.1)
    z, s, q = O.ln_gelu_amax(X, W, b, R, None, None, 1e-5)
    Pm = _mm_exact(X, W)
    for i in range(3):
        x = [Pm[i][j] + Fraction(float(b[j])) + Fraction(float(R[i, j])) for j in range(5)]
        _, _, y = _ln_mp(x, np.ones(5), np.zeros(5), 1e-5)
        zr = [v * mpmath.ncdf(v) for v in y]
        np.testing.assert_allclose(z[i], [float(v) for v in zr], rtol=1e-13, atol=1e-14)
        a = max(abs(v) for v in zr)
        assert s[i] == pytest.approx(float(a / 448), rel=1e-14)
        enc = [int(O.e4m3_encode(np.array([float(v / (a / 448))]))[0]) for v in zr]
        assert list(q[i]) == enc


def test_ffn_special_case_and_brute_force():
    X = _small((6, 8), 17, 0)
    W1, b1 = _small((8, 16), 17, 1, 0.3), _small((16,), 17, 2, 0.05)
    Y = O.ffn_b2b(X, W1, b1, np.zeros((16, 8)), np.zeros(8))
    np.testing.assert_allclose(Y, O.layernorm(X), rtol=1e-15, atol=1e-15)
    W2, b2 = _small((16, 8), 17, 3, 0.3), _small((8,), 17, 4, 0.05)
    Y = O.ffn_b2b(X, W1, b1, W2, b2)
    P = _mm_exact(X, W1)
    for i in range(6):
        h = [mpmath.mpf(P[i][j].numerator) / P[i][j].denominator + mpmath.mpf(float(b1[j])) for j in range(16)]
        h = [v * mpmath.ncdf(v) for v in h]
        u = [mpmath.fsum(h[j] * mpmath.mpf(float(W2[j, c])) for j in range(16)) + mpmath.mpf(float(b2[c]))
             + mpmath.mpf(float(X[i, c])) for c in range(8)]
        mu = mpmath.fsum(u) / 8
        var = mpmath.fsum((v - mu) ** 2 for v in u) / 8
        yr = [(v - mu) / mpmath.sqrt(var + mpmath.mpf(1e-5)) for v in u]
        np.testing.assert_allclose(Y[i], [float(v) for v in yr], rtol=1e-12, atol=1e-13)


def test_rowamax_quant_f32_matches_f64_off_ties():
    # Decided in fp32 or fp64, codes agree except at rounding ties; on random
    # data almost every code must agree, and the scales agree to fp32 rounding.
    z = (np.random.default_rng(21).standard_normal((64, 512)) * 3).astype(np.float32)
    s64, q64 = O.rowamax_quant(z)
    s32, q32 = O.rowamax_quant_f32(z)
    np.testing.assert_allclose(s32, s64, rtol=2 ** -23)
    diff = q32 != q64
    assert diff.mean() < 1e-3
    assert np.all(np.abs(O.e4m3_decode(q32[diff]) - O.e4m3_decode(q64[diff])) <=
                  np.abs(O.e4m3_decode(q64[diff])) * 0.125 + 2 ** -9)
    zero = np.zeros((2, 8), np.float32)
    s, q = O.rowamax_quant_f32(zero)
    assert np.all(s == 0) and np.all(q == 0)


# ---------------------------------------------------------------- B2B MLP (DLRM pattern)
def test_mlp_b2b_brute_force():
    X = _small((4, 6), 40, 0)
    W1, b1 = _small((6, 5), 40, 1, 0.5), _small((5,), 40, 2, 0.3)
    W2, b2 = _small((5, 3), 40, 3, 0.5), _small((3,), 40, 4, 0.3)
    P = _mm_exact(X, W1)
    for out_relu in (False, True):
        got = O.mlp_b2b(X, W1, b1, W2, b2, out_relu=out_relu)
        for i in range(4):
            h = [max(P[i][j] + Fraction(float(b1[j])), Fraction(0)) for j in range(5)]
            for c in range(3):
                o = sum(h[j] * Fraction(float(W2[j, c])) for j in range(5)) + Fraction(float(b2[c]))
                if out_relu:
                    o = max(o, Fraction(0))
                assert abs(float(got[i, c]) - float(o)) <= 1e-14 * (1 + abs(float(o)))


def test_mlp_b2b_special_cases():
    rng = np.random.default_rng(41)
    X, W1, b1 = rng.standard_normal((7, 16)), rng.standard_normal((16, 12)), rng.standard_normal(12)
    W2, b2 = rng.standard_normal((12, 4)), rng.standard_normal(4)
    # W2 = 0: every row is b2 (and ReLU(b2) with the output activation)
    np.testing.assert_array_equal(O.mlp_b2b(X, W1, b1, np.zeros_like(W2), b2), np.broadcast_to(b2, (7, 4)))
    np.testing.assert_array_equal(O.mlp_b2b(X, W1, b1, np.zeros_like(W2), b2, out_relu=True),
                                  np.broadcast_to(np.maximum(b2, 0), (7, 4)))
    # all pre-activations negative: S = 0, O = b2
    np.testing.assert_array_equal(O.mlp_b2b(X, np.zeros_like(W1), -np.abs(b1) - 1, W2, b2), np.broadcast_to(b2, (7, 4)))
    # positive pre-activations: ReLU is the identity, the MLP is linear (associativity, library matmul)
    Xp, W1p, b1p = np.abs(X), np.abs(W1), np.abs(b1)
    np.testing.assert_allclose(O.mlp_b2b(Xp, W1p, b1p, W2, b2), Xp @ (W1p @ W2) + (b1p @ W2 + b2), rtol=1e-12)
    # the partial-sum identity of the N1 split: O = sum over hidden chunks of S_c W2_c
    S = np.maximum(X @ W1 + b1, 0)
    parts = sum(S[:, c:c + 4] @ W2[c:c + 4] for c in range(0, 12, 4))
    np.testing.assert_allclose(O.mlp_b2b(X, W1, b1, W2, b2), parts + b2, rtol=1e-12, atol=1e-12)
