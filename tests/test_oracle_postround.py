"""Pins for the oracle's post-round MXNorm (the post-round appendix): the
series f(sigma) = E[max_i r(|X_i|)] against Monte Carlo (which also pins the
reading of the appendix's reversed difference), its homogeneity and
monotonicity, the exact and tabulated inverses, calibration on Gaussian
rows, and the special rows."""
import numpy as np
import pytest

import oracle
from paper_2603_13180_amd import synth


@pytest.mark.parametrize("B", [16, 32, 64])
@pytest.mark.parametrize("sigma", [0.37, 1.0, 5.3])
def test_f_matches_monte_carlo(B, sigma):
    rng = np.random.default_rng(B * 7 + int(sigma * 100))
    n = 200000
    m = np.abs(rng.standard_normal((n, B)) * sigma).max(axis=1)
    r = 2.0 ** np.floor(np.log2(m))
    se = r.std() / np.sqrt(n)
    assert abs(oracle.postround_f(sigma, B) - r.mean()) <= 4 * se


@pytest.mark.parametrize("B", [16, 32, 64])
def test_f_homogeneous_and_increasing(B):
    base = [0.61, 0.83, 1.0, 1.37]
    for s in base:
        f1 = oracle.postround_f(s, B)
        for k in range(-3, 4):
            assert oracle.postround_f(s * 2.0 ** k, B) == pytest.approx(f1 * 2.0 ** k, rel=1e-12)
    grid = np.linspace(0.5, 2.0, 301)
    vals = np.array([oracle.postround_f(s, B) for s in grid])
    assert (np.diff(vals) > 0).all()
    # not the linear function it resembles: f(sigma) / sigma varies with log2 sigma
    ratio = vals / grid
    assert ratio.max() - ratio.min() > 1e-3


@pytest.mark.parametrize("B", [16, 32, 64])
def test_exact_inverse(B):
    for s in (0.3, 0.77, 1.0, 1.9, 12.5):
        assert oracle.postround_finv_exact(oracle.postround_f(s, B), B) == pytest.approx(s, rel=1e-12)


@pytest.mark.parametrize("B", [16, 32, 64])
def test_table_and_its_interpolation(B):
    xs, vs = oracle.postround_lut(B)
    assert xs[0] == 1.0 and xs[-1] == 2.0 and len(xs) == oracle.POSTROUND_A + 1
    assert np.array_equal(xs, np.exp2(np.arange(65) / 64.0).astype(np.float32))
    assert vs[-1] == pytest.approx(2 * vs[0], rel=1e-6)   # f^-1(2) = 2 f^-1(1)
    lut = (xs, vs)
    # linear interpolation of the inverse on a 2^(1/64) grid: within 2e-3 of
    # the exact inverse (worst seen: 4e-5, 1.5e-4, 6.6e-4 for B = 16, 32, 64;
    # the larger the block, the more f curves), also across binades (the
    # 2^k identity); a table off by one point would be ~1.1% off
    for X in np.concatenate([np.linspace(1.0, 2.0, 257)[:-1], [0.013, 0.5, 3.3, 7.999, 1e4]]):
        got = oracle.postround_finv_lut(X, B, lut)
        assert got == pytest.approx(oracle.postround_finv_exact(X, B), rel=2e-3)
    # the table points themselves come back (to the float rounding of v_i)
    for i in (0, 13, 40, 63):
        assert oracle.postround_finv_lut(float(xs[i]), B, lut) == float(vs[i])


@pytest.mark.parametrize("B", [16, 32, 64])
def test_calibrated_on_gaussian_rows(B):
    # sigma varies per row; the estimate tracks each row's sigma
    rng = np.random.default_rng(B)
    T, d = 256, 4096
    sig = np.exp(rng.uniform(-3, 3, T)).astype(np.float32)
    x = synth.f32_to_bf16_bits((rng.standard_normal((T, d)) * sig[:, None]).astype(np.float32))
    _, _, rho, _ = oracle.mxnorm_postround_mx(x, B=B, eps=0.0)
    rms = np.sqrt(np.mean(synth.bf16_bits_to_f32(x).astype(np.float64) ** 2, axis=1))
    ratio = rho.astype(np.float64) * rms
    assert abs(ratio.mean() - 1.0) < 0.01
    assert ratio.std() < 0.08


def test_homogeneous_in_x_and_cast_is_plain_cast():
    x = synth.gaussian(16, 1024, seed=4, scale=0.9)
    c1, s1, r1, g1 = oracle.mxnorm_postround_mx(x, B=32, eps=0.0)
    x2 = synth.f32_to_bf16_bits(synth.bf16_bits_to_f32(x) * np.float32(2.0))
    c2, s2, r2, g2 = oracle.mxnorm_postround_mx(x2, B=32, eps=0.0)
    assert np.array_equal(g2, 2 * g1) and np.array_equal(r2 * 2, r1)
    assert np.array_equal(c1, c2) and np.array_equal(s1, s2)
    # the cast stage is the plain MX cast of RN32(x rho~)
    y = (synth.bf16_bits_to_f32(x) * r1[:, None]).astype(np.float32)
    for elem in ("e4m3", "e2m1"):
        c, s, r, _ = oracle.mxnorm_postround_mx(x, B=32, elem=elem, eps=0.0)
        wc, ws = oracle.mxcast(y, B=32, elem=elem)
        assert np.array_equal(c, wc) and np.array_equal(s, ws)


def test_special_rows():
    d = 256
    rows = np.zeros((4, d), np.uint16)
    rows[1] = synth.f32_to_bf16_bits(np.full(d, -3.0, np.float32))     # constant
    rows[2, 7] = 0x7F80                                                # +Inf
    rows[3, 9] = 0x7FC0                                                # NaN
    _, _, rho, sig = oracle.mxnorm_postround_mx(rows, B=32, eps=0.0)
    assert rho[0] == 0.0 and sig[0] == 0.0                 # zero row (eps = 0)
    xs, vs = oracle.postround_lut(32)
    # constant row: every r(m~) = 2, Xbar = 2, sigma = 2 f^-1(1) = 2 v_0
    assert sig[1] == 2.0 * float(vs[0])
    assert rho[1] == np.float32(1.0 / (2.0 * float(vs[0])))
    assert rho[2] == 0.0 and np.isinf(sig[2])
    assert np.isnan(rho[3])
    _, _, rho_e, _ = oracle.mxnorm_postround_mx(rows[:1], B=32, eps=1e-6)
    assert rho_e[0] == np.float32(1e3)
