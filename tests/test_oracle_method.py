"""Pins for the oracle's MXNorm / RMSNorm + MX-cast semantics.

What fixes the expected values here (never the oracle itself):
  * the coefficient table of the implementation appendix, re-derived by
    numerical quadrature of Theorem 1's constant c^(p,B);
  * the bound values the paper prints (Sec. 4.3, from Lemmas 1 and 2);
  * blocks worked by hand from Algorithm 2 (tests/golden/hand_blocks.json);
  * closed forms: constant rows, power-of-two rows, zero rows, single-spike
    rows (the equality case of both lemmas);
  * invariants: homogeneity (the scale-family argument of Theorem 1's proof),
    sign symmetry, within-block permutation, the RCEIL code range;
  * the Gaussian calibration of the estimator (Theorem 1 with Gaussian Z).
"""
import json
import math
import os

import numpy as np
import pytest
import torch
from scipy import integrate, special

import oracle
from paper_2603_13180_amd import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def bf16(a):
    return synth.f32_to_bf16_bits(np.asarray(a, np.float32))


def row_with(d, nonzero):
    x = np.zeros((1, d), np.float32)
    for i, v in nonzero.items():
        x[0, int(i)] = v
    return bf16(x)


# ------------------------------------------------------ the coefficient --

def c_quadrature(B, p):
    """Theorem 1: c^(p,B) = (E[max_b |Z_b|^p])^(1/p), Z ~ N(0,1); uses
    E[M^p] = int_0^inf p x^(p-1) P(M > x) dx with P(M <= x) = erf(x/sqrt 2)^B."""
    f = lambda x: p * x ** (p - 1) * (1.0 - special.erf(x / math.sqrt(2.0)) ** B)
    val, _ = integrate.quad(f, 0, np.inf, epsabs=1e-13, epsrel=1e-12, limit=200)
    return val ** (1.0 / p)


def test_coef_table_is_inverse_of_theorem1_constant():
    table = json.load(open(os.path.join(GOLD, "coef_table.json")))["table"]
    for B, p, printed in table:
        assert oracle.coef(B, p) == np.float32(printed)
        # the table is RMS/G = 1/c to four digits (Monte-Carlo), reading R1
        assert abs(printed - 1.0 / c_quadrature(B, p)) < 1e-4, (B, p)


# ------------------------------------------------------- worked blocks --

def test_hand_worked_mxfp8_block():
    g = json.load(open(os.path.join(GOLD, "hand_blocks.json")))["mxfp8"]
    x = row_with(g["d"], g["nonzero"])
    codes, scales, r32, _ = oracle.mxnorm_mxfp8(x, p=g["p"], eps=g["eps"], mode=g["mode"])
    assert abs(r32[0] - g["rho"]) < 1e-6
    assert scales[0].tolist() == g["scales"]
    want = np.zeros(g["d"], np.uint8)
    for i, c in g["codes_nonzero"].items():
        want[int(i)] = c
    assert np.array_equal(codes[0], want)


def test_hand_worked_nvfp4_block():
    g = json.load(open(os.path.join(GOLD, "hand_blocks.json")))["nvfp4"]
    x = row_with(g["d"], g["nonzero"])
    s_g = float(np.float32(math.sqrt(2) / 0.4688 / 2688))
    codes, scales, r32, _ = oracle.mxnorm_nvfp4(x, s_g, p=g["p"], eps=g["eps"])
    assert abs(r32[0] - g["rho"]) < 1e-6
    assert scales[0].tolist() == g["scales"]
    want = np.zeros(g["d"] // 2, np.uint8)
    for i, c in g["packed_nonzero"].items():
        want[int(i)] = c
    assert np.array_equal(codes[0], want)


# ---------------------------------------------------------- closed forms --

@pytest.mark.parametrize("c", [1.0, -3.0, 0.15625, 1000.0])
@pytest.mark.parametrize("p,code", [(2, 0x7A), (1, 0x79)])
def test_constant_rows(c, p, code):
    # x == c: every m~ = |c|, G_p = |c|, rho~ = 1/(coef |c|).  Then
    # t = 1/coef = 2.3895 (p=2) or 2.3469 (p=1); a in (1.75, 3.5] -> e = -7,
    # byte 120; v = t * 128 = 305.9 -> 320 = 1.25*2^8 (0x7A) for p=2, and
    # 300.4 -> 288 = 1.125*2^8 (0x79) for p=1.
    x = bf16(np.full((3, 256), c))
    codes, scales, r32, _ = oracle.mxnorm_mxfp8(x, p=p, eps=0.0)
    coef = oracle.coef(32, p)
    assert np.allclose(r32, 1.0 / (coef * abs(c)), rtol=2e-7)
    assert np.all(scales == 120)
    assert np.all(codes == (code | (0x80 if c < 0 else 0)))


def test_constant_row_nvfp4_default_global_scale():
    # d = 4096, B = 16, p = 2: s_g = 16/0.4688/2688; t = 1/coef; q = t/(6 s_g)
    # = 2688/96 = 28 -> E4M3 28 = 1.75*2^4 = 0x5E; v = t/(28 s_g) = 6 -> 0x7.
    d = 4096
    s_g = float(np.float32(oracle.mxnorm_default_global_scale(d, 16, 2)))
    assert abs(s_g - 16 / 0.4688 / 2688) < 1e-9
    x = bf16(np.full((2, d), 0.75))
    codes, scales, _, _ = oracle.mxnorm_nvfp4(x, s_g, p=2, eps=0.0)
    assert np.all(scales == 0x5E)
    assert np.all(codes == 0x77)


def test_power_of_two_rows_are_homogeneous():
    # every block absmax is 2^j -> rho~ = 2^-j / coef up to one rounding
    rng = np.random.default_rng(11)
    base = rng.standard_normal((4, 512)).astype(np.float32)
    base = np.clip(base, -0.9, 0.9)
    base[:, ::32] = 1.0                       # block absmax exactly 1
    for j in (-20, -3, 0, 5, 40):
        x = bf16(base * np.float32(2.0 ** j))
        c0, s0, r0, _ = oracle.mxnorm_mxfp8(bf16(base), eps=0.0)
        c1, s1, r1, _ = oracle.mxnorm_mxfp8(x, eps=0.0)
        assert np.allclose(r1, 2.0 ** -j / oracle.coef(32, 2), rtol=1.2e-7)
        assert np.array_equal(c0, c1) and np.array_equal(s0, s1)


def test_zero_rows():
    x = bf16(np.zeros((2, 128)))
    x[1] = 0x8000                              # -0.0 everywhere
    codes, scales, r32, _ = oracle.mxnorm_mxfp8(x, eps=1e-6)
    assert np.allclose(r32, 1000.0, rtol=1e-6)
    assert np.all(scales == 0) and np.all(codes[0] == 0) and np.all(codes[1] == 0x80)
    codes, scales, r32, _ = oracle.mxnorm_mxfp8(x, eps=0.0)
    assert np.all(r32 == 0.0) and np.all(scales == 0)
    codes, scales, r32, _ = oracle.rmsnorm_mxfp8(x, eps=0.0)
    assert np.all(r32 == 0.0) and np.all(scales == 0)


# ------------------------------------------------------------- lemmas --

def test_single_spike_reaches_printed_lemma2_bounds():
    g = json.load(open(os.path.join(GOLD, "lemma2_bounds.json")))
    d = g["d"]
    x = row_with(d, {"77": 3.0})
    for p, printed in ((2, g["mxnorm_p2"]), (1, g["mxnorm_p1"])):
        _, _, r32, r64 = oracle.mxnorm_nvfp4(x, 1.0, p=p, eps=0.0)
        assert round(3.0 * r64[0], 2) == printed
    _, _, r32, r64 = oracle.rmsnorm_nvfp4(x, 1.0, eps=0.0)
    assert abs(3.0 * r64[0] - g["rmsnorm"]) < 1e-12


def test_lemma_bounds_hold_on_random_rows():
    rng = np.random.default_rng(12)
    for d in (256, 768, 4096):
        x = rng.standard_t(2, (64, d)).astype(np.float32)
        xb = bf16(x)
        xf = synth.bf16_bits_to_f32(xb).astype(np.float64)
        K = d // 32
        for p in (1, 2):
            _, _, _, r64 = oracle.mxnorm_mxfp8(xb, p=p, eps=0.0)
            bound = (K ** (1.0 / p)) / oracle.coef(32, p)
            assert np.all(np.abs(xf).max(1) * r64 <= bound * (1 + 1e-12))
        _, _, _, r64 = oracle.rmsnorm_mxfp8(xb, eps=0.0)
        assert np.all(np.abs(xf).max(1) * r64 <= math.sqrt(d) * (1 + 1e-12))


# ----------------------------------------------------------- invariants --

def test_sign_flip_and_permutation():
    rng = np.random.default_rng(13)
    x = bf16(rng.standard_normal((8, 1024)))
    c, s, r, _ = oracle.mxnorm_mxfp8(x)
    cn, sn, rn, _ = oracle.mxnorm_mxfp8(x ^ np.uint16(0x8000))
    assert np.array_equal(s, sn) and np.array_equal(r, rn)
    assert np.array_equal(cn, c ^ np.uint8(0x80))
    perm = np.concatenate([rng.permutation(32) + 32 * k for k in range(32)])
    cp, sp, rp, _ = oracle.mxnorm_mxfp8(x[:, perm])
    assert np.array_equal(sp, s) and np.array_equal(rp, r)
    assert np.array_equal(cp, c[:, perm])


def test_rceil_block_maximum_code_range_and_floor_saturation():
    rng = np.random.default_rng(14)
    x = bf16(rng.standard_normal((32, 2048)) * np.exp(rng.uniform(-8, 8, (32, 1))))
    codes, scales, _, _ = oracle.mxnorm_mxfp8(x, mode="rceil")
    vals = np.abs(oracle.e4m3_value(np.arange(256, dtype=np.uint8))[codes])
    bmax = vals.reshape(32, -1, 32).max(-1)
    # a 2^-e lies in (224, 448]; rounding to E4M3 can bring it down to 224
    assert np.all((bmax >= 224) & (bmax <= 448))
    codes, _, _, _ = oracle.mxnorm_mxfp8(x, mode="floor")
    vals = np.abs(oracle.e4m3_value(np.arange(256, dtype=np.uint8))[codes])
    bmax = vals.reshape(32, -1, 32).max(-1)
    assert np.all((bmax >= 256) & (bmax <= 448))


def test_cast_stage_reduces_to_plain_mx_cast():
    # Alg. 2's scale comes from a = RN(m~ rho~); by monotonicity that is
    # max_b |RN(x rho~)|, so the whole cast equals the plain MX cast
    # (eq. blockscale / blockvals) of t = RN32(x rho~).  The RMSNorm baseline
    # without gain is likewise the plain cast of RN32(x rho).
    rng = np.random.default_rng(15)
    x = bf16(rng.standard_normal((16, 768)) * 3)
    xf = synth.bf16_bits_to_f32(x)
    for mode in ("rceil", "floor"):
        c, s, r32, _ = oracle.mxnorm_mxfp8(x, mode=mode)
        c2, s2 = oracle.mxcast_mxfp8((xf * r32[:, None]).astype(np.float32), mode=mode)
        assert np.array_equal(c, c2) and np.array_equal(s, s2)
        c, s, r32, _ = oracle.rmsnorm_mxfp8(x, mode=mode)
        c2, s2 = oracle.mxcast_mxfp8((xf * r32[:, None]).astype(np.float32), mode=mode)
        assert np.array_equal(c, c2) and np.array_equal(s, s2)


def test_plain_cast_values_are_nearest_e4m3_by_torch():
    # with the scale fixed, each code is the nearest E4M3 value of y / 2^e;
    # checked against PyTorch's own float8_e4m3fn conversion
    rng = np.random.default_rng(16)
    y = (rng.standard_normal((8, 256)) * 5).astype(np.float32)
    codes, scales = oracle.mxcast_mxfp8(y)
    e = scales.astype(np.int32) - 127
    v = (y.reshape(8, -1, 32) * np.exp2(-e)[..., None].astype(np.float32)).reshape(8, 256)
    ref = torch.from_numpy(v.astype(np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(codes, ref)


def test_gain_applied_after_normalisation():
    # eq. (gain): y = rho x gamma; gamma = 2 doubles every value, so the
    # scale byte moves up by one and the codes are unchanged
    rng = np.random.default_rng(17)
    x = bf16(rng.standard_normal((4, 512)))
    g1 = bf16(np.ones(512))
    g2 = bf16(np.full(512, 2.0))
    c1, s1, _, _ = oracle.rmsnorm_mxfp8(x, g1)
    c2, s2, _, _ = oracle.rmsnorm_mxfp8(x, g2)
    c0, s0, _, _ = oracle.rmsnorm_mxfp8(x, None)
    assert np.array_equal(c1, c0) and np.array_equal(s1, s0)
    assert np.array_equal(c2, c1) and np.array_equal(s2, s1 + 1)


def test_non_finite_rows():
    x = bf16(np.ones((3, 64)))
    x[0, 5] = 0x7FC0                          # NaN
    x[1, 40] = 0x7F80                         # +Inf in block 1
    x[2, 3] = 0xFF80                          # -Inf in block 0
    x[2, 1] = 0xBF80                          # -1.0
    codes, scales, r32, _ = oracle.mxnorm_mxfp8(x, eps=1e-6)
    assert np.isnan(r32[0]) and np.all(scales[0] == 0xFF) and np.all(codes[0] == 0x7F)
    # Inf: sum of squares is Inf -> rho~ = 0; the Inf block's a = Inf*0 = NaN
    assert r32[1] == 0.0 and scales[1].tolist() == [0x00, 0xFF]
    assert np.all(codes[1, :32] == 0x00) and np.all(codes[1, 32:] == 0x7F)
    assert scales[2].tolist() == [0xFF, 0x00]
    assert codes[2, 3] == 0xFF and codes[2, 1] == 0xFF and codes[2, 0] == 0x7F
    assert np.all(codes[2, 32:] == 0x00)


# ------------------------------------------------ epsilon (reading R3) --

@pytest.mark.parametrize("eps", [1e-6, 1e-2])
def test_rmsnorm_epsilon_matches_torch_rms_norm(eps):
    # The baseline's rho against torch's own RMSNorm (a separate
    # implementation): y = x (mean x^2 + eps)^(-1/2), so rho = y / x.  Rows
    # of magnitude 1e-4 .. 1 put mean x^2 below, near and above eps, where
    # eps added to the RMS, to the sum or after the inversion would differ.
    rng = np.random.default_rng(23)
    mags = np.array([1e-4, 3e-4, 1e-3, 3e-3, 1e-2, 0.1, 1.0])
    x = bf16(rng.standard_normal((len(mags), 256)) * mags[:, None])
    _, _, r32, r64 = oracle.rmsnorm_mxfp8(x, None, eps=eps)
    xf = torch.from_numpy(synth.bf16_bits_to_f32(x).astype(np.float64))
    # the boundary's eps is a float32 argument
    y = torch.nn.functional.rms_norm(xf, (256,), eps=float(np.float32(eps)))
    nz = xf != 0
    want = (y[nz] / xf[nz]).reshape(len(mags), -1)[:, 0].numpy()
    assert np.allclose(r64, want, rtol=1e-12, atol=0)
    assert np.array_equal(r32, r64.astype(np.float32))


# --------------------------------------------------------- calibration --

@pytest.mark.parametrize("d", [2048, 4096])
def test_gaussian_calibration(d):
    # Theorem 1 with Gaussian Z: rho~ / rho -> 1 as K grows; a coef used the
    # wrong way round would give about coef^2 = 0.175 instead
    x = synth.gaussian(2048, d, seed=d)
    _, _, _, rt = oracle.mxnorm_mxfp8(x, eps=0.0)
    _, _, _, rr = oracle.rmsnorm_mxfp8(x, eps=0.0)
    ratio = rt / rr
    assert abs(ratio.mean() - 1.0) < 0.005
    assert ratio.std() < 0.03


def test_dequantised_mxnorm_tracks_rmsnorm():
    # Sec. 3.6: the dequantised MXNorm output approximates RMSNorm + MXCast,
    # with r^2 close to 1 for a few dozen blocks or more
    x = synth.gaussian(256, 2048, seed=3)
    lut = oracle.e4m3_value(np.arange(256, dtype=np.uint8))
    def deq(codes, scales):
        return (lut[codes].reshape(256, -1, 32) *
                oracle.e8m0_value(np.arange(256, dtype=np.uint8))[scales][..., None]).reshape(256, -1)
    a = deq(*oracle.mxnorm_mxfp8(x)[:2])
    b = deq(*oracle.rmsnorm_mxfp8(x)[:2])
    r2 = 1 - ((a - b) ** 2).sum() / ((b - b.mean()) ** 2).sum()
    assert r2 > 0.99
