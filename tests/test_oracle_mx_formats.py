"""Pins for the oracle's generic MX cast: block sizes 16, 32, 64 and E4M3 or
E2M1 elements with E8M0 scales (the block size and element dtype are
parameters of the paper's mx_quantise / mx_norm).  The values come from the
fp32-division RCEIL recipe, hand-worked blocks, closed forms, Lemma 2 and the
Gaussian calibration -- never from the oracle itself."""
import json
import math
import os

import numpy as np
import pytest

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


def rceil_recipe(a, maxval):
    desc = (a.astype(np.float32) / np.float32(maxval)).astype(np.float32)
    bits = desc.view(np.uint32)
    exp = ((bits >> 23) & 0xFF).astype(np.int64) - 127 + ((bits & 0x7FFFFF) != 0)
    return np.clip(exp, -127, 127)


def test_e2m1_rceil_matches_fp32_division_recipe():
    sig = np.arange(0, 1 << 23, dtype=np.uint32)
    parts = [((np.uint32(127 + E) << 23) | sig).view(np.float32) for E in (-5, 1, 9)]
    rng = np.random.default_rng(31)
    parts.append(rng.integers(0x00800000, 0x7F000000, 400_000, dtype=np.uint32).view(np.float32))
    a = np.concatenate(parts)
    a = a[(a / 6.0 >= 2.0 ** -126) & (a / 6.0 < 2.0 ** 127)]
    assert np.array_equal(oracle.scale_exponent(a, "rceil", "e2m1"), rceil_recipe(a, 6.0))


def test_e2m1_scale_ranges():
    rng = np.random.default_rng(32)
    a = np.exp2(rng.uniform(-100, 100, 100_000)).astype(np.float32)
    e = oracle.scale_exponent(a, "rceil", "e2m1").astype(np.float64)
    v = a * np.exp2(-e)
    assert np.all((v > 3.0) & (v <= 6.0))
    e = oracle.scale_exponent(a, "floor", "e2m1").astype(np.float64)
    v = a * np.exp2(-e)
    assert np.all((v >= 4.0) & (v < 8.0))
    edge = np.array([6.0, np.nextafter(np.float32(6), np.float32(7)), 3.0, 1.0, 0.0], np.float32)
    assert oracle.scale_exponent(edge, "rceil", "e2m1").tolist() == [0, 1, -1, -2, -127]
    assert oracle.scale_exponent(edge, "floor", "e2m1").tolist() == [0, 0, -1, -2, -127]


def test_hand_worked_mxfp4_block():
    g = json.load(open(os.path.join(GOLD, "hand_blocks_mx.json")))["mxfp4_b32"]
    codes, scales, r32, _ = oracle.mxnorm_mx(row_with(g["d"], g["nonzero"]), B=g["B"],
                                             elem=g["elem"], p=g["p"], eps=g["eps"])
    assert abs(r32[0] - g["rho"]) < 1e-6
    assert scales[0].tolist() == g["scales"]
    want = np.zeros(g["d"] // 2, np.uint8)
    for i, c in g["packed_nonzero"].items():
        want[int(i)] = c
    assert np.array_equal(codes[0], want)


def test_hand_worked_b64_block():
    g = json.load(open(os.path.join(GOLD, "hand_blocks_mx.json")))["mxfp8_b64"]
    codes, scales, r32, _ = oracle.mxnorm_mx(row_with(g["d"], g["nonzero"]), B=g["B"],
                                             elem=g["elem"], p=g["p"], eps=g["eps"])
    assert abs(r32[0] - g["rho"]) < 1e-6
    assert scales[0].tolist() == g["scales"]
    want = np.zeros(g["d"], np.uint8)
    for i, c in g["codes_nonzero"].items():
        want[int(i)] = c
    assert np.array_equal(codes[0], want)


# x == c: rho~ = 1/(coef |c|), t = 1/coef.  E4M3 (RCEIL): t in (1.75, 3.5] ->
# e = -7, byte 120, v = 128 t.  E2M1: t in (1.5, 3] -> e = -1, byte 126,
# v = 2 t.  B=16: t = 2.1331 -> v = 273.04 -> 288 (0x79) | 4.266 -> 4 (6);
# B=32: 2.3895 -> 305.85 -> 320 (0x7A) | 4.779 -> 4 (6);
# B=64: 2.6295 -> 336.58 -> 352 (0x7B) | 5.259 -> 6 (7).
@pytest.mark.parametrize("B,e4m3_code,e2m1_code", [(16, 0x79, 6), (32, 0x7A, 6), (64, 0x7B, 7)])
@pytest.mark.parametrize("c", [1.0, -0.3])
def test_constant_rows(B, e4m3_code, e2m1_code, c):
    x = bf16(np.full((2, 256), c))
    neg = c < 0
    codes, scales, _, _ = oracle.mxnorm_mx(x, B=B, elem="e4m3", eps=0.0)
    assert np.all(scales == 120) and np.all(codes == (e4m3_code | (0x80 if neg else 0)))
    codes, scales, _, _ = oracle.mxnorm_mx(x, B=B, elem="e2m1", eps=0.0)
    nib = e2m1_code | (0x8 if neg else 0)
    assert np.all(scales == 126) and np.all(codes == (nib | (nib << 4)))


@pytest.mark.parametrize("B", [16, 32, 64])
def test_single_spike_reaches_lemma2_bound(B):
    d = 1024
    K = d // B
    x = row_with(d, {"100": -5.0})
    for p in (1, 2):
        _, _, _, r64 = oracle.mxnorm_mx(x, B=B, p=p, eps=0.0)
        bound = K ** (1.0 / p) / oracle.coef(B, p)
        assert abs(5.0 * r64[0] - bound) <= 1e-9 * bound


@pytest.mark.parametrize("B", [16, 64])
def test_gaussian_calibration_other_block_sizes(B):
    x = synth.gaussian(2048, 4096, seed=B)
    _, _, _, rt = oracle.mxnorm_mx(x, B=B, eps=0.0)
    _, _, _, rr = oracle.rmsnorm_mx(x, B=B, eps=0.0)
    assert abs((rt / rr).mean() - 1.0) < 0.01


@pytest.mark.parametrize("B", [16, 32, 64])
@pytest.mark.parametrize("elem", ["e4m3", "e2m1"])
@pytest.mark.parametrize("mode", ["rceil", "floor"])
def test_cast_stage_reduces_to_plain_mx_cast(B, elem, mode):
    rng = np.random.default_rng(B)
    x = bf16(rng.standard_normal((8, 512)) * np.exp(rng.uniform(-4, 4, (8, 1))))
    xf = synth.bf16_bits_to_f32(x)
    c, s, r32, _ = oracle.mxnorm_mx(x, B=B, elem=elem, mode=mode)
    c2, s2 = oracle.mxcast((xf * r32[:, None]).astype(np.float32), B=B, elem=elem, mode=mode)
    assert np.array_equal(c, c2) and np.array_equal(s, s2)
    c, s, r32, _ = oracle.rmsnorm_mx(x, B=B, elem=elem, mode=mode)
    c2, s2 = oracle.mxcast((xf * r32[:, None]).astype(np.float32), B=B, elem=elem, mode=mode)
    assert np.array_equal(c, c2) and np.array_equal(s, s2)


def test_mxfp4_code_range_sign_and_nan():
    rng = np.random.default_rng(33)
    x = bf16(rng.standard_normal((16, 1024)))
    codes, scales, _, _ = oracle.mxnorm_mx(x, B=32, elem="e2m1")
    lut = oracle.e2m1_value(np.arange(16, dtype=np.uint8))
    nib = np.stack([codes & 0xF, codes >> 4], -1).reshape(16, -1)
    bmax = np.abs(lut[nib]).reshape(16, -1, 32).max(-1)
    assert np.all((bmax >= 3.0) & (bmax <= 6.0))        # a 2^-e in (3, 6]
    cn, sn, _, _ = oracle.mxnorm_mx(x ^ np.uint16(0x8000), B=32, elem="e2m1")
    assert np.array_equal(sn, scales) and np.array_equal(cn, codes ^ np.uint8(0x88))
    y = x.copy()
    y[0, 40] = 0x7FC0
    y[1, 3] = 0xFF80
    c, s, r, _ = oracle.mxnorm_mx(y, B=32, elem="e2m1")
    assert np.all(s[0] == 0xFF) and np.all((c[0] & 0x77) == 0x77)
    assert s[1, 0] == 0xFF and np.all(s[1, 1:] == 0) and r[1] == 0.0


def test_mxfp8_b32_generic_equals_specialised():
    x = synth.gaussian(40, 768, seed=34)
    a = oracle.mxnorm_mx(x, B=32, elem="e4m3")
    b = oracle.mxnorm_mxfp8(x)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)


@pytest.mark.parametrize("B", [16, 32, 64])
@pytest.mark.parametrize("elem", ["e4m3", "e2m1"])
@pytest.mark.parametrize("mode", ["rceil", "floor"])
def test_cast_given_rho_is_the_cast_stage(B, elem, mode):
    # with the oracle's own rho it reproduces Algorithm 2 exactly, non-finite
    # and zero rows included; with any other rho it is the plain MX cast of
    # RN32(x rho), itself pinned above and in the codec tests
    rng = np.random.default_rng(B + len(elem) + len(mode))
    x = bf16(rng.standard_normal((12, 512)) * np.exp(rng.uniform(-6, 6, (12, 1))))
    x[3] = 0
    x[4, 7] = 0x7FC0                      # NaN
    x[5, 100] = 0xFF80                    # -Inf
    x[6] = bf16(np.full(512, 2.5))
    c, s, r32, _ = oracle.mxnorm_mx(x, B=B, elem=elem, mode=mode)
    c2, s2 = oracle.cast_given_rho(x, r32, B=B, elem=elem, mode=mode)
    assert np.array_equal(c, c2) and np.array_equal(s, s2)
    fin = np.isfinite(synth.bf16_bits_to_f32(x)).all(1)
    rho = np.nextafter(r32, np.float32(np.inf)) * np.float32(3.0)
    c3, s3 = oracle.cast_given_rho(x[fin], rho[fin], B=B, elem=elem, mode=mode)
    xf = synth.bf16_bits_to_f32(x[fin])
    c4, s4 = oracle.mxcast((xf * rho[fin][:, None]).astype(np.float32), B=B, elem=elem, mode=mode)
    assert np.array_equal(c3, c4) and np.array_equal(s3, s4)
