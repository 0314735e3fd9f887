"""Pins for the oracle's number-format code (E4M3, E2M1, E8M0 scale rules).

Each check ties the oracle to something outside itself: the formats' published
properties (bias, largest finite value, NaN encoding), PyTorch's independent
float8_e4m3fn conversion (on every fp32 value of the range that matters), a
round-to-nearest-even definition of E2M1 by midpoint counting (likewise on
every fp32 value of its range), the RCEIL rule as implemented with an fp32 division
and a ceil-of-log2 on the exponent bits (the MXFP8 recipe the paper's
experiments use, Sec. 3.2), and hand-listed E2M1 rounding boundaries.
"""
import numpy as np
import pytest
import torch

import oracle

ALL = np.arange(256, dtype=np.uint8)


def f32(bits):
    return np.array(bits, dtype=np.uint32).view(np.float32)


def next_up(x):
    return np.nextafter(np.float32(x), np.float32(np.inf), dtype=np.float32)


def next_down(x):
    return np.nextafter(np.float32(x), np.float32(-np.inf), dtype=np.float32)


# ----------------------------------------------------------------- E4M3 ----

def test_e4m3_decode_matches_format_properties():
    vals = oracle.e4m3_value(ALL)
    # NaN only at S.1111.111 (OCP E4M3 "FN": no infinities)
    assert np.isnan(vals[0x7F]) and np.isnan(vals[0xFF])
    assert np.isnan(vals).sum() == 2
    assert vals[0x7E] == 448.0                  # largest finite, 1.75 * 2^8
    assert vals[0x08] == 2.0 ** -6              # smallest normal
    assert vals[0x01] == 2.0 ** -9              # smallest subnormal
    assert vals[0x07] == 7 * 2.0 ** -9          # largest subnormal
    assert vals[0x38] == 1.0                    # bias 7
    assert vals[0x00] == 0.0 and np.signbit(vals[0x80])
    pos = vals[:0x7F]
    assert np.all(np.diff(pos) > 0), "positive codes must increase strictly"
    assert np.array_equal(vals[0x80:0xFF], -pos)


def test_e4m3_decode_matches_torch_float8():
    ref = torch.from_numpy(ALL.copy()).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    ours = oracle.e4m3_value(ALL)
    finite = ~np.isnan(ref)
    assert np.array_equal(np.isnan(ours), ~finite)
    assert np.array_equal(ours[finite], ref[finite])


def test_e4m3_encode_round_trip_every_code():
    vals = oracle.e4m3_value(ALL).astype(np.float32)
    enc = oracle.e4m3_encode(vals)
    finite = ~np.isnan(vals)
    assert np.array_equal(enc[finite], ALL[finite])
    assert enc[0x7F] & 0x7F == 0x7F and enc[0xFF] & 0x7F == 0x7F


def test_e4m3_midpoints_tie_to_even_and_neighbours_go_nearer():
    vals = oracle.e4m3_value(np.arange(0x7F, dtype=np.uint8))
    for c in range(0x7E):
        lo, hi = vals[c], vals[c + 1]
        mid = np.float32((lo + hi) / 2)          # exact: few significant bits
        assert float(mid) == (lo + hi) / 2
        even = c if c % 2 == 0 else c + 1
        got = oracle.e4m3_encode(np.array([mid, next_down(mid), next_up(mid)], np.float32))
        assert got[0] == even, (c, mid)
        assert got[1] == c and got[2] == c + 1, (c, mid)
        neg = oracle.e4m3_encode(np.array([-mid], np.float32))
        assert neg[0] == (0x80 | even)


def test_e4m3_encode_matches_torch_random_sweep():
    rng = np.random.default_rng(1)
    # log-uniform magnitudes across the whole E4M3 range and below it
    mag = np.exp2(rng.uniform(-14, np.log2(447.9), 400_000)).astype(np.float32)
    sign = np.where(rng.random(mag.size) < 0.5, -1, 1).astype(np.float32)
    v = mag * sign
    # every fp32 value of one binade per exponent near the subnormal boundary
    extra = [np.arange(0x3A800000, 0x3A800000 + (1 << 16), 7, dtype=np.uint32),
             np.arange(0x3C000000, 0x3C000000 + (1 << 16), 5, dtype=np.uint32)]
    v = np.concatenate([v] + [e.view(np.float32) for e in extra])
    ref = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(oracle.e4m3_encode(v), ref)


def test_e4m3_encode_every_fp32_in_range_matches_torch():
    # every positive fp32 bit pattern from 2^-12 (below half the smallest
    # subnormal, 2^-9, everything rounds to zero) up to 464 (above it torch's
    # conversion gives NaN where the oracle saturates), 22 binades, one at a
    # time; negative values on every 7th pattern
    sig = np.arange(1 << 23, dtype=np.uint32)
    for e in range(127 - 12, 127 + 9):
        pos = ((np.uint32(e) << 23) | sig).view(np.float32)
        pos = pos[pos < 464.0]
        for v in (pos, -pos[::7]):
            ref = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
            got = oracle.e4m3_encode(v)
            assert np.array_equal(got, ref), (e, int(np.flatnonzero(got != ref)[0]))


def test_e4m3_saturation_nan_and_signed_zero():
    v = np.array([448.0, next_up(448.0), 464.0, 480.0, 1e30, np.inf, -np.inf, -500.0,
                  np.nan, -0.0, 0.0, -1e-30, 2.0 ** -10, -(2.0 ** -10),
                  next_up(2.0 ** -10), 3 * 2.0 ** -10], np.float32)
    got = oracle.e4m3_encode(v).tolist()
    assert got[:8] == [0x7E, 0x7E, 0x7E, 0x7E, 0x7E, 0x7E, 0xFE, 0xFE]
    assert got[8] & 0x7F == 0x7F
    assert got[9:14] == [0x80, 0x00, 0x80, 0x00, 0x80]   # 2^-10 ties down to 0
    assert got[14] == 0x01
    assert got[15] == 0x02                                # 3*2^-10 ties to even 2*2^-9


# ----------------------------------------------------------------- E2M1 ----

def test_e2m1_decode_table():
    vals = oracle.e2m1_value(np.arange(16, dtype=np.uint8))
    assert vals[:8].tolist() == [0, 0.5, 1, 1.5, 2, 3, 4, 6]
    assert np.array_equal(vals[8:], -vals[:8])
    assert np.signbit(vals[8])


# Boundaries listed by hand from the value set {0, .5, 1, 1.5, 2, 3, 4, 6}:
# a midpoint goes to the code with a zero mantissa bit.
E2M1_CASES = [
    (0.0, 0), (0.25, 0), (0.2500001, 1), (0.5, 1), (0.7499999, 1), (0.75, 2),
    (1.0, 2), (1.25, 2), (1.2500001, 3), (1.5, 3), (1.7499999, 3), (1.75, 4),
    (2.0, 4), (2.5, 4), (2.5000002, 5), (3.0, 5), (3.4999998, 5), (3.5, 6),
    (4.0, 6), (5.0, 6), (5.0000005, 7), (6.0, 7), (7.0, 7), (1e30, 7), (np.inf, 7),
]


@pytest.mark.parametrize("v,code", E2M1_CASES)
def test_e2m1_boundaries(v, code):
    assert oracle.e2m1_encode(np.array([v], np.float32))[0] == code
    assert oracle.e2m1_encode(np.array([-v], np.float32))[0] == (0x8 | code)


def e2m1_rne_by_midpoints(v):
    """Round-to-nearest-even E2M1 magnitude code of |v|, from the definition:
    the number of midpoints of the value set below |v|, with a value on a
    midpoint going to the neighbour whose mantissa bit (the code's low bit)
    is 0; above 6 the largest code (saturation)."""
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0], np.float32)
    a = np.abs(v)
    idx = np.searchsorted(mids, a, side="left")            # midpoints strictly below
    on_mid = (idx < 7) & (a == mids[np.minimum(idx, 6)])
    return np.where(on_mid & (idx % 2 == 1), idx + 1, idx).astype(np.uint8)


def test_e2m1_encode_every_fp32_in_range_matches_rne_definition():
    # every fp32 bit pattern in [2^-4, 16), both signs: below 2^-4 all round
    # to zero and above 6 all saturate (both checked by the boundary cases)
    sig = np.arange(1 << 23, dtype=np.uint32)
    for e in range(127 - 4, 127 + 4):
        pos = ((np.uint32(e) << 23) | sig).view(np.float32)
        want = e2m1_rne_by_midpoints(pos)
        assert np.array_equal(oracle.e2m1_encode(pos), want), e
        assert np.array_equal(oracle.e2m1_encode(-pos), want | np.uint8(8)), e


def test_e2m1_nearest_on_random_values():
    rng = np.random.default_rng(2)
    v = rng.uniform(-7, 7, 200_000).astype(np.float32)
    got = oracle.e2m1_encode(v)
    table = oracle.e2m1_value(np.arange(16, dtype=np.uint8))
    dec = table[got]
    best = np.min(np.abs(np.clip(np.abs(v), 0, 6)[:, None] - table[None, :8]), axis=1)
    assert np.all(np.abs(np.abs(dec) - np.clip(np.abs(v), 0, 6)) == best)
    assert np.all(np.signbit(dec) == np.signbit(v))


# ------------------------------------------------------- E8M0 scale rules --

def rceil_via_fp32_division(a):
    """The MXFP8 recipe's RCEIL: descale = RN32(a / 448); e = ceil(log2 descale)
    read from the fp32 exponent field (+1 when any mantissa bit is set)."""
    desc = (a.astype(np.float32) / np.float32(448.0)).astype(np.float32)
    bits = desc.view(np.uint32)
    exp = ((bits >> 23) & 0xFF).astype(np.int64) - 127
    exp = exp + ((bits & 0x7FFFFF) != 0)
    return np.clip(exp, -127, 127)


def test_rceil_matches_fp32_division_recipe_all_significands():
    # every significand of three binades, plus random normal magnitudes
    sig = np.arange(0, 1 << 23, dtype=np.uint32)
    parts = [((np.uint32(127 + E) << 23) | sig).view(np.float32) for E in (-3, 0, 8)]
    rng = np.random.default_rng(3)
    bits = rng.integers(0x00800000, 0x7F000000, 500_000, dtype=np.uint32)
    parts.append(bits.view(np.float32))
    a = np.concatenate(parts)
    # keep a / 448 a normal fp32 number, where the recipe's bit trick is valid
    a = a[(a / 448.0 >= 2.0 ** -126) & (a / 448.0 < 2.0 ** 127)]
    assert np.array_equal(oracle.scale_exponent(a, "rceil"), rceil_via_fp32_division(a))


def test_rceil_range_property_and_clamps():
    rng = np.random.default_rng(4)
    a = np.exp2(rng.uniform(-110, 120, 200_000)).astype(np.float32)
    e = oracle.scale_exponent(a, "rceil").astype(np.float64)
    scaled = a.astype(np.float64) * np.exp2(-e)
    assert np.all(scaled <= 448.0) and np.all(scaled > 224.0)
    tiny = np.array([0.0, 1e-45, 2.0 ** -126, 2.0 ** -118], np.float32)
    assert oracle.scale_exponent(tiny, "rceil").tolist() == [-127, -127, -127, -126]
    edge = np.array([448.0, next_up(448.0), 224.0, next_up(224.0), 1.0, 1.75], np.float32)
    assert oracle.scale_exponent(edge, "rceil").tolist() == [0, 1, -1, 0, -8, -8]


def test_floor_rule():
    a = np.array([256.0, 511.99997, 512.0, next_down(256.0), 1.0, 0.0, 1e-45,
                  np.finfo(np.float32).max], np.float32)
    assert oracle.scale_exponent(a, "floor").tolist() == [0, 0, 1, -1, -8, -127, -127, 119]
    rng = np.random.default_rng(5)
    a = np.exp2(rng.uniform(-110, 120, 100_000)).astype(np.float32)
    e = oracle.scale_exponent(a, "floor").astype(np.float64)
    scaled = a.astype(np.float64) * np.exp2(-e)
    assert np.all(scaled >= 256.0) and np.all(scaled < 512.0)


def test_e8m0_decode():
    v = oracle.e8m0_value(ALL)
    assert np.isnan(v[255]) and np.isnan(v).sum() == 1
    assert v[127] == 1.0 and v[0] == 2.0 ** -127 and v[254] == 2.0 ** 127
