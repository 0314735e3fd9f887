"""The hardware scaled conversions the norm/cast kernels use, on every fp32
input of the ranges that matter, against round-to-nearest-even written out.

v_cvt_scalef32_pk_fp8_f32 and v_cvt_scalef32_pk_fp4_f32 (through the test
aid tests/hw_convert.hip) must give, for every fp32 v and scale byte b, the
E4M3 / E2M1 code of v / 2^(b - 127) rounded to nearest, ties to the even
code, with v's sign: the rule the oracle's encoders implement (they are
pinned to it on the CPU).  The reference here is that rule written as a
count of the format's midpoints below |v| / 2^e (midpoints taken from the
oracle's decoded value tables; a value on a midpoint goes to the code with
a zero mantissa bit).  E2M1 saturates at 6; E4M3 is checked below 464, the
point above which the instruction returns NaN (the kernels never pass it
such a value: RCEIL keeps |t / 2^e| <= 448 and FLOOR clamps first).
"""
import ctypes
import os

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhwconvert.so")


@pytest.fixture(scope="module")
def hwc():
    if not torch.cuda.is_available():
        raise RuntimeError("the conversion-instruction test needs a GPU (run it with -m gpu)")
    if not os.path.exists(LIB):
        pytest.fail("tests/libhwconvert.so is missing: run __graft_entry__.build()")
    lib = ctypes.CDLL(LIB)
    for f in (lib.hwc_e4m3, lib.hwc_e2m1):
        f.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint32,
                      ctypes.c_void_p]
        f.restype = ctypes.c_int
    lib.hwc_bf16.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    lib.hwc_bf16.restype = ctypes.c_int
    return lib


def _patterns(field, dev):
    """Every fp32 bit pattern with biased exponent field `field`, positive."""
    sig = torch.arange(1 << 23, dtype=torch.int32, device=dev)
    return (sig | (field << 23)).view(torch.float32)


def _rne(a, values):
    """Code index of a >= 0 on the value table `values` (ascending, code
    order), nearest with ties to the even index; above the last midpoint the
    last code."""
    v = np.asarray(values, np.float64)
    mids_np = (v[:-1] + v[1:]) / 2
    assert np.all(mids_np.astype(np.float32).astype(np.float64) == mids_np)  # exact in fp32
    mids = torch.tensor(mids_np, dtype=torch.float32, device=a.device)
    idx = torch.searchsorted(mids, a, right=False)          # midpoints strictly below a
    on_mid = (idx < mids.numel()) & (a == mids[idx.clamp(max=mids.numel() - 1)])
    return torch.where(on_mid & (idx % 2 == 1), idx + 1, idx).to(torch.uint8)


def _sweep(fn, values, sign_bit, e, fields, limit, dev):
    stream = torch.cuda.current_stream().cuda_stream
    checked = 0
    for field in fields:
        pos = _patterns(field, dev)
        a = pos * (2.0 ** -e)                                # exact: a power of two
        keep = a < limit
        pos, a = pos[keep], a[keep]
        want = _rne(a, values)
        for v, w in ((pos, want), (-pos, want | sign_bit)):
            v = v.contiguous()
            out = torch.empty(v.numel(), dtype=torch.uint8, device=dev)
            rc = fn(v.data_ptr(), out.data_ptr(), v.numel(), 127 + e, stream)
            assert rc == 0
            torch.cuda.synchronize()
            bad = torch.nonzero(out != w)
            if bad.numel():
                i = int(bad[0])
                raise AssertionError("e=%d field=%d v=%r got %#x want %#x" % (
                    e, field, float(v[i]), int(out[i]), int(w[i])))
            checked += v.numel()
    return checked


@pytest.mark.parametrize("e", [0, -7, 5, -127])
def test_e4m3_conversion_every_input(hwc, e):
    dev = torch.device("cuda:0")
    values = oracle.e4m3_value(np.arange(0x7F, dtype=np.uint8))   # codes 0..126 ascending
    # |v| / 2^e from 2^-13 (all round to zero) up to 464; fp32 subnormal
    # inputs (field 0) where the range reaches them
    lo = max(0, 127 - 13 + e)
    hi = 127 + 8 + e
    n = _sweep(hwc.hwc_e4m3, values, 0x80, e, range(lo, hi + 1), 464.0, dev)
    assert n > 100_000_000 if e != -127 else n > 50_000_000


@pytest.mark.parametrize("e", [0, -3, 2, -127])
def test_e2m1_conversion_every_input(hwc, e):
    dev = torch.device("cuda:0")
    values = oracle.e2m1_value(np.arange(8, dtype=np.uint8))      # 0, .5, 1, ..., 6
    # |v| / 2^e from 2^-5 (all round to zero) up to 16 (saturated at 6)
    lo = max(0, 127 - 5 + e)
    hi = 127 + 3 + e
    n = _sweep(hwc.hwc_e2m1, values, 0x8, e, range(lo, hi + 1), 16.0, dev)
    assert n > 50_000_000 if e != -127 else n > 8_000_000


def _bf16_rne_bits(u):
    """float -> bf16 by round to nearest, ties to even, written on the bits:
    add half a bf16 ulp less one, plus the lowest kept bit, then truncate
    (a carry into the exponent is the correct rounding up, up to Inf)."""
    u = u.astype(np.uint64)
    return (((u + 0x7FFF + ((u >> 16) & 1)) >> 16) & 0xFFFF).astype(np.uint16)


def test_bf16_conversion_on_every_rounding_case(hwc):
    # every upper half-word (sign, exponent, the 7 kept mantissa bits) with
    # the lower halves that decide the rounding (0, just above 0, just below
    # and at the tie, just above it, all ones) and random ones; then every
    # lower half under the upper halves of 1.0, the fp32 subnormals, the
    # smallest normal and the largest finite values
    rng = np.random.default_rng(3)
    hi = np.arange(1 << 16, dtype=np.uint32)
    lows = np.concatenate([[0x0000, 0x0001, 0x3FFF, 0x7FFF, 0x8000, 0x8001, 0xBFFF, 0xFFFF],
                           rng.integers(0, 1 << 16, 8)]).astype(np.uint32)
    u1 = ((hi[:, None] << 16) | lows[None, :]).ravel()
    every_low = np.arange(1 << 16, dtype=np.uint32)
    u2 = np.concatenate([(h << 16) | every_low for h in
                         (0x3F80, 0x0000, 0x8000, 0x0080, 0x7F7F, 0xFF7F, 0x4B12)])
    u = np.concatenate([u1, u2]).astype(np.uint32)
    dev = torch.device("cuda:0")
    x = torch.from_numpy(u.view(np.int32)).to(dev).view(torch.float32)
    out = torch.empty(u.size, dtype=torch.int16, device=dev)
    assert hwc.hwc_bf16(x.data_ptr(), out.data_ptr(), u.size,
                        torch.cuda.current_stream().cuda_stream) == 0
    got = out.cpu().numpy().view(np.uint16)
    nan_in = (u & 0x7FFFFFFF) > 0x7F800000
    want = _bf16_rne_bits(u)
    bad = np.nonzero((got != want) & ~nan_in)[0]
    if bad.size:
        i = bad[0]
        raise AssertionError("%d of %d differ, first %#010x: got %#06x want %#06x"
                             % (bad.size, u.size, u[i], got[i], want[i]))
    # NaN in, NaN out
    g = got[nan_in]
    assert ((g & 0x7F80) == 0x7F80).all() and ((g & 0x7F) != 0).all()


def test_bad_arguments_launch_nothing(hwc):
    assert hwc.hwc_e4m3(None, None, 3, 127, None) == -1      # odd n
    assert hwc.hwc_e2m1(None, None, 2, 255, None) == -1      # NaN scale byte
    assert hwc.hwc_e4m3(None, None, 0, 127, None) == 0       # empty
    assert hwc.hwc_bf16(None, None, 5, None) == -1
