"""GPU parity: the HIP kernels (called through the C ABI) against the CPU
oracle, element by element, on the same seeded inputs.

Bar (the two-part contract): E8M0 / E4M3 scale bytes and E4M3 / E2M1 codes
bit-exact; the per-row inverse RMS (estimate) bit-equal to the oracle's float
value and within 1e-6 relative of its double value.  Both sides round rho to
float from a double computation; everything deciding a code is float.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from paper_2603_13180_amd import mxnorm, synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
KINDS = ("mxnorm_mxfp8", "rmsnorm_mxfp8", "mxnorm_nvfp4", "rmsnorm_nvfp4")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU parity tests need a GPU (run them with -m gpu on an MI355X)")
    mxnorm.load()


def dev_bf16(xb):
    return torch.from_numpy(np.ascontiguousarray(xb).view(np.int16)).view(torch.bfloat16).to(DEV)


def sg_mxnorm(d, p=2):
    return float(np.float32(oracle.mxnorm_default_global_scale(d, 16, p)))


def sg_rmsnorm(d, gamma_bits=None):
    gmax = 1.0 if gamma_bits is None else float(np.abs(synth.bf16_bits_to_f32(gamma_bits)).max())
    return float(np.float32(oracle.rmsnorm_default_global_scale(d, gmax)))


def run_gpu(kind, xb, gb=None, p=2, eps=1e-6, mode="rceil", coef=0.0, s_g=None):
    x = dev_bf16(xb)
    g = None if gb is None else dev_bf16(gb)
    if kind == "mxnorm_mxfp8":
        out = mxnorm.mxnorm_mxfp8_fwd(x, p=p, coef=coef, eps=eps, scale_mode=mode)
    elif kind == "rmsnorm_mxfp8":
        out = mxnorm.rmsnorm_mxfp8_fwd(x, g, eps=eps, scale_mode=mode)
    elif kind == "mxnorm_nvfp4":
        out = mxnorm.mxnorm_nvfp4_fwd(x, s_g, p=p, coef=coef, eps=eps)
    else:
        out = mxnorm.rmsnorm_nvfp4_fwd(x, g, s_g, eps=eps)
    torch.cuda.synchronize()
    return tuple(t.cpu().numpy() for t in out)


def run_oracle(kind, xb, gb=None, p=2, eps=1e-6, mode="rceil", coef=0.0, s_g=None):
    c = None if coef <= 0 else coef
    if kind == "mxnorm_mxfp8":
        return oracle.mxnorm_mxfp8(xb, p=p, coef_=c, eps=eps, mode=mode)
    if kind == "rmsnorm_mxfp8":
        return oracle.rmsnorm_mxfp8(xb, gb, eps=eps, mode=mode)
    if kind == "mxnorm_nvfp4":
        return oracle.mxnorm_nvfp4(xb, s_g, p=p, coef_=c, eps=eps)
    return oracle.rmsnorm_nvfp4(xb, s_g, gb, eps=eps)


def assert_parity(kind, got, want, ctx=""):
    codes, scales, rho = got
    wc, ws, w32, w64 = want
    bad_s = np.argwhere(scales != ws)
    assert bad_s.size == 0, "%s %s: %d scale bytes differ, first %s: got %d want %d" % (
        kind, ctx, len(bad_s), bad_s[0], scales[tuple(bad_s[0])], ws[tuple(bad_s[0])])
    bad_c = np.argwhere(codes != wc)
    assert bad_c.size == 0, "%s %s: %d codes differ, first %s: got %#x want %#x" % (
        kind, ctx, len(bad_c), bad_c[0], codes[tuple(bad_c[0])], wc[tuple(bad_c[0])])
    same = (rho == w32) | (np.isnan(rho) & np.isnan(w32))
    assert same.all(), "%s %s: rho differs in %d rows" % (kind, ctx, (~same).sum())
    # the relative bound applies where rho is representable in float; a row
    # whose estimate exceeds FLT_MAX (eps = 0, all-subnormal input) is +Inf
    # on both sides, which the bit-equality above already checks
    fin = np.isfinite(w64) & (w64 != 0) & np.isfinite(w32)
    rel = np.abs(rho[fin].astype(np.float64) - w64[fin]) / np.abs(w64[fin])
    assert rel.size == 0 or rel.max() <= 1e-6


def check(kind, xb, gb=None, **kw):
    if "nvfp4" in kind and kw.get("s_g") is None:
        kw["s_g"] = sg_mxnorm(xb.shape[1], kw.get("p", 2)) if kind.startswith("mxnorm") \
            else sg_rmsnorm(xb.shape[1], gb)
    assert_parity(kind, run_gpu(kind, xb, gb, **kw), run_oracle(kind, xb, gb, **kw),
                  "shape=%s %s" % (xb.shape, kw))


# --------------------------------------------------------------- shapes --

SHAPES = [(1, 32), (3, 64), (65, 96), (7, 768), (130, 1024), (33, 1280), (5, 1792),
          (257, 2048), (1000, 4096), (9, 8192), (17, 16384), (3, 32768)]


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("T,d", SHAPES)
def test_shapes(kind, T, d):
    xb = synth.gaussian(T, d, seed=T * 7 + d, scale=1.5)
    gb = synth.f32_to_bf16_bits(np.random.default_rng(d).uniform(0.5, 1.5, d).astype(np.float32))
    check(kind, xb, gb if kind.startswith("rmsnorm") else None)


@pytest.mark.parametrize("kind", ["mxnorm_mxfp8", "mxnorm_nvfp4"])
@pytest.mark.parametrize("p", [1, 2])
@pytest.mark.parametrize("eps", [0.0, 1e-6, 0.5])
def test_p_and_eps(kind, p, eps):
    xb = synth.gaussian(300, 2048, seed=p * 10 + int(eps * 100), scale=0.7)
    check(kind, xb, p=p, eps=eps)


def test_coef_override_and_floor_mode():
    xb = synth.gaussian(200, 1024, seed=21)
    check("mxnorm_mxfp8", xb, coef=0.5)
    check("mxnorm_mxfp8", xb, mode="floor")
    check("rmsnorm_mxfp8", xb, mode="floor")
    gb = synth.f32_to_bf16_bits(np.full(1024, 3.0, np.float32))
    check("rmsnorm_mxfp8", xb, gb, mode="floor")
    check("mxnorm_nvfp4", xb, coef=0.3, s_g=0.01)


def test_rmsnorm_gamma_and_no_gamma():
    xb = synth.gaussian(128, 4096, seed=22)
    gb = synth.f32_to_bf16_bits(np.random.default_rng(3).normal(1, 0.5, 4096).astype(np.float32))
    for kind in ("rmsnorm_mxfp8", "rmsnorm_nvfp4"):
        check(kind, xb, gb)
        check(kind, xb, None)


# ----------------------------------------------------------- edge rows --

def adversarial_rows(d, seed=0):
    rng = np.random.default_rng(seed)
    rows = []
    def f(a):
        with np.errstate(over="ignore"):
            return synth.f32_to_bf16_bits(np.asarray(a, np.float32))
    rows.append(f(rng.standard_normal(d) * np.exp(rng.uniform(-40, 40, d))))   # huge range
    rows.append(f(rng.standard_normal(d) * 1e-39))                              # subnormals
    rows.append(f(np.zeros(d)))                                                 # +0
    rows.append(np.full(d, 0x8000, np.uint16))                                  # -0
    r = f(rng.standard_normal(d)); r[d // 3] = 0x7FC0; rows.append(r)           # NaN
    r = f(rng.standard_normal(d)); r[5] = 0x7F80; rows.append(r)                # +Inf
    r = f(rng.standard_normal(d)); r[d - 1] = 0xFF80; r[0] = 0xFFC1; rows.append(r)  # -Inf, -NaN
    rows.append(f(np.full(d, -2.75)))                                           # constant
    r = np.zeros(d, np.float32); r[d // 2] = 3e38; rows.append(f(r))            # single huge spike
    r = np.zeros(d, np.float32); r[1] = 1e-38; rows.append(f(r))                # single tiny spike
    rows.append(f(np.where(rng.random(d) < 0.5, 448.0, -448.0)))                # +-448
    r = f(rng.standard_normal(d)); r[::7] = 0x0001; rows.append(r)              # min subnormal
    rows.append(f(rng.standard_normal(d) * 3e38))                               # overflowing squares
    rows.append(f(np.exp2(rng.integers(-126, 127, d)).astype(np.float32)))      # powers of two
    return np.stack(rows)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("eps", [0.0, 1e-6])
def test_adversarial_rows(kind, eps):
    for d in (64, 1024, 4096):
        xb = adversarial_rows(d, seed=d)
        gb = synth.f32_to_bf16_bits(np.linspace(-2, 2, d).astype(np.float32)) \
            if kind.startswith("rmsnorm") else None
        kw = dict(eps=eps)
        if "nvfp4" in kind:
            kw["s_g"] = 0.01
        check(kind, xb, gb, **kw)
        if kind.endswith("mxfp8"):
            check(kind, xb, gb, mode="floor", **kw)


def _sum_of_four_squares(n):
    # Lagrange: every natural number is a sum of four squares; small n only
    import math
    for a in range(int(math.isqrt(n)), -1, -1):
        r1 = n - a * a
        for b in range(min(a, int(math.isqrt(r1))), -1, -1):
            r2 = r1 - b * b
            for c in range(min(b, int(math.isqrt(r2))), -1, -1):
                r3 = r2 - c * c
                e = int(math.isqrt(r3))
                if e * e == r3 and e <= c:
                    return [a, b, c, e]
    raise ValueError(n)


def tie_rows(d, block, values, block_max, k, rng, n_rows=8):
    """Rows whose mean square is exactly 4^k, so that with eps = 0 the
    RMSNorm factor is rho = 2^-k exactly and t = x * 2^-k is exact.  Every
    block but the last holds the integer block_max once and otherwise integers
    drawn from `values`; after the block scale those land on the format's
    rounding midpoints.  The last block balances the sum of squares with
    integers <= 256 (exact in bf16)."""
    rows = []
    nb = d // block
    for _ in range(n_rows):
        x = rng.choice(values, d).astype(np.int64)
        for b in range(nb - 1):
            x[b * block + rng.integers(block)] = block_max
        x[-block:] = 0
        x *= rng.choice([-1, 1], d)
        rem = d * 4 ** k - int((x * x).sum())
        assert rem >= 0
        fill = []
        while rem > 65536:
            fill.append(256)
            rem -= 65536
        fill += _sum_of_four_squares(rem)
        assert len(fill) <= block
        x[d - block:d - block + len(fill)] = fill
        assert np.abs(x).max() <= 256 and (x * x).sum() == d * 4 ** k
        rows.append(synth.f32_to_bf16_bits(x.astype(np.float32)))
    return np.stack(rows)


def test_e4m3_ties_through_rmsnorm():
    # mean square 4^5 -> rho = 2^-5, t = x/32.  A block maximum of 31 gives
    # a = 0.96875 -> e = -8 (RCEIL and FLOOR) and v = 8x.  E4M3 values in
    # [128, 256) are spaced by 16, so v = 8 * (odd 17..31) are all midpoints.
    rng = np.random.default_rng(5)
    xb = tie_rows(1024, 32, np.arange(17, 32, 2), 31, 5, rng)
    xf = synth.bf16_bits_to_f32(xb).astype(np.float64)
    assert np.all((xf ** 2).mean(1) == 4.0 ** 5)
    check("rmsnorm_mxfp8", xb, eps=0.0)
    check("rmsnorm_mxfp8", xb, eps=0.0, mode="floor")


def test_e2m1_ties_through_rmsnorm_nvfp4():
    # mean square 4^4 -> rho = 2^-4, t = x/16.  A block maximum of 24 gives
    # a = 1.5; with s_g = 2^-4 (or 2^-8): q = a / (6 s_g) = 4 (or 64), a power
    # of two, so den = dec(S) s_g = 0.25 and v = x/4: x in {1,3,5,7,10,14,20}
    # lands on the E2M1 midpoints {0.25,0.75,1.25,1.75,2.5,3.5,5}.
    rng = np.random.default_rng(6)
    xb = tie_rows(512, 16, np.array([1, 3, 5, 7, 10, 14, 20, 24]), 24, 4, rng)
    check("rmsnorm_nvfp4", xb, eps=0.0, s_g=2.0 ** -4)
    check("rmsnorm_nvfp4", xb, eps=0.0, s_g=2.0 ** -8)


# ---------------------------------------------------- full-size presets --
#
# Every workload preset at its real shape, in the launch configuration the
# bench times: every row of the four d <= 4096 presets, and at the
# [131072, 4096] stress preset 4096 random rows plus every zero and constant
# row, in both scale modes.  The oracle runs over row chunks on threads (its
# C calls release the GIL).

WORKERS = max(1, min(16, os.cpu_count() or 1))


def oracle_rows(fn, x, *args, **kw):
    """fn(x, ...) -> (codes, scales, rho32, rho64), computed over contiguous
    row chunks of x on WORKERS threads and joined."""
    fn(x[:1], *args, **kw)  # load the library before the threads start
    chunks = [c for c in np.array_split(np.arange(len(x)), 4 * WORKERS) if len(c)]
    with ThreadPoolExecutor(WORKERS) as ex:
        parts = list(ex.map(lambda ix: fn(x[ix[0]:ix[-1] + 1], *args, **kw), chunks))
    return tuple(np.concatenate([p[i] for p in parts]) for i in range(4))


def gpu_rows(out, rows=None):
    if rows is None:
        return tuple(t.cpu().numpy() for t in out)
    ri = torch.from_numpy(rows).to(DEV)
    return tuple(t[ri].cpu().numpy() for t in out)


def check_preset(w, x, g, xs, rows, modes, name):
    T, d = w.preset.T, w.preset.d
    if w.preset.fmt == "mxfp8":
        for mode in modes:
            got = gpu_rows(mxnorm.mxnorm_mxfp8_fwd(x, scale_mode=mode), rows)
            assert_parity("mxnorm_mxfp8", got, oracle_rows(oracle.mxnorm_mxfp8, xs, mode=mode),
                          name + " " + mode)
            got = gpu_rows(mxnorm.rmsnorm_mxfp8_fwd(x, g, scale_mode=mode), rows)
            assert_parity("rmsnorm_mxfp8", got,
                          oracle_rows(oracle.rmsnorm_mxfp8, xs, w.gamma, mode=mode),
                          name + " " + mode)
    else:
        s_g = sg_mxnorm(d)
        got = gpu_rows(mxnorm.mxnorm_nvfp4_fwd(x, s_g), rows)
        assert_parity("mxnorm_nvfp4", got, oracle_rows(oracle.mxnorm_nvfp4, xs, s_g), name)
        s_r = sg_rmsnorm(d, w.gamma)
        got = gpu_rows(mxnorm.rmsnorm_nvfp4_fwd(x, g, s_r), rows)
        assert_parity("rmsnorm_nvfp4", got, oracle_rows(oracle.rmsnorm_nvfp4, xs, s_r, w.gamma),
                      name)


@pytest.mark.parametrize("name", ["llama3-125m-d768", "llama3-1b-d2048", "llama3-8b-d4096",
                                  "llama3-8b-d4096-nvfp4"])
def test_full_size_presets_every_row(name):
    w = synth.generate(name)
    check_preset(w, dev_bf16(w.x), dev_bf16(w.gamma), w.x, None, ("rceil", "floor"), name)


def test_stress_preset_every_zero_and_constant_row():
    name = "llama3-8b-longctx-stress"
    w = synth.generate(name)
    P = w.preset
    aux = synth._aux(P, 0)
    zero, const = np.asarray(aux["zero_rows"]), np.asarray(aux["const_rows"])
    assert len(zero) == len(const) == P.T // 100
    rng = np.random.default_rng(7)
    rows = np.array(sorted(set(rng.choice(P.T, 4096, replace=False).tolist())
                           | set(zero.tolist()) | set(const.tolist()) | {0, P.T - 1}))
    xs = np.ascontiguousarray(w.x[rows])
    assert (xs[np.searchsorted(rows, zero)] & 0x7FFF == 0).all()
    check_preset(w, dev_bf16(w.x), dev_bf16(w.gamma), xs, rows, ("rceil", "floor"), name)


# ------------------------------------------------------ two-part contract --
#
# The reading of R7: a kernel's rho within 1e-6 of the oracle's double, and
# its scale bytes and codes bit-exact against the oracle's cast of the
# kernel's own rho.  The tests above demand more (rho bit-equal to the
# oracle's float); this holds the cast stage to its own definition whatever
# rho came out, so a change in the statistic's rounding could not hide a
# cast error behind a rho mismatch, or the other way round.

@pytest.mark.parametrize("B,elem", [(16, "e4m3"), (32, "e4m3"), (64, "e4m3"), (16, "e2m1"),
                                    (32, "e2m1"), (64, "e2m1")])
def test_cast_follows_the_kernels_own_rho(B, elem):
    xs = [synth.generate("llama3-8b-d4096", rows=np.arange(2048)).x,
          adversarial_rows(1024, seed=B), synth.gaussian(333, 2048, seed=B, scale=0.01)]
    for xb in xs:
        x = dev_bf16(xb)
        for mode in ("rceil", "floor"):
            codes, scales, rho = mxnorm.mxnorm_mx_fwd(x, block=B, elem=elem, scale_mode=mode)
            c, sc, r = codes.cpu().numpy(), scales.cpu().numpy(), rho.cpu().numpy()
            wc, ws = oracle.cast_given_rho(xb, r, B=B, elem=elem, mode=mode)
            assert np.array_equal(sc, ws), "scales differ (B=%d %s %s)" % (B, elem, mode)
            assert np.array_equal(c, wc), "codes differ (B=%d %s %s)" % (B, elem, mode)
            _, _, _, r64 = oracle.mxnorm_mx(xb, B=B, elem=elem, mode=mode)
            fin = np.isfinite(r64) & (r64 != 0) & np.isfinite(r)
            assert (np.abs(r[fin] - r64[fin]) <= 1e-6 * np.abs(r64[fin])).all()


# ------------------------------------------------------- buffer hygiene --

def test_canaries_untouched_and_outputs_fully_written():
    T, d = 77, 1280
    xb = synth.gaussian(T, d, seed=9)
    x = dev_bf16(xb)
    pad = 256
    for kind, ncode, nscale in (("mxnorm_mxfp8", T * d, T * d // 32),
                                ("rmsnorm_mxfp8", T * d, T * d // 32),
                                ("mxnorm_nvfp4", T * d // 2, T * d // 16),
                                ("rmsnorm_nvfp4", T * d // 2, T * d // 16)):
        cbuf = torch.full((ncode + 2 * pad,), 0xA5, dtype=torch.uint8, device=DEV)
        sbuf = torch.full((nscale + 2 * pad,), 0xA5, dtype=torch.uint8, device=DEV)
        rbuf = torch.full((T + 2 * pad,), -7.0, dtype=torch.float32, device=DEV)
        codes = cbuf[pad:pad + ncode].view(T, -1)
        scales = sbuf[pad:pad + nscale].view(T, -1)
        rho = rbuf[pad:pad + T]
        if kind == "mxnorm_mxfp8":
            mxnorm.mxnorm_mxfp8_fwd(x, codes=codes, scales=scales, rho=rho)
        elif kind == "rmsnorm_mxfp8":
            mxnorm.rmsnorm_mxfp8_fwd(x, codes=codes, scales=scales, rho=rho)
        elif kind == "mxnorm_nvfp4":
            mxnorm.mxnorm_nvfp4_fwd(x, sg_mxnorm(d), codes=codes, scales=scales, rho=rho)
        else:
            mxnorm.rmsnorm_nvfp4_fwd(x, None, sg_rmsnorm(d), codes=codes, scales=scales, rho=rho)
        torch.cuda.synchronize()
        cb, sb, rb = cbuf.cpu().numpy(), sbuf.cpu().numpy(), rbuf.cpu().numpy()
        assert np.all(cb[:pad] == 0xA5) and np.all(cb[-pad:] == 0xA5), kind
        assert np.all(sb[:pad] == 0xA5) and np.all(sb[-pad:] == 0xA5), kind
        assert np.all(rb[:pad] == -7.0) and np.all(rb[-pad:] == -7.0), kind
        want = run_oracle(kind, xb, s_g=sg_mxnorm(d) if kind == "mxnorm_nvfp4" else sg_rmsnorm(d))
        assert_parity(kind, (codes.cpu().numpy(), scales.cpu().numpy(), rho.cpu().numpy()), want)


def test_empty_input_and_null_rho():
    x = torch.empty(0, 4096, dtype=torch.bfloat16, device=DEV)
    c, s, r = mxnorm.mxnorm_mxfp8_fwd(x)
    assert c.shape == (0, 4096) and s.shape == (0, 128) and r.shape == (0,)
    xb = synth.gaussian(40, 512, seed=4)
    c, s, r = mxnorm.mxnorm_mxfp8_fwd(dev_bf16(xb), want_rho=False)
    torch.cuda.synchronize()
    wc, ws, _, _ = oracle.mxnorm_mxfp8(xb)
    assert r is None and np.array_equal(c.cpu().numpy(), wc) and np.array_equal(s.cpu().numpy(), ws)


def test_side_stream_and_determinism():
    xb = synth.gaussian(333, 4096, seed=10)
    x = dev_bf16(xb)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        a = mxnorm.mxnorm_mxfp8_fwd(x)
        b = mxnorm.mxnorm_mxfp8_fwd(x)
    s.synchronize()
    for u, v in zip(a, b):
        assert torch.equal(u, v)
    assert_parity("mxnorm_mxfp8", tuple(t.cpu().numpy() for t in a), oracle.mxnorm_mxfp8(xb))


def test_device_errors_raise():
    x = torch.zeros(4, 48, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(mxnorm.MXNormError, match="multiple of 32"):
        mxnorm.mxnorm_mxfp8_fwd(x)
    x = torch.zeros(4, 65536, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(mxnorm.MXNormError, match="MX_EUNSUPPORTED"):
        mxnorm.mxnorm_mxfp8_fwd(x)


@pytest.mark.parametrize("offset", [1, 4, 8])
def test_unaligned_scale_pointer(offset):
    # the library picks 16-, 4- or 1-byte scale stores from K and the pointer
    T, d = 50, 4096
    xb = synth.gaussian(T, d, seed=11)
    x = dev_bf16(xb)
    for kind, K in (("mxnorm_mxfp8", d // 32), ("mxnorm_nvfp4", d // 16)):
        buf = torch.full((T * K + 64,), 0xA5, dtype=torch.uint8, device=DEV)
        scales = buf[offset:offset + T * K].view(T, K)
        if kind == "mxnorm_mxfp8":
            c, s, r = mxnorm.mxnorm_mxfp8_fwd(x, scales=scales)
            want = oracle.mxnorm_mxfp8(xb)
        else:
            c, s, r = mxnorm.mxnorm_nvfp4_fwd(x, sg_mxnorm(d), scales=scales)
            want = oracle.mxnorm_nvfp4(xb, sg_mxnorm(d))
        torch.cuda.synchronize()
        b = buf.cpu().numpy()
        assert np.all(b[:offset] == 0xA5) and np.all(b[offset + T * K:] == 0xA5)
        assert_parity(kind, (c.cpu().numpy(), s.cpu().numpy(), r.cpu().numpy()), want)


# the hidden sizes of the paper's kernel sweep: k * 2^r, k in {1,3,5,7}, in [1024, 16384]
SWEEP_D = sorted({k * 2 ** r for k in (1, 3, 5, 7) for r in range(15) if 1024 <= k * 2 ** r <= 16384})


def test_sweep_hidden_sizes_listed():
    assert len(SWEEP_D) == 17 and SWEEP_D[0] == 1024 and SWEEP_D[-1] == 16384


@pytest.mark.parametrize("d", SWEEP_D)
def test_sweep_hidden_sizes(d):
    xb = synth.gaussian(21, d, seed=d + 1)
    for kind in KINDS:
        check(kind, xb)


def test_graph_replay_matches_eager():
    # the sweep times HIP-graph replays; every replay must equal the eager result
    xb = synth.gaussian(300, 2560, seed=12)
    x = dev_bf16(xb)
    eager = [t.clone() for t in mxnorm.mxnorm_mxfp8_fwd(x)]
    codes = torch.empty_like(eager[0]); scales = torch.empty_like(eager[1]); rho = torch.empty_like(eager[2])
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        mxnorm.mxnorm_mxfp8_fwd(x, codes=codes, scales=scales, rho=rho)
    for _ in range(3):
        codes.zero_(); scales.zero_(); rho.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(codes, eager[0]) and torch.equal(scales, eager[1]) and torch.equal(rho, eager[2])
        # eager work between replays
        mxnorm.rmsnorm_mxfp8_fwd(x)
    assert_parity("mxnorm_mxfp8", (codes.cpu().numpy(), scales.cpu().numpy(), rho.cpu().numpy()),
                  oracle.mxnorm_mxfp8(xb))



# ----------------------------------------------------- general MX formats --

MX_FORMATS = [(16, "e4m3"), (32, "e4m3"), (64, "e4m3"), (16, "e2m1"), (32, "e2m1"), (64, "e2m1")]


def check_mx(xb, block, elem, gb=None, mxn=True, **kw):
    x = dev_bf16(xb)
    if mxn:
        got = mxnorm.mxnorm_mx_fwd(x, block=block, elem=elem, **kw)
        c = kw.pop("coef", 0.0)
        want = oracle.mxnorm_mx(xb, B=block, elem=elem, coef_=None if c <= 0 else c,
                                p=kw.get("p", 2), eps=kw.get("eps", 1e-6),
                                mode=kw.get("scale_mode", "rceil"))
    else:
        g = None if gb is None else dev_bf16(gb)
        got = mxnorm.rmsnorm_mx_fwd(x, g, block=block, elem=elem, **kw)
        want = oracle.rmsnorm_mx(xb, gb, B=block, elem=elem, eps=kw.get("eps", 1e-6),
                                 mode=kw.get("scale_mode", "rceil"))
    torch.cuda.synchronize()
    assert_parity("mx B=%d %s %s" % (block, elem, "mxnorm" if mxn else "rmsnorm"),
                  tuple(t.cpu().numpy() for t in got), want, "shape=%s %s" % (xb.shape, kw))


@pytest.mark.parametrize("block,elem", MX_FORMATS)
@pytest.mark.parametrize("T,d", [(3, 64), (65, 192), (130, 1024), (33, 1280), (257, 4096),
                                 (9, 10240), (4, 32768)])
def test_mx_formats_shapes(block, elem, T, d):
    xb = synth.gaussian(T, d, seed=T + d + block, scale=2.0)
    gb = synth.f32_to_bf16_bits(np.random.default_rng(d).uniform(0.5, 1.5, d).astype(np.float32))
    check_mx(xb, block, elem)
    check_mx(xb, block, elem, gb, mxn=False)
    check_mx(xb, block, elem, None, mxn=False)


@pytest.mark.parametrize("block,elem", MX_FORMATS)
def test_mx_formats_modes_p_eps_and_edge_rows(block, elem):
    xb = synth.gaussian(100, 2048, seed=block, scale=0.5)
    for p in (1, 2):
        for eps in (0.0, 1e-6):
            check_mx(xb, block, elem, p=p, eps=eps)
            check_mx(xb, block, elem, p=p, eps=eps, scale_mode="floor")
    check_mx(xb, block, elem, coef=0.77)
    for d in (64, 1024):
        ab = adversarial_rows(d, seed=block + d)
        for mode in ("rceil", "floor"):
            for eps in (0.0, 1e-6):
                check_mx(ab, block, elem, eps=eps, scale_mode=mode)
                check_mx(ab, block, elem, None, mxn=False, eps=eps, scale_mode=mode)


def test_mx_b32_e4m3_equals_mxfp8_entry_point():
    xb = synth.gaussian(77, 4096, seed=3)
    x = dev_bf16(xb)
    a = mxnorm.mxnorm_mx_fwd(x, block=32, elem="e4m3")
    b = mxnorm.mxnorm_mxfp8_fwd(x)
    torch.cuda.synchronize()
    for u, v in zip(a, b):
        assert torch.equal(u, v)


# ------------------------------------------- gain-folded weight cast --

def check_cast(wb, gb, block, elem, mode="rceil"):
    w = dev_bf16(wb)
    g = None if gb is None else dev_bf16(gb)
    codes, scales = mxnorm.mx_cast_fwd(w, g, block=block, elem=elem, scale_mode=mode)
    torch.cuda.synchronize()
    wc, ws = oracle.mxcast_gain(wb, gb, B=block, elem=elem, mode=mode)
    ctx = "cast B=%d %s %s shape=%s gamma=%s" % (block, elem, mode, wb.shape, gb is not None)
    s, c = scales.cpu().numpy(), codes.cpu().numpy()
    bad = np.argwhere(s != ws)
    assert bad.size == 0, "%s: %d scale bytes differ, first %s" % (ctx, len(bad), bad[0])
    bad = np.argwhere(c != wc)
    assert bad.size == 0, "%s: %d codes differ, first %s" % (ctx, len(bad), bad[0])


@pytest.mark.parametrize("block,elem", MX_FORMATS)
@pytest.mark.parametrize("N,d", [(1, 64), (67, 192), (130, 1024), (257, 4096), (5, 14336)])
def test_weight_cast_with_folded_gain(block, elem, N, d):
    # weights of a linear layer: small Gaussian entries; gain around 1
    wb = synth.gaussian(N, d, seed=N * d + block, scale=0.02)
    gb = synth.f32_to_bf16_bits(np.random.default_rng(d).uniform(0.2, 3.0, d).astype(np.float32))
    for mode in ("rceil", "floor"):
        check_cast(wb, gb, block, elem, mode)
        check_cast(wb, None, block, elem, mode)


@pytest.mark.parametrize("block,elem", MX_FORMATS)
def test_weight_cast_edge_rows(block, elem):
    for d in (64, 1024):
        ab = adversarial_rows(d, seed=d + block)
        gb = synth.f32_to_bf16_bits(np.linspace(-3, 3, d).astype(np.float32))
        check_cast(ab, gb, block, elem)
        check_cast(ab, None, block, elem, "floor")


# ------------------------------------------------------- post-round MXNorm --

def check_post(xb, block, elem, eps=1e-6, mode="rceil"):
    x = dev_bf16(xb)
    got = mxnorm.mxnorm_postround_mx_fwd(x, block=block, elem=elem, eps=eps, scale_mode=mode)
    torch.cuda.synchronize()
    wc, ws, w32, _ = oracle.mxnorm_postround_mx(xb, B=block, elem=elem, eps=eps, mode=mode)
    codes, scales, rho = (t.cpu().numpy() for t in got)
    ctx = "postround B=%d %s %s eps=%g shape=%s" % (block, elem, mode, eps, xb.shape)
    same = (rho == w32) | (np.isnan(rho) & np.isnan(w32))
    assert same.all(), "%s: rho differs in %d rows, first %s" % (ctx, (~same).sum(),
                                                                  np.argwhere(~same)[0])
    bad = np.argwhere(scales != ws)
    assert bad.size == 0, "%s: %d scale bytes differ, first %s" % (ctx, len(bad), bad[0])
    bad = np.argwhere(codes != wc)
    assert bad.size == 0, "%s: %d codes differ, first %s" % (ctx, len(bad), bad[0])


@pytest.mark.parametrize("block,elem", MX_FORMATS)
@pytest.mark.parametrize("T,d", [(3, 64), (65, 192), (130, 1024), (33, 1280), (257, 4096),
                                 (9, 10240), (4, 32768)])
def test_postround_shapes(block, elem, T, d):
    # rows with sigma spread over many octaves: every table segment and
    # power-of-two scaling is exercised
    rng = np.random.default_rng(T * d + block)
    sig = np.exp2(rng.uniform(-20, 20, T)).astype(np.float32)
    xb = synth.f32_to_bf16_bits((rng.standard_normal((T, d)) * sig[:, None]).astype(np.float32))
    check_post(xb, block, elem)


@pytest.mark.parametrize("block,elem", MX_FORMATS)
def test_postround_modes_eps_and_edge_rows(block, elem):
    xb = synth.gaussian(100, 2048, seed=block + 1, scale=0.3)
    for mode in ("rceil", "floor"):
        for eps in (0.0, 1e-6, 0.5):
            check_post(xb, block, elem, eps=eps, mode=mode)
    for d in (64, 1024):
        ab = adversarial_rows(d, seed=block + d + 3)
        for mode in ("rceil", "floor"):
            for eps in (0.0, 1e-6):
                check_post(ab, block, elem, eps=eps, mode=mode)
