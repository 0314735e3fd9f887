"""The oracle's host mirror of the library's forward boundary (mxref_*): the
same argument lists with host pointers and no stream.

What fixes the expectations: the library itself for the status of every
rejected argument list (validation happens on the host, before any launch,
so no GPU is needed), and the oracle's own entry points for the outputs of
accepted ones (the mirror adds argument handling only: coef <= 0 selecting
the table, rho optional)."""
import ctypes

import numpy as np
import pytest

import oracle
from paper_2603_13180_amd import mxnorm, synth

# fake pointers for rejected calls: validation must fail before any access
A16, OUT = 0x10000, 0x20000
NAN, INF = float("nan"), float("inf")


def lib_and_ref():
    return mxnorm.load(), oracle._load()


CASES_MXFP8 = [dict(x=None), dict(codes=None), dict(scales=None), dict(T=-1), dict(d=0),
               dict(d=48), dict(d=65536), dict(p=3), dict(p=0), dict(coef=NAN),
               dict(coef=INF), dict(eps=-1.0), dict(eps=NAN), dict(eps=INF), dict(mode=2),
               dict(T=0), dict(T=0, x=None, codes=None, scales=None),
               dict(T=0, d=48, x=None, codes=None, scales=None)]


@pytest.mark.parametrize("kw", CASES_MXFP8)
def test_mxnorm_mxfp8_status_matches_library(kw):
    lib, ref = lib_and_ref()
    a = dict(x=A16, T=4, d=64, p=2, coef=0.0, eps=1e-6, mode=0, codes=OUT, scales=OUT)
    a.update(kw)
    want = lib.mxnorm_mxfp8_fwd(a["x"], a["T"], a["d"], a["p"], a["coef"], a["eps"], a["mode"],
                                a["codes"], a["scales"], None, None)
    got = ref.mxref_mxnorm_mxfp8_fwd(a["x"], a["T"], a["d"], a["p"], a["coef"], a["eps"],
                                     a["mode"], a["codes"], a["scales"], None)
    assert want != 0 or a["T"] == 0
    assert got == want, (kw, got, want)


@pytest.mark.parametrize("kw", [dict(x=None), dict(T=-1), dict(d=40), dict(d=65536),
                                dict(p=3), dict(coef=NAN), dict(eps=-1.0), dict(sg=0.0),
                                dict(sg=-1.0), dict(sg=NAN), dict(sg=INF), dict(sg=1e-39),
                                dict(sg=1e38), dict(T=0)])
def test_nvfp4_status_matches_library(kw):
    lib, ref = lib_and_ref()
    a = dict(x=A16, T=4, d=64, p=2, coef=0.0, eps=1e-6, sg=0.01)
    a.update(kw)
    want = lib.mxnorm_nvfp4_fwd(a["x"], a["T"], a["d"], a["p"], a["coef"], a["eps"], a["sg"],
                                OUT, OUT, None, None)
    got = ref.mxref_mxnorm_nvfp4_fwd(a["x"], a["T"], a["d"], a["p"], a["coef"], a["eps"],
                                     a["sg"], OUT, OUT, None)
    assert got == want, (kw, got, want)
    if "p" not in kw and "coef" not in kw:
        want = lib.rmsnorm_nvfp4_fwd(a["x"], None, a["T"], a["d"], a["eps"], a["sg"], OUT, OUT,
                                     None, None)
        got = ref.mxref_rmsnorm_nvfp4_fwd(a["x"], None, a["T"], a["d"], a["eps"], a["sg"], OUT,
                                          OUT, None)
        assert got == want, (kw, got, want)


@pytest.mark.parametrize("kw", [dict(x=None), dict(T=-1), dict(d=48), dict(d=65536),
                                dict(eps=NAN), dict(mode=5), dict(T=0)])
def test_rmsnorm_mxfp8_status_matches_library(kw):
    lib, ref = lib_and_ref()
    a = dict(x=A16, T=4, d=64, eps=1e-6, mode=0)
    a.update(kw)
    want = lib.rmsnorm_mxfp8_fwd(a["x"], None, a["T"], a["d"], a["eps"], a["mode"], OUT, OUT,
                                 None, None)
    got = ref.mxref_rmsnorm_mxfp8_fwd(a["x"], None, a["T"], a["d"], a["eps"], a["mode"], OUT,
                                      OUT, None)
    assert got == want, (kw, got, want)


def p_(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def test_accepted_calls_equal_the_oracle():
    ref = oracle._load()
    T, d = 9, 256
    x = synth.gaussian(T, d, seed=4, scale=2.0)
    g = synth.f32_to_bf16_bits(np.linspace(0.5, 1.5, d).astype(np.float32))
    for p in (1, 2):
        c = np.empty((T, d), np.uint8); s = np.empty((T, d // 32), np.uint8)
        r = np.empty(T, np.float32)
        assert ref.mxref_mxnorm_mxfp8_fwd(p_(x), T, d, p, 0.0, 1e-6, 0, p_(c), p_(s), p_(r)) == 0
        wc, ws, wr, _ = oracle.mxnorm_mxfp8(x, p=p)
        assert np.array_equal(c, wc) and np.array_equal(s, ws) and np.array_equal(r, wr)
        # the cast stage for that rho reproduces the codes (the two-part contract)
        c2 = np.empty_like(c); s2 = np.empty_like(s)
        assert ref.mxref_cast_given_rho(p_(x), p_(r), T, d, 0, p_(c2), p_(s2)) == 0
        assert np.array_equal(c2, wc) and np.array_equal(s2, ws)
    c = np.empty((T, d), np.uint8); s = np.empty((T, d // 32), np.uint8)
    assert ref.mxref_rmsnorm_mxfp8_fwd(p_(x), p_(g), T, d, 1e-6, 1, p_(c), p_(s), None) == 0
    wc, ws, _, _ = oracle.rmsnorm_mxfp8(x, g, mode="floor")
    assert np.array_equal(c, wc) and np.array_equal(s, ws)
    sg = oracle.mxnorm_default_global_scale(d, 16, 2)
    c = np.empty((T, d // 2), np.uint8); s = np.empty((T, d // 16), np.uint8)
    assert ref.mxref_mxnorm_nvfp4_fwd(p_(x), T, d, 2, 0.0, 1e-6, sg, p_(c), p_(s), None) == 0
    wc, ws, _, _ = oracle.mxnorm_nvfp4(x, sg)
    assert np.array_equal(c, wc) and np.array_equal(s, ws)
    c = np.empty((T, d // 2), np.uint8); s = np.empty((T, d // 16), np.uint8)
    assert ref.mxref_rmsnorm_nvfp4_fwd(p_(x), p_(g), T, d, 1e-6, 0.01, p_(c), p_(s), None) == 0
    wc, ws, _, _ = oracle.rmsnorm_nvfp4(x, 0.01, g)
    assert np.array_equal(c, wc) and np.array_equal(s, ws)


def test_cast_given_rho_rejects_missing_rho():
    ref = oracle._load()
    assert ref.mxref_cast_given_rho(A16, None, 4, 64, 0, OUT, OUT) == 1
    assert ref.mxref_cast_given_rho(A16, None, 0, 64, 0, OUT, OUT) == 0
