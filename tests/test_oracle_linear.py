"""Pins for the oracle's MXNormLinear pieces (Sec. 3.7, eq. (mx-matmul); the
implementation appendix's mx_norm_linear_forward): the gain fold MXCast(W
gamma) and the MX matmul.  Independent references: numpy's float64 matmul of
operands dequantised through torch's float8 decoder and 2^(s-127); closed
forms; and the associativity the paper relies on."""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_13180_amd import synth


def dequant_e4m3(codes, scales, B=32):
    v = torch.from_numpy(np.ascontiguousarray(codes)).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    s = np.exp2(scales.astype(np.float64) - 127.0)
    return (v.reshape(v.shape[0], -1, B) * s[..., None]).reshape(v.shape)


E2M1 = np.array([0, .5, 1, 1.5, 2, 3, 4, 6, -0., -.5, -1, -1.5, -2, -3, -4, -6])


def dequant_e2m1(codes, scales, B=32):
    nib = np.stack([codes & 0xF, codes >> 4], -1).reshape(codes.shape[0], -1)
    v = E2M1[nib]
    s = np.exp2(scales.astype(np.float64) - 127.0)
    return (v.reshape(v.shape[0], -1, B) * s[..., None]).reshape(v.shape)


@pytest.mark.parametrize("elem,deq", [("e4m3", dequant_e4m3), ("e2m1", dequant_e2m1)])
@pytest.mark.parametrize("B", [16, 32, 64])
def test_mx_matmul_equals_library_matmul_of_dequantised(elem, deq, B):
    rng = np.random.default_rng(B)
    x = synth.f32_to_bf16_bits(rng.standard_normal((13, 256)).astype(np.float32))
    w = synth.f32_to_bf16_bits((rng.standard_normal((7, 256)) * 0.05).astype(np.float32))
    ac, as_, _, _ = oracle.mxnorm_mx(x, B=B, elem=elem)
    wc, ws = oracle.mxcast_gain(w, None, B=B, elem=elem)
    h = oracle.mx_matmul(ac, as_, wc, ws, 256, B=B, elem=elem)
    ref = deq(ac, as_, B) @ deq(wc, ws, B).T
    assert np.allclose(h, ref, rtol=1e-12, atol=1e-300)


def test_gain_fold_indexes_columns():
    rng = np.random.default_rng(1)
    w = synth.f32_to_bf16_bits(rng.standard_normal((5, 128)).astype(np.float32))
    ones = synth.f32_to_bf16_bits(np.ones(128, np.float32))
    c1, s1 = oracle.mxcast_gain(w, ones)
    c0, s0 = oracle.mxcast_gain(w, None)
    assert np.array_equal(c1, c0) and np.array_equal(s1, s0)
    # gamma = 2^3 on the second 32-column block only: that block's scale
    # moves up by 3 in every row, its codes are unchanged, the rest is untouched
    g = np.ones(128, np.float32)
    g[32:64] = 8.0
    c8, s8 = oracle.mxcast_gain(w, synth.f32_to_bf16_bits(g))
    assert np.array_equal(c8, c0)
    assert np.array_equal(s8[:, 1], s0[:, 1] + 3)
    assert np.array_equal(np.delete(s8, 1, 1), np.delete(s0, 1, 1))
    # a general gain equals the plain cast of the float product w * gamma
    gg = synth.f32_to_bf16_bits(rng.uniform(0.5, 1.5, 128).astype(np.float32))
    cg, sg = oracle.mxcast_gain(w, gg)
    y = synth.bf16_bits_to_f32(w) * synth.bf16_bits_to_f32(gg)[None, :]
    cy, sy = oracle.mxcast(y.astype(np.float32))
    assert np.array_equal(cg, cy) and np.array_equal(sg, sy)


def test_one_hot_matmul():
    # A row with a single 1.0 at column j and B = I-like rows: H picks entries
    K = 64
    x = np.zeros((2, K), np.float32)
    x[0, 5] = 1.0
    x[1, 40] = -2.0
    w = np.zeros((3, K), np.float32)
    w[0, 5] = 3.0
    w[1, 40] = 0.5
    w[2, :] = 1.0
    xb, wb = synth.f32_to_bf16_bits(x), synth.f32_to_bf16_bits(w)
    c, s = oracle.mxcast(x)
    wc, ws = oracle.mxcast(w)
    h = oracle.mx_matmul(c, s, wc, ws, K)
    assert np.array_equal(h, np.array([[3.0, 0.0, 1.0], [0.0, -1.0, -2.0]]))


@pytest.mark.parametrize("elem,tol", [("e4m3", 0.05), ("e2m1", 0.25)])
def test_mxnorm_linear_approximates_rmsnorm_linear(elem, tol):
    # Sec. 3.7: normalising by MXNorm and folding gamma into W approximates
    # RMSNorm(X; gamma) W^T; Gaussian data, K = 1024 (32 blocks)
    rng = np.random.default_rng(7)
    x = synth.f32_to_bf16_bits(rng.standard_normal((64, 1024)).astype(np.float32))
    w = synth.f32_to_bf16_bits((rng.standard_normal((48, 1024)) / 32).astype(np.float32))
    g = synth.f32_to_bf16_bits(rng.uniform(0.5, 1.5, 1024).astype(np.float32))
    h, _, _, _ = oracle.mxnorm_linear(x, w, g, elem=elem)
    xf = synth.bf16_bits_to_f32(x).astype(np.float64)
    rms = np.sqrt((xf ** 2).mean(1, keepdims=True))
    ref = (xf / rms * synth.bf16_bits_to_f32(g)) @ synth.bf16_bits_to_f32(w).astype(np.float64).T
    rel = np.linalg.norm(h - ref) / np.linalg.norm(ref)
    assert rel < tol
