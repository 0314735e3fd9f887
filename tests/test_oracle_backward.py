"""Pins for the oracle's MXNormLinear backward pieces (Sec. 3.7; the
RMSNorm-gradient appendix; the implementation appendix's
mx_norm_linear_backward): the straight-through estimator against torch's
float64 autograd of RMSNorm, its invariants, and the column-wise MX cast
against the pinned row cast of the transpose and a hand-worked column."""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_13180_amd import synth


def f32(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


def inputs(T, d, seed, gamma=True):
    x = synth.gaussian(T, d, seed=seed, scale=1.7)
    gz = synth.gaussian(T, d, seed=seed + 1, scale=0.3)
    g = synth.f32_to_bf16_bits(np.random.default_rng(seed).uniform(0.2, 2.0, d)
                               .astype(np.float32)) if gamma else None
    return x, gz, g


def exact_rho(x):
    return (1.0 / np.sqrt(np.mean(f32(x) ** 2, axis=1))).astype(np.float32)


@pytest.mark.parametrize("T,d,gamma", [(3, 32, True), (17, 96, True), (8, 256, False),
                                       (5, 1024, True)])
def test_ste_equals_autograd_of_rmsnorm(T, d, gamma):
    # with rho~ = 1/S the estimator is RMSNorm's exact gradient: compare with
    # torch autograd of Z = (X / S) gamma in float64, loss = sum(Z * grad_Z)
    x, gz, g = inputs(T, d, T * d, gamma)
    rho = exact_rho(x)
    gx, gg = oracle.ste_bwd(x, gz, g, rho)
    xt = torch.tensor(f32(x), requires_grad=True)
    gt = torch.tensor(f32(g) if g is not None else np.ones(d), requires_grad=True)
    # S from the float rho the oracle was given, so that only the formula differs
    S = 1.0 / torch.tensor(rho.astype(np.float64))
    S_live = torch.sqrt(torch.mean(xt * xt, dim=1))
    S_used = S_live + (S - S_live).detach()   # value of S, gradient of S_live
    z = xt / S_used[:, None] * gt
    (z * torch.tensor(f32(gz))).sum().backward()
    # autograd differentiates the exact S while the formula uses the float
    # rho~ (2^-24 relative): 1e-6 of the terms' size; a wrong sign, power or
    # 1/d would be off by O(1)
    scale = np.abs(rho[:, None] * f32(gz)).max()
    assert np.abs(gx - xt.grad.numpy()).max() <= 1e-6 * scale
    assert np.abs(gg - gt.grad.numpy()).max() <= 1e-6 * np.abs(gt.grad.numpy()).max()


def test_ste_gradient_is_orthogonal_to_x_at_exact_rms():
    # RMSNorm is scale invariant, so its input gradient is orthogonal to x
    x, gz, g = inputs(64, 512, 3)
    rho64 = 1.0 / np.sqrt(np.mean(f32(x) ** 2, axis=1))
    gx, _ = oracle.ste_bwd(x, gz, g, rho64.astype(np.float32))
    dot = np.sum(gx * f32(x), axis=1)
    # float rho differs from 1/S by <= 2^-24 relative: the residue is
    # rho u (1 - rho^2 ms), with |1 - rho^2 ms| <= 2^-22
    u = np.sum(f32(gz) * f32(g) * f32(x), axis=1)
    assert (np.abs(dot) <= 2.0 ** -21 * np.abs(rho64 * u) + 1e-12).all()
    assert np.abs(u).max() > 1.0   # not vacuous


def test_ste_linear_in_grad_and_gamma_none_is_ones():
    x, gz, g = inputs(9, 64, 11)
    rho = exact_rho(x) * np.float32(1.3)   # any estimate: the formula is linear in grad_Z
    gx1, gg1 = oracle.ste_bwd(x, gz, g, rho)
    neg = gz ^ np.uint16(0x8000)
    gx2, gg2 = oracle.ste_bwd(x, neg, g, rho)
    assert np.array_equal(gx1, -gx2) and np.array_equal(gg1, -gg2)
    ones = synth.f32_to_bf16_bits(np.ones(64, np.float32))
    a, b = oracle.ste_bwd(x, gz, None, rho), oracle.ste_bwd(x, gz, ones, rho)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_ste_gamma_gradient_is_column_sum():
    # grad_gamma_j = sum_t (rho_t x_tj) grad_Z_tj, independent of gamma
    x, gz, g = inputs(33, 64, 5)
    rho = exact_rho(x)
    _, gg = oracle.ste_bwd(x, gz, g, rho)
    want = np.sum(rho[:, None].astype(np.float64) * f32(x) * f32(gz), axis=0)
    assert np.allclose(gg, want, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("elem", ["e4m3", "e2m1"])
@pytest.mark.parametrize("mode", ["rceil", "floor"])
@pytest.mark.parametrize("with_rho", [False, True])
def test_cast_t_equals_row_cast_of_transpose(elem, mode, with_rho):
    x = synth.gaussian(96, 40, seed=7, scale=3.0)
    rho = (np.random.default_rng(1).uniform(0.05, 4.0, 96).astype(np.float32)
           if with_rho else None)
    y = synth.bf16_bits_to_f32(x).astype(np.float32)
    if with_rho:
        y = (y * rho[:, None]).astype(np.float32)   # IEEE single multiply, RN
    wc, ws = oracle.mxcast(np.ascontiguousarray(y.T), B=32, elem=elem, mode=mode)
    gc, gs = oracle.mxcast_t(x, rho, B=32, elem=elem, mode=mode)
    assert np.array_equal(gc, wc) and np.array_equal(gs, ws)


def test_cast_t_hand_column():
    # column c holds 0, 1, ..., 31 (exact in bf16).  RCEIL: amax 31 needs
    # 448 * 2^e >= 31, smallest e = -3 -> byte 124; codes E4M3(8 i):
    # 8 -> 0x50, 24 = 1.5 * 2^4 -> 0x5C, 248 (midpoint of 240 and 256, ties
    # to the even mantissa) -> 0x78.  The other column is all zero: byte 0,
    # codes 0 (RCEIL of 0 clamps to e = -127).
    x = np.zeros((32, 2), np.uint16)
    x[:, 1] = synth.f32_to_bf16_bits(np.arange(32, dtype=np.float32))
    codes, scales = oracle.mxcast_t(x, None, B=32, elem="e4m3")
    assert scales[1, 0] == 124 and scales[0, 0] == 0
    assert codes[1, 1] == 0x50 and codes[1, 3] == 0x5C and codes[1, 31] == 0x78
    assert (codes[0] == 0).all()


def test_cast_t_nan_block_takes_input_signs():
    x = synth.gaussian(64, 8, seed=2)
    x[40, 3] = 0xFFC0          # -NaN in rows 32..63 of column 3
    codes, scales = oracle.mxcast_t(x, None, B=32, elem="e4m3")
    assert scales[3, 1] == 0xFF and scales[3, 0] != 0xFF
    want = ((x[32:64, 3] >> 15).astype(np.uint8) << 7) | 0x7F
    assert np.array_equal(codes[3, 32:64], want)
