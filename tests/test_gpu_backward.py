"""GPU parity of the MXNormLinear backward pieces against the oracle (Sec.
3.7; the RMSNorm-gradient appendix; the implementation appendix's
mx_norm_linear_backward): the column-wise MX cast (bit-exact), the
straight-through estimator (within bounds derived from its float
arithmetic), the matmul's column gain, and the whole backward composed from
the library's kernels, checked stage by stage."""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_13180_amd import mxnorm, synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU backward tests need a GPU (run them with -m gpu on an MI355X)")
    mxnorm.load()


def dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.bfloat16)


def bits_of(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def f64(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


# ----------------------------------------------------------- column cast --

def check_cast_t(xb, rho, elem, mode):
    x = dev_bf16(xb)
    r = None if rho is None else torch.from_numpy(rho).to(DEV)
    codes, scales = mxnorm.mx_cast_t_fwd(x, r, elem=elem, scale_mode=mode)
    torch.cuda.synchronize()
    wc, ws = oracle.mxcast_t(xb, rho, B=32, elem=elem, mode=mode)
    ctx = "cast_t %s %s %s rho=%s" % (xb.shape, elem, mode, rho is not None)
    s, c = scales.cpu().numpy(), codes.cpu().numpy()
    bad = np.argwhere(s != ws)
    assert bad.size == 0, "%s: %d scale bytes differ, first %s" % (ctx, len(bad), bad[0])
    bad = np.argwhere(c != wc)
    assert bad.size == 0, "%s: %d codes differ, first %s got %#x want %#x" % (
        ctx, len(bad), bad[0], c[tuple(bad[0])], wc[tuple(bad[0])])


@pytest.mark.parametrize("elem", ["e4m3", "e2m1"])
@pytest.mark.parametrize("R,C", [(32, 8), (96, 40), (160, 200), (256, 64), (1024, 1000),
                                 (4096, 256), (64, 8200), (288, 8448), (160, 12296)])
def test_cast_t_shapes(elem, R, C):
    # ragged last column tiles (8200, 8448, 12296) and row tiles (160, 288);
    # from 48 column tiles (12288 columns) on the workgroups visit the tiles
    # in XCD ranges of 64-row-tile groups (12296 x 160: one partial group)
    xb = synth.gaussian(R, C, seed=R + C, scale=2.0)
    rho = np.random.default_rng(R).uniform(0.01, 8.0, R).astype(np.float32)
    for mode in ("rceil", "floor"):
        check_cast_t(xb, None, elem, mode)
        check_cast_t(xb, rho, elem, mode)


@pytest.mark.parametrize("elem", ["e4m3", "e2m1"])
def test_cast_t_edge_columns(elem):
    # the forward's adversarial rows, laid out as columns (one per row of it)
    from test_gpu_parity import adversarial_rows
    for R in (64, 1024):
        xb = np.ascontiguousarray(adversarial_rows(R, seed=R).T)   # [R, 14] -> pad to 16 cols
        xb = np.ascontiguousarray(np.concatenate([xb, xb[:, :2]], axis=1))
        rho = np.full(R, 0.75, np.float32)
        for mode in ("rceil", "floor"):
            check_cast_t(xb, None, elem, mode)
            check_cast_t(xb, rho, elem, mode)


@pytest.mark.parametrize("elem", ["e4m3", "e2m1"])
@pytest.mark.parametrize("R,C", [(16384, 4096), (32768, 4096), (4096, 28672), (16384, 16384),
                                 (8320, 12288)])
def test_cast_t_multi_tile_spans_sampled(elem, R, C):
    """Large shapes: the bench's [32768, 4096], the wide grad_H of the
    gate+up projection at 4096 tokens (112 column tiles, one partial group
    of row tiles in the XCD-range order), [16384, 16384] (two full groups)
    and [8320, 12288] (a full group and a partial one): output rows of sampled columns -- the first and last of column
    tiles and random ones -- against the oracle's cast of those columns
    alone (an output row depends only on its column and rho)."""
    rng = np.random.default_rng(R + C)
    xb = synth.gaussian(R, C, seed=C, scale=3.0)
    rho = rng.uniform(0.01, 8.0, R).astype(np.float32)
    cols = np.unique(np.concatenate([[0, 1, 63, 64, 127, 128, 255, 256, C - 64, C - 1],
                                     rng.choice(C, 24, replace=False)]))
    x = dev_bf16(xb)
    codes, scales = mxnorm.mx_cast_t_fwd(x, torch.from_numpy(rho).to(DEV), elem=elem)
    torch.cuda.synchronize()
    c, sc = codes.cpu().numpy(), scales.cpu().numpy()
    # the oracle casts a column block of 8 (its C must be a multiple of 8)
    for c0 in np.unique(cols // 8 * 8):
        wc, ws = oracle.mxcast_t(np.ascontiguousarray(xb[:, c0:c0 + 8]), rho, B=32, elem=elem,
                                 mode="rceil")
        assert np.array_equal(sc[c0:c0 + 8], ws), "cast_t [%d, %d] %s scales, cols %d.." % (
            R, C, elem, c0)
        assert np.array_equal(c[c0:c0 + 8], wc), "cast_t [%d, %d] %s codes, cols %d.." % (
            R, C, elem, c0)


def test_cast_t_empty():
    x = torch.empty(0, 64, dtype=torch.bfloat16, device=DEV)
    c, s = mxnorm.mx_cast_t_fwd(x)
    assert c.shape == (64, 0) and s.shape == (64, 0)


# ------------------------------------------------------------------- STE --

def ste_bounds(xb, gzb, gb, rho):
    """Size of the two terms of grad_x per element, and of the grad_gamma sum."""
    x, gz = f64(xb), f64(gzb)
    g = f64(gb) if gb is not None else np.ones(x.shape[1])
    r = rho.astype(np.float64)[:, None]
    dxb = gz * g
    u = np.sum(dxb * x, axis=1, keepdims=True)
    c = r ** 3 * u / x.shape[1]
    return np.abs(r * dxb) + np.abs(c * x), np.sum(np.abs(r * x * gz), axis=0)


def check_ste(T, d, gamma, out_dtype, want_gg, seed=0, xb=None):
    rng = np.random.default_rng(seed + T + d)
    if xb is None:
        xb = synth.gaussian(T, d, seed=seed + d, scale=1.5)
    gzb = synth.gaussian(T, d, seed=seed + d + 1, scale=0.2)
    gb = synth.f32_to_bf16_bits(rng.uniform(0.3, 2.0, d).astype(np.float32)) if gamma else None
    rho = rng.uniform(0.2, 3.0, T).astype(np.float32)
    gx, gg = mxnorm.mxnorm_ste_bwd(dev_bf16(xb), dev_bf16(gzb),
                                   None if gb is None else dev_bf16(gb),
                                   torch.from_numpy(rho).to(DEV), out_dtype=out_dtype,
                                   want_grad_gamma=want_gg)
    torch.cuda.synchronize()
    wx, wg = oracle.ste_bwd(xb, gzb, gb, rho)
    terms, gsum = ste_bounds(xb, gzb, gb, rho)
    got = gx.float().cpu().numpy().astype(np.float64)
    # float arithmetic: RN(rho dXb), RN(c x) with c rounded once, their
    # difference rounded: within 2^-21 of the terms plus 2^-22 of the result;
    # bf16 output adds half an ulp (2^-8 relative)
    tol = 2.0 ** -21 * terms + 2.0 ** -22 * np.abs(wx) + 1e-37
    if out_dtype == torch.bfloat16:
        tol = tol + 2.0 ** -8 * np.abs(wx)
    fin = np.isfinite(wx)
    err = np.abs(got - wx)
    bad = fin & (err > tol)
    ctx = "ste T=%d d=%d gamma=%s %s" % (T, d, gamma, out_dtype)
    assert not bad.any(), "%s: %d grad_x off, first %s got %r want %r" % (
        ctx, bad.sum(), np.argwhere(bad)[0], got[tuple(np.argwhere(bad)[0])],
        wx[tuple(np.argwhere(bad)[0])])
    if want_gg:
        # float partial sums over 32 rows (each term rounded twice), then a
        # double sum: within 2^-16 of sum |terms|
        g = gg.cpu().numpy().astype(np.float64)
        assert (np.abs(g - wg) <= 2.0 ** -16 * gsum + 1e-37).all(), ctx + ": grad_gamma"
    else:
        assert gg is None


@pytest.mark.parametrize("T,d", [(1, 8), (33, 64), (100, 1024), (40, 4096), (65, 2048),
                                 (9, 10240), (3, 32768), (70, 2056), (2049, 256), (4100, 512)])
def test_ste_shapes(T, d):
    check_ste(T, d, True, torch.bfloat16, True)
    check_ste(T, d, False, torch.float32, True)


def test_ste_bench_shape():
    # the bench's [32768, 4096]: 64 rows per workgroup (512 workgroups), the
    # three-set row pipeline run to its end, every element of grad_x and
    # grad_gamma compared
    check_ste(32768, 4096, True, torch.bfloat16, True, seed=3)


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("gamma", [True, False])
@pytest.mark.parametrize("want_gg", [True, False])
def test_ste_options(out_dtype, gamma, want_gg):
    check_ste(77, 4096, gamma, out_dtype, want_gg, seed=5)


def test_ste_zero_and_constant_rows():
    T, d = 40, 512
    xb = synth.gaussian(T, d, seed=9)
    xb[3] = 0
    xb[7] = synth.f32_to_bf16_bits(np.full(d, -1.25, np.float32))
    check_ste(T, d, True, torch.float32, True, xb=xb)


def test_ste_deterministic_and_workspace_reuse():
    T, d = 300, 4096
    xb = synth.gaussian(T, d, seed=1)
    gzb = synth.gaussian(T, d, seed=2)
    x, gz = dev_bf16(xb), dev_bf16(gzb)
    rho = torch.rand(T, device=DEV) + 0.5
    ws = torch.empty(mxnorm.load().mxnorm_ste_bwd_workspace_bytes(T, d), dtype=torch.uint8,
                     device=DEV)
    a = mxnorm.mxnorm_ste_bwd(x, gz, None, rho, workspace=ws)
    b = mxnorm.mxnorm_ste_bwd(x, gz, None, rho, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


# ---------------------------------------------------- matmul column gain --

@pytest.mark.parametrize("elem", ["e4m3", "e2m1"])
def test_matmul_column_gain(elem):
    from test_gpu_gemm import random_operand, abs_codes, assert_close
    M, N, K = 130, 272, 512
    rng = np.random.default_rng(3)
    ac, as_ = random_operand(M, K, elem, rng)
    bc, bs = random_operand(N, K, elem, rng)
    gb = synth.f32_to_bf16_bits(rng.uniform(-2, 2, N).astype(np.float32))
    t = [torch.from_numpy(v).to(DEV) for v in (ac, as_, bc, bs)]
    h = mxnorm.mx_matmul_fwd(*t, K, elem=elem, b_gain=dev_bf16(gb))
    torch.cuda.synchronize()
    g = f64(gb)
    want = oracle.mx_matmul(ac, as_, bc, bs, K, elem=elem) * g[None, :]
    mag = oracle.mx_matmul(abs_codes(ac, elem), as_, abs_codes(bc, elem), bs, K,
                           elem=elem) * np.abs(g)[None, :]
    # the gain multiply adds one float rounding (2^-24 of |H| <= sum|ab| |g|),
    # far inside the bound
    assert_close(h.cpu().numpy().astype(np.float64), want, mag, False, "gain %s" % elem)


# ------------------------------------------------------- whole backward --

@pytest.mark.parametrize("elem", ["e4m3", "e2m1"])
def test_mxnorm_linear_backward(elem):
    from test_gpu_gemm import abs_codes, assert_close
    T, d, N = 256, 512, 256
    rng = np.random.default_rng(17)
    xb = synth.gaussian(T, d, seed=21, scale=1.3)
    whb = synth.f32_to_bf16_bits((0.05 * rng.standard_normal((N, d))).astype(np.float32))
    ghb = synth.gaussian(T, N, seed=22, scale=0.1)
    gb = synth.f32_to_bf16_bits(rng.uniform(0.5, 1.5, d).astype(np.float32))
    x, w, gh, g = dev_bf16(xb), dev_bf16(whb), dev_bf16(ghb), dev_bf16(gb)
    _, _, rho = mxnorm.mxnorm_mx_fwd(x, block=32, elem=elem)
    gx, gg, gw = mxnorm.mxnorm_linear_bwd(gh, x, rho, g, w, elem=elem,
                                          grad_x_dtype=torch.float32)
    torch.cuda.synchronize()
    rho_np = rho.cpu().numpy()

    # stage 1: grad_Z = MXCast(grad_H) MXCast_N(W)
    hc, hs = oracle.mxcast_gain(ghb, None, B=32, elem=elem)
    wc, ws = oracle.mxcast_t(whb, None, B=32, elem=elem)
    gz_o = oracle.mx_matmul(hc, hs, wc, ws, N, elem=elem)
    gz_mag = oracle.mx_matmul(abs_codes(hc, elem), hs, abs_codes(wc, elem), ws, N, elem=elem)
    gh_c, gh_s = mxnorm.mx_cast_fwd(gh, None, elem=elem)
    wt_c, wt_s = mxnorm.mx_cast_t_fwd(w, None, elem=elem)
    gz = mxnorm.mx_matmul_fwd(gh_c, gh_s, wt_c, wt_s, N, elem=elem, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert np.array_equal(gh_c.cpu().numpy(), hc) and np.array_equal(wt_c.cpu().numpy(), wc)
    assert_close(gz.float().cpu().numpy().astype(np.float64), gz_o, gz_mag, True, "grad_Z")

    # stage 2: the STE on that grad_Z
    wx, wg = oracle.ste_bwd(xb, bits_of(gz), gb, rho_np)
    terms, gsum = ste_bounds(xb, bits_of(gz), gb, rho_np)
    assert (np.abs(gx.cpu().numpy() - wx) <= 2.0 ** -21 * terms + 2.0 ** -22 * np.abs(wx)
            + 1e-37).all()
    assert (np.abs(gg.cpu().numpy() - wg) <= 2.0 ** -16 * gsum + 1e-37).all()

    # stage 3: grad_W = (MXCast(grad_H^T) MXCast(rho~ X)^T) gamma
    tc, ts = oracle.mxcast_t(ghb, None, B=32, elem=elem)
    xc, xs = oracle.mxcast_t(xb, rho_np, B=32, elem=elem)
    gw_o = oracle.mx_matmul(tc, ts, xc, xs, T, elem=elem) * f64(gb)[None, :]
    gw_mag = oracle.mx_matmul(abs_codes(tc, elem), ts, abs_codes(xc, elem), xs, T,
                              elem=elem) * np.abs(f64(gb))[None, :]
    assert_close(gw.cpu().numpy().astype(np.float64), gw_o, gw_mag, False, "grad_W")

    # and the whole thing approximates the float64 RMSNorm-linear gradient:
    # the oracle's own chain is 5.6% (E4M3) and 16.8% (E2M1) away here, from
    # the 8- or 4-bit casts and rho~'s error at d = 512 (16 blocks per row)
    xs64 = f64(xb)
    S = np.sqrt(np.mean(xs64 ** 2, axis=1, keepdims=True))
    gw_ref = f64(ghb).T @ (xs64 / S) * f64(gb)[None, :]
    rel = np.linalg.norm(gw.cpu().numpy() - gw_ref) / np.linalg.norm(gw_ref)
    assert rel < (0.10 if elem == "e4m3" else 0.30), rel


def test_transpose_stream_reference_moves_the_bytes():
    # the column cast's stream reference (a bandwidth denominator) really
    # reads x and rho and writes the transposed bytes it claims to
    from paper_2603_13180_amd import streamref
    R, C = 256, 512
    g = torch.Generator(device=DEV)
    g.manual_seed(3)
    x = torch.randn(R, C, generator=g, device=DEV).to(torch.bfloat16)
    rho = torch.rand(R, generator=g, device=DEV) + 0.5
    out = torch.empty(C, R, dtype=torch.uint8, device=DEV)
    small = torch.empty(C, R // 32, dtype=torch.uint8, device=DEV)
    streamref.stream_reference_transpose(x, rho, out, small)
    torch.cuda.synchronize()
    xb = x.view(torch.int16).cpu().numpy().astype(np.uint16)
    hi = (xb >> 8).astype(np.uint8)
    assert np.array_equal(out.cpu().numpy(), hi.T)
    rb = rho.cpu().numpy().view(np.uint32)
    want = (hi[0::32, :].T ^ (rb[0::32] & 0xFF)[None, :]).astype(np.uint8)
    assert np.array_equal(small.cpu().numpy(), want)
