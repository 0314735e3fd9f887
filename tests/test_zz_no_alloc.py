"""The allocation-free straight-through-estimator entry point
(mxnorm_ste_bwd_noalloc) against the workspace entry point mxnorm_ste_bwd:
same kernels, so grad_x and grad_gamma must be bit-identical, on two calls
in a row (the second smaller, so it runs on the array the first one left
behind)."""
import numpy as np
import pytest
import torch

from paper_2603_13180_amd import mxnorm

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("the allocation-free entry point test needs a GPU (run it with -m gpu)")
    mxnorm.load()


def inputs(T, d, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    x = torch.randn(T, d, generator=g, device=DEV).to(torch.bfloat16)
    gz = (torch.randn(T, d, generator=g, device=DEV) * 0.01).to(torch.bfloat16)
    gam = (1.0 + 0.1 * torch.randn(d, generator=g, device=DEV)).to(torch.bfloat16)
    rho = torch.rand(T, generator=g, device=DEV) + 0.5
    return x, gz, gam, rho


def same_bits(a, b):
    return torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a.view(torch.int32),
                       b.view(torch.int16) if b.dtype == torch.bfloat16 else b.view(torch.int32))


@pytest.mark.parametrize("out_dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("with_gamma", [True, False])
def test_noalloc_equals_workspace_entry_point(out_dtype, with_gamma):
    # [32768, 4096] is the benchmarked backward shape; [1000, 2048] then runs
    # with fewer workgroups and narrower partial rows on the same array
    for (T, d, seed) in ((32768, 4096, 1), (1000, 2048, 2)):
        x, gz, gam, rho = inputs(T, d, seed)
        if not with_gamma:
            gam = None
        want_gx, want_gg = mxnorm.mxnorm_ste_bwd(x, gz, gam, rho, out_dtype=out_dtype)
        gx = torch.full((T, d), 7.0, dtype=out_dtype, device=DEV)
        gg = torch.full((d,), 7.0, dtype=torch.float32, device=DEV)
        mxnorm.mxnorm_ste_bwd_noalloc(x, gz, gam, rho, gx, gg)
        torch.cuda.synchronize()
        assert same_bits(gx, want_gx), "grad_x differs at [%d, %d]" % (T, d)
        assert same_bits(gg, want_gg), "grad_gamma differs at [%d, %d]" % (T, d)
        assert torch.isfinite(gg).all()


def test_noalloc_without_grad_gamma():
    x, gz, gam, rho = inputs(517, 1024, 3)
    want_gx, _ = mxnorm.mxnorm_ste_bwd(x, gz, gam, rho, want_grad_gamma=False)
    gx = torch.empty_like(want_gx)
    mxnorm.mxnorm_ste_bwd_noalloc(x, gz, gam, rho, gx, None)
    torch.cuda.synchronize()
    assert same_bits(gx, want_gx)

