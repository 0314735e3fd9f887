"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/mxnorm.h declares, and rejects bad arguments on the
host -- before any launch and without touching the GPU."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

from paper_2603_13180_amd import mxnorm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mxnorm.h")

pytestmark = pytest.mark.skipif(not os.path.exists(mxnorm.LIB_PATH),
                                reason="libmxnorm.so not built")


def declared_functions(header=HEADER):
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b([a-z_][a-z0-9_]*)\s*\(", text)) - {"defined"})


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert len(names) >= 10
    lib = ctypes.CDLL(mxnorm.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) >= {"mxnorm_mxfp8_fwd", "rmsnorm_mxfp8_fwd", "mxnorm_nvfp4_fwd",
                          "rmsnorm_nvfp4_fwd"}


def test_every_header_maps_to_a_library_exporting_it():
    from paper_2603_13180_amd import streamref
    libs = {"mxnorm.h": mxnorm.LIB_PATH, "streamref.h": streamref.LIB_PATH}
    headers = sorted(os.listdir(os.path.dirname(HEADER)))
    assert set(headers) == set(libs), headers
    for h in headers:
        lib = ctypes.CDLL(libs[h])
        for n in declared_functions(os.path.join(os.path.dirname(HEADER), h)):
            assert hasattr(lib, n), (h, n)


def test_stream_reference_rejects_bad_arguments():
    from paper_2603_13180_amd import streamref
    lib = streamref.load()
    f = lib.mx_stream_reference
    assert f(A16, 4, 1000, OUT, OUT, 0, None) == 1          # d % 512
    assert f(A16, 4, 8192, OUT, OUT, 0, None) == 1          # d > 4096
    assert f(A16, 4, 4096, OUT, OUT, 5, None) == 1          # mode
    assert f(A8, 4, 4096, OUT, OUT, 0, None) == 1           # alignment
    assert f(A16, -1, 4096, OUT, OUT, 0, None) == 1
    assert f(None, 0, 4096, None, None, 0, None) == 0       # T = 0: no-op


def test_ste_stream_reference_rejects_bad_arguments():
    from paper_2603_13180_amd import streamref
    f = streamref.load().mx_stream_reference_ste
    assert f(A16, A16, 4, 1000, OUT, None) == 1              # d % 512
    assert f(A16, A16, 4, 8192, OUT, None) == 1              # d > 4096
    assert f(A16, A8, 4, 4096, OUT, None) == 1               # alignment
    assert f(A16, A16, -1, 4096, OUT, None) == 1
    assert f(None, None, 0, 4096, None, None) == 0           # T = 0: no-op


def test_transpose_stream_reference_rejects_bad_arguments():
    from paper_2603_13180_amd import streamref
    f = streamref.load().mx_stream_reference_transpose
    assert f(A16, OUT, 200, 256, OUT, OUT, None) == 1        # R % 128
    assert f(A16, OUT, 128, 320, OUT, OUT, None) == 1        # C % 256
    assert f(A8, OUT, 128, 256, OUT, OUT, None) == 1         # x alignment
    assert f(A16, None, 128, 256, OUT, OUT, None) == 1       # rho NULL
    assert f(A16, OUT, -128, 256, OUT, OUT, None) == 1
    assert f(None, None, 0, 256, None, None, None) == 0      # R = 0: no-op


def test_header_compiles_as_c():
    import subprocess
    import tempfile
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "t.c")
        open(src, "w").write('#include "mxnorm.h"\nint main(void){return MX_OK;}\n')
        # host C code that includes HIP's runtime API names the platform
        subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
                        "-I", os.path.dirname(HEADER), "-I", "/opt/rocm/include",
                        "-c", src, "-o", os.path.join(d, "t.o")], check=True)


def test_abi_version_status_strings_and_coefs():
    lib = mxnorm.load()
    assert lib.mxnorm_abi_version() == 1
    for s in range(4):
        assert mxnorm.mx_status_str(s).startswith("MX_")
    assert mxnorm.mxnorm_coef(32, 2) == np.float32(0.4185)
    assert mxnorm.mxnorm_coef(16, 1) == np.float32(0.4814)
    assert math.isnan(mxnorm.mxnorm_coef(8, 2)) and math.isnan(mxnorm.mxnorm_coef(32, 3))


def test_default_global_scales_match_oracle():
    import oracle
    for d in (1024, 4096, 768 * 2):
        for p in (1, 2):
            assert mxnorm.mxnorm_default_global_scale(d, 16, p) == \
                np.float32(oracle.mxnorm_default_global_scale(d, 16, p))
        assert mxnorm.rmsnorm_default_global_scale(d, 1.5) == \
            np.float32(oracle.rmsnorm_default_global_scale(d, 1.5))
    assert math.isnan(mxnorm.mxnorm_default_global_scale(100, 16, 2))
    assert math.isnan(mxnorm.rmsnorm_default_global_scale(64, -1.0))


# Fake host pointers: validation must reject the call before it could be
# dereferenced, launched or written to.
A16 = 0x10000
A8 = 0x10008
OUT = 0x20000


def mxfp8(lib, x=A16, T=4, d=64, p=2, coef=0.0, eps=1e-6, mode=0, codes=OUT, scales=OUT,
          rho=None):
    return lib.mxnorm_mxfp8_fwd(x, T, d, p, coef, eps, mode, codes, scales, rho, None)


@pytest.mark.parametrize("kw,status", [
    (dict(x=None), 1), (dict(codes=None), 1), (dict(scales=None), 1),
    (dict(T=-1), 1), (dict(d=0), 1), (dict(d=48), 1), (dict(d=65536), 2),
    (dict(p=3), 1), (dict(p=0), 1), (dict(coef=float("nan")), 1), (dict(coef=float("inf")), 1),
    (dict(eps=-1.0), 1), (dict(eps=float("nan")), 1), (dict(eps=float("inf")), 1),
    (dict(mode=2), 1), (dict(x=A8), 1), (dict(codes=OUT + 4), 1), (dict(rho=OUT + 2), 1),
])
def test_mxnorm_mxfp8_rejects_bad_arguments(kw, status):
    lib = mxnorm.load()
    assert mxfp8(lib, **kw) == status
    assert mxnorm.mx_last_error() != ""


def test_zero_rows_is_a_no_op_without_launch():
    lib = mxnorm.load()
    assert mxfp8(lib, T=0) == 0
    assert lib.rmsnorm_mxfp8_fwd(A16, None, 0, 64, 1e-6, 0, OUT, OUT, None, None) == 0
    assert lib.mxnorm_nvfp4_fwd(A16, 0, 64, 2, 0.0, 1e-6, 0.01, OUT, OUT, None, None) == 0
    assert lib.rmsnorm_nvfp4_fwd(A16, None, 0, 64, 1e-6, 0.01, OUT, OUT, None, None) == 0
    # an empty tensor may come with NULL data pointers
    assert mxfp8(lib, x=None, T=0, codes=None, scales=None) == 0
    assert lib.mxnorm_nvfp4_fwd(None, 0, 64, 2, 0.0, 1e-6, 0.01, None, None, None, None) == 0
    # shape and scalar arguments are still checked
    assert mxfp8(lib, x=None, T=0, d=48, codes=None, scales=None) == 1


@pytest.mark.parametrize("sg", [0.0, -1.0, float("nan"), float("inf"), 1e-39, 1e38])
def test_nvfp4_rejects_bad_global_scale(sg):
    lib = mxnorm.load()
    assert lib.mxnorm_nvfp4_fwd(A16, 4, 64, 2, 0.0, 1e-6, sg, OUT, OUT, None, None) == 1
    assert lib.rmsnorm_nvfp4_fwd(A16, None, 4, 64, 1e-6, sg, OUT, OUT, None, None) == 1


def test_nvfp4_and_rmsnorm_shape_rules():
    lib = mxnorm.load()
    # NVFP4 needs d % 16 == 0; MXFP8 needs d % 32 == 0
    assert lib.mxnorm_nvfp4_fwd(A16, 4, 40, 2, 0.0, 1e-6, 0.01, OUT, OUT, None, None) == 1
    assert lib.rmsnorm_mxfp8_fwd(A16, None, 4, 48, 1e-6, 0, OUT, OUT, None, None) == 1
    assert lib.rmsnorm_mxfp8_fwd(A16, A8, 4, 64, 1e-6, 0, OUT, OUT, None, None) == 1  # gamma align
    assert lib.rmsnorm_mxfp8_fwd(A16, None, 4, 64, 1e-6, 5, OUT, OUT, None, None) == 1


def test_binding_refuses_cpu_tensors():
    import torch
    x = torch.zeros(4, 64, dtype=torch.bfloat16)
    with pytest.raises(RuntimeError, match="GPU"):
        mxnorm.mxnorm_mxfp8_fwd(x)
    with pytest.raises(TypeError):
        mxnorm.mxnorm_mxfp8_fwd(torch.zeros(4, 64))


@pytest.mark.parametrize("args,status", [
    ((A16, 4, 64, 8, 0), 1),     # block 8
    ((A16, 4, 64, 128, 0), 1),   # block 128
    ((A16, 4, 64, 32, 2), 1),    # element format
    ((A16, 4, 48, 32, 0), 1),    # d % block
    ((A16, 4, 96, 64, 1), 1),    # d % 64
    ((A16, 4, 65536, 64, 0), 2), # d too large
    ((None, 0, 64, 64, 1), 0),   # T = 0
])
def test_generic_mx_entry_points_validate(args, status):
    lib = mxnorm.load()
    x, T, d, block, elem = args
    assert lib.mxnorm_mx_fwd(x, T, d, block, elem, 2, 0.0, 1e-6, 0, OUT if T else None,
                             OUT if T else None, None, None) == status
    assert lib.rmsnorm_mx_fwd(x, None, T, d, block, elem, 1e-6, 0, OUT if T else None,
                              OUT if T else None, None, None) == status
    assert lib.mx_cast_fwd(x, None, T, d, block, elem, 0, OUT if T else None,
                           OUT if T else None, None) == status


def test_mx_cast_rejects_bad_arguments():
    lib = mxnorm.load()
    ok = (A16, None, 4, 64, 32, 0, 0, OUT, OUT, None)
    assert lib.mx_cast_fwd(*ok[:1], A8, *ok[2:]) == 1              # gamma alignment
    assert lib.mx_cast_fwd(*ok[:6], 2, *ok[7:]) == 1               # scale mode
    assert lib.mx_cast_fwd(None, *ok[1:]) == 1                     # x NULL with T > 0
    assert lib.mx_cast_fwd(*ok[:7], None, *ok[8:]) == 1            # codes NULL
    assert lib.mx_cast_fwd(*ok[:2], -1, *ok[3:]) == 1              # T < 0


@pytest.mark.parametrize("args,status", [
    (dict(M=-1), 1), (dict(K=0), 1), (dict(elem=2), 1), (dict(out_dtype=2), 1),
    (dict(block=16), 2), (dict(block=64), 2), (dict(K=96), 2), (dict(K=128, elem=1), 2),
    (dict(N=24), 2), (dict(a=None), 1), (dict(out=None), 1), (dict(a=A8), 1),
    (dict(bs=OUT + 2), 1), (dict(out=A8), 1), (dict(M=0, a=None, out=None), 0),
    (dict(N=0, b=None, out=None), 0), (dict(gain=OUT + 4), 1), (dict(K=1 << 23), 2),
    (dict(out=A8, out_dtype=1), 1),    # bf16 output is stored 16 bytes at a time
    (dict(N=(1 << 24) + 16), 2),       # N beyond MX_MATMUL_MAX_N
])
def test_mx_matmul_rejects_bad_arguments(args, status):
    lib = mxnorm.load()
    kw = dict(a=A16, as_=OUT, b=A16, bs=OUT, M=4, N=32, K=256, block=32, elem=0, gain=None,
              out_dtype=0, out=OUT)
    kw.update(args)
    assert lib.mx_matmul_fwd(kw["a"], kw["as_"], kw["b"], kw["bs"], kw["M"], kw["N"], kw["K"],
                             kw["block"], kw["elem"], kw["gain"], kw["out_dtype"], kw["out"],
                             None) == status
    if status:
        assert mxnorm.mx_last_error() != ""


@pytest.mark.parametrize("args,status", [
    (dict(R=-1), 1), (dict(C=0), 1), (dict(elem=2), 1), (dict(mode=3), 1), (dict(block=16), 2),
    (dict(R=48), 1), (dict(C=12), 1), (dict(x=None), 1), (dict(codes=None), 1), (dict(x=A8), 1),
    (dict(rho=OUT + 2), 1), (dict(R=0, x=None, codes=None, scales=None), 0),
    (dict(C=(1 << 23) + 8), 2), (dict(R=(1 << 31) + 32), 2),
])
def test_mx_cast_t_rejects_bad_arguments(args, status):
    lib = mxnorm.load()
    kw = dict(x=A16, rho=None, R=64, C=16, block=32, elem=0, mode=0, codes=OUT, scales=OUT)
    kw.update(args)
    assert lib.mx_cast_t_fwd(kw["x"], kw["rho"], kw["R"], kw["C"], kw["block"], kw["elem"],
                             kw["mode"], kw["codes"], kw["scales"], None) == status


def test_ste_workspace_size():
    # one float partial row of grad_gamma per workgroup of rpw rows, rpw =
    # clamp(ceil(T / 512), 4, 64)
    lib = mxnorm.load()
    assert lib.mxnorm_ste_bwd_workspace_bytes(0, 4096) == 0
    for T in (1, 4, 5, 32, 33, 2048, 4096, 4097, 32768, 100000):
        rpw = max(4, min(64, -(-T // 512)))
        assert lib.mxnorm_ste_bwd_workspace_bytes(T, 4096) == -(-T // rpw) * 4096 * 4, T


@pytest.mark.parametrize("args,status", [
    (dict(T=-1), 1), (dict(d=0), 1), (dict(d=12), 1), (dict(d=65536), 2), (dict(out=2), 1),
    (dict(x=None), 1), (dict(rho=None), 1), (dict(gx=None), 1), (dict(x=A8), 1),
    (dict(gamma=A8), 1), (dict(gg=OUT, ws=None), 1), (dict(gg=OUT, ws=OUT, wsb=16), 1),
    (dict(gg=OUT + 2), 1), (dict(T=0, x=None, gz=None, rho=None, gx=None), 0),
])
def test_ste_rejects_bad_arguments(args, status):
    lib = mxnorm.load()
    kw = dict(x=A16, gz=A16, gamma=None, rho=OUT, T=4, d=64, out=1, gx=OUT, gg=None, ws=None,
              wsb=0)
    kw.update(args)
    assert lib.mxnorm_ste_bwd(kw["x"], kw["gz"], kw["gamma"], kw["rho"], kw["T"], kw["d"],
                              kw["out"], kw["gx"], kw["gg"], kw["ws"], kw["wsb"], None) == status


def test_ste_noalloc_rejects_sizes_beyond_its_array():
    # the allocation-free entry point holds 32 MiB of grad_gamma workspace per
    # GPU; larger problems are refused on the host, before any HIP call
    lib = mxnorm.load()
    cap = lib.mxnorm_ste_bwd_noalloc_max_workspace()
    assert cap == 32 << 20
    assert lib.mxnorm_ste_bwd_workspace_bytes(32768, 16384) <= cap
    for T, d in ((131072, 8192), (32768, 32768), (1 << 20, 4096)):
        assert lib.mxnorm_ste_bwd_workspace_bytes(T, d) > cap
        assert lib.mxnorm_ste_bwd_noalloc(A16, A16, None, OUT, T, d, 1, OUT, OUT, None) == 2
        assert b"allocation-free" in lib.mx_last_error()


@pytest.mark.parametrize("args,status", [
    (dict(T=-1), 1), (dict(d=12), 1), (dict(d=65536), 2), (dict(out=2), 1), (dict(x=None), 1),
    (dict(rho=None), 1), (dict(gx=None), 1), (dict(x=A8), 1),
    (dict(T=0, x=None, gz=None, rho=None, gx=None), 0),
])
def test_ste_noalloc_rejects_bad_arguments(args, status):
    # without grad_gamma the scratch array is not touched, so every check
    # runs on the host
    lib = mxnorm.load()
    kw = dict(x=A16, gz=A16, gamma=None, rho=OUT, T=4, d=64, out=1, gx=OUT)
    kw.update(args)
    assert lib.mxnorm_ste_bwd_noalloc(kw["x"], kw["gz"], kw["gamma"], kw["rho"], kw["T"], kw["d"],
                                      kw["out"], kw["gx"], None, None) == status


@pytest.mark.parametrize("block", [16, 32, 64])
def test_postround_table_equals_oracle_table(block):
    # computed independently on both sides from the appendix's series; the
    # float-rounded tables agree exactly, so the kernels and the oracle take
    # rho~ from the same numbers
    import oracle
    xs, vs = mxnorm.mxnorm_postround_table(block)
    ox, ov = oracle.postround_lut(block)
    assert np.array_equal(xs, ox) and np.array_equal(vs, ov)


def test_postround_validation():
    lib = mxnorm.load()
    assert lib.mxnorm_postround_table(8, OUT, OUT) == 1
    # bad arguments only: every call below is rejected before any launch
    assert lib.mxnorm_postround_mx_fwd(A16, 4, 64, 8, 0, 1e-6, 0, OUT, OUT, None, None) == 1
    assert lib.mxnorm_postround_mx_fwd(A16, 4, 64, 32, 5, 1e-6, 0, OUT, OUT, None, None) == 1
    assert lib.mxnorm_postround_mx_fwd(A16, 4, 48, 32, 0, 1e-6, 0, OUT, OUT, None, None) == 1
    assert lib.mxnorm_postround_mx_fwd(A16, 4, 64, 32, 0, -1.0, 0, OUT, OUT, None, None) == 1
    assert lib.mxnorm_postround_mx_fwd(A16, 4, 64, 32, 0, 1e-6, 7, OUT, OUT, None, None) == 1
    assert lib.mxnorm_postround_mx_fwd(None, 0, 64, 32, 0, 1e-6, 0, None, None, None, None) == 0
