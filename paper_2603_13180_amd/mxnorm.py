"""ctypes binding of libmxnorm.so (declared in include/mxnorm.h).

Argument marshalling only: each function checks tensor dtypes, devices and
shapes, allocates outputs with ``torch.empty`` when none are given, and calls
the C entry point of the same name on the current HIP stream.  Every step of
the computation runs in the library's HIP kernels.  There is no fallback: if
the library is missing, or a tensor is not on the GPU, a call raises.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmxnorm.so")

MX_OK, MX_EINVAL, MX_EUNSUPPORTED, MX_EHIP = 0, 1, 2, 3
SCALE_MODES = {"rceil": 0, "floor": 1}
OUT_DTYPES = {torch.float32: 0, torch.bfloat16: 1}
ELEMS = {"e4m3": 0, "e2m1": 1}
ABI_VERSION = 1
MAX_D = 32768

_lib = None


class MXNormError(RuntimeError):
    def __init__(self, status, detail):
        super().__init__("%s (%s)" % (detail, _status_name(status)))
        self.status = status


def _status_name(status):
    return {0: "MX_OK", 1: "MX_EINVAL", 2: "MX_EUNSUPPORTED", 3: "MX_EHIP"}.get(status, str(status))


def load():
    """Load libmxnorm.so and declare its signatures (no GPU work)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libmxnorm.so is not built (expected at %s); run "
                           "__graft_entry__.build()" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, I, F = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float
    sigs = {
        "mxnorm_mxfp8_fwd": (I, [P, I64, I64, I, F, F, I, P, P, P, P]),
        "rmsnorm_mxfp8_fwd": (I, [P, P, I64, I64, F, I, P, P, P, P]),
        "mxnorm_nvfp4_fwd": (I, [P, I64, I64, I, F, F, F, P, P, P, P]),
        "rmsnorm_nvfp4_fwd": (I, [P, P, I64, I64, F, F, P, P, P, P]),
        "mxnorm_mx_fwd": (I, [P, I64, I64, I, I, I, F, F, I, P, P, P, P]),
        "rmsnorm_mx_fwd": (I, [P, P, I64, I64, I, I, F, I, P, P, P, P]),
        "mxnorm_postround_mx_fwd": (I, [P, I64, I64, I, I, F, I, P, P, P, P]),
        "mxnorm_postround_table": (I, [I, P, P]),
        "mx_cast_fwd": (I, [P, P, I64, I64, I, I, I, P, P, P]),
        "mx_matmul_fwd": (I, [P, P, P, P, I64, I64, I64, I, I, P, I, P, P]),
        "mx_cast_t_fwd": (I, [P, P, I64, I64, I, I, I, P, P, P]),
        "mxnorm_ste_bwd_workspace_bytes": (ctypes.c_size_t, [I64, I64]),
        "mxnorm_ste_bwd": (I, [P, P, P, P, I64, I64, I, P, P, P, ctypes.c_size_t, P]),
        "mxnorm_ste_bwd_noalloc_max_workspace": (ctypes.c_size_t, []),
        "mxnorm_ste_bwd_noalloc": (I, [P, P, P, P, I64, I64, I, P, P, P]),
        "mxnorm_default_global_scale": (F, [I64, I, I, F]),
        "rmsnorm_default_global_scale": (F, [I64, F]),
        "mxnorm_coef": (F, [I, I]),
        "mx_status_str": (ctypes.c_char_p, [I]),
        "mx_last_error": (ctypes.c_char_p, []),
        "mxnorm_abi_version": (I, []),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if lib.mxnorm_abi_version() != ABI_VERSION:
        raise RuntimeError("libmxnorm.so ABI version %d, binding expects %d"
                           % (lib.mxnorm_abi_version(), ABI_VERSION))
    _lib = lib
    return lib


def _check(status):
    if status != MX_OK:
        raise MXNormError(status, load().mx_last_error().decode() or "error")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _input(x):
    if not isinstance(x, torch.Tensor) or x.dtype != torch.bfloat16 or x.dim() != 2:
        raise TypeError("x must be a 2-D torch.bfloat16 tensor [T, d]")
    if not x.is_cuda:
        raise RuntimeError("x must be on the GPU: libmxnorm has no CPU path")
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    return x.shape[0], x.shape[1]


def _gamma(gamma, x):
    if gamma is None:
        return None
    if gamma.dtype != torch.bfloat16 or gamma.shape != (x.shape[1],) or gamma.device != x.device:
        raise TypeError("gamma must be a bfloat16 [d] tensor on x's device")
    return gamma.contiguous()


def _out(t, shape, dtype, device):
    if t is None:
        return torch.empty(shape, dtype=dtype, device=device)
    if t.shape != shape or t.dtype != dtype or t.device != device or not t.is_contiguous():
        raise ValueError("output tensor must be contiguous %s %s on %s" % (dtype, shape, device))
    return t


def mxnorm_mxfp8_fwd(x, p=2, coef=0.0, eps=1e-6, scale_mode="rceil",
                     codes=None, scales=None, rho=None, want_rho=True):
    """MXNorm (Algorithm 2) with MXFP8 output.

    Returns (codes uint8 [T, d] E4M3, scales uint8 [T, d/32] E8M0,
    rho float32 [T] or None)."""
    T, d = _input(x)
    codes = _out(codes, (T, d), torch.uint8, x.device)
    scales = _out(scales, (T, d // 32), torch.uint8, x.device)
    if want_rho:
        rho = _out(rho, (T,), torch.float32, x.device)
    _check(load().mxnorm_mxfp8_fwd(_ptr(x), T, d, p, coef, eps, SCALE_MODES[scale_mode],
                                   _ptr(codes), _ptr(scales), _ptr(rho) if want_rho else None,
                                   _stream(x.device)))
    return codes, scales, (rho if want_rho else None)


def rmsnorm_mxfp8_fwd(x, gamma=None, eps=1e-6, scale_mode="rceil",
                      codes=None, scales=None, rho=None, want_rho=True):
    """RMSNorm (+ optional gain) then MXFP8 cast (Algorithm 1)."""
    T, d = _input(x)
    g = _gamma(gamma, x)
    codes = _out(codes, (T, d), torch.uint8, x.device)
    scales = _out(scales, (T, d // 32), torch.uint8, x.device)
    if want_rho:
        rho = _out(rho, (T,), torch.float32, x.device)
    _check(load().rmsnorm_mxfp8_fwd(_ptr(x), _ptr(g), T, d, eps, SCALE_MODES[scale_mode],
                                    _ptr(codes), _ptr(scales), _ptr(rho) if want_rho else None,
                                    _stream(x.device)))
    return codes, scales, (rho if want_rho else None)


def mxnorm_nvfp4_fwd(x, global_scale=None, p=2, coef=0.0, eps=1e-6,
                     codes=None, scales=None, rho=None, want_rho=True):
    """MXNorm with NVFP4 output.  global_scale None selects the Lemma-2
    default.  Returns (packed E2M1 codes uint8 [T, d/2], E4M3 scales uint8
    [T, d/16], rho)."""
    T, d = _input(x)
    if global_scale is None:
        global_scale = mxnorm_default_global_scale(d, 16, p, coef)
    codes = _out(codes, (T, d // 2), torch.uint8, x.device)
    scales = _out(scales, (T, d // 16), torch.uint8, x.device)
    if want_rho:
        rho = _out(rho, (T,), torch.float32, x.device)
    _check(load().mxnorm_nvfp4_fwd(_ptr(x), T, d, p, coef, eps, global_scale, _ptr(codes),
                                   _ptr(scales), _ptr(rho) if want_rho else None,
                                   _stream(x.device)))
    return codes, scales, (rho if want_rho else None)


def rmsnorm_nvfp4_fwd(x, gamma=None, global_scale=None, eps=1e-6,
                      codes=None, scales=None, rho=None, want_rho=True):
    T, d = _input(x)
    g = _gamma(gamma, x)
    if global_scale is None:
        if g is not None:
            raise ValueError("pass global_scale when gamma is given; "
                             "rmsnorm_default_global_scale(d, max|gamma|) is the Lemma-1 default")
        global_scale = rmsnorm_default_global_scale(d, 1.0)
    codes = _out(codes, (T, d // 2), torch.uint8, x.device)
    scales = _out(scales, (T, d // 16), torch.uint8, x.device)
    if want_rho:
        rho = _out(rho, (T,), torch.float32, x.device)
    _check(load().rmsnorm_nvfp4_fwd(_ptr(x), _ptr(g), T, d, eps, global_scale, _ptr(codes),
                                    _ptr(scales), _ptr(rho) if want_rho else None,
                                    _stream(x.device)))
    return codes, scales, (rho if want_rho else None)


def _mx_out_shapes(T, d, block, elem):
    if block not in (16, 32, 64) or elem not in ELEMS:
        raise ValueError("block must be 16, 32 or 64 and elem 'e4m3' or 'e2m1'")
    return ((T, d) if elem == "e4m3" else (T, d // 2)), (T, d // block)


def mxnorm_mx_fwd(x, block=32, elem="e4m3", p=2, coef=0.0, eps=1e-6, scale_mode="rceil",
                  codes=None, scales=None, rho=None, want_rho=True):
    """MXNorm with a general MX output: E8M0 scales per `block` elements and
    E4M3 or E2M1 (packed two per byte) codes."""
    T, d = _input(x)
    cs, ss = _mx_out_shapes(T, d, block, elem)
    codes = _out(codes, cs, torch.uint8, x.device)
    scales = _out(scales, ss, torch.uint8, x.device)
    if want_rho:
        rho = _out(rho, (T,), torch.float32, x.device)
    _check(load().mxnorm_mx_fwd(_ptr(x), T, d, block, ELEMS[elem], p, coef, eps,
                                SCALE_MODES[scale_mode], _ptr(codes), _ptr(scales),
                                _ptr(rho) if want_rho else None, _stream(x.device)))
    return codes, scales, (rho if want_rho else None)


def mxnorm_postround_mx_fwd(x, block=32, elem="e4m3", eps=1e-6, scale_mode="rceil",
                            codes=None, scales=None, rho=None, want_rho=True):
    """Post-round MXNorm (the post-round appendix): rho~ from the block
    absmaxes rounded down to powers of two, through the inverse of
    f(sigma) = E[max r(|X|)], then the MX cast of Algorithm 2."""
    T, d = _input(x)
    cs, ss = _mx_out_shapes(T, d, block, elem)
    codes = _out(codes, cs, torch.uint8, x.device)
    scales = _out(scales, ss, torch.uint8, x.device)
    if want_rho:
        rho = _out(rho, (T,), torch.float32, x.device)
    _check(load().mxnorm_postround_mx_fwd(_ptr(x), T, d, block, ELEMS[elem], eps,
                                          SCALE_MODES[scale_mode], _ptr(codes), _ptr(scales),
                                          _ptr(rho) if want_rho else None, _stream(x.device)))
    return codes, scales, (rho if want_rho else None)


def mxnorm_postround_table(block):
    """The library's post-round table: (x, v) float32 arrays of 65 points."""
    import numpy as np
    xs = np.empty(65, np.float32)
    vs = np.empty(65, np.float32)
    _check(load().mxnorm_postround_table(block, xs.ctypes.data_as(ctypes.c_void_p),
                                         vs.ctypes.data_as(ctypes.c_void_p)))
    return xs, vs


def rmsnorm_mx_fwd(x, gamma=None, block=32, elem="e4m3", eps=1e-6, scale_mode="rceil",
                   codes=None, scales=None, rho=None, want_rho=True):
    """RMSNorm (+ optional gain) then the general MX cast."""
    T, d = _input(x)
    g = _gamma(gamma, x)
    cs, ss = _mx_out_shapes(T, d, block, elem)
    codes = _out(codes, cs, torch.uint8, x.device)
    scales = _out(scales, ss, torch.uint8, x.device)
    if want_rho:
        rho = _out(rho, (T,), torch.float32, x.device)
    _check(load().rmsnorm_mx_fwd(_ptr(x), _ptr(g), T, d, block, ELEMS[elem], eps,
                                 SCALE_MODES[scale_mode], _ptr(codes), _ptr(scales),
                                 _ptr(rho) if want_rho else None, _stream(x.device)))
    return codes, scales, (rho if want_rho else None)


def mx_cast_fwd(x, gamma=None, block=32, elem="e4m3", scale_mode="rceil",
                codes=None, scales=None):
    """Plain MX cast of x (or RN(x * gamma)), no normalisation.  With x a
    weight [N, d] and gamma the norm gain this is the gain-folded weight cast
    of the MXNormLinear forward (Sec. 3.7)."""
    T, d = _input(x)
    g = _gamma(gamma, x)
    cs, ss = _mx_out_shapes(T, d, block, elem)
    codes = _out(codes, cs, torch.uint8, x.device)
    scales = _out(scales, ss, torch.uint8, x.device)
    _check(load().mx_cast_fwd(_ptr(x), _ptr(g), T, d, block, ELEMS[elem],
                              SCALE_MODES[scale_mode], _ptr(codes), _ptr(scales),
                              _stream(x.device)))
    return codes, scales


def _mx_operand(codes, scales, K, block, elem, name):
    cw = K if elem == "e4m3" else K // 2
    for t, shape_ok in ((codes, codes.dim() == 2 and codes.shape[1] == cw),
                        (scales, scales.dim() == 2 and scales.shape[1] == K // block)):
        if t.dtype != torch.uint8 or not t.is_cuda or not t.is_contiguous() or not shape_ok:
            raise ValueError("%s: codes must be contiguous uint8 [rows, %d] and scales [rows, %d] "
                             "on the GPU" % (name, cw, K // block))
    if codes.shape[0] != scales.shape[0]:
        raise ValueError("%s: codes and scales disagree on the row count" % name)
    return codes.shape[0]


def mx_matmul_fwd(a_codes, a_scales, b_codes, b_scales, K, block=32, elem="e4m3",
                  out_dtype=torch.float32, out=None, b_gain=None):
    """H = dec(A) dec(B)^T on the block-scaled matrix cores (Sec. 3.7 eq.
    (mx-matmul)).  A: MX codes/scales [M, .] along K; B: [N, .].  b_gain
    (bf16 [N]) multiplies column n of H after the product.  Returns H [M, N]
    in out_dtype (float32 or bfloat16)."""
    if elem not in ELEMS or out_dtype not in OUT_DTYPES:
        raise ValueError("elem must be 'e4m3' or 'e2m1', out_dtype float32 or bfloat16")
    M = _mx_operand(a_codes, a_scales, K, block, elem, "A")
    N = _mx_operand(b_codes, b_scales, K, block, elem, "B")
    if b_gain is not None and (b_gain.dtype != torch.bfloat16 or b_gain.shape != (N,) or
                               b_gain.device != a_codes.device or not b_gain.is_contiguous()):
        raise ValueError("b_gain must be a contiguous bfloat16 [N] tensor on the GPU")
    out = _out(out, (M, N), out_dtype, a_codes.device)
    _check(load().mx_matmul_fwd(_ptr(a_codes), _ptr(a_scales), _ptr(b_codes), _ptr(b_scales),
                                M, N, K, block, ELEMS[elem], _ptr(b_gain),
                                OUT_DTYPES[out_dtype], _ptr(out), _stream(a_codes.device)))
    return out


def mxnorm_linear_fwd(x, w_codes, w_scales, block=32, elem="e4m3", p=2, coef=0.0, eps=1e-6,
                      scale_mode="rceil", out_dtype=torch.bfloat16):
    """The MXNormLinear forward H = MXNorm(X) MXCast(W gamma)^T (Sec. 3.7):
    MXNorm of the activations, then the MX matmul with a weight cast once by
    mx_cast_fwd(W, gamma).  Returns (H, rho~)."""
    codes, scales, rho = mxnorm_mx_fwd(x, block=block, elem=elem, p=p, coef=coef, eps=eps,
                                       scale_mode=scale_mode)
    h = mx_matmul_fwd(codes, scales, w_codes, w_scales, x.shape[1], block=block, elem=elem,
                      out_dtype=out_dtype)
    return h, rho


def mx_cast_t_fwd(x, rho=None, block=32, elem="e4m3", scale_mode="rceil", codes=None,
                  scales=None):
    """Column-wise MX cast (Sec. 3.7): the MX encoding of (rho[:, None] * x)^T,
    blocked along x's rows.  x bf16 [R, C] -> codes [C, R] (E4M3) or
    [C, R/2] (E2M1), scales [C, R/32]."""
    R, C = _input(x)
    if rho is not None and (rho.dtype != torch.float32 or rho.shape != (R,) or
                            rho.device != x.device or not rho.is_contiguous()):
        raise ValueError("rho must be a contiguous float32 [R] tensor on x's device")
    if elem not in ELEMS:
        raise ValueError("elem must be 'e4m3' or 'e2m1'")
    codes = _out(codes, (C, R) if elem == "e4m3" else (C, R // 2), torch.uint8, x.device)
    scales = _out(scales, (C, R // block), torch.uint8, x.device)
    _check(load().mx_cast_t_fwd(_ptr(x), _ptr(rho), R, C, block, ELEMS[elem],
                                SCALE_MODES[scale_mode], _ptr(codes), _ptr(scales),
                                _stream(x.device)))
    return codes, scales


def mxnorm_ste_bwd(x, grad_z, gamma, rho, out_dtype=torch.bfloat16, want_grad_gamma=True,
                   grad_x=None, grad_gamma=None, workspace=None):
    """The straight-through estimator of the MXNorm backward (Sec. 3.7; the
    RMSNorm-gradient appendix with S = 1/rho~).  x, grad_z bf16 [T, d];
    gamma bf16 [d] or None; rho float32 [T] from the forward.  Returns
    (grad_x [T, d] in out_dtype, grad_gamma float32 [d] or None)."""
    T, d = _input(x)
    if grad_z.dtype != torch.bfloat16 or grad_z.shape != x.shape or grad_z.device != x.device \
            or not grad_z.is_contiguous():
        raise ValueError("grad_z must be a contiguous bfloat16 tensor shaped like x")
    g = _gamma(gamma, x)
    if rho.dtype != torch.float32 or rho.shape != (T,) or rho.device != x.device:
        raise ValueError("rho must be float32 [T] on x's device")
    if out_dtype not in OUT_DTYPES:
        raise ValueError("out_dtype must be float32 or bfloat16")
    lib = load()
    grad_x = _out(grad_x, (T, d), out_dtype, x.device)
    ws_bytes = 0
    if want_grad_gamma:
        grad_gamma = _out(grad_gamma, (d,), torch.float32, x.device)
        ws_bytes = int(lib.mxnorm_ste_bwd_workspace_bytes(T, d))
        if workspace is None:
            workspace = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=x.device)
        elif workspace.numel() * workspace.element_size() < ws_bytes:
            raise ValueError("workspace smaller than mxnorm_ste_bwd_workspace_bytes(T, d)")
        ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib.mxnorm_ste_bwd(_ptr(x), _ptr(grad_z), _ptr(g), _ptr(rho.contiguous()), T, d,
                              OUT_DTYPES[out_dtype], _ptr(grad_x),
                              _ptr(grad_gamma) if want_grad_gamma else None,
                              _ptr(workspace) if want_grad_gamma else None, ws_bytes,
                              _stream(x.device)))
    return grad_x, (grad_gamma if want_grad_gamma else None)


def mxnorm_ste_bwd_noalloc(x, grad_z, gamma, rho, grad_x, grad_gamma=None):
    """mxnorm_ste_bwd through the library's allocation-free entry point: the
    grad_gamma workspace is the library's static device array, so neither the
    library nor this call allocates.  The caller passes the outputs: grad_x
    [T, d] (float32 or bfloat16, its dtype selects the output type) and
    grad_gamma float32 [d] or None.  Calls that overlap in time on one GPU
    share that array and race."""
    T, d = _input(x)
    if grad_z.dtype != torch.bfloat16 or grad_z.shape != x.shape or grad_z.device != x.device \
            or not grad_z.is_contiguous():
        raise ValueError("grad_z must be a contiguous bfloat16 tensor shaped like x")
    g = _gamma(gamma, x)
    if rho.dtype != torch.float32 or rho.shape != (T,) or rho.device != x.device \
            or not rho.is_contiguous():
        raise ValueError("rho must be contiguous float32 [T] on x's device")
    if grad_x.dtype not in OUT_DTYPES or grad_x.shape != x.shape or grad_x.device != x.device \
            or not grad_x.is_contiguous():
        raise ValueError("grad_x must be a contiguous float32 or bfloat16 tensor shaped like x")
    if grad_gamma is not None and (grad_gamma.dtype != torch.float32 or grad_gamma.shape != (d,)
                                   or grad_gamma.device != x.device):
        raise ValueError("grad_gamma must be float32 [d] on x's device")
    _check(load().mxnorm_ste_bwd_noalloc(_ptr(x), _ptr(grad_z), _ptr(g), _ptr(rho), T, d,
                                         OUT_DTYPES[grad_x.dtype], _ptr(grad_x),
                                         _ptr(grad_gamma) if grad_gamma is not None else None,
                                         _stream(x.device)))
    return grad_x, grad_gamma


def mxnorm_linear_bwd(grad_h, x, rho, gamma, w, block=32, elem="e4m3",
                      grad_x_dtype=torch.bfloat16):
    """The MXNormLinear backward (Sec. 3.7; the implementation appendix's
    mx_norm_linear_backward), every product and cast in the library:
      grad_Z = MXCast(grad_H) MXCast_N(W)            (W blocked along N)
      grad_X, grad_gamma = STE(X, grad_Z, gamma, rho~)
      grad_W = (MXCast(grad_H^T) MXCast(rho~ X)^T) . gamma
    grad_h bf16 [T, N], x bf16 [T, d], rho float32 [T], gamma bf16 [d],
    w bf16 [N, d].  Returns (grad_x, grad_gamma float32 [d], grad_w float32
    [N, d])."""
    T, N = grad_h.shape
    d = x.shape[1]
    if w.shape != (N, d):
        raise ValueError("w must be [N, d]")
    gh_c, gh_s = mx_cast_fwd(grad_h, None, block=block, elem=elem)
    wt_c, wt_s = mx_cast_t_fwd(w, None, block=block, elem=elem)
    grad_z = mx_matmul_fwd(gh_c, gh_s, wt_c, wt_s, N, block=block, elem=elem,
                           out_dtype=torch.bfloat16)
    grad_x, grad_gamma = mxnorm_ste_bwd(x, grad_z, gamma, rho, out_dtype=grad_x_dtype)
    ght_c, ght_s = mx_cast_t_fwd(grad_h, None, block=block, elem=elem)
    xt_c, xt_s = mx_cast_t_fwd(x, rho, block=block, elem=elem)
    grad_w = mx_matmul_fwd(ght_c, ght_s, xt_c, xt_s, T, block=block, elem=elem,
                           out_dtype=torch.float32, b_gain=gamma)
    return grad_x, grad_gamma, grad_w


def mxnorm_default_global_scale(d, block=16, p=2, coef=0.0):
    return float(load().mxnorm_default_global_scale(d, block, p, coef))


def rmsnorm_default_global_scale(d, gamma_absmax=1.0):
    return float(load().rmsnorm_default_global_scale(d, gamma_absmax))


def mxnorm_coef(block, p):
    return float(load().mxnorm_coef(block, p))


def mx_status_str(status):
    return load().mx_status_str(status).decode()


def mx_last_error():
    return load().mx_last_error().decode()
