"""CPU oracle for MXNorm and RMSNorm + MX cast -- TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never imports, links or calls it, and the two share no
code.  The arithmetic lives in ``mx_oracle.c`` (plain C, one obviously-correct
step at a time, citing the paper's sections, equations and algorithms); this
module only builds that file with gcc and marshals numpy arrays to it.

Paper: "MXNorm: Reusing MXFP block scales for efficient tensor normalisation",
arXiv 2603.13180.  Algorithm 1 (RMSNorm + MXCast), Algorithm 2 (MXNorm),
Sec. 3.1-3.4, and the implementation appendix's mx_norm / mx_quantise.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mx_oracle.c")
_LIB = os.path.join(_HERE, "libmx_oracle.so")

SCALE_MODES = {"rceil": 0, "floor": 1}
ELEMS = {"e4m3": 0, "e2m1": 1}
MAX_D = 65536

_lib = None


def build(force=True):
    """Compile mx_oracle.c with gcc (IEEE arithmetic: no FMA contraction, no
    fast-math) into libmx_oracle.so next to it."""
    if not force and os.path.exists(_LIB):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-std=c99", "-ffp-contract=off",
           "-fno-fast-math", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    F = ctypes.c_float
    I = ctypes.c_int
    sig = {
        "mxo_e4m3_value": (ctypes.c_double, [ctypes.c_uint8]),
        "mxo_e2m1_value": (ctypes.c_double, [ctypes.c_uint8]),
        "mxo_e8m0_value": (ctypes.c_double, [ctypes.c_uint8]),
        "mxo_e4m3_encode": (ctypes.c_uint8, [F]),
        "mxo_e2m1_encode": (ctypes.c_uint8, [F]),
        "mxo_scale_exponent": (I, [F, I]),
        "mxo_coef": (F, [I, I]),
        "mxo_rms_inverse": (ctypes.c_double, [P, I64, F]),
        "mxo_rho_from_absmax": (ctypes.c_double, [P, I64, I, F, F]),
        "mxo_mxcast_mxfp8": (None, [P, I64, I64, I, P, P]),
        "mxo_mxnorm_mxfp8": (None, [P, I64, I64, I, F, F, I, P, P, P, P]),
        "mxo_rmsnorm_mxfp8": (None, [P, P, I64, I64, F, I, P, P, P, P]),
        "mxo_mxnorm_nvfp4": (None, [P, I64, I64, I, F, F, F, P, P, P, P]),
        "mxo_rmsnorm_nvfp4": (None, [P, P, I64, I64, F, F, P, P, P, P]),
        "mxo_mxnorm_default_global_scale": (ctypes.c_double, [I64, I, I, F]),
        "mxo_rmsnorm_default_global_scale": (ctypes.c_double, [I64, F]),
        "mxo_e4m3_encode_array": (None, [P, I64, P]),
        "mxo_e2m1_encode_array": (None, [P, I64, P]),
        "mxo_scale_exponent_array": (None, [P, I64, I, P]),
        "mxo_scale_exponent_fmt_array": (None, [P, I64, I, I, P]),
        "mxo_mxcast": (None, [P, I64, I64, I, I, I, P, P]),
        "mxo_mxnorm_mx": (None, [P, I64, I64, I, I, I, F, F, I, P, P, P, P]),
        "mxo_cast_given_rho": (None, [P, P, I64, I64, I, I, I, P, P]),
        "mxo_rmsnorm_mx": (None, [P, P, I64, I64, I, I, F, I, P, P, P, P]),
        "mxo_mxcast_gain": (None, [P, P, I64, I64, I, I, I, P, P]),
        "mxo_mxcast_t": (ctypes.c_int, [P, P, I64, I64, I, I, I, P, P]),
        "mxo_ste_bwd": (None, [P, P, P, P, I64, I64, P, P]),
        "mxo_postround_f": (ctypes.c_double, [ctypes.c_double, I]),
        "mxo_postround_finv_exact": (ctypes.c_double, [ctypes.c_double, I]),
        "mxo_postround_lut": (None, [I, P, P]),
        "mxo_postround_finv_lut": (ctypes.c_double, [ctypes.c_double, P, P]),
        "mxo_mxnorm_postround_mx": (None, [P, I64, I64, I, I, F, I, P, P, P, P]),
        "mxo_mx_matmul": (ctypes.c_int, [P, P, P, P, I64, I64, I64, I, I, P]),
        # host mirror of the library's forward boundary (status codes as the library's)
        "mxref_mxnorm_mxfp8_fwd": (I, [P, I64, I64, I, F, F, I, P, P, P]),
        "mxref_rmsnorm_mxfp8_fwd": (I, [P, P, I64, I64, F, I, P, P, P]),
        "mxref_mxnorm_nvfp4_fwd": (I, [P, I64, I64, I, F, F, F, P, P, P]),
        "mxref_rmsnorm_nvfp4_fwd": (I, [P, P, I64, I64, F, F, P, P, P]),
        "mxref_cast_given_rho": (I, [P, P, I64, I64, I, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _as_bf16_rows(x):
    x = np.ascontiguousarray(x)
    if x.dtype != np.uint16 or x.ndim != 2:
        raise TypeError("x must be a 2-D uint16 array of bf16 bit patterns")
    if x.shape[1] > MAX_D:
        raise ValueError("the oracle handles d <= %d" % MAX_D)
    return x


def _as_gamma(gamma, d):
    if gamma is None:
        return None
    g = np.ascontiguousarray(gamma)
    if g.dtype != np.uint16 or g.shape != (d,):
        raise TypeError("gamma must be a uint16 array of %d bf16 bit patterns" % d)
    return g


# ----------------------------------------------------------------- formats --

def e4m3_value(codes):
    lib = _load()
    return np.array([lib.mxo_e4m3_value(int(c)) for c in np.ravel(codes)]).reshape(np.shape(codes))


def e2m1_value(codes):
    lib = _load()
    return np.array([lib.mxo_e2m1_value(int(c)) for c in np.ravel(codes)]).reshape(np.shape(codes))


def e8m0_value(bytes_):
    lib = _load()
    return np.array([lib.mxo_e8m0_value(int(c)) for c in np.ravel(bytes_)]).reshape(np.shape(bytes_))


def e4m3_encode(v):
    v = np.ascontiguousarray(v, dtype=np.float32)
    out = np.empty(v.shape, np.uint8)
    _load().mxo_e4m3_encode_array(_ptr(v), v.size, _ptr(out))
    return out


def e2m1_encode(v):
    v = np.ascontiguousarray(v, dtype=np.float32)
    out = np.empty(v.shape, np.uint8)
    _load().mxo_e2m1_encode_array(_ptr(v), v.size, _ptr(out))
    return out


def scale_exponent(a, mode="rceil", elem="e4m3"):
    a = np.ascontiguousarray(a, dtype=np.float32)
    out = np.empty(a.shape, np.int32)
    _load().mxo_scale_exponent_fmt_array(_ptr(a), a.size, SCALE_MODES[mode], ELEMS[elem],
                                         _ptr(out))
    return out


def coef(B, p):
    """absmax_scale_factor(B, p) as a float32 constant."""
    return float(_load().mxo_coef(B, p))


def rms_inverse(x_f32, eps=0.0):
    x = np.ascontiguousarray(x_f32, dtype=np.float32)
    return float(_load().mxo_rms_inverse(_ptr(x), x.size, eps))


def rho_from_absmax(m_f32, p=2, coef_=None, eps=0.0, B=32):
    m = np.ascontiguousarray(m_f32, dtype=np.float32)
    c = coef(B, p) if coef_ is None else coef_
    return float(_load().mxo_rho_from_absmax(_ptr(m), m.size, p, c, eps))


def mxnorm_default_global_scale(d, B=16, p=2, coef_=None):
    c = coef(B, p) if coef_ is None else coef_
    return float(_load().mxo_mxnorm_default_global_scale(d, B, p, c))


def rmsnorm_default_global_scale(d, gamma_absmax=1.0):
    return float(_load().mxo_rmsnorm_default_global_scale(d, gamma_absmax))


# ------------------------------------------------------------------ casts --

def mxcast_mxfp8(y, mode="rceil"):
    """Plain MXFP8 cast (eq. blockscale / blockvals) of float32 y [T, d]."""
    y = np.ascontiguousarray(y, dtype=np.float32)
    T, d = y.shape
    if d % 32:
        raise ValueError("d must be a multiple of 32")
    codes = np.empty((T, d), np.uint8)
    scales = np.empty((T, d // 32), np.uint8)
    _load().mxo_mxcast_mxfp8(_ptr(y), T, d, SCALE_MODES[mode], _ptr(codes), _ptr(scales))
    return codes, scales


def mxnorm_mxfp8(x, p=2, coef_=None, eps=1e-6, mode="rceil"):
    """Algorithm 2 (MXNorm), E4M3 codes + E8M0 scales per 32-element block.
    Returns (codes [T,d] u8, scales [T,d/32] u8, rho32 [T] f32, rho64 [T] f64)."""
    x = _as_bf16_rows(x)
    T, d = x.shape
    if d % 32:
        raise ValueError("d must be a multiple of 32")
    c = coef(32, p) if coef_ is None else coef_
    codes = np.empty((T, d), np.uint8)
    scales = np.empty((T, d // 32), np.uint8)
    r32 = np.empty(T, np.float32)
    r64 = np.empty(T, np.float64)
    _load().mxo_mxnorm_mxfp8(_ptr(x), T, d, p, c, eps, SCALE_MODES[mode], _ptr(codes),
                             _ptr(scales), _ptr(r32), _ptr(r64))
    return codes, scales, r32, r64


def rmsnorm_mxfp8(x, gamma=None, eps=1e-6, mode="rceil"):
    """Algorithm 1 (RMSNorm, optional gain, then MXCast)."""
    x = _as_bf16_rows(x)
    T, d = x.shape
    if d % 32:
        raise ValueError("d must be a multiple of 32")
    g = _as_gamma(gamma, d)
    codes = np.empty((T, d), np.uint8)
    scales = np.empty((T, d // 32), np.uint8)
    r32 = np.empty(T, np.float32)
    r64 = np.empty(T, np.float64)
    _load().mxo_rmsnorm_mxfp8(_ptr(x), _ptr(g), T, d, eps, SCALE_MODES[mode], _ptr(codes),
                              _ptr(scales), _ptr(r32), _ptr(r64))
    return codes, scales, r32, r64


def mxnorm_nvfp4(x, s_g, p=2, coef_=None, eps=1e-6):
    """MXNorm with NVFP4 output: packed E2M1 codes [T, d/2], E4M3 scales [T, d/16]."""
    x = _as_bf16_rows(x)
    T, d = x.shape
    if d % 16:
        raise ValueError("d must be a multiple of 16")
    c = coef(16, p) if coef_ is None else coef_
    codes = np.empty((T, d // 2), np.uint8)
    scales = np.empty((T, d // 16), np.uint8)
    r32 = np.empty(T, np.float32)
    r64 = np.empty(T, np.float64)
    _load().mxo_mxnorm_nvfp4(_ptr(x), T, d, p, c, eps, s_g, _ptr(codes), _ptr(scales),
                             _ptr(r32), _ptr(r64))
    return codes, scales, r32, r64


def rmsnorm_nvfp4(x, s_g, gamma=None, eps=1e-6):
    x = _as_bf16_rows(x)
    T, d = x.shape
    if d % 16:
        raise ValueError("d must be a multiple of 16")
    g = _as_gamma(gamma, d)
    codes = np.empty((T, d // 2), np.uint8)
    scales = np.empty((T, d // 16), np.uint8)
    r32 = np.empty(T, np.float32)
    r64 = np.empty(T, np.float64)
    _load().mxo_rmsnorm_nvfp4(_ptr(x), _ptr(g), T, d, eps, s_g, _ptr(codes), _ptr(scales),
                              _ptr(r32), _ptr(r64))
    return codes, scales, r32, r64


# ------------------------------------------------------- generic MX casts --

def _mx_shapes(T, d, B, elem):
    if B not in (16, 32, 64) or d % B:
        raise ValueError("block must be 16, 32 or 64 and divide d")
    return ((T, d) if elem == "e4m3" else (T, d // 2)), (T, d // B)


def mxcast(y, B=32, elem="e4m3", mode="rceil"):
    """Plain MX cast (eq. blockscale / blockvals) of float32 y [T, d]."""
    y = np.ascontiguousarray(y, dtype=np.float32)
    T, d = y.shape
    cshape, sshape = _mx_shapes(T, d, B, elem)
    codes = np.empty(cshape, np.uint8)
    scales = np.empty(sshape, np.uint8)
    _load().mxo_mxcast(_ptr(y), T, d, B, ELEMS[elem], SCALE_MODES[mode], _ptr(codes),
                       _ptr(scales))
    return codes, scales


def mxnorm_mx(x, B=32, elem="e4m3", p=2, coef_=None, eps=1e-6, mode="rceil"):
    """Algorithm 2 with B-element blocks, E8M0 scales and E4M3 or E2M1 codes
    (E2M1 packed two per byte).  Returns (codes, scales, rho32, rho64)."""
    x = _as_bf16_rows(x)
    T, d = x.shape
    cshape, sshape = _mx_shapes(T, d, B, elem)
    c = coef(B, p) if coef_ is None else coef_
    codes = np.empty(cshape, np.uint8)
    scales = np.empty(sshape, np.uint8)
    r32 = np.empty(T, np.float32)
    r64 = np.empty(T, np.float64)
    _load().mxo_mxnorm_mx(_ptr(x), T, d, B, ELEMS[elem], p, c, eps, SCALE_MODES[mode],
                          _ptr(codes), _ptr(scales), _ptr(r32), _ptr(r64))
    return codes, scales, r32, r64


def cast_given_rho(x, rho32, B=32, elem="e4m3", mode="rceil"):
    """Algorithm 2's cast stage for a given float32 rho per row: scale bytes
    and codes of t = RN32(x rho) (the second part of the two-part contract).
    Returns (codes, scales)."""
    x = _as_bf16_rows(x)
    T, d = x.shape
    rho32 = np.ascontiguousarray(rho32, dtype=np.float32)
    if rho32.shape != (T,):
        raise ValueError("rho32 must be float32 [T]")
    cshape, sshape = _mx_shapes(T, d, B, elem)
    codes = np.empty(cshape, np.uint8)
    scales = np.empty(sshape, np.uint8)
    _load().mxo_cast_given_rho(_ptr(x), _ptr(rho32), T, d, B, ELEMS[elem], SCALE_MODES[mode],
                               _ptr(codes), _ptr(scales))
    return codes, scales


def rmsnorm_mx(x, gamma=None, B=32, elem="e4m3", eps=1e-6, mode="rceil"):
    """Algorithm 1 (RMSNorm, optional gain, then the plain MX cast)."""
    x = _as_bf16_rows(x)
    T, d = x.shape
    cshape, sshape = _mx_shapes(T, d, B, elem)
    g = _as_gamma(gamma, d)
    codes = np.empty(cshape, np.uint8)
    scales = np.empty(sshape, np.uint8)
    r32 = np.empty(T, np.float32)
    r64 = np.empty(T, np.float64)
    _load().mxo_rmsnorm_mx(_ptr(x), _ptr(g), T, d, B, ELEMS[elem], eps, SCALE_MODES[mode],
                           _ptr(codes), _ptr(scales), _ptr(r32), _ptr(r64))
    return codes, scales, r32, r64


# ----------------------------------------------------------- MXNormLinear --

def mxcast_gain(w, gamma=None, B=32, elem="e4m3", mode="rceil"):
    """MXCast(W gamma) of the implementation appendix's mx_norm_linear_forward:
    w bf16 bits [N, d], gamma bf16 bits [d] or None; the product in float."""
    w = _as_bf16_rows(w)
    N, d = w.shape
    cshape, sshape = _mx_shapes(N, d, B, elem)
    g = _as_gamma(gamma, d)
    codes = np.empty(cshape, np.uint8)
    scales = np.empty(sshape, np.uint8)
    _load().mxo_mxcast_gain(_ptr(w), _ptr(g), N, d, B, ELEMS[elem], SCALE_MODES[mode],
                            _ptr(codes), _ptr(scales))
    return codes, scales


def mx_matmul(a_codes, a_scales, b_codes, b_scales, K, B=32, elem="e4m3"):
    """H = dec(A) dec(B)^T in double (eq. mx-matmul), A [M, K], B [N, K]."""
    a_codes = np.ascontiguousarray(a_codes, np.uint8)
    b_codes = np.ascontiguousarray(b_codes, np.uint8)
    a_scales = np.ascontiguousarray(a_scales, np.uint8)
    b_scales = np.ascontiguousarray(b_scales, np.uint8)
    M, N = a_codes.shape[0], b_codes.shape[0]
    h = np.empty((M, N), np.float64)
    if _load().mxo_mx_matmul(_ptr(a_codes), _ptr(a_scales), _ptr(b_codes), _ptr(b_scales), M, N,
                             K, B, ELEMS[elem], _ptr(h)) != 0:
        raise MemoryError("mx_matmul: cannot allocate the decoded operand")
    return h


def mxnorm_linear(x, w, gamma=None, B=32, elem="e4m3", p=2, eps=1e-6, mode="rceil"):
    """The MXNormLinear forward, H = MXNorm(X) MXCast(W gamma)^T (Sec. 3.7),
    composed from the three oracle steps.  Returns (H, activation codes,
    activation scales, rho32)."""
    ac, as_, r32, _ = mxnorm_mx(x, B=B, elem=elem, p=p, eps=eps, mode=mode)
    wc, ws = mxcast_gain(w, gamma, B=B, elem=elem, mode=mode)
    return mx_matmul(ac, as_, wc, ws, x.shape[1], B=B, elem=elem), ac, as_, r32


# ------------------------------------------------------ MXNormLinear backward --

def mxcast_t(x, rho=None, B=32, elem="e4m3", mode="rceil"):
    """Column-wise MX cast of RN32(x * rho) (rho None: x): x bf16 bits [R, C]
    -> codes [C, R] (E4M3) or [C, R/2] (E2M1), scales [C, R/B] -- the cast
    along the token dimension the weight gradient needs (Sec. 3.7)."""
    x = np.ascontiguousarray(x)
    if x.dtype != np.uint16 or x.ndim != 2:
        raise TypeError("x must be a 2-D uint16 array of bf16 bit patterns")
    R, C = x.shape
    cshape, sshape = _mx_shapes(C, R, B, elem)
    r = None if rho is None else np.ascontiguousarray(rho, dtype=np.float32)
    if r is not None and r.shape != (R,):
        raise ValueError("rho must be float32 [R]")
    codes = np.empty(cshape, np.uint8)
    scales = np.empty(sshape, np.uint8)
    if _load().mxo_mxcast_t(_ptr(x), _ptr(r), R, C, B, ELEMS[elem], SCALE_MODES[mode],
                            _ptr(codes), _ptr(scales)) != 0:
        raise MemoryError("mxcast_t: cannot allocate a column buffer")
    return codes, scales


def ste_bwd(x, gz, gamma, rho):
    """Straight-through-estimator gradients (Sec. 3.7; the RMSNorm-gradient
    appendix with S = 1/rho~): x, gz bf16 bits [T, d], gamma bf16 bits [d] or
    None, rho float32 [T].  Returns (grad_x [T, d], grad_gamma [d]) in
    double."""
    x = np.ascontiguousarray(x)
    gz = np.ascontiguousarray(gz)
    if x.dtype != np.uint16 or gz.dtype != np.uint16 or x.shape != gz.shape or x.ndim != 2:
        raise TypeError("x and gz must be 2-D uint16 arrays of bf16 bits of one shape")
    T, d = x.shape
    g = _as_gamma(gamma, d)
    r = np.ascontiguousarray(rho, dtype=np.float32)
    if r.shape != (T,):
        raise ValueError("rho must be float32 [T]")
    gx = np.empty((T, d), np.float64)
    gg = np.empty(d, np.float64)
    _load().mxo_ste_bwd(_ptr(x), _ptr(gz), _ptr(g), _ptr(r), T, d, _ptr(gx), _ptr(gg))
    return gx, gg


# ------------------------------------------------------- post-round MXNorm --

POSTROUND_A = 64


def postround_f(sigma, B):
    """f_B(sigma) = E[max_i r(|X_i|)], X_i ~ N(0, sigma^2), i < B (the
    post-round appendix, with the difference read the right way round)."""
    return float(_load().mxo_postround_f(float(sigma), int(B)))


def postround_finv_exact(x, B):
    return float(_load().mxo_postround_finv_exact(float(x), int(B)))


def postround_lut(B):
    """(x_i, v_i), i = 0 .. A: x_i = RN32(2^(i/A)), v_i = RN32(f_B^-1(x_i))."""
    xs = np.empty(POSTROUND_A + 1, np.float32)
    vs = np.empty(POSTROUND_A + 1, np.float32)
    _load().mxo_postround_lut(int(B), _ptr(xs), _ptr(vs))
    return xs, vs


def postround_finv_lut(X, B, lut=None):
    xs, vs = postround_lut(B) if lut is None else lut
    return float(_load().mxo_postround_finv_lut(float(X), _ptr(xs), _ptr(vs)))


def mxnorm_postround_mx(x, B=32, elem="e4m3", eps=1e-6, mode="rceil"):
    """Post-round MXNorm: rho~ from the power-of-two-rounded block absmaxes
    through f^-1 (the post-round appendix), then Algorithm 2's cast.
    Returns (codes, scales, rho32, sigma64)."""
    x = _as_bf16_rows(x)
    T, d = x.shape
    cshape, sshape = _mx_shapes(T, d, B, elem)
    codes = np.empty(cshape, np.uint8)
    scales = np.empty(sshape, np.uint8)
    r32 = np.empty(T, np.float32)
    s64 = np.empty(T, np.float64)
    _load().mxo_mxnorm_postround_mx(_ptr(x), T, d, B, ELEMS[elem], eps, SCALE_MODES[mode],
                                    _ptr(codes), _ptr(scales), _ptr(r32), _ptr(s64))
    return codes, scales, r32, s64
