"""ctypes binding of libstreamref.so (include/streamref.h): a bandwidth
reference with the MXNorm kernel's traffic and access pattern and no
arithmetic, used by the benchmark as a practical-ceiling denominator."""
import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libstreamref.so")
MODES = {"mixed": 0, "read": 1, "write": 2, "nvfp4": 3}
_lib = None


def load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libstreamref.so is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_PATH)
        lib.mx_stream_reference.restype = ctypes.c_int
        lib.mx_stream_reference.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                            ctypes.c_void_p]
        lib.mx_stream_reference_ste.restype = ctypes.c_int
        lib.mx_stream_reference_ste.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                                ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
        lib.mx_stream_reference_transpose.restype = ctypes.c_int
        lib.mx_stream_reference_transpose.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                                                      ctypes.c_int64, ctypes.c_int64,
                                                      ctypes.c_void_p, ctypes.c_void_p,
                                                      ctypes.c_void_p]
        _lib = lib
    return _lib


def stream_reference(x, out, out_small, mode="mixed"):
    """x bf16 [T, d] (d % 512 == 0, d <= 4096); out uint8 [T, d] (mixed,
    write) or [T, d/2] (nvfp4); out_small uint8 [T, d/32] (mixed, write),
    [T, 16] (read) or [T, d/16] (nvfp4)."""
    T, d = x.shape
    st = load().mx_stream_reference(ctypes.c_void_p(x.data_ptr()), T, d,
                                    ctypes.c_void_p(out.data_ptr()),
                                    ctypes.c_void_p(out_small.data_ptr()), MODES[mode],
                                    ctypes.c_void_p(torch.cuda.current_stream(x.device).cuda_stream))
    if st != 0:
        raise RuntimeError("mx_stream_reference failed with status %d" % st)


def stream_reference_ste(x, grad_z, out):
    """x, grad_z, out: bf16 [T, d] (d % 512 == 0, d <= 4096): the straight-
    through estimator's traffic with no arithmetic."""
    T, d = x.shape
    st = load().mx_stream_reference_ste(ctypes.c_void_p(x.data_ptr()),
                                        ctypes.c_void_p(grad_z.data_ptr()), T, d,
                                        ctypes.c_void_p(out.data_ptr()),
                                        ctypes.c_void_p(torch.cuda.current_stream(x.device).cuda_stream))
    if st != 0:
        raise RuntimeError("mx_stream_reference_ste failed with status %d" % st)


def stream_reference_transpose(x, rho, out, out_small):
    """x bf16 [R, C] (R % 128 == 0, C % 256 == 0), rho float [R], out uint8
    [C, R], out_small uint8 [C, R/32]: the column cast's traffic and tiling
    with no arithmetic."""
    R, C = x.shape
    st = load().mx_stream_reference_transpose(
        ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(rho.data_ptr()), R, C,
        ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(out_small.data_ptr()),
        ctypes.c_void_p(torch.cuda.current_stream(x.device).cuda_stream))
    if st != 0:
        raise RuntimeError("mx_stream_reference_transpose failed with status %d" % st)
