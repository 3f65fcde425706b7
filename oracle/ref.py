"""ctypes wrapper around the fp64 C oracle (ft_oracle.c).

TEST INFRASTRUCTURE ONLY.  The oracle computes the paper's definitions
(FourTune, Sec. 3: Eq. (2) forward, Eq. (3) input gradient, the adapter
gradients of Sec. 3.2, block-wise 4-bit quantization) in double precision.
It shares nothing with the GPU library.  Arrays are numpy; bf16 tensors are
passed as their uint16 bit patterns.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "ft_oracle.c")
LIB = os.path.join(_HERE, "libft_oracle.so")

_c_i64 = ctypes.c_int64
_ptr = ctypes.c_void_p
_lib = None


def build():
    """Compile the oracle with gcc (fp64, no fast-math, OpenMP over rows)."""
    tmp = LIB + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-D_DEFAULT_SOURCE", "-fopenmp",
                           "-shared", "-fPIC", SRC, "-o", tmp, "-lm"])
    os.replace(tmp, LIB)


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        L = ctypes.CDLL(LIB)
        L.fto_e2m1_value.restype = ctypes.c_double
        L.fto_e2m1_value.argtypes = [ctypes.c_int]
        L.fto_e8m0_value.restype = ctypes.c_double
        L.fto_e8m0_value.argtypes = [ctypes.c_int]
        L.fto_quantize.argtypes = [_ptr, _c_i64, _c_i64, ctypes.c_int, _ptr, _ptr]
        L.fto_dequantize.argtypes = [_ptr, _ptr, _c_i64, _c_i64, ctypes.c_int, _ptr]
        L.fto_quantize_ex.argtypes = [_ptr, _c_i64, _c_i64, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                      ctypes.c_uint64, ctypes.c_uint64, _ptr, _ptr]
        L.fto_philox4x32_10.argtypes = [_ptr, _ptr, _ptr]
        L.fto_philox4x32_10.restype = None
        L.fto_sr_bits.argtypes = [ctypes.c_uint64, ctypes.c_uint64, _c_i64]
        L.fto_sr_bits.restype = ctypes.c_uint
        L.fto_e4m3_value.restype = ctypes.c_double
        L.fto_e4m3_value.argtypes = [ctypes.c_int]
        L.fto_nvfp4_tensor_scale.restype = ctypes.c_float
        L.fto_nvfp4_tensor_scale.argtypes = [_ptr, _c_i64]
        L.fto_quantize_nvfp4.argtypes = [_ptr, _c_i64, _c_i64, ctypes.c_int, ctypes.c_float, _ptr, _ptr]
        L.fto_dequantize_nvfp4.argtypes = [_ptr, _ptr, _c_i64, _c_i64, ctypes.c_int, ctypes.c_float, _ptr]
        L.fto_gemm_f64.argtypes = [_ptr, _ptr, _c_i64, _c_i64, _c_i64, ctypes.c_int, _ptr, _ptr]
        L.fto_proj.argtypes = [_ptr, _c_i64, _c_i64, _ptr, _c_i64, ctypes.c_int, _ptr, _ptr]
        L.fto_linear_fwd.argtypes = [_ptr, _ptr, _c_i64, _c_i64, _ptr, _ptr, _c_i64,
                                     _ptr, _ptr, _c_i64, _ptr, _ptr, _ptr, _ptr]
        L.fto_linear_bwd_input.argtypes = [_ptr, _ptr, _c_i64, _c_i64, _ptr, _ptr, _c_i64,
                                           _ptr, _ptr, _c_i64, _ptr, _ptr, _ptr]
        L.fto_lora_grads.argtypes = [_ptr, _c_i64, _c_i64, _ptr, _c_i64, _ptr, _ptr,
                                     _c_i64, _c_i64, _ptr, _ptr, _ptr, _ptr]
        L.fto_gelu.restype = ctypes.c_double
        L.fto_gelu.argtypes = [ctypes.c_double]
        L.fto_gelu_grad.restype = ctypes.c_double
        L.fto_gelu_grad.argtypes = [ctypes.c_double]
        L.fto_gelu_vec.argtypes = [_ptr, _c_i64, _ptr, ctypes.c_int]
        L.fto_num_threads.restype = ctypes.c_int
        L.fto_num_threads.argtypes = []
        for f in ("fto_quantize", "fto_quantize_ex", "fto_dequantize", "fto_quantize_nvfp4", "fto_dequantize_nvfp4",
                  "fto_gemm_f64", "fto_proj", "fto_linear_fwd",
                  "fto_linear_bwd_input", "fto_lora_grads"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def e2m1_value(code):
    return lib().fto_e2m1_value(int(code))


def e8m0_value(code):
    return lib().fto_e8m0_value(int(code))


def quantize(src_bits, block_rows=1):
    """bf16 bits [rows, cols] -> (codes uint8 [rows, cols/2], scales uint8)."""
    src = _c(src_bits, np.uint16)
    rows, cols = src.shape
    codes = np.zeros((rows, cols // 2), np.uint8)
    scales = np.zeros((rows // block_rows, cols // 32), np.uint8)
    rc = lib().fto_quantize(_p(src), rows, cols, block_rows, _p(codes), _p(scales))
    if rc != 0:
        raise ValueError("fto_quantize: unsupported shape %r / block_rows %d" % (src.shape, block_rows))
    return codes, scales


def quantize_ex(src_bits, block_rows=1, scale_rule=0, rounding=0, seed=0, stream=0):
    """quantize with the numerics variants: scale_rule 0 floor / 1 no-clip;
    rounding 0 nearest-even / 1 stochastic (Philox4x32-10 bits from seed and
    stream, element (r, c) of the matrix at counter index r * cols + c)."""
    src = _c(src_bits, np.uint16)
    rows, cols = src.shape
    codes = np.zeros((rows, cols // 2), np.uint8)
    scales = np.zeros((rows // block_rows, cols // 32), np.uint8)
    rc = lib().fto_quantize_ex(_p(src), rows, cols, block_rows, scale_rule, rounding, seed, stream,
                               _p(codes), _p(scales))
    if rc != 0:
        raise ValueError("fto_quantize_ex: unsupported arguments")
    return codes, scales


def philox4x32_10(ctr, key):
    """One Philox4x32-10 block: four 32-bit counter words, two key words."""
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, np.uint32)
    lib().fto_philox4x32_10(_p(c), _p(k), _p(out))
    return out


def sr_bits(seed, stream, idx):
    """The 16-bit uniform the stochastic rounding of element idx draws."""
    return int(lib().fto_sr_bits(seed, stream, idx))


def e4m3_value(code):
    return lib().fto_e4m3_value(int(code))


def nvfp4_tensor_scale(src_bits):
    src = _c(src_bits, np.uint16)
    return float(np.float32(lib().fto_nvfp4_tensor_scale(_p(src), src.size)))


def quantize_nvfp4(src_bits, block_rows=1, tensor_scale=None):
    """NVFP4: (codes [rows, cols/2], E4M3 scales [rows/block_rows, cols/16],
    FP32 tensor scale); block_rows 1 (1x16 blocks) or 16 (16x16 tiles)."""
    src = _c(src_bits, np.uint16)
    rows, cols = src.shape
    st = nvfp4_tensor_scale(src) if tensor_scale is None else float(np.float32(tensor_scale))
    codes = np.zeros((rows, cols // 2), np.uint8)
    scales = np.zeros((rows // block_rows, cols // 16), np.uint8)
    rc = lib().fto_quantize_nvfp4(_p(src), rows, cols, block_rows, st, _p(codes), _p(scales))
    if rc != 0:
        raise ValueError("fto_quantize_nvfp4: unsupported arguments")
    return codes, scales, st


def dequantize_nvfp4(codes, scales, st, cols, block_rows=1):
    codes = _c(codes, np.uint8)
    scales = _c(scales, np.uint8)
    rows = codes.shape[0]
    out = np.zeros((rows, cols), np.float64)
    rc = lib().fto_dequantize_nvfp4(_p(codes), _p(scales), rows, cols, block_rows, float(st), _p(out))
    if rc != 0:
        raise ValueError("fto_dequantize_nvfp4: unsupported arguments")
    return out


def gemm_f64(a, b, trans_b=True, want_s=True):
    """trans_b: y = a b^T (b [N, K]); else y = a b (b [K, N]); with S = sum |terms|."""
    a = _c(a, np.float64)
    b = _c(b, np.float64)
    M, K = a.shape
    N = b.shape[0] if trans_b else b.shape[1]
    y = np.zeros((M, N))
    s = np.zeros((M, N)) if want_s else None
    lib().fto_gemm_f64(_p(a), _p(b), M, N, K, 1 if trans_b else 0, _p(y), _p(s))
    return y, s


def dequantize(codes, scales, cols, block_rows=1):
    codes = _c(codes, np.uint8)
    scales = _c(scales, np.uint8)
    rows = codes.shape[0]
    out = np.zeros((rows, cols), np.float64)
    rc = lib().fto_dequantize(_p(codes), _p(scales), rows, cols, block_rows, _p(out))
    if rc != 0:
        raise ValueError("fto_dequantize: unsupported shape")
    return out


def proj(src_bits, proj_bits, layout):
    """layout 0: proj [cols, R], out = src.proj; layout 1: proj [R, cols], out = src.proj^T."""
    src = _c(src_bits, np.uint16)
    pr = _c(proj_bits, np.uint16)
    rows, cols = src.shape
    R = pr.shape[1] if layout == 0 else pr.shape[0]
    out = np.zeros((rows, R), np.float64)
    out_abs = np.zeros((rows, R), np.float64)
    lib().fto_proj(_p(src), rows, cols, _p(pr), R, layout, _p(out), _p(out_abs))
    return out, out_abs


def linear_fwd(xq, xs, wq, ws, K, P, U_bits, bias_bits=None, Pabs=None, want_s=True):
    xq = _c(xq, np.uint8); xs = _c(xs, np.uint8); wq = _c(wq, np.uint8); ws = _c(ws, np.uint8)
    M, N = xq.shape[0], wq.shape[0]
    R = 0 if P is None else P.shape[1]
    P = _c(P, np.float64) if R else np.zeros((M, 0))
    Pabs = _c(Pabs, np.float64)
    U = _c(U_bits, np.uint16) if R else np.zeros((0, N), np.uint16)
    bias = _c(bias_bits, np.uint16)
    y = np.zeros((M, N), np.float64)
    s = np.zeros((M, N), np.float64) if want_s else None
    rc = lib().fto_linear_fwd(_p(xq), _p(xs), M, K, _p(wq), _p(ws), N, _p(P), _p(Pabs), R,
                              _p(U), _p(bias), _p(y), _p(s))
    if rc != 0:
        raise ValueError("fto_linear_fwd failed (%d)" % rc)
    return y, s


def linear_bwd_input(gq, gs, wq, ws, K, Qp, D_bits, Qpabs=None, want_s=True):
    gq = _c(gq, np.uint8); gs = _c(gs, np.uint8); wq = _c(wq, np.uint8); ws = _c(ws, np.uint8)
    M, N = gq.shape[0], wq.shape[0]
    R = 0 if Qp is None else Qp.shape[1]
    Qp = _c(Qp, np.float64) if R else np.zeros((M, 0))
    Qpabs = _c(Qpabs, np.float64)
    D = _c(D_bits, np.uint16) if R else np.zeros((K, 0), np.uint16)
    dx = np.zeros((M, K), np.float64)
    s = np.zeros((M, K), np.float64) if want_s else None
    rc = lib().fto_linear_bwd_input(_p(gq), _p(gs), M, N, _p(wq), _p(ws), K, _p(Qp), _p(Qpabs),
                                    R, _p(D), _p(dx), _p(s))
    if rc != 0:
        raise ValueError("fto_linear_bwd_input failed (%d)" % rc)
    return dx, s


def lora_grads(x_bits, g_bits, xa, gbt, want_s=True):
    """dA = X^T gbt [K, r], dB = xa^T G [r, N]; xa, gbt are fp64 [M, r]."""
    x = _c(x_bits, np.uint16); g = _c(g_bits, np.uint16)
    xa = _c(xa, np.float64); gbt = _c(gbt, np.float64)
    M, K = x.shape
    N = g.shape[1]
    r = xa.shape[1]
    dA = np.zeros((K, r)); dB = np.zeros((r, N))
    sA = np.zeros((K, r)) if want_s else None
    sB = np.zeros((r, N)) if want_s else None
    lib().fto_lora_grads(_p(x), M, K, _p(g), N, _p(xa), _p(gbt), r, r, _p(dA), _p(dB), _p(sA), _p(sB))
    return dA, dB, sA, sB


def num_threads():
    return int(lib().fto_num_threads())


def gelu(z, derivative=False):
    z = _c(z, np.float64)
    out = np.zeros_like(z)
    lib().fto_gelu_vec(_p(z), z.size, _p(out), 1 if derivative else 0)
    return out
