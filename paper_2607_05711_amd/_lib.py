"""Python binding of libfourtune (ctypes): argument marshalling only.

Each function has the name of the C entry point it calls (include/fourtune.h),
checks dtypes, devices and shapes of torch tensors, allocates missing outputs
with torch (device memory only) and enqueues the library call on the current
HIP stream.  All arithmetic runs in the library's gfx950 kernels; there is no
fallback: if the shared library is not built, every call raises.
"""
import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libfourtune.so")

FT_OK, FT_ERR_NULL, FT_ERR_SHAPE, FT_ERR_ALIGN, FT_ERR_UNSUPPORTED, FT_ERR_HIP = range(6)
FT_BF16, FT_F32 = 0, 1
FT_PROJ_COLS_BY_R, FT_PROJ_R_BY_COLS = 0, 1

EXPORTED = ("ft_quantize_blockwise", "ft_linear_fwd", "ft_linear_bwd_input", "ft_lora_grads",
            "ft_status_string", "ft_last_error")


FT_SCALE_FLOOR, FT_SCALE_NO_CLIP = 0, 1
FT_ROUND_NEAREST_EVEN, FT_ROUND_STOCHASTIC = 0, 1


class QuantMode(ctypes.Structure):
    """ft_quant_mode: scale rule, rounding, Philox seed and stream, per-row tile scales."""
    _fields_ = [("scale_rule", ctypes.c_int32), ("rounding", ctypes.c_int32), ("seed", ctypes.c_uint64),
                ("stream", ctypes.c_uint64), ("scales_per_row", ctypes.c_int32)]


class FourTuneError(RuntimeError):
    def __init__(self, status, detail):
        self.status = status
        super().__init__("%s (status %d): %s" % (status_string(status), status, detail))


_lib = None
_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32 = ctypes.c_int32


def load():
    """Load libfourtune.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise FileNotFoundError(
                "libfourtune.so is not built (expected at %s); run `python -m paper_2607_05711_amd.build` "
                "or __graft_entry__.build()" % LIB_PATH)
        from . import build as _build
        want = _build.source_hash()
        try:
            with open(_build.HASH) as fh:
                have = fh.read().strip()
        except OSError:
            have = None
        if have != want:
            raise RuntimeError(
                "libfourtune.so was not built from the sources in this tree (source hash %s, library built "
                "from %s); rebuild with `python -m paper_2607_05711_amd.build`" % (want[:16], (have or "?")[:16]))
        L = ctypes.CDLL(LIB_PATH)
        _Z = ctypes.c_size_t
        L.ft_quantize_blockwise.argtypes = [_P, _I64, _I64, _I32, _P, _P, _P, _I32, ctypes.c_int, _P, _P, _Z, _P]
        L.ft_quantize_blockwise_mode.argtypes = [_P, _I64, _I64, _I32, _P, _P, _P, _I32, ctypes.c_int, _P, _P, _Z,
                                                 ctypes.POINTER(QuantMode), _P]
        L.ft_quantize_blockwise_mode.restype = ctypes.c_int
        L.ft_quantize_nvfp4.argtypes = [_P, _I64, _I64, _I32, _P, _P, _P, _P]
        L.ft_quantize_nvfp4.restype = ctypes.c_int
        L.ft_linear_fwd_nvfp4.argtypes = [_P, _P, _P, _I64, _I64, _P, _P, _P, _I64, _P, _P]
        L.ft_linear_fwd_nvfp4.restype = ctypes.c_int
        L.ft_linear_bwd_input_nvfp4.argtypes = [_P, _P, _P, _I64, _I64, _P, _P, _P, _I64, _P, _P]
        L.ft_linear_bwd_input_nvfp4.restype = ctypes.c_int
        L.ft_quantize_workspace_size.argtypes = [_I64, _I64, _I32, _I32, ctypes.c_int]
        L.ft_quantize_workspace_size.restype = _Z
        L.ft_linear_fwd.argtypes = [_P, _P, _I64, _I64, _P, _P, _I64, _P, _I32, _P, _P, _P, ctypes.c_int, _P]
        L.ft_linear_bwd_input.argtypes = [_P, _P, _I64, _I64, _P, _P, _I64, _P, _I32, _P, _P, ctypes.c_int, _P]
        L.ft_lora_grads.argtypes = [_P, _I64, _I64, _P, _I64, _P, _P, _I64, _I32, _P, _P, _I32, _P, _Z, _P]
        L.ft_lora_grads_noalloc.argtypes = [_P, _I64, _I64, _P, _I64, _P, _P, _I64, _I32, _P, _P, _I32, _P]
        L.ft_lora_grads_noalloc.restype = ctypes.c_int
        L.ft_lora_grads_workspace_size.argtypes = [_I64, _I64, _I64, _I64, _I32]
        L.ft_lora_grads_workspace_size.restype = _Z
        L.ft_linear_fwd_gelu.argtypes = [_P, _P, _I64, _I64, _P, _P, _I64, _P, _I32, _P, _P,
                                         _P, _P, _P, _P, _P, _I32, _P, _P, _Z, _P]
        L.ft_linear_fwd_gelu.restype = ctypes.c_int
        L.ft_linear_fwd_gelu_workspace_size.argtypes = [_I64, _I64, _I32]
        L.ft_linear_fwd_gelu_workspace_size.restype = _Z
        L.ft_linear_bwd_input_dgelu.argtypes = [_P, _P, _I64, _I64, _P, _P, _I64, _P, _I32, _P,
                                                _P, _P, _P, _P, _P, _I32, _P, _P, _Z, _P]
        L.ft_linear_bwd_input_dgelu.restype = ctypes.c_int
        L.ft_linear_bwd_input_dgelu_workspace_size.argtypes = [_I64, _I64, _I32]
        L.ft_linear_bwd_input_dgelu_workspace_size.restype = _Z
        for f in ("ft_quantize_blockwise", "ft_linear_fwd", "ft_linear_bwd_input", "ft_lora_grads"):
            getattr(L, f).restype = ctypes.c_int
        L.ft_status_string.argtypes = [ctypes.c_int]
        L.ft_status_string.restype = ctypes.c_char_p
        L.ft_last_error.argtypes = []
        L.ft_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def status_string(status):
    return load().ft_status_string(int(status)).decode()


def _check(status):
    if status != FT_OK:
        raise FourTuneError(status, load().ft_last_error().decode())


def _ptr(t, offset_elems=0):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr() + offset_elems * t.element_size())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _need(t, name, dtype, device=None, ndim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if t.device.type != "cuda":
        raise ValueError("%s must be on a GPU, got %s" % (name, t.device))
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, expected %s" % (name, t.device, device))
    if ndim is not None and t.dim() != ndim:
        raise ValueError("%s must be %d-D, got shape %s" % (name, ndim, tuple(t.shape)))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t


def _workspace(nbytes, dev, workspace):
    """The caller's workspace (checked for size) or a new one of nbytes."""
    if nbytes == 0:
        return workspace
    if workspace is None:
        return torch.empty(((nbytes + 15) // 16) * 16, dtype=torch.uint8, device=dev)
    if workspace.numel() * workspace.element_size() < nbytes:
        raise ValueError("workspace of %d bytes, %d required" % (workspace.numel() * workspace.element_size(), nbytes))
    return workspace


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


def ft_quantize_blockwise(src, block_rows=1, proj=None, proj_layout=FT_PROJ_COLS_BY_R,
                          codes=None, scales=None, proj_out=None, workspace=None):
    """MXFP4-quantize bf16 src [rows, cols]; optionally fused down-projection.

    Returns (codes uint8 [rows, cols/2], scales uint8, proj_out fp32 [rows, R] or None).
    `workspace` (device tensor) holds the projection's partial sums; one of the
    size ft_quantize_workspace_size reports is made when it is not given.
    """
    return _quantize(src, block_rows, proj, proj_layout, codes, scales, proj_out, workspace, None)


def ft_quantize_blockwise_mode(src, block_rows=1, proj=None, proj_layout=FT_PROJ_COLS_BY_R, codes=None,
                               scales=None, proj_out=None, workspace=None, scale_rule=FT_SCALE_FLOOR,
                               rounding=FT_ROUND_NEAREST_EVEN, seed=0, stream=0, scales_per_row=False):
    """ft_quantize_blockwise with the numerics variants (no-clip scale rule,
    stochastic rounding keyed by (seed, stream), per-row tile scales for 2-D
    blocked activations)."""
    mode = QuantMode(scale_rule, rounding, seed, stream, 1 if scales_per_row else 0)
    return _quantize(src, block_rows, proj, proj_layout, codes, scales, proj_out, workspace, mode)


def _quantize(src, block_rows, proj, proj_layout, codes, scales, proj_out, workspace, mode):
    L = load()
    _need(src, "src", torch.bfloat16, ndim=2)
    dev = src.device
    rows, cols = src.shape
    srows = rows if (mode is not None and mode.scales_per_row) else rows // block_rows
    if codes is None:
        codes = torch.empty((rows, cols // 2), dtype=torch.uint8, device=dev)
    if scales is None:
        scales = torch.empty((srows, cols // 32), dtype=torch.uint8, device=dev)
    _need(codes, "codes", torch.uint8, dev)
    _need(scales, "scales", torch.uint8, dev)
    if codes.numel() * 2 != rows * cols or scales.numel() * 32 != srows * cols:
        raise ValueError("codes/scales size does not match src %s with block_rows %d" % (tuple(src.shape), block_rows))
    R = 0
    if proj is not None:
        _need(proj, "proj", torch.bfloat16, dev, ndim=2)
        R = proj.shape[1] if proj_layout == FT_PROJ_COLS_BY_R else proj.shape[0]
        other = proj.shape[0] if proj_layout == FT_PROJ_COLS_BY_R else proj.shape[1]
        if other != cols:
            raise ValueError("proj shape %s does not match cols %d" % (tuple(proj.shape), cols))
        if proj_out is None:
            proj_out = torch.empty((rows, R), dtype=torch.float32, device=dev)
        _need(proj_out, "proj_out", torch.float32, dev)
        if proj_out.shape != (rows, R):
            raise ValueError("proj_out must be [%d, %d]" % (rows, R))
    else:
        proj_out = None
    workspace = _workspace(L.ft_quantize_workspace_size(rows, cols, block_rows, R, proj_layout), dev, workspace)
    if mode is None:
        _check(L.ft_quantize_blockwise(_ptr(src), rows, cols, block_rows, _ptr(codes), _ptr(scales),
                                       _ptr(proj), R, proj_layout, _ptr(proj_out), _ptr(workspace),
                                       _nbytes(workspace), _stream(dev)))
    else:
        _check(L.ft_quantize_blockwise_mode(_ptr(src), rows, cols, block_rows, _ptr(codes), _ptr(scales),
                                            _ptr(proj), R, proj_layout, _ptr(proj_out), _ptr(workspace),
                                            _nbytes(workspace), ctypes.byref(mode), _stream(dev)))
    return codes, scales, proj_out


def ft_quantize_workspace_size(rows, cols, block_rows=1, R=0, proj_layout=FT_PROJ_COLS_BY_R):
    return int(load().ft_quantize_workspace_size(rows, cols, block_rows, R, proj_layout))


def ft_linear_fwd(xq, xs, wq, ws, K, P=None, U=None, bias=None, out_dtype=torch.bfloat16, y=None):
    """y[M, N] = DQ(xq) DQ(wq)^T + P U + bias (Eq. 2)."""
    L = load()
    dev = xq.device
    _need(xq, "xq", torch.uint8, ndim=2)
    _need(xs, "xs", torch.uint8, dev)
    _need(wq, "wq", torch.uint8, dev, ndim=2)
    _need(ws, "ws", torch.uint8, dev)
    M, N = xq.shape[0], wq.shape[0]
    if xq.shape[1] * 2 != K or wq.shape[1] * 2 != K or xs.numel() * 32 != M * K or ws.numel() * 1024 != N * K:
        raise ValueError("operand shapes do not match K=%d" % K)
    R = 0
    if P is not None or U is not None:
        _need(P, "P", torch.float32, dev, ndim=2)
        _need(U, "U", torch.bfloat16, dev, ndim=2)
        R = P.shape[1]
        if P.shape[0] != M or U.shape != (R, N):
            raise ValueError("P [M,R] / U [R,N] shapes mismatch")
    if bias is not None:
        _need(bias, "bias", torch.bfloat16, dev)
        if bias.numel() != N:
            raise ValueError("bias must have N elements")
    if y is None:
        y = torch.empty((M, N), dtype=out_dtype, device=dev)
    if y.dtype not in (torch.bfloat16, torch.float32) or y.shape != (M, N):
        raise ValueError("y must be bf16 or fp32 [M, N]")
    _need(y, "y", y.dtype, dev)
    _check(L.ft_linear_fwd(_ptr(xq), _ptr(xs), M, K, _ptr(wq), _ptr(ws), N, _ptr(P), R, _ptr(U), _ptr(bias),
                           _ptr(y), FT_F32 if y.dtype == torch.float32 else FT_BF16, _stream(dev)))
    return y


def ft_linear_bwd_input(gq, gs, wq, ws, K, Qp=None, D=None, out_dtype=torch.bfloat16, dx=None):
    """dx[M, K] = DQ(gq) DQ(wq) + Qp D^T (Eq. 3)."""
    L = load()
    dev = gq.device
    _need(gq, "gq", torch.uint8, ndim=2)
    _need(gs, "gs", torch.uint8, dev)
    _need(wq, "wq", torch.uint8, dev, ndim=2)
    _need(ws, "ws", torch.uint8, dev)
    M, N = gq.shape[0], wq.shape[0]
    if gq.shape[1] * 2 != N or wq.shape[1] * 2 != K or gs.numel() * 32 != M * N or ws.numel() * 1024 != N * K:
        raise ValueError("operand shapes do not match N=%d K=%d" % (N, K))
    R = 0
    if Qp is not None or D is not None:
        _need(Qp, "Qp", torch.float32, dev, ndim=2)
        _need(D, "D", torch.bfloat16, dev, ndim=2)
        R = Qp.shape[1]
        if Qp.shape[0] != M or D.shape != (K, R):
            raise ValueError("Qp [M,R] / D [K,R] shapes mismatch")
    if dx is None:
        dx = torch.empty((M, K), dtype=out_dtype, device=dev)
    if dx.dtype not in (torch.bfloat16, torch.float32) or dx.shape != (M, K):
        raise ValueError("dx must be bf16 or fp32 [M, K]")
    _need(dx, "dx", dx.dtype, dev)
    _check(L.ft_linear_bwd_input(_ptr(gq), _ptr(gs), M, N, _ptr(wq), _ptr(ws), K, _ptr(Qp), R, _ptr(D),
                                 _ptr(dx), FT_F32 if dx.dtype == torch.float32 else FT_BF16, _stream(dev)))
    return dx


def _mlp_outputs(M, C, dev, bf_a, bf_b, codes, scales):
    e = lambda t, shape, dt: torch.empty(shape, dtype=dt, device=dev) if t is None else t
    bf_a = e(bf_a, (M, C), torch.bfloat16)
    bf_b = e(bf_b, (M, C), torch.bfloat16)
    codes = e(codes, (M, C // 2), torch.uint8)
    scales = e(scales, (M, C // 32), torch.uint8)
    for t, n, dt, shape in ((bf_a, "z", torch.bfloat16, (M, C)), (bf_b, "output", torch.bfloat16, (M, C)),
                            (codes, "codes", torch.uint8, (M, C // 2)), (scales, "scales", torch.uint8, (M, C // 32))):
        _need(t, n, dt, dev)
        if tuple(t.shape) != shape:
            raise ValueError("%s must be %s" % (n, shape))
    return bf_a, bf_b, codes, scales


def ft_linear_fwd_gelu(xq, xs, wq, ws, K, P=None, U=None, bias=None, D2=None, z=None, h=None, hq=None, hs=None,
                       P2=None, workspace=None):
    """FC1 forward fused with FC2's input preparation (MLP fusion):
    z = bf16(y), h = bf16(GELU_tanh(z)), (hq, hs) = MXFP4(h), P2 = h D2.
    Returns (z, h, hq, hs, P2 or None)."""
    L = load()
    dev = xq.device
    _need(xq, "xq", torch.uint8, ndim=2)
    _need(xs, "xs", torch.uint8, dev)
    _need(wq, "wq", torch.uint8, dev, ndim=2)
    _need(ws, "ws", torch.uint8, dev)
    M, N = xq.shape[0], wq.shape[0]
    if xq.shape[1] * 2 != K or wq.shape[1] * 2 != K or xs.numel() * 32 != M * K or ws.numel() * 1024 != N * K:
        raise ValueError("operand shapes do not match K=%d" % K)
    R = 0
    if P is not None or U is not None:
        _need(P, "P", torch.float32, dev, ndim=2)
        _need(U, "U", torch.bfloat16, dev, ndim=2)
        R = P.shape[1]
        if P.shape[0] != M or U.shape != (R, N):
            raise ValueError("P [M,R] / U [R,N] shapes mismatch")
    if bias is not None:
        _need(bias, "bias", torch.bfloat16, dev)
        if bias.numel() != N:
            raise ValueError("bias must have N elements")
    z, h, hq, hs = _mlp_outputs(M, N, dev, z, h, hq, hs)
    R2 = 0
    if D2 is not None:
        _need(D2, "D2", torch.bfloat16, dev, ndim=2)
        if D2.shape[0] != N:
            raise ValueError("D2 must be [N, R2]")
        R2 = D2.shape[1]
        if P2 is None:
            P2 = torch.empty((M, R2), dtype=torch.float32, device=dev)
        _need(P2, "P2", torch.float32, dev)
        if P2.shape != (M, R2):
            raise ValueError("P2 must be [M, R2]")
    else:
        P2 = None
    workspace = _workspace(L.ft_linear_fwd_gelu_workspace_size(M, N, R2), dev, workspace)
    _check(L.ft_linear_fwd_gelu(_ptr(xq), _ptr(xs), M, K, _ptr(wq), _ptr(ws), N, _ptr(P), R, _ptr(U), _ptr(bias),
                                _ptr(z), _ptr(h), _ptr(hq), _ptr(hs), _ptr(D2), R2, _ptr(P2),
                                _ptr(workspace), _nbytes(workspace), _stream(dev)))
    return z, h, hq, hs, P2


def ft_linear_bwd_input_dgelu(gq, gs, wq, ws, K, z, Qp=None, D=None, U1=None, dz=None, dzq=None, dzs=None,
                              Qp1=None, workspace=None):
    """FC2 backward-input fused with FC1's gradient preparation:
    dz = bf16(dH * GELU_tanh'(z)) with dH = DQ(gq) DQ(wq) + Qp D^T in fp32,
    (dzq, dzs) = MXFP4(dz), Qp1 = dz U1^T.  Returns (dz, dzq, dzs, Qp1 or None)."""
    L = load()
    dev = gq.device
    _need(gq, "gq", torch.uint8, ndim=2)
    _need(gs, "gs", torch.uint8, dev)
    _need(wq, "wq", torch.uint8, dev, ndim=2)
    _need(ws, "ws", torch.uint8, dev)
    M, N = gq.shape[0], wq.shape[0]
    if gq.shape[1] * 2 != N or wq.shape[1] * 2 != K or gs.numel() * 32 != M * N or ws.numel() * 1024 != N * K:
        raise ValueError("operand shapes do not match N=%d K=%d" % (N, K))
    _need(z, "z", torch.bfloat16, dev)
    if tuple(z.shape) != (M, K):
        raise ValueError("z must be [M, K]")
    R = 0
    if Qp is not None or D is not None:
        _need(Qp, "Qp", torch.float32, dev, ndim=2)
        _need(D, "D", torch.bfloat16, dev, ndim=2)
        R = Qp.shape[1]
        if Qp.shape[0] != M or D.shape != (K, R):
            raise ValueError("Qp [M,R] / D [K,R] shapes mismatch")
    _, dz, dzq, dzs = _mlp_outputs(M, K, dev, z, dz, dzq, dzs)
    R1 = 0
    if U1 is not None:
        _need(U1, "U1", torch.bfloat16, dev, ndim=2)
        if U1.shape[1] != K:
            raise ValueError("U1 must be [R1, K]")
        R1 = U1.shape[0]
        if Qp1 is None:
            Qp1 = torch.empty((M, R1), dtype=torch.float32, device=dev)
        _need(Qp1, "Qp1", torch.float32, dev)
        if Qp1.shape != (M, R1):
            raise ValueError("Qp1 must be [M, R1]")
    else:
        Qp1 = None
    workspace = _workspace(L.ft_linear_bwd_input_dgelu_workspace_size(M, K, R1), dev, workspace)
    _check(L.ft_linear_bwd_input_dgelu(_ptr(gq), _ptr(gs), M, N, _ptr(wq), _ptr(ws), K, _ptr(Qp), R, _ptr(D),
                                       _ptr(z), _ptr(dz), _ptr(dzq), _ptr(dzs), _ptr(U1), R1, _ptr(Qp1),
                                       _ptr(workspace), _nbytes(workspace), _stream(dev)))
    return dz, dzq, dzs, Qp1


def ft_linear_fwd_gelu_workspace_size(M, N, R2):
    return int(load().ft_linear_fwd_gelu_workspace_size(M, N, R2))


def ft_linear_bwd_input_dgelu_workspace_size(M, K, R1):
    return int(load().ft_linear_bwd_input_dgelu_workspace_size(M, K, R1))


def ft_lora_grads_workspace_size(M, K, N, ld, r):
    return int(load().ft_lora_grads_workspace_size(M, K, N, ld, r))


def ft_lora_grads(x, dy, xa, dyb, r, col0=0, dA=None, dB=None, accumulate=False, workspace=None):
    """dA = x^T dyb[:, col0:col0+r] [K, r];  dB = xa[:, col0:col0+r]^T dy [r, N].

    xa and dyb are contiguous fp32 [M, ld] (normally P and Qp, with the adapter
    columns starting at col0 = r_s).
    """
    L = load()
    dev = x.device
    _need(x, "x", torch.bfloat16, ndim=2)
    _need(dy, "dy", torch.bfloat16, dev, ndim=2)
    _need(xa, "xa", torch.float32, dev, ndim=2)
    _need(dyb, "dyb", torch.float32, dev, ndim=2)
    M, K = x.shape
    N = dy.shape[1]
    ld = xa.shape[1]
    if dy.shape[0] != M or xa.shape[0] != M or dyb.shape != xa.shape or col0 + r > ld:
        raise ValueError("x [M,K], dy [M,N], xa/dyb [M,ld] shapes mismatch")
    if dA is None:
        dA = torch.empty((K, r), dtype=torch.float32, device=dev)
    if dB is None:
        dB = torch.empty((r, N), dtype=torch.float32, device=dev)
    _need(dA, "dA", torch.float32, dev)
    _need(dB, "dB", torch.float32, dev)
    if dA.shape != (K, r) or dB.shape != (r, N):
        raise ValueError("dA must be [K, r] and dB [r, N]")
    workspace = _workspace(L.ft_lora_grads_workspace_size(M, K, N, ld, r), dev, workspace)
    _check(L.ft_lora_grads(_ptr(x), M, K, _ptr(dy), N, _ptr(xa, col0), _ptr(dyb, col0), ld, r,
                           _ptr(dA), _ptr(dB), 1 if accumulate else 0, _ptr(workspace), _nbytes(workspace),
                           _stream(dev)))
    return dA, dB


def ft_lora_grads_noalloc(x, dy, xa, dyb, r, col0=0, dA=None, dB=None, accumulate=False):
    """ft_lora_grads without a workspace: the library's static device scratch
    holds the token-chunk partials (for callers that cannot allocate around
    the call; pass dA and dB to allocate nothing here either).  Calls that
    overlap on one GPU race on that scratch."""
    L = load()
    dev = x.device
    _need(x, "x", torch.bfloat16, ndim=2)
    _need(dy, "dy", torch.bfloat16, dev, ndim=2)
    _need(xa, "xa", torch.float32, dev, ndim=2)
    _need(dyb, "dyb", torch.float32, dev, ndim=2)
    M, K = x.shape
    N = dy.shape[1]
    ld = xa.shape[1]
    if dy.shape[0] != M or xa.shape[0] != M or dyb.shape != xa.shape or col0 + r > ld:
        raise ValueError("x [M,K], dy [M,N], xa/dyb [M,ld] shapes mismatch")
    if dA is None:
        dA = torch.empty((K, r), dtype=torch.float32, device=dev)
    if dB is None:
        dB = torch.empty((r, N), dtype=torch.float32, device=dev)
    _need(dA, "dA", torch.float32, dev)
    _need(dB, "dB", torch.float32, dev)
    if dA.shape != (K, r) or dB.shape != (r, N):
        raise ValueError("dA must be [K, r] and dB [r, N]")
    _check(L.ft_lora_grads_noalloc(_ptr(x), M, K, _ptr(dy), N, _ptr(xa, col0), _ptr(dyb, col0), ld, r,
                                   _ptr(dA), _ptr(dB), 1 if accumulate else 0, _stream(dev)))
    return dA, dB


def ft_quantize_nvfp4(src, block_rows=1):
    """NVFP4 emulation: (codes uint8 [rows, cols/2], E4M3 scales uint8
    [rows/block_rows, cols/16], tensor scale fp32 [1]) of bf16 src."""
    L = load()
    _need(src, "src", torch.bfloat16, ndim=2)
    dev = src.device
    rows, cols = src.shape
    codes = torch.empty((rows, cols // 2), dtype=torch.uint8, device=dev)
    scales = torch.empty((rows // block_rows, cols // 16), dtype=torch.uint8, device=dev)
    st = torch.empty((1,), dtype=torch.float32, device=dev)
    _check(L.ft_quantize_nvfp4(_ptr(src), rows, cols, block_rows, _ptr(codes), _ptr(scales), _ptr(st), _stream(dev)))
    return codes, scales, st


def ft_linear_fwd_nvfp4(xq, xs, xt, wq, ws, wt, K):
    """y [M, N] fp32 = xt wt DQ(xq) DQ(wq)^T on NVFP4 operands."""
    L = load()
    dev = xq.device
    M, N = xq.shape[0], wq.shape[0]
    y = torch.empty((M, N), dtype=torch.float32, device=dev)
    _check(L.ft_linear_fwd_nvfp4(_ptr(xq), _ptr(xs), _ptr(xt), M, K, _ptr(wq), _ptr(ws), _ptr(wt), N, _ptr(y),
                                 _stream(dev)))
    return y


def ft_linear_bwd_input_nvfp4(gq, gs, gt, wq, ws, wt, K):
    """dx [M, K] fp32 = gt wt DQ(gq) DQ(wq) on NVFP4 operands (w read transposed)."""
    L = load()
    dev = gq.device
    M, N = gq.shape[0], wq.shape[0]
    dx = torch.empty((M, K), dtype=torch.float32, device=dev)
    _check(L.ft_linear_bwd_input_nvfp4(_ptr(gq), _ptr(gs), _ptr(gt), M, N, _ptr(wq), _ptr(ws), _ptr(wt), K, _ptr(dx),
                                       _stream(dev)))
    return dx
