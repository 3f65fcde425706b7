"""Parity of the NVFP4 emulation (ft_quantize_nvfp4, ft_linear_fwd_nvfp4,
ft_linear_bwd_input_nvfp4) against the fp64 oracle, through the C ABI.

NVFP4 is the format FourTune Sec. 3.1 names (E4M3 scales per 16 elements, an
FP32 tensor scale, 16x16 weight tiles, Sec. 4.3).  Bars: codes, E4M3 scales
and the tensor scale bit-exact; GEMM outputs (fp32) within 1e-5 * S of the
oracle's product of the dequantized operands.  Plus the accuracy cross-check
of the two formats on the FLUX QKV layer's forward product.
"""
import numpy as np
import pytest
import torch

from oracle import ref
from paper_2607_05711_amd import _lib, gen
from tests._helpers import f64, random_rows

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(DEV)


def host(t):
    return t.cpu().numpy()


@pytest.mark.parametrize("block_rows", [1, 16])
@pytest.mark.parametrize("rows,cols,kind", [(16, 16, "normal"), (48, 48, "outliers"), (320, 640, "wide"),
                                            (128, 3072, "student_t"), (64, 256, "tiny"), (32, 512, "huge")])
def test_quantize_nvfp4_bitexact(block_rows, rows, cols, kind):
    bits = random_rows(kind, rows, cols, seed=rows * 3 + cols)
    q, s, st = _lib.ft_quantize_nvfp4(dev_bf16(bits), block_rows)
    torch.cuda.synchronize()
    rq, rs, rst = ref.quantize_nvfp4(bits, block_rows)
    assert np.float32(host(st)[0]) == np.float32(rst)
    assert np.array_equal(host(s), rs)
    assert np.array_equal(host(q), rq)


def test_quantize_nvfp4_ragged_rows():
    bits = random_rows("outliers", 33, 96, seed=1)
    q, s, st = _lib.ft_quantize_nvfp4(dev_bf16(bits), 1)
    torch.cuda.synchronize()
    rq, rs, rst = ref.quantize_nvfp4(bits, 1)
    assert np.float32(host(st)[0]) == np.float32(rst)
    assert np.array_equal(host(s), rs) and np.array_equal(host(q), rq)


@pytest.mark.parametrize("M,K,N", [(1, 16, 16), (130, 272, 208), (256, 1024, 384), (300, 1536, 640)])
def test_nvfp4_gemms_against_oracle(M, K, N):
    rng = np.random.default_rng(M + K + N)
    x = random_rows("outliers", M, K, seed=M)
    w = gen.f32_to_bf16_bits((0.02 * rng.standard_normal((N, K))).astype(np.float32))
    g = gen.f32_to_bf16_bits((1e-3 * rng.standard_t(3, (M, N))).astype(np.float32))
    xq, xs, xt = _lib.ft_quantize_nvfp4(dev_bf16(x), 1)
    wq, ws, wt = _lib.ft_quantize_nvfp4(dev_bf16(w), 16)
    gq, gs, gt = _lib.ft_quantize_nvfp4(dev_bf16(g), 1)
    y = _lib.ft_linear_fwd_nvfp4(xq, xs, xt, wq, ws, wt, K)
    dx = _lib.ft_linear_bwd_input_nvfp4(gq, gs, gt, wq, ws, wt, K)
    torch.cuda.synchronize()
    rq, rs, rt = ref.quantize_nvfp4(x, 1)
    mq, ms, mt = ref.quantize_nvfp4(w, 16)
    nq, ns, nt = ref.quantize_nvfp4(g, 1)
    assert np.array_equal(host(xq), rq) and np.array_equal(host(wq), mq) and np.array_equal(host(gq), nq)
    X, W, G = ref.dequantize_nvfp4(rq, rs, rt, K, 1), ref.dequantize_nvfp4(mq, ms, mt, K, 16), \
        ref.dequantize_nvfp4(nq, ns, nt, N, 1)
    yr, S = ref.gemm_f64(X, W, trans_b=True)
    assert np.all(np.abs(host(y) - yr) <= 1e-5 * S)
    dxr, Sdx = ref.gemm_f64(G, W, trans_b=False)
    assert np.all(np.abs(host(dx) - dxr) <= 1e-5 * Sdx)


def test_format_accuracy_cross_check_flux_qkv():
    """The QKV layer's forward product (4608 x 3072 -> 9216, activations with
    0.5 % outlier channels x30) in both formats against the exact fp64
    product of the bf16 operands, on sampled rows: NVFP4's finer blocks and
    scales are closer than MXFP4's; both GPU results match their oracles."""
    shape = gen.SHAPES["flux_qkv"]
    d = gen.layer_inputs(shape, 0)
    X, W = dev_bf16(d["X"]), dev_bf16(d["W"])
    xq, xs, xt = _lib.ft_quantize_nvfp4(X, 1)
    wq, ws, wt = _lib.ft_quantize_nvfp4(W, 16)
    y_nv = _lib.ft_linear_fwd_nvfp4(xq, xs, xt, wq, ws, wt, shape.K)
    mxq, mxs, _ = _lib.ft_quantize_blockwise(X)
    mwq, mws, _ = _lib.ft_quantize_blockwise(W, block_rows=32)
    y_mx = _lib.ft_linear_fwd(mxq, mxs, mwq, mws, shape.K, out_dtype=torch.float32)
    torch.cuda.synchronize()
    rows = np.array([0, 1000, 2047, 3333, 4607])
    exact = f64(d["X"][rows]) @ f64(d["W"]).T
    e_nv = np.linalg.norm(host(y_nv)[rows] - exact) / np.linalg.norm(exact)
    e_mx = np.linalg.norm(host(y_mx)[rows] - exact) / np.linalg.norm(exact)
    print("relative Frobenius error of the forward product: nvfp4 %.4f  mxfp4 %.4f" % (e_nv, e_mx), flush=True)
    assert e_nv < e_mx < 0.3
    rq, rs, rt = ref.quantize_nvfp4(d["X"][rows], 1, tensor_scale=float(host(xt)[0]))
    assert np.array_equal(host(xq)[rows], rq)
