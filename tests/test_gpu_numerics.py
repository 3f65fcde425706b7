"""Parity of the quantizer's numerics variants (ft_quantize_blockwise_mode)
against the fp64 oracle, through the C ABI.

FourTune Sec. 3.1 leaves the quantizer's scale rule and rounding open; the
variants are the no-clip scale rule, stochastic rounding (Philox4x32-10 bits
keyed by seed and stream, per matrix element) and 2-D (32x32) blocks for
activations.  Bars: codes and scales bit-exact; fused projections within the
fp32 bound (unchanged by the mode); GEMMs fed with variant operands within
1e-5 * S of the oracle on the same operands.
"""
import numpy as np
import pytest
import torch

from oracle import ref
from paper_2607_05711_amd import _lib, gen
from tests._helpers import adversarial_rows, f64, random_rows

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
QR_CW = 384


def dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(DEV)


def host(t):
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


MODES = [(1, 0), (0, 1), (1, 1)]    # (scale_rule, rounding): no-clip, stochastic, both
SEED, STREAM = 0x0123_4567_89AB_CDEF, 42


@pytest.mark.parametrize("rule,rnd", MODES)
@pytest.mark.parametrize("rows,cols,kind", [(1, 32, "normal"), (129, 416, "outliers"), (300, 640, "wide"),
                                            (513, 1184, "student_t"), (64, 4096, "huge"), (33, 96, "tiny")])
def test_quantize_variants_bitexact(rule, rnd, rows, cols, kind):
    bits = random_rows(kind, rows, cols, seed=rows + cols)
    codes, scales, _ = _lib.ft_quantize_blockwise_mode(dev_bf16(bits), scale_rule=rule, rounding=rnd, seed=SEED,
                                                       stream=STREAM)
    torch.cuda.synchronize()
    q, s = ref.quantize_ex(bits, 1, scale_rule=rule, rounding=rnd, seed=SEED, stream=STREAM)
    assert np.array_equal(host(scales), s)
    assert np.array_equal(host(codes), q)


@pytest.mark.parametrize("rule,rnd", MODES)
def test_quantize_variants_adversarial(rule, rnd):
    bits = adversarial_rows(1024, seed=3)
    codes, scales, _ = _lib.ft_quantize_blockwise_mode(dev_bf16(bits), scale_rule=rule, rounding=rnd, seed=7,
                                                       stream=1 << 40)
    torch.cuda.synchronize()
    q, s = ref.quantize_ex(bits, 1, scale_rule=rule, rounding=rnd, seed=7, stream=1 << 40)
    assert np.array_equal(host(scales), s)
    assert np.array_equal(host(codes), q)


@pytest.mark.parametrize("rule,rnd", MODES)
@pytest.mark.parametrize("rows,cols,R,layout", [(300, 640, 48, 0), (2304, 4064, 64, 0), (2200, 1056, 16, 0),
                                                (7001, 288, 64, 0), (8224, 3072, 64, 0), (300, 800, 96, 1),
                                                (2065, 4160, 64, 1), (16640, 12288, 64, 1)])
def test_quantize_variants_with_projection(rule, rnd, rows, cols, R, layout):
    """Every kernel path (column chunks for either projection layout, whole
    rows per workgroup in 24- and 32-row workgroups, workgroups looping over
    two chunks): codes and scales as the oracle's variant, projection as
    without the mode."""
    rng = np.random.default_rng(rows + R)
    bits = random_rows("outliers", rows, cols, seed=rows)
    pshape = (cols, R) if layout == 0 else (R, cols)
    proj = gen.f32_to_bf16_bits((0.02 * rng.standard_normal(pshape)).astype(np.float32))
    codes, scales, P = _lib.ft_quantize_blockwise_mode(dev_bf16(bits), proj=dev_bf16(proj), proj_layout=layout,
                                                       scale_rule=rule, rounding=rnd, seed=SEED, stream=STREAM)
    torch.cuda.synchronize()
    q, s = ref.quantize_ex(bits, 1, scale_rule=rule, rounding=rnd, seed=SEED, stream=STREAM)
    assert np.array_equal(host(scales), s) and np.array_equal(host(codes), q)
    p_ref, p_abs = ref.proj(bits, proj, layout)
    chunks = (cols + QR_CW - 1) // QR_CW
    assert np.all(np.abs(host(P).astype(np.float64) - p_ref) <= (cols + chunks) * 2.0 ** -24 * p_abs)


def test_stochastic_rounding_flux_gradient_shape():
    """dY of the QKV projection (4608 x 9216) with its [R, cols] projection,
    the launch the layer's backward uses: bit-exact against the oracle; a
    different stream changes codes and keeps scales."""
    shape = gen.SHAPES["flux_qkv"]
    d = gen.layer_inputs(shape, 0)
    dY, U = dev_bf16(d["dY"]), dev_bf16(d["U"])
    gq, gs, Qp = _lib.ft_quantize_blockwise_mode(dY, proj=U, proj_layout=_lib.FT_PROJ_R_BY_COLS,
                                                 rounding=_lib.FT_ROUND_STOCHASTIC, seed=5, stream=9)
    gq2, gs2, _ = _lib.ft_quantize_blockwise_mode(dY, proj=U, proj_layout=_lib.FT_PROJ_R_BY_COLS,
                                                  rounding=_lib.FT_ROUND_STOCHASTIC, seed=5, stream=10)
    torch.cuda.synchronize()
    q, s = ref.quantize_ex(d["dY"], 1, rounding=1, seed=5, stream=9)
    assert np.array_equal(host(gs), s) and np.array_equal(host(gq), q)
    assert np.array_equal(host(gs2), s) and not np.array_equal(host(gq2), q)


def test_stochastic_gradient_through_backward_gemm():
    """Stochastically rounded G feeds Eq. (3) unchanged: the input gradient on
    those codes matches the oracle's on the oracle's (identical) codes."""
    shape = gen.custom_shape(520, 1024, 1536, r=32, r_s=32, n_outliers=3, outlier_scale=30.0, dy_kind="student_t3")
    d = gen.layer_inputs(shape, 3)
    W, D, U, dY = (dev_bf16(d[k]) for k in ("W", "D", "U", "dY"))
    wq, ws, _ = _lib.ft_quantize_blockwise(W, block_rows=32)
    gq, gs, Qp = _lib.ft_quantize_blockwise_mode(dY, proj=U, proj_layout=_lib.FT_PROJ_R_BY_COLS,
                                                 scale_rule=_lib.FT_SCALE_NO_CLIP, rounding=_lib.FT_ROUND_STOCHASTIC,
                                                 seed=11, stream=2)
    dx = _lib.ft_linear_bwd_input(gq, gs, wq, ws, shape.K, Qp, D, out_dtype=torch.float32)
    torch.cuda.synchronize()
    q, s = ref.quantize_ex(d["dY"], 1, scale_rule=1, rounding=1, seed=11, stream=2)
    assert np.array_equal(host(gq), q) and np.array_equal(host(gs), s)
    wq_r, ws_r = ref.quantize(d["W"], 32)
    Qr, Qa = ref.proj(d["dY"], d["U"], 1)
    dxr, S = ref.linear_bwd_input(q, s, wq_r, ws_r, shape.K, Qr, d["D"], Qpabs=Qa)
    assert np.all(np.abs(host(dx) - dxr) <= 1e-5 * S)


@pytest.mark.parametrize("rule", [0, 1])
@pytest.mark.parametrize("M,K,N", [(64, 256, 256), (320, 1024, 544)])
def test_two_dimensional_activation_blocks_through_gemm(rule, M, K, N):
    """X quantized in 32x32 tiles with scales written per row (each row its
    tile's): codes and scales as the oracle's tile quantizer, and the forward
    GEMM on them within 1e-5 * S of the oracle."""
    rng = np.random.default_rng(M + K + rule)
    X = random_rows("outliers", M, K, seed=M)
    W = gen.f32_to_bf16_bits((0.02 * rng.standard_normal((N, K))).astype(np.float32))
    bias = gen.f32_to_bf16_bits((0.02 * rng.standard_normal(N)).astype(np.float32))
    xq, xs, _ = _lib.ft_quantize_blockwise_mode(dev_bf16(X), block_rows=32, scale_rule=rule, scales_per_row=True)
    tq, ts, _ = _lib.ft_quantize_blockwise_mode(dev_bf16(X), block_rows=32, scale_rule=rule)
    wq, ws, _ = _lib.ft_quantize_blockwise(dev_bf16(W), block_rows=32)
    y = _lib.ft_linear_fwd(xq, xs, wq, ws, K, None, None, dev_bf16(bias), out_dtype=torch.float32)
    torch.cuda.synchronize()
    q, s = ref.quantize_ex(X, 32, scale_rule=rule)
    assert np.array_equal(host(xq), q) and np.array_equal(host(tq), q)
    assert np.array_equal(host(ts), s)
    assert np.array_equal(host(xs), np.repeat(s, 32, axis=0))
    wq_r, ws_r = ref.quantize(W, 32)
    yr, S = ref.linear_fwd(q, np.repeat(s, 32, axis=0), wq_r, ws_r, K, None, None, bias)
    assert np.all(np.abs(host(y) - yr) <= 1e-5 * S)
