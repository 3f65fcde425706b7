"""Parity of the fused MLP epilogues (FourTune Sec. 3.3, MLP fusion) against
the fp64 oracle, through the C ABI.

FC1 forward (ft_linear_fwd_gelu) and FC2 backward-input
(ft_linear_bwd_input_dgelu) run the same GEMM schedule as ft_linear_fwd /
ft_linear_bwd_input, so:
  * z is exactly bf16 (round to nearest even) of the fp32 forward output, and
    that output is within 1e-5 * S of the oracle;
  * h = bf16(GELU(z)) and dz = bf16(dH * GELU'(z)) are within one bf16 unit of
    the same expressions evaluated in fp64 from the GPU's z and fp32 dH (the
    GPU evaluates GELU in fp32; the two roundings can differ by one unit), plus
    an absolute term for the fp32 evaluation near zeros of GELU';
  * codes and scales are bit-exact against the oracle quantizer applied to the
    GPU's h / dz;
  * P2 / Qp1 are within the fp32 accumulation bound of the oracle projection of
    the GPU's h / dz (partial sums per 256-column tile).
"""
import numpy as np
import pytest
import torch

from oracle import ref
from paper_2607_05711_amd import _lib
from paper_2607_05711_amd import gen
from tests._helpers import f64

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(DEV)


def host(t):
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def bf16(a):
    return gen.f32_to_bf16_bits(np.asarray(a, dtype=np.float32))


def rne_bf16_f64(a):
    """Round fp64 values to bf16 (nearest even), via the exact fp32 step when
    the fp64 value is not a tie at the fp32 level (true for these values)."""
    return bf16(np.asarray(a, dtype=np.float64).astype(np.float32))


def within_one_unit(gpu_bits, ref_f64, abs_slack):
    g, r = f64(gpu_bits), np.asarray(ref_f64, dtype=np.float64)
    return np.abs(g - r) <= 2.0 ** -7 * np.abs(r) + abs_slack


def rand_bf16(rng, shape, scale):
    return bf16(scale * rng.standard_normal(shape).astype(np.float32))


def proj_bound(cols, tiles, pabs):
    return (cols + tiles) * 2.0 ** -24 * pabs


FWD_CASES = [  # M, K, N, R, R2
    (300, 256, 512, 32, 32),     # two column tiles: partials reduced
    (520, 384, 1280, 64, 64),    # five tiles, ragged rows
    (64, 128, 256, 16, 0),       # no projection, one tile
    (130, 512, 288, 0, 16),      # ragged last column tile, no low-rank input
]


@pytest.mark.parametrize("M,K,N,R,R2", FWD_CASES)
def test_fc1_forward_gelu_quantize_project(M, K, N, R, R2):
    rng = np.random.default_rng(M + N + R2)
    X = rand_bf16(rng, (M, K), 1.0)
    W = rand_bf16(rng, (N, K), 0.05)
    bias = rand_bf16(rng, (N,), 0.1)
    Xd, Wd, bd = dev_bf16(X), dev_bf16(W), dev_bf16(bias)
    wq, ws, _ = _lib.ft_quantize_blockwise(Wd, block_rows=32)
    if R:
        D, U = rand_bf16(rng, (K, R), 0.05), rand_bf16(rng, (R, N), 0.05)
        xq, xs, P = _lib.ft_quantize_blockwise(Xd, proj=dev_bf16(D))
        Ud = dev_bf16(U)
    else:
        xq, xs, _ = _lib.ft_quantize_blockwise(Xd)
        P = Ud = None
    D2 = rand_bf16(rng, (N, R2), 0.05) if R2 else None
    y32 = _lib.ft_linear_fwd(xq, xs, wq, ws, K, P, Ud, bd, out_dtype=torch.float32)
    z, h, hq, hs, P2 = _lib.ft_linear_fwd_gelu(xq, xs, wq, ws, K, P, Ud, bd, D2=dev_bf16(D2) if R2 else None)
    torch.cuda.synchronize()
    y32, z, h, hq, hs = host(y32), host(z), host(h), host(hq), host(hs)

    # z: the forward's fp32 result rounded once; that result matches the oracle
    assert np.array_equal(z, bf16(y32))
    xq_h, xs_h = ref.quantize(X, 1)
    wq_h, ws_h = ref.quantize(W, 32)
    if R:
        Pr, Pa = ref.proj(X, D, 0)
        yr, S = ref.linear_fwd(xq_h, xs_h, wq_h, ws_h, K, Pr, U, bias, Pabs=Pa)
    else:
        yr, S = ref.linear_fwd(xq_h, xs_h, wq_h, ws_h, K, None, None, bias)
    assert np.all(np.abs(y32.astype(np.float64) - yr) <= 1e-5 * S)

    # h = bf16(GELU(z))
    href = ref.gelu(f64(z))
    ok = within_one_unit(h, href, 1e-6 * np.abs(f64(z)))
    assert ok.all(), "h: %d of %d outside one bf16 unit" % ((~ok).sum(), ok.size)
    assert np.mean(h == rne_bf16_f64(href)) > 0.99

    # codes and scales of h
    q, s = ref.quantize(h, 1)
    assert np.array_equal(hq, q) and np.array_equal(hs, s)

    # FC2's down-projection of h
    if R2:
        pr, pa = ref.proj(h, D2, 0)
        tiles = (N + 255) // 256
        assert np.all(np.abs(host(P2).astype(np.float64) - pr) <= proj_bound(N, tiles, pa))


BWD_CASES = [  # M, N (FC2 output width), K (MLP width), R, R1
    (300, 256, 512, 32, 32),
    (520, 384, 1280, 64, 64),
    (64, 128, 256, 16, 0),
    (130, 512, 384, 0, 16),
]


@pytest.mark.parametrize("M,N,K,R,R1", BWD_CASES)
def test_fc2_backward_dgelu_quantize_project(M, N, K, R, R1):
    rng = np.random.default_rng(7 * M + K + R1)
    dY = gen.f32_to_bf16_bits((1e-3 * rng.standard_t(3, (M, N))).astype(np.float32))
    W = rand_bf16(rng, (N, K), 0.05)
    Z = rand_bf16(rng, (M, K), 1.5)           # FC1 pre-activation saved by the forward
    dYd, Wd, Zd = dev_bf16(dY), dev_bf16(W), dev_bf16(Z)
    wq, ws, _ = _lib.ft_quantize_blockwise(Wd, block_rows=32)
    if R:
        U, D = rand_bf16(rng, (R, N), 0.05), rand_bf16(rng, (K, R), 0.05)
        gq, gs, Qp = _lib.ft_quantize_blockwise(dYd, proj=dev_bf16(U), proj_layout=_lib.FT_PROJ_R_BY_COLS)
        Dd = dev_bf16(D)
    else:
        gq, gs, _ = _lib.ft_quantize_blockwise(dYd)
        Qp = Dd = None
    U1 = rand_bf16(rng, (R1, K), 0.05) if R1 else None
    dh32 = _lib.ft_linear_bwd_input(gq, gs, wq, ws, K, Qp, Dd, out_dtype=torch.float32)
    dz, dzq, dzs, Qp1 = _lib.ft_linear_bwd_input_dgelu(gq, gs, wq, ws, K, Zd, Qp, Dd,
                                                       U1=dev_bf16(U1) if R1 else None)
    torch.cuda.synchronize()
    dh32, dz, dzq, dzs = host(dh32), host(dz), host(dzq), host(dzs)

    gq_h, gs_h = ref.quantize(dY, 1)
    wq_h, ws_h = ref.quantize(W, 32)
    if R:
        Qr, Qa = ref.proj(dY, U, 1)
        dhr, S = ref.linear_bwd_input(gq_h, gs_h, wq_h, ws_h, K, Qr, D, Qpabs=Qa)
    else:
        dhr, S = ref.linear_bwd_input(gq_h, gs_h, wq_h, ws_h, K, None, None)
    assert np.all(np.abs(dh32.astype(np.float64) - dhr) <= 1e-5 * S)

    # dz = bf16(dH * GELU'(z)), dH unrounded
    dzref = dh32.astype(np.float64) * ref.gelu(f64(Z), derivative=True)
    ok = within_one_unit(dz, dzref, 1e-6 * np.abs(dh32.astype(np.float64)))
    assert ok.all(), "dz: %d of %d outside one bf16 unit" % ((~ok).sum(), ok.size)
    assert np.mean(dz == rne_bf16_f64(dzref)) > 0.99

    q, s = ref.quantize(dz, 1)
    assert np.array_equal(dzq, q) and np.array_equal(dzs, s)

    if R1:
        pr, pa = ref.proj(dz, U1, 1)
        tiles = (K + 255) // 256
        assert np.all(np.abs(host(Qp1).astype(np.float64) - pr) <= proj_bound(K, tiles, pa))


def test_mlp_pair_flux_shape_sampled():
    """FLUX.1-dev MLP at 1024^2 (M = 4608, 3072 -> 12288 -> 3072, ranks 32 + 32)
    in the launch configuration the benchmark times: quantized outputs and
    projections in full, elementwise outputs on sampled rows."""
    M, D_, F = 4608, 3072, 12288
    rng = np.random.default_rng(11)
    X = rand_bf16(rng, (M, D_), 1.0)
    W1 = rand_bf16(rng, (F, D_), 0.02)
    W2 = rand_bf16(rng, (D_, F), 0.02)
    D1, U1 = rand_bf16(rng, (D_, 64), 0.01), rand_bf16(rng, (64, F), 0.01)
    D2, U2 = rand_bf16(rng, (F, 64), 0.01), rand_bf16(rng, (64, D_), 0.01)
    dY = gen.f32_to_bf16_bits((1e-3 * rng.standard_t(3, (M, D_))).astype(np.float32))
    b1 = rand_bf16(rng, (F,), 0.02)
    w1q, w1s, _ = _lib.ft_quantize_blockwise(dev_bf16(W1), block_rows=32)
    w2q, w2s, _ = _lib.ft_quantize_blockwise(dev_bf16(W2), block_rows=32)
    xq, xs, P1 = _lib.ft_quantize_blockwise(dev_bf16(X), proj=dev_bf16(D1))
    z, h, hq, hs, P2 = _lib.ft_linear_fwd_gelu(xq, xs, w1q, w1s, D_, P1, dev_bf16(U1), dev_bf16(b1), D2=dev_bf16(D2))
    gq, gs, Qp2 = _lib.ft_quantize_blockwise(dev_bf16(dY), proj=dev_bf16(U2), proj_layout=_lib.FT_PROJ_R_BY_COLS)
    dz, dzq, dzs, Qp1 = _lib.ft_linear_bwd_input_dgelu(gq, gs, w2q, w2s, F, z, Qp2, dev_bf16(D2), U1=dev_bf16(U1))
    y32 = _lib.ft_linear_fwd(xq, xs, w1q, w1s, D_, P1, dev_bf16(U1), dev_bf16(b1), out_dtype=torch.float32)
    dh32 = _lib.ft_linear_bwd_input(gq, gs, w2q, w2s, F, Qp2, dev_bf16(D2), out_dtype=torch.float32)
    torch.cuda.synchronize()
    z, h, hq, hs, dz, dzq, dzs = (host(t) for t in (z, h, hq, hs, dz, dzq, dzs))
    assert np.array_equal(z, bf16(host(y32)))
    q, s = ref.quantize(h, 1)
    assert np.array_equal(hq, q) and np.array_equal(hs, s)
    q, s = ref.quantize(dz, 1)
    assert np.array_equal(dzq, q) and np.array_equal(dzs, s)
    rows = np.array([0, 1, 777, 2048, 4095, 4607])
    href = ref.gelu(f64(z[rows]))
    assert within_one_unit(h[rows], href, 1e-6 * np.abs(f64(z[rows]))).all()
    dh = host(dh32)[rows].astype(np.float64)
    dzref = dh * ref.gelu(f64(z[rows]), derivative=True)
    assert within_one_unit(dz[rows], dzref, 1e-6 * np.abs(dh)).all()
    pr, pa = ref.proj(h[rows], D2, 0)
    assert np.all(np.abs(host(P2)[rows] - pr) <= proj_bound(F, 48, pa))
    pr, pa = ref.proj(dz[rows], U1, 1)
    assert np.all(np.abs(host(Qp1)[rows] - pr) <= proj_bound(F, 48, pa))


def test_mlp_empty_token_axis():
    """M = 0 through both fused epilogues: the calls succeed and every output
    with a token axis is empty."""
    rng = np.random.default_rng(11)
    K, F, R = 256, 512, 32
    W1 = dev_bf16(rand_bf16(rng, (F, K), 0.05))
    W2 = dev_bf16(rand_bf16(rng, (K, F), 0.05))
    w1q, w1s, _ = _lib.ft_quantize_blockwise(W1, block_rows=32)
    w2q, w2s, _ = _lib.ft_quantize_blockwise(W2, block_rows=32)
    xq, xs, _ = _lib.ft_quantize_blockwise(torch.empty((0, K), dtype=torch.bfloat16, device=DEV))
    D2 = dev_bf16(rand_bf16(rng, (F, R), 0.05))
    z, h, hq, hs, P2 = _lib.ft_linear_fwd_gelu(xq, xs, w1q, w1s, K, D2=D2)
    assert z.shape == (0, F) and h.shape == (0, F) and hq.shape == (0, F // 2) and P2.shape == (0, R)
    gq, gs, _ = _lib.ft_quantize_blockwise(torch.empty((0, K), dtype=torch.bfloat16, device=DEV))
    U1 = dev_bf16(rand_bf16(rng, (R, F), 0.05))
    dz, dzq, dzs, Qp1 = _lib.ft_linear_bwd_input_dgelu(gq, gs, w2q, w2s, F, z, U1=U1)
    torch.cuda.synchronize()
    assert dz.shape == (0, F) and dzq.shape == (0, F // 2) and Qp1.shape == (0, R)
