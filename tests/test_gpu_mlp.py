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
Those checks follow the chain stage by stage.  The chain is also anchored on
oracle-only intermediates: z_or = RNE_bf16(y_oracle), taken wherever no bf16
rounding midpoint lies within the forward's tolerance 1e-5 * S of y_oracle (the
fused z must equal it there, and be one of the two neighbours elsewhere);
h_or = GELU(z_or) and dz_or = dH_oracle * GELU'(z) in fp64; the fused outputs
must lie within one bf16 unit of them, and the projections within the fp32
bound plus what the one-unit differences can move them.
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


def anchored_z(z, yr, S):
    """Check the fused z against the oracle's forward: z == RNE_bf16(yr) where
    the rounding is decided within the tolerance, else one of the two bf16
    values the tolerance interval rounds to.  Returns (z_or, sure)."""
    tol = 1e-5 * S
    lo, hi = rne_bf16_f64(yr - tol), rne_bf16_f64(yr + tol)
    sure = lo == hi
    z_or = rne_bf16_f64(yr)
    assert np.array_equal(z[sure], z_or[sure]), "z differs from RNE_bf16 of the oracle's forward"
    # RNE is monotone: z rounds a value inside the tolerance interval, so it lies
    # between the roundings of the interval's ends (which may be several units
    # apart near zero, where S >> |y|)
    assert np.all((f64(lo) <= f64(z)) & (f64(z) <= f64(hi))), "z outside the rounding interval of the oracle's forward"
    # 1e-5 * S spans a sizeable part of a bf16 unit where S >> |y|: most but
    # not all roundings are decided
    assert sure.mean() > 0.5, sure.mean()
    return z_or, sure


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

    # anchored on the oracle alone: z_or from the oracle's forward, h_or = GELU(z_or)
    z_or, sure = anchored_z(z, yr, S)
    h_or = ref.gelu(f64(z_or))
    ok = within_one_unit(h[sure], h_or[sure], 1e-6 * np.abs(f64(z_or[sure])))
    assert ok.all(), "h: %d of %d outside one bf16 unit of GELU(z_oracle)" % ((~ok).sum(), ok.size)

    # FC2's down-projection of h
    if R2:
        pr, pa = ref.proj(h, D2, 0)
        tiles = (N + 255) // 256
        P2h = host(P2).astype(np.float64)
        assert np.all(np.abs(P2h - pr) <= proj_bound(N, tiles, pa))
        # against h_or = bf16(GELU(z_or)) built by the oracle: the fp32 bound plus
        # what the elements where h and h_or differ (at most one unit) contribute
        h_or16 = rne_bf16_f64(h_or)
        pr_or, pa_or = ref.proj(h_or16, D2, 0)
        moved = np.abs(f64(h) - f64(h_or16)) @ np.abs(f64(D2))
        assert np.all(np.abs(P2h - pr_or) <= proj_bound(N, tiles, pa_or) + moved * (1 + 1e-6))


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

    # anchored on the oracle alone: dz_or = dH_oracle * GELU'(z) in fp64; the
    # GPU's dH carries at most 1e-5 * S, and its bf16 rounding one unit
    gp = ref.gelu(f64(Z), derivative=True)
    dz_or = dhr * gp
    lim = 2.0 ** -7 * np.abs(dz_or) + 1.01e-5 * S * np.abs(gp) + 1e-6 * np.abs(dhr) + 1e-30
    ok = np.abs(f64(dz) - dz_or) <= lim
    assert ok.all(), "dz: %d of %d outside one bf16 unit of dH_oracle GELU'(z)" % ((~ok).sum(), ok.size)

    if R1:
        pr, pa = ref.proj(dz, U1, 1)
        tiles = (K + 255) // 256
        assert np.all(np.abs(host(Qp1).astype(np.float64) - pr) <= proj_bound(K, tiles, pa))


def test_mlp_pair_flux_shape_sampled():
    """FLUX.1-dev MLP at 1024^2 (M = 4608, 3072 -> 12288 -> 3072, ranks 32 + 32)
    in the launch configuration the benchmark times: quantized outputs in full;
    FC1's output and FC2's input gradient against the oracle, and the
    elementwise outputs and projections anchored on the oracle, on the last
    256-row tile and scattered rows."""
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
    rows = np.unique(np.concatenate([[0, 1, 777, 2048, 4095], np.arange(4352, 4608)]))
    href = ref.gelu(f64(z[rows]))
    assert within_one_unit(h[rows], href, 1e-6 * np.abs(f64(z[rows]))).all()
    dh = host(dh32)[rows].astype(np.float64)
    dzref = dh * ref.gelu(f64(z[rows]), derivative=True)
    assert within_one_unit(dz[rows], dzref, 1e-6 * np.abs(dh)).all()
    pr, pa = ref.proj(h[rows], D2, 0)
    assert np.all(np.abs(host(P2)[rows] - pr) <= proj_bound(F, 48, pa))
    pr, pa = ref.proj(dz[rows], U1, 1)
    assert np.all(np.abs(host(Qp1)[rows] - pr) <= proj_bound(F, 48, pa))

    # anchored on the oracle: FC1's output from the oracle's quantization and
    # forward of these rows, then z_or, h_or = GELU(z_or); FC2's input gradient
    # from the oracle's backward, dz_or = dH_oracle GELU'(z_or)
    xq_o, xs_o = ref.quantize(X[rows], 1)
    w1q_o, w1s_o = ref.quantize(W1, 32)
    P1r, P1a = ref.proj(X[rows], D1, 0)
    yr, S = ref.linear_fwd(xq_o, xs_o, w1q_o, w1s_o, D_, P1r, U1, b1, Pabs=P1a)
    y32r = host(y32)[rows].astype(np.float64)
    assert np.all(np.abs(y32r - yr) <= 1e-5 * S), "FC1 output outside 1e-5 * S"
    z_or, sure = anchored_z(z[rows], yr, S)
    h_or = ref.gelu(f64(z_or))
    assert within_one_unit(h[rows][sure], h_or[sure], 1e-6 * np.abs(f64(z_or[sure]))).all()
    gq_o, gs_o = ref.quantize(dY[rows], 1)
    w2q_o, w2s_o = ref.quantize(W2, 32)
    Q2r, Q2a = ref.proj(dY[rows], U2, 1)
    dhr, Sdh = ref.linear_bwd_input(gq_o, gs_o, w2q_o, w2s_o, F, Q2r, D2, Qpabs=Q2a)
    assert np.all(np.abs(dh - dhr) <= 1e-5 * Sdh), "FC2 input gradient outside 1e-5 * S"
    gp = ref.gelu(f64(z_or), derivative=True)
    dz_or = dhr * gp
    lim = 2.0 ** -7 * np.abs(dz_or) + 1.01e-5 * Sdh * np.abs(gp) + 1e-6 * np.abs(dhr) + 1e-30
    assert np.all((np.abs(f64(dz[rows]) - dz_or) <= lim)[sure]), "dz outside one bf16 unit of the oracle's"
    h_or16 = rne_bf16_f64(h_or)
    pr_or, pa_or = ref.proj(h_or16, D2, 0)
    moved = np.abs(f64(h[rows]) - f64(h_or16)) @ np.abs(f64(D2))
    assert np.all(np.abs(host(P2)[rows] - pr_or) <= proj_bound(F, 48, pa_or) + moved * (1 + 1e-6))


@pytest.mark.parametrize("M", [200, 256])
def test_fused_epilogues_are_deterministic(M):
    """Repeated calls on the same inputs give the same bits: z, h, codes,
    scales and P2 of FC1; dz, codes, scales and Qp1 of FC2 (several column
    tiles, a partial row tile at M = 200)."""
    rng = np.random.default_rng(M)
    K, F, R = 256, 1024, 32
    X, W1, W2 = rand_bf16(rng, (M, K), 1.0), rand_bf16(rng, (F, K), 0.05), rand_bf16(rng, (K, F), 0.05)
    D1, U1 = rand_bf16(rng, (K, R), 0.05), rand_bf16(rng, (R, F), 0.05)
    D2, U2 = rand_bf16(rng, (F, R), 0.05), rand_bf16(rng, (R, K), 0.05)
    dY = rand_bf16(rng, (M, K), 0.01)
    w1q, w1s, _ = _lib.ft_quantize_blockwise(dev_bf16(W1), block_rows=32)
    w2q, w2s, _ = _lib.ft_quantize_blockwise(dev_bf16(W2), block_rows=32)
    xq, xs, P1 = _lib.ft_quantize_blockwise(dev_bf16(X), proj=dev_bf16(D1))
    gq, gs, Qp2 = _lib.ft_quantize_blockwise(dev_bf16(dY), proj=dev_bf16(U2), proj_layout=_lib.FT_PROJ_R_BY_COLS)
    runs = []
    for _ in range(4):
        fwd = _lib.ft_linear_fwd_gelu(xq, xs, w1q, w1s, K, P1, dev_bf16(U1), None, D2=dev_bf16(D2))
        bwd = _lib.ft_linear_bwd_input_dgelu(gq, gs, w2q, w2s, F, fwd[0], Qp2, dev_bf16(D2), U1=dev_bf16(U1))
        runs.append([t.clone() for t in list(fwd) + list(bwd)])
    torch.cuda.synchronize()
    names = ["z", "h", "hq", "hs", "P2", "dz", "dzq", "dzs", "Qp1"]
    for k, name in enumerate(names):
        for r in runs[1:]:
            assert torch.equal(runs[0][k], r[k]), name + " differs between identical calls"


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
