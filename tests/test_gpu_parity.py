"""Parity of the gfx950 library against the fp64 CPU oracle, through the C ABI.

Bars (from the layer's contract):
  * E2M1 codes and E8M0 scales: bit-exact;
  * GEMM outputs in fp32 mode: |err| <= 1e-5 * S per element, S = sum of |terms|
    computed in fp64 on the dequantized operands (oracle);
  * bf16 outputs: exactly the round-to-nearest-even of the fp32-mode result, and
    |err| <= 1e-5 * S + 2^-8 |ref|;
  * fused down-projections (fp32): |err| <= (cols + chunks) * 2^-24 * sum|x||d|,
    the worst-case bound of fp32 accumulation of exact bf16 products;
  * adapter gradients: ||g - ref||_F <= 1e-3 ||ref||_F.
Inputs are seeded and synthetic (paper_2607_05711_amd.gen); both sides receive
the same host arrays.
"""
import numpy as np
import pytest
import torch

from oracle import ref
from paper_2607_05711_amd import _lib
from paper_2607_05711_amd import gen
from tests._helpers import adversarial_rows, f64, random_rows

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
QR_CW = 384  # narrowest column chunk of the fused quantize kernel (fp32 partial sums combine per chunk)


def dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(DEV)


def dev_u8(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host(t):
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def bf16_rne_of_f32(a):
    return gen.f32_to_bf16_bits(a.astype(np.float32))


def proj_bound(cols, pabs):
    chunks = (cols + QR_CW - 1) // QR_CW
    return (cols + chunks) * 2.0 ** -24 * pabs


def check_gemm(out32, out16, refv, S, what):
    err = np.abs(out32.astype(np.float64) - refv)
    worst = (err / np.maximum(S, 1e-300)).max()
    print("%s: max err/S = %.3g" % (what, worst), flush=True)
    assert np.all(err <= 1e-5 * S), "%s: max err/S = %.3g" % (what, worst)
    assert np.array_equal(out16, bf16_rne_of_f32(out32)), "%s: bf16 output is not RNE of the fp32 result" % what
    err16 = np.abs(f64(out16) - refv)
    assert np.all(err16 <= 1e-5 * S + 2.0 ** -8 * np.abs(refv)), what


# ------------------------------------------------------------------ quantize
QUANT_SHAPES = [(1, 32), (128, 256), (129, 416), (300, 640), (513, 1184), (64, 4096)]


@pytest.mark.parametrize("rows,cols", QUANT_SHAPES)
@pytest.mark.parametrize("kind", ["normal", "outliers", "student_t", "wide"])
def test_quantize_rows_bitexact(rows, cols, kind):
    bits = random_rows(kind, rows, cols, seed=rows * 7 + cols)
    codes, scales, _ = _lib.ft_quantize_blockwise(dev_bf16(bits))
    torch.cuda.synchronize()
    q, s = ref.quantize(bits, 1)
    assert np.array_equal(host(codes), q)
    assert np.array_equal(host(scales), s)


def test_quantize_rows_adversarial_bitexact():
    bits = adversarial_rows(1024, seed=1)
    codes, scales, _ = _lib.ft_quantize_blockwise(dev_bf16(bits))
    torch.cuda.synchronize()
    q, s = ref.quantize(bits, 1)
    assert np.array_equal(host(scales), s)
    assert np.array_equal(host(codes), q)


@pytest.mark.parametrize("rows,cols", [(32, 32), (96, 160), (256, 256), (320, 3072)])
def test_quantize_tiles_bitexact(rows, cols):
    bits = random_rows("outliers", rows, cols, seed=rows + cols)
    bits[:32, :32] = adversarial_rows(32, seed=2)[:, :32].repeat(3, axis=0)[:32]
    codes, scales, _ = _lib.ft_quantize_blockwise(dev_bf16(bits), block_rows=32)
    torch.cuda.synchronize()
    q, s = ref.quantize(bits, 32)
    assert np.array_equal(host(scales), s)
    assert np.array_equal(host(codes), q)


@pytest.mark.parametrize("rows,cols,R,layout", [(128, 256, 32, 0), (300, 640, 48, 0), (129, 1184, 64, 0),
                                                (200, 416, 128, 0), (128, 256, 32, 1), (300, 800, 96, 1),
                                                (77, 4096, 16, 1), (513, 384, 112, 0),
                                                # enough workgroups for 384-column chunks
                                                (8224, 3072, 64, 0),
                                                # rows longer than 4096: column chunks, ragged last chunk
                                                (2304, 10976, 64, 0),
                                                # ... in 640-column chunks (R <= 64) or 512 (R = 96) when
                                                # those still make 256 workgroups; ragged rows, last chunks
                                                # of one step, a step and a half, half a step
                                                (8200, 6464, 64, 0), (8200, 5216, 32, 0), (8200, 5152, 96, 0),
                                                # ... and for rows of at most 4096 when those fill a round
                                                (13200, 3136, 64, 0), (11000, 3104, 96, 0),
                                                # [cols, R] with whole rows per workgroup (64..256 workgroups
                                                # of 24 rows, or of 32 when 24 would need more than 256; rows
                                                # up to 4096): ragged rows, a last half step, fewer steps than
                                                # waves, projections narrower than their 32-column tiles
                                                (2304, 4064, 64, 0), (2200, 1056, 16, 0), (2100, 160, 64, 0),
                                                (8192, 800, 48, 0), (2080, 96, 32, 0), (1601, 512, 64, 0),
                                                (7001, 288, 64, 0),
                                                # [R, cols] at the same row counts (column chunks: 256 columns
                                                # where 768 would make fewer than 128 workgroups, 512 for
                                                # R = 96) and with 768-column chunks and a ragged last one
                                                (2065, 4160, 64, 1), (3000, 2080, 32, 1), (2080, 640, 48, 1),
                                                (1000, 5152, 96, 1), (4352, 6400, 64, 1),
                                                # workgroups looping over several chunks: ragged rows, a
                                                # last group of one ragged chunk ([R, cols]: 22 chunks of
                                                # 768, 3 per group; [cols, R]: 26 of 640, 5 per group)
                                                (16640, 16384, 64, 1), (16640, 16384, 64, 0)])
def test_quantize_fused_projection(rows, cols, R, layout):
    rng = np.random.default_rng(rows + cols + R)
    bits = random_rows("outliers", rows, cols, seed=rows)
    pshape = (cols, R) if layout == 0 else (R, cols)
    proj = gen.f32_to_bf16_bits((0.02 * rng.standard_normal(pshape)).astype(np.float32))
    codes, scales, P = _lib.ft_quantize_blockwise(dev_bf16(bits), proj=dev_bf16(proj), proj_layout=layout)
    torch.cuda.synchronize()
    q, s = ref.quantize(bits, 1)
    assert np.array_equal(host(codes), q) and np.array_equal(host(scales), s)
    p_ref, p_abs = ref.proj(bits, proj, layout)
    err = np.abs(host(P).astype(np.float64) - p_ref)
    assert np.all(err <= proj_bound(cols, p_abs)), (err / np.maximum(p_abs, 1e-300)).max()


# ------------------------------------------------------------- linear layer
def make_case(shape, seed, stab="random"):
    if stab == "svd":
        def residual(w):
            wq, ws = ref.quantize(w, 32)
            return f64(w) - ref.dequantize(wq, ws, shape.K, 32)
        return gen.layer_inputs(shape, seed, residual_fn=residual)
    return gen.layer_inputs(shape, seed)


def run_gpu_layer(d, shape, with_bias=True):
    X, W, D, U, dY = (dev_bf16(d[k]) for k in ("X", "W", "D", "U", "dY"))
    bias = dev_bf16(d["bias"]) if with_bias else None
    wq, ws, _ = _lib.ft_quantize_blockwise(W, block_rows=32)
    R = shape.R
    xq, xs, P = _lib.ft_quantize_blockwise(X, proj=D if R else None, proj_layout=_lib.FT_PROJ_COLS_BY_R)
    y32 = _lib.ft_linear_fwd(xq, xs, wq, ws, shape.K, P, U if R else None, bias, out_dtype=torch.float32)
    y16 = _lib.ft_linear_fwd(xq, xs, wq, ws, shape.K, P, U if R else None, bias, out_dtype=torch.bfloat16)
    gq, gs, Qp = _lib.ft_quantize_blockwise(dY, proj=U if R else None, proj_layout=_lib.FT_PROJ_R_BY_COLS)
    dx32 = _lib.ft_linear_bwd_input(gq, gs, wq, ws, shape.K, Qp, D if R else None, out_dtype=torch.float32)
    dx16 = _lib.ft_linear_bwd_input(gq, gs, wq, ws, shape.K, Qp, D if R else None, out_dtype=torch.bfloat16)
    out = dict(wq=wq, ws=ws, xq=xq, xs=xs, P=P, y32=y32, y16=y16, gq=gq, gs=gs, Qp=Qp, dx32=dx32, dx16=dx16)
    if shape.r and R:
        dA, dB = _lib.ft_lora_grads(X, dY, P, Qp, shape.r, col0=shape.r_s)
        out.update(dA=dA, dB=dB)
    torch.cuda.synchronize()
    return {k: host(v) for k, v in out.items() if v is not None}


def check_layer(d, shape, g, rows=None, with_bias=True):
    """Compare GPU results g with the oracle on all rows or on sampled rows."""
    K, N, R = shape.K, shape.N, shape.R
    wq, ws = ref.quantize(d["W"], 32)
    assert np.array_equal(g["wq"], wq) and np.array_equal(g["ws"], ws)
    X, dY = d["X"], d["dY"]
    sel = slice(None) if rows is None else rows
    Xs, dYs = X[sel], dY[sel]
    xq, xs = ref.quantize(Xs, 1)
    assert np.array_equal(g["xq"][sel], xq) and np.array_equal(g["xs"][sel], xs)
    gq, gs = ref.quantize(dYs, 1)
    assert np.array_equal(g["gq"][sel], gq) and np.array_equal(g["gs"][sel], gs)
    bias = d["bias"] if with_bias else None
    if R:
        P, Pabs = ref.proj(Xs, d["D"], 0)
        Qp, Qpabs = ref.proj(dYs, d["U"], 1)
        assert np.all(np.abs(g["P"][sel] - P) <= proj_bound(K, Pabs))
        assert np.all(np.abs(g["Qp"][sel] - Qp) <= proj_bound(N, Qpabs))
        y, S = ref.linear_fwd(xq, xs, wq, ws, K, P, d["U"], bias, Pabs=Pabs)
        dx, Sdx = ref.linear_bwd_input(gq, gs, wq, ws, K, Qp, d["D"], Qpabs=Qpabs)
    else:
        y, S = ref.linear_fwd(xq, xs, wq, ws, K, None, None, bias)
        dx, Sdx = ref.linear_bwd_input(gq, gs, wq, ws, K, None, None)
    check_gemm(g["y32"][sel], g["y16"][sel], y, S, "forward")
    check_gemm(g["dx32"][sel], g["dx16"][sel], dx, Sdx, "backward-input")
    if "dA" in g and rows is None:
        rs = shape.r_s
        Pf, _ = ref.proj(X, d["D"], 0)
        Qf, _ = ref.proj(dY, d["U"], 1)
        dA, dB, _, _ = ref.lora_grads(X, dY, Pf[:, rs:], Qf[:, rs:], want_s=False)
        assert np.linalg.norm(g["dA"] - dA) <= 1e-3 * np.linalg.norm(dA)
        assert np.linalg.norm(g["dB"] - dB) <= 1e-3 * np.linalg.norm(dB)


def test_layer_tiny_svd_stabilizer():
    """128x256 -> 256, LoRA rank 16, stabilizer rank 16 from the SVD of the
    weight's quantization residual; every output compared."""
    shape = gen.SHAPES["tiny"]
    d = make_case(shape, 0, stab="svd")
    check_layer(d, shape, run_gpu_layer(d, shape))


@pytest.mark.parametrize("M,K,N,r,rs", [(300, 640, 608, 16, 32), (1, 32, 32, 16, 16), (257, 288, 544, 32, 0),
                                        (64, 512, 256, 0, 0), (520, 1056, 800, 64, 32), (33, 96, 1312, 8, 8),
                                        # both reductions multiples of 512 (the A scales of two stages load
                                        # together, the kernels the benchmark times), 3x6 forward and 3x4
                                        # backward tiles with a ragged last row tile, R = 64 and a bias
                                        (520, 1024, 1536, 32, 32)])
def test_layer_ragged(M, K, N, r, rs):
    shape = gen.custom_shape(M, K, N, r=r, r_s=rs, n_outliers=3, outlier_scale=30.0, dy_kind="student_t3")
    d = make_case(shape, 1)
    check_layer(d, shape, run_gpu_layer(d, shape, with_bias=(M % 2 == 0)), with_bias=(M % 2 == 0))


def test_lora_grads_accumulate():
    shape = gen.custom_shape(200, 320, 416, r=32, r_s=16)
    d = make_case(shape, 2)
    X, dY, D, U = (dev_bf16(d[k]) for k in ("X", "dY", "D", "U"))
    _, _, P = _lib.ft_quantize_blockwise(X, proj=D)
    _, _, Qp = _lib.ft_quantize_blockwise(dY, proj=U, proj_layout=_lib.FT_PROJ_R_BY_COLS)
    dA, dB = _lib.ft_lora_grads(X, dY, P, Qp, 32, col0=16)
    dA2, dB2 = dA.clone(), dB.clone()
    _lib.ft_lora_grads(X, dY, P, Qp, 32, col0=16, dA=dA2, dB=dB2, accumulate=True)
    torch.cuda.synchronize()
    # partial sums are added in a fixed order, so the second pass adds exactly dA
    assert torch.equal(dA2, 2 * dA) and torch.equal(dB2, 2 * dB)


def test_empty_token_axis():
    """M = 0: every output with a token axis is empty and the calls succeed; the
    adapter gradients are sums over no tokens, so they come out as exact zeros,
    or unchanged when accumulating."""
    K, N, r = 256, 320, 16
    rng = np.random.default_rng(5)
    W = dev_bf16(gen.f32_to_bf16_bits(rng.standard_normal((N, K)).astype(np.float32)))
    wq, ws, _ = _lib.ft_quantize_blockwise(W, block_rows=32)
    D = dev_bf16(gen.f32_to_bf16_bits(rng.standard_normal((K, 2 * r)).astype(np.float32)))
    U = dev_bf16(gen.f32_to_bf16_bits(rng.standard_normal((2 * r, N)).astype(np.float32)))
    X = torch.empty((0, K), dtype=torch.bfloat16, device=DEV)
    dY = torch.empty((0, N), dtype=torch.bfloat16, device=DEV)
    xq, xs, P = _lib.ft_quantize_blockwise(X, proj=D)
    gq, gs, Qp = _lib.ft_quantize_blockwise(dY, proj=U, proj_layout=_lib.FT_PROJ_R_BY_COLS)
    assert xq.shape == (0, K // 2) and P.shape == (0, 2 * r) and Qp.shape == (0, 2 * r)
    y = _lib.ft_linear_fwd(xq, xs, wq, ws, K, P=P, U=U)
    dx = _lib.ft_linear_bwd_input(gq, gs, wq, ws, K, Qp=Qp, D=D, out_dtype=torch.float32)
    assert y.shape == (0, N) and dx.shape == (0, K)
    dA = torch.full((K, r), 7.0, device=DEV)
    dB = torch.full((r, N), -3.0, device=DEV)
    _lib.ft_lora_grads(X, dY, P, Qp, r, col0=r, dA=dA, dB=dB, accumulate=True)
    torch.cuda.synchronize()
    assert bool((dA == 7.0).all()) and bool((dB == -3.0).all())
    _lib.ft_lora_grads(X, dY, P, Qp, r, col0=r, dA=dA, dB=dB)
    torch.cuda.synchronize()
    assert torch.equal(dA, torch.zeros_like(dA)) and torch.equal(dB, torch.zeros_like(dB))


def test_projection_and_lora_grads_are_reproducible():
    """Partial sums over column and token chunks are combined in a fixed order:
    two runs give the same bits."""
    shape = gen.custom_shape(700, 2080, 1600, r=32, r_s=32)
    d = make_case(shape, 3)
    X, dY, D, U = (dev_bf16(d[k]) for k in ("X", "dY", "D", "U"))
    runs = []
    for _ in range(2):
        _, _, P = _lib.ft_quantize_blockwise(X, proj=D)
        _, _, Qp = _lib.ft_quantize_blockwise(dY, proj=U, proj_layout=_lib.FT_PROJ_R_BY_COLS)
        dA, dB = _lib.ft_lora_grads(X, dY, P, Qp, 32, col0=32)
        torch.cuda.synchronize()
        runs.append([host(t) for t in (P, Qp, dA, dB)])
    for a, b in zip(*runs):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


@pytest.mark.parametrize("M,K,N,r,ld", [(1, 32, 32, 1, 4), (100, 160, 96, 8, 8), (700, 416, 1312, 40, 64),
                                        (257, 3072, 288, 96, 96), (130, 256, 544, 128, 128),
                                        (513, 1184, 2080, 32, 64)])
def test_lora_grads_shapes(M, K, N, r, ld):
    """Adapter gradients with fp32 factors given directly: every rank tile
    count, row strides above r, column counts that leave partial 128-column
    groups and token counts that leave partial 64-row stages."""
    rng = np.random.default_rng(M + K + r)
    X = gen.f32_to_bf16_bits(rng.standard_normal((M, K)).astype(np.float32))
    dY = gen.f32_to_bf16_bits((1e-3 * rng.standard_t(3, (M, N))).astype(np.float32))
    xa = np.zeros((M, ld), np.float32)
    gbt = np.zeros((M, ld), np.float32)
    xa[:, :r] = rng.standard_normal((M, r)).astype(np.float32)
    gbt[:, :r] = (1e-3 * rng.standard_normal((M, r))).astype(np.float32)
    xa[:, r:] = np.float32(7.0)   # columns past r must not reach the outputs
    gbt[:, r:] = np.float32(-5.0)
    dA, dB = _lib.ft_lora_grads(dev_bf16(X), dev_bf16(dY), torch.from_numpy(xa).to(DEV),
                                torch.from_numpy(gbt).to(DEV), r, col0=0)
    torch.cuda.synchronize()
    dAr, dBr, _, _ = ref.lora_grads(X, dY, xa[:, :r].astype(np.float64), gbt[:, :r].astype(np.float64),
                                    want_s=False)
    assert host(dA).shape == (K, r) and host(dB).shape == (r, N)
    assert np.linalg.norm(host(dA) - dAr) <= 1e-3 * np.linalg.norm(dAr)
    assert np.linalg.norm(host(dB) - dBr) <= 1e-3 * np.linalg.norm(dBr)


def test_gemm_random_codes():
    """Arbitrary code bytes (all 16 E2M1 codes) and scales over a wide range,
    with fp32 P given directly: forward and backward against the oracle."""
    rng = np.random.default_rng(5)
    M, K, N, R = 200, 704, 352, 32
    xq = rng.integers(0, 256, (M, K // 2)).astype(np.uint8)
    xs = rng.integers(100, 150, (M, K // 32)).astype(np.uint8)
    wq = rng.integers(0, 256, (N, K // 2)).astype(np.uint8)
    ws = rng.integers(100, 150, (N // 32, K // 32)).astype(np.uint8)
    P = rng.standard_normal((M, R)).astype(np.float32)
    U = gen.f32_to_bf16_bits(rng.standard_normal((R, N)).astype(np.float32))
    y = _lib.ft_linear_fwd(dev_u8(xq), dev_u8(xs), dev_u8(wq), dev_u8(ws), K, torch.from_numpy(P).to(DEV),
                           dev_bf16(U), None, out_dtype=torch.float32)
    gq = rng.integers(0, 256, (M, N // 2)).astype(np.uint8)
    gs = rng.integers(100, 150, (M, N // 32)).astype(np.uint8)
    Qp = rng.standard_normal((M, R)).astype(np.float32)
    D = gen.f32_to_bf16_bits(rng.standard_normal((K, R)).astype(np.float32))
    dx = _lib.ft_linear_bwd_input(dev_u8(gq), dev_u8(gs), dev_u8(wq), dev_u8(ws), K, torch.from_numpy(Qp).to(DEV),
                                  dev_bf16(D), out_dtype=torch.float32)
    torch.cuda.synchronize()
    yr, S = ref.linear_fwd(xq, xs, wq, ws, K, P.astype(np.float64), U, None)
    assert np.all(np.abs(host(y) - yr) <= 1e-5 * S)
    dxr, Sdx = ref.linear_bwd_input(gq, gs, wq, ws, K, Qp.astype(np.float64), D)
    assert np.all(np.abs(host(dx) - dxr) <= 1e-5 * Sdx)


@pytest.mark.parametrize("M,K,N,R", [(300, 640, 384, 48), (129, 128, 128, 16), (257, 1280, 896, 80),
                                     (64, 2304, 640, 0), (520, 1408, 1152, 128), (256, 768, 512, 32),
                                     # paired A-scale stages in both directions, 2x2 tiles and more, R = 64
                                     (520, 1024, 1536, 64), (512, 2048, 512, 64)])
def test_gemm_pipelined_shapes(M, K, N, R):
    """Reduction lengths that are multiples of 128 run the pipelined kernel:
    stage counts from one to nine, a half last stage (length an odd multiple
    of 128) in either direction, low-rank widths with a half last chunk, and
    row counts that leave partial tiles.  Random code bytes and scales, fp32 P;
    both output precisions against the oracle."""
    rng = np.random.default_rng(M + K + N + R)
    xq = rng.integers(0, 256, (M, K // 2)).astype(np.uint8)
    xs = rng.integers(110, 140, (M, K // 32)).astype(np.uint8)
    wq = rng.integers(0, 256, (N, K // 2)).astype(np.uint8)
    ws = rng.integers(110, 140, (N // 32, K // 32)).astype(np.uint8)
    gq = rng.integers(0, 256, (M, N // 2)).astype(np.uint8)
    gs = rng.integers(110, 140, (M, N // 32)).astype(np.uint8)
    bias = gen.f32_to_bf16_bits(rng.standard_normal(N).astype(np.float32))
    Pt = Ut = Qt = Dt = None
    P = U = Qp = D = None
    if R:
        P = rng.standard_normal((M, R)).astype(np.float32)
        U = gen.f32_to_bf16_bits(rng.standard_normal((R, N)).astype(np.float32))
        Qp = rng.standard_normal((M, R)).astype(np.float32)
        D = gen.f32_to_bf16_bits(rng.standard_normal((K, R)).astype(np.float32))
        Pt, Ut = torch.from_numpy(P).to(DEV), dev_bf16(U)
        Qt, Dt = torch.from_numpy(Qp).to(DEV), dev_bf16(D)
    args = (dev_u8(xq), dev_u8(xs), dev_u8(wq), dev_u8(ws), K)
    y32 = _lib.ft_linear_fwd(*args, Pt, Ut, dev_bf16(bias), out_dtype=torch.float32)
    y16 = _lib.ft_linear_fwd(*args, Pt, Ut, dev_bf16(bias), out_dtype=torch.bfloat16)
    gargs = (dev_u8(gq), dev_u8(gs), dev_u8(wq), dev_u8(ws), K)
    dx32 = _lib.ft_linear_bwd_input(*gargs, Qt, Dt, out_dtype=torch.float32)
    dx16 = _lib.ft_linear_bwd_input(*gargs, Qt, Dt, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    f = (lambda a: None if a is None else a.astype(np.float64))
    yr, S = ref.linear_fwd(xq, xs, wq, ws, K, f(P), U, bias)
    check_gemm(host(y32), host(y16), yr, S, "forward")
    dxr, Sdx = ref.linear_bwd_input(gq, gs, wq, ws, K, f(Qp), D)
    check_gemm(host(dx32), host(dx16), dxr, Sdx, "backward-input")


@pytest.mark.parametrize("K", [12288, 15360])
def test_long_reduction_rounds_once_per_mfma_step(K):
    """One fp32 accumulator per output over the whole reduction, rounded once
    per 64-element MFMA step.  Adversarial codes: the first step contributes
    1, every later one a single product of 2^-24 = half an ulp of the running
    sum, which round-half-to-even drops.  The error may then reach
    (K/64 - 1) 2^-24 S, above 1e-5 S from K = 10752 on, but never more than
    K/64 roundings of at most 2^-24 of the running |sum| allow."""
    M, N = 40, 64
    steps = K // 64
    xq = np.zeros((M, K // 2), np.uint8)
    wq = np.zeros((N, K // 2), np.uint8)
    xq[:, ::32] = 0x02            # element 64 j = 1.0 (E2M1 code 2, low nibble)
    wq[:, ::32] = 0x02
    xs = np.full((M, K // 32), 127, np.uint8)
    ws = np.full((N // 32, K // 32), 127, np.uint8)
    xs[:, 2::2] = 115             # blocks holding k = 64 j, j >= 1: 2^-12
    ws[:, 2::2] = 115             # so every later product is 2^-12 * 2^-12 = 2^-24
    y32 = host(_lib.ft_linear_fwd(dev_u8(xq), dev_u8(xs), dev_u8(wq), dev_u8(ws), K, out_dtype=torch.float32))
    torch.cuda.synchronize()
    yr, S = ref.linear_fwd(xq, xs, wq, ws, K, None, None)
    assert np.all(yr == 1.0 + (steps - 1) * 2.0 ** -24)
    err = np.abs(y32.astype(np.float64) - yr)
    print("K = %d: max err / S = %.3g (1e-5 bar; bound %d x 2^-24 = %.3g)" % (K, (err / S).max(), steps,
                                                                            steps * 2.0 ** -24), flush=True)
    assert np.all(err <= steps * 2.0 ** -24 * S)


def test_layer_flux_qkv_full_size_sampled():
    """FLUX.1-dev QKV projection at 1024^2 (M=4608, K=3072, N=9216, r = r_s = 32)
    in the launch configuration the benchmark times: quantized operands
    compared in full, GEMM outputs on two whole 256-row tiles (an interior one
    and the last) and scattered rows, adapter gradients in full."""
    shape = gen.SHAPES["flux_qkv"]
    d = make_case(shape, 0)
    g = run_gpu_layer(d, shape)
    # every row of an interior 256-row tile and of the last one (each output
    # position of the 256x256 tile, i.e. every wave and accumulator slot), plus
    # scattered rows
    rows = np.unique(np.concatenate([[0, 1, 31, 32, 255, 256, 1000, 3333, 4095],
                                     np.arange(2048, 2304), np.arange(4352, 4608)]))
    wq, ws = ref.quantize(d["W"], 32)
    assert np.array_equal(g["wq"], wq) and np.array_equal(g["ws"], ws)
    xq, xs = ref.quantize(d["X"], 1)
    assert np.array_equal(g["xq"], xq) and np.array_equal(g["xs"], xs)
    gq, gs = ref.quantize(d["dY"], 1)
    assert np.array_equal(g["gq"], gq) and np.array_equal(g["gs"], gs)
    check_layer(d, shape, g, rows=rows)
    rs = shape.r_s
    Pf, _ = ref.proj(d["X"], d["D"], 0)
    Qf, _ = ref.proj(d["dY"], d["U"], 1)
    dA, dB, _, _ = ref.lora_grads(d["X"], d["dY"], Pf[:, rs:], Qf[:, rs:], want_s=False)
    assert np.linalg.norm(g["dA"] - dA) <= 1e-3 * np.linalg.norm(dA)
    assert np.linalg.norm(g["dB"] - dB) <= 1e-3 * np.linalg.norm(dB)


@pytest.mark.parametrize("name", ["flux_single_linear1", "flux_single_linear2"])
def test_layer_flux_single_stream_full_size_sampled(name):
    """FLUX.1-dev single-stream block linears at batch 4 (M = 18432 tokens;
    3072 -> 21504 and 15360 -> 3072; LoRA rank 64, stabilizer rank 32), as in
    the stack step: quantized operands and adapter gradients in full, GEMM
    outputs on two whole 256-row tiles (an interior one and the last) and
    scattered rows."""
    shape = gen.SHAPES[name]
    d = make_case(shape, 4)
    g = run_gpu_layer(d, shape)
    rows = np.unique(np.concatenate([[0, 255, 256, 5000, 9999],
                                     np.arange(9984, 10240), np.arange(18176, 18432)]))
    xq, xs = ref.quantize(d["X"], 1)
    assert np.array_equal(g["xq"], xq) and np.array_equal(g["xs"], xs)
    gq, gs = ref.quantize(d["dY"], 1)
    assert np.array_equal(g["gq"], gq) and np.array_equal(g["gs"], gs)
    check_layer(d, shape, g, rows=rows)
    rs = shape.r_s
    Pf, _ = ref.proj(d["X"], d["D"], 0)
    Qf, _ = ref.proj(d["dY"], d["U"], 1)
    dA, dB, _, _ = ref.lora_grads(d["X"], d["dY"], Pf[:, rs:], Qf[:, rs:], want_s=False)
    assert np.linalg.norm(g["dA"] - dA) <= 1e-3 * np.linalg.norm(dA)
    assert np.linalg.norm(g["dB"] - dB) <= 1e-3 * np.linalg.norm(dB)
