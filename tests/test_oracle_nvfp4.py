"""Pins of the oracle's NVFP4 emulation (CPU only).

NVFP4 is the format FourTune Sec. 3.1 names: E2M1 elements with one FP8 E4M3
scale per 16 elements and one FP32 scale per tensor; Sec. 4.3 uses 16x16
blocks for the weight.  The build's native format is MXFP4 (E8M0 per 32);
this emulation is an accuracy cross-check.  Pinned against: the E4M3 bit-field
definition, torch's float8_e4m3fn conversion (a library routine, round to
nearest even), an exact-rational element quantizer, the transpose property
of 16x16 tiles, a hand-worked tensor (tests/golden/nvfp4_blocks.txt) and
numpy products.
"""
import os
import struct
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import quant_exact, ref
from tests._helpers import f64, random_rows

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "nvfp4_blocks.txt")
E2M1 = [Fraction(0), Fraction(1, 2), Fraction(1), Fraction(3, 2), Fraction(2), Fraction(3), Fraction(4), Fraction(6)]


def e4m3_from_bits(code):
    s, e, m = (code >> 7) & 1, (code >> 3) & 15, code & 7
    if e == 15 and m == 7:
        return None
    v = Fraction(m, 8) * Fraction(1, 64) if e == 0 else (1 + Fraction(m, 8)) * Fraction(2) ** (e - 7)
    return -v if s else v


def test_e4m3_decode_all_codes():
    for code in range(256):
        want = e4m3_from_bits(code)
        got = ref.e4m3_value(code)
        if want is None:
            assert np.isnan(got)
        else:
            assert Fraction(got) == want, code
    assert ref.e4m3_value(0x7E) == 448.0 and ref.e4m3_value(1) == 2.0 ** -9


def test_block_scale_encoding_matches_torch_float8():
    """The block scale is the E4M3 value nearest to amax_b / (6 st): checked
    against torch's float8_e4m3fn conversion of the same fp32 quotient."""
    bits = random_rows("wide", 48, 512, seed=3)
    q, s, st = ref.quantize_nvfp4(bits, 1)
    amax_b = np.abs(f64(bits)).reshape(48, 32, 16).max(axis=2).astype(np.float32)
    d = amax_b / np.float32(np.float32(6.0) * np.float32(st))
    assert d.max() <= 448.0 * (1 + 2 ** -20)
    want = torch.from_numpy(np.minimum(d, np.float32(448.0))).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(s, want)


def test_tensor_scale_is_amax_over_2688_in_fp32():
    bits = random_rows("outliers", 64, 256, seed=4)
    amax = np.float32(np.abs(f64(bits)).max())
    assert ref.nvfp4_tensor_scale(bits) == float(amax / np.float32(2688.0))


def test_elements_match_exact_rational_nearest():
    bits = random_rows("student_t", 24, 128, seed=5)
    q, s, st = ref.quantize_nvfp4(bits, 1)
    stf = Fraction(st)
    codes = np.stack([q & 15, q >> 4], -1).reshape(24, 128)
    for r in range(24):
        for c in range(128):
            mag, sign = quant_exact.bf16_fraction(int(bits[r, c]))
            bs = Fraction(ref.e4m3_value(int(s[r, c // 16]))) * stf
            t = mag / bs if bs else Fraction(0)
            if t >= 6:
                want = 7
            else:
                dist = [abs(t - g) for g in E2M1]
                best = min(dist)
                cands = [i for i, dd in enumerate(dist) if dd == best]
                want = min(cands, key=lambda i: (i & 1, i))    # a tie goes to the even code
            assert int(codes[r, c]) == want | (sign << 3), (r, c)


def test_dequantized_values_and_transpose_property():
    w = random_rows("normal", 64, 96, seed=6)
    q, s, st = ref.quantize_nvfp4(w, 16)
    qt, stt, st2 = ref.quantize_nvfp4(np.ascontiguousarray(w.T), 16)
    assert st2 == st and np.array_equal(stt, s.T)
    d, dt = ref.dequantize_nvfp4(q, s, st, 96, 16), ref.dequantize_nvfp4(qt, stt, st, 64, 16)
    assert np.array_equal(dt, d.T)
    # every value is within half an element step of its input, and none exceeds 6 * E4M3 * st
    v = f64(w)
    bs = np.repeat(np.repeat(np.array([[ref.e4m3_value(int(c)) for c in row] for row in s]), 16, 0), 16, 1) * st
    assert np.all(np.abs(d) <= 6 * bs * (1 + 1e-12))
    assert np.all((np.abs(np.abs(d) - np.abs(v)) <= 1.0 * bs) | (np.abs(v) > 6 * bs))


def _golden():
    out = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        name, blocks, st, scales, codes = [p.strip() for p in line.split("|")]
        bits = np.zeros((1, 48), np.uint16)
        for blk in blocks.split(";"):
            i, vals = blk.split(":")
            v = [int(x, 16) for x in vals.split()]
            bits[0, 16 * int(i):16 * int(i) + len(v)] = v
        out.append((name, bits, struct.unpack(">f", bytes.fromhex(st))[0], [int(x, 16) for x in scales.split()],
                    bytes(int(x, 16) for x in codes.split())))
    return out


@pytest.mark.parametrize("case", _golden(), ids=lambda c: c[0])
def test_golden_nvfp4(case):
    name, bits, st_want, scales, codes = case
    q, s, st = ref.quantize_nvfp4(bits, 1)
    assert st == st_want
    assert list(s[0]) == scales
    assert bytes(q[0]) == codes


def test_gemm_f64_against_numpy_and_rationals():
    rng = np.random.default_rng(7)
    a = rng.integers(-8, 8, (5, 48)) / 4.0
    b = rng.integers(-8, 8, (6, 48)) / 8.0
    y, s = ref.gemm_f64(a, b, trans_b=True)
    for m in range(5):
        for n in range(6):
            assert Fraction(y[m, n]) == sum(Fraction(a[m, k]) * Fraction(b[n, k]) for k in range(48))
            assert Fraction(s[m, n]) == sum(abs(Fraction(a[m, k]) * Fraction(b[n, k])) for k in range(48))
    bt = np.ascontiguousarray(b.T)
    y2, _ = ref.gemm_f64(a, bt, trans_b=False)
    assert np.array_equal(y, y2)
    A = rng.standard_normal((40, 64)); B = rng.standard_normal((30, 64))
    y3, s3 = ref.gemm_f64(A, B)
    assert np.all(np.abs(y3 - A @ B.T) <= 1e-12 * s3)


def test_nvfp4_versus_mxfp4_accuracy():
    """Accuracy cross-check of the two formats on an activation with outlier
    channels times a weight (the layer's forward product, no low-rank terms):
    NVFP4's 16-element blocks with E4M3 scales track the exact product more
    closely than MXFP4's 32-element power-of-two blocks."""
    x = random_rows("outliers", 64, 512, seed=8)
    w = random_rows("normal", 96, 512, seed=9)
    exact = f64(x) @ f64(w).T
    xq, xs = ref.quantize(x, 1); wq, ws = ref.quantize(w, 32)
    y_mx, _ = ref.gemm_f64(ref.dequantize(xq, xs, 512, 1), ref.dequantize(wq, ws, 512, 32))
    nq, ns, nt = ref.quantize_nvfp4(x, 1); mq, ms, mt = ref.quantize_nvfp4(w, 16)
    y_nv, _ = ref.gemm_f64(ref.dequantize_nvfp4(nq, ns, nt, 512, 1), ref.dequantize_nvfp4(mq, ms, mt, 512, 16))
    e_mx = np.linalg.norm(y_mx - exact) / np.linalg.norm(exact)
    e_nv = np.linalg.norm(y_nv - exact) / np.linalg.norm(exact)
    assert e_nv < e_mx < 0.3, (e_nv, e_mx)
