"""Pins of the oracle's number formats and block quantizer (CPU only).

The oracle's quantizer is checked against things it does not itself contain:
the E2M1/E8M0 bit-field definitions, an exact-rational threshold quantizer
written differently, the rule's invariants, hand-worked blocks, the
re-quantization identity and the 32x32 transpose property the backward pass
relies on (FourTune Sec. 3.2).
"""
import math
import os
import zlib

import numpy as np
import pytest

from oracle import quant_exact, ref
from paper_2607_05711_amd.gen import bf16_bits_to_f32, f32_to_bf16_bits
from tests._helpers import adversarial_rows, on_grid_rows, random_rows

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "mxfp4_blocks.txt")


def e2m1_from_bits(code):
    """E2M1 by its bit fields: sign | 2-bit exponent (bias 1) | 1-bit mantissa."""
    s, e, m = (code >> 3) & 1, (code >> 1) & 3, code & 1
    mag = (m / 2.0) if e == 0 else 2.0 ** (e - 1) * (1 + m / 2.0)
    return -mag if s else mag


def test_e2m1_decode_all_codes():
    for code in range(16):
        got = ref.e2m1_value(code)
        want = e2m1_from_bits(code)
        assert got == want and math.copysign(1, got) == math.copysign(1, want), code


def test_e8m0_decode_all_codes():
    for code in range(255):
        assert ref.e8m0_value(code) == math.ldexp(1.0, code - 127)
    assert math.isnan(ref.e8m0_value(255))


def _load_golden():
    cases = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        name, inp, scale, codes = [p.strip() for p in line.split("|")]
        bits = np.zeros(32, np.uint16)
        vals = [int(x, 16) for x in inp.split()]
        bits[: len(vals)] = vals
        cases.append((name, bits, int(scale, 16), bytes(int(x, 16) for x in codes.split())))
    return cases


@pytest.mark.parametrize("case", _load_golden(), ids=lambda c: c[0])
def test_golden_blocks(case):
    name, bits, scale, codes = case
    rule = 1 if name.startswith("noclip-") else 0
    q, s = ref.quantize_ex(bits[None, :], 1, scale_rule=rule) if rule else ref.quantize(bits[None, :], 1)
    assert int(s[0, 0]) == scale, name
    assert bytes(q[0]) == codes, name
    # the exact-rational formulation agrees on the worked example too
    pq, ps = quant_exact.quantize_rows(bits[None, :].tolist(), scale_rule=rule)
    assert ps[0][0] == scale and bytes(pq[0]) == codes


@pytest.mark.parametrize("kind", ["normal", "outliers", "laplace", "student_t", "tiny", "huge", "wide"])
def test_matches_exact_rational_quantizer(kind):
    bits = random_rows(kind, 24, 256, seed=zlib.crc32(kind.encode()) % 1000)
    q, s = ref.quantize(bits, 1)
    pq, ps = quant_exact.quantize_rows(bits.tolist())
    assert np.array_equal(q, np.array(pq, np.uint8))
    assert np.array_equal(s, np.array(ps, np.uint8))


def test_matches_exact_rational_quantizer_adversarial():
    bits = adversarial_rows(256, seed=3)
    q, s = ref.quantize(bits, 1)
    pq, ps = quant_exact.quantize_rows(bits.tolist())
    assert np.array_equal(q, np.array(pq, np.uint8))
    assert np.array_equal(s, np.array(ps, np.uint8))


def test_matches_exact_rational_quantizer_tiles():
    bits = random_rows("outliers", 64, 64, seed=5)
    q, s = ref.quantize(bits, 32)
    pq, ps = quant_exact.quantize_rows(bits.tolist(), block_rows=32)
    assert np.array_equal(q, np.array(pq, np.uint8))
    assert np.array_equal(s, np.array(ps, np.uint8))


def _unpack(q):
    return np.stack([q & 0xF, q >> 4], axis=-1).reshape(q.shape[0], -1)


@pytest.mark.parametrize("kind", ["normal", "laplace", "wide", "huge"])
def test_scale_invariant_and_nearest(kind):
    """amax * 2^-e lies in [4, 8) unless e is clamped at -127, and every code
    is a nearest E2M1 magnitude of |v| 2^-e (brute force over all 8)."""
    bits = random_rows(kind, 64, 256, seed=11)
    q, s = ref.quantize(bits, 1)
    v = bf16_bits_to_f32(bits).astype(np.float64)
    e = s.astype(np.int64) - 127
    blocks = np.abs(v).reshape(64, 8, 32)
    amax = blocks.max(axis=2)
    t = amax * np.exp2(-e.astype(np.float64))
    ok = (t >= 4) & (t < 8) | ((e == -127) & (t < 8)) | (amax == 0)
    assert ok.all()
    codes = _unpack(q).reshape(64, 8, 32)
    tt = blocks * np.exp2(-e.astype(np.float64))[:, :, None]
    grid = np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6])
    chosen = grid[codes & 7]
    best = np.abs(tt[..., None] - grid).min(axis=-1)
    assert np.all(np.abs(tt - chosen) == best)
    # sign bit copied
    neg = np.signbit(v).reshape(64, 8, 32)
    assert np.array_equal((codes >> 3).astype(bool), neg)


@pytest.mark.parametrize("kind", ["normal", "outliers", "laplace", "student_t", "tiny", "huge", "wide"])
def test_round_trip_identity(kind):
    """Q(DQ(Q(x))) == Q(x): dequantized blocks are bf16-exact and requantize
    to the same codes and scales (2^14 blocks per distribution)."""
    bits = random_rows(kind, 512, 1024, seed=7)
    q, s = ref.quantize(bits, 1)
    dq = ref.dequantize(q, s, 1024, 1)
    f = dq.astype(np.float32)
    assert np.array_equal(f.astype(np.float64), dq)  # exact in fp32
    b2 = f32_to_bf16_bits(f)
    assert np.array_equal(bf16_bits_to_f32(b2).astype(np.float64), dq)  # exact in bf16
    q2, s2 = ref.quantize(b2, 1)
    assert np.array_equal(q2, q) and np.array_equal(s2, s)


def test_round_trip_identity_tiles_and_adversarial():
    bits = adversarial_rows(1024, seed=9)
    q, s = ref.quantize(bits, 1)
    b2 = f32_to_bf16_bits(ref.dequantize(q, s, 1024, 1).astype(np.float32))
    q2, s2 = ref.quantize(b2, 1)
    assert np.array_equal(q2, q) and np.array_equal(s2, s)
    w = random_rows("outliers", 256, 512, seed=2)
    q, s = ref.quantize(w, 32)
    b2 = f32_to_bf16_bits(ref.dequantize(q, s, 512, 32).astype(np.float32))
    q2, s2 = ref.quantize(b2, 32)
    assert np.array_equal(q2, q) and np.array_equal(s2, s)


def test_on_grid_inputs_are_fixed_points():
    bits = on_grid_rows(64, 256, seed=1)
    q, s = ref.quantize(bits, 1)
    assert np.array_equal(ref.dequantize(q, s, 256, 1), bf16_bits_to_f32(bits).astype(np.float64))


def test_tile_transpose_property():
    """32x32 tiles: quantizing W^T gives the transposed codes and scale grid,
    so the backward GEMM can read Q(W) transposed without re-quantizing."""
    w = random_rows("outliers", 96, 160, seed=4)
    q, s = ref.quantize(w, 32)
    qt, st = ref.quantize(np.ascontiguousarray(w.T), 32)
    assert np.array_equal(st, s.T)
    assert np.array_equal(_unpack(qt), _unpack(q).T)


def test_tile_scale_covers_whole_tile():
    """One scale per 32x32 tile: an outlier anywhere in the tile sets it."""
    w = np.full((64, 64), f32_to_bf16_bits(np.array([1.0], np.float32))[0], np.uint16)
    w[37, 5] = f32_to_bf16_bits(np.array([100.0], np.float32))[0]
    _, s = ref.quantize(w, 32)
    assert s[1, 0] == 127 + 6 - 2 and s[0, 0] == s[0, 1] == s[1, 1] == 125


def test_rejects_bad_shapes():
    with pytest.raises(ValueError):
        ref.quantize(np.zeros((2, 48), np.uint16), 1)
    with pytest.raises(ValueError):
        ref.quantize(np.zeros((48, 64), np.uint16), 32)
