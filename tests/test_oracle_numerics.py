"""Pins of the oracle's numerics variants of Q(.) (CPU only).

FourTune Sec. 3.1 fixes the 4-bit format but not the quantizer's scale rule or
rounding; these variants cover the readings the layer's default leaves out:
  * the no-clip shared exponent (smallest e with max|v| <= 6 * 2^e);
  * stochastic rounding of the elements, with random bits from Philox4x32-10
    (Salmon, Moraes, Dror, Shaw, SC 2011);
  * 2-D (32x32) blocks for activations.
Pinned against: the generator's published known-answer vectors, an
exact-rational second quantizer (oracle/quant_exact.py, a different
formulation), the rules' invariants, hand-worked blocks
(tests/golden/mxfp4_blocks.txt), and the unbiasedness of stochastic rounding.
"""
import numpy as np
import pytest

from oracle import quant_exact, ref
from tests._helpers import adversarial_rows, random_rows

E2M1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


# Known-answer vectors of Philox4x32-10 from the generator's reference
# distribution (Random123): (counter, key) -> output.
PHILOX_KAT = [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2, (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


@pytest.mark.parametrize("ctr,key,want", PHILOX_KAT)
def test_philox_known_answers(ctr, key, want):
    assert tuple(int(x) for x in ref.philox4x32_10(ctr, key)) == want


def test_sr_bits_layout_and_uniformity():
    seed, stream = 0x1234_5678_9ABC_DEF0, 7
    # element idx takes half idx % 2 of word (idx % 8) / 2 of the block idx / 8
    for idx in (0, 1, 2, 7, 8, 13, 1 << 33 | 5):
        q = idx >> 3
        out = ref.philox4x32_10((q & 0xFFFFFFFF, q >> 32, stream, 0), (seed & 0xFFFFFFFF, seed >> 32))
        assert ref.sr_bits(seed, stream, idx) == (int(out[(idx & 7) >> 1]) >> (16 * (idx & 1))) & 0xFFFF
    u = np.array([ref.sr_bits(3, 0, i) for i in range(1 << 15)])
    for part in (u >> 12, u & 15):            # top and bottom 4 bits: 16 bins, chi-square with 15 dof
        h = np.bincount(part, minlength=16)
        chi2 = ((h - len(u) / 16) ** 2 / (len(u) / 16)).sum()
        assert chi2 < 50, chi2


def _blocks():
    rows = [adversarial_rows(256, seed=4)]
    for i, kind in enumerate(("normal", "outliers", "student_t", "wide", "tiny", "huge")):
        rows.append(random_rows(kind, 8, 256, seed=40 + i))
    return np.concatenate(rows)


def test_no_clip_rule_invariants():
    bits = _blocks()
    q, s = ref.quantize_ex(bits, 1, scale_rule=1)
    vals = np.array([[quant_exact.bf16_fraction(int(b))[0] for b in row] for row in bits], dtype=object)
    for r in range(bits.shape[0]):
        for b in range(8):
            amax = max(vals[r, 32 * b:32 * b + 32])
            e = int(s[r, b]) - 127
            if amax == 0:
                assert e == -127
                continue
            # the block maximum fits 6 * 2^e, and 2^(e-1) would not fit it (unless clamped)
            assert amax <= 6 * quant_exact._pow2(e)
            assert e == -127 or amax > 6 * quant_exact._pow2(e - 1)
    # nothing saturates: every |DQ| is within half a grid step of |v| (no value is cut to 6 * 2^e)
    d = ref.dequantize(q, s, 256)
    v = np.array([[float(m) for m in row] for row in vals])
    scale = np.repeat(2.0 ** (s.astype(np.int64) - 127), 32, axis=1)
    assert np.all(np.abs(np.abs(d) - v) <= 1.0 * scale + 1e-300)


def test_no_clip_matches_exact_rational_quantizer():
    bits = _blocks()
    q, s = ref.quantize_ex(bits, 1, scale_rule=1)
    pq, ps = quant_exact.quantize_rows(bits.tolist(), scale_rule=1)
    assert np.array_equal(s, np.array(ps, np.uint8))
    assert np.array_equal(q, np.array(pq, np.uint8))
    q32, s32 = ref.quantize_ex(bits[:32], 32, scale_rule=1)
    pq, ps = quant_exact.quantize_rows(bits[:32].tolist(), block_rows=32, scale_rule=1)
    assert np.array_equal(s32, np.array(ps, np.uint8)) and np.array_equal(q32, np.array(pq, np.uint8))


def test_no_clip_value_round_trip():
    """Re-quantizing dequantized values keeps every value (the grid of 2^e is
    contained in that of 2^(e-1) where the maximum allows it) although the
    scale byte may drop by one (golden block noclip-H)."""
    bits = _blocks()
    q, s = ref.quantize_ex(bits, 1, scale_rule=1)
    d = ref.dequantize(q, s, 256)
    # Rounding up may carry a block maximum near the top of the bf16 range to
    # 2^128, past the largest finite bf16: such rows have no bf16 round trip.
    fits = np.all(np.abs(d) < 2.0 ** 127, axis=1)
    assert fits.sum() >= d.shape[0] - 8 and not fits.all()
    d = d[fits]
    from paper_2607_05711_amd.gen import bf16_bits_to_f32, f32_to_bf16_bits
    d_bits = f32_to_bf16_bits(d.astype(np.float32))
    assert np.array_equal(d, bf16_bits_to_f32(d_bits).astype(np.float64)), "dequantized values are bf16-exact"
    q2, s2 = ref.quantize_ex(d_bits, 1, scale_rule=1)
    assert np.array_equal(ref.dequantize(q2, s2, 256), d)
    assert np.any(s2 != s[fits])


def _uniforms(rows, cols, seed, stream):
    return np.array([[ref.sr_bits(seed, stream, r * cols + c) for c in range(cols)] for r in range(rows)])


@pytest.mark.parametrize("rule", [0, 1])
def test_stochastic_rounding_matches_exact_rational(rule):
    bits = _blocks()[:40, :128].copy()
    seed, stream = 99, 3
    q, s = ref.quantize_ex(bits, 1, scale_rule=rule, rounding=1, seed=seed, stream=stream)
    u = _uniforms(bits.shape[0], 128, seed, stream)
    pq, ps = quant_exact.quantize_rows(bits.tolist(), scale_rule=rule, uniforms=u)
    assert np.array_equal(s, np.array(ps, np.uint8))
    assert np.array_equal(q, np.array(pq, np.uint8))
    # the scales are the rounding-independent ones
    assert np.array_equal(s, ref.quantize_ex(bits, 1, scale_rule=rule)[1])


def test_stochastic_rounding_picks_a_neighbour():
    bits = _blocks()
    q, s = ref.quantize_ex(bits, 1, rounding=1, seed=5, stream=11)
    d = np.abs(ref.dequantize(q, s, 256))
    v = np.array([[float(quant_exact.bf16_fraction(int(b))[0]) for b in row] for row in bits])
    scale = np.repeat(2.0 ** (s.astype(np.int64) - 127), 32, axis=1)
    t, g = v / scale, d / scale
    lo = np.array([E2M1[E2M1 <= x].max() if x < 6 else 6.0 for x in t.ravel()]).reshape(t.shape)
    hi = np.array([E2M1[E2M1 > x].min() if x < 6 else 6.0 for x in t.ravel()]).reshape(t.shape)
    on_grid = np.isin(t, E2M1)
    assert np.all((g == lo) | (g == hi))
    assert np.all(g[on_grid] == t[on_grid])          # grid values never move


@pytest.mark.parametrize("rule", [0, 1])
def test_stochastic_rounding_is_unbiased(rule):
    """Averaged over many independent streams, DQ(SR(v)) converges to v: the
    mean error of each element is within 6 standard errors.  Under the floor
    rule a block maximum above 6 * 2^e saturates, which no rounding undoes:
    those elements are left out there; the no-clip rule has none."""
    rng = np.random.default_rng(0)
    from paper_2607_05711_amd.gen import f32_to_bf16_bits
    bits = f32_to_bf16_bits(rng.standard_normal((1, 64)).astype(np.float32))
    v = np.array([float(quant_exact.bf16_fraction(int(b))[0]) * (-1 if b >> 15 else 1) for b in bits[0]])
    n = 3000
    acc = np.zeros(64)
    acc2 = np.zeros(64)
    for st in range(n):
        q, s = ref.quantize_ex(bits, 1, scale_rule=rule, rounding=1, seed=1, stream=st)
        d = ref.dequantize(q, s, 64)[0]
        acc += d
        acc2 += d * d
    mean = acc / n
    sd = np.sqrt(np.maximum(acc2 / n - mean ** 2, 0)) + 1e-12
    scale = np.repeat(2.0 ** (s[0].astype(np.int64) - 127), 32)
    keep = np.abs(v) <= 6 * scale
    assert keep.sum() >= 56 and (rule == 0 or keep.all())
    assert np.all((np.abs(mean - v) <= 6 * sd / np.sqrt(n) + 2.0 ** -16 * np.abs(v))[keep])
    # nearest-even, on the same values, is biased by more than that
    rq, rs = ref.quantize_ex(bits, 1, scale_rule=rule)
    assert np.abs(ref.dequantize(rq, rs, 64)[0] - v)[keep].max() > 10 * np.abs(mean - v)[keep].max()


def test_stochastic_rounding_depends_only_on_seed_stream_and_index():
    bits = random_rows("normal", 16, 256, seed=2)
    a = ref.quantize_ex(bits, 1, rounding=1, seed=7, stream=1)
    b = ref.quantize_ex(bits, 1, rounding=1, seed=7, stream=1)
    c = ref.quantize_ex(bits, 1, rounding=1, seed=7, stream=2)
    assert np.array_equal(a[0], b[0]) and not np.array_equal(a[0], c[0])
    # a row block quantized on its own draws the same bits as inside the matrix only when its
    # element indices are the same: rows are keyed by their index in the matrix
    top = ref.quantize_ex(bits[:8], 1, rounding=1, seed=7, stream=1)
    assert np.array_equal(top[0], a[0][:8])


def test_two_dimensional_activation_blocks():
    """2-D (32x32) blocks for activations: the tile rule of the weight applied
    to X; one scale per tile, shared by its 32 rows.  The per-row layout the
    GEMM reads is each row carrying its tile's scale."""
    bits = random_rows("outliers", 64, 256, seed=9)
    q, s = ref.quantize(bits, 32)
    pq, ps = quant_exact.quantize_rows(bits.tolist(), block_rows=32)
    assert np.array_equal(q, np.array(pq, np.uint8)) and np.array_equal(s, np.array(ps, np.uint8))
    per_row = np.repeat(s, 32, axis=0)
    assert np.array_equal(ref.dequantize(q, per_row, 256, 1), ref.dequantize(q, s, 256, 32))
