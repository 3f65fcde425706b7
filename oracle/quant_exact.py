"""Exact-rational second opinion on the block quantizer.

TEST INFRASTRUCTURE ONLY.  A deliberately different formulation of the same
MXFP4 rule as ft_oracle.c (OCP Microscaling formats, cited in FourTune
Sec. 2.3; block-wise use in Sec. 3.2):

  * bf16 inputs are decoded from their bit fields into Fractions (no float
    conversion);
  * the shared exponent is found by walking powers of two, not by frexp;
  * an element's code is the number of decision thresholds its scaled
    magnitude passes, where each threshold is the midpoint of two adjacent
    E2M1 magnitudes and a magnitude exactly on a midpoint goes to the side
    whose code is even -- instead of a nearest-value search;
  * the no-clip exponent walks down from the top of the E8M0 range while the
    block maximum still fits 6 * 2^e, instead of correcting the floor rule;
  * stochastic rounding compares exact fractions, not floating point.

Pure Python loops: use on small inputs only.
"""
from fractions import Fraction

# (midpoint between code c and c+1, True if a value exactly on it rounds up)
# Codes 0..7 are the magnitudes 0, 1/2, 1, 3/2, 2, 3, 4, 6; the even code of
# each adjacent pair wins the tie.
_THRESHOLDS = [
    (Fraction(1, 4), False),   # 0   | 1/2 : tie -> code 0
    (Fraction(3, 4), True),    # 1/2 | 1   : tie -> code 2
    (Fraction(5, 4), False),   # 1   | 3/2 : tie -> code 2
    (Fraction(7, 4), True),    # 3/2 | 2   : tie -> code 4
    (Fraction(5, 2), False),   # 2   | 3   : tie -> code 4
    (Fraction(7, 2), True),    # 3   | 4   : tie -> code 6
    (Fraction(5, 1), False),   # 4   | 6   : tie -> code 6
]


def bf16_fraction(bits):
    """Exact value of a bf16 bit pattern (finite only) and its sign bit."""
    sign = (bits >> 15) & 1
    exp = (bits >> 7) & 0xFF
    man = bits & 0x7F
    if exp == 0xFF:
        raise ValueError("non-finite bf16")
    if exp == 0:
        mag = Fraction(man, 1 << 7) * Fraction(1, 1 << 126)
    else:
        mag = Fraction(128 + man, 128)
        e = exp - 127
        mag = mag * (Fraction(1 << e) if e >= 0 else Fraction(1, 1 << -e))
    return mag, sign


def _pow2(e):
    return Fraction(1 << e) if e >= 0 else Fraction(1, 1 << -e)


def _floor_log2(x):
    """Largest k with 2^k <= x, for a positive Fraction x."""
    k = 0
    while _pow2(k) > x:
        k -= 1
    while _pow2(k + 1) <= x:
        k += 1
    return k


# E2M1 magnitudes in code order, as exact fractions.
_GRID = [Fraction(0), Fraction(1, 2), Fraction(1), Fraction(3, 2), Fraction(2), Fraction(3), Fraction(4),
         Fraction(6)]


def _no_clip_exponent(amax):
    """The smallest e in [-127, 127] with amax <= 6 * 2^e, found by walking
    down from an exponent that satisfies it."""
    e = 127
    while e > -127 and amax <= 6 * _pow2(e - 1):
        e -= 1
    return e


def quantize_block(bits_list, scale_rule=0, uniforms=None):
    """bf16 bit patterns of one block -> (E8M0 code, list of 4-bit codes).

    scale_rule 0: the floor rule; 1: the no-clip rule (smallest exponent at
    which the block maximum is not above 6).  uniforms: None for
    nearest-even rounding, else one 16-bit integer u per element for
    stochastic rounding: a magnitude strictly between two grid values lo < hi
    moves up when (t - lo) / (hi - lo) > (2u + 1) / 2^17."""
    vals = [bf16_fraction(b) for b in bits_list]
    amax = max(m for m, _ in vals)
    if amax == 0:
        e = -127
    elif scale_rule == 0:
        e = max(-127, min(127, _floor_log2(amax) - 2))
    else:
        e = _no_clip_exponent(amax)
    codes = []
    for i, (mag, sign) in enumerate(vals):
        t = mag / _pow2(e)
        if uniforms is None:
            code = 0
            for thr, tie_up in _THRESHOLDS:
                if t > thr or (t == thr and tie_up):
                    code += 1
        elif t >= 6:
            code = 7
        else:
            code = max(c for c in range(8) if _GRID[c] <= t)
            if _GRID[code] != t and (t - _GRID[code]) / (_GRID[code + 1] - _GRID[code]) > \
                    Fraction(2 * int(uniforms[i]) + 1, 1 << 17):
                code += 1
        codes.append(code | (sign << 3))
    return e + 127, codes


def quantize_rows(bits, block_rows=1, scale_rule=0, uniforms=None):
    """bits: 2-D list/array of bf16 patterns -> (packed codes, scales) as lists.

    Packing: element 2i of a row in bits 3:0 of byte i, element 2i+1 in 7:4.
    uniforms: None (nearest-even) or a 2-D array of 16-bit integers, one per
    element (stochastic rounding).
    """
    rows = len(bits)
    cols = len(bits[0])
    nibbles = [[0] * cols for _ in range(rows)]
    scales = [[0] * (cols // 32) for _ in range(rows // block_rows)]
    for br in range(rows // block_rows):
        for bc in range(cols // 32):
            block = [int(bits[br * block_rows + i][bc * 32 + j])
                     for i in range(block_rows) for j in range(32)]
            u = None if uniforms is None else [int(uniforms[br * block_rows + i][bc * 32 + j])
                                               for i in range(block_rows) for j in range(32)]
            s, codes = quantize_block(block, scale_rule, u)
            scales[br][bc] = s
            n = 0
            for i in range(block_rows):
                for j in range(32):
                    nibbles[br * block_rows + i][bc * 32 + j] = codes[n]
                    n += 1
    packed = [[nibbles[r][2 * i] | (nibbles[r][2 * i + 1] << 4) for i in range(cols // 2)]
              for r in range(rows)]
    return packed, scales
