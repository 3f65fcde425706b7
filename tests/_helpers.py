"""Input builders shared by the CPU and GPU tests (numpy only)."""
import numpy as np

from paper_2607_05711_amd.gen import bf16_bits_to_f32, f32_to_bf16_bits

E2M1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def adversarial_rows(cols, seed=0):
    """Rows of bf16 bit patterns that stress the block rule: exact ties,
    signed zeros, subnormals, E8M0 extremes, lone outliers, all-zero blocks."""
    g = np.random.default_rng(seed)
    rows = []
    # ties between adjacent E2M1 magnitudes at assorted exponents (amax pinned to 6*2^e)
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])
    for e in (-120, -10, -3, 0, 3, 60, 120):
        v = g.choice(np.concatenate([mids, E2M1, -mids, -E2M1]), cols).astype(np.float64)
        v[::32] = 6.0
        rows.append(f32_to_bf16_bits((v * 2.0 ** e).astype(np.float32)))
    # signed zeros and all-zero blocks
    z = np.zeros(cols, np.uint16)
    z[1::2] = 0x8000
    rows.append(z)
    rows.append(np.zeros(cols, np.uint16))
    rows.append(np.full(cols, 0x8000, np.uint16))
    # subnormal bf16 magnitudes (including the smallest) and mixed tiny blocks
    rows.append(g.integers(0, 0x80, cols).astype(np.uint16) | (g.integers(0, 2, cols).astype(np.uint16) << 15))
    t = g.integers(0, 0x80, cols).astype(np.uint16)
    t[::7] = 0x0080  # smallest normal
    rows.append(t)
    # largest finite magnitudes
    rows.append((g.integers(0x7F00, 0x7F80, cols).astype(np.uint16)) | (g.integers(0, 2, cols).astype(np.uint16) << 15))
    # one huge outlier per block among small values
    v = g.standard_normal(cols).astype(np.float32) * 1e-3
    v[5::32] = 3.0e4
    rows.append(f32_to_bf16_bits(v))
    # saturation band: values in (6, 8) * 2^e next to the block max
    v = g.uniform(-8, 8, cols).astype(np.float32)
    v[::32] = 7.99
    rows.append(f32_to_bf16_bits(v))
    # every bf16 exponent once per row segment
    ex = np.arange(cols) % 254 + 1
    bits = (ex.astype(np.uint16) << 7) | g.integers(0, 0x80, cols).astype(np.uint16)
    rows.append(bits.astype(np.uint16))
    return np.stack(rows)


def random_rows(kind, rows, cols, seed=0):
    g = np.random.default_rng(seed)
    if kind == "normal":
        v = g.standard_normal((rows, cols))
    elif kind == "outliers":
        v = g.standard_normal((rows, cols))
        v[:, g.choice(cols, max(1, cols // 128), replace=False)] *= 50
    elif kind == "laplace":
        v = g.laplace(0, 1e-3, (rows, cols))
    elif kind == "student_t":
        v = 1e-3 * g.standard_t(3, (rows, cols))
    elif kind == "tiny":
        v = g.standard_normal((rows, cols)) * 2.0 ** -128
    elif kind == "huge":
        v = g.standard_normal((rows, cols)) * 2.0 ** 120
    elif kind == "wide":
        v = g.standard_normal((rows, cols)) * 2.0 ** g.integers(-60, 60, (rows, cols))
    else:
        raise ValueError(kind)
    return f32_to_bf16_bits(v.astype(np.float32))


def on_grid_rows(rows, cols, seed=0, e_lo=-6, e_hi=2):
    """bf16 values already on the MXFP4 grid of their own 1x32 blocks, so that
    quantizing them returns them unchanged: every block holds E2M1 multiples
    of 2^e with one element at magnitude 4 or 6 (times 2^e)."""
    g = np.random.default_rng(seed)
    nb = cols // 32
    e = g.integers(e_lo, e_hi + 1, (rows, nb))
    mags = g.choice(E2M1, (rows, nb, 32))
    mags[:, :, g.integers(0, 32)] = g.choice([4.0, 6.0], (rows, nb))
    sign = np.where(g.random((rows, nb, 32)) < 0.5, -1.0, 1.0)
    v = (sign * mags * (2.0 ** e)[:, :, None]).reshape(rows, cols)
    return f32_to_bf16_bits(v.astype(np.float32))


def f64(bits):
    return bf16_bits_to_f32(bits).astype(np.float64)
