"""Seeded synthetic inputs shaped like FLUX.1-dev linear layers.

This module is shared by the tests, the smoke check and the benchmark on both
sides of the parity check (the GPU library and the CPU oracle).  It only draws
random numbers and rounds them to bf16; it holds none of the layer's
arithmetic (no quantization, no products).  Where an input depends on the
method (the stabilizer factors come from the weight's quantization residual),
the caller passes the residual in.

bf16 tensors are returned as numpy uint16 bit patterns (round-to-nearest-even
from float32 draws).  Every tensor has its own random stream,
``default_rng([seed, tensor_id])``, so draw order never matters.
"""
from dataclasses import dataclass

import numpy as np

TENSOR_IDS = {"X": 1, "W": 2, "A": 3, "B": 4, "STAB": 5, "DY": 6, "BIAS": 7, "OUTLIER": 8}


def rng(seed, name):
    return np.random.default_rng([int(seed), TENSOR_IDS[name]])


def f32_to_bf16_bits(a):
    """float32 array -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(b):
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass(frozen=True)
class LayerShape:
    """One triple-branch linear: X[M,K] -> Y[M,N]; LoRA rank r, stabilizer rank r_s."""
    name: str
    M: int
    K: int
    N: int
    r: int
    r_s: int
    n_outliers: int          # activation channels (columns of X) scaled up
    outlier_scale: float
    dy_kind: str             # "laplace" or "student_t3"
    dy_scale: float

    @property
    def R(self):
        return self.r + self.r_s


def _n_outliers(K, frac):
    return int(round(frac * K))


# Workloads.  FLUX.1-dev at 1024x1024: 4096 image + 512 text tokens, hidden
# size 3072, MLP width 12288, single-stream fused widths 21504 / 15360.
SHAPES = {
    # small parity case: 2 of 256 channels x50, Laplace(0, 1e-3) gradients
    "tiny": LayerShape("tiny", 128, 256, 256, 16, 16, 2, 50.0, "laplace", 1e-3),
    # attention QKV projection, batch 1
    "flux_qkv": LayerShape("flux_qkv", 4608, 3072, 9216, 32, 32, _n_outliers(3072, 0.005), 30.0,
                           "student_t3", 1e-3),
    # double-stream attention output projection
    "flux_attn_out": LayerShape("flux_attn_out", 4608, 3072, 3072, 32, 32, _n_outliers(3072, 0.005),
                                30.0, "student_t3", 1e-3),
    # MLP pair, batch 1
    "flux_mlp_up": LayerShape("flux_mlp_up", 4608, 3072, 12288, 32, 32, _n_outliers(3072, 0.005),
                              30.0, "student_t3", 1e-3),
    "flux_mlp_down": LayerShape("flux_mlp_down", 4608, 12288, 3072, 32, 32,
                                _n_outliers(12288, 0.005), 30.0, "student_t3", 1e-3),
    # single-stream block linears, batch 4
    "flux_single_linear1": LayerShape("flux_single_linear1", 18432, 3072, 21504, 64, 32,
                                      _n_outliers(3072, 0.005), 30.0, "student_t3", 1e-3),
    "flux_single_linear2": LayerShape("flux_single_linear2", 18432, 15360, 3072, 64, 32,
                                      _n_outliers(15360, 0.005), 30.0, "student_t3", 1e-3),
}


def custom_shape(M, K, N, r=16, r_s=16, n_outliers=2, outlier_scale=50.0,
                 dy_kind="laplace", dy_scale=1e-3, name="custom"):
    return LayerShape(name, M, K, N, r, r_s, n_outliers, outlier_scale, dy_kind, dy_scale)


def draw_x(shape, seed):
    """Activations ~ N(0,1) with n_outliers whole channels scaled up."""
    x = rng(seed, "X").standard_normal((shape.M, shape.K), dtype=np.float32)
    if shape.n_outliers:
        cols = rng(seed, "OUTLIER").choice(shape.K, shape.n_outliers, replace=False)
        x[:, cols] *= np.float32(shape.outlier_scale)
    return f32_to_bf16_bits(x)


def draw_dy(shape, seed):
    g = rng(seed, "DY")
    if shape.dy_kind == "laplace":
        d = g.laplace(0.0, shape.dy_scale, (shape.M, shape.N)).astype(np.float32)
    elif shape.dy_kind == "student_t3":
        d = (shape.dy_scale * g.standard_t(3, (shape.M, shape.N))).astype(np.float32)
    else:
        raise ValueError(shape.dy_kind)
    return f32_to_bf16_bits(d)


def draw_w(shape, seed):
    return f32_to_bf16_bits(0.02 * rng(seed, "W").standard_normal((shape.N, shape.K), dtype=np.float32))


def draw_lora(shape, seed):
    A = f32_to_bf16_bits(0.01 * rng(seed, "A").standard_normal((shape.K, shape.r), dtype=np.float32))
    B = f32_to_bf16_bits(0.01 * rng(seed, "B").standard_normal((shape.r, shape.N), dtype=np.float32))
    return A, B


def draw_bias(shape, seed):
    return f32_to_bf16_bits(0.02 * rng(seed, "BIAS").standard_normal(shape.N, dtype=np.float32))


def stabilizer_from_residual(residual, r_s):
    """Rank-r_s factors of a weight residual E[N, K] (fp64), by exact SVD.

    E^T = V S U'^T  ->  L1 = V_r S_r [K, r_s],  L2 = U'_r^T [r_s, N], rounded to bf16,
    so that L1 L2 approximates E^T (the paper's weight orientation, Eq. (1)).
    """
    Et = np.asarray(residual, dtype=np.float64).T
    V, S, Uh = np.linalg.svd(Et, full_matrices=False)
    L1 = V[:, :r_s] * S[:r_s]
    L2 = Uh[:r_s, :]
    return f32_to_bf16_bits(L1.astype(np.float32)), f32_to_bf16_bits(L2.astype(np.float32))


def stabilizer_random(shape, seed, std1=0.01, std2=0.01):
    """Random stabilizer factors for timing-only or large parity cases."""
    g = rng(seed, "STAB")
    L1 = f32_to_bf16_bits(std1 * g.standard_normal((shape.K, shape.r_s), dtype=np.float32))
    L2 = f32_to_bf16_bits(std2 * g.standard_normal((shape.r_s, shape.N), dtype=np.float32))
    return L1, L2


def layer_inputs(shape, seed=0, residual_fn=None, with_dy=True):
    """All inputs of one layer as bf16 bit patterns.

    residual_fn(W_bits) -> fp64 residual E[N, K]; when given, the stabilizer is
    its rank-r_s SVD, otherwise random factors are drawn.  D = [L1 | A] is
    [K, R] and U = [L2 ; B] is [R, N] with the stabilizer in the first r_s
    columns / rows.
    """
    X = draw_x(shape, seed)
    W = draw_w(shape, seed)
    A, B = draw_lora(shape, seed)
    bias = draw_bias(shape, seed)
    if residual_fn is not None:
        L1, L2 = stabilizer_from_residual(residual_fn(W), shape.r_s)
    else:
        L1, L2 = stabilizer_random(shape, seed)
    D = np.ascontiguousarray(np.concatenate([L1, A], axis=1))
    U = np.ascontiguousarray(np.concatenate([L2, B], axis=0))
    out = dict(X=X, W=W, A=A, B=B, L1=L1, L2=L2, D=D, U=U, bias=bias)
    if with_dy:
        out["dY"] = draw_dy(shape, seed)
    return out


# ------------------------------------------------------------- device draws
def layer_inputs_torch(shape, seed, device):
    """Same distributions drawn on the device with a seeded torch generator
    (for large timing workloads, where host generation would dominate).
    Returns torch tensors: bf16 X, W, D, U, bias, dY."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1000003 + 17)

    def normal(shape_, std):
        return torch.randn(shape_, generator=g, device=device, dtype=torch.float32) * std

    X = normal((shape.M, shape.K), 1.0)
    if shape.n_outliers:
        cols = torch.randperm(shape.K, generator=g, device=device)[: shape.n_outliers]
        X[:, cols] *= shape.outlier_scale
    W = normal((shape.N, shape.K), 0.02)
    D = torch.cat([normal((shape.K, shape.r_s), 0.01), normal((shape.K, shape.r), 0.01)], dim=1)
    U = torch.cat([normal((shape.r_s, shape.N), 0.01), normal((shape.r, shape.N), 0.01)], dim=0)
    bias = normal((shape.N,), 0.02)
    if shape.dy_kind == "student_t3":
        z = torch.randn((shape.M, shape.N), generator=g, device=device)
        chi = sum(torch.randn((shape.M, shape.N), generator=g, device=device) ** 2 for _ in range(3))
        dY = shape.dy_scale * z / torch.sqrt(chi / 3.0)
    else:
        u = torch.rand((shape.M, shape.N), generator=g, device=device) - 0.5
        dY = -shape.dy_scale * torch.sign(u) * torch.log1p(-2.0 * u.abs())
    bf = torch.bfloat16
    return dict(X=X.to(bf), W=W.to(bf), D=D.to(bf).contiguous(), U=U.to(bf).contiguous(),
                bias=bias.to(bf), dY=dY.to(bf))
