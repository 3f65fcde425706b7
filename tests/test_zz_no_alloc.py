"""The allocation-free adapter-gradient entry point (ft_lora_grads_noalloc)
against ft_lora_grads, through the C ABI: both run the same kernels with the
same partial-sum order, so the results must be bit-identical.  Two calls in a
row, the second with a smaller input (the static scratch keeps the first
call's contents), plus accumulation and a size that needs no partials."""
import numpy as np
import pytest
import torch

from paper_2607_05711_amd import _lib, gen

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def case(M, K, N, r, rs, seed):
    rng = np.random.default_rng(seed)
    bf = lambda a: torch.from_numpy(gen.f32_to_bf16_bits(a.astype(np.float32)).view(np.int16)).view(
        torch.bfloat16).to(DEV)
    X = bf(rng.standard_normal((M, K)))
    dY = bf(1e-3 * rng.standard_t(3, (M, N)))
    P = torch.from_numpy(rng.standard_normal((M, r + rs)).astype(np.float32)).to(DEV)
    Qp = torch.from_numpy((1e-3 * rng.standard_normal((M, r + rs))).astype(np.float32)).to(DEV)
    return X, dY, P, Qp


def same_bits(a, b):
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


@pytest.mark.parametrize("big,small", [((4608, 3072, 9216, 32, 32), (1000, 1024, 2048, 32, 32)),
                                       ((18432, 3072, 21504, 64, 32), (700, 416, 1312, 40, 24))])
def test_noalloc_matches_workspace_entry_point(big, small):
    for shape, seed in ((big, 1), (small, 2)):
        M, K, N, r, rs = shape
        assert _lib.ft_lora_grads_workspace_size(M, K, N, r + rs, r) > 0      # partials go through the scratch
        X, dY, P, Qp = case(M, K, N, r, rs, seed)
        dA_ref, dB_ref = _lib.ft_lora_grads(X, dY, P, Qp, r, col0=rs)
        dA = torch.full((K, r), float("nan"), device=DEV)
        dB = torch.full((r, N), float("nan"), device=DEV)
        _lib.ft_lora_grads_noalloc(X, dY, P, Qp, r, col0=rs, dA=dA, dB=dB)
        torch.cuda.synchronize()
        print("no-alloc lora grads", shape, flush=True)
        assert same_bits(dA, dA_ref) and same_bits(dB, dB_ref), shape
        # accumulate: adds exactly the same sums
        _lib.ft_lora_grads_noalloc(X, dY, P, Qp, r, col0=rs, dA=dA, dB=dB, accumulate=True)
        torch.cuda.synchronize()
        assert torch.equal(dA, 2 * dA_ref) and torch.equal(dB, 2 * dB_ref), shape


def test_noalloc_without_partials_and_empty():
    # one 64-row stage: no token chunks, nothing goes through the scratch
    X, dY, P, Qp = case(64, 256, 320, 16, 16, 3)
    assert _lib.ft_lora_grads_workspace_size(64, 256, 320, 32, 16) == 0
    dA_ref, dB_ref = _lib.ft_lora_grads(X, dY, P, Qp, 16, col0=16)
    dA, dB = _lib.ft_lora_grads_noalloc(X, dY, P, Qp, 16, col0=16)
    torch.cuda.synchronize()
    assert same_bits(dA, dA_ref) and same_bits(dB, dB_ref)
    # no tokens: zeros
    X0, dY0 = X[:0], dY[:0]
    dA0, dB0 = _lib.ft_lora_grads_noalloc(X0, dY0, P[:0], Qp[:0], 16, col0=16)
    torch.cuda.synchronize()
    assert bool((dA0 == 0).all()) and bool((dB0 == 0).all())
