"""The synthetic DiT training step (paper Sec. 4, "Efficiency Results": a
FLUX DiT training step with the 4-bit layers) at a small size, through the
library: the autograd wrappers against the fp64 oracle, the fused MLP pair
against the same calls made one by one, and training steps that lower the
loss and repeat bit for bit."""
import numpy as np
import pytest
import torch

from oracle import ref
from paper_2607_05711_amd import _lib, dit, gen
from tests._helpers import f64

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TINY = dit.DiTConfig(hidden=256, heads=2, mlp=1024, double_blocks=2, single_blocks=2, img_tokens=256,
                     txt_tokens=64, lora_rank=16, stab_rank=16)


def bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def test_triple_branch_autograd_against_oracle():
    g = torch.Generator(device=DEV)
    g.manual_seed(3)
    M, K, N, r, rs = 300, 256, 384, 16, 16
    layer = dit.FourTuneLinear(K, N, r, rs, g, DEV)
    with torch.no_grad():
        layer.B.copy_(torch.randn((r, N), generator=g, device=DEV) * 0.05)
        layer.wq.copy_(_lib.ft_quantize_blockwise((torch.randn((N, K), generator=g, device=DEV) * 0.02).to(
            torch.bfloat16), block_rows=32)[0])
    layer.sync()
    x = torch.randn((M, K), generator=g, device=DEV).to(torch.bfloat16).requires_grad_(True)
    dy = (torch.randn((M, N), generator=g, device=DEV) * 1e-2).to(torch.bfloat16)
    y = layer(x)
    y.backward(dy)
    torch.cuda.synchronize()
    X, DY, D, U, b = bits(x.detach()), bits(dy), bits(layer.D), bits(layer.U), bits(layer.bias)
    wq, ws = layer.wq.cpu().numpy(), layer.ws.cpu().numpy()
    xq, xs = ref.quantize(X, 1)
    P, Pa = ref.proj(X, D, 0)
    yr, S = ref.linear_fwd(xq, xs, wq, ws, K, P, U, b, Pabs=Pa)
    assert np.all(np.abs(f64(bits(y.detach())) - yr) <= 1e-5 * S + 2.0 ** -8 * np.abs(yr))
    gq, gs = ref.quantize(DY, 1)
    Qp, Qa = ref.proj(DY, U, 1)
    dxr, Sdx = ref.linear_bwd_input(gq, gs, wq, ws, K, Qp, D, Qpabs=Qa)
    assert np.all(np.abs(f64(bits(x.grad)) - dxr) <= 1e-5 * Sdx + 2.0 ** -8 * np.abs(dxr))
    dA, dB, _, _ = ref.lora_grads(X, DY, P[:, rs:], Qp[:, rs:], want_s=False)
    assert np.linalg.norm(layer.A.grad.cpu().numpy() - dA) <= 1e-3 * np.linalg.norm(dA)
    assert np.linalg.norm(layer.B.grad.cpu().numpy() - dB) <= 1e-3 * np.linalg.norm(dB)


def test_mlp_pair_autograd_equals_library_calls():
    g = torch.Generator(device=DEV)
    g.manual_seed(4)
    M, Dm, Fm = 200, 256, 1024
    mlp = dit.FourTuneMLP(Dm, Fm, 16, 16, g, DEV)
    with torch.no_grad():
        mlp.fc1.B.normal_(0, 0.05, generator=g)
        mlp.fc2.B.normal_(0, 0.05, generator=g)
    mlp.sync()
    x = torch.randn((M, Dm), generator=g, device=DEV).to(torch.bfloat16).requires_grad_(True)
    dy = (torch.randn((M, Dm), generator=g, device=DEV) * 1e-2).to(torch.bfloat16)
    y = mlp(x)
    y.backward(dy)
    f1, f2 = mlp.fc1, mlp.fc2
    xq, xs, P1 = _lib.ft_quantize_blockwise(x.detach(), proj=f1.D)
    z, h, hq, hs, P2 = _lib.ft_linear_fwd_gelu(xq, xs, f1.wq, f1.ws, Dm, P1, f1.U, f1.bias, D2=f2.D)
    y2 = _lib.ft_linear_fwd(hq, hs, f2.wq, f2.ws, Fm, P2, f2.U, f2.bias)
    gq, gs, Qp2 = _lib.ft_quantize_blockwise(dy, proj=f2.U, proj_layout=_lib.FT_PROJ_R_BY_COLS)
    dz, dzq, dzs, Qp1 = _lib.ft_linear_bwd_input_dgelu(gq, gs, f2.wq, f2.ws, Fm, z, Qp2, f2.D, U1=f1.U)
    dx = _lib.ft_linear_bwd_input(dzq, dzs, f1.wq, f1.ws, Dm, Qp1, f1.D)
    dA1, dB1 = _lib.ft_lora_grads(x.detach(), dz, P1, Qp1, 16, col0=16)
    torch.cuda.synchronize()
    assert torch.equal(y, y2) and torch.equal(x.grad, dx)
    assert torch.equal(f1.A.grad, dA1) and torch.equal(f1.B.grad, dB1)


def _train(kind, steps, seed=0):
    model = dit.DiT(TINY, kind, seed, DEV)
    trainer = dit.Trainer(model, lr=3e-3)
    batch = dit.synthetic_batch(TINY, seed + 1, DEV)
    losses = [float(trainer.step(*batch)) for _ in range(steps)]
    torch.cuda.synchronize()
    return model, losses


def test_dit_training_steps_lower_the_loss_and_repeat():
    model, losses = _train("fp4", 6)
    print("fp4 DiT losses", losses, flush=True)
    assert all(np.isfinite(losses))
    assert losses[-1] < losses[0]
    for p in model.lora_parameters():
        assert p.grad is not None and bool(torch.isfinite(p.grad).all())
    _, again = _train("fp4", 6)
    assert again == losses                     # fixed summation orders: bit-reproducible


def test_bf16_lora_dit_step_runs():
    _, losses = _train("bf16", 3)
    assert all(np.isfinite(losses)) and losses[-1] < losses[0]
