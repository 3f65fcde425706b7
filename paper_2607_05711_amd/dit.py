"""A synthetic FLUX.1-dev-shaped DiT training step built on the W4A4G4 layer.

The paper times whole DiT training steps (Sec. 4, "Efficiency Results": one
FLUX.1-dev DiT step with the 4-bit layers against BF16 LoRA).  This module
builds that step around the library: every linear of the double- and
single-stream blocks is a triple-branch layer (frozen MXFP4 weight, frozen
low-rank stabilizer, trainable LoRA) whose forward and backward run in the
library's kernels through the C ABI, wrapped as torch autograd functions; the
MLPs of the double blocks use the fused GELU / dGELU epilogues (Sec. 3.3,
MLP fusion).  The rest of a DiT block is not part of the paper's method and
runs as torch operations: LayerNorm with adaLN modulation, RMSNorm of q and
k, rotary position embeddings, joint attention (fused attention kernels
only), gated residuals.  AdamW updates the LoRA factors (fp32 masters; the
library reads their bf16 copies).

The same model with 16-bit LoRA linears (bf16 weights and adapters as torch
matmuls) is the paper's BF16 LoRA baseline.

Weights are random (timing does not depend on values); inputs are seeded
synthetic tensors with FLUX.1-dev's shapes at 1024x1024 (4096 image + 512
text tokens, hidden 3072, 24 heads of 128, MLP 12288, 19 double and 38 single
blocks).
"""
from dataclasses import dataclass

import torch
import torch.nn.functional as F

from . import _lib

BF = torch.bfloat16


@dataclass(frozen=True)
class DiTConfig:
    hidden: int = 3072
    heads: int = 24
    mlp: int = 12288
    double_blocks: int = 19
    single_blocks: int = 38
    img_tokens: int = 4096
    txt_tokens: int = 512
    lora_rank: int = 32
    stab_rank: int = 32

    @property
    def head_dim(self):
        return self.hidden // self.heads


FLUX_DEV = DiTConfig()


# ----------------------------------------------------------------- autograd
class _TripleBranchFn(torch.autograd.Function):
    """y = Q(x) Q(W)^T + x [L1|A] [L2;B] + bias (Eq. 2); backward Eq. (3) and
    the adapter gradients, all in the library."""

    @staticmethod
    def forward(ctx, x, A, B, layer):
        x = x.contiguous()
        xq, xs, P = _lib.ft_quantize_blockwise(x, proj=layer.D)
        y = _lib.ft_linear_fwd(xq, xs, layer.wq, layer.ws, layer.K, P, layer.U, layer.bias)
        ctx.save_for_backward(x, P)
        ctx.layer = layer
        return y

    @staticmethod
    def backward(ctx, dy):
        x, P = ctx.saved_tensors
        L = ctx.layer
        dy = dy.contiguous()
        gq, gs, Qp = _lib.ft_quantize_blockwise(dy, proj=L.U, proj_layout=_lib.FT_PROJ_R_BY_COLS)
        dx = _lib.ft_linear_bwd_input(gq, gs, L.wq, L.ws, L.K, Qp, L.D) if ctx.needs_input_grad[0] else None
        dA, dB = _lib.ft_lora_grads(x, dy, P, Qp, L.r, col0=L.rs)
        return dx, dA, dB, None


class _MlpPairFn(torch.autograd.Function):
    """FC1 -> GELU(tanh) -> FC2 with the fused epilogues (MLP fusion)."""

    @staticmethod
    def forward(ctx, x, A1, B1, A2, B2, fc1, fc2):
        x = x.contiguous()
        xq, xs, P1 = _lib.ft_quantize_blockwise(x, proj=fc1.D)
        z, h, hq, hs, P2 = _lib.ft_linear_fwd_gelu(xq, xs, fc1.wq, fc1.ws, fc1.K, P1, fc1.U, fc1.bias, D2=fc2.D)
        y = _lib.ft_linear_fwd(hq, hs, fc2.wq, fc2.ws, fc2.K, P2, fc2.U, fc2.bias)
        ctx.save_for_backward(x, P1, z, h, P2)
        ctx.fc = (fc1, fc2)
        return y

    @staticmethod
    def backward(ctx, dy):
        x, P1, z, h, P2 = ctx.saved_tensors
        fc1, fc2 = ctx.fc
        dy = dy.contiguous()
        gq, gs, Qp2 = _lib.ft_quantize_blockwise(dy, proj=fc2.U, proj_layout=_lib.FT_PROJ_R_BY_COLS)
        dz, dzq, dzs, Qp1 = _lib.ft_linear_bwd_input_dgelu(gq, gs, fc2.wq, fc2.ws, fc2.K, z, Qp2, fc2.D, U1=fc1.U)
        dx = _lib.ft_linear_bwd_input(dzq, dzs, fc1.wq, fc1.ws, fc1.K, Qp1, fc1.D)
        dA2, dB2 = _lib.ft_lora_grads(h, dy, P2, Qp2, fc2.r, col0=fc2.rs)
        dA1, dB1 = _lib.ft_lora_grads(x, dz, P1, Qp1, fc1.r, col0=fc1.rs)
        return dx, dA1, dB1, dA2, dB2, None, None


# ------------------------------------------------------------------- layers
class FourTuneLinear(torch.nn.Module):
    """A triple-branch linear K -> N: frozen MXFP4 weight (a random N(0,
    0.02^2) weight quantized by the library), frozen stabilizer L1 L2,
    trainable LoRA A B (fp32 masters, B
    initialised to zero), frozen bias.  D = [L1 | A] and U = [L2 ; B] are the
    bf16 buffers the library reads; sync() refreshes their adapter part."""

    def __init__(self, K, N, r, rs, gen, device, bias=True):
        super().__init__()
        self.K, self.N, self.r, self.rs = K, N, r, rs
        # frozen weight N(0, 0.02^2), quantized once in 32x32 tiles (offline in the method)
        W = (torch.randn((N, K), generator=gen, device=device) * 0.02).to(BF)
        self.wq, self.ws, _ = _lib.ft_quantize_blockwise(W, block_rows=32)
        del W
        L1 = torch.randn((K, rs), generator=gen, device=device) * 0.01
        L2 = torch.randn((rs, N), generator=gen, device=device) * 0.01
        self.A = torch.nn.Parameter(torch.randn((K, r), generator=gen, device=device) * (1.0 / K ** 0.5))
        self.B = torch.nn.Parameter(torch.zeros((r, N), device=device))
        self.D = torch.cat([L1, self.A.detach()], 1).to(BF).contiguous()
        self.U = torch.cat([L2, self.B.detach()], 0).to(BF).contiguous()
        self.bias = (torch.randn((N,), generator=gen, device=device) * 0.02).to(BF) if bias else None

    @torch.no_grad()
    def sync(self):
        self.D[:, self.rs:].copy_(self.A)
        self.U[self.rs:].copy_(self.B)

    def forward(self, x):
        shape = x.shape
        y = _TripleBranchFn.apply(x.reshape(-1, self.K), self.A, self.B, self)
        return y.reshape(*shape[:-1], self.N)


class FourTuneMLP(torch.nn.Module):
    """MLP pair D -> F -> D (GELU tanh) of two triple-branch linears, forward
    and backward through the fused epilogues."""

    def __init__(self, Dm, Fm, r, rs, gen, device):
        super().__init__()
        self.fc1 = FourTuneLinear(Dm, Fm, r, rs, gen, device)
        self.fc2 = FourTuneLinear(Fm, Dm, r, rs, gen, device)

    def sync(self):
        self.fc1.sync()
        self.fc2.sync()

    def forward(self, x):
        f1, f2 = self.fc1, self.fc2
        shape = x.shape
        y = _MlpPairFn.apply(x.reshape(-1, f1.K), f1.A, f1.B, f2.A, f2.B, f1, f2)
        return y.reshape(*shape[:-1], f2.N)


class Bf16LoraLinear(torch.nn.Module):
    """16-bit LoRA linear (the paper's BF16 LoRA baseline): frozen bf16
    weight, trainable bf16 A B, y = x W^T + b + (x A) B as torch matmuls."""

    def __init__(self, K, N, r, rs, gen, device, bias=True):
        super().__init__()
        self.K, self.N = K, N
        self.W = (torch.randn((N, K), generator=gen, device=device) * 0.02).to(BF)
        self.A = torch.nn.Parameter((torch.randn((K, r), generator=gen, device=device) * (1.0 / K ** 0.5)).to(BF))
        self.B = torch.nn.Parameter(torch.zeros((r, N), device=device, dtype=BF))
        self.bias = (torch.randn((N,), generator=gen, device=device) * 0.02).to(BF) if bias else None

    def sync(self):
        pass

    def forward(self, x):
        y = F.linear(x, self.W, self.bias)
        return y + (x @ self.A) @ self.B


class Bf16LoraMLP(torch.nn.Module):
    def __init__(self, Dm, Fm, r, rs, gen, device):
        super().__init__()
        self.fc1 = Bf16LoraLinear(Dm, Fm, r, rs, gen, device)
        self.fc2 = Bf16LoraLinear(Fm, Dm, r, rs, gen, device)

    def sync(self):
        pass

    def forward(self, x):
        return self.fc2(F.gelu(self.fc1(x), approximate="tanh"))


# -------------------------------------------------------------------- blocks
def _layer_norm(x):
    return F.layer_norm(x.float(), (x.shape[-1],), eps=1e-6)


def _modulate(x, shift, scale):
    return (_layer_norm(x) * (1.0 + scale.float()) + shift.float()).to(BF)


def _rms_norm(x, w):
    xf = x.float()
    return (xf * torch.rsqrt(xf.pow(2).mean(-1, keepdim=True) + 1e-6) * w.float()).to(BF)


def _rope(x, cos, sin):
    """Rotary embedding on consecutive pairs of the head dimension:
    x [tokens, heads, head_dim]; cos, sin [tokens, 1, head_dim / 2]."""
    xf = x.float().unflatten(-1, (-1, 2))
    x0, x1 = xf[..., 0], xf[..., 1]
    return torch.stack([x0 * cos - x1 * sin, x0 * sin + x1 * cos], -1).flatten(-2).to(BF)


def rope_tables(cfg, device):
    """FLUX's three-axis rotary table (axes of 16, 56 and 56 of the 128 head
    dimensions: a text index, then the image's row and column); text tokens
    sit at position 0 of every axis."""
    hd = cfg.head_dim
    axes = (hd // 8, (hd - hd // 8) // 2, hd - hd // 8 - (hd - hd // 8) // 2)
    side = int(round(cfg.img_tokens ** 0.5))
    ids = torch.zeros((cfg.txt_tokens + cfg.img_tokens, 3), device=device)
    r = torch.arange(cfg.img_tokens, device=device)
    ids[cfg.txt_tokens:, 1] = (r // side).float()
    ids[cfg.txt_tokens:, 2] = (r % side).float()
    angles = []
    for a, dim in enumerate(axes):
        freq = 1.0 / (10000.0 ** (torch.arange(0, dim, 2, device=device).float() / dim))
        angles.append(ids[:, a:a + 1] * freq[None, :])
    ang = torch.cat(angles, -1)[:, None, :]          # [L, 1, hd / 2]
    return torch.cos(ang), torch.sin(ang)


def _attention(q, k, v):
    """Joint attention over all tokens; q, k, v [L, heads, head_dim] bf16.
    Only fused attention kernels are allowed (no unfused matmul fallback)."""
    from torch.nn.attention import SDPBackend, sdpa_kernel
    q, k, v = (t.transpose(0, 1).unsqueeze(0) for t in (q, k, v))     # [1, heads, L, hd]
    with sdpa_kernel([SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]):
        o = F.scaled_dot_product_attention(q, k, v)
    return o.squeeze(0).transpose(0, 1).reshape(q.shape[2], -1)


class DoubleBlock(torch.nn.Module):
    """Image and text streams with their own weights, joint attention."""

    def __init__(self, cfg, make_linear, make_mlp, gen, device):
        super().__init__()
        H, r, rs = cfg.hidden, cfg.lora_rank, cfg.stab_rank
        self.cfg = cfg
        self.mod = {s: (torch.randn((H, 6 * H), generator=gen, device=device) * 0.01).to(BF) for s in ("img", "txt")}
        self.qkv = torch.nn.ModuleDict({s: make_linear(H, 3 * H, r, rs, gen, device) for s in ("img", "txt")})
        self.out = torch.nn.ModuleDict({s: make_linear(H, H, r, rs, gen, device) for s in ("img", "txt")})
        self.mlp = torch.nn.ModuleDict({s: make_mlp(H, cfg.mlp, r, rs, gen, device) for s in ("img", "txt")})
        self.qn = {s: torch.ones(cfg.head_dim, device=device, dtype=BF) for s in ("img", "txt")}
        self.kn = {s: torch.ones(cfg.head_dim, device=device, dtype=BF) for s in ("img", "txt")}

    def forward(self, img, txt, vec, rope):
        cfg = self.cfg
        x = {"img": img, "txt": txt}
        mods, qkv = {}, {}
        for s in ("img", "txt"):
            mods[s] = (F.silu(vec) @ self.mod[s]).chunk(6, -1)
            sh1, sc1 = mods[s][0], mods[s][1]
            q, k, v = self.qkv[s](_modulate(x[s], sh1, sc1)).view(-1, 3, cfg.heads, cfg.head_dim).unbind(1)
            qkv[s] = (_rms_norm(q, self.qn[s]), _rms_norm(k, self.kn[s]), v)
        cos, sin = rope
        q = _rope(torch.cat([qkv["txt"][0], qkv["img"][0]], 0), cos, sin)
        k = _rope(torch.cat([qkv["txt"][1], qkv["img"][1]], 0), cos, sin)
        v = torch.cat([qkv["txt"][2], qkv["img"][2]], 0)
        o = _attention(q, k, v)
        att = {"txt": o[:cfg.txt_tokens], "img": o[cfg.txt_tokens:]}
        for s in ("img", "txt"):
            _, _, g1, sh2, sc2, g2 = mods[s]
            x[s] = x[s] + g1 * self.out[s](att[s])
            x[s] = x[s] + g2 * self.mlp[s](_modulate(x[s], sh2, sc2))
        return x["img"], x["txt"]


class SingleBlock(torch.nn.Module):
    """Fused QKV + MLP-in linear, attention and GELU, one output linear."""

    def __init__(self, cfg, make_linear, gen, device):
        super().__init__()
        H, r, rs = cfg.hidden, cfg.lora_rank, cfg.stab_rank
        self.cfg = cfg
        self.mod = (torch.randn((H, 3 * H), generator=gen, device=device) * 0.01).to(BF)
        self.linear1 = make_linear(H, 3 * H + cfg.mlp, r, rs, gen, device)
        self.linear2 = make_linear(H + cfg.mlp, H, r, rs, gen, device)
        self.qn = torch.ones(cfg.head_dim, device=device, dtype=BF)
        self.kn = torch.ones(cfg.head_dim, device=device, dtype=BF)

    def forward(self, x, vec, rope):
        cfg = self.cfg
        sh, sc, g = (F.silu(vec) @ self.mod).chunk(3, -1)
        h = self.linear1(_modulate(x, sh, sc))
        qkv, mlp = h.split([3 * cfg.hidden, cfg.mlp], -1)
        q, k, v = qkv.reshape(-1, 3, cfg.heads, cfg.head_dim).unbind(1)
        cos, sin = rope
        o = _attention(_rope(_rms_norm(q, self.qn), cos, sin), _rope(_rms_norm(k, self.kn), cos, sin), v)
        return x + g * self.linear2(torch.cat([o, F.gelu(mlp, approximate="tanh")], -1))


class DiT(torch.nn.Module):
    """The double- and single-stream blocks of a FLUX-shaped DiT (the
    embedders and the final projection are small and left out)."""

    def __init__(self, cfg, kind, seed, device):
        super().__init__()
        gen = torch.Generator(device=device)
        gen.manual_seed(seed)
        if kind == "fp4":
            make_linear, make_mlp = FourTuneLinear, FourTuneMLP
        elif kind == "bf16":
            make_linear, make_mlp = Bf16LoraLinear, Bf16LoraMLP
        else:
            raise ValueError(kind)
        self.cfg = cfg
        self.double_stream = torch.nn.ModuleList(
            [DoubleBlock(cfg, make_linear, make_mlp, gen, device) for _ in range(cfg.double_blocks)])
        self.single_stream = torch.nn.ModuleList([SingleBlock(cfg, make_linear, gen, device) for _ in range(cfg.single_blocks)])
        self.rope = rope_tables(cfg, device)

    def lora_parameters(self):
        return [p for n, p in self.named_parameters() if n.endswith(".A") or n.endswith(".B")]

    def sync(self):
        for m in self.modules():
            if m is not self and hasattr(m, "sync") and isinstance(m, (FourTuneLinear, Bf16LoraLinear)):
                m.sync()

    def forward(self, img, txt, vec):
        for blk in self.double_stream:
            img, txt = blk(img, txt, vec, self.rope)
        x = torch.cat([txt, img], 0)
        for blk in self.single_stream:
            x = blk(x, vec, self.rope)
        return x[self.cfg.txt_tokens:]


def synthetic_batch(cfg, seed, device):
    """Image and text token states, the conditioning vector and a target."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    img = torch.randn((cfg.img_tokens, cfg.hidden), generator=g, device=device).to(BF)
    txt = torch.randn((cfg.txt_tokens, cfg.hidden), generator=g, device=device).to(BF)
    vec = torch.randn((1, cfg.hidden), generator=g, device=device).to(BF)
    target = torch.randn((cfg.img_tokens, cfg.hidden), generator=g, device=device).to(BF)
    return img, txt, vec, target


class Trainer:
    """One training step: forward, mean-squared loss against the target,
    backward, AdamW on the LoRA factors, refresh of the bf16 copies."""

    def __init__(self, model, lr=1e-4):
        self.model = model
        self.params = model.lora_parameters()
        self.opt = torch.optim.AdamW(self.params, lr=lr, weight_decay=0.0)

    def step(self, img, txt, vec, target):
        self.opt.zero_grad(set_to_none=True)
        out = self.model(img, txt, vec)
        loss = (out.float() - target.float()).pow(2).mean()
        loss.backward()
        self.opt.step()
        self.model.sync()
        return loss.detach()
