"""Benchmark: W4A4G4 triple-branch linear layers, forward + backward, on one GPU.

The default workload (flux_qkv) is one step of the hot path over one batch of
synthetic FLUX.1-dev-shaped input (attention QKV projection at 1024x1024:
M = 4096 image + 512 text tokens, K = 3072, N = 9216, LoRA rank 32,
stabilizer rank 32):

  quantize X (1x32 MXFP4) + P = X [L1|A]          ft_quantize_blockwise
  Y  = Q(X) Q(W)^T + P [L2;B] + bias   (bf16)      ft_linear_fwd
  quantize dY + Qp = dY [L2;B]^T                    ft_quantize_blockwise
  dX = Q(dY) Q(W) + Qp [L1|A]^T        (bf16)      ft_linear_bwd_input
  dA = X^T (dY B^T), dB = (X A)^T dY   (fp32)      ft_lora_grads

Other workloads: flux_mlp (the MLP pair 3072 -> 12288 -> 3072 with the fused
GELU / dGELU epilogues), flux_single (the single-stream block linears at batch
4) and flux_stack (every linear of the FLUX.1-dev stack, one training step).

The frozen weights are quantized once before timing (offline in the method).
Inputs are drawn on the device with a seeded generator and are resident in HBM
when the timed region starts.  Prints one JSON line.
"""
import argparse
import hashlib
import json
import os
import signal
import subprocess
import sys
import tempfile
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

MXFP4_PEAK_TFLOPS = 10100.0      # MI355X dense MXFP4 MFMA (256 CU x 2.4 GHz x 16384 flop/clk)
HBM_PEAK_GBS = 8000.0


def layer_flops(M, K, N, r, R):
    fp4 = 2 * (2.0 * M * N * K)                      # fwd + bwd-input 4-bit GEMMs
    lowrank = 2.0 * M * R * (K + N) * 2               # down + up projections, fwd and bwd
    lora = 2.0 * r * M * (N + K)                      # dA and dB
    return fp4, lowrank, lora


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed steps before the timed ones (default: 200 for flux_qkv, 100 for flux_mlp, 20 for "
                         "flux_single and the --ablation / --numerics modes, 3 for flux_stack and --dit; the clock "
                         "takes some 30 ms of back-to-back steps to settle)")
    ap.add_argument("--workload", default="flux_qkv", choices=["flux_qkv", "flux_mlp", "flux_single", "flux_stack"])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-workloads", action="store_true",
                    help="flux_qkv: skip the flux_mlp / flux_single / flux_stack measurements under other_workloads")
    ap.add_argument("--cpu-rows", type=int, default=0, help="token rows in the oracle sample (0: auto)")
    ap.add_argument("--ablation", action="store_true",
                    help="flux_qkv / flux_mlp: time the fused step against an unfused one, print one JSON line, exit")
    ap.add_argument("--numerics", action="store_true",
                    help="time the quantizer's numerics variants at the QKV shapes, print one JSON line, exit")
    ap.add_argument("--dit", action="store_true",
                    help="time one synthetic FLUX DiT training step, W4A4G4 against BF16 LoRA; print one JSON line")
    ap.add_argument("--stability", action="store_true",
                    help="run the synthetic gradient-norm stability probe, print one JSON line, exit")
    ap.add_argument("--no-clock-sample", action="store_true",
                    help="skip the rocm-smi clock sample (2 s of back-to-back forward GEMMs) of the default line")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB three times (scales HBM counters), then exit")
    return ap.parse_args()


# Sources whose compiled code the GEMM traffic record was measured on; the record
# is reported only while they hash the same.
GEMM_SOURCES = ("paper_2607_05711_amd/csrc/gemm_fp4.hip", "paper_2607_05711_amd/csrc/ft_device.h",
                "paper_2607_05711_amd/csrc/ft_kernels.h")
TRAFFIC_RECORD = "profiles/gemm_fp4_flux_qkv_traffic.md"


def sources_sha256(paths=GEMM_SOURCES):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(direction):
    """HBM bytes per launch of the forward or backward-input GEMM from the
    committed counter record (FETCH_SIZE + WRITE_SIZE, each scaled by the
    factor a plain copy of known size gives), or None when the record is
    missing or was taken on other kernel sources."""
    path = os.path.join(ROOT, TRAFFIC_RECORD)
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as f:
        for line in f:
            m = line.strip().strip("`").split(":", 1)
            if len(m) == 2 and m[0].strip().startswith(("source_sha256", "traffic_bytes_")):
                rec[m[0].strip()] = m[1].strip()
    if rec.get("source_sha256") != sources_sha256():
        return None
    v = rec.get("traffic_bytes_" + direction)
    return float(v) if v else None


def copy_calibration(mib):
    import torch
    n = mib << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 3}), flush=True)


# ----------------------------------------------------------------- workloads
# A workload is a list of layers: ("linear", M, K, N, r, r_s) runs the five
# steps of one triple-branch linear; ("mlp", M, D, F, r, r_s) runs the MLP pair
# D -> F -> D with the fused GELU / dGELU epilogues.  One step is every
# layer's forward in order, then every layer's backward in reverse order.
def workload_layers(name):
    if name == "flux_qkv":
        return [("linear", 4608, 3072, 9216, 32, 32)]
    if name == "flux_mlp":
        return [("mlp", 4608, 3072, 12288, 32, 32)]
    if name == "flux_single":
        return [("linear", 18432, 3072, 21504, 64, 32), ("linear", 18432, 15360, 3072, 64, 32)]
    if name == "flux_stack":
        layers = []
        for _ in range(19):              # double-stream blocks: image (4096 tokens) and text (512) streams
            for m in (4096, 512):
                layers += [("linear", m, 3072, 9216, 32, 32), ("linear", m, 3072, 3072, 32, 32),
                           ("mlp", m, 3072, 12288, 32, 32)]
        for _ in range(38):              # single-stream blocks over all 4608 tokens
            layers += [("linear", 4608, 3072, 21504, 32, 32), ("linear", 4608, 15360, 3072, 32, 32)]
        return layers
    raise SystemExit("unknown workload %r" % name)


def workload_lanes(name, layers):
    """(group, lane) of every layer.  Within a group, lane-1 layers run on a
    second HIP stream beside the lane-0 layers: the image (lane 0) and text
    (lane 1) streams of a double block have separate weights and inputs, so
    their linears are independent, and the short text stream's kernels fill
    CUs the image stream's last round of tiles leaves idle.  Groups run in
    order (forward) and in reverse order (backward)."""
    if name != "flux_stack":
        return [(i, 0) for i in range(len(layers))]
    out = []
    for b in range(19):
        out += [(b, 0)] * 3 + [(b, 1)] * 3
    out += [(19 + i, 0) for i in range(len(layers) - len(out))]
    return out


WORKLOAD_TEXT = {
    "flux_qkv": "FLUX.1-dev attention QKV linear, batch 1 at 1024^2 (M=4608 tokens, 3072 -> 9216)",
    "flux_mlp": "FLUX.1-dev MLP pair, batch 1 at 1024^2 (M=4608, 3072 -> 12288 -> 3072, GELU-tanh)",
    "flux_single": "FLUX.1-dev single-stream block linears, batch 4 (M=18432: 3072 -> 21504, 15360 -> 3072)",
    "flux_stack": "FLUX.1-dev linear stack, one training step (19 double blocks x {image 4096, text 512} tokens x "
                  "{QKV, out, MLP pair} + 38 single blocks x {3072 -> 21504, 15360 -> 3072} at 4608 tokens)",
}


def linear_counts(M, K, N, r, R):
    """(FP4 flops, low-rank flops, adapter-gradient flops, quantize bytes, adapter-gradient bytes)."""
    fp4, lowrank, lora = layer_flops(M, K, N, r, R)
    qbytes = M * K * (2 + 0.5 + 1 / 32) + M * R * 4 + K * R * 2 + M * N * (2 + 0.5 + 1 / 32) + M * R * 4 + N * R * 2
    lbytes = 2.0 * M * (K + N) + 2 * M * r * 4 + 4.0 * r * (K + N)
    return fp4, lowrank, lora, qbytes, lbytes


class Builder:
    """Device buffers and launch closures.  Inputs are seeded synthetic draws
    (activations N(0,1) with 0.5% outlier channels x30, gradients 1e-3 *
    Student-t(3), adapter and stabilizer factors N(0, 0.01^2), bias N(0,
    0.02^2)); weights are N(0, 0.02^2) quantized once before timing, or random
    FP4 codes and E8M0 scales for the stack (timing does not depend on values).
    Activation buffers are shared between layers of the same shape."""

    def __init__(self, torch, lib, dev, seed, random_weights):
        self.t, self.L, self.dev = torch, lib, dev
        self.g = torch.Generator(device=dev)
        self.g.manual_seed(seed)
        self.random_weights = random_weights
        self.shared = {}
        self.lane = 0   # buffers written by layers on different streams are never shared

    def normal(self, shape, std):
        return (self.t.randn(shape, generator=self.g, device=self.dev) * std).to(self.t.bfloat16)

    def activations(self, M, K):
        key = ("x", M, K)
        if key not in self.shared:
            x = self.t.randn((M, K), generator=self.g, device=self.dev)
            cols = self.t.randperm(K, generator=self.g, device=self.dev)[:max(1, round(0.005 * K))]
            x[:, cols] *= 30.0
            self.shared[key] = x.to(self.t.bfloat16)
        return self.shared[key]

    def gradient(self, M, N):
        key = ("dy", M, N)
        if key not in self.shared:
            z = self.t.randn((M, N), generator=self.g, device=self.dev)
            chi = sum(self.t.randn((M, N), generator=self.g, device=self.dev) ** 2 for _ in range(3))
            self.shared[key] = (1e-3 * z / self.t.sqrt(chi / 3.0)).to(self.t.bfloat16)
        return self.shared[key]

    def buf(self, tag, shape, dtype):
        key = (self.lane, tag, tuple(shape), dtype)
        if key not in self.shared:
            self.shared[key] = self.t.empty(shape, dtype=dtype, device=self.dev)
        return self.shared[key]

    def weight(self, N, K):
        t = self.t
        if self.random_weights:
            wq = t.randint(0, 256, (N, K // 2), generator=self.g, device=self.dev, dtype=t.uint8)
            ws = t.randint(118, 124, (N // 32, K // 32), generator=self.g, device=self.dev, dtype=t.uint8)
            return wq, ws
        wq, ws, _ = self.L.ft_quantize_blockwise(self.normal((N, K), 0.02), block_rows=32)
        return wq, ws

    def wspace(self, nbytes):
        return self.buf("ws%d" % nbytes, (max(nbytes, 16),), self.t.uint8)

    def linear(self, M, K, N, r, rs, given=None):
        """Closures for one linear: forward [(kind, fn)], backward [(kind, fn)],
        counts.  `given` may supply X, dY, wq, ws, D, U, bias."""
        t, L = self.t, self.L
        u8, f32, bf = t.uint8, t.float32, t.bfloat16
        R = r + rs
        if given:
            X, dY, wq, ws = given["X"], given["dY"], given["wq"], given["ws"]
            D, U, bias = given["D"], given["U"], given["bias"]
        else:
            X, dY = self.activations(M, K), self.gradient(M, N)
            wq, ws = self.weight(N, K)
            D, U, bias = self.normal((K, R), 0.01), self.normal((R, N), 0.01), self.normal((N,), 0.02)
        xq, xs = self.buf("xq", (M, K // 2), u8), self.buf("xs", (M, K // 32), u8)
        P, Qp = self.buf("P", (M, R), f32), self.buf("Qp", (M, R), f32)
        Y, dX = self.buf("y", (M, N), bf), self.buf("dx", (M, K), bf)
        gq, gs = self.buf("gq", (M, N // 2), u8), self.buf("gs", (M, N // 32), u8)
        dA, dB = self.buf("dA", (K, r), f32), self.buf("dB", (r, N), f32)
        wx = self.wspace(L.ft_quantize_workspace_size(M, K, 1, R, L.FT_PROJ_COLS_BY_R))
        wd = self.wspace(L.ft_quantize_workspace_size(M, N, 1, R, L.FT_PROJ_R_BY_COLS))
        wl = self.wspace(L.ft_lora_grads_workspace_size(M, K, N, R, r))
        fwd = [("quantize_x", lambda: L.ft_quantize_blockwise(X, proj=D, codes=xq, scales=xs, proj_out=P, workspace=wx)),
               ("gemm_fwd", lambda: L.ft_linear_fwd(xq, xs, wq, ws, K, P, U, bias, y=Y))]
        bwd = [("quantize_dy", lambda: L.ft_quantize_blockwise(dY, proj=U, proj_layout=L.FT_PROJ_R_BY_COLS, codes=gq,
                                                              scales=gs, proj_out=Qp, workspace=wd)),
               ("gemm_bwd", lambda: L.ft_linear_bwd_input(gq, gs, wq, ws, K, Qp, D, dx=dX)),
               ("lora_grads", lambda: L.ft_lora_grads(X, dY, P, Qp, r, col0=rs, dA=dA, dB=dB, workspace=wl))]
        fp4, lowrank, lora, qb, lb = linear_counts(M, K, N, r, R)
        counts = {"flops": fp4 + lowrank + lora, "gemm_fwd": fp4 / 2, "gemm_bwd": fp4 / 2,
                  "quantize_x": M * K * (2 + 0.5 + 1 / 32) + M * R * 4 + K * R * 2,
                  "quantize_dy": M * N * (2 + 0.5 + 1 / 32) + M * R * 4 + N * R * 2, "lora_grads": lb}
        return fwd, bwd, counts

    def mlp(self, M, Dm, F, r, rs):
        """MLP pair Dm -> F -> Dm: FC1 forward fused with GELU and FC2's input
        preparation, FC2 backward-input fused with dGELU and FC1's gradient
        preparation."""
        t, L = self.t, self.L
        u8, f32, bf = t.uint8, t.float32, t.bfloat16
        R = r + rs
        X, dY = self.activations(M, Dm), self.gradient(M, Dm)
        w1q, w1s = self.weight(F, Dm)
        w2q, w2s = self.weight(Dm, F)
        D1, U1, b1 = self.normal((Dm, R), 0.01), self.normal((R, F), 0.01), self.normal((F,), 0.02)
        D2, U2, b2 = self.normal((F, R), 0.01), self.normal((R, Dm), 0.01), self.normal((Dm,), 0.02)
        xq, xs = self.buf("xq", (M, Dm // 2), u8), self.buf("xs", (M, Dm // 32), u8)
        P1, P2 = self.buf("P1", (M, R), f32), self.buf("P2", (M, R), f32)
        Qp1, Qp2 = self.buf("Qp1", (M, R), f32), self.buf("Qp2", (M, R), f32)
        z, h = self.buf("z", (M, F), bf), self.buf("h", (M, F), bf)
        hq, hs = self.buf("hq", (M, F // 2), u8), self.buf("hs", (M, F // 32), u8)
        Y = self.buf("y", (M, Dm), bf)
        gq, gs = self.buf("gq", (M, Dm // 2), u8), self.buf("gs", (M, Dm // 32), u8)
        dz = self.buf("dz", (M, F), bf)
        dzq, dzs = self.buf("dzq", (M, F // 2), u8), self.buf("dzs", (M, F // 32), u8)
        dX = self.buf("dx", (M, Dm), bf)
        dA1, dB1 = self.buf("dA1", (Dm, r), f32), self.buf("dB1", (r, F), f32)
        dA2, dB2 = self.buf("dA2", (F, r), f32), self.buf("dB2", (r, Dm), f32)
        wx = self.wspace(L.ft_quantize_workspace_size(M, Dm, 1, R, L.FT_PROJ_COLS_BY_R))
        wd = self.wspace(L.ft_quantize_workspace_size(M, Dm, 1, R, L.FT_PROJ_R_BY_COLS))
        wg = self.wspace(L.ft_linear_fwd_gelu_workspace_size(M, F, R))
        wdg = self.wspace(L.ft_linear_bwd_input_dgelu_workspace_size(M, F, R))
        wl1 = self.wspace(L.ft_lora_grads_workspace_size(M, Dm, F, R, r))
        wl2 = self.wspace(L.ft_lora_grads_workspace_size(M, F, Dm, R, r))
        fwd = [("quantize_x", lambda: L.ft_quantize_blockwise(X, proj=D1, codes=xq, scales=xs, proj_out=P1, workspace=wx)),
               ("gemm_fwd_gelu", lambda: L.ft_linear_fwd_gelu(xq, xs, w1q, w1s, Dm, P1, U1, b1, D2=D2, z=z, h=h,
                                                               hq=hq, hs=hs, P2=P2, workspace=wg)),
               ("gemm_fwd", lambda: L.ft_linear_fwd(hq, hs, w2q, w2s, F, P2, U2, b2, y=Y))]
        bwd = [("quantize_dy", lambda: L.ft_quantize_blockwise(dY, proj=U2, proj_layout=L.FT_PROJ_R_BY_COLS, codes=gq,
                                                              scales=gs, proj_out=Qp2, workspace=wd)),
               ("gemm_bwd_dgelu", lambda: L.ft_linear_bwd_input_dgelu(gq, gs, w2q, w2s, F, z, Qp2, D2, U1=U1, dz=dz,
                                                                       dzq=dzq, dzs=dzs, Qp1=Qp1, workspace=wdg)),
               ("gemm_bwd", lambda: L.ft_linear_bwd_input(dzq, dzs, w1q, w1s, Dm, Qp1, D1, dx=dX)),
               ("lora_grads", lambda: L.ft_lora_grads(h, dY, P2, Qp2, r, col0=rs, dA=dA2, dB=dB2, workspace=wl2)),
               ("lora_grads", lambda: L.ft_lora_grads(X, dz, P1, Qp1, r, col0=rs, dA=dA1, dB=dB1, workspace=wl1))]
        c1, c2 = linear_counts(M, Dm, F, r, R), linear_counts(M, F, Dm, r, R)
        counts = {"flops": sum(c1[:3]) + sum(c2[:3]),
                  "gemm_fwd_gelu": c1[0] / 2, "gemm_fwd": c2[0] / 2, "gemm_bwd_dgelu": c2[0] / 2, "gemm_bwd": c1[0] / 2,
                  "quantize_x": M * Dm * (2 + 0.5 + 1 / 32) + M * R * 4 + Dm * R * 2,
                  "quantize_dy": M * Dm * (2 + 0.5 + 1 / 32) + M * R * 4 + Dm * R * 2, "lora_grads": c1[4] + c2[4]}
        return fwd, bwd, counts


def fusion_ablation(torch, L, d, wq, ws, shape, steps, warmup):
    """The layer step with and without the low-rank fusion (the paper's LoRA
    fusion, Sec. 3.3), same inputs.  Unfused: quantization without the
    projection, the FP4 GEMMs without the low-rank branch, and the low-rank
    down- and up-projections and adapter gradients as separate bf16 library
    matmuls (each re-reading its [M, K] or [M, N] operand).  A timing
    comparison only: the unfused step keeps its low-rank intermediates in
    bf16."""
    M, K, N, r, rs = shape.M, shape.K, shape.N, shape.r, shape.r_s
    R = r + rs
    dev = d["X"].device
    X, dY, D, U, bias = d["X"], d["dY"], d["D"], d["U"], d["bias"]
    u8, f32, bf = torch.uint8, torch.float32, torch.bfloat16
    e = lambda sh, t: torch.empty(sh, dtype=t, device=dev)
    xq, xs, gq, gs = e((M, K // 2), u8), e((M, K // 32), u8), e((M, N // 2), u8), e((M, N // 32), u8)
    P, Qp = e((M, R), f32), e((M, R), f32)
    Y, dX = e((M, N), bf), e((M, K), bf)
    dA, dB = e((K, r), f32), e((r, N), f32)
    wx = e((max(16, L.ft_quantize_workspace_size(M, K, 1, R, L.FT_PROJ_COLS_BY_R)),), u8)
    wd = e((max(16, L.ft_quantize_workspace_size(M, N, 1, R, L.FT_PROJ_R_BY_COLS)),), u8)
    wl = e((max(16, L.ft_lora_grads_workspace_size(M, K, N, R, r)),), u8)
    Ut, Dt = U.t().contiguous(), D.t().contiguous()       # [N, R], [R, K]: contiguous matmul operands
    dBb, dAtb = e((r, N), bf), e((r, K), bf)

    def fused():
        L.ft_quantize_blockwise(X, proj=D, codes=xq, scales=xs, proj_out=P, workspace=wx)
        L.ft_linear_fwd(xq, xs, wq, ws, K, P, U, bias, y=Y)
        L.ft_quantize_blockwise(dY, proj=U, proj_layout=L.FT_PROJ_R_BY_COLS, codes=gq, scales=gs, proj_out=Qp,
                                workspace=wd)
        L.ft_linear_bwd_input(gq, gs, wq, ws, K, Qp, D, dx=dX)
        L.ft_lora_grads(X, dY, P, Qp, r, col0=rs, dA=dA, dB=dB, workspace=wl)

    def unfused():
        L.ft_quantize_blockwise(X, codes=xq, scales=xs)
        Pb = torch.mm(X, D)                                   # [M, R] bf16, re-reads X
        L.ft_linear_fwd(xq, xs, wq, ws, K, None, None, bias, y=Y)
        Y.add_(torch.mm(Pb, U))                               # up-projection, then a pass over Y
        L.ft_quantize_blockwise(dY, codes=gq, scales=gs)
        Qb = torch.mm(dY, Ut)                                 # [M, R], re-reads dY
        L.ft_linear_bwd_input(gq, gs, wq, ws, K, dx=dX)
        dX.add_(torch.mm(Qb, Dt))
        torch.mm(Pb[:, rs:].t().contiguous(), dY, out=dBb)   # dB = (XA)^T dY
        torch.mm(Qb[:, rs:].t().contiguous(), X, out=dAtb)   # dA^T = (dY B^T)^T X

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / steps

    bf16_step = bf16_lora_linear(torch, d["W"], d["D"][:, rs:].contiguous(), d["U"][rs:].contiguous(), bias, X, dY)
    tf, tu = timed(fused), timed(unfused)
    tb = timed(bf16_step)
    tf2 = timed(fused)
    tf = min(tf, tf2)
    return {"metric": "layer step time, low-rank fusion ablation and BF16 LoRA (flux_qkv)", "unit": "ms",
            "fused_ms": round(tf, 4), "unfused_ms": round(tu, 4), "fusion_speedup": round(tu / tf, 3),
            "unfused": "quantize without projection; FP4 GEMMs without the low-rank branch; down-, up-projections "
                       "and adapter gradients as separate bf16 library matmuls",
            "bf16_lora_ms": round(tb, 4), "speedup_vs_bf16_lora": round(tb / tf, 3),
            "bf16_lora": BF16_LORA_TEXT,
            "steps": steps, "warmup": warmup, "data": "synthetic"}


BF16_LORA_TEXT = ("16-bit LoRA (W16A16G16): bf16 weight, activations and gradients; the weight and adapter "
                  "products as bf16 library matmuls (hipBLASLt through torch) with fp32 accumulation, no stabilizer; "
                  "forward, input gradient and adapter gradients")


def bf16_lora_linear(torch, W, A, B, bias, X, dY):
    """One step of the 16-bit LoRA linear the paper compares against (BF16
    LoRA): Y = X W^T + bias + (X A) B, then dX = dY W + (dY B^T) A^T,
    dA = X^T (dY B^T), dB = (X A)^T dY, all bf16 matmuls with fp32
    accumulation.  The frozen weight is kept in both layouts so that no
    product takes a transposed right operand."""
    Wt = W.t().contiguous()                    # [K, N]

    def step():
        XA = torch.mm(X, A)                    # [M, r]
        torch.addmm(bias, X, Wt).addmm_(XA, B)
        G_Bt = torch.mm(dY, B.t().contiguous())    # [M, r]
        torch.mm(dY, W).addmm_(G_Bt, A.t().contiguous())
        torch.mm(X.t(), G_Bt)                  # dA [K, r]
        torch.mm(XA.t(), dY)                   # dB [r, N]
    return step


def bf16_lora_mlp(torch, W1, A1, B1, b1, W2, A2, B2, b2, X, dY):
    """The MLP pair as 16-bit LoRA: z = X W1^T + b1 + (X A1) B1, h = GELU(z),
    y = h W2^T + b2 + (h A2) B2, and the backward through both linears and
    the GELU, with the four adapter gradients."""
    W1t, W2t = W1.t().contiguous(), W2.t().contiguous()
    F = torch.nn.functional

    def step():
        XA1 = torch.mm(X, A1)
        z = torch.addmm(b1, X, W1t).addmm_(XA1, B1)
        h = F.gelu(z, approximate="tanh")
        hA2 = torch.mm(h, A2)
        torch.addmm(b2, h, W2t).addmm_(hA2, B2)
        G_B2t = torch.mm(dY, B2.t().contiguous())
        dh = torch.mm(dY, W2).addmm_(G_B2t, A2.t().contiguous())
        torch.mm(h.t(), G_B2t)                 # dA2
        torch.mm(hA2.t(), dY)                  # dB2
        dz = torch.ops.aten.gelu_backward(dh, z, approximate="tanh")
        dz_B1t = torch.mm(dz, B1.t().contiguous())
        torch.mm(dz, W1).addmm_(dz_B1t, A1.t().contiguous())
        torch.mm(X.t(), dz_B1t)                # dA1
        torch.mm(XA1.t(), dz)                  # dB1
    return step


def mlp_ablation(torch, L, dev, seed, steps, warmup, M=4608, Dm=3072, F=12288, r=32, rs=32):
    """The MLP pair step with and without the MLP fusion (Sec. 3.3): the
    fused step runs FC1 with the GELU / quantize / projection epilogue and
    FC2's backward-input with the dGELU epilogue; the unfused step writes z
    and dH from plain GEMMs and applies GELU-tanh and its derivative as
    library elementwise kernels before quantizing h and dz with their
    projections.  Both keep the low-rank fusion.  A timing comparison only."""
    t, R = torch, r + rs
    g = t.Generator(device=dev)
    g.manual_seed(seed)
    u8, f32, bf = t.uint8, t.float32, t.bfloat16
    e = lambda sh, dt: t.empty(sh, dtype=dt, device=dev)
    nrm = lambda sh, sd: (t.randn(sh, generator=g, device=dev) * sd).to(bf)
    X, dY = nrm((M, Dm), 1.0), nrm((M, Dm), 1e-3)
    w1q, w1s, _ = L.ft_quantize_blockwise(nrm((F, Dm), 0.02), block_rows=32)
    w2q, w2s, _ = L.ft_quantize_blockwise(nrm((Dm, F), 0.02), block_rows=32)
    D1, U1, b1 = nrm((Dm, R), 0.01), nrm((R, F), 0.01), nrm((F,), 0.02)
    D2, U2, b2 = nrm((F, R), 0.01), nrm((R, Dm), 0.01), nrm((Dm,), 0.02)
    xq, xs = e((M, Dm // 2), u8), e((M, Dm // 32), u8)
    P1, P2, Qp1, Qp2 = (e((M, R), f32) for _ in range(4))
    z, h, dz, dH = (e((M, F), bf) for _ in range(4))
    hq, hs, dzq, dzs = e((M, F // 2), u8), e((M, F // 32), u8), e((M, F // 2), u8), e((M, F // 32), u8)
    Y, dX = e((M, Dm), bf), e((M, Dm), bf)
    gq, gs = e((M, Dm // 2), u8), e((M, Dm // 32), u8)
    dA1, dB1, dA2, dB2 = e((Dm, r), f32), e((r, F), f32), e((F, r), f32), e((r, Dm), f32)
    ws = lambda n: e((max(16, n),), u8)
    wx = ws(L.ft_quantize_workspace_size(M, Dm, 1, R, L.FT_PROJ_COLS_BY_R))
    wd = ws(L.ft_quantize_workspace_size(M, Dm, 1, R, L.FT_PROJ_R_BY_COLS))
    wh = ws(L.ft_quantize_workspace_size(M, F, 1, R, L.FT_PROJ_COLS_BY_R))
    wz = ws(L.ft_quantize_workspace_size(M, F, 1, R, L.FT_PROJ_R_BY_COLS))
    wg = ws(L.ft_linear_fwd_gelu_workspace_size(M, F, R))
    wdg = ws(L.ft_linear_bwd_input_dgelu_workspace_size(M, F, R))
    wl1, wl2 = ws(L.ft_lora_grads_workspace_size(M, Dm, F, R, r)), ws(L.ft_lora_grads_workspace_size(M, F, Dm, R, r))

    def common_tail():
        L.ft_linear_bwd_input(dzq, dzs, w1q, w1s, Dm, Qp1, D1, dx=dX)
        L.ft_lora_grads(h, dY, P2, Qp2, r, col0=rs, dA=dA2, dB=dB2, workspace=wl2)
        L.ft_lora_grads(X, dz, P1, Qp1, r, col0=rs, dA=dA1, dB=dB1, workspace=wl1)

    def fused():
        L.ft_quantize_blockwise(X, proj=D1, codes=xq, scales=xs, proj_out=P1, workspace=wx)
        L.ft_linear_fwd_gelu(xq, xs, w1q, w1s, Dm, P1, U1, b1, D2=D2, z=z, h=h, hq=hq, hs=hs, P2=P2, workspace=wg)
        L.ft_linear_fwd(hq, hs, w2q, w2s, F, P2, U2, b2, y=Y)
        L.ft_quantize_blockwise(dY, proj=U2, proj_layout=L.FT_PROJ_R_BY_COLS, codes=gq, scales=gs, proj_out=Qp2,
                                workspace=wd)
        L.ft_linear_bwd_input_dgelu(gq, gs, w2q, w2s, F, z, Qp2, D2, U1=U1, dz=dz, dzq=dzq, dzs=dzs, Qp1=Qp1,
                                    workspace=wdg)
        common_tail()

    def unfused():
        L.ft_quantize_blockwise(X, proj=D1, codes=xq, scales=xs, proj_out=P1, workspace=wx)
        L.ft_linear_fwd(xq, xs, w1q, w1s, Dm, P1, U1, b1, y=z)
        t.ops.aten.gelu.out(z, approximate="tanh", out=h)
        L.ft_quantize_blockwise(h, proj=D2, codes=hq, scales=hs, proj_out=P2, workspace=wh)
        L.ft_linear_fwd(hq, hs, w2q, w2s, F, P2, U2, b2, y=Y)
        L.ft_quantize_blockwise(dY, proj=U2, proj_layout=L.FT_PROJ_R_BY_COLS, codes=gq, scales=gs, proj_out=Qp2,
                                workspace=wd)
        L.ft_linear_bwd_input(gq, gs, w2q, w2s, F, Qp2, D2, dx=dH)
        t.ops.aten.gelu_backward.grad_input(dH, z, approximate="tanh", grad_input=dz)
        L.ft_quantize_blockwise(dz, proj=U1, proj_layout=L.FT_PROJ_R_BY_COLS, codes=dzq, scales=dzs, proj_out=Qp1,
                                workspace=wz)
        common_tail()

    def timed(fn):
        for _ in range(warmup):
            fn()
        t.cuda.synchronize()
        a, b = t.cuda.Event(enable_timing=True), t.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            fn()
        b.record()
        t.cuda.synchronize()
        return a.elapsed_time(b) / steps

    W1b, W2b = nrm((F, Dm), 0.02), nrm((Dm, F), 0.02)
    bf16_step = bf16_lora_mlp(t, W1b, D1[:, rs:].contiguous(), U1[rs:].contiguous(), b1, W2b,
                              D2[:, rs:].contiguous(), U2[rs:].contiguous(), b2, X, dY)
    tf, tu = timed(fused), timed(unfused)
    tb = timed(bf16_step)
    tf = min(tf, timed(fused))
    return {"metric": "MLP pair step time, MLP fusion ablation and BF16 LoRA (flux_mlp)", "unit": "ms",
            "fused_ms": round(tf, 4), "unfused_ms": round(tu, 4), "fusion_speedup": round(tu / tf, 3),
            "unfused": "FC1 and FC2 backward-input as plain GEMMs writing z and dH; GELU-tanh and its derivative "
                       "as library elementwise kernels; h and dz quantized with their projections separately",
            "bf16_lora_ms": round(tb, 4), "speedup_vs_bf16_lora": round(tb / tf, 3),
            "bf16_lora": BF16_LORA_TEXT,
            "steps": steps, "warmup": warmup, "data": "synthetic"}


def numerics_timing(torch, L, dev, seed, steps, warmup):
    """Time the quantizer's numerics variants at the QKV shapes (X 4608 x 3072
    with its [cols, R] projection; dY 4608 x 9216 with its [R, cols]
    projection), one HIP stream, events around the calls."""
    shape = __import__("paper_2607_05711_amd.gen", fromlist=["SHAPES"]).SHAPES["flux_qkv"]
    from paper_2607_05711_amd import gen
    d = gen.layer_inputs_torch(shape, seed, dev)
    M, K, N, R = shape.M, shape.K, shape.N, shape.R
    u8, f32 = torch.uint8, torch.float32
    e = lambda sh, dt: torch.empty(sh, dtype=dt, device=dev)
    out = {}
    for name, src, proj, layout, cols in (("quantize_x", d["X"], d["D"], L.FT_PROJ_COLS_BY_R, K),
                                          ("quantize_dy", d["dY"], d["U"], L.FT_PROJ_R_BY_COLS, N)):
        codes, scales, po = e((M, cols // 2), u8), e((M, cols // 32), u8), e((M, R), f32)
        ws = e((max(16, L.ft_quantize_workspace_size(M, cols, 1, R, layout)),), u8)
        nbytes = M * cols * (2 + 0.5 + 1 / 32) + M * R * 4 + cols * R * 2
        for mode, (rule, rnd) in (("floor_nearest", (0, 0)), ("noclip_nearest", (1, 0)),
                                  ("floor_stochastic", (0, 1)), ("noclip_stochastic", (1, 1))):
            fn = lambda: L.ft_quantize_blockwise_mode(src, proj=proj, proj_layout=layout, codes=codes, scales=scales,
                                                      proj_out=po, workspace=ws, scale_rule=rule, rounding=rnd,
                                                      seed=seed, stream=1)
            for _ in range(warmup):
                fn()
            torch.cuda.synchronize()
            a_, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a_.record()
            for _ in range(steps):
                fn()
            b_.record()
            torch.cuda.synchronize()
            us = 1e3 * a_.elapsed_time(b_) / steps
            out["%s_%s" % (name, mode)] = {"us": round(us, 2), "hbm_frac": round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
    return {"metric": "quantize + fused projection time by numerics variant (flux_qkv shapes)", "unit": "us",
            "variants": out, "steps": steps, "warmup": warmup, "data": "synthetic"}


def stability_probe(torch, L, dev, seed, steps=150, M=4096, K=1024, N=1024, r=16, rs=16, lr=2e-3):
    """A synthetic gradient-norm stability probe (the paper's stabilizer and
    precision ablation, Sec. 4.3): LoRA fine-tuning of one triple-branch
    linear toward a teacher whose weight differs from the frozen one by a
    low-rank term, with Adam on A and B.  Activations carry 1 % outlier
    channels x30 and the frozen weight is heavy-tailed, so 4-bit quantization
    error matters.  Variants: the W4A4G4 layer with the stabilizer (L1 L2 from
    a rank-rs SVD of the weight's quantization residual), without it,
    with stochastic rounding of the gradient, with the no-clip scale rule;
    and an unquantized fp32 reference of the same model.  Per step it records
    the loss and the Frobenius norms of dA and dB; the JSON line summarizes
    them against the reference."""
    t = torch
    g = t.Generator(device=dev)
    g.manual_seed(seed)
    f32, bf = t.float32, t.bfloat16
    nrm = lambda sh, sd: t.randn(sh, generator=g, device=dev, dtype=f32) * sd
    # frozen weight: Student-t(3)-like tails
    z = nrm((N, K), 1.0)
    chi = sum(nrm((N, K), 1.0) ** 2 for _ in range(3)) / 3.0
    W0 = (0.02 * z / t.sqrt(chi)).to(bf)
    delta = nrm((N, 8), 0.05) @ nrm((8, K), 0.05)               # what the adapter should learn
    W_teacher = W0.float() + delta
    wq, ws, _ = L.ft_quantize_blockwise(W0, block_rows=32)
    # dequantized weight (offline set-up of the stabilizer; not the probe's step)
    lut = t.tensor([0, .5, 1, 1.5, 2, 3, 4, 6, -0., -.5, -1, -1.5, -2, -3, -4, -6], device=dev, dtype=f32)
    codes = t.stack([wq & 15, wq >> 4], dim=-1).reshape(N, K).long()
    scale = t.exp2(ws.float() - 127.0).repeat_interleave(32, 0).repeat_interleave(32, 1)
    Wd = lut[codes] * scale
    Uv, Sv, Vh = t.linalg.svd((W0.float() - Wd).double(), full_matrices=False)
    L1 = (Vh[:rs].T * Sv[:rs]).float().to(bf)                    # [K, rs]
    L2 = Uv[:, :rs].T.float().to(bf)                             # [rs, N]

    def batch(step):
        gb = t.Generator(device=dev)
        gb.manual_seed(seed * 7919 + step)
        x = t.randn((M, K), generator=gb, device=dev, dtype=f32)
        cols = t.randperm(K, generator=gb, device=dev)[: K // 100]
        x[:, cols] *= 30.0
        return x

    def run(variant):
        stab = variant != "no_stabilizer"
        A = (nrm((K, r), 1.0) / K ** 0.5).requires_grad_(True)
        B = t.zeros((r, N), device=dev, dtype=f32, requires_grad=True)
        opt = t.optim.Adam([A, B], lr=lr)
        rule = 1 if variant == "no_clip" else 0
        rnd = 1 if variant == "sr_grad" else 0
        hist = []
        for step in range(steps):
            x = batch(step)
            xb = x.to(bf)
            target = x @ W_teacher.T
            if variant == "fp32_reference":
                y = x @ W0.float().T + (x @ A) @ B
                loss = 0.5 * ((y - target) ** 2).sum() / M
                opt.zero_grad()
                loss.backward()
                gA, gB = A.grad, B.grad
            else:
                D = (t.cat([L1, A.detach().to(bf)], 1) if stab else A.detach().to(bf)).contiguous()
                U = (t.cat([L2, B.detach().to(bf)], 0) if stab else B.detach().to(bf)).contiguous()
                xq, xs, P = L.ft_quantize_blockwise_mode(xb, proj=D, scale_rule=rule)
                y = L.ft_linear_fwd(xq, xs, wq, ws, K, P, U, None, out_dtype=f32)
                diff = y - target
                loss = 0.5 * (diff ** 2).sum() / M
                dY = (diff / M).to(bf)
                gq, gs, Qp = L.ft_quantize_blockwise_mode(dY, proj=U, proj_layout=L.FT_PROJ_R_BY_COLS,
                                                          scale_rule=rule, rounding=rnd, seed=seed, stream=step)
                dA, dB = L.ft_lora_grads(xb, dY, P, Qp, r, col0=rs if stab else 0)
                opt.zero_grad()
                A.grad, B.grad = dA, dB
                gA, gB = dA, dB
            hist.append((float(loss.detach()), float(gA.norm()), float(gB.norm())))
            opt.step()
        return hist

    variants = ["fp32_reference", "w4a4g4", "no_stabilizer", "sr_grad", "no_clip"]
    hists = {v: run(v) for v in variants}
    ref_h = hists["fp32_reference"]
    summary = {}
    for v, h in hists.items():
        gn = [(a ** 2 + b ** 2) ** 0.5 for _, a, b in h]
        gr = [(a ** 2 + b ** 2) ** 0.5 for _, a, b in ref_h]
        summary[v] = {"loss": {str(k): round(h[k][0], 6) for k in (0, 10, 50, steps // 2, steps - 1)},
                      "grad_norm": {str(k): round(gn[k], 6) for k in (0, 10, 50, steps // 2, steps - 1)},
                      "grad_norm_max_over_min": round(max(gn[1:]) / max(min(gn[1:]), 1e-30), 3),
                      "grad_norm_rel_dev_vs_reference": round(sum(abs(a / b - 1) for a, b in zip(gn[1:], gr[1:]))
                                                              / (len(gn) - 1), 4)}
    return {"metric": "synthetic gradient-norm stability probe (LoRA fine-tuning of one triple-branch linear)",
            "shape": {"M": M, "K": K, "N": N, "r": r, "r_s": rs}, "steps": steps, "optimizer": "Adam lr %g" % lr,
            "data": "synthetic: X N(0,1) with 1%% channels x30, heavy-tailed frozen W, teacher W + rank-8 delta",
            "variants": summary}


LIBRARY_GEMM_TEXT = ("hipBLASLt's MXFP4 GEMM through torch._scaled_mm (E2M1 operands, one E8M0 scale per 1x32 "
                     "block of each operand, bf16 output) against this library's FP4 GEMM without the low-rank "
                     "branch and the bias, on the same random codes and scales (the weight's 32x32 tile scales "
                     "repeated per row for the library); for the backward-input shape the library gets a "
                     "pre-transposed weight (random codes of that shape), while this library reads the forward's "
                     "codes transposed. Back-to-back calls, warm. Context only: neither is the layer step.")


def library_gemm(torch, _lib, dev, seed, steps=20, warmup=5):
    """Plain MXFP4 GEMM times (us) of the vendor library and of this library at
    the FLUX shapes: forward Q(X) Q(W)^T and backward-input Q(dY) Q(W)."""
    g = torch.Generator(device=dev)
    g.manual_seed(seed)

    def codes(r, c):
        return torch.randint(0, 256, (r, c // 2), dtype=torch.uint8, device=dev, generator=g)

    def scales(r, c):
        return torch.randint(120, 131, (r, c), dtype=torch.uint8, device=dev, generator=g)

    def time_us(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps * 1e3

    e2m1, e8m0 = torch.float4_e2m1fn_x2, torch.float8_e8m0fnu
    out = {"what": LIBRARY_GEMM_TEXT}
    for name, M, K, N in (("qkv", 4608, 3072, 9216), ("mlp_fc1", 4608, 3072, 12288)):
        wq, ws = codes(N, K), scales(N // 32, K // 32)
        ws_rows = ws.repeat_interleave(32, dim=0).contiguous()
        # forward: [M, K] x [N, K]^T
        xq, xs = codes(M, K), scales(M, K // 32)
        lib_f = time_us(lambda: torch._scaled_mm(xq.view(e2m1), wq.view(e2m1).t(), xs.view(e8m0), ws_rows.view(e8m0),
                                                 out_dtype=torch.bfloat16))
        ours_f = time_us(lambda: _lib.ft_linear_fwd(xq, xs, wq, ws, K))
        # backward-input: [M, N] x [N, K]; the library takes W^T [K, N] with scales along N
        gq, gs = codes(M, N), scales(M, N // 32)
        wtq = codes(K, N)
        wts = ws.t().repeat_interleave(32, dim=0).contiguous()
        lib_b = time_us(lambda: torch._scaled_mm(gq.view(e2m1), wtq.view(e2m1).t(), gs.view(e8m0), wts.view(e8m0),
                                                 out_dtype=torch.bfloat16))
        ours_b = time_us(lambda: _lib.ft_linear_bwd_input(gq, gs, wq, ws, K))
        fl = 2.0 * M * N * K
        out[name] = {"shape": [M, K, N],
                     "fwd_us": {"library": round(lib_f, 2), "ours": round(ours_f, 2)},
                     "bwd_us": {"library": round(lib_b, 2), "ours": round(ours_b, 2)},
                     "fwd_tflops": {"library": round(fl / lib_f / 1e6, 1), "ours": round(fl / ours_f / 1e6, 1)},
                     "bwd_tflops": {"library": round(fl / lib_b / 1e6, 1), "ours": round(fl / ours_b / 1e6, 1)}}
        torch.cuda.empty_cache()
    return out


def dit_step_timing(torch, dev, seed, steps, warmup, cfg=None):
    """One synthetic FLUX.1-dev DiT training step (19 double + 38 single
    blocks at 4096 image + 512 text tokens; forward, loss, backward, AdamW on
    the LoRA factors) with the W4A4G4 layers, and the same step with BF16
    LoRA linears (the paper's comparison, Sec. 4 "Efficiency Results")."""
    from paper_2607_05711_amd import dit
    cfg = cfg or dit.FLUX_DEV
    out = {}
    for kind in ("fp4", "bf16"):
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats(dev)
        model = dit.DiT(cfg, kind, seed, dev)
        trainer = dit.Trainer(model)
        batch = dit.synthetic_batch(cfg, seed + 1, dev)
        wbytes = sum(t.numel() * t.element_size() for m in model.modules()
                     for t in ([m.wq, m.ws] if isinstance(m, dit.FourTuneLinear) else
                               [m.W] if isinstance(m, dit.Bf16LoraLinear) else []))
        for _ in range(warmup):
            trainer.step(*batch)
        torch.cuda.synchronize()
        a_, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a_.record()
        for _ in range(steps):
            loss = trainer.step(*batch)
        b_.record()
        torch.cuda.synchronize()
        out[kind] = {"ms_per_step": round(a_.elapsed_time(b_) / steps, 2), "loss": round(float(loss), 5),
                     "peak_memory_gb": round(torch.cuda.max_memory_allocated(dev) / 1e9, 2),
                     "linear_weight_gb": round(wbytes / 1e9, 2)}
        del model, trainer, batch
        print("dit %s: %.2f ms/step" % (kind, out[kind]["ms_per_step"]), file=sys.stderr, flush=True)
    return {"metric": "synthetic FLUX.1-dev DiT training step time, W4A4G4 vs BF16 LoRA", "unit": "ms",
            "w4a4g4": out["fp4"], "bf16_lora": out["bf16"],
            "speedup_vs_bf16_lora": round(out["bf16"]["ms_per_step"] / out["fp4"]["ms_per_step"], 3),
            "config": {"double_blocks": cfg.double_blocks, "single_blocks": cfg.single_blocks,
                       "img_tokens": cfg.img_tokens, "txt_tokens": cfg.txt_tokens, "hidden": cfg.hidden,
                       "heads": cfg.heads, "mlp": cfg.mlp, "lora_rank": cfg.lora_rank,
                       "stabilizer_rank": cfg.stab_rank},
            "step": "forward, MSE loss, backward, AdamW on every LoRA factor; attention, norms, modulation "
                    "and RoPE as torch operations (fused attention kernels only)",
            "steps": steps, "warmup": warmup, "data": "synthetic, random weights"}


def start_clock_sampler():
    """rocm-smi's clocks and power, sampled every few tenths of a second by a shell loop
    started before this process touches the GPU (so no child process is
    started from a process holding a GPU context).  Lines: '<unix time> <json>'.
    Returns (process, path) or (None, None) when rocm-smi is not there."""
    if not any(os.access(os.path.join(d, "rocm-smi"), os.X_OK) for d in os.environ.get("PATH", "").split(os.pathsep)):
        return None, None
    fd, path = tempfile.mkstemp(prefix="ft_clock_", suffix=".txt")
    # it polls only while <path>.go exists, so the timed steps run without it
    script = ("while true; do if [ -e '%s.go' ]; then t=$(date +%%s.%%N); "
              "o=$(timeout 10 rocm-smi --showclocks --showpower --json 2>/dev/null | tr -d '\\n'); "
              "echo \"$t $o\"; sleep 0.2; else sleep 0.05; fi; done") % path
    proc = subprocess.Popen(["bash", "-c", script], stdout=fd, stderr=subprocess.DEVNULL, start_new_session=True)
    os.close(fd)
    return proc, path


def stop_clock_sampler(proc, path):
    if proc is None:
        return
    try:
        os.killpg(proc.pid, signal.SIGTERM)
    except ProcessLookupError:
        pass
    proc.wait(timeout=10)
    for p in (path, path + ".go"):
        try:
            os.unlink(p)
        except OSError:
            pass


def clock_under_load(torch, fn, path, seconds=2.0):
    """Run fn back to back for `seconds` and return the rocm-smi samples taken
    meanwhile: graphics clock (MHz) and package power (W)."""
    if path is None:
        return {"error": "rocm-smi not found"}
    fn()
    torch.cuda.synchronize()
    open(path + ".go", "w").close()
    t0 = time.time()
    calls = 0
    while time.time() - t0 < seconds:
        for _ in range(10):
            fn()
        calls += 10
        torch.cuda.synchronize()
    t1 = time.time()
    time.sleep(1.0)   # let a sample taken in the window finish writing
    os.unlink(path + ".go")
    sclk, mclk, power = [], [], []
    with open(path) as f:
        for line in f:
            parts = line.strip().split(" ", 1)
            if len(parts) != 2:
                continue
            try:
                t, d = float(parts[0]), json.loads(parts[1]).get("card0", {})
            except ValueError:
                continue
            if not t0 + 0.2 <= t <= t1 - 0.5:   # the sample's rocm-smi call ran inside the window
                continue
            for k, v in d.items():
                if k.startswith("sclk clock speed"):
                    sclk.append(float(v.strip("()").lower().replace("mhz", "")))
                elif k.startswith("mclk clock speed"):
                    mclk.append(float(v.strip("()").lower().replace("mhz", "")))
                elif "power" in k.lower() and "max" not in k.lower():
                    try:
                        power.append(float(str(v).split()[0]))
                    except ValueError:
                        pass
    return {"what": "rocm-smi samples while the forward GEMM of the QKV step runs back to back",
            "seconds": round(t1 - t0, 2), "calls": calls, "sclk_mhz": sclk, "mclk_mhz": mclk,
            "power_w": power if power else "not reported by rocm-smi here"}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the layer's data-parallel shards are independent and the "
              "library runs no collectives; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return

    default_line = not (args.numerics or args.dit or args.stability or args.ablation)
    sample = default_line and args.workload == "flux_qkv" and not args.no_clock_sample
    sampler, sample_path = start_clock_sampler() if sample else (None, None)
    try:
        run(args, sample_path)
    finally:
        stop_clock_sampler(sampler, sample_path)


DEFAULT_WARMUP = {"flux_qkv": 200, "flux_mlp": 100, "flux_single": 20, "flux_stack": 3}


def resolve_warmup(args):
    """Warm-up steps: --warmup if given, else the mode's default."""
    if args.warmup is not None:
        return args.warmup
    return 3 if args.dit else 20 if (args.ablation or args.numerics) else DEFAULT_WARMUP[args.workload]


def run(args, sample_path):
    import torch
    from paper_2607_05711_amd import _lib, gen

    args.warmup = resolve_warmup(args)

    _lib.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.numerics:
        print(json.dumps(numerics_timing(torch, _lib, dev, args.seed, args.steps, args.warmup)), flush=True)
        return
    if args.dit:
        print(json.dumps(dit_step_timing(torch, dev, args.seed, args.steps, args.warmup)), flush=True)
        return
    if args.stability:
        print(json.dumps(stability_probe(torch, _lib, dev, args.seed)), flush=True)
        return
    if args.ablation and args.workload == "flux_mlp":
        print(json.dumps(mlp_ablation(torch, _lib, dev, args.seed, args.steps, args.warmup)), flush=True)
        return
    if args.ablation:
        if args.workload != "flux_qkv":
            raise SystemExit("--ablation is defined for flux_qkv and flux_mlp")
        d = gen.layer_inputs_torch(gen.SHAPES["flux_qkv"], args.seed, dev)
        wq, ws, _ = _lib.ft_quantize_blockwise(d["W"], block_rows=32)
        print(json.dumps(fusion_ablation(torch, _lib, d, wq, ws, gen.SHAPES["flux_qkv"], args.steps, args.warmup)),
              flush=True)
        return
    rec = measure_workload(torch, _lib, gen, dev, args.workload, args.steps, args.warmup, args.seed)
    d = rec.pop("_inputs")
    out = {
        "metric": "fused W4A4 linear fwd+bwd TFLOP/s at FLUX 1024^2 shapes; % MXFP4 MFMA peak",
        "value": rec["tflops"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": rec["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "mxfp4",
        "data": "synthetic",
        "config": rec["config"],
    }
    out.update({k: v for k, v in rec.items() if k not in ("tflops", "ms_per_step", "config")})
    if sample_path is not None:
        try:
            K = d["X"].shape[1]
            xq, xs, P = _lib.ft_quantize_blockwise(d["X"], proj=d["D"])
            wq, ws, _ = _lib.ft_quantize_blockwise(d["W"], block_rows=32)
            ybuf = torch.empty((d["X"].shape[0], d["W"].shape[0]), dtype=torch.bfloat16, device=dev)
            gc = clock_under_load(
                torch, lambda: _lib.ft_linear_fwd(xq, xs, wq, ws, K, P, d["U"], d["bias"], y=ybuf), sample_path)
            rf = out.get("roofline") or {}
            if gc.get("sclk_mhz") and rf.get("achieved") and rf.get("peak"):
                mhz = sorted(gc["sclk_mhz"])[len(gc["sclk_mhz"]) // 2]
                # the dense MXFP4 peak scales with the clock: 16384 FLOP per clock per CU
                gc["gemm_fwd_frac_at_median_sclk"] = round(rf["achieved"] / (rf["peak"] * mhz / 2400.0), 4)
            out["gpu_clock"] = gc
            del xq, xs, P, wq, ws, ybuf
        except Exception as e:   # noqa: BLE001
            out["gpu_clock"] = {"error": "%s: %s" % (type(e).__name__, e)}
    if args.workload == "flux_qkv" and not args.no_other_workloads:
        # the other FLUX configurations, each as its own whole step (fewer steps)
        others = {}
        for name, st, wu in (("flux_mlp", 20, 10), ("flux_single", 10, 5), ("flux_stack", 3, 2)):
            o = measure_workload(torch, _lib, gen, dev, name, st, wu, args.seed, per_kernel=name != "flux_stack")
            o.pop("_inputs")
            others[name] = {"ms_per_step": o["ms_per_step"], "tflops": o["tflops"],
                            "pct_mxfp4_peak": o["pct_mxfp4_peak"], "steps": st, "warmup": wu,
                            "step_ms": o["step_ms"], "workload": o["config"]["workload"]}
            for k in ("kernels_us", "kernels_frac", "kernels_frac_flushed"):
                if k in o:
                    others[name][k] = o[k]
            torch.cuda.empty_cache()
            print("measured %s: %.3f ms/step" % (name, o["ms_per_step"]), file=sys.stderr, flush=True)
        # the synthetic DiT training step, W4A4G4 against BF16 LoRA; a failure here is reported, not hidden
        try:
            others["flux_dit"] = dit_step_timing(torch, dev, args.seed, 3, 2)
        except Exception as e:   # noqa: BLE001
            others["flux_dit"] = {"error": "%s: %s" % (type(e).__name__, e)}
        torch.cuda.empty_cache()
        out["other_workloads"] = others
        try:
            out["library_gemm"] = library_gemm(torch, _lib, dev, args.seed)
        except Exception as e:   # noqa: BLE001
            out["library_gemm"] = {"error": "%s: %s" % (type(e).__name__, e)}
        # the fusion ablations of --ablation (fused against unfused steps, and BF16 LoRA), fewer steps
        try:
            wq_a, ws_a, _ = _lib.ft_quantize_blockwise(d["W"], block_rows=32)
            out["fusion_ablation"] = {
                "flux_qkv": fusion_ablation(torch, _lib, d, wq_a, ws_a, gen.SHAPES["flux_qkv"], 20, 20),
                "flux_mlp": mlp_ablation(torch, _lib, dev, args.seed, 20, 20)}
            del wq_a, ws_a
        except Exception as e:   # noqa: BLE001
            out["fusion_ablation"] = {"error": "%s: %s" % (type(e).__name__, e)}
        torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        if d is None:
            shape = gen.SHAPES["flux_qkv"]
            d = gen.layer_inputs_torch(shape, args.seed, dev)
        out["cpu_baseline"] = cpu_baseline(d, gen.SHAPES["flux_qkv"], args.cpu_rows)
        if args.workload != "flux_qkv":
            out["cpu_baseline"]["sample"] += " (the QKV linear, the oracle's per-linear rate)"
    print(json.dumps(out), flush=True)


def measure_workload(torch, _lib, gen, dev, workload, steps, warmup, seed, per_kernel=True):
    """Build one workload's buffers, time its step, and return the measured
    figures (the layers' inputs for flux_qkv under "_inputs")."""
    layers = workload_layers(workload)
    b = Builder(torch, _lib, dev, seed, random_weights=workload == "flux_stack")
    fwd_ops, bwd_ops, counts = [], [], {}
    d = given = None
    if workload == "flux_qkv":
        # the headline layer keeps the seeded recipe of the parity tests
        d = gen.layer_inputs_torch(gen.SHAPES["flux_qkv"], seed, dev)
        wq, ws, _ = _lib.ft_quantize_blockwise(d["W"], block_rows=32)     # offline weight preparation
        given = dict(X=d["X"], dY=d["dY"], wq=wq, ws=ws, D=d["D"], U=d["U"], bias=d["bias"])
    lanes = workload_lanes(workload, layers)
    for (kind, M, K, N, r, rs), (_, lane) in zip(layers, lanes):
        b.lane = lane
        if kind == "linear":
            f, bw, c = b.linear(M, K, N, r, rs, given)
        else:
            f, bw, c = b.mlp(M, K, N, r, rs)
        fwd_ops.append(f)
        bwd_ops.append(bw)
        for k, v in c.items():
            counts[k] = counts.get(k, 0.0) + v
    ops = [op for f in fwd_ops for op in f] + [op for bw in reversed(bwd_ops) for op in bw]
    torch.cuda.synchronize()

    # The timed step: each group's lane-1 layers on a second stream (default
    # priority) that starts after the group's preceding work and is joined at
    # the group's end.  Per-kernel timing below runs everything on one stream.
    groups = []
    for i, (g, lane) in enumerate(lanes):
        if not groups or groups[-1][0] != g:
            groups.append((g, [[], []]))
        groups[-1][1][lane].append(i)
    side = torch.cuda.Stream(device=dev) if any(lane for _, lane in lanes) else None
    ev_pool = [torch.cuda.Event() for _ in range(4 * len(groups))]

    def run_group(members, ops_of, k):
        main_ids, side_ids = members
        if not side_ids:
            for i in main_ids:
                for _, fn in ops_of(i):
                    fn()
            return
        main = torch.cuda.current_stream()
        ev0, ev1 = ev_pool[2 * k], ev_pool[2 * k + 1]
        ev0.record(main)
        side.wait_event(ev0)
        with torch.cuda.stream(side):
            for i in side_ids:
                for _, fn in ops_of(i):
                    fn()
            ev1.record(side)
        for i in main_ids:
            for _, fn in ops_of(i):
                fn()
        main.wait_event(ev1)

    def step_timed():
        for k, (_, members) in enumerate(groups):
            run_group(members, lambda i: fwd_ops[i], k)
        for k, (_, members) in enumerate(reversed(groups)):
            run_group([list(reversed(members[0])), list(reversed(members[1]))], lambda i: bwd_ops[i],
                      len(groups) + k)

    flush_buf = torch.ones(1 << 30, dtype=torch.uint8, device=dev)

    def flush():
        flush_buf.sum(dtype=torch.int64)

    def step(ev=None, flushed=False):
        for i, (_, fn) in enumerate(ops):
            if flushed:
                flush()
            if ev is not None:
                ev[2 * i].record()
            fn()
            if ev is not None:
                ev[2 * i + 1].record()

    for _ in range(warmup):
        step_timed()
    torch.cuda.synchronize()

    # whole-step timing: no events between kernels
    t0 = torch.cuda.Event(enable_timing=True); t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for _ in range(steps):
        step_timed()
    t1.record()
    torch.cuda.synchronize()
    ms_per_step = t0.elapsed_time(t1) / steps

    # per-step times: warm (back to back) and with the caches flushed before
    # every step by reading a 1 GiB buffer (L2 and the 256 MB last-level
    # cache then hold that buffer's clean lines, not the step's inputs)
    nps = min(steps, 20)

    def per_step(flushed):
        evs_ = []
        for _ in range(nps):
            if flushed:
                flush()
            a_, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a_.record()
            step_timed()
            b_.record()
            evs_.append((a_, b_))
        torch.cuda.synchronize()
        return sorted(a_.elapsed_time(b_) for a_, b_ in evs_)

    def summary(v):
        q = lambda p: v[min(len(v) - 1, int(round(p * (len(v) - 1))))]
        return {"median": round(q(0.5), 4), "p10": round(q(0.1), 4), "p90": round(q(0.9), 4)}

    step_warm, step_flushed = summary(per_step(False)), summary(per_step(True))
    tflops = counts["flops"] / (ms_per_step * 1e-3) / 1e12
    rec = {
        "ms_per_step": round(ms_per_step, 4),
        "tflops": round(tflops, 2),
        "config": {"workload": "%s: %s" % (workload, WORKLOAD_TEXT[workload]),
                   "layers": len(layers), "lora_rank": layers[0][4], "stabilizer_rank": layers[0][5],
                   "outputs": "activations and input gradients bf16; dA, dB fp32", "parallelism": "single GPU"},
        "pct_mxfp4_peak": round(100.0 * tflops / MXFP4_PEAK_TFLOPS, 2),
        "schedule": ("image and text streams of each double block on two HIP streams; per-kernel times on one"
                     if side is not None else "one HIP stream"),
        "step_ms": {"steps": nps, "warm": step_warm, "flushed": step_flushed,
                    "flush": "1 GiB read before each step (L2 and last-level cache hold no inputs)",
                    "flushed_tflops_median": round(counts["flops"] / (step_flushed["median"] * 1e-3) / 1e12, 2)},
        "_inputs": d,
    }
    if not per_kernel:
        del flush_buf
        return rec

    # per-kernel timing: events around each call, same stream, warm (calls
    # back to back) and flushed (the 1 GiB read before every call, outside
    # its events: each kernel finds its inputs in HBM only)
    kinds = []
    for k, _ in ops:
        if k not in kinds:
            kinds.append(k)

    def per_kernel_us(flushed):
        psteps = min(steps, 20 if len(ops) < 50 else 2)
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2 * len(ops))] for _ in range(psteps)]
        for s_ in range(psteps):
            step(evs[s_], flushed)
        torch.cuda.synchronize()
        tot_us = {k: 0.0 for k in kinds}
        calls = {k: 0 for k in kinds}
        for s_ in range(psteps):
            for i, (k, _) in enumerate(ops):
                tot_us[k] += 1e3 * evs[s_][2 * i].elapsed_time(evs[s_][2 * i + 1])
                calls[k] += 1
        return {k: tot_us[k] / psteps for k in kinds}, {k: tot_us[k] / calls[k] for k in kinds}, \
            {k: calls[k] / psteps for k in kinds}

    step_us, launch_us, calls_per_step = per_kernel_us(False)
    step_us_fl, _, _ = per_kernel_us(True)
    del flush_buf

    def fracs(us):
        frac = {}
        for k in kinds:
            if k.startswith("gemm"):
                frac[k + "_mxfp4"] = round(counts[k] / (us[k] * 1e-6) / 1e12 / MXFP4_PEAK_TFLOPS, 4)
            else:
                frac[k + "_hbm"] = round(counts[k] / (us[k] * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)
        return frac

    gemms = [k for k in kinds if k.startswith("gemm")]
    gemm = max(gemms, key=lambda k: step_us[k])
    per_call_flops = counts[gemm] / calls_per_step[gemm]
    achieved = counts[gemm] / (step_us[gemm] * 1e-6) / 1e12
    kname = {"gemm_fwd": "ft::k_gemm_fp4_pipe<false, false, 0, true> (forward)",
             "gemm_bwd": "ft::k_gemm_fp4_pipe<true, false, 0, true> (backward-input)",
             "gemm_fwd_gelu": "ft::k_gemm_fp4_pipe<false, false, 1, true> (forward, GELU epilogue)",
             "gemm_bwd_dgelu": "ft::k_gemm_fp4_pipe<true, false, 2, true> (backward-input, dGELU epilogue)"}[gemm]
    rec.update({
        "roofline": {"bound": "mfma", "kernel": kname,
                     "achieved": round(achieved, 1), "peak": MXFP4_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / MXFP4_PEAK_TFLOPS, 4),
                     "traffic": measured_traffic("bwd" if gemm == "gemm_bwd" else "fwd")
                     if workload == "flux_qkv" else None,
                     "per_launch_flops": per_call_flops, "avg_launch_us": round(launch_us[gemm], 2)},
        "kernels_us": {k: round(step_us[k], 2) for k in kinds},
        "kernels_frac": fracs(step_us),
        "kernels_us_flushed": {k: round(step_us_fl[k], 2) for k in kinds},
        "kernels_frac_flushed": fracs(step_us_fl),
    })
    return rec


def cpu_baseline(d, shape, rows):
    """The fp64 oracle, as it stands, over the first `rows` token rows of the
    same inputs (whole step: both quantizations and projections, forward,
    backward-input, adapter gradients over those rows).  With rows == 0 a
    32-row pass sizes the sample to about 12 s of CPU work."""
    import numpy as np
    import torch

    from oracle import ref

    M, K, N, r, rs, R = shape.M, shape.K, shape.N, shape.r, shape.r_s, shape.R
    bits = lambda t: t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    W, D, U, bias = bits(d["W"]), bits(d["D"]), bits(d["U"]), bits(d["bias"])
    wq, ws = ref.quantize(W, 32)                 # offline in the method; not timed

    def run(n):
        X, dY = bits(d["X"][:n]), bits(d["dY"][:n])
        t = time.perf_counter()
        xq, xs = ref.quantize(X, 1)
        P, Pa = ref.proj(X, D, 0)
        ref.linear_fwd(xq, xs, wq, ws, K, P, U, bias, Pabs=Pa)
        gq, gs = ref.quantize(dY, 1)
        Qp, Qa = ref.proj(dY, U, 1)
        ref.linear_bwd_input(gq, gs, wq, ws, K, Qp, D, Qpabs=Qa)
        ref.lora_grads(X, dY, P[:, rs:], Qp[:, rs:])
        return time.perf_counter() - t

    if not rows:
        t32 = run(min(32, M))
        rows = int(min(M, max(32, 12.0 / max(t32 / min(32, M), 1e-6))))
    dt = run(rows)
    fp4, lowrank, lora = layer_flops(rows, K, N, r, R)
    return {"value": round((fp4 + lowrank + lora) / dt / 1e12, 6), "unit": "TFLOP/s",
            "cores": ref.num_threads(), "kind": "oracle",
            "sample": "first %d of %d token rows through the whole layer step, fp64 (%.1f s)" % (rows, M, dt)}


if __name__ == "__main__":
    main()
