"""Benchmark: one W4A4G4 triple-branch linear layer, forward + backward, on one GPU.

A step is the whole hot path over one batch of synthetic FLUX.1-dev-shaped
input (attention QKV projection at 1024x1024: M = 4096 image + 512 text tokens,
K = 3072, N = 9216, LoRA rank 32, stabilizer rank 32):

  quantize X (1x32 MXFP4) + P = X [L1|A]          ft_quantize_blockwise
  Y  = Q(X) Q(W)^T + P [L2;B] + bias   (bf16)      ft_linear_fwd
  quantize dY + Qp = dY [L2;B]^T                    ft_quantize_blockwise
  dX = Q(dY) Q(W) + Qp [L1|A]^T        (bf16)      ft_linear_bwd_input
  dA = X^T (dY B^T), dB = (X A)^T dY   (fp32)      ft_lora_grads

The frozen weight is quantized once before timing (offline in the method).
Inputs are drawn on the device with a seeded generator and are resident in HBM
when the timed region starts.  Prints one JSON line.
"""
import argparse
import hashlib
import json
import os
import sys
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
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="flux_qkv")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=0, help="token rows in the oracle sample (0: auto)")
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


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the layer's data-parallel shards are independent and this "
              "build runs no collectives; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return

    import torch
    from paper_2607_05711_amd import _lib, gen

    _lib.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    shape = gen.SHAPES[args.workload]
    M, K, N, r, rs, R = shape.M, shape.K, shape.N, shape.r, shape.r_s, shape.R

    d = gen.layer_inputs_torch(shape, args.seed, dev)
    X, W, D, U, dY, bias = d["X"], d["W"], d["D"], d["U"], d["dY"], d["bias"]
    wq, ws, _ = _lib.ft_quantize_blockwise(W, block_rows=32)            # offline weight preparation
    u8, f32, bf = torch.uint8, torch.float32, torch.bfloat16
    xq = torch.empty((M, K // 2), dtype=u8, device=dev); xs = torch.empty((M, K // 32), dtype=u8, device=dev)
    P = torch.empty((M, R), dtype=f32, device=dev)
    Y = torch.empty((M, N), dtype=bf, device=dev)
    gq = torch.empty((M, N // 2), dtype=u8, device=dev); gs = torch.empty((M, N // 32), dtype=u8, device=dev)
    Qp = torch.empty((M, R), dtype=f32, device=dev)
    dX = torch.empty((M, K), dtype=bf, device=dev)
    dA = torch.empty((K, r), dtype=f32, device=dev); dB = torch.empty((r, N), dtype=f32, device=dev)
    # workspaces for the partial sums (allocated once, outside the timed region)
    wspace = lambda n: torch.empty(max(n, 16), dtype=u8, device=dev)
    ws_x = wspace(_lib.ft_quantize_workspace_size(M, K, 1, R, _lib.FT_PROJ_COLS_BY_R))
    ws_dy = wspace(_lib.ft_quantize_workspace_size(M, N, 1, R, _lib.FT_PROJ_R_BY_COLS))
    ws_lg = wspace(_lib.ft_lora_grads_workspace_size(M, K, N, R, r))

    names = ["quantize_x", "gemm_fwd", "quantize_dy", "gemm_bwd", "lora_grads"]

    def step(ev=None):
        def mark(i):
            if ev is not None:
                ev[i].record()
        mark(0)
        _lib.ft_quantize_blockwise(X, proj=D, proj_layout=_lib.FT_PROJ_COLS_BY_R, codes=xq, scales=xs, proj_out=P,
                                   workspace=ws_x)
        mark(1)
        _lib.ft_linear_fwd(xq, xs, wq, ws, K, P, U, bias, y=Y)
        mark(2)
        _lib.ft_quantize_blockwise(dY, proj=U, proj_layout=_lib.FT_PROJ_R_BY_COLS, codes=gq, scales=gs, proj_out=Qp,
                                   workspace=ws_dy)
        mark(3)
        _lib.ft_linear_bwd_input(gq, gs, wq, ws, K, Qp, D, dx=dX)
        mark(4)
        _lib.ft_lora_grads(X, dY, P, Qp, r, col0=rs, dA=dA, dB=dB, workspace=ws_lg)
        mark(5)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # whole-step timing: no events between kernels
    t0 = torch.cuda.Event(enable_timing=True); t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for _ in range(args.steps):
        step()
    t1.record()
    torch.cuda.synchronize()
    ms_per_step = t0.elapsed_time(t1) / args.steps

    # per-kernel timing: events around each launch, same stream
    per = {n: [] for n in names}
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(args.steps)]
    for s in range(args.steps):
        step(evs[s])
    torch.cuda.synchronize()
    for s in range(args.steps):
        for i, n in enumerate(names):
            per[n].append(evs[s][i].elapsed_time(evs[s][i + 1]))
    avg_us = {n: 1e3 * sum(v) / len(v) for n, v in per.items()}

    fp4, lowrank, lora = layer_flops(M, K, N, r, R)
    total = fp4 + lowrank + lora
    tflops = total / (ms_per_step * 1e-3) / 1e12

    gemm = max(("gemm_fwd", "gemm_bwd"), key=lambda n: avg_us[n])
    gemm_flops = 2.0 * M * N * K
    achieved = gemm_flops / (avg_us[gemm] * 1e-6) / 1e12
    quant_bytes = M * K * (2 + 0.5 + 1 / 32) + M * R * 4 + K * R * 2
    qdy_bytes = M * N * (2 + 0.5 + 1 / 32) + M * R * 4 + N * R * 2
    lora_bytes = 2.0 * M * (K + N) + 2 * M * r * 4 + 4.0 * r * (K + N)

    out = {
        "metric": "fused W4A4 linear fwd+bwd TFLOP/s at FLUX 1024^2 shapes; % MXFP4 MFMA peak",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "mxfp4",
        "data": "synthetic",
        "config": {"workload": "FLUX.1-dev attention QKV linear, batch 1 at 1024^2 (%s)" % shape.name,
                   "M": M, "K": K, "N": N, "lora_rank": r, "stabilizer_rank": rs,
                   "outputs": "Y, dX bf16; dA, dB fp32", "parallelism": "single GPU"},
        "pct_mxfp4_peak": round(100.0 * tflops / MXFP4_PEAK_TFLOPS, 2),
        "roofline": {"bound": "mfma", "kernel": "ft::k_gemm_fp4_pipe<%s> (%s)" % (("true, false", "backward-input") if gemm == "gemm_bwd" else ("false, false", "forward")),
                     "achieved": round(achieved, 1), "peak": MXFP4_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / MXFP4_PEAK_TFLOPS, 4),
                     "traffic": measured_traffic("bwd" if gemm == "gemm_bwd" else "fwd"),
                     "per_launch_flops": gemm_flops, "avg_launch_us": round(avg_us[gemm], 2)},
        "kernels_us": {n: round(v, 2) for n, v in avg_us.items()},
        "kernels_frac": {
            "gemm_fwd_mxfp4": round(gemm_flops / (avg_us["gemm_fwd"] * 1e-6) / 1e12 / MXFP4_PEAK_TFLOPS, 4),
            "gemm_bwd_mxfp4": round(gemm_flops / (avg_us["gemm_bwd"] * 1e-6) / 1e12 / MXFP4_PEAK_TFLOPS, 4),
            "quantize_x_hbm": round(quant_bytes / (avg_us["quantize_x"] * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "quantize_dy_hbm": round(qdy_bytes / (avg_us["quantize_dy"] * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "lora_grads_hbm": round(lora_bytes / (avg_us["lora_grads"] * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
        },
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(d, shape, args.cpu_rows)
    print(json.dumps(out), flush=True)


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
