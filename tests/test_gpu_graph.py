"""One whole layer step (fused quantization of X and dY with their
projections, forward GEMM, backward-input GEMM, adapter gradients through the
allocation-free entry point) captured in a HIP graph and replayed: every
replay, with other GPU work and host synchronisation between replays, gives
the same bits as the eager step.  Every output buffer and workspace is
allocated before capture, and the library itself allocates nothing and
records no memset, so the captured launches are the library's kernels only."""
import pytest
import torch

from paper_2607_05711_amd import _lib, gen

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.mark.parametrize("M,K,N", [(1000, 1024, 1536), (4608, 3072, 9216)])
def test_layer_step_replays_in_hip_graph(M, K, N):
    r, rs = 32, 32
    R = r + rs
    shape = gen.custom_shape(M, K, N, r=r, r_s=rs)
    d = gen.layer_inputs_torch(shape, 5, DEV)
    X, dY, D, U, bias = d["X"], d["dY"], d["D"], d["U"], d["bias"]
    wq, ws, _ = _lib.ft_quantize_blockwise(d["W"], block_rows=32)
    bf, f32, u8 = torch.bfloat16, torch.float32, torch.uint8

    # every output and workspace before capture
    xq, xs = torch.empty((M, K // 2), dtype=u8, device=DEV), torch.empty((M, K // 32), dtype=u8, device=DEV)
    gq, gs = torch.empty((M, N // 2), dtype=u8, device=DEV), torch.empty((M, N // 32), dtype=u8, device=DEV)
    P, Qp = torch.empty((M, R), dtype=f32, device=DEV), torch.empty((M, R), dtype=f32, device=DEV)
    y, dx = torch.empty((M, N), dtype=bf, device=DEV), torch.empty((M, K), dtype=bf, device=DEV)
    dA, dB = torch.empty((K, r), dtype=f32, device=DEV), torch.empty((r, N), dtype=f32, device=DEV)
    wsx = torch.empty(max(1, _lib.ft_quantize_workspace_size(M, K, 1, R, _lib.FT_PROJ_COLS_BY_R)), dtype=u8,
                      device=DEV)
    wsg = torch.empty(max(1, _lib.ft_quantize_workspace_size(M, N, 1, R, _lib.FT_PROJ_R_BY_COLS)), dtype=u8,
                      device=DEV)
    outs = (xq, xs, P, y, gq, gs, Qp, dx, dA, dB)

    def step():
        _lib.ft_quantize_blockwise(X, proj=D, codes=xq, scales=xs, proj_out=P, workspace=wsx)
        _lib.ft_linear_fwd(xq, xs, wq, ws, K, P, U, bias, y=y)
        _lib.ft_quantize_blockwise(dY, proj=U, proj_layout=_lib.FT_PROJ_R_BY_COLS, codes=gq, scales=gs,
                                   proj_out=Qp, workspace=wsg)
        _lib.ft_linear_bwd_input(gq, gs, wq, ws, K, Qp, D, dx=dx)
        _lib.ft_lora_grads_noalloc(X, dY, P, Qp, r, col0=rs, dA=dA, dB=dB)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()

    for rep in range(3):
        for t in outs:   # eager work between replays: scribble over every output
            t.view(u8).fill_(0xA5)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        print("graph replay", rep, (M, K, N), flush=True)
        for name, a, b in zip(("xq", "xs", "P", "y", "gq", "gs", "Qp", "dx", "dA", "dB"), outs, ref):
            assert torch.equal(a.view(u8), b.view(u8)), "%s differs on replay %d" % (name, rep)
