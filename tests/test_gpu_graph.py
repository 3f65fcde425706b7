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


@pytest.mark.parametrize("M,Dm,F", [(1000, 1024, 4096)])
def test_mlp_pair_step_replays_in_hip_graph(M, Dm, F):
    """The MLP pair (Sec. 3.3, MLP fusion): FC1 with the GELU / quantize /
    projection epilogue, FC2's forward, FC2's backward-input with the dGELU
    epilogue, FC1's backward-input and both adapter gradients, captured and
    replayed; the fused epilogues' projection partials go through their
    workspaces and the reduction kernel, with no memset in the graph."""
    r, rs = 32, 32
    R = r + rs
    bf, f32, u8 = torch.bfloat16, torch.float32, torch.uint8
    g = torch.Generator(device=DEV)
    g.manual_seed(17)
    nrm = lambda sh, sd: (torch.randn(sh, generator=g, device=DEV) * sd).to(bf)
    X, dY = nrm((M, Dm), 1.0), nrm((M, Dm), 1e-3)
    w1q, w1s, _ = _lib.ft_quantize_blockwise(nrm((F, Dm), 0.02), block_rows=32)
    w2q, w2s, _ = _lib.ft_quantize_blockwise(nrm((Dm, F), 0.02), block_rows=32)
    D1, U1, b1 = nrm((Dm, R), 0.01), nrm((R, F), 0.01), nrm((F,), 0.02)
    D2, U2, b2 = nrm((F, R), 0.01), nrm((R, Dm), 0.01), nrm((Dm,), 0.02)
    e = lambda sh, dt: torch.empty(sh, dtype=dt, device=DEV)
    xq, xs, gq, gs = e((M, Dm // 2), u8), e((M, Dm // 32), u8), e((M, Dm // 2), u8), e((M, Dm // 32), u8)
    P1, P2, Qp1, Qp2 = (e((M, R), f32) for _ in range(4))
    z, h, dz = (e((M, F), bf) for _ in range(3))
    hq, hs, dzq, dzs = e((M, F // 2), u8), e((M, F // 32), u8), e((M, F // 2), u8), e((M, F // 32), u8)
    Y, dX = e((M, Dm), bf), e((M, Dm), bf)
    dA1, dB1, dA2, dB2 = e((Dm, r), f32), e((r, F), f32), e((F, r), f32), e((r, Dm), f32)
    ws = lambda n: e((max(16, n),), u8)
    wx = ws(_lib.ft_quantize_workspace_size(M, Dm, 1, R, _lib.FT_PROJ_COLS_BY_R))
    wd = ws(_lib.ft_quantize_workspace_size(M, Dm, 1, R, _lib.FT_PROJ_R_BY_COLS))
    wg, wdg = ws(_lib.ft_linear_fwd_gelu_workspace_size(M, F, R)), ws(_lib.ft_linear_bwd_input_dgelu_workspace_size(M, F, R))
    wl1, wl2 = ws(_lib.ft_lora_grads_workspace_size(M, Dm, F, R, r)), ws(_lib.ft_lora_grads_workspace_size(M, F, Dm, R, r))
    assert wg.numel() > 16 and wdg.numel() > 16   # several column tiles: partials and their reduction
    outs = (xq, xs, P1, z, h, hq, hs, P2, Y, gq, gs, Qp2, dz, dzq, dzs, Qp1, dX, dA1, dB1, dA2, dB2)

    def step():
        _lib.ft_quantize_blockwise(X, proj=D1, codes=xq, scales=xs, proj_out=P1, workspace=wx)
        _lib.ft_linear_fwd_gelu(xq, xs, w1q, w1s, Dm, P1, U1, b1, D2=D2, z=z, h=h, hq=hq, hs=hs, P2=P2, workspace=wg)
        _lib.ft_linear_fwd(hq, hs, w2q, w2s, F, P2, U2, b2, y=Y)
        _lib.ft_quantize_blockwise(dY, proj=U2, proj_layout=_lib.FT_PROJ_R_BY_COLS, codes=gq, scales=gs,
                                   proj_out=Qp2, workspace=wd)
        _lib.ft_linear_bwd_input_dgelu(gq, gs, w2q, w2s, F, z, Qp2, D2, U1=U1, dz=dz, dzq=dzq, dzs=dzs, Qp1=Qp1,
                                       workspace=wdg)
        _lib.ft_linear_bwd_input(dzq, dzs, w1q, w1s, Dm, Qp1, D1, dx=dX)
        _lib.ft_lora_grads(h, dY, P2, Qp2, r, col0=rs, dA=dA2, dB=dB2, workspace=wl2)
        _lib.ft_lora_grads(X, dz, P1, Qp1, r, col0=rs, dA=dA1, dB=dB1, workspace=wl1)

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

    names = ("xq", "xs", "P1", "z", "h", "hq", "hs", "P2", "Y", "gq", "gs", "Qp2", "dz", "dzq", "dzs", "Qp1", "dX",
             "dA1", "dB1", "dA2", "dB2")
    for rep in range(3):
        for t in outs + (wg, wdg):   # eager work between replays: scribble over every output and partial
            t.view(u8).fill_(0xA5)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        print("mlp graph replay", rep, (M, Dm, F), flush=True)
        for name, a, b in zip(names, outs, ref):
            assert torch.equal(a.view(u8), b.view(u8)), "%s differs on replay %d" % (name, rep)
