"""The C ABI library loads, exports every entry point its header declares, and
rejects invalid arguments before launching anything (CPU only: none of these
calls reaches a kernel launch)."""
import ctypes
import os
import re

import pytest

from paper_2607_05711_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fourtune.h")

def _gpu_visible():
    import torch
    return torch.cuda.is_available()


# The validation tests pass fake device addresses that a correct library never
# dereferences; they run only where no GPU is visible, so that a regression in
# validation can never turn into a launch on bogus pointers.
pytestmark = [pytest.mark.skipif(not os.path.exists(_lib.LIB_PATH), reason="libfourtune.so not built"),
              pytest.mark.skipif(_gpu_visible(), reason="host-logic checks with fake pointers run without a GPU")]


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ft_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("ft_quantize_blockwise", "ft_linear_fwd", "ft_linear_bwd_input", "ft_lora_grads",
              "ft_linear_fwd_gelu", "ft_linear_bwd_input_dgelu", "ft_quantize_workspace_size",
              "ft_lora_grads_workspace_size", "ft_status_string", "ft_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(_lib.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings():
    L = _lib.load()
    for code, text in [(0, "ok"), (1, "null pointer"), (2, "invalid shape"), (3, "misaligned pointer"),
                       (4, "unsupported argument"), (5, "HIP runtime error")]:
        assert _lib.status_string(code) == text
    assert _lib.status_string(99) == "unknown status"
    assert L.ft_last_error() is not None


ALIGNED = ctypes.c_void_p(0x100000)      # never dereferenced: validation fails first
ALIGNED2 = ctypes.c_void_p(0x200000)
MISALIGNED = ctypes.c_void_p(0x100008)
NULL = None


def q(src, rows, cols, block_rows, codes, scales, proj=NULL, R=0, layout=0, out=NULL, ws=NULL, wsb=0):
    return _lib.load().ft_quantize_blockwise(src, rows, cols, block_rows, codes, scales, proj, R, layout, out,
                                             ws, wsb, NULL)


def test_quantize_validation():
    assert q(ALIGNED, 4, 48, 1, ALIGNED, ALIGNED) == _lib.FT_ERR_SHAPE          # cols % 32
    assert q(ALIGNED, -1, 64, 1, ALIGNED, ALIGNED) == _lib.FT_ERR_SHAPE
    assert q(ALIGNED, 48, 64, 32, ALIGNED, ALIGNED) == _lib.FT_ERR_SHAPE        # rows % 32 for tiles
    assert q(ALIGNED, 4, 64, 2, ALIGNED, ALIGNED) == _lib.FT_ERR_UNSUPPORTED
    assert q(NULL, 4, 64, 1, ALIGNED, ALIGNED) == _lib.FT_ERR_NULL
    assert q(MISALIGNED, 4, 64, 1, ALIGNED, ALIGNED) == _lib.FT_ERR_ALIGN
    assert q(ALIGNED, 4, 64, 1, ALIGNED, MISALIGNED) == _lib.FT_ERR_ALIGN      # scales too
    assert q(ALIGNED, 64, 64, 32, ALIGNED, ctypes.c_void_p(0x100004)) == _lib.FT_ERR_ALIGN
    assert q(ALIGNED, 4, 64, 1, ALIGNED, ALIGNED, ALIGNED2, 20, 0, ALIGNED2) == _lib.FT_ERR_UNSUPPORTED
    assert q(ALIGNED, 4, 64, 1, ALIGNED, ALIGNED, ALIGNED2, 144, 0, ALIGNED2) == _lib.FT_ERR_UNSUPPORTED
    assert q(ALIGNED, 4, 64, 1, ALIGNED, ALIGNED, ALIGNED2, 32, 0, NULL) == _lib.FT_ERR_NULL
    assert q(ALIGNED, 4, 64, 1, ALIGNED, ALIGNED, ALIGNED2, 32, 7, ALIGNED2) == _lib.FT_ERR_UNSUPPORTED
    assert q(ALIGNED, 64, 64, 32, ALIGNED, ALIGNED, ALIGNED2, 32, 0, ALIGNED2) == _lib.FT_ERR_UNSUPPORTED
    # empty input is a no-op, even with NULL buffers
    assert q(NULL, 0, 64, 1, NULL, NULL) == _lib.FT_OK
    # a projection over several column chunks needs the workspace the size query reports
    need = _lib.ft_quantize_workspace_size(512, 3072, 1, 64, 0)
    assert need == 12 * 512 * 64 * 4       # 256-column chunks: 384 would leave fewer workgroups than CUs
    assert _lib.ft_quantize_workspace_size(8224, 3072, 1, 64, 0) == 8 * 8224 * 64 * 4     # 384 otherwise
    # the widest chunk that fits LDS (512 for R = 96, 640 for R <= 64) while it still makes a full
    # round of workgroups, else as above
    # long rows: several chunks per workgroup ([cols, R]: up to 6 while 384 workgroups remain, 30 chunks
    # in 6 groups; [R, cols]: up to 4 while 512 remain)
    assert _lib.ft_quantize_workspace_size(18432, 15360, 1, 96, 0) == 6 * 18432 * 96 * 4
    assert _lib.ft_quantize_workspace_size(18432, 21504, 1, 96, 1) == 11 * 18432 * 96 * 4   # [R, cols]: 42 chunks
    assert _lib.ft_quantize_workspace_size(16640, 16384, 1, 64, 1) == 8 * 16640 * 64 * 4    # 22 chunks, 3 per group
    assert _lib.ft_quantize_workspace_size(16640, 16384, 1, 64, 0) == 6 * 16640 * 64 * 4    # 26 chunks, 5 per group
    assert _lib.ft_quantize_workspace_size(4608, 15360, 1, 64, 0) == 24 * 4608 * 64 * 4
    assert _lib.ft_quantize_workspace_size(2304, 10976, 1, 64, 0) == 29 * 2304 * 64 * 4     # 640 would make 162
    assert _lib.ft_quantize_workspace_size(18432, 3072, 1, 96, 0) == 6 * 18432 * 96 * 4
    assert _lib.ft_quantize_workspace_size(4608, 9216, 1, 64, 1) == 12 * 4608 * 64 * 4   # 768 for [R, cols]
    assert _lib.ft_quantize_workspace_size(512, 9216, 1, 64, 1) == 36 * 512 * 64 * 4     # 256: 768 makes 24
    assert _lib.ft_quantize_workspace_size(512, 9216, 1, 96, 1) == 18 * 512 * 96 * 4     # 512 at R = 96
    assert _lib.ft_quantize_workspace_size(512, 256, 1, 64, 0) == 0                      # one chunk: none
    # whole rows per workgroup for [cols, R] (64..256 workgroups of 24 or 32 rows, R <= 64): no partial sums
    assert _lib.ft_quantize_workspace_size(4608, 3072, 1, 64, 0) == 0
    assert _lib.ft_quantize_workspace_size(4608, 15360, 1, 64, 0) > 0                    # rows > 4096: chunks
    assert _lib.ft_quantize_workspace_size(4608, 9216, 1, 64, 1) == 12 * 4608 * 64 * 4   # [R, cols]: chunks
    assert _lib.ft_quantize_workspace_size(4608, 3072, 1, 96, 0) > 0                     # R > 64: chunks
    assert _lib.ft_quantize_workspace_size(4608, 3072, 1, 0, 0) == 0                     # no projection: none
    assert _lib.ft_quantize_workspace_size(4608, 3072, 32, 0, 0) == 0
    big = (ALIGNED, 512, 3072, 1, ALIGNED, ALIGNED, ALIGNED2, 64, 0, ALIGNED2)
    assert q(*big) == _lib.FT_ERR_NULL
    assert q(*big, ws=ALIGNED2, wsb=need - 16) == _lib.FT_ERR_SHAPE
    assert q(*big, ws=MISALIGNED, wsb=need) == _lib.FT_ERR_ALIGN


def test_linear_validation():
    L = _lib.load()
    f = L.ft_linear_fwd
    assert f(ALIGNED, ALIGNED, 8, 48, ALIGNED, ALIGNED, 64, NULL, 0, NULL, NULL, ALIGNED, 0, NULL) == _lib.FT_ERR_SHAPE
    assert f(ALIGNED, ALIGNED, 8, 64, ALIGNED, ALIGNED, 40, NULL, 0, NULL, NULL, ALIGNED, 0, NULL) == _lib.FT_ERR_SHAPE
    assert f(ALIGNED, ALIGNED, 8, 64, ALIGNED, ALIGNED, 64, NULL, 0, NULL, NULL, ALIGNED, 3, NULL) == _lib.FT_ERR_UNSUPPORTED
    assert f(ALIGNED, NULL, 8, 64, ALIGNED, ALIGNED, 64, NULL, 0, NULL, NULL, ALIGNED, 0, NULL) == _lib.FT_ERR_NULL
    assert f(MISALIGNED, ALIGNED, 8, 64, ALIGNED, ALIGNED, 64, NULL, 0, NULL, NULL, ALIGNED, 0, NULL) == _lib.FT_ERR_ALIGN
    # the scale arrays are moved in 4- and 16-byte units: they must be aligned like the rest
    assert f(ALIGNED, MISALIGNED, 8, 64, ALIGNED, ALIGNED, 64, NULL, 0, NULL, NULL, ALIGNED, 0, NULL) == _lib.FT_ERR_ALIGN
    assert f(ALIGNED, ALIGNED, 8, 64, ALIGNED, MISALIGNED, 64, NULL, 0, NULL, NULL, ALIGNED, 0, NULL) == _lib.FT_ERR_ALIGN
    assert f(ALIGNED, ALIGNED, 8, 64, ALIGNED, ALIGNED, 64, ALIGNED2, 32, NULL, NULL, ALIGNED, 0, NULL) == _lib.FT_ERR_NULL
    assert f(ALIGNED, ALIGNED, 8, 64, ALIGNED, ALIGNED, 64, ALIGNED2, 24, ALIGNED2, NULL, ALIGNED, 0, NULL) == _lib.FT_ERR_UNSUPPORTED
    assert f(ALIGNED, ALIGNED, 8, 64, ALIGNED, ALIGNED, 64, NULL, 0, ALIGNED2, NULL, ALIGNED, 0, NULL) == _lib.FT_ERR_UNSUPPORTED
    assert f(ALIGNED, ALIGNED, 8, 0, ALIGNED, ALIGNED, 64, NULL, 0, NULL, NULL, ALIGNED, 0, NULL) == _lib.FT_ERR_SHAPE
    assert f(NULL, NULL, 0, 64, NULL, NULL, 64, NULL, 0, NULL, NULL, NULL, 0, NULL) == _lib.FT_OK
    b = L.ft_linear_bwd_input
    assert b(ALIGNED, ALIGNED, 8, 48, ALIGNED, ALIGNED, 64, NULL, 0, NULL, ALIGNED, 0, NULL) == _lib.FT_ERR_SHAPE
    assert b(ALIGNED, ALIGNED, 8, 64, ALIGNED, ALIGNED, 64, ALIGNED2, 32, NULL, ALIGNED, 0, NULL) == _lib.FT_ERR_NULL
    assert b(ALIGNED, ALIGNED, 8, 64, ALIGNED, ALIGNED, 64, NULL, 0, NULL, MISALIGNED, 1, NULL) == _lib.FT_ERR_ALIGN
    assert b(ALIGNED, MISALIGNED, 8, 64, ALIGNED, ALIGNED, 64, NULL, 0, NULL, ALIGNED, 1, NULL) == _lib.FT_ERR_ALIGN
    assert b(ALIGNED, ALIGNED, 8, 64, ALIGNED, MISALIGNED, 64, NULL, 0, NULL, ALIGNED, 1, NULL) == _lib.FT_ERR_ALIGN
    assert b(NULL, NULL, 0, 64, NULL, NULL, 64, NULL, 0, NULL, NULL, 0, NULL) == _lib.FT_OK


def test_lora_validation():
    f = _lib.load().ft_lora_grads
    args = lambda **kw: [kw.get("x", ALIGNED), kw.get("M", 8), kw.get("K", 64), kw.get("dy", ALIGNED), kw.get("N", 64),
                         kw.get("xa", ALIGNED2), kw.get("dyb", ALIGNED2), kw.get("ld", 32), kw.get("r", 16),
                         kw.get("dA", ALIGNED), kw.get("dB", ALIGNED), kw.get("acc", 0), kw.get("ws", NULL),
                         kw.get("wsb", 0), NULL]
    assert f(*args(r=0)) == _lib.FT_ERR_UNSUPPORTED
    assert f(*args(r=129, ld=132)) == _lib.FT_ERR_UNSUPPORTED
    assert f(*args(ld=8)) == _lib.FT_ERR_SHAPE
    assert f(*args(ld=33)) == _lib.FT_ERR_SHAPE
    assert f(*args(K=40)) == _lib.FT_ERR_SHAPE
    assert f(*args(acc=2)) == _lib.FT_ERR_UNSUPPORTED
    assert f(*args(dA=NULL)) == _lib.FT_ERR_NULL
    assert f(*args(x=NULL)) == _lib.FT_ERR_NULL
    assert f(*args(dy=MISALIGNED)) == _lib.FT_ERR_ALIGN
    assert f(*args(xa=MISALIGNED)) == _lib.FT_ERR_ALIGN
    assert f(*args(dyb=MISALIGNED)) == _lib.FT_ERR_ALIGN
    assert f(*args(N=(1 << 24) + 32)) == _lib.FT_ERR_UNSUPPORTED
    # no output columns at all: nothing to compute (the token-window sizing divides by max(K, N))
    assert f(*args(K=0, N=0)) == _lib.FT_OK
    assert f(*args(K=0, N=0, dA=NULL, dB=NULL, x=NULL, dy=NULL)) == _lib.FT_OK
    assert _lib.ft_lora_grads_workspace_size(4608, 0, 0, 64, 32) == 0
    # token chunks leave partial sums in the workspace
    need = _lib.ft_lora_grads_workspace_size(4608, 3072, 9216, 64, 32)
    assert need > 0 and need % (32 * (3072 + 9216) * 4) == 0
    assert _lib.ft_lora_grads_workspace_size(64, 3072, 9216, 64, 32) == 0        # one 64-row stage: no chunks
    big = dict(M=4608, K=3072, N=9216, ld=64, r=32)
    assert f(*args(**big)) == _lib.FT_ERR_NULL
    assert f(*args(**big, ws=ALIGNED2, wsb=need - 4)) == _lib.FT_ERR_SHAPE
    assert f(*args(**big, ws=MISALIGNED, wsb=need)) == _lib.FT_ERR_ALIGN


def test_mlp_fused_validation():
    L = _lib.load()
    f = L.ft_linear_fwd_gelu
    # xq, xs, M, K, wq, ws, N, P, R, U, bias, z, h, hq, hs, D2, R2, P2, ws, wsb, stream
    base = dict(xq=ALIGNED, xs=ALIGNED, M=8, K=256, wq=ALIGNED, ws=ALIGNED, N=256, P=NULL, R=0, U=NULL, bias=NULL,
                z=ALIGNED, h=ALIGNED, hq=ALIGNED, hs=ALIGNED, D2=NULL, R2=0, P2=NULL, wsp=NULL, wsb=0)
    order = ["xq", "xs", "M", "K", "wq", "ws", "N", "P", "R", "U", "bias", "z", "h", "hq", "hs", "D2", "R2", "P2",
             "wsp", "wsb"]
    call = lambda **kw: f(*[{**base, **kw}[k] for k in order], NULL)
    assert call(K=160) == _lib.FT_ERR_UNSUPPORTED                     # K % 128 != 0: no fused kernel
    assert call(R2=8, D2=ALIGNED2, P2=ALIGNED2) == _lib.FT_ERR_UNSUPPORTED
    assert call(R2=80, D2=ALIGNED2, P2=ALIGNED2) == _lib.FT_ERR_UNSUPPORTED
    assert call(R2=32, D2=ALIGNED2) == _lib.FT_ERR_NULL
    assert call(h=NULL) == _lib.FT_ERR_NULL
    assert call(z=MISALIGNED) == _lib.FT_ERR_ALIGN
    assert call(xs=MISALIGNED) == _lib.FT_ERR_ALIGN
    assert call(hs=MISALIGNED) == _lib.FT_ERR_ALIGN
    need = _lib.ft_linear_fwd_gelu_workspace_size(4608, 12288, 64)
    assert need == 48 * 4608 * 64 * 4                                  # one partial per 256-column tile
    assert _lib.ft_linear_fwd_gelu_workspace_size(4608, 256, 64) == 0  # one tile: written directly
    assert _lib.ft_linear_fwd_gelu_workspace_size(4608, 12288, 0) == 0
    assert call(M=4608, N=12288, R2=64, D2=ALIGNED2, P2=ALIGNED2) == _lib.FT_ERR_NULL
    g = L.ft_linear_bwd_input_dgelu
    base_b = dict(gq=ALIGNED, gs=ALIGNED, M=8, N=256, wq=ALIGNED, ws=ALIGNED, K=256, Qp=NULL, R=0, D=NULL,
                  z=ALIGNED, dz=ALIGNED, dzq=ALIGNED, dzs=ALIGNED, U1=NULL, R1=0, Qp1=NULL, wsp=NULL, wsb=0)
    order_b = ["gq", "gs", "M", "N", "wq", "ws", "K", "Qp", "R", "D", "z", "dz", "dzq", "dzs", "U1", "R1", "Qp1",
               "wsp", "wsb"]
    call_b = lambda **kw: g(*[{**base_b, **kw}[k] for k in order_b], NULL)
    assert call_b(N=160) == _lib.FT_ERR_UNSUPPORTED                   # reduction not a multiple of 128
    assert call_b(K=224) == _lib.FT_ERR_UNSUPPORTED
    assert call_b(z=NULL) == _lib.FT_ERR_NULL
    assert call_b(gs=MISALIGNED) == _lib.FT_ERR_ALIGN
    assert call_b(dzs=MISALIGNED) == _lib.FT_ERR_ALIGN
    assert call_b(R1=48, U1=ALIGNED2) == _lib.FT_ERR_NULL
    assert _lib.ft_linear_bwd_input_dgelu_workspace_size(4608, 12288, 64) == 48 * 4608 * 64 * 4
    assert call_b(M=0) == _lib.FT_OK


def test_load_refuses_a_library_built_from_other_sources(monkeypatch):
    """The binding ties the shared library to the sources in the tree: a
    library whose recorded source hash differs is refused, never loaded."""
    from paper_2607_05711_amd import build
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(build, "source_hash", lambda: "0" * 64)
    with pytest.raises(RuntimeError, match="not built from the sources"):
        _lib.load()


def test_lora_noalloc_validation():
    """The allocation-free adapter-gradient entry point validates like
    ft_lora_grads (no workspace arguments)."""
    f = _lib.load().ft_lora_grads_noalloc
    args = lambda **kw: [kw.get("x", ALIGNED), kw.get("M", 8), kw.get("K", 64), kw.get("dy", ALIGNED), kw.get("N", 64),
                         kw.get("xa", ALIGNED2), kw.get("dyb", ALIGNED2), kw.get("ld", 32), kw.get("r", 16),
                         kw.get("dA", ALIGNED), kw.get("dB", ALIGNED), kw.get("acc", 0), NULL]
    assert f(*args(r=0)) == _lib.FT_ERR_UNSUPPORTED
    assert f(*args(ld=33)) == _lib.FT_ERR_SHAPE
    assert f(*args(K=40)) == _lib.FT_ERR_SHAPE
    assert f(*args(acc=2)) == _lib.FT_ERR_UNSUPPORTED
    assert f(*args(dB=NULL)) == _lib.FT_ERR_NULL
    assert f(*args(xa=MISALIGNED)) == _lib.FT_ERR_ALIGN
    assert f(*args(K=0, N=0, dA=NULL, dB=NULL)) == _lib.FT_OK


def test_quantize_mode_validation():
    """ft_quantize_blockwise_mode rejects unknown options and the combinations
    it does not offer before launching anything."""
    f = _lib.load().ft_quantize_blockwise_mode
    M = _lib.QuantMode
    call = lambda mode, block_rows=1, rows=64: f(ALIGNED, rows, 64, block_rows, ALIGNED, ALIGNED2, NULL, 0, 0,
                                                 NULL, NULL, 0, ctypes.byref(mode) if mode else None, NULL)
    assert call(M(2, 0, 0, 0, 0)) == _lib.FT_ERR_UNSUPPORTED                 # scale rule
    assert call(M(0, 5, 0, 0, 0)) == _lib.FT_ERR_UNSUPPORTED                 # rounding
    assert call(M(0, 0, 0, 0, 2)) == _lib.FT_ERR_UNSUPPORTED                 # scales_per_row
    assert call(M(0, 1, 0, 0, 0), block_rows=32) == _lib.FT_ERR_UNSUPPORTED  # stochastic 32x32
    assert call(M(0, 0, 0, 0, 1), block_rows=1) == _lib.FT_ERR_UNSUPPORTED   # per-row scales of 1x32
    assert call(M(0, 0, 0, 0, 0), rows=-1) == _lib.FT_ERR_SHAPE
    assert f(ALIGNED, 64, 64, 1, ALIGNED, MISALIGNED, NULL, 0, 0, NULL, NULL, 0, None, NULL) == _lib.FT_ERR_ALIGN
    assert f(NULL, 0, 64, 1, NULL, NULL, NULL, 0, 0, NULL, NULL, 0, None, NULL) == _lib.FT_OK


def test_nvfp4_validation():
    L = _lib.load()
    q = L.ft_quantize_nvfp4
    assert q(ALIGNED, 16, 24, 1, ALIGNED, ALIGNED2, ALIGNED, NULL) == _lib.FT_ERR_SHAPE        # cols % 16
    assert q(ALIGNED, 24, 32, 16, ALIGNED, ALIGNED2, ALIGNED, NULL) == _lib.FT_ERR_SHAPE       # rows % 16 for tiles
    assert q(ALIGNED, 16, 32, 8, ALIGNED, ALIGNED2, ALIGNED, NULL) == _lib.FT_ERR_UNSUPPORTED
    assert q(ALIGNED, 16, 32, 1, ALIGNED, ALIGNED2, NULL, NULL) == _lib.FT_ERR_NULL
    assert q(ALIGNED, 16, 32, 1, ALIGNED, MISALIGNED, ALIGNED, NULL) == _lib.FT_ERR_ALIGN
    assert q(NULL, 0, 32, 1, NULL, NULL, NULL, NULL) == _lib.FT_OK
    f = L.ft_linear_fwd_nvfp4
    assert f(ALIGNED, ALIGNED, ALIGNED, 8, 40, ALIGNED, ALIGNED, ALIGNED, 32, ALIGNED2, NULL) == _lib.FT_ERR_SHAPE
    assert f(ALIGNED, ALIGNED, NULL, 8, 32, ALIGNED, ALIGNED, ALIGNED, 32, ALIGNED2, NULL) == _lib.FT_ERR_NULL
    assert f(ALIGNED, ALIGNED, ALIGNED, 8, 0, ALIGNED, ALIGNED, ALIGNED, 32, ALIGNED2, NULL) == _lib.FT_ERR_SHAPE
    b = L.ft_linear_bwd_input_nvfp4
    assert b(ALIGNED, ALIGNED, ALIGNED, 8, 32, ALIGNED, ALIGNED, ALIGNED, 48, MISALIGNED, NULL) == _lib.FT_ERR_ALIGN
    assert b(NULL, NULL, NULL, 0, 32, NULL, NULL, NULL, 48, NULL, NULL) == _lib.FT_OK
