"""MI355X (gfx950) W4A4G4 triple-branch linear layer (FourTune, arXiv 2607.05711).

The compute path is libfourtune.so (hand-written HIP kernels behind the C ABI
in include/fourtune.h); `paper_2607_05711_amd._lib` is its ctypes binding.
Importing this package does not load the library; the binding loads it on
first use and raises if it has not been built.
"""
__all__ = ["ft_quantize_blockwise", "ft_linear_fwd", "ft_linear_bwd_input", "ft_lora_grads",
           "ft_linear_fwd_gelu", "ft_linear_bwd_input_dgelu"]


def __getattr__(name):
    if name in __all__:
        from . import _lib
        return getattr(_lib, name)
    raise AttributeError(name)
