"""libwamdit: one denoising step of a block-causal video/action DiT on MI355X (gfx950).

The compute path is the HIP library ``libwamdit.so`` (hand-written gfx950 kernels
behind a C ABI declared in ``include/wamdit.h``); this package is its ctypes binding.
"""
from .binding import *  # noqa: F401,F403
from .binding import (lib, WamError, make_chunks, cached_chunks, append_chunks, make_dims,  # noqa: F401
                      make_model, make_denoise_params, make_block_fp8)
