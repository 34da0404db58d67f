"""fp64 CPU oracle for one denoising step of the block-causal video/action DiT.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it.  The product (the HIP library and
its Python binding) never imports, calls or links anything here, and this package
imports nothing from the product.

It is the plain definition of what the hot path computes, in numpy float64 with no
intermediate rounding, written for a reader to check by eye against the paper:

* chunked autoregressive denoising with a KV cache of earlier chunks, and the
  attention rule "the current chunk sees every earlier chunk and itself"
  (section 3.1, Model Inference; Appendix C, Figure 10);
* the velocity call u_theta(x_t; KV, c, t) of the closed-loop inference algorithm
  (Appendix C, Algorithm 2, the denoising-loop forward with update=False), its cache
  update pass (update=True) and the denoising loop around it (solver step, guidance,
  DiT caching);
* the block internals the paper leaves unstated follow fixed readings, stated with
  each function: AdaLN-modulated LayerNorm (shift, scale, gate per branch), 3D RoPE,
  cross-attention to text behind an affine LayerNorm with no gate, tanh-GELU FFN.

Every function is pinned by ``tests/test_oracle_pins.py`` against brute force,
closed forms, invariants and library routines.
"""
from .layers import linear, layernorm, modulate, gelu_tanh, silu, timestep_sinusoid  # noqa: F401
from .rope import rope_split, rope_angles, apply_rope, chunk_positions  # noqa: F401
from .attention import attention  # noqa: F401
from .model import (time_embedding, text_projection, patchify, unpatchify,  # noqa: F401
                    embed, dit_block, head, dit_step, dit_update)
from .denoise import (euler_step, cfg_combine, cosine_similarity, denoise,  # noqa: F401
                      unipc_lambda, unipc_update, unipc_denoise)
from . import fp8  # noqa: F401
