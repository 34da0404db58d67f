"""The five synthetic workloads, named by what they are.

Shapes follow the paper's chunking (K=2 latent frames per chunk, up to four cached
chunks; Appendix C) and a Wan-style 14B DiT backbone (d=5120, 40 heads of 128,
FFN 13824, 40 blocks; section 4.1 names the Wan2.1-I2V-14B initialisation).  The
paper prints no resolution or token counts; the grids below (30x52 and, for three
views tiled along the width as in section 3.1, 30x156) stand in for its 480P video.
"""
from __future__ import annotations

import dataclasses


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    B: int = 1
    d: int = 5120
    H: int = 40
    Dh: int = 128
    ffn: int = 13824
    n_layers: int = 40
    latent_ch: int = 16
    F: int = 2            # latent frames per chunk (K in the paper)
    Hl: int = 60          # latent height
    Wl: int = 104         # latent width (all views tiled)
    A: int = 32           # action tokens per chunk
    act_dim: int = 16
    n_cached: int = 2     # earlier chunks held in the KV cache
    Lc: int = 512         # text tokens
    text_dim: int = 4096
    freq_dim: int = 256
    eps: float = 1e-6
    mod_std: float = 0.02  # std of the per-block modulation table

    @property
    def Hg(self):
        return self.Hl // 2

    @property
    def Wg(self):
        return self.Wl // 2

    @property
    def Lv(self):
        return self.F * self.Hg * self.Wg

    @property
    def L(self):
        return self.Lv + self.A

    @property
    def cache_rows(self):
        return self.n_cached * self.L

    @property
    def Lk(self):
        return self.cache_rows + self.L

    @property
    def Lcap(self):
        return self.Lk

    @property
    def patch_dim(self):
        return self.latent_ch * 1 * 2 * 2

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    # algorithmic flop counts (2*M*N*K per GEMM; 4*Dh per visible (q,k) pair)
    def block_flops(self, cross_kv: bool = True) -> dict:
        M, d, F, Lc, B = self.B * self.L, self.d, self.ffn, self.Lc, self.B
        f = {
            "qkv": 2 * M * d * 3 * d,
            "o": 2 * M * d * d,
            "cq": 2 * M * d * d,
            "co": 2 * M * d * d,
            "ffn1": 2 * M * d * F,
            "ffn2": 2 * M * F * d,
            "self_attn": 4 * self.H * self.Dh * M * self.Lk,
            "cross_attn": 4 * self.H * self.Dh * M * Lc,
        }
        if cross_kv:
            f["ckv"] = 2 * B * Lc * d * 2 * d
        return f

    def step_flops(self, cross_kv: bool = True, text_proj: bool = True) -> float:
        per_block = sum(self.block_flops(cross_kv).values())
        total = self.n_layers * per_block
        M, d = self.B * self.L, self.d
        total += 2 * self.B * self.Lv * self.patch_dim * d + 2 * self.B * self.A * self.act_dim * d
        total += 2 * M * d * self.patch_dim  # head (upper bound: video head over all rows)
        if text_proj:
            total += 2 * self.B * self.Lc * (self.text_dim * d + d * d)
        return float(total)


WORKLOADS = {
    # one small block: d=512, 8 heads of 64, FFN 2048, 2x8x8 video + 16 action tokens,
    # no cache, 32 text tokens of width 512, modulation vector N(0,1)
    "block_d512": Workload("block_d512", seed=0, d=512, H=8, Dh=64, ffn=2048, n_layers=1,
                           Hl=16, Wl=16, A=16, n_cached=0, Lc=32, text_dim=512, mod_std=1.0),
    # block-causal attention alone: 40x128 heads, 3152 queries, 2 cached chunks (9456 keys)
    "attn_q3152_k9456": Workload("attn_q3152_k9456", seed=1, n_layers=1, n_cached=2),
    # one 14B-class block with a 2-chunk cache and 512x4096 text
    "block_14b": Workload("block_14b", seed=2, n_layers=1, n_cached=2),
    # full 40-block denoising step, 4 cached chunks per layer
    "step_14b": Workload("step_14b", seed=3, n_layers=40, n_cached=4),
    # 40-block step at batch 2, three views tiled along the width, 6 cached chunks
    "step_14b_b2_3view": Workload("step_14b_b2_3view", seed=4, B=2, n_layers=40,
                                  Wl=312, n_cached=6),
}
