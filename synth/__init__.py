"""Seeded synthetic inputs shared by the oracle-side tests and the GPU-side tests.

This module holds no arithmetic of the method: it only draws random numbers, rounds
them to the storage types (bf16 round-to-nearest-even, fp32) and describes the
workload shapes.  Both the fp64 oracle and the HIP path consume what it returns;
neither is imported here.

Every tensor comes from its own seeded stream
``Generator(PCG64(SeedSequence([cfg_seed, tensor_id, layer])))`` so a test can
regenerate one layer at a time without holding a whole 40-layer model in host RAM.
"""
from __future__ import annotations

import concurrent.futures
import os

import numpy as np

from .workloads import WORKLOADS, Workload  # noqa: F401

# Stable tensor ids: changing one changes every seeded input that uses it.
TENSOR_IDS = {
    # activations / inputs
    "x": 1, "e0": 2, "ctx": 3, "text": 4, "t": 5, "z_t": 6, "a_t": 7,
    "q": 8, "k": 9, "v": 10, "k_cache": 11, "v_cache": 12, "o_init": 13,
    "pos_perm": 14, "probe": 15, "z_clean": 16, "t_action": 17,
    # per-block weights
    "w_qkv": 20, "b_qkv": 21, "w_o": 22, "b_o": 23, "w_cq": 24, "b_cq": 25,
    "w_ckv": 26, "b_ckv": 27, "w_co": 28, "b_co": 29, "w_f1": 30, "b_f1": 31,
    "w_f2": 32, "b_f2": 33, "mod6": 34, "lnc_gamma": 35, "lnc_beta": 36,
    # model-level weights
    "w_t1": 40, "b_t1": 41, "w_t2": 42, "b_t2": 43, "w_t6": 44, "b_t6": 45,
    "w_x1": 46, "b_x1": 47, "w_x2": 48, "b_x2": 49, "w_patch": 50, "b_patch": 51,
    "w_ain": 52, "b_ain": 53, "w_hv": 54, "b_hv": 55, "w_ha": 56, "b_ha": 57,
    "head_mod2": 58,
}

WEIGHT_STD = 0.02


def rng(cfg_seed: int, tensor: str, layer: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [int(cfg_seed), TENSOR_IDS[tensor], int(layer)])))


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round to bfloat16 (round-to-nearest-even) and return the raw uint16 bits."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32)
    nan = np.isnan(f)
    # u + 0x7FFF + lsb cannot wrap for non-NaN inputs (NaNs are fixed up below)
    r = ((u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) >> np.uint32(16)).astype(np.uint16)
    if nan.any():
        r[nan] = 0x7FC0
    return r


def bf16_from_bits(bits: np.ndarray) -> np.ndarray:
    """Widen raw bfloat16 bits to float64 (exact)."""
    u = bits.astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Values of ``a`` after bf16 RNE rounding, as float64."""
    return bf16_from_bits(bf16_bits(a))


def round_f32(a: np.ndarray) -> np.ndarray:
    return np.asarray(a, dtype=np.float32).astype(np.float64)


class Tensor:
    """A seeded input in its storage type: ``bits`` (uint16 for bf16 / float32 array)
    and ``f64`` (exact float64 widening, what the oracle consumes)."""

    __slots__ = ("dtype", "data", "f64")

    def __init__(self, dtype: str, data: np.ndarray):
        self.dtype = dtype
        self.data = data
        self.f64 = bf16_from_bits(data) if dtype == "bf16" else data.astype(np.float64)

    @property
    def shape(self):
        return self.data.shape


def normal(cfg_seed: int, tensor: str, shape, std: float = 1.0, layer: int = 0,
           dtype: str = "bf16") -> Tensor:
    """N(0, std^2) draws (float32 ziggurat), stored as bf16 (RNE) or fp32."""
    g = rng(cfg_seed, tensor, layer)
    if std:
        a = g.standard_normal(size=shape, dtype=np.float32)
        if std != 1.0:
            a *= np.float32(std)
    else:
        a = np.zeros(shape, np.float32)
    if dtype == "bf16":
        return Tensor("bf16", bf16_bits(a))
    return Tensor("f32", a)


def device_normal(cfg_seed: int, tensor: str, shape, std: float = 1.0, layer: int = 0, dtype: str = "bf16"):
    """N(0, std^2) drawn on the GPU from a seeded stream (torch's generator seeded
    from SeedSequence([cfg_seed, tensor_id, layer])), stored as bf16 (RNE) or fp32, for
    inputs too large to draw on the host in a test's time (a 65744-key cache is 337M
    values per sample).  Both sides read the same device tensor: the oracle gets its
    host copy."""
    import torch
    seed = int(np.random.SeedSequence([int(cfg_seed), TENSOR_IDS[tensor], int(layer)]).generate_state(1,
                                                                                                   np.uint64)[0])
    g = torch.Generator(device="cuda")
    g.manual_seed(seed & 0x7FFFFFFFFFFFFFFF)
    a = torch.randn(shape, generator=g, device="cuda", dtype=torch.float32) * std
    return a.to(torch.bfloat16) if dtype == "bf16" else a


def zeros(shape, dtype: str = "f32") -> Tensor:
    if dtype == "bf16":
        return Tensor("bf16", np.zeros(shape, np.uint16))
    return Tensor("f32", np.zeros(shape, np.float32))


def uniform(cfg_seed: int, tensor: str, shape, layer: int = 0) -> Tensor:
    g = rng(cfg_seed, tensor, layer)
    return Tensor("f32", g.random(size=shape, dtype=np.float64).astype(np.float32))


# ---------------------------------------------------------------------------------
# Model parameters.  Matrices are bf16 in [out][in] layout, vectors fp32; biases are
# zero unless ``bias_std`` is given (tests use non-zero biases to exercise epilogues).
# ---------------------------------------------------------------------------------

def _draw_all(jobs: dict) -> dict:
    """Draw several seeded tensors at once: name -> (normal's positional args, dtype).
    Every tensor has its own stream, so drawing them on threads (numpy releases the GIL
    while it fills and rounds large arrays) gives the same values as one by one."""
    workers = max(1, min(len(jobs), 8, len(os.sched_getaffinity(0))))
    with concurrent.futures.ThreadPoolExecutor(workers) as ex:
        futs = {k: ex.submit(normal, *args, dtype=dt) for k, (args, dt) in jobs.items()}
        return {k: f.result() for k, f in futs.items()}


def block_params(wl: "Workload", layer: int, bias_std: float = 0.0,
                 mod_std: float = WEIGHT_STD, seed: int | None = None) -> dict:
    s = wl.seed if seed is None else seed
    d, F = wl.d, wl.ffn
    jobs = {
        "w_qkv": ((s, "w_qkv", (3 * d, d), WEIGHT_STD, layer), "bf16"),
        "w_o": ((s, "w_o", (d, d), WEIGHT_STD, layer), "bf16"),
        "w_cq": ((s, "w_cq", (d, d), WEIGHT_STD, layer), "bf16"),
        "w_ckv": ((s, "w_ckv", (2 * d, d), WEIGHT_STD, layer), "bf16"),
        "w_co": ((s, "w_co", (d, d), WEIGHT_STD, layer), "bf16"),
        "w_f1": ((s, "w_f1", (F, d), WEIGHT_STD, layer), "bf16"),
        "w_f2": ((s, "w_f2", (d, F), WEIGHT_STD, layer), "bf16"),
        "mod6": ((s, "mod6", (6, d), mod_std, layer), "f32"),
    }
    p = _draw_all(jobs)
    p["lnc_gamma"] = Tensor("f32", np.ones(d, np.float32))
    p["lnc_beta"] = zeros((d,))
    for b, n in (("b_qkv", 3 * d), ("b_o", d), ("b_cq", d), ("b_ckv", 2 * d),
                 ("b_co", d), ("b_f1", F), ("b_f2", d)):
        p[b] = normal(s, b, (n,), bias_std, layer, dtype="f32") if bias_std else zeros((n,))
    return p


def model_params(wl: "Workload", bias_std: float = 0.0, seed: int | None = None) -> dict:
    s = wl.seed if seed is None else seed
    d = wl.d
    p = _draw_all({
        "w_t1": ((s, "w_t1", (d, wl.freq_dim), WEIGHT_STD), "bf16"),
        "w_t2": ((s, "w_t2", (d, d), WEIGHT_STD), "bf16"),
        "w_t6": ((s, "w_t6", (6 * d, d), WEIGHT_STD), "bf16"),
        "w_x1": ((s, "w_x1", (d, wl.text_dim), WEIGHT_STD), "bf16"),
        "w_x2": ((s, "w_x2", (d, d), WEIGHT_STD), "bf16"),
        "w_patch": ((s, "w_patch", (d, wl.patch_dim), WEIGHT_STD), "bf16"),
        "w_ain": ((s, "w_ain", (d, wl.act_dim), WEIGHT_STD), "bf16"),
        "w_hv": ((s, "w_hv", (wl.patch_dim, d), WEIGHT_STD), "bf16"),
        "w_ha": ((s, "w_ha", (wl.act_dim, d), WEIGHT_STD), "bf16"),
        "head_mod2": ((s, "head_mod2", (2, d), WEIGHT_STD), "f32"),
    })
    for b, n in (("b_t1", d), ("b_t2", d), ("b_t6", 6 * d), ("b_x1", d), ("b_x2", d),
                 ("b_patch", d), ("b_ain", d), ("b_hv", wl.patch_dim), ("b_ha", wl.act_dim)):
        p[b] = normal(s, b, (n,), bias_std, dtype="f32") if bias_std else zeros((n,))
    return p


def kv_cache(wl: "Workload", layer: int, B: int | None = None, seed: int | None = None):
    """Cached K (stored after RoPE) and V of the earlier chunks: N(0,1) bf16,
    shape (B, n_cached_rows, H, Dh)."""
    s = wl.seed if seed is None else seed
    B = wl.B if B is None else B
    shape = (B, wl.cache_rows, wl.H, wl.Dh)
    kv = _draw_all({"k": ((s, "k_cache", shape, 1.0, layer), "bf16"), "v": ((s, "v_cache", shape, 1.0, layer), "bf16")})
    return kv["k"], kv["v"]
