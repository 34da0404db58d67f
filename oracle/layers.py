"""Token-wise layers of the DiT block, float64.

The paper names LayerNorm only in passing (Appendix D.2, where LayerNorm and RoPE
are kept in higher precision); AdaLN modulation, the tanh-GELU FFN and the
sinusoidal timestep embedding are the Wan-style block the backbone inherits
(section 4.1).  Their exact forms are readings, stated with each function.
"""
import numpy as np


def linear(x, w, b=None):
    """PyTorch-style Linear: y = x W^T + b, with W stored [out][in]."""
    y = np.matmul(x, np.swapaxes(w, -1, -2))
    if b is not None:
        y = y + b
    return y


def layernorm(x, eps, gamma=None, beta=None):
    """LayerNorm over the last axis: (x - mean) / sqrt(var + eps), var biased (/n).
    Optional elementwise affine gamma, beta."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    y = (x - mu) / np.sqrt(var + eps)
    if gamma is not None:
        y = y * gamma
    if beta is not None:
        y = y + beta
    return y


def modulate(x, shift, scale, eps):
    """AdaLN: affine-free LayerNorm, then scaled by (1 + scale) and shifted."""
    return layernorm(x, eps) * (1.0 + scale) + shift


def gelu_tanh(u):
    """tanh approximation of GELU (Hendrycks & Gimpel, 2016)."""
    return 0.5 * u * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (u + 0.044715 * u ** 3)))


def silu(u):
    """x * sigmoid(x)."""
    with np.errstate(over="ignore"):
        return u / (1.0 + np.exp(-u))


def timestep_sinusoid(t, dim=256, t_scale=1000.0, base=10000.0):
    """Sinusoidal embedding of the per-sample timestep t (the t argument of the
    velocity call in Algorithm 2): [cos(s*w_k), sin(s*w_k)] for k < dim/2 with
    s = t_scale * t and w_k = base^(-k/(dim/2))."""
    half = dim // 2
    omega = base ** (-np.arange(half, dtype=np.float64) / half)
    arg = t_scale * np.asarray(t, dtype=np.float64)[:, None] * omega[None, :]
    return np.concatenate([np.cos(arg), np.sin(arg)], axis=-1)
