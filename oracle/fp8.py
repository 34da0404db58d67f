"""FP8 (E4M3) quantization by definition, float64.

The paper's deployment quantizes to FP8 E4M3 on its GPUs (section 3.2, Appendix D.2);
this is the reading used for the FP8 path here:

* E4M3 (the OCP 8-bit float with 4 exponent bits, bias 7, 3 mantissa bits, no
  infinities): normal values (1 + m/8) 2^(e-7) for e = 1..15 (m = 0..6 when e = 15,
  largest 448), subnormals m/8 2^-6, round to nearest, ties to the even mantissa,
  values beyond 448 in magnitude saturate to +-448;
* activations are quantized per row (per token) with scale = max|row| / 448, weights
  per output channel the same way; a zero row gets scale 1;
* an FP8 GEMM computes sum_k q_a[m][k] q_w[n][k] exactly and multiplies by
  scale_a[m] scale_w[n];
* attention in FP8 (the paper quantizes QKV and the softmax): q and k in 32-element
  blocks along the head dimension, each block with its own power-of-two scale 2^e
  (an 8-bit biased exponent, as the OCP microscaling formats define it), e the
  smallest integer with max|block| <= 448 * 2^e, so no element saturates; v with one
  scale per tensor, code = E4M3(x * (1 / scale)) with the reciprocal and the product
  rounded to fp32;
* the same block rule over 64 consecutive elements of a row for a projection input
  that a producer writes already quantized (the FFN's hidden activations): the FP8
  GEMM then computes sum_k q_a[m][k] 2^e(m, k/64) q_w[n][k] exactly, times scale_w[n].
"""
import numpy as np

E4M3_MAX = 448.0


def e4m3_values():
    """All 127 non-negative finite E4M3 values in increasing order (code 0x00..0x7E)."""
    vals = [m / 8 * 2.0 ** -6 for m in range(8)]
    for e in range(1, 16):
        for m in range(8):
            if e == 15 and m == 7:
                continue  # 0x7F is NaN
            vals.append((1 + m / 8) * 2.0 ** (e - 7))
    return np.array(vals)


_VALS = e4m3_values()


def round_e4m3(x):
    """Nearest E4M3 value to each element (ties to the even code), saturating at 448."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), E4M3_MAX)
    i = np.searchsorted(_VALS, a)              # first grid value >= a
    i = np.clip(i, 1, len(_VALS) - 1)
    lo, hi = _VALS[i - 1], _VALS[i]
    pick_hi = (hi - a < a - lo) | ((hi - a == a - lo) & (i % 2 == 0))  # even code wins a tie
    r = np.where(pick_hi, hi, lo)
    r = np.where(a == 0, 0.0, r)
    return np.copysign(r, x)


def quantize_rows(x):
    """Per-row E4M3 quantization: returns (q, scale) with q = round_e4m3(x / scale) and
    scale = max|row| / 448 (1 for an all-zero row); x ~ q * scale."""
    x = np.asarray(x, dtype=np.float64)
    amax = np.max(np.abs(x), axis=-1)
    scale = np.where(amax > 0, amax / E4M3_MAX, 1.0)
    return round_e4m3(x / scale[..., None]), scale


def fp8_linear(q_a, s_a, q_w, s_w, bias=None):
    """y[m][n] = (sum_k q_a[m][k] q_w[n][k]) s_a[m] s_w[n] + bias[n]."""
    y = (q_a @ q_w.T) * s_a[..., None] * s_w
    return y if bias is None else y + bias


MX_BLOCK = 32
MX_EMIN, MX_EMAX = -127, 127   # exponent range of the 8-bit biased scale (bias 127)


def mx_exponent(amax):
    """Shared exponent of each block with maximum magnitude amax: the smallest integer e
    with amax <= 448 * 2^e, clamped to [-127, 127]; 0 for an all-zero block."""
    amax = np.asarray(amax, dtype=np.float64)
    _, E = np.frexp(amax)              # amax = f 2^E, 0.5 <= f < 1, so 2^(E-1) <= amax < 2^E
    e = E.astype(np.int64) - 1 - 8     # amax / 2^e in [256, 512)
    e = np.where(amax > E4M3_MAX * np.ldexp(1.0, e), e + 1, e)
    e = np.clip(e, MX_EMIN, MX_EMAX)
    return np.where(amax == 0, 0, e)


def quantize_mx(x, block=MX_BLOCK):
    """Block quantization along the last axis (length a multiple of block): returns
    (q, e) with e [..., n/block] the block exponents and q the E4M3 values of x / 2^e."""
    x = np.asarray(x, dtype=np.float64)
    blocks = x.reshape(x.shape[:-1] + (x.shape[-1] // block, block))
    e = mx_exponent(np.max(np.abs(blocks), axis=-1))
    q = round_e4m3(blocks * 2.0 ** (-e[..., None].astype(np.float64)))
    return q.reshape(x.shape), e


def decode_mx(q, e, block=MX_BLOCK):
    """x ~ q * 2^e with each exponent applied to its block of consecutive elements."""
    return np.asarray(q, dtype=np.float64) * np.repeat(2.0 ** np.asarray(e, dtype=np.float64), block, axis=-1)


def quantize_scaled(x, scale):
    """One-scale E4M3 quantization evaluated in fp32: round_e4m3(fp32(x * fp32(1/scale)))."""
    inv = np.float32(1.0) / np.float32(scale)
    y = np.asarray(x, dtype=np.float32) * inv
    return round_e4m3(y.astype(np.float64))
