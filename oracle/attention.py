"""Block-causal softmax attention, float64, by its plain definition.

Rule (section 3.1, Model Inference; Appendix C, Figure 10b): a query of chunk i sees
every key of chunks <= i — the cached, clean earlier chunks and its own chunk —
and nothing later.  Inside a chunk attention is bidirectional.
"""
import numpy as np


def attention(q, k, v, q_chunk, k_chunk, scale=None):
    """q: (Lq, H, Dh); k, v: (Lk, H, Dh); q_chunk (Lq,), k_chunk (Lk,) chunk ids.
    o[i] = sum_j softmax_j(q_i . k_j * scale) v_j over visible j (k_chunk[j] <= q_chunk[i]).
    scale defaults to 1/sqrt(Dh).  A query that sees no key is an error."""
    Lq, H, Dh = q.shape
    scale = 1.0 / np.sqrt(Dh) if scale is None else scale
    visible = np.asarray(k_chunk)[None, :] <= np.asarray(q_chunk)[:, None]
    if Lq and not visible.any(axis=1).all():
        raise ValueError("a query row sees no key")
    o = np.empty((Lq, H, v.shape[-1]), dtype=np.float64)
    for h in range(H):
        s = np.matmul(q[:, h, :], k[:, h, :].T) * scale
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        o[:, h, :] = np.matmul(p, v[:, h, :])
    return o
