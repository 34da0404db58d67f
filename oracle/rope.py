"""3D rotary position embedding over (frame, row, column) positions, float64.

The paper keeps RoPE in higher precision (Appendix D.2) but does not spell it out;
the split of a 128-dim head into 44/42/42 dims for (t, h, w) and "action tokens take
positions after the last frame" come from the workload description.  Readings:
segments of (Dh - 4*floor(Dh/6), 2*floor(Dh/6), 2*floor(Dh/6)) contiguous dims,
base 10000, rotation of adjacent pairs inside each segment.
"""
import numpy as np


def rope_split(Dh):
    a = Dh // 6
    return (Dh - 4 * a, 2 * a, 2 * a)


def rope_angles(pos, Dh, theta=10000.0):
    """Rotation angle of every adjacent pair of a head vector: for the segment of
    axis a with D_a dims and position p_a, pair i rotates by p_a * theta^(-2i/D_a).
    pos: (L, 3) integer (t, h, w) positions.  Returns (L, Dh/2)."""
    pos = np.asarray(pos, dtype=np.float64)
    parts = []
    for axis, Da in enumerate(rope_split(Dh)):
        i = np.arange(Da // 2, dtype=np.float64)
        parts.append(pos[:, axis:axis + 1] * theta ** (-2.0 * i / Da)[None, :])
    return np.concatenate(parts, axis=-1)


def apply_rope(x, pos, theta=10000.0):
    """Rotate each head vector of x (..., L, H, Dh): (x0, x1) -> (x0 cos - x1 sin,
    x0 sin + x1 cos) on every adjacent pair, angle from rope_angles."""
    Dh = x.shape[-1]
    phi = rope_angles(pos, Dh, theta)[:, None, :]  # (L, 1, Dh/2)
    c, s = np.cos(phi), np.sin(phi)
    x0, x1 = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x, dtype=np.float64)
    out[..., 0::2] = x0 * c - x1 * s
    out[..., 1::2] = x0 * s + x1 * c
    return out


def chunk_positions(c, F, Hg, Wg, A):
    """(t, h, w) positions of the tokens of chunk c: video token (f, r, s) of the
    chunk's F latent frames sits at (F*c + f, r, s); action token j sits after the
    chunk's last frame at (F*c + F + j, 0, 0).  Multi-view frames are one wide frame
    (section 3.1), so s runs over the tiled width."""
    f, r, s = np.meshgrid(np.arange(F), np.arange(Hg), np.arange(Wg), indexing="ij")
    video = np.stack([F * c + f.ravel(), r.ravel(), s.ravel()], axis=1)
    j = np.arange(A)
    action = np.stack([F * c + F + j, np.zeros(A, int), np.zeros(A, int)], axis=1)
    return np.concatenate([video, action], axis=0).astype(np.int64)
