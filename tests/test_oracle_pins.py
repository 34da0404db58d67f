"""Pins of the fp64 oracle against things other than itself: brute force on tiny
inputs, closed forms, invariants, library routines and the paper's Figure 10
visibility pattern.  Each group names the mistake it is there to catch."""
import math
import os

import numpy as np
import pytest

import oracle
from oracle import attention, rope_split, rope_angles, apply_rope, chunk_positions

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rnd(*shape, seed=0):
    return np.random.default_rng(seed).standard_normal(shape)


# ----------------------------------------------------------------------------- P1
def brute_attention(q, k, v, visible, scale):
    """Triple loop, explicit boolean mask, no vectorisation."""
    Lq, H, Dh = q.shape
    Lk = k.shape[0]
    o = np.zeros((Lq, H, v.shape[2]))
    for h in range(H):
        for i in range(Lq):
            scores = []
            for j in range(Lk):
                if visible[i][j]:
                    s = 0.0
                    for c in range(Dh):
                        s += q[i, h, c] * k[j, h, c]
                    scores.append((j, s * scale))
            mx = max(s for _, s in scores)
            den = sum(math.exp(s - mx) for _, s in scores)
            for j, s in scores:
                w = math.exp(s - mx) / den
                for c in range(v.shape[2]):
                    o[i, h, c] += w * v[j, h, c]
    return o


def test_attention_matches_brute_force_with_explicit_mask():
    # B=1, H=2, Dh=8, three chunks of five tokens; queries from chunks 0..2
    k_chunk = np.repeat([0, 1, 2], 5)
    q_chunk = np.array([0, 0, 1, 1, 1, 2, 2, 0, 2])
    q, k, v = rnd(9, 2, 8, seed=1), rnd(15, 2, 8, seed=2), rnd(15, 2, 8, seed=3)
    visible = [[k_chunk[j] <= q_chunk[i] for j in range(15)] for i in range(9)]
    ref = brute_attention(q, k, v, visible, 1 / math.sqrt(8))
    got = attention(q, k, v, q_chunk, k_chunk)
    assert np.max(np.abs(got - ref)) <= 1e-12


def test_attention_explicit_scale_and_empty_rows():
    q, k, v = rnd(4, 1, 8, seed=4), rnd(6, 1, 8, seed=5), rnd(6, 1, 8, seed=6)
    vis = [[True] * 6] * 4
    ref = brute_attention(q, k, v, vis, 0.37)
    assert np.max(np.abs(attention(q, k, v, np.zeros(4), np.zeros(6), 0.37) - ref)) <= 1e-12
    with pytest.raises(ValueError):
        attention(q, k, v, np.zeros(4), np.ones(6))


# ----------------------------------------------------------------------------- Figure 10
def read_visibility():
    cases = {}
    with open(os.path.join(GOLDEN, "fig10b_chunk_visibility.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            head, vis = line.split(":")
            case, qc = head.split()
            cases.setdefault(case, {})[int(qc)] = set(int(x) for x in vis.split())
    return cases


def test_attention_visibility_matches_figure_10():
    cases = read_visibility()
    n = 4
    k_chunk = np.repeat(np.arange(n), 3)
    k, v = rnd(12, 2, 8, seed=7), rnd(12, 2, 8, seed=8)
    for case, table in cases.items():
        for qc, vis in table.items():
            q = rnd(2, 2, 8, seed=9 + qc)
            qch = np.full(2, qc)
            base = attention(q, k, v, qch, k_chunk)
            for kc in range(n):
                v2 = v.copy()
                v2[k_chunk == kc] += 1.0
                changed = np.max(np.abs(attention(q, k, v2, qch, k_chunk) - base)) > 1e-9
                assert changed == (kc in vis), (case, qc, kc)


# ----------------------------------------------------------------------------- P5, P6, P7
def test_softmax_invariants():
    k_chunk = np.repeat([0, 1, 2], 4)
    q_chunk = np.array([0, 1, 2, 2])
    q, k = rnd(4, 2, 8, seed=10), rnd(12, 2, 8, seed=11)
    row = rnd(1, 2, 8, seed=12)
    v_const = np.repeat(row, 12, axis=0)
    # constant V rows -> that row
    assert np.allclose(attention(q, k, v_const, q_chunk, k_chunk), np.repeat(row, 4, 0), atol=1e-13)
    # q = 0 -> mean of the visible V
    v = rnd(12, 2, 8, seed=13)
    o = attention(np.zeros_like(q), k, v, q_chunk, k_chunk)
    for i, c in enumerate(q_chunk):
        assert np.allclose(o[i], v[k_chunk <= c].mean(axis=0), atol=1e-13)
    # adding the same amount to every score of a query changes nothing: shift every
    # key along that query's direction
    q1 = q[:1]
    alpha = 3.7
    shift = alpha * q1[0] / np.sum(q1[0] ** 2, axis=-1, keepdims=True) * math.sqrt(8)
    a = attention(q1, k, v, q_chunk[:1], k_chunk)
    b = attention(q1, k + shift[None], v, q_chunk[:1], k_chunk)
    assert np.allclose(a, b, atol=1e-12)
    # one visible key -> its value
    o1 = attention(q[:1], k[:1], v[:1], np.zeros(1), np.zeros(1))
    assert np.allclose(o1, v[:1], atol=1e-15)


def test_future_independence_and_permutation():
    k_chunk = np.repeat([0, 1, 2], 5)
    q_chunk = np.repeat([0, 1, 2], 5)
    q, k, v = rnd(15, 2, 8, seed=14), rnd(15, 2, 8, seed=15), rnd(15, 2, 8, seed=16)
    base = attention(q, k, v, q_chunk, k_chunk)
    k2, v2 = k.copy(), v.copy()
    k2[10:] = rnd(5, 2, 8, seed=17)
    v2[10:] = rnd(5, 2, 8, seed=18)
    o2 = attention(q, k2, v2, q_chunk, k_chunk)
    assert np.array_equal(o2[:10], base[:10])
    # permuting tokens inside chunk 1 (queries and keys alike) permutes the outputs
    perm = np.arange(15)
    perm[5:10] = [8, 5, 9, 7, 6]
    o3 = attention(q[perm], k[perm], v[perm], q_chunk, k_chunk)
    assert np.allclose(o3, base[perm], atol=1e-13)


# ----------------------------------------------------------------------------- KV-cache equivalence (P4)
def test_attention_kv_cache_equivalence():
    sizes = [4, 6, 5]
    k_chunk = np.repeat(np.arange(3), sizes)
    q, k, v = rnd(15, 3, 16, seed=20), rnd(15, 3, 16, seed=21), rnd(15, 3, 16, seed=22)
    full = attention(q, k, v, k_chunk, k_chunk)
    off = np.concatenate([[0], np.cumsum(sizes)])
    for c in range(3):
        rows = slice(off[c], off[c + 1])
        cached = attention(q[rows], k[:off[c + 1]], v[:off[c + 1]],
                           np.full(sizes[c], c), k_chunk[:off[c + 1]])
        assert np.allclose(cached, full[rows], atol=1e-13)


# ----------------------------------------------------------------------------- RoPE (P2)
def test_rope_split_matches_44_42_42():
    assert rope_split(128) == (44, 42, 42)
    assert sum(rope_split(64)) == 64 and all(s % 2 == 0 for s in rope_split(64))


def test_rope_rotation_properties():
    Dh = 128
    x = rnd(7, 3, Dh, seed=30)
    pos = np.array([[0, 0, 0], [1, 2, 3], [5, 29, 51], [9, 0, 0], [3, 7, 155], [2, 2, 2], [33, 1, 0]])
    y = apply_rope(x, pos)
    # norm preserved per head vector, and per rotated pair
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), atol=1e-12)
    assert np.allclose(y[..., 0::2] ** 2 + y[..., 1::2] ** 2, x[..., 0::2] ** 2 + x[..., 1::2] ** 2)
    # R(0) = I
    assert np.array_equal(y[0], x[0])
    # each axis only moves its own segment: 44 dims for t, 42 for h, 42 for w
    seg = np.cumsum([0] + list(rope_split(Dh)))
    for axis in range(3):
        p = np.zeros((1, 3), int)
        p[0, axis] = 5
        z = apply_rope(x[:1], p)
        moved = np.any(np.abs(z - x[:1]) > 0, axis=(0, 1))
        assert moved[seg[axis]:seg[axis + 1]].all()
        assert not moved[:seg[axis]].any() and not moved[seg[axis + 1]:].any()


def test_rope_angles_first_pair_and_geometric_spectrum():
    Dh = 128
    seg = rope_split(Dh)
    # measure the rotation of unit pairs: rotate e0 = (1, 0) in every pair
    e = np.zeros((1, 1, Dh))
    e[..., 0::2] = 1.0
    for axis in range(3):
        p = np.zeros((1, 3), int)
        p[0, axis] = 1
        r = apply_rope(e, p)[0, 0]
        ang = np.arctan2(r[1::2], r[0::2])
        start = sum(seg[:axis]) // 2
        a = ang[start:start + seg[axis] // 2]
        assert abs(a[0] - 1.0) < 1e-15  # first pair turns by exactly p radians
        ratio = a[1:] / a[:-1]  # geometric with ratio 10000^(-2/D_a)
        assert np.allclose(ratio, 10000.0 ** (-2.0 / seg[axis]), rtol=1e-12)
        assert a[-1] > 1e-4 and a[-1] < 1.0


def test_rope_relative_position_invariance():
    Dh = 64
    qv, kv = rnd(1, 2, Dh, seed=31), rnd(1, 2, Dh, seed=32)
    p, pp = np.array([[3, 4, 5]]), np.array([[1, 9, 2]])
    base = np.sum(apply_rope(qv, p) * apply_rope(kv, pp), axis=-1)
    for s in ([7, 0, 0], [0, 11, 0], [0, 0, 13], [2, 3, 4]):
        s = np.array([s])
        sh = np.sum(apply_rope(qv, p + s) * apply_rope(kv, pp + s), axis=-1)
        assert np.allclose(sh, base, atol=1e-12)


def test_chunk_positions():
    pos = chunk_positions(2, 2, 3, 4, 5)
    assert pos.shape == (2 * 3 * 4 + 5, 3)
    # video tokens run frame-major, then row, then column, frames 2c .. 2c+1
    assert pos[0].tolist() == [4, 0, 0] and pos[1].tolist() == [4, 0, 1]
    assert pos[4].tolist() == [4, 1, 0] and pos[12].tolist() == [5, 0, 0]
    assert pos[23].tolist() == [5, 2, 3]
    # action tokens come after the chunk's last frame
    assert pos[24:].tolist() == [[6 + j, 0, 0] for j in range(5)]


# ----------------------------------------------------------------------------- LN, AdaLN, GELU, Linear
def test_layernorm_moments_and_closed_form():
    eps = 1e-6
    x = rnd(5, 64, seed=40) * 3 + 2
    y = oracle.layernorm(x, eps)
    var = x.var(axis=-1)
    assert np.allclose(y.mean(axis=-1), 0, atol=1e-13)
    assert np.allclose(y.var(axis=-1), var / (var + eps), rtol=1e-12)
    a = 0.3
    assert np.allclose(oracle.layernorm(np.array([a, -a]), eps), np.array([a, -a]) / math.sqrt(a * a + eps))
    g, b = rnd(64, seed=41), rnd(64, seed=42)
    assert np.allclose(oracle.layernorm(x, eps, g, b), y * g + b)
    # invariance under per-row affine change of the input (up to eps)
    assert np.allclose(oracle.layernorm(5 * x + 7, 0.0), oracle.layernorm(x, 0.0), atol=1e-12)


def test_adaln_zero_modulation_is_layernorm():
    x = rnd(3, 32, seed=43)
    z = np.zeros(32)
    assert np.array_equal(oracle.modulate(x, z, z, 1e-6), oracle.layernorm(x, 1e-6))
    sc, sh = rnd(32, seed=44), rnd(32, seed=45)
    m = oracle.modulate(x, sh, sc, 1e-6)
    assert np.allclose(oracle.layernorm(m - sh, 0.0), oracle.layernorm(oracle.layernorm(x, 1e-6) * (1 + sc), 0.0))


def test_gelu_tanh():
    u = np.linspace(-8, 8, 2001)
    g = oracle.gelu_tanh(u)
    assert oracle.gelu_tanh(np.array(0.0)) == 0.0
    assert np.allclose(g - oracle.gelu_tanh(-u), u, atol=1e-14)
    erf_gelu = np.array([0.5 * x * (1 + math.erf(x / math.sqrt(2))) for x in u])
    err = np.max(np.abs(g - erf_gelu))
    assert 1e-5 < err < 1e-3  # a close approximation of GELU, but not GELU itself
    assert abs(oracle.gelu_tanh(np.array(30.0)) - 30.0) < 1e-12
    assert abs(oracle.gelu_tanh(np.array(-30.0))) < 1e-12


def test_silu():
    u = np.linspace(-20, 20, 101)
    ref = np.array([x / (1 + math.exp(-x)) for x in u])
    assert np.allclose(oracle.silu(u), ref, rtol=1e-14, atol=1e-300)


def test_linear_brute_force():
    x, w, b = rnd(2, 3, 5, seed=46), rnd(4, 5, seed=47), rnd(4, seed=48)
    y = oracle.linear(x, w, b)
    for i in range(2):
        for j in range(3):
            for o in range(4):
                assert abs(y[i, j, o] - (sum(x[i, j, c] * w[o, c] for c in range(5)) + b[o])) < 1e-13


def test_timestep_sinusoid():
    s = oracle.timestep_sinusoid(np.array([0.0, 0.3, 1.0]))
    assert s.shape == (3, 256)
    assert np.array_equal(s[0], np.concatenate([np.ones(128), np.zeros(128)]))
    # cos and sin of the same frequency are paired
    assert np.allclose(s[:, :128] ** 2 + s[:, 128:] ** 2, 1.0)
    # measured angular frequencies are geometric from 1000 rad per unit t down by 10^4
    t = 1e-5
    a = np.arctan2(oracle.timestep_sinusoid(np.array([t]))[0, 128:], oracle.timestep_sinusoid(np.array([t]))[0, :128]) / t
    assert abs(a[0] - 1000.0) < 1e-6
    assert np.allclose(a[1:] / a[:-1], 10000.0 ** (-1 / 128), rtol=1e-9)


# ----------------------------------------------------------------------------- patchify (P8)
def test_patchify_roundtrip_and_layout():
    B, C, F, Hl, Wl = 2, 3, 2, 4, 6
    z = rnd(B, C, F, Hl, Wl, seed=50)
    tok = oracle.patchify(z)
    assert tok.shape == (B, F * 2 * 3, C * 4)
    assert np.array_equal(oracle.unpatchify(tok, C, F, Hl, Wl), z)
    # coordinate-encoded latent: decode every token feature back to its coordinates
    c, f, y, x = np.meshgrid(np.arange(C), np.arange(F), np.arange(Hl), np.arange(Wl), indexing="ij")
    code = (c * 1000 + f * 100 + y * 10 + x).astype(float)[None]
    t = oracle.patchify(code)[0]
    for ti in range(t.shape[0]):
        fi, rem = divmod(ti, 2 * 3)
        r, s = divmod(rem, 3)
        for fe in range(C * 4):
            cc, rest = divmod(fe, 4)
            ph, pw = divmod(rest, 2)
            assert t[ti, fe] == cc * 1000 + fi * 100 + (2 * r + ph) * 10 + (2 * s + pw)


# ----------------------------------------------------------------------------- block-level pins
def small_block_weights(d, F, seed, zero_gates=False):
    g = np.random.default_rng(seed)
    W = {
        "w_qkv": g.standard_normal((3 * d, d)) * 0.1, "b_qkv": g.standard_normal(3 * d) * 0.1,
        "w_o": g.standard_normal((d, d)) * 0.1, "b_o": g.standard_normal(d) * 0.1,
        "w_cq": g.standard_normal((d, d)) * 0.1, "b_cq": g.standard_normal(d) * 0.1,
        "w_ckv": g.standard_normal((2 * d, d)) * 0.1, "b_ckv": g.standard_normal(2 * d) * 0.1,
        "w_co": g.standard_normal((d, d)) * 0.1, "b_co": g.standard_normal(d) * 0.1,
        "w_f1": g.standard_normal((F, d)) * 0.1, "b_f1": g.standard_normal(F) * 0.1,
        "w_f2": g.standard_normal((d, F)) * 0.1, "b_f2": g.standard_normal(d) * 0.1,
        "mod6": g.standard_normal((6, d)) * 0.3,
        "lnc_gamma": 1 + 0.1 * g.standard_normal(d), "lnc_beta": 0.1 * g.standard_normal(d),
    }
    return W


def test_block_kv_cache_equivalence():
    """Three chunks in one masked call equal three sequential cached calls, each
    appending its post-RoPE K and V to the cache (Figure 10b, section 3.1)."""
    d, H, Fh, B = 24, 2, 40, 2
    Fg, Hg, Wg, A = 2, 2, 3, 2
    W = small_block_weights(d, Fh, 60)
    Lc = 5
    ctx = rnd(B, Lc, d, seed=61)
    e0 = rnd(B, 6, d, seed=62) * 0.5
    Lch = Fg * Hg * Wg + A
    pos = np.concatenate([chunk_positions(c, Fg, Hg, Wg, A) for c in range(3)])
    chunk = np.repeat(np.arange(3), Lch)
    x = rnd(B, 3 * Lch, d, seed=63)
    full, k_full, v_full = oracle.dit_block(x, e0, W, H, 1e-6, pos, chunk, ctx=ctx)
    kc = vc = pc = None
    for c in range(3):
        rows = slice(c * Lch, (c + 1) * Lch)
        out, k, v = oracle.dit_block(x[:, rows], e0, W, H, 1e-6, pos[rows], chunk[rows], kc, vc, pc, ctx=ctx)
        assert np.allclose(out, full[:, rows], atol=1e-12)
        kc = k if kc is None else np.concatenate([kc, k], 1)
        vc = v if vc is None else np.concatenate([vc, v], 1)
        pc = chunk[rows] if pc is None else np.concatenate([pc, chunk[rows]])
    assert np.allclose(kc, k_full, atol=1e-13) and np.allclose(vc, v_full, atol=1e-13)


def test_block_zero_gates():
    d, H, Fh, B, L = 16, 2, 32, 1, 7
    W = small_block_weights(d, Fh, 70)
    W["mod6"][2] = 0.0  # gate1
    W["mod6"][5] = 0.0  # gate2
    e0 = rnd(B, 6, d, seed=71)
    e0[:, 2] = 0.0
    e0[:, 5] = 0.0
    x = rnd(B, L, d, seed=72)
    ctx = rnd(B, 4, d, seed=73)
    pos = chunk_positions(0, 1, 1, 5, 2)
    ch = np.zeros(L, int)
    out, _, _ = oracle.dit_block(x, e0, W, H, 1e-6, pos, ch, ctx=ctx)
    # with both gates zero the self-attention and FFN weights do not matter
    W2 = dict(W)
    for n in ("w_qkv", "w_o", "w_f1", "w_f2", "b_qkv", "b_o", "b_f1", "b_f2"):
        W2[n] = W[n] * -3.0 + 1.0
    out2, _, _ = oracle.dit_block(x, e0, W2, H, 1e-6, pos, ch, ctx=ctx)
    assert np.allclose(out, out2, atol=1e-13)
    assert np.max(np.abs(out - x)) > 1e-2  # the ungated cross-attention branch still moves x
    # ... and with the cross-attention output projection zeroed the block is the identity
    W2["w_co"] = np.zeros_like(W["w_co"])
    W2["b_co"] = np.zeros_like(W["b_co"])
    out3, _, _ = oracle.dit_block(x, e0, W2, H, 1e-6, pos, ch, ctx=ctx)
    assert np.array_equal(out3, x)


def test_block_token_permutation_equivariance():
    d, H, Fh, B, L = 16, 2, 32, 1, 8
    W = small_block_weights(d, Fh, 80)
    e0 = rnd(B, 6, d, seed=81)
    x = rnd(B, L, d, seed=82)
    ctx = rnd(B, 3, d, seed=83)
    pos = chunk_positions(1, 1, 2, 3, 2)
    ch = np.full(L, 1)
    kp, vp = rnd(B, 4, H, d // H, seed=84), rnd(B, 4, H, d // H, seed=85)
    pc = np.zeros(4, int)
    out, k, v = oracle.dit_block(x, e0, W, H, 1e-6, pos, ch, kp, vp, pc, ctx=ctx)
    perm = np.array([3, 0, 7, 1, 2, 6, 4, 5])
    out_p, k_p, _ = oracle.dit_block(x[:, perm], e0, W, H, 1e-6, pos[perm], ch, kp, vp, pc, ctx=ctx)
    assert np.allclose(out_p, out[:, perm], atol=1e-12)
    assert np.allclose(k_p, k[:, perm], atol=1e-13)


def test_block_precomputed_cross_kv():
    d, H, Fh, B, L = 16, 2, 32, 2, 5
    W = small_block_weights(d, Fh, 90)
    x, e0, ctx = rnd(B, L, d, seed=91), rnd(B, 6, d, seed=92), rnd(B, 3, d, seed=93)
    pos = chunk_positions(0, 1, 1, 3, 2)
    ch = np.zeros(L, int)
    a, _, _ = oracle.dit_block(x, e0, W, H, 1e-6, pos, ch, ctx=ctx)
    kv = oracle.linear(ctx, W["w_ckv"], W["b_ckv"])
    b, _, _ = oracle.dit_block(x, e0, W, H, 1e-6, pos, ch, ctx_kv=kv)
    assert np.array_equal(a, b)


def test_block_row_subset_equals_rows_of_the_full_block():
    """The row-sampled block (queries and token-wise work for listed rows only, every
    row's K and V) equals those rows of the full block: with a cache, batch 2, a
    per-sample and a per-token modulation, rows in any order."""
    d, H, Fh, B = 16, 2, 32, 2
    W = small_block_weights(d, Fh, 550)
    Fg, Hg, Wg, A = 2, 2, 2, 2
    L = Fg * Hg * Wg + A
    pos = chunk_positions(1, Fg, Hg, Wg, A)
    ch = np.full(L, 1)
    kp, vp = rnd(B, 5, H, d // H, seed=551), rnd(B, 5, H, d // H, seed=552)
    pc = np.zeros(5, int)
    x, ctx = rnd(B, L, d, seed=553), rnd(B, 3, d, seed=554)
    rows = np.array([7, 0, 9, 3])
    for e0 in (rnd(B, 6, d, seed=555) * 0.5, rnd(B, L, 6, d, seed=556) * 0.5):
        full, kf, vf = oracle.dit_block(x, e0, W, H, 1e-6, pos, ch, kp, vp, pc, ctx=ctx)
        sub, ks, vs = oracle.dit_block(x, e0, W, H, 1e-6, pos, ch, kp, vp, pc, ctx=ctx, rows=rows)
        assert sub.shape == (B, len(rows), d)
        assert np.max(np.abs(sub - full[:, rows])) <= 1e-12
        assert np.array_equal(ks, kf) and np.array_equal(vs, vf)


# ----------------------------------------------------------------------------- every branch live, by hand
def _ln_by_hand(v, eps):
    n = len(v)
    mu = sum(v) / n
    var = sum((a - mu) ** 2 for a in v) / n
    return [(a - mu) / math.sqrt(var + eps) for a in v]


def _matvec(W, b, v):
    return [sum(W[r][c] * v[c] for c in range(len(v))) + b[r] for r in range(len(W))]


def _softmax_mix(q, keys, vals, scale):
    s = [scale * sum(qa * ka for qa, ka in zip(q, k)) for k in keys]
    m = max(s)
    w = [math.exp(a - m) for a in s]
    z = sum(w)
    return [sum(w[j] * vals[j][c] for j in range(len(keys))) / z for c in range(len(vals[0]))]


def test_block_every_branch_by_hand():
    """A block with every branch live, recomputed token by token with scalar loops:
    gates g1 != g2 (both non-zero), non-zero W_co and b_co, cross LayerNorm with
    gamma != 1 and beta != 0, non-zero biases, a cached key of an earlier chunk (visible)
    and one of a later chunk (hidden).  Dh = 6 splits into three one-pair RoPE segments
    (t | h | w), each turned by its position in radians.  This fixes the block's wiring:
    g1 scales the self-attention branch and g2 the FFN, the cross branch has no gate and
    reads LN(x) gamma + beta of the residual after the self-attention update, the FFN reads
    the residual after the cross update."""
    d, H, Dh, Fh, eps = 12, 2, 6, 10, 1e-6
    g = np.random.default_rng(500)
    W = small_block_weights(d, Fh, 501)
    e0 = g.standard_normal((1, 6, d)) * 0.5
    m = W["mod6"] + e0[0]
    sh1, sc1, g1, sh2, sc2, g2 = (list(m[i]) for i in range(6))
    assert min(abs(a - b) for a, b in zip(g1, g2)) > 1e-3 and min(map(abs, g1 + g2)) > 1e-3
    x = g.standard_normal((1, 2, d))
    pos = np.array([[2, 1, 3], [3, 0, 2]])
    ctx = g.standard_normal((1, 3, d))
    k_prev = g.standard_normal((1, 2, H, Dh))
    v_prev = g.standard_normal((1, 2, H, Dh))
    prev_chunk = np.array([0, 2])
    out, k_cur, v_cur = oracle.dit_block(x, e0, W, H, eps, pos, np.array([1, 1]), k_prev, v_prev, prev_chunk,
                                         ctx=ctx)

    L_ = lambda a: [list(r) for r in np.asarray(a)]  # noqa: E731
    Wqkv, Wo, Wcq, Wckv, Wco, W1, W2 = (L_(W[n]) for n in ("w_qkv", "w_o", "w_cq", "w_ckv", "w_co", "w_f1", "w_f2"))
    bqkv, bo, bcq, bckv, bco, b1, b2 = (list(W[n]) for n in ("b_qkv", "b_o", "b_cq", "b_ckv", "b_co", "b_f1", "b_f2"))
    gam, bet = list(W["lnc_gamma"]), list(W["lnc_beta"])

    def rope(vec, p):  # one head: pairs (0,1) by p_t, (2,3) by p_h, (4,5) by p_w radians
        r = list(vec)
        for a in range(3):
            c, s = math.cos(p[a]), math.sin(p[a])
            x0, x1 = vec[2 * a], vec[2 * a + 1]
            r[2 * a], r[2 * a + 1] = x0 * c - x1 * s, x0 * s + x1 * c
        return r

    # self-attention inputs of both current tokens
    q_t, k_t, v_t = [], [], []
    for i in range(2):
        n1 = _ln_by_hand(list(x[0, i]), eps)
        h1 = [n1[c] * (1 + sc1[c]) + sh1[c] for c in range(d)]
        qkv = _matvec(Wqkv, bqkv, h1)
        q_t.append([rope(qkv[hh * Dh:(hh + 1) * Dh], pos[i]) for hh in range(H)])
        k_t.append([rope(qkv[d + hh * Dh:d + (hh + 1) * Dh], pos[i]) for hh in range(H)])
        v_t.append([qkv[2 * d + hh * Dh:2 * d + (hh + 1) * Dh] for hh in range(H)])
    ctx_k = [_matvec([r for r in Wckv[:d]], bckv[:d], list(ctx[0, j])) for j in range(3)]
    ctx_v = [_matvec([r for r in Wckv[d:]], bckv[d:], list(ctx[0, j])) for j in range(3)]
    for i in range(2):
        # keys visible to chunk 1: the cached row of chunk 0 and both current rows
        o = []
        for hh in range(H):
            keys = [list(k_prev[0, 0, hh]), k_t[0][hh], k_t[1][hh]]
            vals = [list(v_prev[0, 0, hh]), v_t[0][hh], v_t[1][hh]]
            o += _softmax_mix(q_t[i][hh], keys, vals, 1 / math.sqrt(Dh))
        ao = _matvec(Wo, bo, o)
        x1 = [x[0, i, c] + g1[c] * ao[c] for c in range(d)]
        nc = _ln_by_hand(x1, eps)
        hc = [nc[c] * gam[c] + bet[c] for c in range(d)]
        cq = _matvec(Wcq, bcq, hc)
        oc = []
        for hh in range(H):
            sl = slice(hh * Dh, (hh + 1) * Dh)
            oc += _softmax_mix(cq[sl], [k[sl] for k in ctx_k], [v[sl] for v in ctx_v], 1 / math.sqrt(Dh))
        co = _matvec(Wco, bco, oc)
        x2 = [x1[c] + co[c] for c in range(d)]
        n2 = _ln_by_hand(x2, eps)
        h2 = [n2[c] * (1 + sc2[c]) + sh2[c] for c in range(d)]
        u = [0.5 * a * (1 + math.tanh(math.sqrt(2 / math.pi) * (a + 0.044715 * a ** 3))) for a in _matvec(W1, b1, h2)]
        f = _matvec(W2, b2, u)
        x3 = [x2[c] + g2[c] * f[c] for c in range(d)]
        assert np.max(np.abs(out[0, i] - np.array(x3))) <= 1e-12
        for hh in range(H):
            assert np.max(np.abs(k_cur[0, i, hh] - np.array(k_t[i][hh]))) <= 1e-12
            assert np.max(np.abs(v_cur[0, i, hh] - np.array(v_t[i][hh]))) <= 1e-12


def test_block_gate_assignment():
    """g1 gates only the self-attention branch and g2 only the FFN: with g2 = 0 the FFN
    weights cannot matter while the O projection does; with g1 = 0 the reverse."""
    d, H, Fh, B, L = 16, 2, 32, 1, 6
    base = small_block_weights(d, Fh, 510)
    x = rnd(B, L, d, seed=511)
    ctx = rnd(B, 4, d, seed=512)
    pos = chunk_positions(0, 1, 1, 4, 2)
    ch = np.zeros(L, int)
    for zero_gate, dead, live in ((5, ("w_f1", "w_f2", "b_f1", "b_f2"), ("w_o", "b_o")),
                                  (2, ("w_qkv", "w_o", "b_qkv", "b_o"), ("w_f2", "b_f2"))):
        W = dict(base)
        W["mod6"] = base["mod6"].copy()
        W["mod6"][zero_gate] = 0.0
        e0 = rnd(B, 6, d, seed=513)
        e0[:, zero_gate] = 0.0
        out, _, _ = oracle.dit_block(x, e0, W, H, 1e-6, pos, ch, ctx=ctx)
        Wd = dict(W)
        for n in dead:
            Wd[n] = W[n] * -2.0 + 0.5
        out_d, _, _ = oracle.dit_block(x, e0, Wd, H, 1e-6, pos, ch, ctx=ctx)
        assert np.allclose(out, out_d, atol=1e-13)
        Wl = dict(W)
        for n in live:
            Wl[n] = W[n] * -2.0 + 0.5
        out_l, _, _ = oracle.dit_block(x, e0, Wl, H, 1e-6, pos, ch, ctx=ctx)
        assert np.max(np.abs(out - out_l)) > 1e-3


def test_block_cross_branch_reads_the_affine_layernorm_only():
    """With g1 = g2 = 0 only the cross-attention branch moves x.  That branch takes no
    AdaLN shift or scale (changing them changes nothing), and its LayerNorm is affine:
    with gamma = 0 every token's cross query is W_cq beta + b_cq, so every token receives
    the same increment."""
    d, H, Fh, B, L = 16, 2, 32, 1, 7
    W = small_block_weights(d, Fh, 520)
    W["mod6"][2] = W["mod6"][5] = 0.0
    e0 = rnd(B, 6, d, seed=521)
    e0[:, 2] = e0[:, 5] = 0.0
    x = rnd(B, L, d, seed=522)
    ctx = rnd(B, 4, d, seed=523)
    pos = chunk_positions(0, 1, 1, 5, 2)
    ch = np.zeros(L, int)
    out, _, _ = oracle.dit_block(x, e0, W, H, 1e-6, pos, ch, ctx=ctx)
    assert np.max(np.abs(out - x)) > 1e-2  # the cross branch is live
    e0b = e0.copy()
    for i in (0, 1, 3, 4):
        e0b[:, i] = rnd(B, d, seed=530 + i) * 2.0
    out_b, _, _ = oracle.dit_block(x, e0b, W, H, 1e-6, pos, ch, ctx=ctx)
    assert np.allclose(out_b, out, atol=1e-13)
    Wg = dict(W)
    Wg["lnc_gamma"] = np.zeros(d)
    out_g, _, _ = oracle.dit_block(x, e0, Wg, H, 1e-6, pos, ch, ctx=ctx)
    inc = out_g - x
    assert np.allclose(inc, inc[:, :1], atol=1e-13)
    # that shared increment is the cross attention of the query W_cq beta + b_cq
    cq = W["w_cq"] @ W["lnc_beta"] + W["b_cq"]
    kv = W["w_ckv"] @ ctx[0].T + W["b_ckv"][:, None]
    o = []
    for hh in range(H):
        sl = slice(hh * 8, (hh + 1) * 8)
        o += _softmax_mix(list(cq[sl]), [list(kv[:d][sl, j]) for j in range(4)],
                          [list(kv[d:][sl, j]) for j in range(4)], 1 / math.sqrt(8))
    assert np.allclose(inc[0, 0], W["w_co"] @ np.array(o) + W["b_co"], atol=1e-12)


def test_text_projection_by_hand():
    """Text features -> context: Linear, then tanh-GELU, then Linear, token by token."""
    g = np.random.default_rng(540)
    B, Lc, tdim, d = 2, 3, 7, 5
    text = g.standard_normal((B, Lc, tdim))
    w1, b1 = g.standard_normal((d, tdim)), g.standard_normal(d)
    w2, b2 = g.standard_normal((d, d)) * 0.5, g.standard_normal(d)
    got = oracle.text_projection(text, w1, b1, w2, b2)
    for b in range(B):
        for j in range(Lc):
            hid = []
            for r in range(d):
                a = b1[r] + sum(w1[r, c] * text[b, j, c] for c in range(tdim))
                hid.append(0.5 * a * (1 + math.tanh(math.sqrt(2 / math.pi) * (a + 0.044715 * a ** 3))))
            for r in range(d):
                want = b2[r] + sum(w2[r, c] * hid[c] for c in range(d))
                assert abs(got[b, j, r] - want) <= 1e-12


# ----------------------------------------------------------------------------- step (P12)
def test_step_identity_blocks_reduce_to_embed_and_head():
    """All gates zero and W_co = b_co = 0 in every block => every block is the identity,
    so the velocity is head(embed(z, a)); this checks the step's wiring of time
    embedding, patchify, embeddings, head and unpatchify."""
    g = np.random.default_rng(100)
    B, C, F, Hl, Wl, A, ad, d, H = 2, 4, 2, 4, 6, 3, 5, 16, 2
    tdim, Lc = 12, 4
    P = {"w_t1": g.standard_normal((d, 256)) * 0.1, "b_t1": g.standard_normal(d) * 0.1,
         "w_t2": g.standard_normal((d, d)) * 0.1, "b_t2": g.standard_normal(d) * 0.1,
         "w_t6": g.standard_normal((6 * d, d)) * 0.1, "b_t6": g.standard_normal(6 * d) * 0.1,
         "w_x1": g.standard_normal((d, tdim)) * 0.1, "b_x1": np.zeros(d),
         "w_x2": g.standard_normal((d, d)) * 0.1, "b_x2": np.zeros(d),
         "w_patch": g.standard_normal((d, C * 4)), "b_patch": g.standard_normal(d),
         "w_ain": g.standard_normal((d, ad)), "b_ain": g.standard_normal(d),
         "w_hv": g.standard_normal((C * 4, d)), "b_hv": g.standard_normal(C * 4),
         "w_ha": g.standard_normal((ad, d)), "b_ha": g.standard_normal(ad),
         "head_mod2": g.standard_normal((2, d)) * 0.1}
    # zero the gate rows of the time projection so e0's gates are exactly zero
    for gate in (2, 5):
        P["w_t6"][gate * d:(gate + 1) * d] = 0.0
        P["b_t6"][gate * d:(gate + 1) * d] = 0.0
    W = small_block_weights(d, 32, 101)
    W["mod6"][2] = W["mod6"][5] = 0.0
    W["w_co"] = np.zeros((d, d))
    W["b_co"] = np.zeros(d)
    z, a = g.standard_normal((B, C, F, Hl, Wl)), g.standard_normal((B, A, ad))
    t = np.array([0.25, 0.8])
    text = g.standard_normal((B, Lc, tdim))
    Lv = F * (Hl // 2) * (Wl // 2)
    pos = chunk_positions(1, F, Hl // 2, Wl // 2, A)
    kp = g.standard_normal((B, 6, H, d // H))
    vv, va = oracle.dit_step(z, a, t, text, P, lambda l: (W, kp, kp), 3, H, 1e-6, 1, pos,
                             prev_chunk=np.zeros(6, int))
    # independent composition: tokens -> head, per token, written out by hand
    e = np.zeros((B, d))
    for b in range(B):
        s = np.array([math.cos(1000 * t[b] * 10000 ** (-k / 128)) for k in range(128)]
                     + [math.sin(1000 * t[b] * 10000 ** (-k / 128)) for k in range(128)])
        h1 = P["w_t1"] @ s + P["b_t1"]
        h1 = h1 / (1 + np.exp(-h1))
        e[b] = P["w_t2"] @ h1 + P["b_t2"]
    for b in range(B):
        sh, sc = P["head_mod2"][0] + e[b], P["head_mod2"][1] + e[b]
        for tok in range(Lv + A):
            if tok < Lv:
                f, rem = divmod(tok, (Hl // 2) * (Wl // 2))
                r, s_ = divmod(rem, Wl // 2)
                feat = np.array([z[b, c, f, 2 * r + ph, 2 * s_ + pw]
                                 for c in range(C) for ph in range(2) for pw in range(2)])
                xt = P["w_patch"] @ feat + P["b_patch"]
            else:
                xt = P["w_ain"] @ a[b, tok - Lv] + P["b_ain"]
            ht = (xt - xt.mean()) / math.sqrt(xt.var() + 1e-6) * (1 + sc) + sh
            if tok < Lv:
                out = P["w_hv"] @ ht + P["b_hv"]
                for c in range(C):
                    for ph in range(2):
                        for pw in range(2):
                            assert abs(vv[b, c, f, 2 * r + ph, 2 * s_ + pw] - out[c * 4 + ph * 2 + pw]) < 1e-10
            else:
                assert np.allclose(va[b, tok - Lv], P["w_ha"] @ ht + P["b_ha"], atol=1e-10)



def test_step_depth_taps_equal_shallower_steps():
    """dit_step(depths=[1, 3]) gives the velocities of the 1-block and the 3-block steps."""
    g = np.random.default_rng(560)
    B, C, F, Hl, Wl, A, ad, d, H, tdim, Lc = 1, 4, 2, 4, 4, 2, 5, 16, 2, 6, 3
    P = small_model_params(g, d, C, ad, tdim)
    Ws = [small_block_weights(d, 24, 561 + l) for l in range(3)]
    z, a = g.standard_normal((B, C, F, Hl, Wl)), g.standard_normal((B, A, ad))
    t, text = np.array([0.3]), g.standard_normal((B, Lc, tdim))
    pos = chunk_positions(0, F, Hl // 2, Wl // 2, A)
    taps = oracle.dit_step(z, a, t, text, P, lambda l: (Ws[l], None, None), 3, H, 1e-6, 0, pos, depths=[1, 3])
    for (tv, ta), n in zip(taps, (1, 3)):
        rv, ra = oracle.dit_step(z, a, t, text, P, lambda l: (Ws[l], None, None), n, H, 1e-6, 0, pos)
        assert np.array_equal(tv, rv) and np.array_equal(ta, ra)


# ----------------------------------------------------------------------------- update pass
def small_model_params(g, d, C, ad, tdim):
    return {"w_t1": g.standard_normal((d, 256)) * 0.1, "b_t1": g.standard_normal(d) * 0.1,
            "w_t2": g.standard_normal((d, d)) * 0.1, "b_t2": g.standard_normal(d) * 0.1,
            "w_t6": g.standard_normal((6 * d, d)) * 0.1, "b_t6": g.standard_normal(6 * d) * 0.1,
            "w_x1": g.standard_normal((d, tdim)) * 0.1, "b_x1": np.zeros(d),
            "w_x2": g.standard_normal((d, d)) * 0.1, "b_x2": np.zeros(d),
            "w_patch": g.standard_normal((d, C * 4)), "b_patch": g.standard_normal(d),
            "w_ain": g.standard_normal((d, ad)), "b_ain": g.standard_normal(d),
            "w_hv": g.standard_normal((C * 4, d)), "b_hv": g.standard_normal(C * 4),
            "w_ha": g.standard_normal((ad, d)), "b_ha": g.standard_normal(ad),
            "head_mod2": g.standard_normal((2, d)) * 0.1}


def test_update_two_chunks_equal_two_sequential_updates():
    """Algorithm 2's cache update with two clean chunks in one call (block-causal mask,
    Figure 10b) appends exactly what two successive single-chunk updates append, each
    layer seeing its own cache (section 3.1, Model Inference)."""
    g = np.random.default_rng(110)
    B, C, F, Hl, Wl, ad, d, H, n_layers, Lc, tdim = 2, 4, 2, 4, 6, 5, 16, 2, 3, 3, 12
    P = small_model_params(g, d, C, ad, tdim)
    Ws = [small_block_weights(d, 32, 111 + l) for l in range(n_layers)]
    Hg, Wg = Hl // 2, Wl // 2
    Lch = F * Hg * Wg
    # one cached chunk (id 0) per layer, then clean chunks 1 and 2 (video only)
    kc0 = [g.standard_normal((B, Lch, H, d // H)) for _ in range(n_layers)]
    vc0 = [g.standard_normal((B, Lch, H, d // H)) for _ in range(n_layers)]
    z = g.standard_normal((B, C, 2 * F, Hl, Wl))  # frames of chunks 1 and 2
    a = np.zeros((B, 0, ad))
    t = np.array([1.0, 1.0])
    text = g.standard_normal((B, Lc, tdim))
    pos = np.concatenate([chunk_positions(1, F, Hg, Wg, 0), chunk_positions(2, F, Hg, Wg, 0)])
    q_chunk = np.repeat([1, 2], Lch)
    joint = oracle.dit_update(z, a, t, text, P, lambda l: (Ws[l], kc0[l], vc0[l]), n_layers, H, 1e-6,
                              pos, q_chunk, prev_chunk=np.zeros(Lch, int))
    first = oracle.dit_update(z[:, :, :F], a, t, text, P, lambda l: (Ws[l], kc0[l], vc0[l]), n_layers, H,
                              1e-6, pos[:Lch], q_chunk[:Lch], prev_chunk=np.zeros(Lch, int))
    kc1 = [np.concatenate([kc0[l], first[l][0]], 1) for l in range(n_layers)]
    vc1 = [np.concatenate([vc0[l], first[l][1]], 1) for l in range(n_layers)]
    second = oracle.dit_update(z[:, :, F:], a, t, text, P, lambda l: (Ws[l], kc1[l], vc1[l]), n_layers, H,
                               1e-6, pos[Lch:], q_chunk[Lch:], prev_chunk=np.repeat([0, 1], Lch))
    for l in range(n_layers):
        assert np.allclose(joint[l][0][:, :Lch], first[l][0], atol=1e-12)
        assert np.allclose(joint[l][1][:, :Lch], first[l][1], atol=1e-12)
        assert np.allclose(joint[l][0][:, Lch:], second[l][0], atol=1e-12)
        assert np.allclose(joint[l][1][:, Lch:], second[l][1], atol=1e-12)
    # chunk 1's rows must not see chunk 2: perturbing chunk 2's latents leaves them unchanged
    z2 = z.copy()
    z2[:, :, F:] += 1.0
    pert = oracle.dit_update(z2, a, t, text, P, lambda l: (Ws[l], kc0[l], vc0[l]), n_layers, H, 1e-6,
                             pos, q_chunk, prev_chunk=np.zeros(Lch, int))
    for l in range(n_layers):
        assert np.array_equal(pert[l][0][:, :Lch], joint[l][0][:, :Lch])
        assert not np.allclose(pert[l][0][:, Lch:], joint[l][0][:, Lch:])


def test_update_identity_blocks_closed_form():
    """With every block the identity (zero gates, W_co = b_co = 0), each layer's residual
    input is the patch embedding of the clean latents, so the appended K and V of layer l
    are that layer's projection of LN(x)(1+scale)+shift, with K rotated pair by pair at
    the token's (frame, row, column) position; written out here token by token."""
    g = np.random.default_rng(120)
    B, C, F, Hl, Wl, ad, d, H, n_layers, Lc, tdim = 1, 2, 2, 4, 4, 3, 12, 1, 2, 2, 8
    Dh = d // H
    P = small_model_params(g, d, C, ad, tdim)
    for gate in (2, 5):
        P["w_t6"][gate * d:(gate + 1) * d] = 0.0
        P["b_t6"][gate * d:(gate + 1) * d] = 0.0
    Ws = []
    for l in range(n_layers):
        W = small_block_weights(d, 24, 121 + l)
        W["mod6"][2] = W["mod6"][5] = 0.0
        W["w_co"] = np.zeros((d, d))
        W["b_co"] = np.zeros(d)
        Ws.append(W)
    z = g.standard_normal((B, C, F, Hl, Wl))
    t = np.array([0.6])
    text = g.standard_normal((B, Lc, tdim))
    c = 3  # chunk index of the clean chunk; no cache rows
    Hg, Wg = Hl // 2, Wl // 2
    pos = chunk_positions(c, F, Hg, Wg, 0)
    kv = oracle.dit_update(z, np.zeros((B, 0, ad)), t, text, P, lambda l: (Ws[l], None, None), n_layers, H,
                           1e-6, pos, np.full(F * Hg * Wg, c))
    # e0 by hand
    s = np.array([math.cos(1000 * t[0] * 10000 ** (-k / 128)) for k in range(128)]
                 + [math.sin(1000 * t[0] * 10000 ** (-k / 128)) for k in range(128)])
    h1 = P["w_t1"] @ s + P["b_t1"]
    h1 = h1 / (1 + np.exp(-h1))
    e = P["w_t2"] @ h1 + P["b_t2"]
    se = e / (1 + np.exp(-e))
    e0 = (P["w_t6"] @ se + P["b_t6"]).reshape(6, d)
    seg = (Dh - 4 * (Dh // 6), 2 * (Dh // 6), 2 * (Dh // 6))
    for l in range(n_layers):
        m = Ws[l]["mod6"] + e0
        for tok in range(F * Hg * Wg):
            f, rem = divmod(tok, Hg * Wg)
            r, s_ = divmod(rem, Wg)
            feat = np.array([z[0, ch, f, 2 * r + ph, 2 * s_ + pw] for ch in range(C) for ph in range(2)
                             for pw in range(2)])
            xt = P["w_patch"] @ feat + P["b_patch"]
            ht = (xt - xt.mean()) / math.sqrt(xt.var() + 1e-6) * (1 + m[1]) + m[0]
            kraw = Ws[l]["w_qkv"][d:2 * d] @ ht + Ws[l]["b_qkv"][d:2 * d]
            vraw = Ws[l]["w_qkv"][2 * d:] @ ht + Ws[l]["b_qkv"][2 * d:]
            p3 = (F * c + f, r, s_)
            krot = kraw.copy()
            for hd in range(H):
                base = hd * Dh
                for ax in range(3):
                    for i in range(seg[ax] // 2):
                        ang = p3[ax] * 10000.0 ** (-2.0 * i / seg[ax])
                        x0, x1 = kraw[base + 2 * i], kraw[base + 2 * i + 1]
                        krot[base + 2 * i] = x0 * math.cos(ang) - x1 * math.sin(ang)
                        krot[base + 2 * i + 1] = x0 * math.sin(ang) + x1 * math.cos(ang)
                    base += seg[ax]
            assert np.allclose(kv[l][0][0, tok].reshape(d), krot, atol=1e-10)
            assert np.allclose(kv[l][1][0, tok].reshape(d), vraw, atol=1e-10)


# ----------------------------------------------------------------------------- DreamZero-Flash
def flash_case(seed):
    g = np.random.default_rng(seed)
    B, C, F, Hl, Wl, A, ad, d, H, tdim, Lc = 2, 2, 2, 4, 4, 3, 5, 16, 2, 12, 4
    P = small_model_params(g, d, C, ad, tdim)
    Ws = [small_block_weights(d, 32, seed + 1 + l) for l in range(2)]
    z, a = g.standard_normal((B, C, F, Hl, Wl)), g.standard_normal((B, A, ad))
    text = g.standard_normal((B, Lc, tdim))
    kp = g.standard_normal((B, 6, H, d // H))
    pos = chunk_positions(1, F, Hl // 2, Wl // 2, A)
    return P, Ws, z, a, text, kp, pos, H


def test_flash_equal_timesteps_reduce_to_the_shared_step():
    P, Ws, z, a, text, kp, pos, H = flash_case(160)
    t = np.array([0.3, 0.9])
    run = lambda ta: oracle.dit_step(z, a, t, text, P, lambda l: (Ws[l], kp, kp), 2, H, 1e-6, 1, pos,
                                     prev_chunk=np.zeros(6, int), t_action=ta)
    v0, a0 = run(None)
    v1, a1 = run(t.copy())
    assert np.allclose(v0, v1, atol=1e-12) and np.allclose(a0, a1, atol=1e-12)
    # a different action timestep changes both outputs (the action rows feed attention)
    v2, a2 = run(np.array([0.7, 0.1]))
    assert not np.allclose(a0, a2) and not np.allclose(v0, v2)


def test_block_per_token_modulation_is_row_wise():
    """With the self-attention gate and the cross-attention output at zero the block acts
    on each token alone, so a per-token modulation must give every row what a uniform
    modulation equal to that row's gives it."""
    g = np.random.default_rng(161)
    B, L, d, H = 2, 5, 16, 2
    W = small_block_weights(d, 32, 162)
    W["mod6"][2] = 0.0
    W["w_co"] = np.zeros((d, d))
    W["b_co"] = np.zeros(d)
    x = g.standard_normal((B, L, d))
    e0 = g.standard_normal((B, L, 6, d)) * 0.5
    e0[:, :, 2] = 0.0
    ctx = g.standard_normal((B, 3, d))
    pos = chunk_positions(0, 1, 1, 3, 2)
    ch = np.zeros(L, int)
    out, _, _ = oracle.dit_block(x, e0, W, H, 1e-6, pos, ch, ctx=ctx)
    for i in range(L):
        row, _, _ = oracle.dit_block(x, e0[:, i], W, H, 1e-6, pos, ch, ctx=ctx)
        assert np.allclose(out[:, i], row[:, i], atol=1e-12)


def test_flash_identity_blocks_closed_form():
    """Identity blocks: the velocity is the head applied to the embeddings, with the video
    rows modulated by e(t) and the action rows by e(t_action), written out per token."""
    P, Ws, z, a, text, kp, pos, H = flash_case(163)
    d = P["w_t2"].shape[0]
    for gate in (2, 5):
        P["w_t6"][gate * d:(gate + 1) * d] = 0.0
        P["b_t6"][gate * d:(gate + 1) * d] = 0.0
    for W in Ws:
        W["mod6"][2] = W["mod6"][5] = 0.0
        W["w_co"] = np.zeros((d, d))
        W["b_co"] = np.zeros(d)
    B, C, F, Hl, Wl = z.shape
    A = a.shape[1]
    t, ta = np.array([0.2, 0.6]), np.array([0.95, 0.05])
    vv, va = oracle.dit_step(z, a, t, text, P, lambda l: (Ws[l], kp, kp), 2, H, 1e-6, 1, pos,
                             prev_chunk=np.zeros(6, int), t_action=ta)

    def e_of(tt):
        s = np.array([math.cos(1000 * tt * 10000 ** (-k / 128)) for k in range(128)]
                     + [math.sin(1000 * tt * 10000 ** (-k / 128)) for k in range(128)])
        h1 = P["w_t1"] @ s + P["b_t1"]
        h1 = h1 / (1 + np.exp(-h1))
        return P["w_t2"] @ h1 + P["b_t2"]

    Hg, Wg = Hl // 2, Wl // 2
    for b in range(B):
        ev, ea = e_of(t[b]), e_of(ta[b])
        for tok in range(F * Hg * Wg + A):
            e = ev if tok < F * Hg * Wg else ea
            sh, sc = P["head_mod2"][0] + e, P["head_mod2"][1] + e
            if tok < F * Hg * Wg:
                f, rem = divmod(tok, Hg * Wg)
                r, s_ = divmod(rem, Wg)
                feat = np.array([z[b, c, f, 2 * r + ph, 2 * s_ + pw] for c in range(C) for ph in range(2)
                                 for pw in range(2)])
                xt = P["w_patch"] @ feat + P["b_patch"]
            else:
                xt = P["w_ain"] @ a[b, tok - F * Hg * Wg] + P["b_ain"]
            ht = (xt - xt.mean()) / math.sqrt(xt.var() + 1e-6) * (1 + sc) + sh
            if tok < F * Hg * Wg:
                out = P["w_hv"] @ ht + P["b_hv"]
                got = np.array([vv[b, c, f, 2 * r + ph, 2 * s_ + pw] for c in range(C) for ph in range(2)
                                for pw in range(2)])
                assert np.allclose(got, out, atol=1e-10)
            else:
                assert np.allclose(va[b, tok - F * Hg * Wg], P["w_ha"] @ ht + P["b_ha"], atol=1e-10)


# ----------------------------------------------------------------------------- denoising loop
def test_euler_follows_the_straight_path_of_eq2():
    """With the path's own velocity z1 - z0 (constant along Eq. 2's interpolation), every
    Euler step lands on the path: after step i the state is t_{i+1} z1 + (1 - t_{i+1}) z0,
    and the last step reaches the clean sample z1, for any schedule."""
    g = np.random.default_rng(130)
    z0, z1 = g.standard_normal((3, 5)), g.standard_normal((3, 5))
    ts = np.array([0.0, 0.03, 0.2, 0.21, 0.6, 0.95, 1.0])
    x = z0.copy()
    for i in range(len(ts) - 1):
        x = oracle.euler_step(x, z1 - z0, ts[i], ts[i + 1])
        assert np.allclose(x, ts[i + 1] * z1 + (1 - ts[i + 1]) * z0, atol=1e-14)
    xN, computed = oracle.denoise(z0, lambda xin, t: z1 - z0, ts)
    assert np.allclose(xN, z1, atol=1e-14) and all(computed)


def test_euler_closed_form_on_a_linear_ode():
    """dx/dt = -x with N uniform Euler steps from 0 to 1 gives x0 (1 - 1/N)^N exactly
    (and tends to x0/e)."""
    x0 = np.array([1.5, -2.0, 0.25])
    for N in (1, 4, 16):
        ts = np.linspace(0.0, 1.0, N + 1)
        xN, _ = oracle.denoise(x0, lambda xin, t: -xin, ts)
        assert np.allclose(xN, x0 * (1 - 1 / N) ** N, rtol=1e-13)


def test_cfg_combine_and_cosine_similarity():
    g = np.random.default_rng(131)
    vc, vu = g.standard_normal(7), g.standard_normal(7)
    assert np.allclose(oracle.cfg_combine(vc, vu, 1.0), vc, atol=1e-15)
    assert np.array_equal(oracle.cfg_combine(vc, vu, 0.0), vu)
    s = 4.5
    assert np.allclose(oracle.cfg_combine(vc, vu, s), [vu[i] + s * (vc[i] - vu[i]) for i in range(7)], atol=1e-15)
    a, b = g.standard_normal(9), g.standard_normal(9)
    dot = sum(a[i] * b[i] for i in range(9))
    na = math.sqrt(sum(x * x for x in a))
    nb = math.sqrt(sum(x * x for x in b))
    assert abs(oracle.cosine_similarity(a, b) - dot / (na * nb)) < 1e-14
    assert abs(oracle.cosine_similarity(a, 3 * a) - 1) < 1e-15
    assert abs(oracle.cosine_similarity(a, -a) + 1) < 1e-15
    assert oracle.cosine_similarity(np.array([1.0, 0.0]), np.array([0.0, 2.0])) == 0.0


def test_dit_caching_skips_a_window_after_similar_velocities():
    """Algorithm 2 with DiT caching: once two successive computed velocities are more
    similar than tau, the next `window` steps reuse the latest one."""
    calls = []

    def const_v(xin, t):
        calls.append(t)
        return np.ones(4)

    ts = np.linspace(0, 1, 9)
    x, computed = oracle.denoise(np.zeros(4), const_v, ts, tau=0.9, window=2)
    assert computed == [True, True, False, False, True, False, False, True]
    assert len(calls) == 4 and np.allclose(x, 1.0)
    # tau above 1 never skips; no tau or a zero window disables caching
    for tau, window in ((1.5, 2), (None, 2), (0.5, 0)):
        _, computed = oracle.denoise(np.zeros(4), const_v, ts, tau=tau, window=window)
        assert all(computed)
    # dissimilar successive velocities never trigger a skip
    flip = {"s": 1.0}

    def alt_v(xin, t):
        flip["s"] = -flip["s"]
        return flip["s"] * np.ones(4)

    _, computed = oracle.denoise(np.zeros(4), alt_v, ts, tau=0.5, window=3)
    assert all(computed)


def _gauss_flow(mu, sd, z):
    """Straight-path flow of Eq. 2 from N(0, 1) noise to N(mu, sd^2) data: its exact
    velocity field E[x1 - x0 | x_t] and the closed-form trajectory x_t = t mu +
    sqrt(t^2 sd^2 + (1 - t)^2) z of the noise sample z."""
    var = lambda t: t * t * sd * sd + (1 - t) ** 2
    vel = lambda x, t: mu + (t * sd * sd - (1 - t)) / var(t) * (x - t * mu)
    path = lambda t: t * mu + np.sqrt(var(t)) * z
    return vel, path


def _lambda_grid(t0, t1, n):
    lam = np.linspace(math.log(t0 / (1 - t0)), math.log(t1 / (1 - t1)), n + 1)
    return [float(v) for v in 1 / (1 + np.exp(-lam))]


def test_unipc_predictor_of_order_one_is_euler():
    """UniP-1 on the straight path (no corrector) is the explicit Euler step: for any
    velocity field, state by state."""
    g = np.random.default_rng(175)
    x0 = g.standard_normal(6)
    vel = lambda x, t: np.sin(3 * x) + t * x - 0.5
    ts = [0.02, 0.1, 0.25, 0.5, 0.8, 0.97, 1.0]
    xe, _ = oracle.denoise(x0, vel, ts)
    xu, _ = oracle.unipc_denoise(x0, vel, ts, order=1, corrector=False)
    assert np.allclose(xu, xe, rtol=1e-13, atol=1e-13)
    assert np.allclose(oracle.unipc_update(x0, 0.3, 0.55, x0 + 0.7 * vel(x0, 0.3)),
                       oracle.euler_step(x0, vel(x0, 0.3), 0.3, 0.55), atol=1e-14)


def test_unipc_update_is_exact_for_polynomial_data_predictions():
    """With data predictions m(lambda) a polynomial P of degree K in lambda = log(t/(1-t)),
    the ODE dx/dt = (m - x)/(1 - t) integrates in closed form, x_t / sigma_t - x_s / sigma_s
    = F(lambda_t) - F(lambda_s) with F = e^lambda sum_k (-1)^k P^(k) (repeated integration
    by parts); one UniPC update with K other data predictions reproduces it, whether the
    points lie before t_s (predictor) or include t itself (corrector)."""
    g = np.random.default_rng(176)
    lam = lambda t: math.log(t / (1 - t))
    for K in range(4):
        c = g.standard_normal((K + 1, 3))                      # P(lambda) = sum_j c_j lambda^j
        P = lambda u: sum(c[j] * u ** j for j in range(K + 1))

        def F(u):
            out, d = 0.0, c.copy()
            for k in range(K + 1):
                out = out + (-1) ** k * sum(d[j] * u ** j for j in range(len(d)))
                d = np.array([j * d[j] for j in range(1, len(d))]) if len(d) > 1 else np.zeros((0, 3))
            return math.exp(u) * out

        x_s = g.standard_normal(3)
        for t_s, t, pts in ((0.4, 0.62, [0.3, 0.21, 0.1]), (0.4, 0.62, [0.62, 0.3, 0.21]),
                            (0.15, 0.5, [0.5, 0.08, 0.04])):
            pts = pts[:K]
            exact = (1 - t) * (x_s / (1 - t_s) + F(lam(t)) - F(lam(t_s)))
            got = oracle.unipc_update(x_s, t_s, t, P(lam(t_s)), [(tj, P(lam(tj))) for tj in pts])
            assert np.allclose(got, exact, rtol=1e-9, atol=1e-9), (K, t_s, t, pts)


def test_unipc_constant_data_prediction_is_exact_at_every_order():
    """Straight paths to one clean sample (m constant): every order lands on the path at
    every corrected state and returns the clean sample at t = 1."""
    g = np.random.default_rng(177)
    x1, z = g.standard_normal(5), g.standard_normal(5)
    ts = [0.05, 0.2, 0.45, 0.7, 0.9, 1.0]
    for order in (1, 2, 3):
        states = []
        xN, computed = oracle.unipc_denoise(ts[0] * x1 + (1 - ts[0]) * z, lambda x, t: (x1 - x) / (1 - t), ts,
                                            order=order, states=states)
        assert np.allclose(xN, x1, atol=1e-12) and all(computed) and len(states) == len(ts) - 2
        for i, st in enumerate(states, start=1):
            assert np.allclose(st, ts[i] * x1 + (1 - ts[i]) * z, atol=1e-12)


def test_unipc_converges_at_order_p_plus_one():
    """On Gaussian data, whose flow is known in closed form, halving the steps of a grid
    uniform in lambda divides the error by ~2^q: q = 1 for Euler and q = p + 1 for UniPC-p
    (the corrector adds one order); without the corrector UniP-p is of order at least p."""
    z = np.linspace(-2.0, 2.0, 9)
    vel, path = _gauss_flow(0.7, 0.4, z)

    def err(n, **kw):
        ts = _lambda_grid(0.05, 0.95, n)
        if kw:
            xN, _ = oracle.unipc_denoise(path(ts[0]), vel, ts, **kw)
        else:
            xN, _ = oracle.denoise(path(ts[0]), vel, ts)
        return np.abs(xN - path(ts[-1])).max()

    def rate(**kw):
        return math.log2(err(32, **kw) / err(64, **kw))

    assert 0.9 < rate() < 1.1
    assert 1.9 < rate(order=1) < 2.1
    assert 2.9 < rate(order=2) < 3.2
    assert 3.7 < rate(order=3) < 4.3
    assert 1.9 < rate(order=2, corrector=False) < 2.2
    assert 2.8 < rate(order=3, corrector=False)
    # the corrected higher orders are also far more accurate at few steps
    assert err(8, order=2) < 0.3 * err(8)


def test_unipc_with_caching_and_schedule_checks():
    """Caching decisions follow the same rule as the Euler loop; schedules that start at
    t = 0 (lambda = -inf) or are not increasing are rejected."""
    ts = list(np.linspace(0.05, 1.0, 9))
    _, computed = oracle.unipc_denoise(np.zeros(4), lambda x, t: np.ones(4), ts, tau=0.9, window=2)
    assert computed == [True, True, False, False, True, False, False, True]
    for bad in ([0.0, 0.5, 1.0], [0.1, 0.5, 0.5, 1.0], [0.2, 0.1, 1.0]):
        with pytest.raises(ValueError):
            oracle.unipc_denoise(np.zeros(2), lambda x, t: x, bad)
    with pytest.raises(ValueError):
        oracle.unipc_denoise(np.zeros(2), lambda x, t: x, [0.1, 1.0], order=4)


# ----------------------------------------------------------------------------- FP8 (E4M3)
def test_e4m3_grid_matches_torch_float8():
    """The E4M3 value set against torch's float8_e4m3fn decoding of every finite code."""
    torch = pytest.importorskip("torch")
    vals = oracle.fp8.e4m3_values()
    assert len(vals) == 127 and vals[-1] == 448.0 and vals[1] == 2.0 ** -9 and np.all(np.diff(vals) > 0)
    codes = torch.arange(0, 127, dtype=torch.uint8).view(torch.float8_e4m3fn)
    assert np.array_equal(codes.to(torch.float64).numpy(), vals)


def test_e4m3_rounding_matches_torch_and_ties_go_even():
    torch = pytest.importorskip("torch")
    g = np.random.default_rng(170)
    x = np.concatenate([g.standard_normal(20000) * s for s in (0.003, 0.1, 1.0, 30.0, 150.0)])
    x = np.clip(x, -448.0, 448.0).astype(np.float32).astype(np.float64)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(oracle.fp8.round_e4m3(x), ref)
    vals = oracle.fp8.e4m3_values()
    mid = (vals[:-1] + vals[1:]) / 2
    got = oracle.fp8.round_e4m3(mid)
    even = np.where(np.arange(len(vals) - 1) % 2 == 0, vals[:-1], vals[1:])
    assert np.array_equal(got, even)
    assert np.array_equal(oracle.fp8.round_e4m3(np.array([500.0, -1e6, 448.0])), [448.0, -448.0, 448.0])


def test_fp8_row_quantization_error_bound():
    """Per-row scales map each row's largest magnitude to 448 exactly; every element in
    the normal range is reproduced within half a unit of its 3-bit mantissa (2^-4)."""
    g = np.random.default_rng(171)
    x = g.standard_normal((16, 300))
    x[3] = 0.0
    q, s = oracle.fp8.quantize_rows(x)
    assert s[3] == 1.0 and not q[3].any()
    rows = [r for r in range(16) if r != 3]
    assert np.allclose(np.max(np.abs(q[rows]), axis=1), 448.0)
    deq = q * s[:, None]
    normal = np.abs(x / s[:, None]) >= 2.0 ** -6
    assert np.all(np.abs(deq - x)[normal] <= 2.0 ** -4 * np.abs(x)[normal] + 1e-300)
    y = oracle.fp8.fp8_linear(q[:2], s[:2], q[2:5], s[2:5])
    assert np.allclose(y, (q[:2] * s[:2, None]) @ (q[2:5] * s[2:5, None]).T, atol=1e-12)


def test_mx_exponent_is_smallest_without_saturation():
    """The block exponent against a brute-force search for the smallest e in [-127, 127]
    with max|block| <= 448 * 2^e, at the boundaries 448 * 2^e and 224 * 2^e (the largest
    magnitude that still takes the exponent below) and over random magnitudes."""
    f = oracle.fp8.mx_exponent

    def brute(a):
        if a == 0.0:
            return 0
        for e in range(-127, 128):
            if a <= 448.0 * 2.0 ** e:
                return e
        return 127

    for e in (-20, -3, 0, 1, 7, 40):
        top = 448.0 * 2.0 ** e
        assert f(top) == e and f(np.nextafter(top, np.inf)) == e + 1
        assert f(224.0 * 2.0 ** e) == e - 1 and f(np.nextafter(224.0 * 2.0 ** e, np.inf)) == e
    g = np.random.default_rng(172)
    amax = np.abs(g.standard_normal(500)) * 10.0 ** g.uniform(-30, 30, 500)
    assert np.array_equal(f(amax), [brute(a) for a in amax])
    assert f(0.0) == 0 and f(2.0 ** -140) == -127 and f(3.0e38) == brute(3.0e38)


@pytest.mark.parametrize("bl", [32, 64])
def test_mx_block_quantization(bl):
    """Blocks of bl elements along the last axis: codes equal torch's float8_e4m3fn rounding
    of x / 2^e, each block's largest scaled magnitude lies in (224, 448], every normal-range
    element is within half a mantissa unit, a block whose maximum is exactly 448 * 2^e gets
    the per-row quantizer's codes, and blocks do not influence each other."""
    torch = pytest.importorskip("torch")
    g = np.random.default_rng(173 + bl)
    nb = 256 // bl
    x = g.standard_normal((6, 256)) * np.repeat(10.0 ** g.uniform(-4, 4, (6, nb)), bl, axis=1)
    x = x.astype(np.float32).astype(np.float64)
    x[2, 2 * bl:3 * bl] = 0.0
    q, e = oracle.fp8.quantize_mx(x, bl)
    assert e.shape == (6, nb) and e[2, 2] == 0 and not q[2, 2 * bl:3 * bl].any()
    scaled = x * np.repeat(2.0 ** -e.astype(np.float64), bl, axis=1)
    ref = torch.from_numpy(scaled).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(q, ref)
    bmax = np.max(np.abs(scaled.reshape(6, nb, bl)), axis=-1)
    nz = bmax > 0
    assert np.all(bmax[nz] > 224.0) and np.all(bmax[nz] <= 448.0)
    deq = oracle.fp8.decode_mx(q, e, bl)
    normal = np.abs(scaled) >= 2.0 ** -6
    assert np.all(np.abs(deq - x)[normal] <= 2.0 ** -4 * np.abs(x)[normal])
    blk = g.standard_normal(bl)
    blk = blk / np.max(np.abs(blk)) * (448.0 * 2.0 ** 5)  # the largest magnitude exactly 448 * 2^5
    qb, eb = oracle.fp8.quantize_mx(blk, bl)
    qr, sr = oracle.fp8.quantize_rows(blk[None])
    assert eb[0] == 5 and sr[0] == 2.0 ** 5 and np.array_equal(qb, qr[0])
    x2 = x.copy()
    x2[:, bl:2 * bl] *= 1000.0
    q2, e2 = oracle.fp8.quantize_mx(x2, bl)
    keep = np.ones(256, bool)
    keep[bl:2 * bl] = False
    assert np.array_equal(q2[:, keep], q[:, keep]) and np.array_equal(np.delete(e2, 1, 1), np.delete(e, 1, 1))


def test_scaled_quantization_in_fp32():
    """One-scale quantization: torch's float8 conversion of the fp32 product x * (1/s),
    and for a power-of-two scale the exact quotient's rounding."""
    torch = pytest.importorskip("torch")
    g = np.random.default_rng(174)
    x = (g.standard_normal(5000) * 3.0).astype(np.float32)
    s = 0.0123
    inv = torch.tensor(1.0, dtype=torch.float32) / torch.tensor(s, dtype=torch.float32)
    ref = (torch.from_numpy(x) * inv).clamp(-448.0, 448.0).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(oracle.fp8.quantize_scaled(x, s), ref)
    assert np.array_equal(oracle.fp8.quantize_scaled(x, 0.125), oracle.fp8.round_e4m3(x.astype(np.float64) / 0.125))


# ----------------------------------------------------------------------------- shared input generator
def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    from synth import bf16_bits
    x = np.concatenate([rnd(10000, seed=110) * 10.0 ** np.arange(-3, 7).repeat(1000),
                        [0.0, -0.0, 1.0, 65504.0, 3.0e38, 1e-40]]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bf16_bits(x), ref)
