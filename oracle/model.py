"""The velocity network u_theta for one chunk, float64: embeddings, DiT block, head.

One denoising step is the call u_theta([z_t, a_t]; KV, c, t, update=False) of the
closed-loop inference algorithm (Appendix C, Algorithm 2): it returns the velocity
of the chunk's video latents and of its action chunk, attending to a KV cache of
earlier chunks (section 3.1, Model Inference; Figure 10b).  The block structure is
the Wan-style DiT the backbone inherits (section 4.1); the paper does not list its
internals, so the forms below are readings.
"""
import numpy as np

from .attention import attention
from .layers import gelu_tanh, layernorm, linear, modulate, silu, timestep_sinusoid
from .rope import apply_rope


def time_embedding(t, w_t1, b_t1, w_t2, b_t2, w_t6, b_t6, freq_dim=256):
    """t (B,) -> e (B, d) = Linear(SiLU(Linear(sinusoid(t)))) and the six AdaLN
    vectors e0 (B, 6, d) = Linear(SiLU(e)), one set per sample since all tokens of a
    chunk share one timestep (section 3.1, Training Objective)."""
    s = timestep_sinusoid(t, freq_dim)
    e = linear(silu(linear(s, w_t1, b_t1)), w_t2, b_t2)
    e0 = linear(silu(e), w_t6, b_t6)
    return e, e0.reshape(e.shape[0], 6, e.shape[1])


def text_projection(text, w_x1, b_x1, w_x2, b_x2):
    """Text-encoder features (B, Lc, text_dim) -> context c (B, Lc, d):
    Linear -> tanh-GELU -> Linear."""
    return linear(gelu_tanh(linear(text, w_x1, b_x1)), w_x2, b_x2)


def patchify(z, ph=2, pw=2):
    """Latent (B, C, F, Hl, Wl) -> tokens (B, F*Hg*Wg, C*ph*pw) with 1x2x2 patches.
    Tokens run frame-major, then row, then column; a token's features run over
    (channel, patch row, patch column)."""
    B, C, F, Hl, Wl = z.shape
    t = z.reshape(B, C, F, Hl // ph, ph, Wl // pw, pw)
    t = t.transpose(0, 2, 3, 5, 1, 4, 6)  # B, f, r, s, C, ph, pw
    return t.reshape(B, F * (Hl // ph) * (Wl // pw), C * ph * pw)


def unpatchify(tok, C, F, Hl, Wl, ph=2, pw=2):
    """Exact inverse of patchify."""
    B = tok.shape[0]
    t = tok.reshape(B, F, Hl // ph, Wl // pw, C, ph, pw)
    t = t.transpose(0, 4, 1, 2, 5, 3, 6)  # B, C, f, r, ph, s, pw
    return t.reshape(B, C, F, Hl, Wl)


def embed(z_t, a_t, w_patch, b_patch, w_ain, b_ain):
    """Chunk tokens: patch-embedded video latents followed by the encoded action
    tokens (the action encoder is a Linear; section 3.1 adds only light encoders)."""
    xv = linear(patchify(z_t), w_patch, b_patch)
    xa = linear(a_t, w_ain, b_ain)
    return np.concatenate([xv, xa], axis=1)


def dit_block(x, e0, W, H, eps, pos, q_chunk, k_prev=None, v_prev=None, prev_chunk=None,
              ctx=None, ctx_kv=None, rows=None):
    """One DiT block over the current chunk rows.

    x (B, L, d) residual; e0 (B, 6, d) time modulation, or (B, L, 6, d) for a
    per-token modulation (DreamZero-Flash: video and action tokens at their own
    timesteps, Appendix D.3); W the block's weights;
    pos (L, 3) RoPE positions and q_chunk (L,) chunk ids of the current rows;
    k_prev / v_prev (B, Lp, H, Dh) the cached K (after RoPE) and V of earlier rows,
    prev_chunk (Lp,) their chunk ids; ctx (B, Lc, d) projected text, or ctx_kv
    (B, Lc, 2d) its precomputed cross K|V.

    Returns (x_out, k_cur, v_cur): the new residual and the current rows' K (after
    RoPE) and V, i.e. what an update pass would append to the cache.

    rows (optional index array): x_out holds only those rows of the new residual.  Every
    row's K and V are still computed (each query sees them), but the queries and all
    token-wise work after the self-attention keys are computed for the listed rows only;
    the block has no other coupling between rows, so this is a row subset of the full
    result.
    """
    B, L, d = x.shape
    Dh = d // H
    if e0.ndim == 4:
        m = W["mod6"][None, None] + e0
        sh1, sc1, g1, sh2, sc2, g2 = (m[:, :, i] for i in range(6))
    else:
        m = W["mod6"][None] + e0
        sh1, sc1, g1, sh2, sc2, g2 = (m[:, i][:, None, :] for i in range(6))

    # self-attention against cache + current chunk; the fused projection's output
    # columns are q | k | v
    h = modulate(x, sh1, sc1, eps)
    w_qkv, b_qkv = W["w_qkv"], W["b_qkv"]
    kv = linear(h, w_qkv[d:], None if b_qkv is None else b_qkv[d:])
    k = apply_rope(kv[..., :d].reshape(B, L, H, Dh), pos)
    v = kv[..., d:].reshape(B, L, H, Dh)
    cur_chunk = np.asarray(q_chunk)
    if rows is not None:
        rows = np.asarray(rows)
        x, h, pos, q_chunk = x[:, rows], h[:, rows], np.asarray(pos)[rows], cur_chunk[rows]
        L = len(rows)
        if e0.ndim == 4:
            sh1, sc1, g1, sh2, sc2, g2 = (a[:, rows] for a in (sh1, sc1, g1, sh2, sc2, g2))
    q = linear(h, w_qkv[:d], None if b_qkv is None else b_qkv[:d]).reshape(B, L, H, Dh)
    q = apply_rope(q, pos)
    if k_prev is None:
        k_all, v_all, k_chunk = k, v, cur_chunk
    else:
        k_all = np.concatenate([k_prev, k], axis=1)
        v_all = np.concatenate([v_prev, v], axis=1)
        k_chunk = np.concatenate([np.asarray(prev_chunk), cur_chunk])
    o = np.stack([attention(q[b], k_all[b], v_all[b], q_chunk, k_chunk) for b in range(B)])
    x = x + g1 * linear(o.reshape(B, L, d), W["w_o"], W["b_o"])

    # cross-attention to the text context: affine LayerNorm, no gate, no RoPE
    hc = layernorm(x, eps, W.get("lnc_gamma"), W.get("lnc_beta"))
    cq = linear(hc, W["w_cq"], W["b_cq"]).reshape(B, L, H, Dh)
    if ctx_kv is None:
        ctx_kv = linear(ctx, W["w_ckv"], W["b_ckv"])
    Lc = ctx_kv.shape[1]
    ck = ctx_kv[..., :d].reshape(B, Lc, H, Dh)
    cv = ctx_kv[..., d:].reshape(B, Lc, H, Dh)
    zq, zk = np.zeros(L, int), np.zeros(Lc, int)
    oc = np.stack([attention(cq[b], ck[b], cv[b], zq, zk) for b in range(B)])
    x = x + linear(oc.reshape(B, L, d), W["w_co"], W["b_co"])

    # feed-forward
    u = gelu_tanh(linear(modulate(x, sh2, sc2, eps), W["w_f1"], W["b_f1"]))
    x = x + g2 * linear(u, W["w_f2"], W["b_f2"])
    return x, k, v


def head(x, e, head_mod2, Lv, w_hv, b_hv, w_ha, b_ha, eps, C, F, Hl, Wl):
    """Output head: AdaLN with (shift, scale) = head_mod2 + e (e of shape (B, d), or
    (B, L, d) per token), then the video decoder (Linear to patch features,
    unpatchified) on the first Lv rows and the action decoder (Linear) on the rest."""
    e = e[:, None, :] if e.ndim == 2 else e
    m = head_mod2[None, None] + e[:, :, None, :]
    h = modulate(x, m[:, :, 0], m[:, :, 1], eps)
    v_video = unpatchify(linear(h[:, :Lv], w_hv, b_hv), C, F, Hl, Wl)
    v_action = linear(h[:, Lv:], w_ha, b_ha)
    return v_video, v_action


def dit_step(z_t, a_t, t, text, P, layers, n_layers, H, eps, chunk_index, pos,
             prev_chunk=None, q_chunk=None, ctx=None, t_action=None, depths=None):
    """u_theta([z_t, a_t]; KV, c, t, update=False) for one chunk.

    z_t (B, C, F, Hl, Wl) noisy latents; a_t (B, A, act_dim) noisy actions; t (B,);
    text (B, Lc, text_dim) text features; P the model-level weights; layers(l)
    returns (W_l, k_prev_l, v_prev_l), so callers can stream one layer at a time.
    t_action (B,), when given, is the action tokens' own timestep (DreamZero-Flash,
    Appendix D.3): their AdaLN and head modulation come from it, the video tokens'
    from t.  Returns (v_video, v_action); with depths (a list of block counts), the
    list of (v_video, v_action) the head gives after each of those many blocks."""
    B, C, F, Hl, Wl = z_t.shape
    e, e0 = time_embedding(t, P["w_t1"], P["b_t1"], P["w_t2"], P["b_t2"], P["w_t6"], P["b_t6"])
    if t_action is not None:
        ea, e0a = time_embedding(t_action, P["w_t1"], P["b_t1"], P["w_t2"], P["b_t2"], P["w_t6"], P["b_t6"])
        Lv_, A_ = F * (Hl // 2) * (Wl // 2), a_t.shape[1]
        e = np.concatenate([np.repeat(e[:, None], Lv_, 1), np.repeat(ea[:, None], A_, 1)], axis=1)
        e0 = np.concatenate([np.repeat(e0[:, None], Lv_, 1), np.repeat(e0a[:, None], A_, 1)], axis=1)
    if ctx is None:
        ctx = text_projection(text, P["w_x1"], P["b_x1"], P["w_x2"], P["b_x2"])
    x = embed(z_t, a_t, P["w_patch"], P["b_patch"], P["w_ain"], P["b_ain"])
    L = x.shape[1]
    if q_chunk is None:
        q_chunk = np.full(L, chunk_index)
    Lv = F * (Hl // 2) * (Wl // 2)

    def velocity(x):
        return head(x, e, P["head_mod2"], Lv, P["w_hv"], P["b_hv"], P["w_ha"], P["b_ha"], eps, C, F, Hl, Wl)

    taps = []
    for layer in range(n_layers):
        W, kp, vp = layers(layer)
        x, _, _ = dit_block(x, e0, W, H, eps, pos, q_chunk, kp, vp, prev_chunk, ctx=ctx)
        if depths is not None and layer + 1 in depths:
            taps.append(velocity(x))
    return velocity(x) if depths is None else taps


def dit_update(z, a, t, text, P, layers, n_layers, H, eps, pos, q_chunk, prev_chunk=None, ctx=None):
    """u_theta([z, a]; KV, c, t, update=True): the cache-update pass of the
    closed-loop algorithm (Appendix C, Algorithm 2), run on clean observed latents
    (the algorithm passes no actions, i.e. a with zero rows; the chunk's timestep t
    is whatever the caller uses for clean content).

    The current rows may span several chunks (q_chunk holds each row's chunk id,
    pos its RoPE position); each attends to the cached rows and to the current rows
    of its own and earlier chunks (Figure 10b).  Returns [(k_l, v_l)] per layer: the
    K (after RoPE) and V of the current rows that the pass appends to layer l's
    cache.  The velocities of this call are discarded by the algorithm and are not
    computed."""
    e, e0 = time_embedding(t, P["w_t1"], P["b_t1"], P["w_t2"], P["b_t2"], P["w_t6"], P["b_t6"])
    if ctx is None:
        ctx = text_projection(text, P["w_x1"], P["b_x1"], P["w_x2"], P["b_x2"])
    x = embed(z, a, P["w_patch"], P["b_patch"], P["w_ain"], P["b_ain"])
    new_kv = []
    for layer in range(n_layers):
        W, kp, vp = layers(layer)
        x, k, v = dit_block(x, e0, W, H, eps, pos, q_chunk, kp, vp, prev_chunk, ctx=ctx)
        new_kv.append((k, v))
    return new_kv
