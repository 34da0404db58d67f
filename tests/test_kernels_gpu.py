"""GPU parity of each kernel of the step, through its C-ABI entry point, against the
fp64 oracle on the same seeded bf16/fp32 inputs.

Tolerances (relative L2): a bf16 output costs about 2^-9/sqrt(3) = 1.1e-3 from its
final rounding alone, so bf16 results are held to 3e-3 (5e-3 where a bf16
intermediate is rounded as well); fp32 results of fp32 accumulations to 1e-5."""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import dev, host, log, rel_l2, workspace

pytestmark = pytest.mark.gpu


def lib():
    import paper_2602_15922_amd as w
    return w


# ----------------------------------------------------------------------------- LN + modulate
@pytest.mark.parametrize("d,B,L", [(512, 1, 144), (5120, 2, 37), (1280, 3, 5)])
def test_adaln_ln_mod(d, B, L):
    import torch
    w = lib()
    log(f"ln_mod d={d} B={B} L={L}")
    x = synth.normal(5, "x", (B, L, d), 3.0, d, dtype="f32")
    tab = synth.normal(5, "mod6", (6, d), 0.5, d, dtype="f32")
    e0 = synth.normal(5, "e0", (B, 6, d), 0.5, d, dtype="f32")
    xd, tabd, e0d = dev(x), dev(tab), dev(e0)
    h = torch.empty((B, L, d), dtype=torch.bfloat16, device="cuda")
    w.wam_adaln_ln_mod(xd, h, 1e-6, L, shift_a=tabd[0], shift_v=e0d[:, 0], scale_a=tabd[1],
                       scale_v=e0d[:, 1], mod_stride=6 * d)
    torch.cuda.synchronize()
    m = tab.f64[None] + e0.f64
    ref = oracle.modulate(x.f64, m[:, 0][:, None], m[:, 1][:, None], 1e-6)
    assert rel_l2(host(h), ref) <= 3e-3
    # affine LayerNorm without modulation
    g = synth.normal(5, "lnc_gamma", (d,), 0.3, d, dtype="f32")
    bt = synth.normal(5, "lnc_beta", (d,), 0.3, d, dtype="f32")
    w.wam_adaln_ln_mod(xd, h, 1e-6, L, gamma=dev(g), beta=dev(bt))
    torch.cuda.synchronize()
    ref = oracle.layernorm(x.f64, 1e-6, g.f64, bt.f64)
    assert rel_l2(host(h), ref) <= 3e-3


# ----------------------------------------------------------------------------- RoPE + KV append
@pytest.mark.parametrize("Dh,H,B,L,c", [(128, 3, 1, 2 * 3 * 5 + 4, 2), (64, 4, 2, 2 * 2 * 4 + 3, 0)])
def test_rope_qkv_and_cache_append(Dh, H, B, L, c):
    import torch
    w = lib()
    log(f"rope Dh={Dh} H={H} B={B} L={L}")
    d = H * Dh
    Hg, Wg = (3, 5) if Dh == 128 else (2, 4)
    A = L - 2 * Hg * Wg
    pos = w.wam_chunk_positions(c, 2, Hg, Wg, A)
    assert np.array_equal(pos, oracle.chunk_positions(c, 2, Hg, Wg, A))
    cos, sin = w.wam_rope_tables(pos, Dh)
    qkv = synth.normal(6, "x", (B, L, 3 * d), 1.0, Dh)
    Lcap, row0 = L + 23, 11
    kc = torch.full((B, Lcap, H, Dh), 5.0, dtype=torch.bfloat16, device="cuda")
    vc = kc.clone()
    q = torch.empty((B, L, H, Dh), dtype=torch.bfloat16, device="cuda")
    w.wam_rope_qkv(dev(qkv), dev(cos), dev(sin), q, kc, vc, row0, H, Dh)
    torch.cuda.synchronize()
    f = qkv.f64.reshape(B, L, 3, H, Dh)
    assert rel_l2(host(q), oracle.apply_rope(f[:, :, 0], pos)) <= 3e-3
    assert rel_l2(host(kc[:, row0:row0 + L]), oracle.apply_rope(f[:, :, 1], pos)) <= 3e-3
    # v is copied bit for bit; rows outside the chunk's slot are untouched
    assert np.array_equal(host(vc[:, row0:row0 + L]), f[:, :, 2])
    assert (host(kc[:, :row0]) == 5.0).all() and (host(kc[:, row0 + L:]) == 5.0).all()
    assert (host(vc[:, :row0]) == 5.0).all() and (host(vc[:, row0 + L:]) == 5.0).all()


# ----------------------------------------------------------------------------- GEMM epilogues
GEMM_SHAPES = [
    (300, 200, 136),     # small tiles, ragged M, N and K (K % 64 != 0)
    (3152, 5100, 520),   # 128x256 tiles (500 of them, 2 rounds), ragged M, N and K
    (17, 16, 16),        # the action embedding's K
    (130, 203, 72),      # N % 4 != 0: the last column group is stored element by element
    (1000, 12700, 520),  # 256x256 tiles (200, one round), ragged M, N and K
    (570, 15300, 136),   # 192x256 tiles (180, one round, against 300 of 128 rows), ragged M, N and K
    (3152, 13700, 136),  # two column ranges in one launch: 39 columns of 256-row tiles, 15 of 192
    (1347, 16590, 72),   # two column ranges: 256- and 128-row tiles
    (903, 16590, 136),   # two column ranges: 192- and 128-row tiles
]


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
@pytest.mark.parametrize("epi", ["bf16", "gelu", "resid", "f32"])
def test_gemm_epilogues(M, N, K, epi):
    import torch
    w = lib()
    log(f"gemm {epi} M={M} N={N} K={K}")
    A = synth.normal(7, "x", (M, K), 1.0, K)
    W = synth.normal(7, "w_qkv", (N, K), 0.05, K)
    bias = synth.normal(7, "b_qkv", (N,), 0.1, K, dtype="f32")
    acc = oracle.linear(A.f64, W.f64, bias.f64)
    Ad, Wd, bd = dev(A), dev(W), dev(bias)
    N4 = (N + 3) // 4 * 4  # output and gate row strides must be multiples of 4
    if epi in ("bf16", "gelu"):
        out = torch.zeros((M, N4), dtype=torch.bfloat16, device="cuda")
        w.wam_gemm_bf16(Ad, Wd, out, w.WAM_EPI_BF16 if epi == "bf16" else w.WAM_EPI_GELU_BF16, bias=bd)
        torch.cuda.synchronize()
        ref = acc if epi == "bf16" else oracle.gelu_tanh(acc)
        assert rel_l2(host(out[:, :N]), ref) <= 3e-3
        assert not out[:, N:].any()  # padding columns untouched
    elif epi == "f32":
        out = torch.zeros((M, N4), dtype=torch.float32, device="cuda")
        w.wam_gemm_bf16(Ad, Wd, out, w.WAM_EPI_F32, bias=bd)
        torch.cuda.synchronize()
        assert rel_l2(host(out[:, :N]), acc) <= 1e-5
        assert not out[:, N:].any()
    else:
        # x += (gate_a + gate_v[batch]) * (A W^T + b), batches of `rows` rows
        rows = max(1, M // 3)
        nb = (M + rows - 1) // rows
        x0 = synth.normal(7, "e0", (M, N4), 1.0, K, dtype="f32")
        ga = synth.normal(7, "mod6", (N,), 0.5, K, dtype="f32")
        gv = synth.normal(7, "mod6", (nb, 2 * N4), 0.5, K + 1, dtype="f32")
        out = dev(x0)
        gvd = dev(gv)
        w.wam_gemm_bf16(Ad, Wd, out, w.WAM_EPI_RESID_F32, bias=bd, gate_a=dev(ga), gate_v=gvd[:, N4:],
                        gate_stride=2 * N4, gate_rows=rows)
        torch.cuda.synchronize()
        gate = ga.f64[None] + gv.f64[np.arange(M) // rows, N4:N4 + N]
        ref = x0.f64[:, :N] + gate * acc
        got = host(out)
        assert rel_l2(got[:, :N] - x0.f64[:, :N], ref - x0.f64[:, :N]) <= 1e-5
        assert np.array_equal(got[:, N:], x0.f64[:, N:])


def test_gemm_row_remap():
    """A rows and output rows in per-batch groups inside larger buffers (as the
    embedding and head use them)."""
    import torch
    w = lib()
    log("gemm row remap")
    B, R, gapA, gapO, K, N = 3, 50, 70, 64, 128, 96
    A = synth.normal(8, "x", (B, gapA, K), 1.0)
    W = synth.normal(8, "w_o", (N, K), 0.05)
    out = torch.full((B, gapO, N), -1.0, dtype=torch.float32, device="cuda")
    Ad = dev(A)
    w.wam_gemm_bf16(Ad[:, 5:], dev(W), out[:, 3:], w.WAM_EPI_F32, M=B * R, lda=K, a_rows=R,
                    a_batch_stride=gapA * K, ldo=N, out_rows=R, out_batch_stride=gapO * N)
    torch.cuda.synchronize()
    o = host(out)
    ref = oracle.linear(A.f64[:, 5:5 + R], W.f64)
    assert rel_l2(o[:, 3:3 + R], ref) <= 1e-5
    assert (o[:, :3] == -1).all() and (o[:, 3 + R:] == -1).all()


# ----------------------------------------------------------------------------- model pieces
def small_model(wl, bias_std=0.05):
    w = lib()
    P = synth.model_params(wl, bias_std=bias_std)
    top = {k: dev(v) for k, v in P.items()}
    dims = w.make_dims(wl.d, wl.H, wl.Dh, wl.ffn, 0, wl.latent_ch, wl.act_dim, wl.text_dim, wl.freq_dim, wl.eps)
    return P, top, w.make_model(dims, top, [])


def test_time_embedding():
    import torch
    w = lib()
    wl = synth.WORKLOADS["block_d512"].replace(B=3)
    P, top, m = small_model(wl)
    t = synth.uniform(wl.seed, "t", (3,))
    log("time embedding")
    e = torch.empty((3, wl.d), dtype=torch.float32, device="cuda")
    e0 = torch.empty((3, 6, wl.d), dtype=torch.float32, device="cuda")
    w.wam_time_embed_fwd(m, dev(t), e, e0, workspace(w.wam_time_embed_workspace_bytes(m.dims, 3)))
    torch.cuda.synchronize()
    f = {k: v.f64 for k, v in P.items()}
    re, re0 = oracle.time_embedding(t.f64, f["w_t1"], f["b_t1"], f["w_t2"], f["b_t2"], f["w_t6"], f["b_t6"])
    assert rel_l2(host(e), re) <= 1e-4
    assert rel_l2(host(e0), re0) <= 1e-4


def test_text_projection():
    import torch
    w = lib()
    wl = synth.WORKLOADS["block_d512"].replace(text_dim=1024, Lc=40)
    P, top, m = small_model(wl)
    text = synth.normal(wl.seed, "text", (2, wl.Lc, wl.text_dim), 1.0)
    log("text projection")
    ctx = torch.empty((2, wl.Lc, wl.d), dtype=torch.bfloat16, device="cuda")
    w.wam_text_proj_fwd(m, dev(text), ctx, workspace(w.wam_text_proj_workspace_bytes(m.dims, 2, wl.Lc)))
    torch.cuda.synchronize()
    f = {k: v.f64 for k, v in P.items()}
    ref = oracle.text_projection(text.f64, f["w_x1"], f["b_x1"], f["w_x2"], f["b_x2"])
    assert rel_l2(host(ctx), ref) <= 5e-3


def test_embed_and_head():
    import torch
    w = lib()
    wl = synth.WORKLOADS["block_d512"]
    P, top, m = small_model(wl)
    B, C, F, Hl, Wl, A = 2, wl.latent_ch, wl.F, wl.Hl, wl.Wl, wl.A
    z = synth.normal(wl.seed, "z_t", (B, C, F, Hl, Wl), 1.0)
    a = synth.normal(wl.seed, "a_t", (B, A, wl.act_dim), 1.0)
    log("embed + head")
    L = wl.L
    x = torch.full((B, L, wl.d), float("nan"), dtype=torch.float32, device="cuda")
    w.wam_embed_fwd(m, dev(z), dev(a), x, workspace(w.wam_embed_workspace_bytes(m.dims, B, F, Hl, Wl)))
    torch.cuda.synchronize()
    f = {k: v.f64 for k, v in P.items()}
    ref_x = oracle.embed(z.f64, a.f64, f["w_patch"], f["b_patch"], f["w_ain"], f["b_ain"])
    xh = host(x)
    assert np.isfinite(xh).all()
    assert rel_l2(xh, ref_x) <= 1e-5
    e = synth.normal(wl.seed, "e0", (B, wl.d), 0.3, dtype="f32")
    vv = torch.empty((B, C, F, Hl, Wl), dtype=torch.float32, device="cuda")
    va = torch.empty((B, A, wl.act_dim), dtype=torch.float32, device="cuda")
    w.wam_head_fwd(m, x, dev(e), vv, va, workspace(w.wam_head_workspace_bytes(m.dims, B, F, Hl, Wl, A)))
    torch.cuda.synchronize()
    rv, ra = oracle.head(xh, e.f64, f["head_mod2"], wl.Lv, f["w_hv"], f["b_hv"], f["w_ha"], f["b_ha"],
                         wl.eps, C, F, Hl, Wl)
    assert rel_l2(host(vv), rv) <= 5e-3
    assert rel_l2(host(va), ra) <= 5e-3
