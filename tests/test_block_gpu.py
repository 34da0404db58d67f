"""GPU parity of wam_dit_block_fwd against the fp64 oracle (relative L2 <= 2e-2 on the
block output), the cache rows it appends, and the block-level properties: zero-gate
identity (exact) and KV-cache equivalence (bitwise)."""
import numpy as np
import pytest

import oracle
import synth
from dit_cases import BlockCase, dims_of, f64, gpu_rope_tables, oracle_positions, prev_chunk_ids, upload_cache
from gpu_helpers import dev, host, log, rel_l2, workspace

pytestmark = pytest.mark.gpu
TOL = 2e-2


def lib():
    import paper_2602_15922_amd as w
    return w


def check_block(case, x, kc, vc, tol=TOL, ref=None):
    wl = case.wl
    rx, rk, rv = case.run_oracle() if ref is None else ref
    xg = host(x)
    x0 = case.x.f64
    err, derr = rel_l2(xg, rx), rel_l2(xg - x0, rx - x0)
    print(f"  block rel L2 {err:.2e}, of the update {derr:.2e}", flush=True)
    assert err <= tol and derr <= tol
    rows = slice(wl.cache_rows, wl.cache_rows + wl.L)
    assert rel_l2(host(kc[:, rows]), rk) <= 5e-3
    assert rel_l2(host(vc[:, rows]), rv) <= 5e-3
    if wl.cache_rows:  # cached rows are read, never written
        assert np.array_equal(host(kc[:, :wl.cache_rows]), case.kc.f64)


@pytest.mark.parametrize("variant", ["plain", "bias_cache_batch2"])
def test_block_d512(variant):
    """d=512, 8 heads of 64, FFN 2048, 2x8x8 video + 16 action tokens, 32 text tokens,
    modulation vector N(0,1)."""
    wl = synth.WORKLOADS["block_d512"]
    bias = 0.0
    if variant != "plain":
        wl = wl.replace(B=2, n_cached=2)
        bias = 0.05
    log(f"block d512 {variant}")
    case = BlockCase(wl, bias_std=bias, e0=synth.normal(wl.seed, "e0", (wl.B, 6, wl.d), 0.3, dtype="f32")
                     if variant != "plain" else None)
    x, kc, vc = case.run_gpu()
    check_block(case, x, kc, vc)


def test_block_14b_with_time_and_text_conditioning():
    """One 14B-class block (d=5120, 40x128, FFN 13824) over 3152 rows with a 6304-row
    cache; e0 from the time MLP of t ~ U(0,1) and ctx from the text projection of
    512x4096 features, all on the GPU, against the same chain in the oracle."""
    import torch
    w = lib()
    wl = synth.WORKLOADS["block_14b"]
    log("block 14b: inputs")
    P = synth.model_params(wl)
    t = synth.uniform(wl.seed, "t", (1,))
    text = synth.normal(wl.seed, "text", (1, wl.Lc, wl.text_dim), 1.0)
    top = {k: dev(v) for k, v in P.items()}
    m = w.make_model(dims_of(wl, 0), top, [])
    e = torch.empty((1, wl.d), dtype=torch.float32, device="cuda")
    e0 = torch.empty((1, 6, wl.d), dtype=torch.float32, device="cuda")
    ctx = torch.empty((1, wl.Lc, wl.d), dtype=torch.bfloat16, device="cuda")
    log("block 14b: time embedding + text projection")
    w.wam_time_embed_fwd(m, dev(t), e, e0, workspace(w.wam_time_embed_workspace_bytes(m.dims, 1)))
    w.wam_text_proj_fwd(m, dev(text), ctx, workspace(w.wam_text_proj_workspace_bytes(m.dims, 1, wl.Lc)))
    torch.cuda.synchronize()
    f = f64(P)
    _, re0 = oracle.time_embedding(t.f64, f["w_t1"], f["b_t1"], f["w_t2"], f["b_t2"], f["w_t6"], f["b_t6"])
    rctx = oracle.text_projection(text.f64, f["w_x1"], f["b_x1"], f["w_x2"], f["b_x2"])
    case = BlockCase(wl)
    log("block 14b: block on the GPU")
    x, kc, vc = case.run_gpu(e0_dev=e0, ctx_dev=ctx)
    # the oracle consumes its own e0 and ctx (the fp64 chain), not the GPU's
    log("block 14b: oracle")
    check_block(case, x, kc, vc, ref=case.run_oracle(e0=re0, ctx=rctx))


def test_block_zero_gates_is_exact_identity_at_14b_shape():
    """gate1 = gate2 = 0 and W_co = b_co = 0: the fp32 residual passes through untouched."""
    import torch
    w = lib()
    wl = synth.WORKLOADS["block_14b"]
    d, L = wl.d, wl.L
    log("block 14b zero gates")
    g = torch.Generator(device="cuda").manual_seed(5)

    def rn(*s, std=0.02):
        return (torch.randn(*s, generator=g, device="cuda") * std).to(torch.bfloat16)

    Wd = {"w_qkv": rn(3 * d, d), "w_o": rn(d, d), "w_cq": rn(d, d), "w_ckv": rn(2 * d, d),
          "w_co": torch.zeros(d, d, dtype=torch.bfloat16, device="cuda"), "w_f1": rn(wl.ffn, d),
          "w_f2": rn(d, wl.ffn), "mod6": torch.randn(6, d, generator=g, device="cuda") * 0.1}
    Wd["mod6"][2] = 0.0
    Wd["mod6"][5] = 0.0
    e0 = torch.randn(1, 6, d, generator=g, device="cuda") * 0.3
    e0[:, 2] = 0.0
    e0[:, 5] = 0.0
    x = torch.randn(1, L, d, generator=g, device="cuda")
    x_in = x.clone()
    kc = rn(1, wl.Lcap, wl.H, wl.Dh, std=1.0)
    vc = rn(1, wl.Lcap, wl.H, wl.Dh, std=1.0)
    ctx = rn(1, wl.Lc, d, std=1.0)
    cos, sin = gpu_rope_tables(wl)
    dims = dims_of(wl, 1)
    w.wam_dit_block_fwd(dims, w.make_block_weights(Wd), x, e0, cos, sin, kc, vc, wl.cache_rows,
                        w.cached_chunks(wl.cache_rows, L), ctx=ctx,
                        ws=workspace(w.wam_block_workspace_bytes(dims, 1, L, wl.Lc)))
    torch.cuda.synchronize()
    assert torch.equal(x, x_in)


def test_block_kv_cache_equivalence_bitwise():
    """Three chunks in one block call (block-causal mask) equal three sequential cached
    calls, each appending its chunk's K/V (Figure 10b): every per-row computation is the
    same, so the results agree bit for bit."""
    import torch
    w = lib()
    wl = synth.WORKLOADS["block_d512"].replace(n_cached=0)
    B, d, H, Dh, L, Lc = 1, wl.d, wl.H, wl.Dh, wl.L, wl.Lc
    W = {k: dev(v) for k, v in synth.block_params(wl, 3, 0.05, mod_std=0.3).items()}
    e0 = dev(synth.normal(0, "e0", (B, 6, d), 0.3, 3, dtype="f32"))
    ctx = dev(synth.normal(0, "ctx", (B, Lc, d), 1.0, 3))
    x3 = dev(synth.normal(0, "x", (B, 3 * L, d), 1.0, 3, dtype="f32"))
    pos = np.concatenate([w.wam_chunk_positions(c, wl.F, wl.Hg, wl.Wg, wl.A) for c in range(3)])
    cos, sin = (dev(a) for a in w.wam_rope_tables(pos, Dh))
    dims = dims_of(wl, 1)
    log("block kv-cache equivalence")
    # one call, three query chunks
    kA = torch.zeros((B, 3 * L, H, Dh), dtype=torch.bfloat16, device="cuda")
    vA = torch.zeros_like(kA)
    xA = x3.clone()
    w.wam_dit_block_fwd(dims, w.make_block_weights(W), xA, e0, cos, sin, kA, vA, 0,
                        w.make_chunks([L] * 3, [L] * 3, [0, 1, 2]), ctx=ctx,
                        ws=workspace(w.wam_block_workspace_bytes(dims, B, 3 * L, Lc)))
    # three cached calls
    kB = torch.zeros_like(kA)
    vB = torch.zeros_like(kA)
    ws = workspace(w.wam_block_workspace_bytes(dims, B, L, Lc))
    outs = []
    for c in range(3):
        xc = x3[:, c * L:(c + 1) * L].clone()
        w.wam_dit_block_fwd(dims, w.make_block_weights(W), xc, e0, cos[c * L:(c + 1) * L].contiguous(),
                            sin[c * L:(c + 1) * L].contiguous(), kB, vB, c * L,
                            w.make_chunks([L] * (c + 1), [L], [c]), ctx=ctx, ws=ws)
        outs.append(xc)
    torch.cuda.synchronize()
    assert torch.equal(kA, kB) and torch.equal(vA, vB)
    assert torch.equal(xA, torch.cat(outs, dim=1))


def test_block_precomputed_cross_kv_matches():
    import torch
    w = lib()
    wl = synth.WORKLOADS["block_d512"].replace(B=2)
    case = BlockCase(wl, bias_std=0.05)
    log("block precomputed cross kv")
    x1, _, _ = case.run_gpu()
    Wd = {k: dev(v) for k, v in case.W.items()}
    ctx = dev(case.ctx)
    kv = torch.empty((wl.B, wl.Lc, 2 * wl.d), dtype=torch.bfloat16, device="cuda")
    w.wam_gemm_bf16(ctx.view(-1, wl.d), Wd["w_ckv"], kv.view(-1, 2 * wl.d), w.WAM_EPI_BF16, bias=Wd["b_ckv"])
    x = dev(case.x)
    kc, vc = upload_cache(wl, None, None, wl.B)
    cos, sin = gpu_rope_tables(wl)
    dims = dims_of(wl, 1)
    w.wam_dit_block_fwd(dims, w.make_block_weights(Wd), x, dev(case.e0), cos, sin, kc, vc, 0,
                        w.cached_chunks(0, wl.L), ctx_kv=kv,
                        ws=workspace(w.wam_block_workspace_bytes(dims, wl.B, wl.L, wl.Lc)))
    torch.cuda.synchronize()
    assert torch.equal(x, x1)


@pytest.mark.timeout(900)
def test_block_b2_3view_sampled_rows():
    """One 14B-class block at the two-sample, three-view shape: batch 2 of 9392 rows
    (2 frames x 30 x 156 patches + 32 actions) after six cached chunks (56352 rows, 65744
    keys), e0 from the time MLP of two different t and ctx from the text projection, all
    on the GPU.  The oracle takes every row's K and V (they are appended, and every query
    sees them) and the rest of the block on sampled rows of both samples.  The residual,
    the cache and the cached rows are drawn on the device from seeded streams (the host
    generator would take minutes at this size); the oracle reads host copies."""
    import torch
    w = lib()
    wl = synth.WORKLOADS["step_14b_b2_3view"]
    B, L, d, H, Dh = wl.B, wl.L, wl.d, wl.H, wl.Dh
    log(f"block b2 3-view B={B} L={L} Lk={wl.Lk}: inputs")
    P = synth.model_params(wl)
    t = synth.uniform(wl.seed, "t", (B,))
    assert abs(float(t.f64[0] - t.f64[1])) > 1e-3
    text = synth.normal(wl.seed, "text", (B, wl.Lc, wl.text_dim), 1.0)
    W = synth.block_params(wl, 0)
    top = {k: dev(v) for k, v in P.items()}
    m = w.make_model(dims_of(wl, 0), top, [])
    e = torch.empty((B, d), dtype=torch.float32, device="cuda")
    e0 = torch.empty((B, 6, d), dtype=torch.float32, device="cuda")
    ctx = torch.empty((B, wl.Lc, d), dtype=torch.bfloat16, device="cuda")
    w.wam_time_embed_fwd(m, dev(t), e, e0, workspace(w.wam_time_embed_workspace_bytes(m.dims, B)))
    w.wam_text_proj_fwd(m, dev(text), ctx, workspace(w.wam_text_proj_workspace_bytes(m.dims, B, wl.Lc)))
    x = synth.device_normal(wl.seed, "x", (B, L, d), 1.0, dtype="f32")
    kc = torch.zeros((B, wl.Lcap, H, Dh), dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    kc[:, :wl.cache_rows] = synth.device_normal(wl.seed, "k_cache", (B, wl.cache_rows, H, Dh))
    vc[:, :wl.cache_rows] = synth.device_normal(wl.seed, "v_cache", (B, wl.cache_rows, H, Dh))
    x_in = host(x)
    Wd = {k: dev(v) for k, v in W.items()}
    cos, sin = gpu_rope_tables(wl)
    dims = dims_of(wl, 1)
    log("block b2 3-view: GPU")
    w.wam_dit_block_fwd(dims, w.make_block_weights(Wd), x, e0, cos, sin, kc, vc, wl.cache_rows,
                        w.cached_chunks(wl.cache_rows, L), ctx=ctx,
                        ws=workspace(w.wam_block_workspace_bytes(dims, B, L, wl.Lc)))
    torch.cuda.synchronize()
    del Wd
    rng = np.random.default_rng(7)
    rows = sorted({0, 1, 127, 128, 4679, 4680, 9215, 9216, wl.Lv - 1, wl.Lv, L - 1}
                  | set(rng.integers(0, L, 53).tolist()))
    rows = np.array(rows)
    xg = host(x[:, rows])
    app = slice(wl.cache_rows, wl.cache_rows + L)
    kg, vg = host(kc[:, app]), host(vc[:, app])
    log("block b2 3-view: oracle")
    f = f64(P)
    _, re0 = oracle.time_embedding(t.f64, f["w_t1"], f["b_t1"], f["w_t2"], f["b_t2"], f["w_t6"], f["b_t6"])
    rctx = oracle.text_projection(text.f64, f["w_x1"], f["b_x1"], f["w_x2"], f["b_x2"])
    kp, vp = host(kc[:, :wl.cache_rows]), host(vc[:, :wl.cache_rows])
    del kc, vc
    rx, rk, rv = oracle.dit_block(x_in, re0, f64(W), H, wl.eps, oracle_positions(wl), np.full(L, wl.n_cached),
                                  kp, vp, prev_chunk_ids(wl), ctx=rctx, rows=rows)
    x0 = x_in[:, rows]
    err, derr = rel_l2(xg, rx), rel_l2(xg - x0, rx - x0)
    ek, ev = rel_l2(kg, rk), rel_l2(vg, rv)
    print(f"  {len(rows)} rows per sample: block rel L2 {err:.2e}, of the update {derr:.2e}; "
          f"appended K {ek:.2e} V {ev:.2e}", flush=True)
    for b in range(B):
        print(f"  sample {b}: update rel L2 {rel_l2(xg[b] - x0[b], rx[b] - x0[b]):.2e}", flush=True)
    assert err <= TOL and derr <= TOL
    assert ek <= 5e-3 and ev <= 5e-3
