"""Host-only checks of the C ABI (no GPU needed): the library loads, exports every
symbol the header declares, and rejects bad arguments with a status and a message
before touching the GPU."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def lib():
    import paper_2602_15922_amd as w
    return w


def header_functions():
    src = open(os.path.join(ROOT, "include", "wamdit.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(wam_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    w = lib()
    declared = header_functions()
    assert len(declared) >= 20
    L = w.lib()
    for name in declared:
        assert hasattr(L, name), name
    assert sorted(w.binding.EXPORTED) == declared
    assert w.wam_abi_version() == 7


def test_struct_sizes_match_the_header_layout():
    w = lib()
    b = w.binding
    assert C.sizeof(b.wam_chunks) == 4 * (1 + 17 + 1 + 17 + 16)
    assert C.sizeof(b.wam_dims) == 10 * 4
    assert C.sizeof(b.wam_block_weights) == 18 * 8
    assert C.sizeof(b.wam_block_fp8) == 14 * 8
    # sizes printed by a C++ compile of include/wamdit.h
    assert C.sizeof(b.wam_flow_dims) == 32
    assert C.sizeof(b.wam_denoise_params) == 56
    assert C.sizeof(b.wam_unipc_coef) == 44
    assert C.sizeof(b.wam_step_io) == 368
    assert C.sizeof(b.wam_block_io) == 312
    assert C.sizeof(b.wam_model) == 200


def _status(fn, *args):
    return fn(*args)


def test_attention_rejects_bad_arguments_without_a_gpu():
    w = lib()
    b = w.binding
    L = w.lib()

    def call(**kw):
        d = b.wam_attn_desc(B=1, H=2, Dh=128, Lq=10, Lk=20, q_tok_stride=256, q_batch_stride=2560,
                            kv_tok_stride=256, kv_batch_stride=5120, o_tok_stride=256, o_batch_stride=2560,
                            scale=0.0, ch=w.make_chunks([10, 10], [10], [1]))
        ptrs = dict(q=4096, k=8192, v=12288, o=16384)
        for k_, v_ in kw.items():
            if k_ in ptrs:
                ptrs[k_] = v_
            elif k_ == "ch":
                d.ch = v_
            else:
                setattr(d, k_, v_)
        return L.wam_attn_blockcausal(C.byref(d), ptrs["q"], ptrs["k"], ptrs["v"], ptrs["o"], None)

    assert call(Dh=96) == b.WAM_EUNSUPPORTED
    assert call(q=0) == b.WAM_EINVAL and b"q is NULL" in L.wam_last_error()
    assert call(k=8200) == b.WAM_EINVAL and b"aligned" in L.wam_last_error()
    assert call(q_tok_stride=100) == b.WAM_EINVAL
    assert call(Lk=21) == b.WAM_EINVAL  # chunks do not cover Lk
    assert call(ch=w.make_chunks([10, 10], [10], [2])) == b.WAM_EINVAL  # chunk id out of range
    assert call(ch=w.make_chunks([0, 20], [10], [0])) == b.WAM_EINVAL  # sees no key
    assert call(ch=w.make_chunks([10, 10], [5, 5], [1, 0])) == b.WAM_EINVAL  # ids decreasing
    assert call(B=-1) == b.WAM_EINVAL
    # nothing to do is not an error, and needs no valid pointers
    assert call(Lq=0, ch=w.make_chunks([10, 10], [0], [1]), q=0, o=0) == b.WAM_OK


def test_gemm_and_block_reject_bad_arguments():
    w = lib()
    b = w.binding
    L = w.lib()
    g = b.wam_gemm_desc(M=10, N=10, K=12, epilogue=0, A=4096, lda=16, W=8192, ldw=16, out=16384, ldo=10)
    assert L.wam_gemm_bf16(C.byref(g), None) == b.WAM_EINVAL  # K % 8
    g.K = 16
    g.epilogue = 9
    assert L.wam_gemm_bf16(C.byref(g), None) == b.WAM_EINVAL
    dims = w.make_dims(d=512, H=8, Dh=64, ffn=2048, n_layers=1)
    wts = b.wam_block_weights()
    io = b.wam_block_io(B=1, L=10, Lc=4, Lcap=8, cache_len=0, ch=w.cached_chunks(0, 10))
    assert L.wam_dit_block_fwd(C.byref(dims), C.byref(wts), C.byref(io), None, 0, None) == b.WAM_EINVAL
    bad = w.make_dims(d=500, H=5, Dh=100, ffn=2048, n_layers=1)
    assert L.wam_dit_block_fwd(C.byref(bad), C.byref(wts), C.byref(io), None, 0, None) == b.WAM_EUNSUPPORTED
    assert L.wam_block_workspace_bytes(C.byref(dims), 1, 144, 32) > 0
    assert L.wam_dit_step_fwd(None, None, None, 0, None) == b.WAM_EINVAL
    assert L.wam_dit_update_fwd(None, None, None, 0, None) == b.WAM_EINVAL
    assert L.wam_denoise_chunk(None, None, None, None, 0, None) == b.WAM_EINVAL
    fd = b.wam_flow_dims(B=3, cfg=1, cfg_scale=2.0, n_video=8, n_action=0)
    assert L.wam_flow_step(C.byref(fd), None, None, None, 4096, None, 0.0, 0.1, 8192, None, None) == b.WAM_EINVAL
    assert L.wam_cosine_similarity(4096, 8192, 16, None, 0, 12288, None) == b.WAM_EWORKSPACE


def test_rope_tables_and_positions_agree_with_the_oracle():
    w = lib()
    for Dh, (c, F, Hg, Wg, A) in [(128, (3, 2, 30, 52, 32)), (64, (0, 2, 8, 8, 16))]:
        pos = w.wam_chunk_positions(c, F, Hg, Wg, A)
        assert np.array_equal(pos, oracle.chunk_positions(c, F, Hg, Wg, A))
        cos, sin = w.wam_rope_tables(pos, Dh)
        phi = oracle.rope_angles(pos, Dh)
        # double-precision tables rounded to fp32: within one fp32 ulp of 1
        assert np.max(np.abs(cos - np.cos(phi))) <= 1.2e-7
        assert np.max(np.abs(sin - np.sin(phi))) <= 1.2e-7


def test_loader_fails_loudly_without_the_library(monkeypatch, tmp_path):
    w = lib()
    monkeypatch.setattr(w.binding, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(w.binding, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        w.binding.lib()


def test_fp8_entry_points_reject_bad_arguments_without_a_gpu():
    """Every check below fails before any launch (fake device addresses, no GPU)."""
    w = lib()
    b = w.binding
    L = w.lib()

    def attn(Dh=128, v_scale=1.0, q=4096, qe=8192, k=12288, ke=16384, v=20480, o=24576, **kw):
        d = b.wam_attn_desc(B=1, H=2, Dh=Dh, Lq=10, Lk=20, q_tok_stride=256, q_batch_stride=2560,
                            kv_tok_stride=256, kv_batch_stride=5120, o_tok_stride=256, o_batch_stride=2560,
                            scale=0.0, ch=w.make_chunks([10, 10], [10], [1]))
        for k_, v_ in kw.items():
            setattr(d, k_, v_)
        return L.wam_attn_blockcausal_fp8(C.byref(d), q, qe, k, ke, v, v_scale, o, None)

    assert attn(Dh=64) == b.WAM_EUNSUPPORTED
    assert attn(v_scale=0.0) == b.WAM_EINVAL and b"v_scale" in L.wam_last_error()
    assert attn(v_scale=float("nan")) == b.WAM_EINVAL
    assert attn(qe=0) == b.WAM_EINVAL and b"q_exp is NULL" in L.wam_last_error()
    assert attn(q=4100) == b.WAM_EINVAL and b"aligned" in L.wam_last_error()
    assert attn(ke=8194) == b.WAM_EINVAL and b"aligned" in L.wam_last_error()
    assert attn(q_tok_stride=320) == b.WAM_EINVAL  # not a multiple of Dh bytes
    assert attn(Lk=21) == b.WAM_EINVAL  # chunks do not cover Lk
    q = L.wam_quantize_mx_fp8
    assert q(4, 33, 4096, 40, 8192, 40, 12288, None) == b.WAM_EINVAL  # cols % 32
    assert q(4, 64, 4096, 68, 8192, 64, 12288, None) == b.WAM_EINVAL  # ldx % 8
    assert q(4, 64, 4100, 64, 8192, 64, 12288, None) == b.WAM_EINVAL  # x alignment
    assert L.wam_quantize_scaled_fp8(7, 4096, 1.0, 8192, None) == b.WAM_EINVAL
    assert L.wam_quantize_scaled_fp8(8, 4096, -1.0, 8192, None) == b.WAM_EINVAL
    r = L.wam_rope_qkv_fp8
    assert r(1, 4, 2, 64, 4096, 8192, 8192, 0, 0, 12288, 16384, 20480, 1.0, 8, 0, None) == b.WAM_EUNSUPPORTED
    assert r(1, 4, 2, 128, 4096, 8192, 8192, 24576, 0, 12288, 16384, 20480, 1.0, 8, 0, None) == b.WAM_EINVAL
    assert r(1, 4, 2, 128, 4096, 8192, 8192, 0, 0, 12288, 16384, 20480, 1.0, 8, 5, None) == b.WAM_EINVAL  # row0+L>Lcap

    def gm(M=300, N=256, K=256, epi=b.WAM_EPI_BF16, a_scale=None, a_exp=4096, a_lde=None, out_exp=None, o_lde=0,
           out=8192):
        g = b.wam_gemm_desc(M=M, N=N, K=K, epilogue=epi, A=12288, lda=K, a_batch_stride=0, a_rows=0, W=16384,
                            ldw=K, bias=None, out=out, ldo=N, out_batch_stride=0, out_rows=0, gate_a=None,
                            gate_v=None, gate_stride=0, gate_rows=0)
        return L.wam_gemm_fp8_mx(C.byref(g), a_scale, a_exp, 4 * M if a_lde is None else a_lde, 20480, out_exp,
                                 o_lde, None)

    gelu = b.WAM_EPI_GELU_BF16
    assert gm(a_scale=24576) == b.WAM_EINVAL and b"exactly one" in L.wam_last_error()
    assert gm(a_exp=None) == b.WAM_EINVAL
    assert gm(K=192) == b.WAM_EUNSUPPORTED  # block-scaled A: K % 128
    assert gm(epi=gelu) == b.WAM_EUNSUPPORTED  # block-scaled A: bf16 or residual epilogue
    assert gm(a_lde=4 * 300 - 4) == b.WAM_EINVAL and b"a_lde" in L.wam_last_error()
    assert gm(a_exp=4098) == b.WAM_EINVAL and b"aligned" in L.wam_last_error()
    assert gm(out_exp=28672, o_lde=1200, epi=gelu) == b.WAM_EUNSUPPORTED  # both sides block-scaled
    blk_out = dict(a_exp=None, a_scale=24576, out_exp=28672, o_lde=1200)
    assert gm(epi=b.WAM_EPI_BF16, **blk_out) == b.WAM_EUNSUPPORTED  # a block-scaled output is GELU's
    assert gm(epi=gelu, N=192, **blk_out) == b.WAM_EUNSUPPORTED  # N % 128
    assert gm(epi=gelu, out=8194, **blk_out) == b.WAM_EINVAL and b"aligned" in L.wam_last_error()
    assert gm(epi=gelu, **dict(blk_out, o_lde=1198)) == b.WAM_EINVAL  # o_lde % 4, >= 4 M

    def am(Dh=128, o8=24576, oe=28672, lde=80, fp8=False, **kw):
        d = b.wam_attn_desc(B=2, H=2, Dh=Dh, Lq=10, Lk=20, q_tok_stride=256, q_batch_stride=2560,
                            kv_tok_stride=256, kv_batch_stride=5120, o_tok_stride=256, o_batch_stride=2560,
                            scale=0.0, ch=w.make_chunks([10, 10], [10], [1]))
        for k_, v_ in kw.items():
            setattr(d, k_, v_)
        if fp8:
            return L.wam_attn_blockcausal_fp8_mx(C.byref(d), 4096, 8192, 12288, 16384, 20480, 1.0, o8, oe, lde, None)
        return L.wam_attn_blockcausal_mx(C.byref(d), 4096, 12288, 20480, o8, oe, lde, None)

    for f8 in (False, True):
        assert am(fp8=f8, oe=0) == b.WAM_EINVAL and b"o_exp" in L.wam_last_error()
        assert am(fp8=f8, lde=76) == b.WAM_EINVAL and b"o_lde" in L.wam_last_error()  # < 4 B Lq
        assert am(fp8=f8, lde=82) == b.WAM_EINVAL  # not a multiple of 4
        assert am(fp8=f8, oe=28674) == b.WAM_EINVAL and b"aligned" in L.wam_last_error()
        assert am(fp8=f8, o_batch_stride=2816) == b.WAM_EINVAL and b"plain rows" in L.wam_last_error()
    assert am(Dh=64, q_tok_stride=128, kv_tok_stride=128, o_tok_stride=128, q_batch_stride=1280,
              kv_batch_stride=2560, o_batch_stride=1280) == b.WAM_EUNSUPPORTED


def _apply_unipc_weights(coef, x0, vels):
    """The documented semantics of wam_unipc_step applied in numpy: returns the final
    state and the corrected states."""
    x, x_last, ring, states = np.array(x0, dtype=np.float64), None, {}, []
    for i, v in enumerate(vels):
        c = coef[i]
        m = x + c.s_v * v
        hist = [ring.get(i - 1 - q) for q in range(3)]
        xc = x
        if c.correct:
            xc = c.c_x * x_last + c.c_new * m + sum(c.c_m[q] * hist[q] for q in range(3) if c.c_m[q] != 0.0)
            states.append(xc)
        x = c.p_x * xc + c.p_new * m + sum(c.p_m[q] * hist[q] for q in range(2) if c.p_m[q] != 0.0)
        ring[i], x_last = m, xc
    return x, states


def test_unipc_plan_reproduces_the_oracle_solver():
    """The library's host-side UniPC weights, applied as the step kernel applies them,
    follow the oracle's UniPC over whole schedules (orders 1-3, ending inside (0, 1) or
    at 1) up to the fp32 rounding of the weights."""
    w = lib()
    g = np.random.default_rng(178)
    for ts in ([0.02, 0.1, 0.23, 0.41, 0.6, 0.78, 0.93, 1.0], [0.3, 0.35, 0.5, 0.52, 0.7, 0.9],
               [0.5, 1.0], [0.001, 0.002, 0.5]):
        ts = [float(t) for t in np.float32(ts)]
        vels = [g.standard_normal(50) for _ in range(len(ts) - 1)]
        x0 = g.standard_normal(50)
        for order in (1, 2, 3):
            it = iter(vels)
            states = []
            ref, _ = oracle.unipc_denoise(x0, lambda x, t: next(it), ts, order=order, states=states)
            got, got_states = _apply_unipc_weights(w.wam_unipc_plan(ts, order), x0, vels)
            scale = 1.0 + np.abs(ref).max()
            assert np.abs(got - ref).max() < 1e-5 * scale, (ts, order)
            assert len(got_states) == len(states)
            for a, b in zip(got_states, states):
                assert np.abs(a - b).max() < 1e-5 * scale


def test_unipc_plan_and_step_reject_bad_arguments_without_a_gpu():
    w = lib()
    b = w.binding
    L = w.lib()
    out = (b.wam_unipc_coef * 4)()

    def plan(ts, order=2, n=None):
        t = np.asarray(ts, dtype=np.float32)
        return L.wam_unipc_plan(t.ctypes.data_as(C.POINTER(C.c_float)), len(t) - 1 if n is None else n, order, out)

    assert plan([0.1, 0.5, 1.0]) == b.WAM_OK
    for ts in ([0.0, 0.5, 1.0], [0.1, 0.5, 0.5], [0.5, 0.2, 1.0], [0.1, 0.5, 1.5]):
        assert plan(ts) == b.WAM_EINVAL, ts
    assert plan([0.1, 0.5, 1.0], order=0) == b.WAM_EINVAL
    assert plan([0.1, 0.5, 1.0], order=4) == b.WAM_EINVAL
    assert plan([0.1], n=0) == b.WAM_EINVAL
    assert L.wam_unipc_plan(None, 2, 2, out) == b.WAM_EINVAL
    # a correcting first step, and a missing history buffer, are rejected before any launch
    d = b.wam_flow_dims(B=1, cfg=0, cfg_scale=1.0, n_video=8, n_action=0)
    ring = (C.c_void_p * 4)(4096, 8192, 12288, 16384)
    c = b.wam_unipc_coef(s_v=0.5, correct=1, c_x=1.0)
    assert L.wam_unipc_step(C.byref(d), 4096, None, None, 4096, 4096, ring, 0, C.byref(c), None, 4096, None,
                            None) == b.WAM_EINVAL
    c = b.wam_unipc_coef(s_v=0.5, correct=0, p_x=1.0)
    c.p_m[1] = 0.5
    assert L.wam_unipc_step(C.byref(d), 4096, None, None, 4096, 4096, ring, 1, C.byref(c), None, 4096, None,
                            None) == b.WAM_EINVAL
    assert L.wam_unipc_step(C.byref(d), None, None, None, 4096, 4096, ring, 0, C.byref(b.wam_unipc_coef()), None,
                            4096, None, None) == b.WAM_EINVAL


def test_step_workspace_holds_every_blocks_cross_kv_without_ctx_kv():
    """Without precomputed cross K|V the step projects every block's into its workspace
    (the last region): the size grows by exactly n_layers * align256(B * Lc * 2d * 2)
    bytes over the size with ctx_kv given."""
    w = lib()
    b = w.binding
    for (d, H, n_layers, B, Lc) in ((5120, 40, 40, 1, 512), (512, 4, 3, 2, 77)):
        m = b.wam_model()
        m.dims = w.make_dims(d, H, 128, 4 * d, n_layers)
        io = b.wam_step_io(B=B, F=2, Hl=8, Wl=8, A=4, Lc=Lc, Lcap=200, cache_len=0)
        without = w.lib().wam_step_workspace_bytes(C.byref(m), C.byref(io))
        given = (C.c_void_p * n_layers)(*([4096] * n_layers))
        io.ctx_kv = C.cast(given, C.POINTER(C.c_void_p))
        with_kv = w.lib().wam_step_workspace_bytes(C.byref(m), C.byref(io))
        per_layer = (B * Lc * 2 * d * 2 + 255) // 256 * 256
        assert without - with_kv == n_layers * per_layer, (d, without, with_kv)


def test_block_validates_its_whole_launch_sequence_before_the_first_launch():
    """Checks that belong to launches deep inside a block (the attention's 2 GiB key span,
    an FP8 projection's K % 16) fail before the first launch: with fake device addresses
    on a host without a GPU, a launch would return WAM_EHIP, so the status shows that
    nothing was launched (and so nothing of x or the cache was touched)."""
    w = lib()
    b = w.binding
    L = w.lib()
    fake = iter(range(1 << 20, 1 << 30, 1 << 16))

    def weights(fp8=False):
        wts = b.wam_block_weights()
        for n in ("w_qkv", "w_o", "w_cq", "w_ckv", "w_co", "w_f1", "w_f2", "mod6"):
            setattr(wts, n, next(fake))
        if fp8:
            f = b.wam_block_fp8()
            for n in ("w_qkv", "w_o", "w_cq", "w_ckv", "w_co", "w_f1", "w_f2"):
                setattr(f, n, next(fake))
                setattr(f, "s" + n[1:], next(fake))
            wts.fp8 = C.pointer(f)
            wts._f = f
        return wts

    def io(cache_len, Lq):
        return b.wam_block_io(x=next(fake), e0=next(fake), rope_cos=next(fake), rope_sin=next(fake),
                              k_cache=next(fake), v_cache=next(fake), Lcap=cache_len + Lq, cache_len=cache_len,
                              ch=w.cached_chunks(cache_len, Lq), ctx=next(fake), B=1, L=Lq, Lc=512)

    ws = 1 << 32
    dims = w.make_dims(d=5120, H=40, Dh=128, ffn=13824, n_layers=1)
    # 209000 cached keys of 5120 bf16: one sample's keys span more than 2 GiB
    big = io(209000, 1000)
    st = L.wam_dit_block_fwd(C.byref(dims), C.byref(weights()), C.byref(big), ws, 1 << 40, None)
    assert st == b.WAM_EUNSUPPORTED and b"keys span" in L.wam_last_error()
    # FP8 projections need K % 16 == 0; FFN2's K is ffn = 13832 (a multiple of 8 only)
    odd = w.make_dims(d=5120, H=40, Dh=128, ffn=13832, n_layers=1)
    st = L.wam_dit_block_fwd(C.byref(odd), C.byref(weights(fp8=True)), C.byref(io(0, 64)), ws, 1 << 40, None)
    assert st == b.WAM_EINVAL and b"K%16==0" in L.wam_last_error()
    # the same block with bf16 projections passes validation and reaches the first launch,
    # which fails here for want of a GPU
    st = L.wam_dit_block_fwd(C.byref(odd), C.byref(weights()), C.byref(io(0, 64)), ws, 1 << 40, None)
    assert st == b.WAM_EHIP


def test_block_event_kinds_match_the_header():
    w = lib()
    src = open(os.path.join(ROOT, "include", "wamdit.h")).read()
    kinds = {int(v): n.lower() for n, v in re.findall(r"\bWAM_EV_([A-Z0-9_]+)\s*=\s*(\d+)", src)}
    assert [kinds[i] for i in range(len(kinds))] == list(w.binding.BLOCK_EVENT_NAMES)
    assert int(re.search(r"WAM_BLOCK_EVENTS\s*=\s*(\d+)", src).group(1)) == w.binding.WAM_BLOCK_EVENTS
