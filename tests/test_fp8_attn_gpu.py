"""GPU parity of the FP8 attention path (wam_quantize_mx_fp8, wam_quantize_scaled_fp8,
wam_rope_qkv_fp8, wam_attn_blockcausal_fp8) against the oracle's E4M3 definitions: the
quantizers bit-exact, the attention against the fp64 softmax attention of the decoded
operands (exactly, up to fp32 accumulation and the bf16 output, when every probability
is a power of two; within the E4M3 rounding of the probabilities otherwise), and the FP8
KV cache inside a block and a 14B-shaped step against the unquantized fp64 model."""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import dev, host, log, rel_l2

pytestmark = pytest.mark.gpu

# Bar for random operands.  Every probability is rounded to E4M3 (3 mantissa bits: a
# relative error up to 2^-4, RMS ~2^-4/sqrt(3) ~ 3.6% for round-to-nearest).  For
# attention over many keys with random values the output is a weighted mean whose norm
# shrinks like the noise it averages, so the relative error of o stays near that RMS;
# measured 2-3%.  Twice the RMS leaves room without admitting a mis-paired key (error of
# order 1).
TOL_RANDOM = 8e-2
# Probabilities that are powers of two are rounded exactly: only fp32 accumulation and
# the bf16 output remain (2^-9 / sqrt(3) ~ 1.1e-3 for the output rounding).
TOL_EXACT = 3e-3


def lib():
    import paper_2602_15922_amd as w
    return w


def codes_dev(vals):
    """float64 values on the E4M3 grid -> uint8 codes on the device."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(vals)).to(torch.float8_e4m3fn).view(torch.uint8).cuda()


def decode(q_u8):
    import torch
    return q_u8.view(torch.float8_e4m3fn).to(torch.float64).cpu().numpy()


def exps_dev(e):
    """Unbiased block exponents [..., H, 4] -> int32 [..., H] (byte j = block j + 127)."""
    import torch
    b = np.ascontiguousarray((np.asarray(e) + 127).astype(np.uint8))
    return torch.from_numpy(b.view(np.int32)[..., 0].copy()).cuda()


def exps_host(e32):
    """int32 [..., H] device -> unbiased exponents [..., H, 4]."""
    b = e32.contiguous().cpu().numpy().astype(np.int32).view(np.uint8).reshape(tuple(e32.shape) + (4,))
    return b.astype(np.int64) - 127


def fp8_operands(q, k, v):
    """Oracle quantization of float64 q, k, v [..., H, 128]: MX blocks for q and k, one
    fp32 scale max|v| / 448 for v.  Returns the device operands and the decoded values."""
    qq, qe = oracle.fp8.quantize_mx(q)
    kq, ke = oracle.fp8.quantize_mx(k)
    vs = float(np.float32(np.max(np.abs(v)) / 448.0))
    vq = oracle.fp8.quantize_scaled(v, vs)
    devs = dict(q8=codes_dev(qq), q_exp=exps_dev(qe), k8=codes_dev(kq), k_exp=exps_dev(ke), v8=codes_dev(vq),
                v_scale=vs)
    dec = (oracle.fp8.decode_mx(qq, qe), oracle.fp8.decode_mx(kq, ke), vq * vs)
    return devs, dec


def run_fp8(ops, ch, Lq_shape, scale=0.0):
    import torch
    w = lib()
    o = torch.empty(Lq_shape, dtype=torch.bfloat16, device="cuda")
    w.wam_attn_blockcausal_fp8(ops["q8"], ops["q_exp"], ops["k8"], ops["k_exp"], ops["v8"], ops["v_scale"], o, ch,
                               scale=scale)
    torch.cuda.synchronize()
    return o


def chunk_ids(sizes):
    return np.repeat(np.arange(len(sizes)), sizes)


# --------------------------------------------------------------------------- quantizers
@pytest.mark.parametrize("M,K", [(37, 512), (300, 5120), (4, 32)])
def test_quantize_mx_matches_definition(M, K):
    """Codes and block exponents bit-exact against the oracle's block quantizer, on rows
    whose blocks span 16 binary orders of magnitude, with an all-zero block."""
    import torch
    w = lib()
    g = np.random.default_rng(M + K)
    x = g.standard_normal((M, K)) * np.repeat(2.0 ** g.integers(-8, 8, (M, K // 32)), 32, axis=1)
    x[0, :32] = 0.0
    xb = synth.Tensor("bf16", synth.bf16_bits(x.astype(np.float32)))
    log(f"quantize mx M={M} K={K}")
    ldq = K + 16
    q8 = torch.zeros((M, ldq), dtype=torch.uint8, device="cuda")
    ex = torch.zeros((M, K // 32), dtype=torch.uint8, device="cuda")
    w.wam_quantize_mx_fp8(dev(xb), q8, ex)
    torch.cuda.synchronize()
    qr, er = oracle.fp8.quantize_mx(xb.f64)
    assert np.array_equal(ex.cpu().numpy().astype(np.int64) - 127, er)
    assert np.array_equal(decode(q8[:, :K]), qr)
    assert not q8[:, K:].any()


def test_quantize_scaled_matches_definition():
    import torch
    w = lib()
    g = np.random.default_rng(7)
    x = synth.Tensor("bf16", synth.bf16_bits((g.standard_normal(40000) * 3.0).astype(np.float32)))
    s = 0.0123
    log("quantize scaled")
    q8 = torch.empty(40000, dtype=torch.uint8, device="cuda")
    w.wam_quantize_scaled_fp8(dev(x), s, q8)
    torch.cuda.synchronize()
    assert np.array_equal(decode(q8), oracle.fp8.quantize_scaled(x.f64, s))


@pytest.mark.parametrize("B,L,c", [(1, 62, 3), (2, 45, 0)])
def test_rope_fp8_append(B, L, c):
    """Rotated q and k encoded in 32-dim blocks from their fp32 rotation: block exponents
    equal to the oracle's on the fp64 rotation, codes equal except where the fp32 rotation
    lands on the other side of a rounding midpoint (then one E4M3 step apart); v codes
    bit-exact; cache rows outside the chunk's slot untouched."""
    import torch
    w = lib()
    H, Dh = 3, 128
    d = H * Dh
    Hg, Wg = 3, 5
    A = L - 2 * Hg * Wg
    pos = w.wam_chunk_positions(c, 2, Hg, Wg, A)
    cos, sin = w.wam_rope_tables(pos, Dh)
    qkv = synth.normal(8, "x", (B, L, 3 * d), 1.0, 300 + L)
    Lcap, row0 = L + 19, 7
    vs = 0.02
    log(f"rope fp8 B={B} L={L}")
    k8 = torch.full((B, Lcap, H, Dh), 0x11, dtype=torch.uint8, device="cuda")
    v8 = k8.clone()
    ke = torch.full((B, Lcap, H), 0x22222222, dtype=torch.int32, device="cuda")
    q8 = torch.empty((B, L, H, Dh), dtype=torch.uint8, device="cuda")
    qe = torch.empty((B, L, H), dtype=torch.int32, device="cuda")
    w.wam_rope_qkv_fp8(dev(qkv), dev(cos), dev(sin), q8, qe, k8, ke, v8, vs, row0, H, Dh)
    torch.cuda.synchronize()
    f = qkv.f64.reshape(B, L, 3, H, Dh)
    vals = oracle.fp8.e4m3_values()
    for got_q, got_e, x in ((q8, qe, f[:, :, 0]), (k8[:, row0:row0 + L], ke[:, row0:row0 + L], f[:, :, 1])):
        rq, re = oracle.fp8.quantize_mx(oracle.apply_rope(x, pos))
        assert np.array_equal(exps_host(got_e), re)
        gq = decode(got_q)
        diff = gq != rq
        assert diff.mean() < 1e-3
        # a mismatch is a neighbouring grid value
        idx_g = np.searchsorted(vals, np.abs(gq[diff]))
        idx_r = np.searchsorted(vals, np.abs(rq[diff]))
        assert np.all(np.abs(idx_g - idx_r) == 1)
    assert np.array_equal(decode(v8[:, row0:row0 + L]), oracle.fp8.quantize_scaled(f[:, :, 2], vs))
    for t, fill in ((k8, 0x11), (v8, 0x11)):
        assert (t[:, :row0] == fill).all() and (t[:, row0 + L:] == fill).all()
    assert (ke[:, :row0] == 0x22222222).all() and (ke[:, row0 + L:] == 0x22222222).all()


# --------------------------------------------------------------------------- attention
CASES = [
    # name, B, H, key chunk sizes, query chunks (indices into the key chunks)
    ("decode_ragged", 1, 2, [100, 77], [1]),
    ("prefill3_masked", 2, 3, [50, 70, 45], [0, 1, 2]),
    ("cached_tail", 1, 2, [130, 64, 200], [1, 2]),
    ("one_token", 1, 1, [1], [0]),
    ("mid_tile_boundaries", 1, 2, [31, 97, 1, 129], [0, 1, 2, 3]),
    ("many_chunks", 2, 2, [40] * 16, list(range(16))),
]


def layout(ks, qc):
    k_chunk = chunk_ids(ks)
    off = np.concatenate([[0], np.cumsum(ks)])
    q_rows = np.concatenate([np.arange(off[c], off[c + 1]) for c in qc])
    return k_chunk, k_chunk[q_rows], len(q_rows), int(off[-1])


@pytest.mark.parametrize("name,B,H,ks,qc", CASES)
def test_attention_fp8_exact_probabilities(name, B, H, ks, qc):
    """Scores chosen so every probability the kernel rounds is a power of two: q and k
    take values in {-1, 0, 1} on six dims (zero elsewhere), which the block quantizer
    represents exactly (exponent -8, code 256), so q.k is an integer in [-6, 6]; with
    scale = ln 2, exp(scale s) = 2^s.  The kernel's rounding of the probabilities is then
    exact and the result must equal the softmax attention of the decoded operands up to
    fp32 accumulation and the bf16 output, whichever keys a tile pairs."""
    w = lib()
    case = [c[0] for c in CASES].index(name)
    k_chunk, q_chunk, Lq, Lk = layout(ks, qc)
    g = np.random.default_rng(500 + case)
    q = np.zeros((B, Lq, H, 128))
    k = np.zeros((B, Lk, H, 128))
    q[..., :6] = g.integers(-1, 2, (B, Lq, H, 6))
    k[..., :6] = g.integers(-1, 2, (B, Lk, H, 6))
    v = g.standard_normal((B, Lk, H, 128))
    ops, (qd, kd, vd) = fp8_operands(q, k, v)
    assert np.array_equal(qd, q) and np.array_equal(kd, k)  # represented exactly
    scale = float(np.float32(np.log(2.0)))
    ch = w.make_chunks(ks, [ks[c] for c in qc], qc)
    log(f"attn fp8 exact {name} B={B} H={H} Lq={Lq} Lk={Lk}")
    o = host(run_fp8(ops, ch, (B, Lq, H, 128), scale=scale))
    for b in range(B):
        ref = oracle.attention(qd[b], kd[b], vd[b], q_chunk, k_chunk, scale=scale)
        err = rel_l2(o[b], ref)
        print(f"  {name} b={b}: rel L2 {err:.2e}", flush=True)
        assert err <= TOL_EXACT, (name, b, err)


@pytest.mark.parametrize("name,B,H,ks,qc", CASES)
def test_attention_fp8_random_operands(name, B, H, ks, qc):
    """Gaussian q, k, v quantized by the oracle; the kernel against the fp64 attention of
    the decoded operands, the difference being the E4M3 rounding of the probabilities."""
    w = lib()
    case = [c[0] for c in CASES].index(name)
    k_chunk, q_chunk, Lq, Lk = layout(ks, qc)
    q = synth.normal(2, "q", (B, Lq, H, 128), 1.0, 600 + case).f64
    k = synth.normal(2, "k", (B, Lk, H, 128), 1.0, 600 + case).f64
    v = synth.normal(2, "v", (B, Lk, H, 128), 1.0, 600 + case).f64
    ops, (qd, kd, vd) = fp8_operands(q, k, v)
    ch = w.make_chunks(ks, [ks[c] for c in qc], qc)
    log(f"attn fp8 random {name} B={B} H={H} Lq={Lq} Lk={Lk}")
    o = host(run_fp8(ops, ch, (B, Lq, H, 128)))
    for b in range(B):
        ref = oracle.attention(qd[b], kd[b], vd[b], q_chunk, k_chunk)
        err = rel_l2(o[b], ref)
        print(f"  {name} b={b}: rel L2 {err:.2e}", flush=True)
        assert err <= TOL_RANDOM, (name, b, err)


@pytest.mark.parametrize("name,B,H,ks,qc", CASES)
def test_attention_fp8_block_scaled_output(name, B, H, ks, qc):
    """wam_attn_blockcausal_fp8_mx writes, bit for bit, the oracle's 64-element MX
    quantization of the bf16 output that wam_attn_blockcausal_fp8 writes for the same
    operands, in the a_exp layout of the O projection; other exponent bytes untouched."""
    import torch
    from gpu_helpers import check_block_output
    w = lib()
    case = [c[0] for c in CASES].index(name)
    k_chunk, q_chunk, Lq, Lk = layout(ks, qc)
    q = synth.normal(3, "q", (B, Lq, H, 128), 1.0, 700 + case).f64
    k = synth.normal(3, "k", (B, Lk, H, 128), 1.0, 700 + case).f64
    v = synth.normal(3, "v", (B, Lk, H, 128), 1.0, 700 + case).f64
    ops, _ = fp8_operands(q, k, v)
    ch = w.make_chunks(ks, [ks[c] for c in qc], qc)
    log(f"attn fp8 block-scaled output {name} B={B} H={H} Lq={Lq} Lk={Lk}")
    o = host(run_fp8(ops, ch, (B, Lq, H, 128)))
    o8 = torch.full((B, Lq, H, 128), 0x7F, dtype=torch.uint8, device="cuda")
    lde = 4 * B * Lq + 8
    oe = torch.full((H * lde,), 0xAB, dtype=torch.uint8, device="cuda")
    w.wam_attn_blockcausal_fp8_mx(ops["q8"], ops["q_exp"], ops["k8"], ops["k_exp"], ops["v8"], ops["v_scale"], o8,
                                  oe, lde, ch)
    torch.cuda.synchronize()
    check_block_output(o8.view(B * Lq, H * 128), oe, o.reshape(B * Lq, H * 128), lde)


def test_attention_fp8_deterministic_and_future_independent():
    """Bitwise: the same inputs give the same output, and chunk 0's rows do not change
    when chunk 1's keys and values do."""
    import torch
    w = lib()
    B, H, ks = 1, 2, [70, 90]
    k_chunk, q_chunk, Lq, Lk = layout(ks, [0, 1])
    g = np.random.default_rng(9)
    q, k, v = (g.standard_normal((B, n, H, 128)) for n in (Lq, Lk, Lk))
    ops, _ = fp8_operands(q, k, v)
    ch = w.make_chunks(ks, ks, [0, 1])
    log("attn fp8 determinism")
    o1 = run_fp8(ops, ch, (B, Lq, H, 128))
    o2 = run_fp8(ops, ch, (B, Lq, H, 128))
    assert torch.equal(o1, o2)
    ops["k8"][:, 70:] = codes_dev(np.full((B, 90, H, 128), 3.0))
    ops["v8"][:, 70:] = codes_dev(np.full((B, 90, H, 128), -5.0))
    o3 = run_fp8(ops, ch, (B, Lq, H, 128))
    assert torch.equal(o1[:, :70], o3[:, :70]) and not torch.equal(o1[:, 70:], o3[:, 70:])


def test_attention_fp8_full_size_sampled_rows():
    """40 heads x 128, 3152 queries of chunk 4 against 15760 keys (four cached chunks of
    3152 plus the chunk): the step's self-attention shape.  Oracle on sampled rows."""
    w = lib()
    wl = synth.WORKLOADS["step_14b"]
    B, H, L, Lk = 1, wl.H, wl.L, wl.Lk
    q = synth.normal(wl.seed, "q", (B, L, H, 128), 1.0, 700).f64
    k = synth.normal(wl.seed, "k", (B, Lk, H, 128), 1.0, 700).f64
    v = synth.normal(wl.seed, "v", (B, Lk, H, 128), 1.0, 700).f64
    log(f"attn fp8 full size Lq={L} Lk={Lk}: quantize")
    ops, (qd, kd, vd) = fp8_operands(q, k, v)
    log("attn fp8 full size: GPU")
    o = host(run_fp8(ops, w.cached_chunks(Lk - L, L), (B, L, H, 128)))
    g = np.random.default_rng(3)
    rows = np.unique(np.concatenate([[0, 1, 127, 128, L - 2, L - 1], g.integers(0, L, 40)]))
    log("attn fp8 full size: oracle")
    n_ch = Lk // L
    ref = oracle.attention(qd[0, rows], kd[0], vd[0], np.full(len(rows), n_ch - 1), np.repeat(np.arange(n_ch), L))
    err = rel_l2(o[0, rows], ref)
    print(f"  full size rel L2 {err:.2e}", flush=True)
    assert err <= TOL_RANDOM


def test_attention_fp8_b2_3view_sampled_rows():
    """The two-sample, three-view configuration: batch 2, 9392 queries of chunk 6 against
    65744 keys, 40 heads of 128.  Inputs are drawn on the device from seeded streams and
    quantized by the library's own quantizers (bit-exact against the oracle's above); the
    fp64 oracle attends with the decoded operands on sampled query rows of both samples,
    every head, all keys."""
    import torch
    w = lib()
    wl = synth.WORKLOADS["step_14b_b2_3view"]
    B, H, Dh, L, Lk = wl.B, wl.H, wl.Dh, wl.L, wl.Lk
    log(f"attn fp8 b2 3-view B={B} Lq={L} Lk={Lk}: inputs")
    ops = {}
    for name, rows in (("q", L), ("k", Lk)):
        x = synth.device_normal(wl.seed, name, (B, rows, H, Dh))
        c = torch.empty((B, rows, H, Dh), dtype=torch.uint8, device="cuda")
        e = torch.empty((B, rows, H), dtype=torch.int32, device="cuda")
        w.wam_quantize_mx_fp8(x.view(B * rows, H * Dh), c.view(B * rows, H * Dh),
                              e.view(torch.uint8).view(B * rows, H * 4))
        ops[name] = (c, e)
        del x
    v = synth.device_normal(wl.seed, "v", (B, Lk, H, Dh))
    vs = float(v.abs().max().float()) / 448.0
    v8 = torch.empty((B, Lk, H, Dh), dtype=torch.uint8, device="cuda")
    w.wam_quantize_scaled_fp8(v, vs, v8)
    del v
    log("attn fp8 b2 3-view: GPU")
    o = torch.empty((B, L, H, Dh), dtype=torch.bfloat16, device="cuda")
    w.wam_attn_blockcausal_fp8(ops["q"][0], ops["q"][1], ops["k"][0], ops["k"][1], v8, vs, o,
                               w.cached_chunks(wl.cache_rows, L))
    torch.cuda.synchronize()
    g = np.random.default_rng(4)
    rows = np.unique(np.concatenate([[0, 127, 128, 9215, 9216, L - 1], g.integers(0, L, 18)]))
    kc = np.repeat(np.arange(wl.n_cached + 1), L)
    for b in range(B):
        log(f"attn fp8 b2 3-view: oracle, sample {b}")
        qd = oracle.fp8.decode_mx(decode(ops["q"][0][b, rows]), exps_host(ops["q"][1][b, rows]))
        kd = oracle.fp8.decode_mx(decode(ops["k"][0][b]), exps_host(ops["k"][1][b]))
        vd = decode(v8[b]) * vs
        ref = oracle.attention(qd, kd, vd, np.full(len(rows), wl.n_cached), kc)
        err = rel_l2(host(o[b, rows]), ref)
        print(f"  sample {b}: {len(rows)} rows, rel L2 {err:.2e}", flush=True)
        assert err <= TOL_RANDOM
        del kd, vd


def test_attention_fp8_rejects_bad_arguments():
    import torch
    w = lib()
    q8 = torch.zeros((1, 4, 1, 128), dtype=torch.uint8, device="cuda")
    qe = torch.zeros((1, 4, 1), dtype=torch.int32, device="cuda")
    o = torch.zeros((1, 4, 1, 128), dtype=torch.bfloat16, device="cuda")
    ch = w.make_chunks([4], [4], [0])
    with pytest.raises(w.WamError):
        w.wam_attn_blockcausal_fp8(q8, qe, q8, qe, q8, 0.0, o, ch)  # v_scale must be positive
    q64 = torch.zeros((1, 4, 2, 64), dtype=torch.uint8, device="cuda")
    qe2 = torch.zeros((1, 4, 2), dtype=torch.int32, device="cuda")
    with pytest.raises(w.WamError):
        w.wam_attn_blockcausal_fp8(q64, qe2, q64, qe2, q64, 1.0, o, ch)  # Dh = 128 only


# --------------------------------------------------------------------------- in the step
# The bar of the FP8 step (each E4M3 projection ~4%, chains of three ~7%); the FP8 cache
# adds the rounding of k, v and the probabilities inside the self-attention, whose output
# is one gated branch of the residual update.
FP8_TOL_STEP = 1e-1


@pytest.mark.parametrize("fp8_proj", [False, True])
def test_fp8_cache_step_14b_shapes_one_block(fp8_proj):
    """The 14B step at depth 1 (3152 rows after 4 cached chunks, Lk 15760) with an FP8 KV
    cache, so the RoPE/append writes E4M3 codes and the self-attention runs in FP8, with
    bf16 or FP8 projections, against the unquantized fp64 oracle."""
    from dit_cases import StepCase
    wl = synth.WORKLOADS["step_14b"].replace(n_layers=1)
    log(f"fp8 cache step 14b depth 1 (fp8 projections: {fp8_proj}): inputs + calibration step")
    case = StepCase(wl, 1)
    case.upload(fp8=fp8_proj)
    case.run_gpu()
    case.make_fp8_cache()
    log("fp8 cache step: GPU")
    vv, va = case.run_gpu(fp8_cache=True)
    log("fp8 cache step: oracle")
    rv, ra = case.run_oracle()
    ev, ea = rel_l2(host(vv), rv), rel_l2(host(va), ra)
    print(f"  fp8 cache step rel L2 video {ev:.3e} action {ea:.3e}", flush=True)
    assert ev <= FP8_TOL_STEP and ea <= FP8_TOL_STEP


def test_fp8_cache_update_pass_14b_shapes():
    """The cache-update pass writing an FP8 cache at the 14B block shapes: 3120 clean video
    rows after two cached chunks (9360 keys), two layers (a full block with the FP8
    self-attention, then the K/V-only last layer).  The appended K (decoded blocks) and V
    (codes times the layer's scale) against the oracle's unquantized pass; the cached rows'
    codes untouched.  V's scales come from a bf16 pass over the same rows (calibration),
    whose appended rows are then cleared from the FP8 caches."""
    import torch
    from dit_cases import UpdateCase, fp8_caches
    wl = synth.WORKLOADS["block_14b"].replace(A=0, n_cached=2, n_layers=2)
    log("fp8 update 14b: inputs + calibration pass")
    case = UpdateCase(wl, 2, 1)
    case.upload()
    case.run_gpu()
    r0, r1 = wl.cache_rows, wl.cache_rows + case.L
    k8s, kes, v8s, vsc = fp8_caches(case.kcs, case.vcs, r1)
    before = [(k8[:, :r0].clone(), ke[:, :r0].clone(), v8[:, :r0].clone()) for k8, ke, v8 in zip(k8s, kes, v8s)]
    for k8, ke, v8 in zip(k8s, kes, v8s):
        k8[:, r0:].zero_()
        ke[:, r0:].zero_()
        v8[:, r0:].zero_()
    log("fp8 update 14b: GPU")
    case.run_gpu(fp8_cache=(k8s, kes, v8s, vsc))
    log("fp8 update 14b: oracle")
    ref = case.run_oracle()
    for l, (k_ref, v_ref) in enumerate(ref):
        kd = oracle.fp8.decode_mx(decode(k8s[l][:, r0:r1]), exps_host(kes[l][:, r0:r1]))
        vd = decode(v8s[l][:, r0:r1]) * vsc[l]
        ek, ev = rel_l2(kd, k_ref), rel_l2(vd, v_ref)
        print(f"  layer {l}: appended K rel L2 {ek:.2e}, V {ev:.2e}", flush=True)
        assert ek <= FP8_TOL_STEP and ev <= FP8_TOL_STEP
        k8, ke, v8 = before[l]
        assert torch.equal(k8s[l][:, :r0], k8) and torch.equal(kes[l][:, :r0], ke) and torch.equal(v8s[l][:, :r0], v8)
        assert not k8s[l][:, r1:].any() and not v8s[l][:, r1:].any()
