"""GPU parity of the FP8 (E4M3) path: the per-row quantizer against the E4M3 definition
(codes bit-exact, decided in fp32 on both sides), and the FP8 GEMM with every epilogue
against the exact product of the decoded operands times their scales."""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import dev, host, log, rel_l2

pytestmark = pytest.mark.gpu


def lib():
    import paper_2602_15922_amd as w
    return w


def decode(q_u8):
    """uint8 E4M3 codes (device) -> float64 (numpy), through torch's float8 decoding."""
    import torch
    return q_u8.view(torch.float8_e4m3fn).to(torch.float64).cpu().numpy()


def expected_quant(x_bf16):
    """The quantizer's definition in fp32: inv = 448/amax, q = E4M3(x * inv)."""
    x32 = x_bf16.f64.astype(np.float32)
    amax = np.max(np.abs(x32), axis=1)
    inv = np.where(amax > 0, np.float32(448.0) / np.where(amax > 0, amax, 1), np.float32(1.0)).astype(np.float32)
    scale = np.where(amax > 0, amax / np.float32(448.0), np.float32(1.0)).astype(np.float32)
    xs = np.clip((x32 * inv[:, None]).astype(np.float32), -448, 448)
    return oracle.fp8.round_e4m3(xs.astype(np.float64)), scale


# one shape per register tier of the quantizer (rows up to 2048 / 4096 / 6144 / 14336 wide)
# and one row longer than all of them (the two-pass kernel)
@pytest.mark.parametrize("M,K", [(37, 520), (5, 8), (9, 3000), (130, 5120), (33, 13824), (4, 16392)])
def test_quantize_rows_fp8(M, K):
    import torch
    w = lib()
    log(f"fp8 quantize M={M} K={K}")
    x = synth.normal(21, "x", (M, K), 3.0)
    bits = x.data.copy()
    bits[min(2, M - 1)] = 0  # an all-zero row
    x = synth.Tensor("bf16", bits)
    ldq = (K + 15) // 16 * 16
    q = torch.zeros((M, ldq), dtype=torch.uint8, device="cuda")
    s = torch.zeros(M, dtype=torch.float32, device="cuda")
    w.wam_quantize_rows_fp8(dev(x), q, s)
    torch.cuda.synchronize()
    ref_q, ref_s = expected_quant(x)
    assert np.array_equal(host(s), ref_s.astype(np.float64))
    assert np.array_equal(decode(q[:, :K].contiguous()), ref_q)


# ----------------------------------------------------------------------------- LayerNorm to FP8
@pytest.mark.parametrize("d,B,L", [(512, 1, 144), (5120, 2, 37), (2560, 3, 5)])
def test_ln_mod_fp8_is_ln_then_quantize(d, B, L):
    """The LayerNorm that writes E4M3 rows: codes and scales bit for bit those of the bf16
    LayerNorm followed by the row quantizer (both through the C ABI), modulated and affine,
    and the decoded rows against the fp64 LayerNorm at E4M3's resolution."""
    import torch
    w = lib()
    log(f"ln_mod_fp8 d={d} B={B} L={L}")
    x = synth.normal(5, "x", (B, L, d), 3.0, d, dtype="f32")
    tab = synth.normal(5, "mod6", (6, d), 0.5, d, dtype="f32")
    e0 = synth.normal(5, "e0", (B, 6, d), 0.5, d, dtype="f32")
    g = synth.normal(5, "lnc_gamma", (d,), 0.3, d, dtype="f32")
    bt = synth.normal(5, "lnc_beta", (d,), 0.3, d, dtype="f32")
    xd, tabd, e0d = dev(x), dev(tab), dev(e0)
    M, ldq = B * L, (d + 15) // 16 * 16 + 16  # a row stride past d: padding bytes stay untouched
    m = tab.f64[None] + e0.f64
    cases = (
        (dict(shift_a=tabd[0], shift_v=e0d[:, 0], scale_a=tabd[1], scale_v=e0d[:, 1], mod_stride=6 * d),
         oracle.modulate(x.f64, m[:, 0][:, None], m[:, 1][:, None], 1e-6)),
        (dict(gamma=dev(g), beta=dev(bt)), oracle.layernorm(x.f64, 1e-6, g.f64, bt.f64)),
    )
    for kw, ref in cases:
        h = torch.empty((M, d), dtype=torch.bfloat16, device="cuda")
        w.wam_adaln_ln_mod(xd, h, 1e-6, L, **kw)
        q_ref = torch.zeros((M, ldq), dtype=torch.uint8, device="cuda")
        s_ref = torch.zeros(M, dtype=torch.float32, device="cuda")
        w.wam_quantize_rows_fp8(h, q_ref, s_ref)
        q = torch.full((M, ldq), 7, dtype=torch.uint8, device="cuda")
        s = torch.zeros(M, dtype=torch.float32, device="cuda")
        w.wam_adaln_ln_mod_fp8(xd, q, s, 1e-6, L, **kw)
        torch.cuda.synchronize()
        assert torch.equal(q[:, :d], q_ref[:, :d])
        assert torch.equal(s, s_ref)
        assert bool((q[:, d:] == 7).all())
        got = decode(q[:, :d].contiguous()) * host(s)[:, None]
        assert rel_l2(got, ref.reshape(M, d)) <= 4e-2  # E4M3: 3 mantissa bits (relative step 2^-4)


def test_ln_mod_fp8_rejects_widths_it_does_not_take():
    import torch
    w = lib()
    x = torch.zeros((2, 1280), dtype=torch.float32, device="cuda")
    q = torch.zeros((2, 1280), dtype=torch.uint8, device="cuda")
    s = torch.zeros(2, dtype=torch.float32, device="cuda")
    with pytest.raises(w.WamError):
        w.wam_adaln_ln_mod_fp8(x, q, s, 1e-6, 2)


GEMM_SHAPES = [(300, 200, 144), (3152, 5192, 528), (17, 16, 16), (3152, 13700, 144)]  # the last: two column ranges


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
@pytest.mark.parametrize("epi", ["bf16", "gelu", "resid", "f32"])
def test_gemm_fp8_epilogues(M, N, K, epi):
    import torch
    w = lib()
    log(f"gemm fp8 {epi} M={M} N={N} K={K}")
    A = synth.normal(9, "x", (M, K), 1.0, K)
    W = synth.normal(9, "w_qkv", (N, K), 0.05, K)
    bias = synth.normal(9, "b_qkv", (N,), 0.1, K, dtype="f32")
    qa = torch.empty((M, K), dtype=torch.uint8, device="cuda")
    qw = torch.empty((N, K), dtype=torch.uint8, device="cuda")
    sa = torch.empty(M, dtype=torch.float32, device="cuda")
    sw = torch.empty(N, dtype=torch.float32, device="cuda")
    w.wam_quantize_rows_fp8(dev(A), qa, sa)
    w.wam_quantize_rows_fp8(dev(W), qw, sw)
    torch.cuda.synchronize()
    acc = oracle.fp8.fp8_linear(decode(qa), host(sa), decode(qw), host(sw), bias.f64)
    bd = dev(bias)
    if epi in ("bf16", "gelu"):
        out = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
        w.wam_gemm_fp8(qa, qw, out, w.WAM_EPI_BF16 if epi == "bf16" else w.WAM_EPI_GELU_BF16, sa, sw, bias=bd)
        torch.cuda.synchronize()
        ref = acc if epi == "bf16" else oracle.gelu_tanh(acc)
        assert rel_l2(host(out), ref) <= 3e-3
    elif epi == "f32":
        out = torch.empty((M, N), dtype=torch.float32, device="cuda")
        w.wam_gemm_fp8(qa, qw, out, w.WAM_EPI_F32, sa, sw, bias=bd)
        torch.cuda.synchronize()
        # the FP8 matrix instruction's internal accumulation is slightly coarser than
        # IEEE fp32 (measured ~1.4e-5 relative even at K = 16)
        assert rel_l2(host(out), acc) <= 5e-5
    else:
        rows = max(1, M // 3)
        nb = (M + rows - 1) // rows
        x0 = synth.normal(9, "e0", (M, N), 1.0, K, dtype="f32")
        ga = synth.normal(9, "mod6", (N,), 0.5, K, dtype="f32")
        gv = synth.normal(9, "mod6", (nb, 2 * N), 0.5, K + 1, dtype="f32")
        out = dev(x0)
        gvd = dev(gv)
        w.wam_gemm_fp8(qa, qw, out, w.WAM_EPI_RESID_F32, sa, sw, bias=bd, gate_a=dev(ga), gate_v=gvd[:, N:],
                       gate_stride=2 * N, gate_rows=rows)
        torch.cuda.synchronize()
        gate = ga.f64[None] + gv.f64[np.arange(M) // rows, N:]
        ref = x0.f64 + gate * acc
        assert rel_l2(host(out) - x0.f64, ref - x0.f64) <= 5e-5


def test_gemm_fp8_against_the_unquantized_product():
    """The quantization error itself, at the QKV shape: per-row E4M3 of activations and
    per-channel E4M3 of weights reproduce the bf16 product within the error E4M3's
    3-bit mantissa allows (about 2^-4 / sqrt(3) per operand, i.e. ~5% relative L2)."""
    import torch
    w = lib()
    M, N, K = 3152, 1024, 5120
    log("gemm fp8 vs unquantized")
    A = synth.normal(10, "x", (M, K), 1.0)
    W = synth.normal(10, "w_qkv", (N, K), 0.02)
    qa = torch.empty((M, K), dtype=torch.uint8, device="cuda")
    qw = torch.empty((N, K), dtype=torch.uint8, device="cuda")
    sa = torch.empty(M, dtype=torch.float32, device="cuda")
    sw = torch.empty(N, dtype=torch.float32, device="cuda")
    w.wam_quantize_rows_fp8(dev(A), qa, sa)
    w.wam_quantize_rows_fp8(dev(W), qw, sw)
    out = torch.empty((M, N), dtype=torch.float32, device="cuda")
    w.wam_gemm_fp8(qa, qw, out, w.WAM_EPI_F32, sa, sw)
    torch.cuda.synchronize()
    e = rel_l2(host(out), A.f64 @ W.f64.T)
    print(f"  fp8 vs unquantized rel L2 {e:.3e}", flush=True)
    assert e <= 6e-2


# ------------------------------------------------------- block-scaled projection inputs
def pack_block_exps(e, lde, fill=0xAB):
    """Unbiased exponents [M][nb] of 64-column blocks -> the library's layout: per pair of
    blocks all rows in order, 4 bytes per row, block kb of row m at byte
    (kb // 2) * lde + 4 m + kb % 2; the two unused bytes of each word hold `fill`."""
    M, nb = e.shape
    buf = np.full((nb + 1) // 2 * lde, fill, dtype=np.uint8)
    kb = np.arange(nb)
    idx = (kb // 2 * lde + kb % 2)[None, :] + 4 * np.arange(M)[:, None]
    buf[idx] = (np.asarray(e) + 127).astype(np.uint8)
    return buf


def unpack_block_exps(buf, M, nb, lde):
    kb = np.arange(nb)
    idx = (kb // 2 * lde + kb % 2)[None, :] + 4 * np.arange(M)[:, None]
    return buf[idx].astype(np.int64) - 127


def codes_dev(vals):
    """float64 values on the E4M3 grid -> uint8 codes on the device."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(vals)).to(torch.float8_e4m3fn).view(torch.uint8).cuda()


MXA_SHAPES = [(300, 200, 512), (1000, 640, 384), (37, 256, 128), (129, 256, 256), (3152, 5120, 13824)]


@pytest.mark.parametrize("M,N,K", MXA_SHAPES)
@pytest.mark.parametrize("epi", ["bf16", "resid"])
def test_gemm_fp8_block_scaled_a(M, N, K, epi):
    """A as E4M3 codes with one power-of-two scale per 64 columns of a row (as FFN1 writes
    the FFN's hidden activations), blocks spread over 10^-3..10^3 so the exponents differ
    from block to block, against the oracle's fp64 product of the decoded blocks times the
    per-channel W scales (fp32 accumulation and the bf16 output rounding remain).  The
    shapes cover one, two and three slices of 128 columns (fewer than the prefetch ring's
    stages), ragged row and column tiles, and the FFN2 shape (oracle on sampled rows)."""
    import torch
    w = lib()
    log(f"gemm fp8 block-scaled A {epi} M={M} N={N} K={K}")
    g = np.random.default_rng(M + N + K)
    nb = K // 64
    x = g.standard_normal((M, K)) * np.repeat(10.0 ** g.uniform(-3, 3, (M, nb)), 64, axis=1)
    qa, ea = oracle.fp8.quantize_mx(x, 64)
    W = synth.normal(11, "w_f2", (N, K), 0.05, K)
    bias = synth.normal(11, "b_f2", (N,), 0.1, K, dtype="f32")
    qw = torch.empty((N, K), dtype=torch.uint8, device="cuda")
    sw = torch.empty(N, dtype=torch.float32, device="cuda")
    w.wam_quantize_rows_fp8(dev(W), qw, sw)
    lde = 4 * M + 64
    exps = torch.from_numpy(pack_block_exps(ea, lde)).cuda()
    a8 = codes_dev(qa)
    rows = np.arange(M) if M <= 1000 else sampled_rows(M)
    acc = oracle.fp8.fp8_linear(oracle.fp8.decode_mx(qa[rows], ea[rows], 64), np.ones(len(rows)), decode(qw),
                                host(sw), bias.f64)
    if epi == "bf16":
        out = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
        w.wam_gemm_fp8_mx(a8, qw, out, w.WAM_EPI_BF16, sw, a_exp=exps, a_lde=lde, bias=dev(bias))
        torch.cuda.synchronize()
        assert rel_l2(host(out)[rows], acc) <= 3e-3
    else:
        x0 = synth.normal(11, "e0", (M, N), 1.0, K, dtype="f32")
        ga = synth.normal(11, "mod6", (N,), 0.5, K, dtype="f32")
        out = dev(x0)
        w.wam_gemm_fp8_mx(a8, qw, out, w.WAM_EPI_RESID_F32, sw, a_exp=exps, a_lde=lde, bias=dev(bias),
                          gate_a=dev(ga))
        torch.cuda.synchronize()
        upd = host(out)[rows] - x0.f64[rows]
        assert rel_l2(upd, ga.f64[None] * acc) <= 5e-5


def sampled_rows(M):
    """Row-tile boundaries of the 128-, 192- and 256-row tiles and the ragged end, plus random rows."""
    r = {0, 1, M - 1, M - 2}
    for t in (128, 192, 256):
        for b in range(t, M, t):
            r.update([b - 1, b])
    r.update(np.random.default_rng(M).integers(0, M, 24).tolist())
    return np.array(sorted(i for i in r if 0 <= i < M))


MX8_SHAPES = [(300, 512, 512), (130, 1280, 256), (3152, 13824, 5120)]


@pytest.mark.parametrize("M,N,K", MX8_SHAPES)
def test_gemm_fp8_gelu_block_output(M, N, K):
    """The GELU epilogue written block-scaled is, bit for bit, the oracle's 64-element MX
    quantization of the bf16 GELU output that wam_gemm_fp8 writes for the same inputs:
    every code and exponent (the same accumulators, the same bf16 rounding, the block
    exponent rule of wam_quantize_mx_fp8), the unused exponent bytes untouched.  The last
    shape is FFN1's (two column ranges of 256- and 192-row tiles), checked on sampled rows."""
    import torch
    w = lib()
    log(f"gemm fp8 gelu block output M={M} N={N} K={K}")
    A = synth.normal(12, "x", (M, K), 1.0, K)
    W = synth.normal(12, "w_f1", (N, K), 0.05, K)
    bias = synth.normal(12, "b_f1", (N,), 0.1, K, dtype="f32")
    qa = torch.empty((M, K), dtype=torch.uint8, device="cuda")
    qw = torch.empty((N, K), dtype=torch.uint8, device="cuda")
    sa = torch.empty(M, dtype=torch.float32, device="cuda")
    sw = torch.empty(N, dtype=torch.float32, device="cuda")
    w.wam_quantize_rows_fp8(dev(A), qa, sa)
    w.wam_quantize_rows_fp8(dev(W), qw, sw)
    bd = dev(bias)
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    w.wam_gemm_fp8(qa, qw, y, w.WAM_EPI_GELU_BF16, sa, sw, bias=bd)
    lde = 4 * M + 32
    nb = N // 64
    u8 = torch.full((M, N), 0x7F, dtype=torch.uint8, device="cuda")
    ue = torch.full(((nb + 1) // 2 * lde,), 0xAB, dtype=torch.uint8, device="cuda")
    w.wam_gemm_fp8_mx(qa, qw, u8, w.WAM_EPI_GELU_BF16, sw, a_scale=sa, out_exp=ue, o_lde=lde, bias=bd)
    torch.cuda.synchronize()
    rows = np.arange(M) if M <= 1000 else sampled_rows(M)
    q, e = oracle.fp8.quantize_mx(host(y)[rows], 64)
    assert np.array_equal(decode(u8)[rows], q)
    ueh = ue.cpu().numpy()
    assert np.array_equal(unpack_block_exps(ueh, M, nb, lde)[rows], e)
    used = np.zeros(ueh.size, bool)
    kb = np.arange(nb)
    used[((kb // 2 * lde + kb % 2)[None, :] + 4 * np.arange(M)[:, None]).ravel()] = True
    assert np.all(ueh[~used] == 0xAB)


# ------------------------------------------------------------------------------ FP8 blocks
# Against the fp64 oracle of the unquantized model: each FP8 projection carries ~4%
# relative error (measured above at the QKV shape) and a branch chains up to three of
# them (cross-Q, cross-K|V, cross-O: ~sqrt(3) x 4% ~ 7%), so a block's residual update,
# its appended K/V and the step's velocities (the ungated cross-attention branch moves
# the residual by O(1) even when the gates are small) are held to 0.1.
FP8_TOL_UPDATE = 1e-1
FP8_TOL_STEP = 1e-1


def test_fp8_block_small():
    from dit_cases import BlockCase
    wl = synth.WORKLOADS["block_d512"].replace(B=2, n_cached=1)
    log("fp8 block d512")
    case = BlockCase(wl, bias_std=0.05)
    x, kc, vc = case.run_gpu(fp8=True)
    ref, k_ref, v_ref = case.run_oracle()
    x0 = case.x.f64
    eu = rel_l2(host(x) - x0, ref - x0)
    r0, r1 = wl.cache_rows, wl.cache_rows + wl.L
    ek = rel_l2(host(kc[:, r0:r1]), k_ref)
    ev = rel_l2(host(vc[:, r0:r1]), v_ref)
    print(f"  fp8 block: update rel L2 {eu:.3e}, K {ek:.3e}, V {ev:.3e}", flush=True)
    assert eu <= FP8_TOL_UPDATE and ek <= FP8_TOL_UPDATE and ev <= FP8_TOL_UPDATE


def test_fp8_step_14b_shapes_one_block():
    from dit_cases import StepCase
    wl = synth.WORKLOADS["step_14b"].replace(n_layers=1)
    log("fp8 step 14b depth 1: inputs + GPU")
    case = StepCase(wl, 1)
    case.upload(fp8=True)
    vv, va = case.run_gpu()
    log("fp8 step 14b depth 1: oracle")
    rv, ra = case.run_oracle()
    ev, ea = rel_l2(host(vv), rv), rel_l2(host(va), ra)
    print(f"  fp8 step rel L2 video {ev:.3e} action {ea:.3e}", flush=True)
    assert ev <= FP8_TOL_STEP and ea <= FP8_TOL_STEP
