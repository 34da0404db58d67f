"""Throughput of one DiT denoising step on one MI355X, through libwamdit's C ABI.

Workload (the 14B-class step): 40 blocks, d=5120, 40 heads of 128, FFN 13824; one chunk of
2 latent frames x 30x52 patches (3120 video tokens) + 32 action tokens; 4 cached chunks per
layer (12608 rows; 15760 keys per query); 512 text tokens of width 4096.  Weights are
random bf16 N(0, 0.02^2), ~28 GB resident; inputs are synthetic Gaussians of the paper's
shapes (no trained weights or datasets exist here).  A step is the whole velocity call:
time embedding, text projection, patch/action embedding, 40 blocks (each recomputing its
cross-attention K/V of the text) and the output head.

Prints one JSON line: steps/s, plus the self-attention kernel's achieved bf16 TFLOP/s
against the MFMA peak (per-launch durations from HIP events recorded around every
self-attention launch inside the timed steps) and its HBM bytes per launch (from the
committed counter profile; null once the kernel source differs from the profiled one),
the fp64 oracle timed on the host cores on a bounded sample (one full-shape block),
scaled to steps/s, and (`extras`) the Flash step, the cache-update pass, a 4-step
denoising loop and the step with FP8 projections on the same model.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MI355X_BF16_DENSE_TFLOPS = 2500.0  # published dense bf16 MFMA peak
MI355X_FP8_DENSE_TFLOPS = 5000.0  # published dense FP8 MFMA peak
WORKLOAD = "step_14b"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extras", action="store_true",
                   help="skip the Flash step / update pass / denoising loop timings")
    p.add_argument("--workload", default=WORKLOAD)
    p.add_argument("--probe-attn", type=int, default=0, metavar="N",
                   help="counter-collection mode: one plain 1 GiB device copy, then N self-attention "
                        "launches at the workload's shape; prints what ran and exits")
    p.add_argument("--probe-attn-fp8", type=int, default=0, metavar="N",
                   help="the same with the FP8 self-attention (operands quantized by the library)")
    p.add_argument("--probe", choices=("gemm", "gemm_fp8", "ln", "rope", "torch_linear"), default=None,
                   help="counter-collection mode: the calibration copy, then --probe-n launches of each "
                        "of the block's six projections (gemm), of the AdaLN LayerNorm (ln) or of the "
                        "RoPE/KV-append kernel (rope) at the workload's shapes")
    p.add_argument("--probe-n", type=int, default=3)
    p.add_argument("--profile-steps", type=int, default=2,
                   help="untimed steps after the timed ones with events around every launch of every "
                        "block (per-role kernel times: the GEMM fractions of the JSON line)")
    p.add_argument("--pmc-summary", default=None, metavar="DIR",
                   help="no GPU: print per-kernel averages of a rocprofv3 counter CSV under DIR")
    p.add_argument("--trace-summary", default=None, metavar="DIR",
                   help="no GPU: print per-kernel and per-launch-shape times of a rocprofv3 kernel trace "
                        "under DIR (with --trace-steps: the dispatches of that many steps per step)")
    p.add_argument("--trace-steps", type=int, default=0)
    return p.parse_args()


def build_model(wl, torch):
    import paper_2602_15922_amd as w
    d, dev = wl.d, "cuda"
    g = torch.Generator(device=dev).manual_seed(1234)

    def rn(*shape, std=0.02):
        t = torch.randn(*shape, generator=g, device=dev, dtype=torch.bfloat16)
        return t.mul_(std) if std != 1.0 else t

    def zf(n):
        return torch.zeros(n, dtype=torch.float32, device=dev)

    top = {"w_t1": rn(d, wl.freq_dim), "w_t2": rn(d, d), "w_t6": rn(6 * d, d), "w_x1": rn(d, wl.text_dim),
           "w_x2": rn(d, d), "w_patch": rn(d, wl.patch_dim), "w_ain": rn(d, wl.act_dim),
           "w_hv": rn(wl.patch_dim, d), "w_ha": rn(wl.act_dim, d),
           "head_mod2": torch.randn(2, d, generator=g, device=dev) * 0.02}
    for n, k in (("b_t1", d), ("b_t2", d), ("b_t6", 6 * d), ("b_x1", d), ("b_x2", d), ("b_patch", d),
                 ("b_ain", d), ("b_hv", wl.patch_dim), ("b_ha", wl.act_dim)):
        top[n] = zf(k)
    blocks, kcs, vcs = [], [], []
    for _ in range(wl.n_layers):
        b = {"w_qkv": rn(3 * d, d), "w_o": rn(d, d), "w_cq": rn(d, d), "w_ckv": rn(2 * d, d), "w_co": rn(d, d),
             "w_f1": rn(wl.ffn, d), "w_f2": rn(d, wl.ffn),
             "mod6": torch.randn(6, d, generator=g, device=dev) * 0.02,
             "lnc_gamma": torch.ones(d, device=dev), "lnc_beta": zf(d)}
        for n, k in (("b_qkv", 3 * d), ("b_o", d), ("b_cq", d), ("b_ckv", 2 * d), ("b_co", d),
                     ("b_f1", wl.ffn), ("b_f2", d)):
            b[n] = zf(k)
        blocks.append(b)
        kcs.append(rn(wl.B, wl.Lcap, wl.H, wl.Dh, std=1.0))
        vcs.append(rn(wl.B, wl.Lcap, wl.H, wl.Dh, std=1.0))
    dims = w.make_dims(d, wl.H, wl.Dh, wl.ffn, wl.n_layers, wl.latent_ch, wl.act_dim, wl.text_dim,
                       wl.freq_dim, wl.eps)
    model = w.make_model(dims, top, blocks)
    inputs = {
        "z": rn(wl.B, wl.latent_ch, wl.F, wl.Hl, wl.Wl, std=1.0),
        "a": rn(wl.B, wl.A, wl.act_dim, std=1.0),
        "t": torch.rand(wl.B, generator=g, device=dev),
        "text": rn(wl.B, wl.Lc, wl.text_dim, std=1.0),
    }
    pos = w.wam_chunk_positions(wl.n_cached, wl.F, wl.Hg, wl.Wg, wl.A)
    cos, sin = w.wam_rope_tables(pos, wl.Dh)
    inputs["cos"] = torch.from_numpy(cos).to(dev)
    inputs["sin"] = torch.from_numpy(sin).to(dev)
    return model, (top, blocks), kcs, vcs, inputs


# Per-role algorithmic work of one block launch at the workload's shapes: flops for the
# matrix kernels (2*M*N*K per projection, 4*Dh per visible (q, k) pair per head for
# attention), bytes for the memory-bound ones (LayerNorm: fp32 row in, bf16 row out;
# RoPE/append: the bf16 q|k|v row in, q, k and v out).
def role_work(wl, ln_out_bytes=2):
    """Algorithmic work of each role per launch: flops, or bytes (a LayerNorm reads 4 and
    writes ln_out_bytes per element: 2 for bf16 rows, 1 for the E4M3 rows of the FP8 step)."""
    M, d, F = wl.B * wl.L, wl.d, wl.ffn
    ln = M * d * (4 + ln_out_bytes)
    return {
        "ln1": ("GB/s", ln), "qkv": ("TFLOP/s", 2 * M * d * 3 * d), "rope": ("GB/s", M * 3 * d * 2 * 2),
        "self_attn": ("TFLOP/s", 4 * wl.H * wl.Dh * M * wl.Lk), "o": ("TFLOP/s", 2 * M * d * d),
        "lnc": ("GB/s", ln), "cq": ("TFLOP/s", 2 * M * d * d),
        "cross_attn": ("TFLOP/s", 4 * wl.H * wl.Dh * M * wl.Lc), "co": ("TFLOP/s", 2 * M * d * d),
        "ln2": ("GB/s", ln), "ffn1": ("TFLOP/s", 2 * M * d * F), "ffn2": ("TFLOP/s", 2 * M * F * d),
    }


MI355X_HBM_GBPS = 8000.0  # published HBM3E peak


def profiled_roles(wl, model, kcs, vcs, inp, vv, va, torch, n_steps, mfma_peak=None, ln_out_bytes=2, rope_fused=False,
                   **io_kw):
    """Per-role average launch time over n_steps untimed steps that record events around
    every launch of every block, with each role's achieved rate and fraction of its peak
    (dense MFMA at mfma_peak, bf16's by default, for GEMMs and attention; HBM for LayerNorm
    and RoPE; rope_fused: the step runs RoPE and the K/V append in the QKV projection's
    epilogue, as the bf16 step does, so its events bracket no launch).  io_kw: extra step
    inputs (the FP8 KV cache's exponents and scales)."""
    import paper_2602_15922_amd as w
    names = w.binding.BLOCK_EVENT_NAMES
    nk = len(names)
    chunks = w.cached_chunks(wl.cache_rows, wl.L)
    sums = [0.0] * nk
    ws = None
    for _ in range(n_steps):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * nk * wl.n_layers)]
        io = w.make_step_io(inp["z"], inp["a"], inp["t"], inp["text"], kcs, vcs, inp["cos"], inp["sin"],
                            wl.cache_rows, chunks, vv, va, block_events=ev, **io_kw)
        if ws is None:
            ws = torch.empty(w.wam_step_workspace_bytes(model, io), dtype=torch.uint8, device="cuda")
        w.wam_dit_step_fwd(model, io, ws)
        torch.cuda.synchronize()
        for l in range(wl.n_layers):
            for k in range(nk):
                sums[k] += ev[2 * (l * nk + k)].elapsed_time(ev[2 * (l * nk + k) + 1])
    work = role_work(wl, ln_out_bytes)
    out = {}
    for k, name in enumerate(names):
        ms = sums[k] / (n_steps * wl.n_layers)
        unit, amount = work[name]
        if name == "rope" and rope_fused:
            out[name] = {"ms": round(ms, 4), "achieved": None, "unit": unit, "frac": None,
                         "work_per_launch": amount, "fused": "in the QKV projection's epilogue"}
            continue
        if unit == "TFLOP/s":
            rate = amount / (ms * 1e-3) / 1e12
            peak = mfma_peak or MI355X_BF16_DENSE_TFLOPS
        else:
            rate = amount / (ms * 1e-3) / 1e9
            peak = MI355X_HBM_GBPS
        out[name] = {"ms": round(ms, 4), "achieved": round(rate, 1), "unit": unit, "frac": round(rate / peak, 4),
                     "work_per_launch": amount}
    return out


def attn_traffic():
    """HBM bytes per self-attention launch from the committed counter profile, or None
    when the attention kernel's source has changed since the counters were taken."""
    import hashlib
    prof = os.path.join(ROOT, "profiles", "attn_fwd_step_14b_traffic.md")
    if not os.path.exists(prof):
        return None
    fields = {}
    for line in open(prof):
        if ":" in line and line.split(":")[0] in ("traffic_bytes_per_launch", "kernel_source_sha256"):
            k, v = line.split(":", 1)
            fields[k] = v.strip()
    h = hashlib.sha256()
    for f in ("attn.hip", "common.h"):
        with open(os.path.join(ROOT, "paper_2602_15922_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    if fields.get("kernel_source_sha256") != h.hexdigest():
        return None
    return int(fields["traffic_bytes_per_launch"])


def extras(wl, model, keep, kcs, vcs, inp, torch, reps=3):
    """Timings of the other entry points on the same model and workload (milliseconds,
    HIP events on the current stream, after one warm-up call each): the DreamZero-Flash
    step (actions at their own timestep), the cache-update pass over one clean video-only
    chunk (3120 rows after the cached ones), a 4-step Euler denoising loop, the step with
    the text's projection and cross K|V cached per episode (computed once, passed in), the
    step with every block's seven projections as FP8 (E4M3) GEMMs, and that step with an FP8
    KV cache (self-attention in FP8; also its average self-attention launch, from events
    recorded around each launch of the last timed call)."""
    import numpy as np
    import paper_2602_15922_amd as w
    B = wl.B
    dev = "cuda"

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    out = {}
    vv = torch.empty((B, wl.latent_ch, wl.F, wl.Hl, wl.Wl), dtype=torch.float32, device=dev)
    va = torch.empty((B, wl.A, wl.act_dim), dtype=torch.float32, device=dev)
    chunks = w.cached_chunks(wl.cache_rows, wl.L)
    t_act = torch.full((B,), 0.9, device=dev)
    io_f = w.make_step_io(inp["z"], inp["a"], inp["t"], inp["text"], kcs, vcs, inp["cos"], inp["sin"],
                          wl.cache_rows, chunks, vv, va, t_action=t_act)
    ws = torch.empty(w.wam_step_workspace_bytes(model, io_f), dtype=torch.uint8, device=dev)
    out["flash_step_ms"] = round(timed(lambda: w.wam_dit_step_fwd(model, io_f, ws)), 3)

    # update pass: the clean chunk's video rows only (Algorithm 2 passes no actions)
    Lu = wl.Lv
    a0 = torch.empty((B, 0, wl.act_dim), dtype=torch.bfloat16, device=dev)
    pos = w.wam_chunk_positions(wl.n_cached, wl.F, wl.Hg, wl.Wg, 0)
    cu, su = (torch.from_numpy(x).to(dev) for x in w.wam_rope_tables(pos, wl.Dh))
    io_u = w.make_step_io(inp["z"], a0, inp["t"], inp["text"], kcs, vcs, cu, su, wl.cache_rows,
                          w.cached_chunks(wl.cache_rows, Lu), None, None)
    ws_u = torch.empty(w.wam_update_workspace_bytes(model, io_u), dtype=torch.uint8, device=dev)
    out["update_pass_ms"] = round(timed(lambda: w.wam_dit_update_fwd(model, io_u, ws_u)), 3)

    # 4-step Euler loop of one chunk, no guidance, no caching
    n = wl.latent_ch * wl.F * wl.Hl * wl.Wl + wl.A * wl.act_dim
    x = torch.randn(B, n, device=dev)
    x0 = x.clone()
    tl = torch.zeros(B, device=dev)
    io_l = w.make_step_io(inp["z"], inp["a"], tl, inp["text"], kcs, vcs, inp["cos"], inp["sin"],
                          wl.cache_rows, chunks, vv, va)
    p = w.make_denoise_params(np.linspace(0.0, 1.0, 5), x)
    ws_l = torch.empty(w.wam_denoise_workspace_bytes(model, io_l, p), dtype=torch.uint8, device=dev)

    def loop():
        x.copy_(x0)
        w.wam_denoise_chunk(model, io_l, p, ws_l)

    out["denoise_4step_ms"] = round(timed(loop), 3)
    assert torch.isfinite(x).all()
    # the same loop with UniPC of order 2 (its schedule starts just after t = 0)
    p_u = w.make_denoise_params([0.02, 0.27, 0.51, 0.76, 1.0], x, solver=w.binding.WAM_SOLVER_UNIPC, order=2)
    ws_u2 = torch.empty(w.wam_denoise_workspace_bytes(model, io_l, p_u), dtype=torch.uint8, device=dev)

    def loop_u():
        x.copy_(x0)
        w.wam_denoise_chunk(model, io_l, p_u, ws_u2)

    out["denoise_4step_unipc_ms"] = round(timed(loop_u), 3)
    assert torch.isfinite(x).all()

    # the step with the text conditioning cached per episode: the text projection and every
    # block's cross K|V computed once (by the library's own entry points) and passed in
    top, blocks = keep
    ctx = torch.empty((B, wl.Lc, wl.d), dtype=torch.bfloat16, device=dev)
    ws_t = torch.empty(w.wam_text_proj_workspace_bytes(model.dims, B, wl.Lc), dtype=torch.uint8, device=dev)
    w.wam_text_proj_fwd(model, inp["text"], ctx, ws_t)
    kvs = []
    for b in blocks:
        kv = torch.empty((B, wl.Lc, 2 * wl.d), dtype=torch.bfloat16, device=dev)
        w.wam_gemm_bf16(ctx.view(-1, wl.d), b["w_ckv"], kv.view(-1, 2 * wl.d), w.WAM_EPI_BF16, bias=b["b_ckv"])
        kvs.append(kv)
    io_c = w.make_step_io(inp["z"], inp["a"], inp["t"], inp["text"], kcs, vcs, inp["cos"], inp["sin"],
                          wl.cache_rows, chunks, vv, va, ctx_kv=kvs)
    ws_c = torch.empty(w.wam_step_workspace_bytes(model, io_c), dtype=torch.uint8, device=dev)
    out["step_text_cached_ms"] = round(timed(lambda: w.wam_dit_step_fwd(model, io_c, ws_c)), 3)
    del kvs, ws_c

    # FP8 projections: E4M3 copies of every block's matrices, made on the device
    blocks8 = [dict(b, fp8=w.make_block_fp8(b)) for b in blocks]
    model8 = w.make_model(model.dims, top, blocks8)
    io8 = w.make_step_io(inp["z"], inp["a"], inp["t"], inp["text"], kcs, vcs, inp["cos"], inp["sin"],
                         wl.cache_rows, chunks, vv, va)
    ws8 = torch.empty(w.wam_step_workspace_bytes(model8, io8), dtype=torch.uint8, device=dev)
    out["fp8_step_ms"] = round(timed(lambda: w.wam_dit_step_fwd(model8, io8, ws8)), 3)
    assert torch.isfinite(vv).all()

    # FP8 projections and an FP8 KV cache (FP8 self-attention): E4M3 caches made from the
    # bf16 ones with the library's quantizers, V's per-layer scale max|V| / 448 over the
    # rows the step reads and writes (the bf16 steps above wrote this chunk's rows: a
    # calibration pass)
    rows = wl.cache_rows + wl.L
    k8s, kes, v8s, vsc = [], [], [], []
    for kc, vc in zip(kcs, vcs):
        Bc, Lcap, H, Dh = kc.shape
        k8 = torch.empty((Bc, Lcap, H, Dh), dtype=torch.uint8, device=dev)
        ke = torch.empty((Bc, Lcap, H), dtype=torch.int32, device=dev)
        w.wam_quantize_mx_fp8(kc.view(Bc * Lcap, H * Dh), k8.view(Bc * Lcap, H * Dh),
                              ke.view(torch.uint8).view(Bc * Lcap, H * 4))
        vs = float(vc[:, :rows].abs().max().float()) / 448.0
        v8 = torch.empty_like(k8)
        w.wam_quantize_scaled_fp8(vc, vs, v8)
        k8s.append(k8)
        kes.append(ke)
        v8s.append(v8)
        vsc.append(vs)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * wl.n_layers)]
    io8a = w.make_step_io(inp["z"], inp["a"], inp["t"], inp["text"], k8s, v8s, inp["cos"], inp["sin"],
                          wl.cache_rows, chunks, vv, va, events=ev, k_exps=kes, v_scales=vsc)
    out["fp8_attn_step_ms"] = round(timed(lambda: w.wam_dit_step_fwd(model8, io8a, ws8)), 3)
    torch.cuda.synchronize()
    out["fp8_attn_kernel_ms"] = round(sum(ev[2 * l].elapsed_time(ev[2 * l + 1]) for l in range(wl.n_layers))
                                      / wl.n_layers, 4)
    assert torch.isfinite(vv).all()
    # the same step with events around every launch of every block: per-role times of the
    # FP8 path, MFMA roles against the FP8 dense peak (the O, cross-O and FFN2 roles include
    # the row quantization of their input; the three LayerNorms write E4M3 rows themselves
    # where the width allows it, a byte per element)
    ln8 = wl.d % 512 == 0 and 512 <= wl.d <= 5120
    roles8 = profiled_roles(wl, model8, k8s, v8s, inp, vv, va, torch, 1, mfma_peak=MI355X_FP8_DENSE_TFLOPS,
                            ln_out_bytes=1 if ln8 else 2, k_exps=kes, v_scales=vsc)
    out["fp8_roles"] = {k: {"ms": v["ms"], "achieved": v["achieved"], "unit": v["unit"], "frac": v["frac"]}
                        for k, v in roles8.items()}
    del blocks8, model8, ws8, k8s, v8s, kes
    return out


def cpu_baseline(wl):
    """The fp64 oracle on one full-shape block of the workload (a 1/40 sample of the
    step's blocks), scaled to steps/s; inputs come from the seeded generators."""
    import numpy as np
    import oracle
    import synth
    threads, vendor = None, "unknown"
    try:
        from threadpoolctl import threadpool_info
        blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if blas:
            threads = max(i.get("num_threads", 1) for i in blas)
            vendor = ", ".join(sorted({f"{i.get('internal_api')} {i.get('version')}" for i in blas}))
    except Exception:  # pragma: no cover
        pass
    cores = len(os.sched_getaffinity(0))
    threads = threads or cores
    cpu_model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:  # pragma: no cover
        pass
    W = {k: v.f64 for k, v in synth.block_params(wl, 0).items()}
    kc, vc = synth.kv_cache(wl, 0)
    x = synth.normal(wl.seed, "x", (wl.B, wl.L, wl.d), 1.0, dtype="f32").f64
    e0 = synth.normal(wl.seed, "e0", (wl.B, 6, wl.d), 0.02, dtype="f32").f64
    ctx = synth.normal(wl.seed, "ctx", (wl.B, wl.Lc, wl.d), 1.0).f64
    pos = oracle.chunk_positions(wl.n_cached, wl.F, wl.Hg, wl.Wg, wl.A)
    t0 = time.perf_counter()
    oracle.dit_block(x, e0, W, wl.H, wl.eps, pos, np.full(wl.L, wl.n_cached), kc.f64, vc.f64,
                     np.repeat(np.arange(wl.n_cached), wl.L), ctx=ctx)
    dt = time.perf_counter() - t0
    step_s = dt * wl.n_layers
    return {"value": 1.0 / step_s, "unit": "steps/s", "cores": int(threads), "kind": "oracle",
            "affinity_cores": cores, "blas_threads": int(threads), "blas": vendor, "cpu_model": cpu_model,
            "sample": f"one full-shape block ({dt:.1f} s fp64 numpy on {threads} BLAS threads), "
                      f"x{wl.n_layers} blocks; embeddings and head not timed"}


def probe_attn(wl, n):
    """Launch a plain device-to-device copy of known size (the calibration for HBM byte
    counters) and n self-attention launches of the step's shape (queries of one chunk
    against the cached chunks plus itself), with nothing else on the GPU in between."""
    import torch
    import paper_2602_15922_amd as w
    torch.cuda.set_device(0)
    g = torch.Generator(device="cuda").manual_seed(7)
    copy_bytes = 1 << 30
    src = torch.randn(copy_bytes // 2, generator=g, device="cuda", dtype=torch.bfloat16)
    dst = torch.empty_like(src)
    q = torch.randn(wl.B, wl.L, wl.H, wl.Dh, generator=g, device="cuda", dtype=torch.bfloat16)
    k = torch.randn(wl.B, wl.Lk, wl.H, wl.Dh, generator=g, device="cuda", dtype=torch.bfloat16)
    v = torch.randn_like(k)
    o = torch.empty_like(q)
    chunks = w.cached_chunks(wl.cache_rows, wl.L)
    torch.cuda.synchronize()
    torch.mul(src, 1, out=dst)  # one elementwise kernel: reads and writes copy_bytes
    torch.cuda.synchronize()
    for _ in range(n):
        w.wam_attn_blockcausal(q, k, v, o, chunks)
    torch.cuda.synchronize()
    assert torch.isfinite(o).all()
    print(json.dumps({"probe": "attn", "workload": wl.name, "copy_bytes": copy_bytes, "attn_launches": n,
                      "q": list(q.shape), "kv": list(k.shape)}), flush=True)


def probe_attn_fp8(wl, n):
    """The same as probe_attn for the FP8 attention: the calibration copy, the operands
    quantized by the library (MX blocks for q and k, one scale for v), then n FP8
    self-attention launches of the step's shape."""
    import torch
    import paper_2602_15922_amd as w
    torch.cuda.set_device(0)
    g = torch.Generator(device="cuda").manual_seed(7)
    copy_bytes = 1 << 30
    src = torch.randn(copy_bytes // 2, generator=g, device="cuda", dtype=torch.bfloat16)
    dst = torch.empty_like(src)
    B, L, Lk, H, Dh = wl.B, wl.L, wl.Lk, wl.H, wl.Dh
    ops = {}
    for name, rows in (("q", L), ("k", Lk)):
        x = torch.randn(B * rows, H * Dh, generator=g, device="cuda", dtype=torch.bfloat16)
        c = torch.empty((B, rows, H, Dh), dtype=torch.uint8, device="cuda")
        e = torch.empty((B, rows, H), dtype=torch.int32, device="cuda")
        w.wam_quantize_mx_fp8(x, c.view(B * rows, H * Dh), e.view(torch.uint8).view(B * rows, H * 4))
        ops[name] = (c, e)
    v = torch.randn(B, Lk, H, Dh, generator=g, device="cuda", dtype=torch.bfloat16)
    vs = float(v.abs().max().float()) / 448.0
    v8 = torch.empty((B, Lk, H, Dh), dtype=torch.uint8, device="cuda")
    w.wam_quantize_scaled_fp8(v, vs, v8)
    o = torch.empty((B, L, H, Dh), dtype=torch.bfloat16, device="cuda")
    chunks = w.cached_chunks(wl.cache_rows, L)
    torch.cuda.synchronize()
    torch.mul(src, 1, out=dst)
    torch.cuda.synchronize()
    for _ in range(n):
        w.wam_attn_blockcausal_fp8(ops["q"][0], ops["q"][1], ops["k"][0], ops["k"][1], v8, vs, o, chunks)
    torch.cuda.synchronize()
    assert torch.isfinite(o).all()
    print(json.dumps({"probe": "attn_fp8", "workload": wl.name, "copy_bytes": copy_bytes, "attn_launches": n,
                      "q": [B, L, H, Dh], "kv": [B, Lk, H, Dh]}), flush=True)


def _calibration_copy(torch, g):
    """One elementwise kernel that reads and writes 1 GiB: the known traffic that scales
    the HBM byte counters."""
    copy_bytes = 1 << 30
    src = torch.randn(copy_bytes // 2, generator=g, device="cuda", dtype=torch.bfloat16)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    torch.mul(src, 1, out=dst)
    torch.cuda.synchronize()
    return copy_bytes


def probe_kernels(wl, kind, n):
    """Counter-collection mode for the non-attention kernels: the calibration copy, then n
    launches of each of the block's six projections with their epilogues (qkv, o, cq, co,
    ffn1, ffn2, in that order) at the step's shapes, or n launches of the AdaLN LayerNorm,
    or of the RoPE/KV-append kernel."""
    import torch
    import paper_2602_15922_amd as w
    torch.cuda.set_device(0)
    g = torch.Generator(device="cuda").manual_seed(7)
    M, d, F = wl.B * wl.L, wl.d, wl.ffn

    def rn(*shape, std=1.0):
        return (torch.randn(*shape, generator=g, device="cuda") * std).to(torch.bfloat16)

    copy_bytes = _calibration_copy(torch, g)
    ran = []
    if kind == "torch_linear":
        # reference point, not part of the library: PyTorch's linear (hipBLASLt) on the same
        # projection shapes, plain bf16 output, no fused epilogue
        for name, K, N in (("qkv", d, 3 * d), ("o", d, d), ("ffn1", d, F), ("ffn2", F, d)):
            A, Wt = rn(M, K), rn(N, K, std=0.02)
            torch.cuda.synchronize()
            for _ in range(n):
                out = torch.nn.functional.linear(A, Wt)
            torch.cuda.synchronize()
            ran.append({"role": name, "M": M, "N": N, "K": K, "launches": n, "out": list(out.shape)})
            del A, Wt, out
    elif kind == "gemm":
        x = torch.randn(M, d, generator=g, device="cuda")
        gate = torch.randn(6, d, generator=g, device="cuda") * 0.02
        roles = (("qkv", d, 3 * d, w.WAM_EPI_BF16), ("o", d, d, w.WAM_EPI_RESID_F32),
                 ("cq", d, d, w.WAM_EPI_BF16), ("co", d, d, w.WAM_EPI_RESID_F32),
                 ("ffn1", d, F, w.WAM_EPI_GELU_BF16), ("ffn2", F, d, w.WAM_EPI_RESID_F32))
        for name, K, N, epi in roles:
            A, Wt = rn(M, K), rn(N, K, std=0.02)
            bias = torch.zeros(N, device="cuda")
            out = x if epi == w.WAM_EPI_RESID_F32 else torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
            gated = name in ("o", "ffn2")
            torch.cuda.synchronize()
            for _ in range(n):
                w.wam_gemm_bf16(A, Wt, out, epi, bias=bias, gate_a=gate[2] if gated else None,
                                gate_v=gate[3] if gated else None, gate_rows=wl.L if gated else 0)
            torch.cuda.synchronize()
            ran.append({"role": name, "M": M, "N": N, "K": K, "epilogue": epi, "launches": n})
            del A, Wt
        assert torch.isfinite(x).all()
    elif kind == "gemm_fp8":
        # the FP8-attention step's projections: E4M3 operands, per-channel weight scales; QKV,
        # cross-Q and FFN1 read row-scaled rows (as the LayerNorms write them), O, cross-O and
        # FFN2 block-scaled ones (as the attentions and FFN1 write them), FFN1 writes its output
        # block-scaled.  Random codes (no NaN code), unit block exponents: the counters depend
        # on the shapes and the code path, not on the values.
        def codes(*shape):
            c = torch.randint(0, 0x70, shape, generator=g, device="cuda", dtype=torch.int32)
            return (c | (torch.randint(0, 2, shape, generator=g, device="cuda", dtype=torch.int32) << 7)).to(torch.uint8)

        x = torch.randn(M, d, generator=g, device="cuda")
        gate = torch.randn(6, d, generator=g, device="cuda") * 0.02
        roles = (("qkv", d, 3 * d, w.WAM_EPI_BF16, "rows"), ("o", d, d, w.WAM_EPI_RESID_F32, "blocks"),
                 ("cq", d, d, w.WAM_EPI_BF16, "rows"), ("co", d, d, w.WAM_EPI_RESID_F32, "blocks"),
                 ("ffn1", d, F, w.WAM_EPI_GELU_BF16, "rows"), ("ffn2", F, d, w.WAM_EPI_RESID_F32, "blocks"))
        for name, K, N, epi, a_kind in roles:
            A, Wt = codes(M, K), codes(N, K)
            sw = torch.rand(N, generator=g, device="cuda") * 1e-3
            bias = torch.zeros(N, device="cuda")
            lde = 4 * M
            if a_kind == "rows":
                sa, ae = torch.rand(M, generator=g, device="cuda") * 1e-2, None
            else:
                sa, ae = None, torch.full(((K // 128) * lde,), 127, dtype=torch.uint8, device="cuda")
            oe = None
            if epi == w.WAM_EPI_RESID_F32:
                out = x
            elif epi == w.WAM_EPI_GELU_BF16:
                out = torch.empty(M, N, dtype=torch.uint8, device="cuda")
                oe = torch.empty(((N // 128) * lde,), dtype=torch.uint8, device="cuda")
            else:
                out = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
            gated = name in ("o", "ffn2")
            torch.cuda.synchronize()
            for _ in range(n):
                w.wam_gemm_fp8_mx(A, Wt, out, epi, sw, a_scale=sa, a_exp=ae, a_lde=lde if ae is not None else 0,
                                  out_exp=oe, o_lde=lde if oe is not None else 0, bias=bias,
                                  gate_a=gate[2] if gated else None)
            torch.cuda.synchronize()
            ran.append({"role": name, "M": M, "N": N, "K": K, "epilogue": epi, "a": a_kind,
                        "out": "blocks" if oe is not None else "plain", "launches": n})
            del A, Wt
        assert torch.isfinite(x).all()
    elif kind == "ln":
        x = torch.randn(M, d, generator=g, device="cuda")
        h = torch.empty(M, d, dtype=torch.bfloat16, device="cuda")
        mod = torch.randn(4, d, generator=g, device="cuda") * 0.02
        torch.cuda.synchronize()
        for _ in range(n):
            w.wam_adaln_ln_mod(x, h, wl.eps, wl.L, shift_a=mod[0], shift_v=mod[1], scale_a=mod[2], scale_v=mod[3])
        torch.cuda.synchronize()
        ran.append({"kernel": "ln_mod", "rows": M, "d": d, "launches": n})
    else:
        qkv = rn(wl.B, wl.L, 3 * d)
        q = torch.empty(wl.B, wl.L, d, dtype=torch.bfloat16, device="cuda")
        kc = torch.zeros(wl.B, wl.Lcap, wl.H, wl.Dh, dtype=torch.bfloat16, device="cuda")
        vc = torch.zeros_like(kc)
        pos = w.wam_chunk_positions(wl.n_cached, wl.F, wl.Hg, wl.Wg, wl.A)
        cos, sin = (torch.from_numpy(a).to("cuda") for a in w.wam_rope_tables(pos, wl.Dh))
        torch.cuda.synchronize()
        for _ in range(n):
            w.wam_rope_qkv(qkv, cos, sin, q, kc, vc, wl.cache_rows, wl.H, wl.Dh)
        torch.cuda.synchronize()
        ran.append({"kernel": "rope_qkv", "rows": M, "d": d, "launches": n})
    print(json.dumps({"probe": kind, "workload": wl.name, "copy_bytes": copy_bytes, "ran": ran}), flush=True)


def pmc_summary(path):
    """Per-kernel averages of the counters in a rocprofv3 counter-collection CSV (one row
    per dispatch and counter), in dispatch order of each kernel's first appearance.  The
    CSV's GRBM_GUI_ACTIVE is the sum over the 8 XCDs, so where the inputs are present it
    adds rocprofv3's MfmaUtil formula, sum(SQ_VALU_MFMA_BUSY_CYCLES) / (max over XCDs of
    GRBM_GUI_ACTIVE x 1024 SIMDs), with the max taken as the sum / 8, and the shader clock
    implied by GRBM_GUI_ACTIVE / 8 over the dispatch's duration."""
    import csv
    import glob
    files = sorted(glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True))
    if not files:
        sys.exit(f"no counter_collection.csv under {path}")
    disp = {}
    for f in files:
        for r in csv.DictReader(open(f)):
            key = (f, int(r["Dispatch_Id"]))
            dd = disp.setdefault(key, {"kernel": r["Kernel_Name"], "ns": int(r["End_Timestamp"]) -
                                       int(r["Start_Timestamp"]), "grid": r["Grid_Size"], "c": {}})
            dd["c"][r["Counter_Name"]] = float(r["Counter_Value"])
    kern = {}  # (kernel, grid size) -> dispatches: one row per launch shape
    for key in sorted(disp):
        dd = disp[key]
        name = dd["kernel"].replace("(anonymous namespace)::", "").split("(")[0][:100]
        kern.setdefault(f"{name}` grid {dd['grid']}", []).append(dd)
    counters = sorted({c for dd in disp.values() for c in dd["c"]})
    print("| kernel | dispatches | avg µs | " + " | ".join(counters) + " | MfmaUtil % | clock GHz |")
    print("|---|---:|---:|" + "---:|" * (len(counters) + 2))
    for name, ds in kern.items():
        avg = {c: sum(d_["c"].get(c, 0.0) for d_ in ds) / len(ds) for c in counters}
        us = sum(d_["ns"] for d_ in ds) / len(ds) / 1e3
        util = clk = ""
        gui = avg.get("GRBM_GUI_ACTIVE", 0.0) / 8.0
        if "SQ_VALU_MFMA_BUSY_CYCLES" in avg and gui:
            util = f"{100.0 * avg['SQ_VALU_MFMA_BUSY_CYCLES'] / (gui * 1024):.1f}"
        if gui and us > 0:
            clk = f"{gui / (us * 1e3):.2f}"
        print(f"| `{name} | {len(ds)} | {us:.1f} | " + " | ".join(f"{avg[c]:.6g}" for c in counters)
              + f" | {util} | {clk} |")


def trace_summary(path, steps):
    """Kernel time by (kernel, grid size) from a rocprofv3 kernel-trace CSV: calls, average,
    min and max duration, total, share of all kernel time, and (steps > 0) milliseconds per
    step over the dispatches of the run's last `steps` steps, a step being delimited by
    the time-embedding kernel that opens it."""
    import csv
    import glob
    files = sorted(glob.glob(os.path.join(path, "**", "*kernel_trace.csv"), recursive=True))
    if not files:
        sys.exit(f"no kernel_trace.csv under {path}")
    rows = []
    for f in files:
        for r in csv.DictReader(open(f)):
            name = r["Kernel_Name"].replace("(anonymous namespace)::", "").replace("wam::", "")
            rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), name.split("(")[0][:80], r.get("Grid_Size") or r.get("Grid_Size_X")))
    rows.sort()
    total = sum(e - b for b, e, _, _ in rows)
    if steps > 0:
        starts = [i for i, r in enumerate(rows) if r[2].startswith("sinusoid_kernel")]
        if len(starts) >= steps:
            rows_s = rows[starts[-steps]:]
        else:
            rows_s = rows
    agg = {}
    for b, e, n, g in rows:
        a = agg.setdefault((n, g), [0, 0, 1e18, 0])
        a[0] += 1
        a[1] += e - b
        a[2] = min(a[2], e - b)
        a[3] = max(a[3], e - b)
    per_step = {}
    if steps > 0:
        for b, e, n, g in rows_s:
            per_step[(n, g)] = per_step.get((n, g), 0) + e - b
    print("| kernel | grid | calls | avg us | min us | max us | total ms | % |" + (" ms/step |" if steps else ""))
    print("|---|---:|---:|---:|---:|---:|---:|---:|" + ("---:|" if steps else ""))
    for (n, g), a in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        if a[1] < 0.001 * total:
            continue
        line = (f"| `{n}` | {g} | {a[0]} | {a[1] / a[0] / 1e3:.1f} | {a[2] / 1e3:.1f} | {a[3] / 1e3:.1f} | "
                f"{a[1] / 1e6:.1f} | {100.0 * a[1] / total:.1f} |")
        if steps:
            line += f" {per_step.get((n, g), 0) / 1e6 / steps:.3f} |"
        print(line)
    if steps:
        print(f"\nkernel time per step over the last {steps} steps: {sum(per_step.values()) / 1e6 / steps:.2f} ms")


def main():
    args = parse()
    if args.pmc_summary:
        return pmc_summary(args.pmc_summary)
    if args.trace_summary:
        return trace_summary(args.trace_summary, args.trace_steps)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this build runs on one GPU only (no sharding or collectives); "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    import synth
    import paper_2602_15922_amd as w

    wl = synth.WORKLOADS[args.workload]
    if args.probe_attn:
        return probe_attn(wl, args.probe_attn)
    if args.probe_attn_fp8:
        return probe_attn_fp8(wl, args.probe_attn_fp8)
    if args.probe:
        return probe_kernels(wl, args.probe, args.probe_n)
    torch.cuda.set_device(0)
    model, keep, kcs, vcs, inp = build_model(wl, torch)
    B, d = wl.B, wl.d
    vv = torch.empty((B, wl.latent_ch, wl.F, wl.Hl, wl.Wl), dtype=torch.float32, device="cuda")
    va = torch.empty((B, wl.A, wl.act_dim), dtype=torch.float32, device="cuda")
    chunks = w.cached_chunks(wl.cache_rows, wl.L)
    n_ev = 2 * wl.n_layers
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(n_ev)] for _ in range(args.steps)]
    ios = [w.make_step_io(inp["z"], inp["a"], inp["t"], inp["text"], kcs, vcs, inp["cos"], inp["sin"],
                          wl.cache_rows, chunks, vv, va, events=events[i]) for i in range(args.steps)]
    io_plain = w.make_step_io(inp["z"], inp["a"], inp["t"], inp["text"], kcs, vcs, inp["cos"], inp["sin"],
                              wl.cache_rows, chunks, vv, va)
    ws = torch.empty(w.wam_step_workspace_bytes(model, io_plain), dtype=torch.uint8, device="cuda")

    for _ in range(args.warmup):
        w.wam_dit_step_fwd(model, io_plain, ws)
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for i in range(args.steps):
        w.wam_dit_step_fwd(model, ios[i], ws)
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = start.elapsed_time(stop) / args.steps
    assert torch.isfinite(vv).all() and torch.isfinite(va).all()

    attn_ms = [events[i][2 * l].elapsed_time(events[i][2 * l + 1])
               for i in range(args.steps) for l in range(wl.n_layers)]
    attn_avg = sum(attn_ms) / len(attn_ms)
    attn_flop = 4.0 * wl.H * wl.Dh * wl.B * wl.L * wl.Lk  # visible (q, k) pairs x 4 Dh
    attn_tflops = attn_flop / (attn_avg * 1e-3) / 1e12
    step_flop = wl.step_flops()

    rec = {
        "metric": "DiT denoising steps/sec (14B-class chunk); attention TFLOP/s as % bf16 MFMA peak",
        "value": round(1000.0 / ms, 4),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic Gaussians of the workload's shapes; random-init bf16 weights",
        "config": {"workload": f"{wl.name}: {wl.n_layers} blocks, d={d}, {wl.H}x{wl.Dh} heads, FFN {wl.ffn}, "
                               f"chunk {wl.Lv}+{wl.A} tokens, {wl.n_cached} cached chunks (Lk {wl.Lk}), "
                               f"text {wl.Lc}x{wl.text_dim}, batch {B}",
                   "global_batch": B, "seq_len": wl.L, "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "mfma", "kernel": "attn_fwd (block-causal self-attention)",
                     "achieved": round(attn_tflops, 1), "peak": MI355X_BF16_DENSE_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(attn_tflops / MI355X_BF16_DENSE_TFLOPS, 4),
                     "traffic": attn_traffic() if wl.name == WORKLOAD else None, "traffic_unit": "bytes",
                     "avg_launch_ms": round(attn_avg, 4), "flop_per_launch": attn_flop},
        "step_tflops": round(step_flop / (ms * 1e-3) / 1e12, 1),
        "step_mfma_frac": round(step_flop / (ms * 1e-3) / 1e12 / MI355X_BF16_DENSE_TFLOPS, 4),
        "wall_s_timed": round(wall, 3),
    }
    if args.profile_steps > 0:
        roles = profiled_roles(wl, model, kcs, vcs, inp, vv, va, torch, args.profile_steps, rope_fused=wl.d % 64 == 0)
        rec["gemm_roofline"] = {k: roles[k] for k in ("qkv", "o", "cq", "co", "ffn1", "ffn2")}
        rec["gemm_roofline"]["source"] = (f"events around every launch of every block over {args.profile_steps} "
                                          "untimed steps after the timed ones; peak: bf16 dense MFMA")
        rec["kernel_roles"] = {k: roles[k] for k in ("ln1", "rope", "self_attn", "lnc", "cross_attn", "ln2")}
    if not args.no_extras:
        rec["extras"] = extras(wl, model, keep, kcs, vcs, inp, torch)
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
