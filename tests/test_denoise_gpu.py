"""GPU parity of the denoising loop of Algorithm 2 against the fp64 oracle: the fused
guidance + Euler + bf16 re-quantization step, the deterministic cosine similarity, and
wam_denoise_chunk (plain, with classifier-free guidance, with DiT caching) driving the
d=512 network through several steps."""
import numpy as np
import pytest

import oracle
import synth
from dit_cases import StepCase, f64, oracle_positions, prev_chunk_ids
from gpu_helpers import dev, host, log, rel_l2, workspace

pytestmark = pytest.mark.gpu
TOL = 2e-2


def lib():
    import paper_2602_15922_amd as w
    return w


def bf16_round(x):
    return synth.bf16_from_bits(synth.bf16_bits(np.asarray(x, dtype=np.float32)))


@pytest.mark.parametrize("cfg", [False, True])
def test_flow_step_matches_oracle(cfg):
    import torch
    w = lib()
    g = np.random.default_rng(140)
    B, nv, na = (2, 1000, 37) if cfg else (3, 1003, 16)
    nx = 1 if cfg else B
    vv, va = g.standard_normal((B, nv)).astype(np.float32), g.standard_normal((B, na)).astype(np.float32)
    x0 = g.standard_normal((nx, nv + na)).astype(np.float32)
    s, t, tn = 3.5, 0.25, 0.4
    dims = w.binding.wam_flow_dims(B=B, cfg=int(cfg), cfg_scale=s, n_video=nv, n_action=na)
    x = dev(x0)
    z = torch.empty((B, nv), dtype=torch.bfloat16, device="cuda")
    a = torch.empty((B, na), dtype=torch.bfloat16, device="cuda")
    vout = torch.empty((nx, nv + na), dtype=torch.float32, device="cuda")
    log(f"flow step cfg={cfg}")
    w.wam_flow_step(dims, x, z, a, t, tn, v_video=dev(vv), v_action=dev(va), v_out=vout)
    torch.cuda.synchronize()
    v64 = np.concatenate([vv.astype(np.float64), va.astype(np.float64)], axis=1)
    v_eff = oracle.cfg_combine(v64[0], v64[1], s)[None] if cfg else v64
    ref = oracle.euler_step(x0.astype(np.float64), v_eff, t, tn)
    assert rel_l2(host(vout), v_eff) < 1e-6
    assert rel_l2(host(x), ref) < 1e-6
    xg = host(x)
    for b in range(B):
        j = 0 if cfg else b
        assert np.array_equal(host(z[b]), bf16_round(xg[j, :nv]))
        assert np.array_equal(host(a[b]), bf16_round(xg[j, nv:]))
    # a cached velocity instead of the step outputs, then a pure re-quantization
    v_in = g.standard_normal((nx, nv + na)).astype(np.float32)
    x1 = host(x)
    w.wam_flow_step(dims, x, z, a, tn, 0.9, v_in=dev(v_in))
    torch.cuda.synchronize()
    assert rel_l2(host(x), oracle.euler_step(x1, v_in.astype(np.float64), tn, 0.9)) < 1e-6
    x2 = host(x)
    w.wam_flow_step(dims, x, z, a, 0.9, 1.0)
    torch.cuda.synchronize()
    assert np.array_equal(host(x), x2)
    assert np.array_equal(host(z[0]), bf16_round(x2[0, :nv]))


@pytest.mark.parametrize("n", [1, 1000, (1 << 20) + 3])
def test_cosine_similarity(n):
    import torch
    w = lib()
    g = np.random.default_rng(141 + n % 7)
    a = g.standard_normal(n).astype(np.float32)
    b = (0.3 * a + g.standard_normal(n)).astype(np.float32)
    ws = workspace(w.wam_cosine_workspace_bytes())
    out = torch.zeros(1, dtype=torch.float32, device="cuda")
    log(f"cosine n={n}")
    da, db = dev(a), dev(b)
    w.wam_cosine_similarity(da, db, out, ws)
    torch.cuda.synchronize()
    first = out.item()
    assert abs(first - oracle.cosine_similarity(a, b)) < 1e-6
    w.wam_cosine_similarity(da, db, out, ws)
    torch.cuda.synchronize()
    assert out.item() == first  # fixed reduction order
    w.wam_cosine_similarity(da, da, out, ws)
    torch.cuda.synchronize()
    assert abs(out.item() - 1.0) < 1e-6
    w.wam_cosine_similarity(da, -da, out, ws)
    torch.cuda.synchronize()
    assert abs(out.item() + 1.0) < 1e-6


# ------------------------------------------------------------------------------ the loop
class LoopCase(StepCase):
    """The d=512 network (cache of earlier chunks, batch of one chunk or a guidance pair)
    denoised over a schedule, on the GPU through wam_denoise_chunk and in the oracle
    through oracle.denoise with oracle.dit_step as the velocity."""

    def __init__(self, wl, n_layers, cfg_scale=None):
        super().__init__(wl, n_layers, bias_std=0.05)
        self.cfg = cfg_scale is not None
        self.scale = cfg_scale if self.cfg else 1.0
        B = wl.B
        self.nv = wl.latent_ch * wl.F * wl.Hl * wl.Wl
        self.na = wl.A * wl.act_dim
        nx = 1 if self.cfg else B
        g = np.random.default_rng(wl.seed + 150)
        self.x0 = g.standard_normal((nx, self.nv + self.na)).astype(np.float32)

    def velocity(self, x_in, t):
        wl, B = self.wl, self.wl.B
        xs = np.repeat(x_in, B, axis=0) if self.cfg else x_in
        z = xs[:, :self.nv].reshape(B, wl.latent_ch, wl.F, wl.Hl, wl.Wl)
        a = xs[:, self.nv:].reshape(B, wl.A, wl.act_dim)

        def layers(l):
            W, kc, vc = self.layer(l)
            return f64(W), (kc.f64 if kc is not None else None), (vc.f64 if vc is not None else None)

        vv, va = oracle.dit_step(z, a, np.full(B, t), self.text.f64, f64(self.P), layers, self.n_layers, wl.H,
                                 wl.eps, wl.n_cached, oracle_positions(wl),
                                 prev_chunk=prev_chunk_ids(wl) if wl.n_cached else None)
        v = np.concatenate([vv.reshape(B, -1), va.reshape(B, -1)], axis=1)
        return oracle.cfg_combine(v[0], v[1], self.scale)[None] if self.cfg else v

    def run_oracle_loop(self, ts, tau=None, window=0):
        return oracle.denoise(self.x0.astype(np.float64), self.velocity, ts, tau=tau, window=window,
                              to_model_input=bf16_round)

    def gpu_loop_setup(self, ts, tau=0.0, window=0):
        """Device buffers, step io, loop parameters and workspace of one loop call."""
        import torch
        w = lib()
        wl, B = self.wl, self.wl.B
        if not hasattr(self, "model"):
            self.upload()
        vv = torch.empty((B, wl.latent_ch, wl.F, wl.Hl, wl.Wl), dtype=torch.float32, device="cuda")
        va = torch.empty((B, wl.A, wl.act_dim), dtype=torch.float32, device="cuda")
        z = torch.empty((B, wl.latent_ch, wl.F, wl.Hl, wl.Wl), dtype=torch.bfloat16, device="cuda")
        a = torch.empty((B, wl.A, wl.act_dim), dtype=torch.bfloat16, device="cuda")
        t = torch.zeros(B, dtype=torch.float32, device="cuda")
        io = w.make_step_io(z, a, t, self.dtext, self.kcs, self.vcs, self.cos, self.sin, wl.cache_rows,
                            w.cached_chunks(wl.cache_rows, wl.L), vv, va)
        x = dev(self.x0)
        p = w.make_denoise_params(ts, x, cfg=self.cfg, cfg_scale=self.scale, cache_tau=tau, cache_window=window)
        ws = workspace(w.wam_denoise_workspace_bytes(self.model, io, p))
        return dict(io=io, p=p, x=x, ws=ws, keep=(vv, va, z, a, t))

    def run_gpu_loop(self, ts, tau=0.0, window=0):
        import torch
        s = self.gpu_loop_setup(ts, tau, window)
        lib().wam_denoise_chunk(self.model, s["io"], s["p"], s["ws"])
        torch.cuda.synchronize()
        return s["x"], [bool(c) for c in s["p"].computed_steps.cpu().tolist()]


def small_wl(**kw):
    base = dict(B=1, n_cached=1, n_layers=2, mod_std=0.3)
    base.update(kw)
    return synth.WORKLOADS["block_d512"].replace(**base)


def check_loop(case, ts, tau=None, window=0):
    log(f"denoise loop: GPU ({len(ts) - 1} steps, cfg={case.cfg}, window={window})")
    x, computed = case.run_gpu_loop(ts, tau=0.0 if tau is None else tau, window=window)
    log("denoise loop: oracle")
    ref, ref_computed = case.run_oracle_loop(ts, tau=tau, window=window)
    e = rel_l2(host(x), ref)
    print(f"  final state rel L2 {e:.2e}; computed {computed}", flush=True)
    assert computed == ref_computed
    assert e <= TOL


def test_denoise_loop_plain():
    case = LoopCase(small_wl(), 2)
    check_loop(case, [0.0, 0.3, 0.55, 0.8, 1.0])


def test_denoise_loop_guidance_pair():
    """Classifier-free guidance over a batch of two: sample 0 conditional, sample 1
    unconditional (different text and caches), one shared state."""
    case = LoopCase(small_wl(B=2), 2, cfg_scale=3.0)
    check_loop(case, [0.0, 0.4, 0.7, 1.0])


def test_denoise_loop_dit_caching():
    """A threshold every pair of successive velocities passes (-1), window 1: the pattern
    computed / reused alternates after the first two steps, on both sides."""
    case = LoopCase(small_wl(), 2)
    check_loop(case, list(np.linspace(0.0, 1.0, 7)), tau=-1.0, window=1)


def test_denoise_loop_graph_replay():
    """A whole loop call with DiT caching, captured once as a HIP graph (the reuse decision
    is taken on the device, so the call never waits for the host) and replayed three times
    with eager loop calls between the replays: every replay and every eager call gives the
    same final state and computed / reused pattern, bit for bit, and that result matches
    the oracle's loop."""
    graph_replay_check(LoopCase(small_wl(), 2), list(np.linspace(0.0, 1.0, 7)))


def graph_replay_check(case, ts):
    """Capture one loop call with caching (tau -1, window 1) as a HIP graph, replay it
    three times between eager calls, and check every result bitwise against the eager
    call and the eager call against the oracle."""
    import torch
    w = lib()
    s = case.gpu_loop_setup(ts, tau=-1.0, window=1)
    x0 = s["x"].clone()
    flags = s["p"].computed_steps

    def eager():
        s["x"].copy_(x0)
        flags.zero_()
        w.wam_denoise_chunk(case.model, s["io"], s["p"], s["ws"])
        torch.cuda.synchronize()
        return s["x"].clone(), flags.clone()

    log("denoise loop graph: eager call")
    x_ref, f_ref = eager()
    assert f_ref.cpu().tolist() == [1, 1, 0, 1, 0, 1]
    g = torch.cuda.CUDAGraph()
    s["x"].copy_(x0)
    torch.cuda.synchronize()
    log("denoise loop graph: capture")
    with torch.cuda.graph(g):
        w.wam_denoise_chunk(case.model, s["io"], s["p"], s["ws"])
    torch.cuda.synchronize()
    for r in range(3):
        s["x"].copy_(x0)
        flags.zero_()
        log(f"denoise loop graph: replay {r}")
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(s["x"], x_ref), f"replay {r}: state differs from the eager call"
        assert torch.equal(flags, f_ref), f"replay {r}: computed pattern differs"
        x_e, f_e = eager()
        assert torch.equal(x_e, x_ref) and torch.equal(f_e, f_ref)
    del g
    log("denoise loop graph: oracle")
    ref, ref_computed = case.run_oracle_loop(ts, tau=-1.0, window=1)
    assert [bool(c) for c in f_ref.cpu().tolist()] == ref_computed
    e = rel_l2(host(x_ref), ref)
    print(f"  final state rel L2 {e:.2e}", flush=True)
    assert e <= TOL
