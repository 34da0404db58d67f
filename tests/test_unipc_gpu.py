"""GPU parity of the UniPC solver (the paper's Flow-UniPC) against the fp64 oracle:
wam_unipc_step driven by seeded velocities over whole schedules (orders 1-3, plain and
guidance pair, step outputs and cached velocities), and wam_denoise_chunk with UniPC
driving the d=512 network (plain; guidance pair with DiT caching)."""
import numpy as np
import pytest

import oracle
from gpu_helpers import dev, host, log, rel_l2
from test_denoise_gpu import LoopCase, bf16_round, graph_replay_check, small_wl

pytestmark = pytest.mark.gpu
TOL_STEP = 1e-5   # fp32 kernel with fp32 weights against fp64 (weights rounded to 2^-24)
TOL_LOOP = 2e-2   # the bf16 network in the loop, as for the Euler loop


def lib():
    import paper_2602_15922_amd as w
    return w


@pytest.mark.parametrize("order", [1, 2, 3])
@pytest.mark.parametrize("cfg", [False, True])
def test_unipc_steps_match_oracle(order, cfg):
    import torch
    w = lib()
    g = np.random.default_rng(180 + order + 10 * cfg)
    B, nv, na = (2, 3077, 37) if cfg else (3, 1003, 16)
    nx, s = (1 if cfg else B), 2.5
    n = nv + na
    ts = [float(t) for t in np.float32([0.02, 0.1, 0.23, 0.41, 0.6, 0.78, 0.93, 1.0])]
    N = len(ts) - 1
    vv = g.standard_normal((N, B, nv)).astype(np.float32)
    va = g.standard_normal((N, B, na)).astype(np.float32)
    x0 = g.standard_normal((nx, n)).astype(np.float32)
    v64 = np.concatenate([vv.astype(np.float64), va.astype(np.float64)], axis=2)
    v_eff = [oracle.cfg_combine(v64[i, 0], v64[i, 1], s)[None] if cfg else v64[i] for i in range(N)]
    calls = []

    def velocity(x_in, t):
        calls.append(t)
        return v_eff[len(calls) - 1]

    states = []
    ref, _ = oracle.unipc_denoise(x0.astype(np.float64), velocity, ts, order=order, states=states)
    coef = w.wam_unipc_plan(ts, order)
    dims = w.binding.wam_flow_dims(B=B, cfg=int(cfg), cfg_scale=s, n_video=nv, n_action=na)
    x, x_last = dev(x0), torch.zeros((nx, n), dtype=torch.float32, device="cuda")
    ring = [torch.zeros((nx, n), dtype=torch.float32, device="cuda") for _ in range(4)]
    vout = torch.empty((nx, n), dtype=torch.float32, device="cuda")
    z = torch.empty((B, nv), dtype=torch.bfloat16, device="cuda")
    a = torch.empty((B, na), dtype=torch.bfloat16, device="cuda")
    log(f"unipc steps order={order} cfg={cfg}")
    for i in range(N):
        if not cfg and i % 2 == 1:   # a cached velocity instead of the step outputs
            w.wam_unipc_step(dims, None, None, dev(np.concatenate([vv[i], va[i]], axis=1)), x, x_last, ring, i,
                             coef[i], vout, z, a)
        else:
            w.wam_unipc_step(dims, dev(vv[i]), dev(va[i]), None, x, x_last, ring, i, coef[i], vout, z, a)
        torch.cuda.synchronize()
        assert rel_l2(host(vout), v_eff[i]) < 1e-6
        if i >= 1:
            e = rel_l2(host(x_last), states[i - 1])
            assert e < TOL_STEP, (i, e)
    xg = host(x)
    e = rel_l2(xg, ref)
    print(f"  final state rel L2 {e:.2e}", flush=True)
    assert e < TOL_STEP
    for b in range(B):
        j = 0 if cfg else b
        assert np.array_equal(host(z[b]), bf16_round(xg[j, :nv]))
        assert np.array_equal(host(a[b]), bf16_round(xg[j, nv:]))


def test_unipc_step_rejects_bad_arguments():
    import torch
    w = lib()
    b = w.binding
    ts = [0.1, 0.4, 0.7, 1.0]
    coef = w.wam_unipc_plan(ts, 2)
    dims = b.wam_flow_dims(B=1, cfg=0, cfg_scale=1.0, n_video=8, n_action=0)
    x = torch.zeros((1, 8), dtype=torch.float32, device="cuda")
    ring = [torch.zeros_like(x) for _ in range(4)]
    z = torch.empty((1, 8), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(w.WamError):   # step 0 cannot correct
        w.wam_unipc_step(dims, x, None, None, x, x.clone(), ring, 0, coef[1], None, z, None)
    with pytest.raises(w.WamError):   # the history slot step 2 reads is missing
        w.wam_unipc_step(dims, x, None, None, x, x.clone(), ring[:1] + [None] + ring[2:], 2, coef[2], None, z, None)
    with pytest.raises(w.WamError):   # no velocity at all
        w.wam_unipc_step(dims, None, None, None, x, x.clone(), ring, 0, coef[0], None, z, None)
    torch.cuda.synchronize()
    assert np.array_equal(host(x), np.zeros((1, 8), np.float32))


class UnipcLoopCase(LoopCase):
    def run_oracle_loop(self, ts, tau=None, window=0):
        return oracle.unipc_denoise(self.x0.astype(np.float64), self.velocity, ts, order=self.order, tau=tau,
                                    window=window, to_model_input=bf16_round)

    def gpu_loop_setup(self, ts, tau=0.0, window=0):
        s = super().gpu_loop_setup(ts, tau, window)
        s["p"].solver = lib().binding.WAM_SOLVER_UNIPC
        s["p"].solver_order = self.order
        from gpu_helpers import workspace
        s["ws"] = workspace(lib().wam_denoise_workspace_bytes(self.model, s["io"], s["p"]))
        return s


def check_unipc_loop(case, ts, tau=None, window=0):
    log(f"unipc loop: GPU ({len(ts) - 1} steps, order {case.order}, cfg={case.cfg}, window={window})")
    x, computed = case.run_gpu_loop(ts, tau=0.0 if tau is None else tau, window=window)
    log("unipc loop: oracle")
    ref, ref_computed = case.run_oracle_loop(ts, tau=tau, window=window)
    e = rel_l2(host(x), ref)
    print(f"  final state rel L2 {e:.2e}; computed {computed}", flush=True)
    assert computed == ref_computed
    assert e <= TOL_LOOP


def test_denoise_loop_unipc():
    case = UnipcLoopCase(small_wl(), 2)
    case.order = 2
    check_unipc_loop(case, [0.05, 0.3, 0.55, 0.8, 1.0])


def test_denoise_loop_unipc_guidance_and_caching():
    """Order 3 over a guidance pair with DiT caching (every pair of successive velocities
    passes tau = -1, window 1): reused velocities enter the solver like computed ones."""
    case = UnipcLoopCase(small_wl(B=2), 2, cfg_scale=3.0)
    case.order = 3
    check_unipc_loop(case, [float(t) for t in np.float32(np.linspace(0.04, 1.0, 7))], tau=-1.0, window=1)


def test_denoise_loop_unipc_graph_replay():
    """A UniPC loop call with DiT caching captured as a HIP graph: the history buffers are
    written before they are read in every call, so each replay equals the eager call bit
    for bit (and the eager call matches the oracle)."""
    case = UnipcLoopCase(small_wl(), 2)
    case.order = 2
    graph_replay_check(case, [float(t) for t in np.float32(np.linspace(0.05, 1.0, 7))])
