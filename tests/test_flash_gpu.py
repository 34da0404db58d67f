"""GPU parity of the DreamZero-Flash step (Appendix D.3: video and action tokens at their
own timesteps) against the fp64 oracle (relative L2 <= 2e-2 on both velocities), and the
reduction to the plain step when both timesteps are equal (bitwise)."""
import numpy as np
import pytest

import synth
from dit_cases import StepCase
from gpu_helpers import host, log, rel_l2

pytestmark = pytest.mark.gpu
TOL = 2e-2


def check(case, vv, va):
    rv, ra = case.run_oracle()
    ev, ea = rel_l2(host(vv), rv), rel_l2(host(va), ra)
    print(f"  flash step rel L2 video {ev:.2e} action {ea:.2e}", flush=True)
    assert ev <= TOL and ea <= TOL


def test_flash_step_small():
    wl = synth.WORKLOADS["block_d512"].replace(B=2, n_cached=2, n_layers=3, mod_std=0.3)
    log("flash step small")
    case = StepCase(wl, 3, bias_std=0.05, flash=True)
    vv, va = case.run_gpu()
    check(case, vv, va)


def test_flash_equal_timesteps_match_plain_step_bitwise():
    wl = synth.WORKLOADS["block_d512"].replace(B=2, n_cached=1, n_layers=2, mod_std=0.3)
    log("flash step equal timesteps")
    case = StepCase(wl, 2, bias_std=0.05)
    v0, a0 = case.run_gpu()
    v1, a1 = case.run_gpu(t_action=case.dt.clone())
    assert np.array_equal(host(v0), host(v1)) and np.array_equal(host(a0), host(a1))


def test_flash_step_14b_shapes_one_block():
    wl = synth.WORKLOADS["step_14b"].replace(n_layers=1)
    log("flash step 14b depth 1: inputs + GPU")
    case = StepCase(wl, 1, flash=True)
    vv, va = case.run_gpu()
    log("flash step 14b depth 1: oracle")
    check(case, vv, va)
