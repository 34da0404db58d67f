"""The denoising loop of one chunk, float64: flow-matching solver step, classifier-free
guidance and DiT caching (Appendix C, Algorithm 2; section 3.2 and Appendix D.1).

The noisy sample moves along the straight path of Eq. 2, x_t = t x_1 + (1 - t) x_0,
from t = 0 (pure noise) to t = 1 (clean), whose velocity dx/dt = x_1 - x_0 is what the
network predicts (Eq. 3).  Readings where the paper is silent or ambiguous:

* the solver is the explicit Euler step of that ODE, x <- x + (t_next - t) v (the paper
  names Flow-UniPC for its deployment but gives no formula);
* guidance combines the conditional and unconditional velocities as
  v = v_u + s (v_c - v_u) (the classifier-free guidance rule the paper cites);
* DiT caching compares the two most recent computed velocities (the listing's
  CosSim(v_prev, v_last)); when their cosine similarity exceeds tau, the next `window`
  steps reuse the latest computed velocity instead of calling the network;
* the network consumes bf16 inputs, so the state is rounded to bf16 before each call
  (`to_model_input`), while the state itself is carried at full precision.
"""
import numpy as np


def euler_step(x, v, t, t_next):
    """One explicit Euler step of dx/dt = v from t to t_next."""
    return x + (t_next - t) * v


def cfg_combine(v_cond, v_uncond, scale):
    """Classifier-free guidance: v_u + s (v_c - v_u)."""
    return v_uncond + scale * (v_cond - v_uncond)


def cosine_similarity(a, b):
    """<a, b> / (|a| |b|) over all elements (0 when either vector is zero)."""
    a = np.asarray(a, dtype=np.float64).ravel()
    b = np.asarray(b, dtype=np.float64).ravel()
    den = np.linalg.norm(a) * np.linalg.norm(b)
    return float(a @ b / den) if den > 0 else 0.0


def denoise(x0, velocity, t_sched, tau=None, window=1, to_model_input=None):
    """Algorithm 2's denoising loop for one chunk.

    x0: initial noise (any array); velocity(x_in, t) -> v, the network's (already
    guidance-combined) velocity at model input x_in and time t; t_sched: the N+1
    scheduler times t_0 .. t_N; tau None (or window 0) turns DiT caching off.  Returns
    (x_N, computed) with computed[i] True where step i called the network."""
    x = np.array(x0, dtype=np.float64)
    v_last = None     # most recent computed velocity
    v_before = None   # the computed velocity before it
    skip = 0
    computed = []
    for i in range(len(t_sched) - 1):
        t, t_next = float(t_sched[i]), float(t_sched[i + 1])
        if skip > 0:
            v = v_last
            skip -= 1
            computed.append(False)
        else:
            x_in = to_model_input(x) if to_model_input is not None else x
            v = np.asarray(velocity(x_in, t), dtype=np.float64)
            v_before, v_last = v_last, v
            computed.append(True)
            if tau is not None and window > 0 and v_before is not None and \
                    cosine_similarity(v_last, v_before) > tau:
                skip = window
        x = euler_step(x, v, t, t_next)
    return x, computed
