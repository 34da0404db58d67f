"""The denoising loop of one chunk, float64: flow-matching solver step, classifier-free
guidance and DiT caching (Appendix C, Algorithm 2; section 3.2 and Appendix D.1).

The noisy sample moves along the straight path of Eq. 2, x_t = t x_1 + (1 - t) x_0,
from t = 0 (pure noise) to t = 1 (clean), whose velocity dx/dt = x_1 - x_0 is what the
network predicts (Eq. 3).  Readings where the paper is silent or ambiguous:

* the default solver is the explicit Euler step of that ODE, x <- x + (t_next - t) v;
  the paper names Flow-UniPC for its deployment without giving its formulas, so the
  second solver here (`unipc_denoise`) is UniPC (Zhao et al., 2023: a multistep
  predictor UniP-p and the corrector UniC, in its data-prediction form with
  B(h) = e^h - 1) on this path, with alpha_t = t and sigma_t = 1 - t;
* guidance combines the conditional and unconditional velocities as
  v = v_u + s (v_c - v_u) (the classifier-free guidance rule the paper cites);
* DiT caching compares the two most recent computed velocities (the listing's
  CosSim(v_prev, v_last)); when their cosine similarity exceeds tau, the next `window`
  steps reuse the latest computed velocity instead of calling the network;
* the network consumes bf16 inputs, so the state is rounded to bf16 before each call
  (`to_model_input`), while the state itself is carried at full precision.
"""
import math

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


# ----------------------------------------------------------------------------------
# UniPC on the straight path (alpha_t = t, sigma_t = 1 - t).
#
# With the data prediction m = x + (1 - t) v (the clean sample the velocity points at)
# and lambda = log(alpha / sigma), the ODE dx/dt = v has the exact solution
#     x_t = (sigma_t / sigma_s) x_s + sigma_t * integral_{lambda_s}^{lambda_t} e^lambda m d lambda.
# Expanding m around lambda_s and integrating term by term gives
#     x_t = (sigma_t / sigma_s) x_s + alpha_t sum_k m^(k)(lambda_s) I_k(h),
#     I_k(h) = e^-h integral_0^h e^u u^k / k! du,  I_0 = 1 - e^-h,  I_k = h^k / k! - I_(k-1),
# with h = lambda_t - lambda_s.  UniPC replaces the derivatives by divided differences
# D_j = (m_j - m_s) / r_j of data predictions at lambda_s + r_j h and weights a_j chosen
# so that the update is exact for every m of degree <= K in lambda:
#     x_t = (sigma_t / sigma_s) x_s + alpha_t I_0 (m_s + sum_j a_j D_j),
#     sum_j a_j r_j^(k-1) = k! I_k / (h^k I_0),  k = 1 .. K,
# i.e. UniPC's linear system R_p(h) a_p = phi_p(h) / B(h) with B(h) = e^h - 1 written in
# the data-prediction variable.  The predictor UniP-p uses the p - 1 previous data
# predictions; the corrector UniC refits the step just taken once the network has been
# called at its result, adding that new prediction at r = 1 (one order higher, no
# extra network call).
# ----------------------------------------------------------------------------------

def unipc_lambda(t):
    """lambda = log(alpha_t / sigma_t) = log(t / (1 - t))."""
    return math.log(t) - math.log1p(-t)


def unipc_update(x_s, t_s, t, m_s, points=()):
    """One UniPC update from time t_s (state x_s, data prediction m_s) to t.  points:
    (t_j, m_j) pairs of other data predictions, each giving one divided difference (the
    corrector passes the new prediction at t itself).  Exact whenever m is a polynomial
    of degree <= len(points) in lambda."""
    a_s, s_s = t_s, 1.0 - t_s
    a_t, s_t = t, 1.0 - t
    e = (a_s * s_t) / (s_s * a_t)          # e^-h, 0 when t = 1
    i0 = 1.0 - e
    out = (s_t / s_s) * np.asarray(x_s, dtype=np.float64) + a_t * i0 * np.asarray(m_s, dtype=np.float64)
    if not points:
        return out
    h = unipc_lambda(t) - unipc_lambda(t_s)
    K = len(points)
    ik = [i0]
    for k in range(1, K + 1):
        ik.append(h ** k / math.factorial(k) - ik[-1])
    rhs = np.array([math.factorial(k) * ik[k] / (h ** k * i0) for k in range(1, K + 1)])
    r = np.array([(unipc_lambda(tj) - unipc_lambda(t_s)) / h for tj, _ in points])
    R = np.array([[rj ** (k - 1) for rj in r] for k in range(1, K + 1)])
    a = np.linalg.solve(R, rhs)
    corr = sum(a[j] * (np.asarray(points[j][1], dtype=np.float64) - m_s) / r[j] for j in range(K))
    return out + a_t * i0 * corr


def unipc_denoise(x0, velocity, t_sched, order=2, tau=None, window=1, to_model_input=None,
                  corrector=True, states=None):
    """The denoising loop of `denoise` with UniPC of the given order (1..3) in place of
    Euler.  Readings: the schedule must satisfy 0 < t_0 < ... < t_N <= 1 (lambda finite
    wherever a step starts); the predictor's order warms up as min(order, i + 1), and a
    step that ends at t = 1 is order 1 (lambda is infinite there: the step returns its
    data prediction); the corrector
    runs at every step after the first, with the order of the predictor that produced
    the state it corrects; a step that reuses a velocity (DiT caching) treats it as the
    network's output at the current state.  states (a list) receives the corrected state
    of every step after the first.  Returns (x_N, computed)."""
    t_sched = [float(t) for t in t_sched]
    n = len(t_sched) - 1
    if not 1 <= order <= 3:
        raise ValueError("order must be 1, 2 or 3")
    if not (0.0 < t_sched[0] and all(a < b for a, b in zip(t_sched, t_sched[1:])) and t_sched[-1] <= 1.0):
        raise ValueError("UniPC needs 0 < t_0 < t_1 < ... < t_N <= 1")
    x = np.array(x0, dtype=np.float64)   # the state the network is called at
    x_prev = None                        # corrected state at the previous time
    hist = []                            # (t_j, m_j), newest last
    p_prev = 0
    v_last = v_before = None
    skip = 0
    computed = []
    for i in range(n):
        t, t_next = t_sched[i], t_sched[i + 1]
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
        m = x + (1.0 - t) * v
        if i > 0 and corrector:
            t_s, m_s = hist[-1]
            older = hist[-p_prev:-1] if p_prev > 1 else []
            x = unipc_update(x_prev, t_s, t, m_s, list(reversed(older)) + [(t, m)])
            if states is not None:
                states.append(x.copy())
        hist.append((t, m))
        x_prev = x
        p = 1 if t_next == 1.0 else min(order, i + 1)
        older = hist[-p:-1] if p > 1 else []
        x = unipc_update(x, t, t_next, m, list(reversed(older)))
        p_prev = p
    return x, computed
