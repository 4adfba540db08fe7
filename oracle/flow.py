"""Flow-matching action head over a cached context, with latent warm start (reference).

TEST INFRASTRUCTURE ONLY: imported by the tests, never by the product package.

What it computes
----------------
Paper section 3.2.1 lists, among the cached intermediate states, the latent
vectors a diffusion model produces for the actions; section 3.4.2 ("Action
Regeneration") starts the action generation from a previously successful
action vector instead of a random one, which amounts to running further
denoising steps on the existing context.  The paper defines no model; the
readings taken here:

* an action chunk is a latent x of T action tokens with `a` values each;
* the velocity v(x, tau) runs every decoder layer over the T tokens
  e_i = W_in x_i + tau w_t, placed at positions len .. len+T-1 after the row's
  cached sequence (causal attention over the cache and the earlier action
  tokens; their K/V are not kept), then v_i = W_out (h_i / rms(h_i)) with the
  RMSNorm of the model's epsilon and no gain;
* sampling is Euler integration from tau0 to 1 in K equal steps,
  x <- x + dt v(x, tau0 + k dt), dt = (1 - tau0) / K: a cold start draws x at
  tau0 = 0, a warm start takes a stored latent and a later tau0.

Every computation is fp64 NumPy on top of ``decoder.forward``.
"""
from __future__ import annotations

import numpy as np

from . import decoder as D


class FlowHead:
    """w_in [d, a], w_t [d], w_out [a, d] (any float arrays, used in fp64)."""

    def __init__(self, w_in, w_t, w_out):
        self.w_in = np.asarray(w_in, dtype=np.float64)
        self.w_t = np.asarray(w_t, dtype=np.float64)
        self.w_out = np.asarray(w_out, dtype=np.float64)


def velocity(p: D.Params, fh: FlowHead, past, start: int, x: np.ndarray, tau: float) -> np.ndarray:
    """v(x, tau) for one row whose cached K/V (``past``) covers positions 0..start-1."""
    e = np.asarray(x, dtype=np.float64) @ fh.w_in.T + tau * fh.w_t
    h, _ = D.forward(p, e, start=start, past=past)
    u = h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + p.cfg.rms_eps)
    return u @ fh.w_out.T


def sample(p: D.Params, fh: FlowHead, seq: np.ndarray, x0: np.ndarray, tau0: float, n_steps: int) -> np.ndarray:
    """Euler integration of the velocity from tau0 to 1 in n_steps steps over the row's
    sequence ``seq`` (its cached context)."""
    x = np.asarray(x0, dtype=np.float64).copy()
    if n_steps <= 0:
        return x
    _, kv = D.forward(p, np.asarray(seq, dtype=np.float64))
    dt = (1.0 - tau0) / n_steps
    for k in range(n_steps):
        x = x + dt * velocity(p, fh, kv, seq.shape[0], x, tau0 + k * dt)
    return x
