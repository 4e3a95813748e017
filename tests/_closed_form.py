"""Token states that the heavy-hitter recipe implies, in closed form.

Under the 'hh' recipe every relevance score stays provably on one side of tau
(``synth.gen.hh_relevance_bounds``): a cold token is flagged at every step it
attends once it has left the window of the K most recent positions, a hot
token never.  Without recovery every cold token therefore follows the
oracle's own single-token trajectory (Eq. 3 and Algorithm 1), shifted to the
step it leaves the window, and the states of any (layer, sequence) at any step
follow from that trajectory and the hot mask alone.  The CPU test
``test_stress_closed_form_cpu`` checks this against the fully stepped oracle.
"""
import math

import numpy as np

import oracle


def base_trajectory(k_soft, T):
    """(count, frozen, remaining timer) after each of T steps of a token that is
    a freeze candidate from step 1 and flagged whenever it attends: position 0
    of an oracle instance with tau = +inf and no window (1 x 1 rows)."""
    z = np.zeros((1, 1, 1))
    inst = oracle.Instance(z, z, 0, math.inf, k_soft, capacity=T + 2)
    c = np.zeros(T + 1, np.int64)
    f = np.zeros(T + 1, bool)
    r = np.zeros(T + 1, np.int64)
    q = np.zeros((1, 1))
    for t in range(1, T + 1):
        inst.step(q, q, q)
        timer, count, frozen = inst.state()
        c[t], f[t], r[t] = count[0], frozen[0], timer[0]
    return c, f, r


class ClosedForm:
    """Token states implied by the heavy-hitter recipe without recovery."""

    def __init__(self, w, hot, base, seq=0):
        self.w, self.hot = w, hot
        self.c, self.f, self.r = base
        self.P, self.K = w.prefill[seq], w.window_K

    def state(self, t):
        """(count, frozen, remaining timer) of positions 0..n_t-1 after step t."""
        n = self.P + t
        p = np.arange(n)
        t0 = np.maximum(1, p - self.P + self.K + 1)          # first step outside the window
        tau = np.where(self.hot[:n], 0, np.maximum(0, t - t0 + 1))
        return self.c[tau], self.f[tau], np.where(self.f[tau], self.r[tau], 0)

    def active(self, t):
        """Positions attended at step t (after step t - 1), the new token last."""
        if t == 1:
            return np.arange(self.P + 1)
        _, fz, _ = self.state(t - 1)
        return np.concatenate([np.nonzero(~fz)[0], [self.P + t - 1]])
