"""Generalized advantage estimation over rollout segments, in fp64.

Test infrastructure (see the package docstring).

The paper trains with PPO using GAE, lambda = 0.95, with advantages smoothed
over 256-timestep segments (subsection "Optimizing the Policy"; Table
"Hyperparameters").  The GAE recursion itself is the standard one of
Schulman et al. (2016), which the paper cites:

    delta_t = r_t + gamma * (1 - done_t) * V_{t+1} - V_t
    A_t     = delta_t + gamma * lambda * (1 - done_t) * A_{t+1}
    R_t     = A_t + V_t                      (the value-function target)

Readings where the paper is silent: ``done[t] = 1`` marks transition t as
terminal (no bootstrap from V_{t+1} and no carry of A_{t+1}); the final step
of a segment bootstraps from ``v[L]``, the value of the state after the
segment.

Layout is time-major: r, done [L, S]; v [L+1, S] with row L the bootstrap.
"""
import numpy as np

from .precision import F


def gae(r, v, done, gamma, lam):
    """Sequential reverse loop over t = L-1 .. 0.  Returns (adv, ret) [L, S]."""
    r = np.asarray(r, F())
    v = np.asarray(v, F())
    nd = 1.0 - np.asarray(done, F())
    L, S = r.shape
    adv = np.zeros((L, S), F())
    carry = np.zeros(S, F())
    for t in reversed(range(L)):
        delta = r[t] + gamma * nd[t] * v[t + 1] - v[t]
        carry = delta + gamma * lam * nd[t] * carry
        adv[t] = carry
    ret = adv + v[:L]
    return adv, ret


def segments_to_samples(adv, ret, done, T):
    """Cut each length-L segment into L/T samples of T steps.

    Sample b = s * (L/T) + j holds segment steps T*j .. T*j + T - 1 of
    segment s.  Returns (adv_s, ret_s [T, B], reset [T, B] uint8) where
    reset[t, b] = done at the previous step of the same sample (reset[0] = 0:
    the stored rollout state at a sample's start already accounts for it).
    """
    L, S = adv.shape
    J = L // T
    adv_s = np.empty((T, S * J), F())
    ret_s = np.empty((T, S * J), F())
    reset = np.zeros((T, S * J), dtype=np.uint8)
    for s in range(S):
        for j in range(J):
            bidx = s * J + j
            for t in range(T):
                l = T * j + t
                adv_s[t, bidx] = adv[l, s]
                ret_s[t, bidx] = ret[l, s]
                if t > 0:
                    reset[t, bidx] = done[l - 1, s]
    return adv_s, ret_s, reset
