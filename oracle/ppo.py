"""Policy/value heads, PPO loss and its gradient, in fp64.

Test infrastructure (see the package docstring).

What the paper fixes:
* the policy outputs and the value function are linear projections of the
  LSTM state, and policy and value share the network and its gradients
  (appendix "Neural Network Architecture");
* the action is factorised into a primary action and parameter actions, one
  categorical distribution per head; heads that the primary action ignores
  are masked out of the optimisation, and at each timestep action filters
  restrict the choice to the available actions (appendix "Action Space");
* PPO clipped surrogate with clip 0.2, value loss weight 1.0 (Table
  "Hyperparameters"); entropy bonus c * S[pi](s_t) with c = 0.01 (appendix
  "Exploration", subsection "Loss function").

Readings where the paper is silent: one joint probability ratio over the
factorised action (per-head log-probabilities summed under the head mask);
no advantage normalisation; value loss (V - R)^2 without a 1/2 factor and
without clipping; natural-log entropy; means over the N timesteps; the
gradient of the surrogate flows when (A >= 0 and r <= 1+eps) or
(A < 0 and r >= 1-eps), inclusive at the kinks.  Availability: an
unavailable logit is left out of its head's softmax (its probability is 0,
it carries no gradient and it does not enter the entropy); a head with no
available logit in a row contributes log-probability 0, entropy 0 and no
gradient; a taken action that is unavailable has log-probability -inf.  A
head whose mask is 0 contributes nothing whatever its log-probability.

Shapes: h [N, H]; Wp [A+1, H] with the last row the value head; bp [A+1];
act [N, K] (integer index within each head); logp_old, adv, ret [N];
head_mask [N, K] or None (all ones); avail [N, A] (1 = available) or None
(all available).

Unit-selection head (appendix "Neural Network Architecture": the unit
embeddings from the observation processing are carried beside the LSTM and
used by the action heads to choose a unit to target).  Optionally head k
scores its n_k units against per-row embeddings E [N, n_k, d]: a query
q = h Wq^T + bq [N, d], logits z_k[n, u] = <q[n], E[n, u]>.  Reading: the
query is a linear projection of the LSTM state, the score a plain dot
product; the rows of Wp and bp that belong to head k are then unused (zero
gradient).  The gradient reaches Wq, bq and h through q; none is taken into
E (the observation encoder that would produce E is not modelled).
"""
import numpy as np

from .precision import F

STAT_NAMES = ("total", "pg", "vf", "ent", "clipfrac", "approx_kl",
              "mean_ratio", "nonfinite")


def head_offsets(head_sizes):
    off = [0]
    for n in head_sizes:
        off.append(off[-1] + int(n))
    return off


def heads_forward(h, Wp, bp):
    """Logits and value: z = h Wp^T + bp, an [N, A+1] array."""
    return np.asarray(h, F()) @ np.asarray(Wp, F()).T + \
        np.asarray(bp, F())


def head_logprob_entropy(z, act, head_sizes, avail=None):
    """Per-head log-probability of the taken action, entropy and softmax,
    each head's softmax taken over its available logits only.

    Returns (logp [N,K], ent [N,K], probs list of [N, n_k]).
    """
    N = z.shape[0]
    off = head_offsets(head_sizes)
    K = len(head_sizes)
    av_all = np.ones((N, off[-1]), bool) if avail is None else np.asarray(avail) != 0
    logp = np.empty((N, K), F())
    ent = np.empty((N, K), F())
    probs = []
    rows = np.arange(N)
    for k in range(K):
        zk = z[:, off[k]:off[k + 1]]
        av = av_all[:, off[k]:off[k + 1]]
        some = av.any(axis=1)
        zmax = np.where(av, zk, -np.inf).max(axis=1, keepdims=True)
        zmax = np.where(some[:, None], zmax, 0.0)
        e = np.where(av, np.exp(zk - zmax), 0.0)
        se = e.sum(axis=1, keepdims=True)
        lse = np.where(some, (zmax + np.log(np.where(some[:, None], se, 1.0)))[:, 0], 0.0)
        p = np.where(some[:, None], e / np.where(some[:, None], se, 1.0), 0.0)
        taken = av[rows, act[:, k]]
        logp[:, k] = np.where(some, np.where(taken, zk[rows, act[:, k]] - lse, -np.inf), 0.0)
        ent[:, k] = np.where(some, lse - (p * np.where(av, zk, 0.0)).sum(axis=1), 0.0)
        probs.append(p)
    return logp, ent, probs


def unit_logits(h, Wq, bq, E):
    """Query q = h Wq^T + bq and logits z[n, u] = <q[n], E[n, u]>."""
    q = np.asarray(h, F()) @ np.asarray(Wq, F()).T + np.asarray(bq, F())
    return q, np.einsum("nj,nuj->nu", q, np.asarray(E, F()))


def ppo_loss_grad(h, Wp, bp, act, logp_old, adv, ret, head_sizes,
                  clip_eps=0.2, vf_coef=1.0, ent_coef=0.01, head_mask=None,
                  avail=None, unit=None):
    """Loss statistics and gradients with respect to h, Wp and bp.

    Returns (stats dict, dh [N,H], dWp [A+1,H], dbp [A+1], z [N,A+1]); with
    ``unit`` = dict(head=k, Wq=[d,H], bq=[d], E=[N,n_k,d]) also
    (dWq [d,H], dbq [d]) as a sixth element.
    """
    h = np.asarray(h, F())
    Wp = np.asarray(Wp, F())
    act = np.asarray(act, np.int64)
    logp_old = np.asarray(logp_old, F())
    A_ = np.asarray(adv, F())
    R_ = np.asarray(ret, F())
    N = h.shape[0]
    K = len(head_sizes)
    off = head_offsets(head_sizes)
    A = off[-1]
    mask = np.ones((N, K), F()) if head_mask is None else \
        np.asarray(head_mask, F())

    z = heads_forward(h, Wp, bp)
    if unit is not None:
        ku = unit["head"]
        _, z[:, off[ku]:off[ku + 1]] = unit_logits(h, unit["Wq"], unit["bq"], unit["E"])
    V = z[:, A]
    logp, ent_k, probs = head_logprob_entropy(z, act, head_sizes, avail)
    on = mask != 0
    logpi = np.where(on, logp, 0.0).sum(axis=1)
    ratio = np.exp(logpi - logp_old)
    clipped = np.clip(ratio, 1.0 - clip_eps, 1.0 + clip_eps)
    surr = np.minimum(ratio * A_, clipped * A_)
    ent = np.where(on, ent_k, 0.0).sum(axis=1)
    verr = V - R_

    pg = -surr.mean()
    vf = (verr ** 2).mean()
    entm = ent.mean()
    total = pg + vf_coef * vf - ent_coef * entm
    row_loss = -surr + vf_coef * verr ** 2 - ent_coef * ent
    stats = {
        "total": total,
        "pg": pg,
        "vf": vf,
        "ent": entm,
        "clipfrac": (np.abs(ratio - 1.0) > clip_eps).mean(),
        "approx_kl": ((ratio - 1.0) - (logpi - logp_old)).mean(),
        "mean_ratio": ratio.mean(),
        "nonfinite": float((~np.isfinite(row_loss)).sum()),
    }

    # d(loss)/d(logits)
    flow = ((A_ >= 0) & (ratio <= 1.0 + clip_eps)) | \
        ((A_ < 0) & (ratio >= 1.0 - clip_eps))
    g_logpi = -np.where(flow, ratio * A_, 0.0) / N          # dL_pg / d logpi
    dz = np.zeros_like(z)
    rows = np.arange(N)
    av_all = np.ones((N, A), bool) if avail is None else np.asarray(avail) != 0
    for k in range(K):
        zk = z[:, off[k]:off[k + 1]]
        av = av_all[:, off[k]:off[k + 1]]
        p = probs[k]
        onehot = np.zeros_like(p)
        onehot[rows, act[:, k]] = 1.0
        onehot *= av                                           # an unavailable taken action has no gradient
        use = (on[:, k] & av.any(axis=1))[:, None]
        dpg = g_logpi[:, None] * (onehot - p)
        zbar = (p * np.where(av, zk, 0.0)).sum(axis=1, keepdims=True)
        dent = -p * np.where(av, zk - zbar, 0.0)               # dS_k / dz_k
        dz[:, off[k]:off[k + 1]] = np.where(use & av, dpg - (ent_coef / N) * dent, 0.0)
    dz[:, A] = 2.0 * vf_coef * verr / N

    if unit is None:
        dh = dz @ Wp
        dWp = dz.T @ h
        dbp = dz.sum(axis=0)
        return stats, dh, dWp, dbp, z
    # head k's logits come from the query: its gradient goes to q, not to Wp
    ku = unit["head"]
    dz_u = dz[:, off[ku]:off[ku + 1]].copy()
    dz[:, off[ku]:off[ku + 1]] = 0.0
    Wq = np.asarray(unit["Wq"], F())
    dq = np.einsum("nu,nuj->nj", dz_u, np.asarray(unit["E"], F()))
    dh = dz @ Wp + dq @ Wq
    dWp = dz.T @ h
    dbp = dz.sum(axis=0)
    return stats, dh, dWp, dbp, z, (dq.T @ h, dq.sum(axis=0))
