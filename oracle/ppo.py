"""Policy/value heads, PPO loss and its gradient, in fp64.

Test infrastructure (see the package docstring).

What the paper fixes:
* the policy outputs and the value function are linear projections of the
  LSTM state, and policy and value share the network and its gradients
  (appendix "Neural Network Architecture");
* the action is factorised into a primary action and parameter actions, one
  categorical distribution per head; heads that the primary action ignores
  are masked out of the optimisation (appendix "Action Space");
* PPO clipped surrogate with clip 0.2, value loss weight 1.0 (Table
  "Hyperparameters"); entropy bonus c * S[pi](s_t) with c = 0.01 (appendix
  "Exploration", subsection "Loss function").

Readings where the paper is silent: one joint probability ratio over the
factorised action (per-head log-probabilities summed under the head mask);
no advantage normalisation; value loss (V - R)^2 without a 1/2 factor and
without clipping; natural-log entropy; means over the N timesteps; the
gradient of the surrogate flows when (A >= 0 and r <= 1+eps) or
(A < 0 and r >= 1-eps), inclusive at the kinks.

Shapes: h [N, H]; Wp [A+1, H] with the last row the value head; bp [A+1];
act [N, K] (integer index within each head); logp_old, adv, ret [N];
head_mask [N, K] or None (all ones).
"""
import numpy as np

STAT_NAMES = ("total", "pg", "vf", "ent", "clipfrac", "approx_kl",
              "mean_ratio", "nonfinite")


def head_offsets(head_sizes):
    off = [0]
    for n in head_sizes:
        off.append(off[-1] + int(n))
    return off


def heads_forward(h, Wp, bp):
    """Logits and value: z = h Wp^T + bp, an [N, A+1] array."""
    return np.asarray(h, np.float64) @ np.asarray(Wp, np.float64).T + \
        np.asarray(bp, np.float64)


def head_logprob_entropy(z, act, head_sizes):
    """Per-head log-probability of the taken action, entropy and softmax.

    Returns (logp [N,K], ent [N,K], probs list of [N, n_k]).
    """
    N = z.shape[0]
    off = head_offsets(head_sizes)
    K = len(head_sizes)
    logp = np.empty((N, K))
    ent = np.empty((N, K))
    probs = []
    rows = np.arange(N)
    for k in range(K):
        zk = z[:, off[k]:off[k + 1]]
        zmax = zk.max(axis=1, keepdims=True)
        lse = (zmax + np.log(np.exp(zk - zmax).sum(axis=1, keepdims=True)))[:, 0]
        p = np.exp(zk - lse[:, None])
        logp[:, k] = zk[rows, act[:, k]] - lse
        ent[:, k] = lse - (p * zk).sum(axis=1)
        probs.append(p)
    return logp, ent, probs


def ppo_loss_grad(h, Wp, bp, act, logp_old, adv, ret, head_sizes,
                  clip_eps=0.2, vf_coef=1.0, ent_coef=0.01, head_mask=None):
    """Loss statistics and gradients with respect to h, Wp and bp.

    Returns (stats dict, dh [N,H], dWp [A+1,H], dbp [A+1], z [N,A+1]).
    """
    h = np.asarray(h, np.float64)
    Wp = np.asarray(Wp, np.float64)
    act = np.asarray(act, np.int64)
    logp_old = np.asarray(logp_old, np.float64)
    A_ = np.asarray(adv, np.float64)
    R_ = np.asarray(ret, np.float64)
    N = h.shape[0]
    K = len(head_sizes)
    off = head_offsets(head_sizes)
    A = off[-1]
    mask = np.ones((N, K)) if head_mask is None else \
        np.asarray(head_mask, np.float64)

    z = heads_forward(h, Wp, bp)
    V = z[:, A]
    logp, ent_k, probs = head_logprob_entropy(z, act, head_sizes)
    logpi = (mask * logp).sum(axis=1)
    ratio = np.exp(logpi - logp_old)
    clipped = np.clip(ratio, 1.0 - clip_eps, 1.0 + clip_eps)
    surr = np.minimum(ratio * A_, clipped * A_)
    ent = (mask * ent_k).sum(axis=1)
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
    for k in range(K):
        zk = z[:, off[k]:off[k + 1]]
        p = probs[k]
        onehot = np.zeros_like(p)
        onehot[rows, act[:, k]] = 1.0
        dpg = (g_logpi * mask[:, k])[:, None] * (onehot - p)
        zbar = (p * zk).sum(axis=1, keepdims=True)
        dent = -p * (zk - zbar)                                # dS_k / dz_k
        dz[:, off[k]:off[k + 1]] = dpg - (ent_coef / N) * mask[:, k:k + 1] * dent
    dz[:, A] = 2.0 * vf_coef * verr / N

    dh = dz @ Wp
    dWp = dz.T @ h
    dbp = dz.sum(axis=0)
    return stats, dh, dWp, dbp, z
