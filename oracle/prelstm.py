"""The LSTM's input side, in fp64: observation normalisation, the pre-LSTM
fully-connected layer and the cross-hero pool, forward and backward.

Test infrastructure (see the package docstring).

What the paper fixes:
* every float observation is normalised with a running mean and standard
  deviation of all data ever observed: subtract the mean, divide by the
  standard deviation, clip to (-5, 5) (appendix "Observation Space");
* five replica networks, one per hero of the team, each see nearly the same
  observation; before the LSTM the flattened observation (with the
  controlled hero's embedding appended) goes through a fully-connected layer
  and a "cross-hero pool" that max-pools the first 25% of the vector across
  the five replicas (appendix "Neural Network Architecture", Figure
  "Observation processing").

Readings where the paper is silent:
* the running statistics are the exact per-feature count, mean and sum of
  squared deviations of every observation seen so far, this batch included
  (merged pairwise), and the scale is 1 / sqrt(var + eps), eps = 1e-8, so a
  constant feature normalises to 0;
* the fully-connected layer is followed by a ReLU (the paper names the layer,
  not its activation);
* the pooled part is the first floor(D / 4) features; the five replicas of a
  team are five consecutive samples b = 5 q + r of the [T, B, D] layout, so B
  is a multiple of 5; at each timestep each replica's pooled features become
  the maximum over the five, the rest is its own;
* the gradient of the maximum goes to the first replica (lowest r) that
  attains it.

Shapes: obs, o [N, Do] with N = T B rows n = t B + b; W [D, Do], b [D];
y, x, dx [N, D].
"""
import numpy as np

REPLICAS = 5


def merge_stats(a, b):
    """Merge per-feature (count, mean, M2) summaries of disjoint row sets."""
    na, ma, qa = a
    nb, mb, qb = b
    n = na + nb
    if n == 0:
        return (0.0, np.zeros_like(ma), np.zeros_like(qa))
    d = mb - ma
    return (n, ma + d * (nb / n), qa + qb + d * d * (na * nb / n))


def obs_normalize(obs, stats, clip=5.0, eps=1e-8):
    """Merge this batch into the running per-feature statistics, then
    normalise and clip.  Returns (o [N, Do], new stats)."""
    obs = np.asarray(obs, np.float64)
    n = obs.shape[0]
    m = obs.mean(axis=0)
    batch = (float(n), m, ((obs - m) ** 2).sum(axis=0))
    cnt, mean, m2 = stats
    new = merge_stats((float(cnt), np.asarray(mean, np.float64), np.asarray(m2, np.float64)), batch)
    var = new[2] / new[0]
    o = np.clip((obs - new[1]) / np.sqrt(var + eps), -clip, clip)
    return o, new


def pooled_width(D):
    return D // 4


def prelstm_forward(o, W, b, T, B):
    """y = relu(o W^T + b); x = y with its first D/4 features replaced, at
    each timestep, by their maximum over the team's five replicas.
    Returns (x [N, D], y [N, D])."""
    y = np.maximum(np.asarray(o, np.float64) @ np.asarray(W, np.float64).T + np.asarray(b, np.float64), 0.0)
    D = y.shape[1]
    P = pooled_width(D)
    g = y.reshape(T, B // REPLICAS, REPLICAS, D)
    x = g.copy()
    x[..., :P] = g[..., :P].max(axis=2, keepdims=True)
    return x.reshape(T * B, D), y


def prelstm_backward(o, W, y, dx, T, B, want_do=False):
    """Gradients of <dx, x> through the pool, the ReLU and the layer.
    Returns (dW [D, Do], db [D], do [N, Do] or None)."""
    y = np.asarray(y, np.float64)
    dx = np.asarray(dx, np.float64)
    D = y.shape[1]
    P = pooled_width(D)
    gy = y.reshape(T, B // REPLICAS, REPLICAS, D)
    gdx = dx.reshape(T, B // REPLICAS, REPLICAS, D)
    dy = gdx.copy()
    # the pooled features: the five replicas' gradients summed onto the first
    # replica attaining the maximum
    win = gy[..., :P].argmax(axis=2)                       # [T, Q, P]
    tot = gdx[..., :P].sum(axis=2)                         # [T, Q, P]
    r = np.arange(REPLICAS)[None, None, :, None]
    dy[..., :P] = np.where(r == win[:, :, None, :], tot[:, :, None, :], 0.0)
    dpre = (dy * (gy > 0)).reshape(T * B, D)
    o = np.asarray(o, np.float64)
    dW = dpre.T @ o
    db = dpre.sum(axis=0)
    do = dpre @ np.asarray(W, np.float64) if want_do else None
    return dW, db, do
