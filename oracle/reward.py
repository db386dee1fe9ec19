"""Reward post-processing ahead of GAE, in fp64.

Test infrastructure (see the package docstring).

Appendix "Reward Weights" lists three transformations of the per-hero raw
reward, for games of two teams of five heroes:

* game time weighting: every reward except the win/loss outcome is scaled by
  0.6 ** (T / 10 minutes), T the game time at which it is earned;
* team spirit tau: hero i of a team receives (1 - tau) rho_i + tau * mean of
  rho over its own team;
* zero sum: from each hero's reward the average reward of the five enemies
  is subtracted.

Table "Hyperparameters" (note on the value loss weight) adds that rewards are
normalised by a running estimate of their standard deviation.

Readings where the paper is silent:
* team spirit and zero sum are both applied to the time-weighted reward plus
  the outcome; the enemies' average in the zero-sum step is taken over their
  rewards after team spirit.  Both maps are linear and team spirit keeps a
  team's mean, so the order of the two does not matter (pinned in the tests);
* the normalisation divides by the standard deviation and does not subtract
  a mean; the running estimate is the exact variance of every processed
  reward seen so far (counts, means and squared deviations merged batch by
  batch), this batch included; r = z / sqrt(var + eps);
* layout: segment s = 10 g + 5 team + hero of the [L, S] GAE layout, game
  time [L, G] in minutes.
"""
import numpy as np

HEROES = 5   # per team
TEAMS = 2


def time_weight(game_time, base=0.6, period=10.0):
    """The game-time factor base ** (T / period) of the shaped reward."""
    return np.power(base, np.asarray(game_time, np.float64) / period)


def shape(shaped, outcome, game_time, tau, base=0.6, period=10.0):
    """Time weighting, team spirit and zero sum.  shaped, outcome: [L, S]
    with S = 10 G (outcome may be None); game_time [L, G].  Returns z [L, S]."""
    shaped = np.asarray(shaped, np.float64)
    L, S = shaped.shape
    G = S // (TEAMS * HEROES)
    assert G * TEAMS * HEROES == S
    rho = shaped.reshape(L, G, TEAMS, HEROES) * time_weight(game_time, base, period).reshape(L, G, 1, 1)
    if outcome is not None:
        rho = rho + np.asarray(outcome, np.float64).reshape(L, G, TEAMS, HEROES)
    # team spirit: mix each hero's reward with its team's mean
    own_mean = rho.mean(axis=3, keepdims=True)
    tilde = (1.0 - tau) * rho + tau * own_mean
    # zero sum: subtract the enemy team's average
    enemy_mean = tilde.mean(axis=3, keepdims=True)[:, :, ::-1, :]
    z = tilde - enemy_mean
    return z.reshape(L, S)


def merge_stats(a, b):
    """Merge two (count, mean, M2) summaries of disjoint sets of values
    (M2 = sum of squared deviations from the mean): the textbook pairwise
    update of Chan, Golub and LeVeque."""
    na, ma, qa = a
    nb, mb, qb = b
    n = na + nb
    if n == 0:
        return (0.0, 0.0, 0.0)
    d = mb - ma
    return (n, ma + d * nb / n, qa + qb + d * d * na * nb / n)


def batch_stats(z):
    z = np.asarray(z, np.float64).ravel()
    if z.size == 0:
        return (0.0, 0.0, 0.0)
    m = z.mean()
    return (float(z.size), float(m), float(((z - m) ** 2).sum()))


def reward_process(shaped, outcome, game_time, tau, stats, base=0.6, period=10.0, eps=1e-8):
    """One call: returns (r [L, S], new stats).  ``stats`` is the running
    (count, mean, M2) before this batch ((0, 0, 0) at the start)."""
    z = shape(shaped, outcome, game_time, tau, base, period)
    new = merge_stats(tuple(float(x) for x in stats), batch_stats(z))
    var = new[2] / new[0]
    return z / np.sqrt(var + eps), new
