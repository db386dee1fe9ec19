"""Pins for the reward post-processing oracle (appendix "Reward Weights";
Table "Hyperparameters", note on reward normalisation): each test checks a
property the paper's definitions fix, chosen so that a plausible slip (a
missing or mis-signed zero-sum term, team spirit over the wrong heroes, a
wrong averaging count, time weighting applied to the outcome, a wrong
variance merge) fails at least one of them."""
import numpy as np
import pytest

from oracle.reward import batch_stats, merge_stats, reward_process, shape, time_weight


def _inputs(L, G, seed, with_outcome=True):
    rng = np.random.default_rng(seed)
    shaped = rng.standard_normal((L, 10 * G))
    outcome = rng.choice([-1.0, 0.0, 1.0], size=(L, 10 * G), p=[0.01, 0.98, 0.01]) if with_outcome else None
    game_time = rng.uniform(0.0, 60.0, (L, G))
    return shaped, outcome, game_time


def _games(z, L, G):
    return np.asarray(z).reshape(L, G, 2, 5)


@pytest.mark.parametrize("tau", [0.0, 0.3, 1.0])
def test_every_game_sums_to_zero(tau):
    L, G = 7, 5
    shaped, outcome, tm = _inputs(L, G, 1)
    z = _games(shape(shaped, outcome, tm, tau), L, G)
    assert np.max(np.abs(z.sum(axis=(2, 3)))) < 1e-12
    # and the two teams' totals are opposite
    assert np.allclose(z[:, :, 0].sum(-1), -z[:, :, 1].sum(-1), atol=1e-12)


@pytest.mark.parametrize("tau", [0.0, 0.25, 0.8, 1.0])
def test_team_mean_does_not_depend_on_team_spirit(tau):
    # team spirit redistributes within a team; the team's mean reward is its
    # raw mean minus the enemies' raw mean whatever tau is
    L, G = 4, 3
    shaped, _, _ = _inputs(L, G, 2)
    zero = np.zeros((L, G))
    z = _games(shape(shaped, None, zero, tau), L, G)
    raw = _games(shaped, L, G)
    want = raw.mean(-1) - raw.mean(-1)[:, :, ::-1]
    assert np.allclose(z.mean(-1), want, atol=1e-12)


def test_full_team_spirit_shares_equally():
    L, G = 3, 4
    shaped, outcome, tm = _inputs(L, G, 3)
    z = _games(shape(shaped, outcome, tm, 1.0), L, G)
    assert np.max(np.abs(z - z[..., :1])) < 1e-12   # all five heroes of a team equal
    assert np.allclose(z[:, :, 0, 0], -z[:, :, 1, 0], atol=1e-12)


def test_zero_team_spirit_is_selfish_and_enemy_average_has_weight_one_fifth():
    L, G = 2, 2
    shaped, _, _ = _inputs(L, G, 4)
    zero = np.zeros((L, G))
    base = shape(shaped, None, zero, 0.0)
    # a teammate's reward does not reach hero (team 0, hero 0) when tau = 0
    s2 = shaped.copy()
    s2[:, 1] += 3.0
    assert np.allclose(shape(s2, None, zero, 0.0)[:, 0], base[:, 0], atol=1e-12)
    # an enemy's reward enters with weight -1/5, and moves every enemy's own
    # reward only through its own term
    s3 = shaped.copy()
    s3[:, 7] += 2.5
    d = shape(s3, None, zero, 0.0) - base
    assert np.allclose(d[:, 0:5], -0.5, atol=1e-12)
    assert np.allclose(d[:, 7], 2.5, atol=1e-12)
    assert np.allclose(np.delete(d[:, 5:10], 2, axis=1), 0.0, atol=1e-12)


def test_team_spirit_and_zero_sum_commute():
    # the same two maps applied in the other order (zero sum first, on the
    # raw rewards, then team spirit) give the same rewards
    L, G, tau = 5, 3, 0.4
    shaped, outcome, tm = _inputs(L, G, 5)
    rho = _games(shaped * np.repeat(time_weight(tm), 10, axis=1) + outcome, L, G)
    zs = rho - rho.mean(-1, keepdims=True)[:, :, ::-1]
    other = (1 - tau) * zs + tau * zs.mean(-1, keepdims=True)
    assert np.allclose(shape(shaped, outcome, tm, tau), other.reshape(L, -1), atol=1e-12)


def test_time_weighting_decays_shaped_reward_only():
    assert time_weight(0.0) == 1.0
    assert time_weight(10.0) == pytest.approx(0.6, abs=1e-15)
    assert time_weight(20.0) == pytest.approx(0.36, abs=1e-15)
    assert time_weight(5.0) == pytest.approx(np.sqrt(0.6), abs=1e-15)
    L, G = 3, 2
    shaped, outcome, _ = _inputs(L, G, 6)
    t0, t10 = np.zeros((L, G)), np.full((L, G), 10.0)
    # the shaped part scales by 0.6 between minute 0 and minute 10 ...
    assert np.allclose(shape(shaped, None, t10, 0.3), 0.6 * shape(shaped, None, t0, 0.3), atol=1e-12)
    # ... and the outcome does not scale at all
    nothing = np.zeros_like(shaped)
    assert np.allclose(shape(nothing, outcome, t10, 0.3), shape(nothing, outcome, t0, 0.3), atol=1e-15)


def test_fresh_normalisation_gives_unit_variance_and_scale_invariance():
    L, G = 16, 6
    shaped, outcome, tm = _inputs(L, G, 7)
    r, st = reward_process(shaped, outcome, tm, 0.3, (0.0, 0.0, 0.0))
    assert st[0] == L * 10 * G
    assert np.var(r) == pytest.approx(1.0, rel=1e-6)
    r2, _ = reward_process(7.0 * shaped, 7.0 * outcome, tm, 0.3, (0.0, 0.0, 0.0))
    assert np.allclose(r2, r, atol=1e-9)


def test_running_statistics_equal_those_of_all_batches_together():
    L, G = 8, 3
    st = (0.0, 0.0, 0.0)
    seen = []
    for seed in range(4):
        shaped, outcome, tm = _inputs(L, G, 10 + seed)
        r, st = reward_process(shaped, outcome, tm, 0.5, st)
        z = shape(shaped, outcome, tm, 0.5)
        seen.append(z.ravel())
        allz = np.concatenate(seen)
        assert st[0] == allz.size
        assert st[1] == pytest.approx(allz.mean(), abs=1e-12)
        assert st[2] / st[0] == pytest.approx(np.var(allz), rel=1e-12)
        assert np.allclose(r, z / np.sqrt(np.var(allz) + 1e-8), atol=1e-12)


def test_merge_with_empty_summary_is_identity():
    s = batch_stats(np.array([1.0, 2.0, 4.0]))
    assert merge_stats((0.0, 0.0, 0.0), s) == s
    assert merge_stats(s, (0.0, 0.0, 0.0)) == s
    assert s[2] == pytest.approx(np.var([1.0, 2.0, 4.0]) * 3, rel=1e-15)
