"""Pins for the oracle's heads, PPO loss and gradient (CPU only): PPO
invariants, the uniform-policy entropy, finite differences and PyTorch's
float64 Categorical distribution."""
import numpy as np
import pytest
import torch

from oracle.ppo import head_logprob_entropy, head_offsets, heads_forward, ppo_loss_grad

HEADS = (30, 8, 32, 4)


def _inputs(seed, N=24, H=16, heads=HEADS, wscale=0.3):
    rng = np.random.default_rng(seed)
    A1 = sum(heads) + 1
    h = rng.uniform(-1, 1, (N, H))
    Wp = rng.uniform(-wscale, wscale, (A1, H))
    bp = rng.uniform(-wscale, wscale, A1)
    act = np.stack([rng.integers(0, n, N) for n in heads], axis=1)
    adv = rng.standard_normal(N)
    ret = rng.standard_normal(N)
    return h, Wp, bp, act, adv, ret


def _logpi(h, Wp, bp, act, heads, mask=None):
    z = heads_forward(h, Wp, bp)
    logp, _, _ = head_logprob_entropy(z, act, heads)
    if mask is None:
        mask = np.ones_like(logp)
    return (mask * logp).sum(axis=1)


def test_ratio_one_invariant():
    h, Wp, bp, act, adv, ret = _inputs(0)
    logp_old = _logpi(h, Wp, bp, act, HEADS)
    stats, dh, dWp, dbp, z = ppo_loss_grad(h, Wp, bp, act, logp_old, adv, ret, HEADS,
                                           ent_coef=0.0, vf_coef=0.0)
    assert abs(stats["pg"] - (-adv.mean())) < 1e-14
    assert abs(stats["mean_ratio"] - 1.0) < 1e-14
    assert stats["clipfrac"] == 0.0 and abs(stats["approx_kl"]) < 1e-14
    # dL_pg/dz = -(A/N) (onehot - p) on every head
    N = h.shape[0]
    off = head_offsets(HEADS)
    dz = np.zeros_like(z)
    for k, n in enumerate(HEADS):
        zk = z[:, off[k]:off[k + 1]]
        p = np.exp(zk - zk.max(1, keepdims=True))
        p /= p.sum(1, keepdims=True)
        oh = np.eye(n)[act[:, k]]
        dz[:, off[k]:off[k + 1]] = -(adv / N)[:, None] * (oh - p)
    np.testing.assert_allclose(dbp, dz.sum(0), rtol=0, atol=1e-14)
    np.testing.assert_allclose(dWp, dz.T @ h, rtol=0, atol=1e-14)


def test_uniform_policy_entropy():
    h, Wp, bp, act, adv, ret = _inputs(1)
    Wp[:] = 0
    bp[:] = 0
    stats, *_ = ppo_loss_grad(h, Wp, bp, act, np.zeros(len(adv)), adv, ret, HEADS)
    assert abs(stats["ent"] - np.log(30 * 8 * 32 * 4)) < 1e-12
    assert abs(np.log(30720) - 10.332669) < 1e-6   # ln 3 + 11 ln 2 + ln 5


def test_all_ratios_clipped_high_with_positive_advantage():
    h, Wp, bp, act, adv, ret = _inputs(2)
    adv = np.abs(adv) + 0.1
    logp_old = _logpi(h, Wp, bp, act, HEADS) - 0.5      # r = e^0.5 > 1.2
    stats, dh, dWp, dbp, z = ppo_loss_grad(h, Wp, bp, act, logp_old, adv, ret, HEADS,
                                           ent_coef=0.0, vf_coef=0.0)
    assert abs(stats["pg"] - (-(1.2) * adv.mean())) < 1e-14
    assert stats["clipfrac"] == 1.0
    assert not dh.any() and not dWp.any() and not dbp.any()


def test_value_equal_to_return_gives_zero_value_loss():
    h, Wp, bp, act, adv, ret = _inputs(3)
    ret = heads_forward(h, Wp, bp)[:, -1]
    stats, dh, dWp, dbp, _ = ppo_loss_grad(h, Wp, bp, act, np.zeros(len(adv)), adv, ret, HEADS)
    assert abs(stats["vf"]) < 1e-28
    assert abs(dbp[-1]) < 1e-15


def test_categorical_matches_torch():
    h, Wp, bp, act, *_ = _inputs(4)
    z = heads_forward(h, Wp, bp)
    logp, ent, _ = head_logprob_entropy(z, act, HEADS)
    off = head_offsets(HEADS)
    for k in range(len(HEADS)):
        dist = torch.distributions.Categorical(logits=torch.from_numpy(z[:, off[k]:off[k + 1]]))
        np.testing.assert_allclose(logp[:, k], dist.log_prob(torch.from_numpy(act[:, k])).numpy(),
                                   rtol=0, atol=1e-13)
        np.testing.assert_allclose(ent[:, k], dist.entropy().numpy(), rtol=0, atol=1e-13)


def _total(h, Wp, bp, act, logp_old, adv, ret, heads, mask):
    st, *_ = ppo_loss_grad(h, Wp, bp, act, logp_old, adv, ret, heads, 0.2, 0.7, 0.05, mask)
    return st["total"]


@pytest.mark.parametrize("use_mask", [False, True])
def test_gradients_central_finite_differences(use_mask):
    heads = (5, 3, 4)
    h, Wp, bp, act, adv, ret = _inputs(5, N=12, H=6, heads=heads, wscale=0.8)
    rng = np.random.default_rng(7)
    mask = (rng.random((12, 3)) < 0.7).astype(np.float64) if use_mask else None
    lp = _logpi(h, Wp, bp, act, heads, mask)
    # ratios spread over both sides of the clip range but >= 0.02 from the kinks
    shift = np.array([-0.6, -0.3, -0.1, 0.0, 0.1, 0.3, 0.6, -0.05, 0.05, 0.4, -0.4, 0.12])
    logp_old = lp + shift
    r = np.exp(-shift)
    assert np.all(np.abs(r - 1.2) > 0.02) and np.all(np.abs(r - 0.8) > 0.02)
    stats, dh, dWp, dbp, _ = ppo_loss_grad(h, Wp, bp, act, logp_old, adv, ret, heads,
                                           0.2, 0.7, 0.05, mask)
    eps = 1e-6
    for name, arr, analytic in (("h", h, dh), ("Wp", Wp, dWp), ("bp", bp, dbp)):
        num = np.zeros_like(arr)
        it = np.nditer(arr, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            a_p, a_m = arr.copy(), arr.copy()
            a_p[idx] += eps
            a_m[idx] -= eps
            args_p = {"h": h, "Wp": Wp, "bp": bp}
            args_m = dict(args_p)
            args_p[name], args_m[name] = a_p, a_m
            fp = _total(args_p["h"], args_p["Wp"], args_p["bp"], act, logp_old, adv, ret, heads, mask)
            fm = _total(args_m["h"], args_m["Wp"], args_m["bp"], act, logp_old, adv, ret, heads, mask)
            num[idx] = (fp - fm) / (2 * eps)
        rel = np.max(np.abs(num - analytic)) / np.max(np.abs(num))
        assert rel < 1e-7, (name, rel)


def test_head_mask_zero_removes_head():
    heads = (5, 3)
    h, Wp, bp, act, adv, ret = _inputs(6, N=10, H=4, heads=heads)
    mask = np.ones((10, 2))
    mask[:, 1] = 0
    act2 = act.copy()
    act2[:, 1] = (act[:, 1] + 1) % 3          # a masked head's action is irrelevant
    s1, dh1, *_ = ppo_loss_grad(h, Wp, bp, act, np.zeros(10), adv, ret, heads, head_mask=mask)
    s2, dh2, *_ = ppo_loss_grad(h, Wp, bp, act2, np.zeros(10), adv, ret, heads, head_mask=mask)
    assert s1["total"] == s2["total"]
    assert np.array_equal(dh1, dh2)


@pytest.mark.filterwarnings("ignore:invalid value encountered:RuntimeWarning")
def test_nonfinite_count():
    h, Wp, bp, act, adv, ret = _inputs(8, N=10, H=4, heads=(3,))
    adv[2] = np.nan
    ret[7] = np.inf
    stats, *_ = ppo_loss_grad(h, Wp, bp, act, np.zeros(10), adv, ret, (3,))
    assert stats["nonfinite"] == 2.0


def _one_head_rows(z_row, counts):
    """Rows that all share one logit vector z_row (a single head), with
    action a repeated counts[a] times."""
    act = np.concatenate([np.full(c, a) for a, c in enumerate(counts)])[:, None]
    N = len(act)
    Wp = np.zeros((len(z_row) + 1, 1))
    bp = np.append(np.asarray(z_row, np.float64), 0.0)
    h = np.ones((N, 1))
    return h, Wp, bp, act


def test_approx_kl_is_the_exact_kl_when_rows_follow_the_old_policy():
    """Statistics at r != 1 pinned by an identity that does not involve the
    estimator's formula: when the taken actions occur exactly in proportion
    to the behaviour policy p (action a in k_a of M rows, p_a = k_a / M),
    the row mean of (r - 1) - log r with r = q_a / p_a is
    sum_a q_a - 1 + sum_a p_a log(p_a / q_a) = KL(p || q), the exact
    Kullback-Leibler divergence of the new policy q from p; the row mean of
    r is sum_a q_a = 1."""
    from scipy.special import softmax
    from scipy.stats import entropy
    counts = np.array([1, 3, 6, 2, 8])          # p = (1, 3, 6, 2, 8) / 20
    p = counts / counts.sum()
    z = np.array([0.7, -0.2, 0.4, 1.1, -0.5])   # the new policy's logits
    q = softmax(z)
    h, Wp, bp, act = _one_head_rows(z, counts)
    N = len(act)
    logp_old = np.log(p[act[:, 0]])
    adv, ret = np.ones(N), np.zeros(N)
    stats, *_ = ppo_loss_grad(h, Wp, bp, act, logp_old, adv, ret, (5,))
    kl = entropy(p, q)                          # scipy: sum p log(p / q)
    assert kl > 0.1                              # far from r = 1
    assert abs(stats["approx_kl"] - kl) < 1e-14
    assert abs(stats["mean_ratio"] - 1.0) < 1e-14
    # swapping the roles of the two policies (the ratio inverted) gives a
    # different number, so the sign convention of the log-ratio is pinned
    inv = np.mean(p[act[:, 0]] / q[act[:, 0]] - 1.0 - np.log(p[act[:, 0]] / q[act[:, 0]]))
    assert abs(inv - kl) > 1e-3


def test_ratio_statistics_at_hand_chosen_log_ratios():
    """Rows whose log-ratio d = log pi - log pi_old is set by hand: r = e^d.
    The clip range (1 - 0.2, 1 + 0.2) is (e^-0.22314, e^0.18232) in d, so
    of d = (0.18, 0.19, -0.22, -0.23, 0, 1) exactly three rows (0.19, -0.23,
    1) lie outside it; one row of d = 0.3 gives approx_kl = e^0.3 - 1.3 and
    mean_ratio = e^0.3 (e^0.3 = 1.3498588075760032), and one of d = -0.3
    gives e^-0.3 - 0.7 and e^-0.3 (e^-0.3 = 0.7408182206817179)."""
    heads = (4, 3)
    h, Wp, bp, act, adv, ret = _inputs(11, N=6, H=5, heads=heads)
    lp = _logpi(h, Wp, bp, act, heads)
    d = np.array([0.18, 0.19, -0.22, -0.23, 0.0, 1.0])
    stats, *_ = ppo_loss_grad(h, Wp, bp, act, lp - d, adv, ret, heads)
    assert stats["clipfrac"] == 0.5
    for dd, e_d in ((0.3, 1.3498588075760032), (-0.3, 0.7408182206817179)):
        s1, *_ = ppo_loss_grad(h[:1], Wp, bp, act[:1], lp[:1] - dd, adv[:1], ret[:1], heads)
        assert abs(s1["mean_ratio"] - e_d) < 1e-15
        assert abs(s1["approx_kl"] - (e_d - 1.0 - dd)) < 1e-15
        assert s1["clipfrac"] == 1.0
