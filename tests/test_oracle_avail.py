"""Pins for the availability mask of the heads (appendix "Action Space":
action filters restrict each timestep's choice to the available actions),
in the PPO loss and in the sampler: PyTorch's float64 Categorical over
logits set to -inf where unavailable, finite differences, and the
invariances the definition fixes (an unavailable logit is inert, a single
available action is certain, an empty head under a zero head mask adds
nothing)."""
import numpy as np
import pytest
import scipy.stats as sstats
import torch

from oracle.philox import gumbel_max_sample
from oracle.ppo import head_logprob_entropy, head_offsets, heads_forward, ppo_loss_grad


def _avail(rng, N, heads, p=0.6):
    """Random availability with at least one available logit per head; the
    taken actions drawn among the available ones."""
    off = head_offsets(heads)
    av = rng.random((N, off[-1])) < p
    act = np.zeros((N, len(heads)), np.int64)
    for k, n in enumerate(heads):
        blk = av[:, off[k]:off[k + 1]]
        none = ~blk.any(axis=1)
        blk[none, rng.integers(0, n, none.sum())] = True
        for i in range(N):
            act[i, k] = rng.choice(np.flatnonzero(blk[i]))
    return av.astype(np.uint8), act


def _inputs(seed, N, H, heads, wscale=0.8):
    rng = np.random.default_rng(seed)
    A1 = sum(heads) + 1
    h = rng.uniform(-1, 1, (N, H))
    Wp = rng.uniform(-wscale, wscale, (A1, H))
    bp = rng.uniform(-wscale, wscale, A1)
    av, act = _avail(rng, N, heads)
    return h, Wp, bp, av, act, rng.standard_normal(N), rng.standard_normal(N)


def _masked_dist(z, av):
    t = torch.from_numpy(z).masked_fill(torch.from_numpy(av == 0), -float("inf"))
    return torch.distributions.Categorical(logits=t)


def test_masked_categorical_matches_torch():
    heads = (30, 8, 32, 4)
    h, Wp, bp, av, act, *_ = _inputs(1, 40, 12, heads)
    z = heads_forward(h, Wp, bp)
    logp, ent, probs = head_logprob_entropy(z, act, heads, av)
    off = head_offsets(heads)
    for k in range(len(heads)):
        d = _masked_dist(z[:, off[k]:off[k + 1]], av[:, off[k]:off[k + 1]])
        np.testing.assert_allclose(logp[:, k], d.log_prob(torch.from_numpy(act[:, k])).numpy(), rtol=0, atol=1e-13)
        np.testing.assert_allclose(ent[:, k], d.entropy().numpy(), rtol=0, atol=1e-13)
        np.testing.assert_allclose(probs[k], d.probs.numpy(), rtol=0, atol=1e-15)


def test_all_available_equals_no_mask():
    heads = (5, 3, 4)
    h, Wp, bp, _, act, adv, ret = _inputs(2, 16, 6, heads)
    lo = np.zeros(16)
    a = ppo_loss_grad(h, Wp, bp, act, lo, adv, ret, heads)
    b = ppo_loss_grad(h, Wp, bp, act, lo, adv, ret, heads, avail=np.ones((16, 12), np.uint8))
    assert a[0] == b[0]
    for x, y in zip(a[1:], b[1:]):
        assert np.array_equal(x, y)


def test_unavailable_logit_is_inert():
    heads = (5, 3, 4)
    h, Wp, bp, av, act, adv, ret = _inputs(3, 16, 6, heads)
    c = 6                                       # column 1 of head 1: unavailable everywhere
    av[:, c] = 0
    act[act[:, 1] == 1, 1] = 0
    av[:, 5] = 1
    lo = np.zeros(16)
    s1, dh1, dWp1, dbp1, _ = ppo_loss_grad(h, Wp, bp, act, lo, adv, ret, heads, avail=av)
    Wp2, bp2 = Wp.copy(), bp.copy()
    Wp2[c] += 3.0
    bp2[c] -= 5.0
    s2, dh2, *_ = ppo_loss_grad(h, Wp2, bp2, act, lo, adv, ret, heads, avail=av)
    assert s1["total"] == s2["total"]
    assert np.array_equal(dh1, dh2)
    assert dbp1[c] == 0.0 and np.all(dWp1[c] == 0.0)


def test_single_available_action_is_certain():
    heads = (5, 3)
    h, Wp, bp, av, act, adv, ret = _inputs(4, 12, 5, heads)
    av[:, 5:8] = 0
    av[:, 6] = 1                                # head 1: only its action 1 is available
    act[:, 1] = 1
    z = heads_forward(h, Wp, bp)
    logp, ent, probs = head_logprob_entropy(z, act, heads, av)
    assert np.all(logp[:, 1] == 0.0) and np.all(ent[:, 1] == 0.0)
    _, _, _, dbp, _ = ppo_loss_grad(h, Wp, bp, act, np.zeros(12), adv, ret, heads, avail=av)
    assert np.all(dbp[5:8] == 0.0)


def test_empty_head_under_zero_head_mask_adds_nothing():
    heads = (5, 3)
    h, Wp, bp, av, act, adv, ret = _inputs(5, 12, 5, heads)
    mask = np.ones((12, 2))
    mask[::3, 1] = 0
    empty = av.copy()
    empty[::3, 5:8] = 0                         # no available logit where the head is masked
    lo = np.zeros(12)
    a = ppo_loss_grad(h, Wp, bp, act, lo, adv, ret, heads, head_mask=mask, avail=av)
    b = ppo_loss_grad(h, Wp, bp, act, lo, adv, ret, heads, head_mask=mask, avail=empty)
    assert a[0]["total"] == pytest.approx(b[0]["total"], abs=1e-15)
    np.testing.assert_allclose(a[1], b[1], rtol=0, atol=1e-16)


@pytest.mark.parametrize("use_mask", [False, True])
def test_avail_gradients_central_finite_differences(use_mask):
    heads = (5, 3, 4)
    N, H = 12, 6
    h, Wp, bp, av, act, adv, ret = _inputs(6, N, H, heads)
    mask = (np.random.default_rng(9).random((N, 3)) < 0.7).astype(np.float64) if use_mask else None
    z = heads_forward(h, Wp, bp)
    logp, _, _ = head_logprob_entropy(z, act, heads, av)
    lp = (logp * (1.0 if mask is None else mask)).sum(axis=1)
    shift = np.array([-0.6, -0.3, -0.1, 0.0, 0.1, 0.3, 0.6, -0.05, 0.05, 0.4, -0.4, 0.12])
    logp_old = lp + shift

    def total(h_, Wp_, bp_):
        return ppo_loss_grad(h_, Wp_, bp_, act, logp_old, adv, ret, heads, 0.2, 0.7, 0.05, mask, av)[0]["total"]

    _, dh, dWp, dbp, _ = ppo_loss_grad(h, Wp, bp, act, logp_old, adv, ret, heads, 0.2, 0.7, 0.05, mask, av)
    eps = 1e-6
    for name, arr, analytic in (("h", h, dh), ("Wp", Wp, dWp), ("bp", bp, dbp)):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            p_, m_ = arr.copy(), arr.copy()
            p_[idx] += eps
            m_[idx] -= eps
            args_p = {"h_": h, "Wp_": Wp, "bp_": bp}
            args_m = dict(args_p)
            args_p[name + "_"], args_m[name + "_"] = p_, m_
            fp, fm = total(**args_p), total(**args_m)
            num[idx] = (fp - fm) / (2 * eps)
        rel = np.max(np.abs(num - analytic)) / np.max(np.abs(num))
        assert rel < 1e-7, (name, rel)


def test_masked_sampler_frequencies_and_empty_heads():
    rng = np.random.default_rng(7)
    heads = (6, 3)
    z_row = np.concatenate([rng.normal(0, 1.5, 6), rng.normal(0, 0.5, 3), [0.0]])
    av_row = np.array([1, 0, 1, 1, 0, 1, 0, 0, 0], np.uint8)   # head 1 empty
    B = 200_000
    z = np.broadcast_to(z_row, (B, 10))
    av = np.broadcast_to(av_row, (B, 9))
    act, logp, _, _ = gumbel_max_sample(z, heads, seed=3, counter=2, avail=av)
    assert np.all(act[:, 1] == -1)
    counts = np.bincount(act[:, 0], minlength=6)
    assert counts[1] == 0 and counts[4] == 0
    keep = av_row[:6] == 1
    p = np.exp(z_row[:6][keep] - z_row[:6][keep].max())
    p /= p.sum()
    assert sstats.chisquare(counts[keep], B * p).pvalue > 1e-3
    d = _masked_dist(np.ascontiguousarray(z[:64, :6]), np.ascontiguousarray(av[:64, :6]))
    np.testing.assert_allclose(logp[:64], d.log_prob(torch.from_numpy(act[:64, 0]).long()).numpy(), rtol=0, atol=1e-13)
