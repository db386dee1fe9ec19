"""Pins for the LSTM input side (appendix "Observation Space": running
normalisation clipped to +-5; appendix "Neural Network Architecture": the
pre-LSTM fully-connected layer and the cross-hero max-pool of the first 25%
across the five replicas): NumPy statistics of all batches seen, the pool's
defining properties, PyTorch float64 autograd and central finite
differences for the backward, and the tie rule."""
import numpy as np
import pytest
import torch

from oracle.prelstm import REPLICAS, obs_normalize, pooled_width, prelstm_backward, prelstm_forward


def test_running_normalisation_matches_all_batches_together():
    rng = np.random.default_rng(0)
    Do = 7
    st = (0.0, np.zeros(Do), np.zeros(Do))
    seen = []
    for k in range(3):
        obs = rng.normal(3.0, 2.0, (50 + 10 * k, Do))
        o, st = obs_normalize(obs, st)
        seen.append(obs)
        allo = np.concatenate(seen)
        assert st[0] == allo.shape[0]
        np.testing.assert_allclose(st[1], allo.mean(axis=0), rtol=0, atol=1e-12)
        np.testing.assert_allclose(st[2] / st[0], allo.var(axis=0), rtol=1e-12)
        want = np.clip((obs - allo.mean(0)) / np.sqrt(allo.var(0) + 1e-8), -5, 5)
        np.testing.assert_allclose(o, want, rtol=0, atol=1e-12)


def test_fresh_normalisation_standardises_clips_and_zeroes_constants():
    rng = np.random.default_rng(1)
    obs = rng.normal(-2.0, 0.5, (400, 4))
    obs[:, 2] = 7.0                       # a constant feature (e.g. a deprecated observation)
    obs[0, 3] = 1e3                       # an outlier
    o, _ = obs_normalize(obs, (0.0, np.zeros(4), np.zeros(4)))
    np.testing.assert_allclose(o[:, :2].mean(0), 0.0, atol=1e-12)
    np.testing.assert_allclose(o[:, :2].var(0), 1.0, rtol=1e-6)
    assert np.all(o[:, 2] == 0.0)
    assert o[0, 3] == 5.0 and np.all(np.abs(o) <= 5.0)


def _layer(seed, T, B, Do, D):
    rng = np.random.default_rng(seed)
    o = rng.standard_normal((T * B, Do))
    W = rng.standard_normal((D, Do)) / np.sqrt(Do)
    b = rng.standard_normal(D) * 0.1
    return o, W, b


def test_pool_properties():
    T, B, Do, D = 3, 10, 6, 9                # floor(9 / 4) = 2 pooled features
    o, W, b = _layer(2, T, B, Do, D)
    x, y = prelstm_forward(o, W, b, T, B)
    P = pooled_width(D)
    assert P == 2 and np.all(y >= 0)
    gx = x.reshape(T, B // REPLICAS, REPLICAS, D)
    gy = y.reshape(T, B // REPLICAS, REPLICAS, D)
    # the unpooled features are the replica's own; the pooled ones are the
    # same for the five replicas of a team and dominate each of them
    assert np.array_equal(gx[..., P:], gy[..., P:])
    assert np.all(gx[..., :P] == gx[:, :, :1, :P])
    assert np.all(gx[..., :P] >= gy[..., :P])
    assert np.all(np.any(gx[..., :P] == gy[..., :P], axis=2))
    # identical replicas: the pool changes nothing
    o_same = np.repeat(o.reshape(T, B // REPLICAS, REPLICAS, Do)[:, :, :1], REPLICAS, axis=2).reshape(T * B, Do)
    x2, y2 = prelstm_forward(o_same, W, b, T, B)
    assert np.array_equal(x2, y2)


def test_backward_matches_torch_autograd():
    T, B, Do, D = 2, 15, 8, 12
    o, W, b = _layer(3, T, B, Do, D)
    dx = np.random.default_rng(4).standard_normal((T * B, D))
    x, y = prelstm_forward(o, W, b, T, B)
    dW, db, do = prelstm_backward(o, W, y, dx, T, B, want_do=True)
    to = torch.tensor(o, requires_grad=True)
    tW = torch.tensor(W, requires_grad=True)
    tb = torch.tensor(b, requires_grad=True)
    ty = torch.relu(to @ tW.T + tb)
    g = ty.reshape(T, B // REPLICAS, REPLICAS, D)
    P = D // 4
    pooled = g[..., :P].max(dim=2, keepdim=True).values.expand(-1, -1, REPLICAS, -1)
    tx = torch.cat([pooled, g[..., P:]], dim=-1).reshape(T * B, D)
    np.testing.assert_allclose(tx.detach().numpy(), x, rtol=0, atol=1e-14)
    (tx * torch.tensor(dx)).sum().backward()
    np.testing.assert_allclose(dW, tW.grad.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(db, tb.grad.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(do, to.grad.numpy(), rtol=0, atol=1e-12)


def test_backward_central_finite_differences():
    T, B, Do, D = 2, 5, 4, 8
    o, W, b = _layer(5, T, B, Do, D)
    dx = np.random.default_rng(6).standard_normal((T * B, D))

    def f(W_, b_):
        x, _ = prelstm_forward(o, W_, b_, T, B)
        return (x * dx).sum()

    # keep the inputs away from ReLU kinks and from ties of the maximum
    pre = o @ W.T + b
    assert np.min(np.abs(pre)) > 1e-3
    _, y = prelstm_forward(o, W, b, T, B)
    s = np.sort(y.reshape(T, 1, REPLICAS, D)[..., :D // 4], axis=2)
    assert np.min(s[:, :, -1] - s[:, :, -2]) > 1e-3 or np.all(s[:, :, -1] == 0)
    dW, db, _ = prelstm_backward(o, W, y, dx, T, B)
    eps = 1e-6
    for name, arr, analytic in (("W", W, dW), ("b", b, db)):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            p_, m_ = arr.copy(), arr.copy()
            p_[idx] += eps
            m_[idx] -= eps
            fp = f(p_, b) if name == "W" else f(W, p_)
            fm = f(m_, b) if name == "W" else f(W, m_)
            num[idx] = (fp - fm) / (2 * eps)
        assert np.max(np.abs(num - analytic)) / np.max(np.abs(num)) < 1e-7, name


def test_max_tie_sends_the_gradient_to_the_first_replica():
    T, B, Do, D = 1, 5, 3, 4                 # one pooled feature
    W = np.zeros((D, Do))
    b = np.array([2.0, 1.0, 1.0, 1.0])      # every replica's feature 0 equals 2
    o = np.random.default_rng(7).standard_normal((B, Do))
    dx = np.arange(1.0, 1.0 + B * D).reshape(B, D)
    _, y = prelstm_forward(o, W, b, T, B)
    dW, db, _ = prelstm_backward(o, W, y, dx, T, B)
    assert db[0] == dx[:, 0].sum()           # the whole pooled gradient reaches replica 0
    np.testing.assert_array_equal(dW[0], dx[:, 0].sum() * o[0])
