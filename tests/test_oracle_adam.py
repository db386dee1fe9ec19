"""Pins for the oracle's Adam + per-parameter clip (CPU only): PyTorch's
float64 Adam with the clip off, and closed forms of the first step, a
constant gradient, lr = 0 and a clipped spike."""
import numpy as np
import torch

from oracle.adam import adam_step


def test_clip_off_matches_torch_adam():
    rng = np.random.default_rng(0)
    n = 257
    p0 = rng.standard_normal(n)
    grads = [rng.standard_normal(n) * (1 + 3 * k) for k in range(6)]
    tp = torch.nn.Parameter(torch.from_numpy(p0.copy()))
    opt = torch.optim.Adam([tp], lr=5e-3, betas=(0.9, 0.999), eps=1e-8)
    p, m, v = p0.copy(), np.zeros(n), np.zeros(n)
    for step, g in enumerate(grads, start=1):
        tp.grad = torch.from_numpy(g.copy())
        opt.step()
        p, m, v = adam_step(p, m, v, g, 5e-3, 0.9, 0.999, 1e-8, 0.0, step)
        np.testing.assert_allclose(p - p0, tp.detach().numpy() - p0, rtol=1e-12, atol=1e-16)


def test_first_step_closed_form_and_clip_inactive():
    rng = np.random.default_rng(1)
    g = rng.standard_normal(100) * 10.0 ** rng.uniform(-6, 2, 100)
    p = rng.standard_normal(100)
    for k in (5.0, 0.0):
        p1, m1, v1 = adam_step(p, np.zeros(100), np.zeros(100), g, 5e-5, 0.9, 0.999, 1e-8, k, 1)
        np.testing.assert_allclose(p1 - p, -5e-5 * g / (np.abs(g) + 1e-8), rtol=1e-9, atol=0)


def test_constant_gradient_gives_constant_update():
    g = np.array([3.0, -0.25, 1e-3, -7e2])
    p, m, v = np.zeros(4), np.zeros(4), np.zeros(4)
    for step in range(1, 40):
        p_new, m, v = adam_step(p, m, v, g, 1e-3, 0.9, 0.999, 1e-8, 5.0, step)
        np.testing.assert_allclose(p_new - p, -1e-3 * g / (np.abs(g) + 1e-8), rtol=1e-9, atol=0)
        p = p_new


def test_lr_zero_leaves_parameters_bitwise():
    rng = np.random.default_rng(2)
    p = rng.standard_normal(50)
    m = rng.standard_normal(50) * 0.1
    v = rng.random(50)
    g = rng.standard_normal(50)
    p1, m1, v1 = adam_step(p, m, v, g, 0.0, 0.9, 0.999, 1e-8, 5.0, 7)
    assert np.array_equal(p1, p)
    assert not np.array_equal(m1, m) and not np.array_equal(v1, v)


def test_spike_is_clipped_to_five_sqrt_vhat():
    b1, b2 = 0.9, 0.999
    p, m, v = np.zeros(1), np.zeros(1), np.zeros(1)
    g0 = 1e-3
    for step in range(1, 101):
        p, m, v = adam_step(p, m, v, np.array([g0]), 0.0, b1, b2, 1e-8, 5.0, step)
    m_before = m.copy()
    p, m, v = adam_step(p, m, v, np.array([1.0]), 0.0, b1, b2, 1e-8, 5.0, 101)
    # geometric sums: after 100 steps of g0, v = (1 - b2^100) g0^2; then the spike enters v
    v101 = b2 * (1 - b2 ** 100) * g0 ** 2 + (1 - b2) * 1.0
    bound = 5.0 * np.sqrt(v101 / (1 - b2 ** 101))
    assert bound < 1.0
    np.testing.assert_allclose(v, v101, rtol=1e-12)
    np.testing.assert_allclose(m, b1 * m_before + (1 - b1) * bound, rtol=1e-12)
    np.testing.assert_allclose(m_before, (1 - b1 ** 100) * g0, rtol=1e-12)
