"""Pins for the oracle's GAE (CPU only): closed forms, special cases and an
O(L^2) brute-force sum, none of which shares the reverse recursion."""
import numpy as np
import pytest

from oracle.gae import gae, segments_to_samples


def _inputs(seed, L=37, S=5, p_done=0.1):
    rng = np.random.default_rng(seed)
    r = rng.standard_normal((L, S))
    v = rng.standard_normal((L + 1, S))
    d = (rng.random((L, S)) < p_done).astype(np.uint8)
    return r, v, d


def test_lambda_zero_is_td_residual():
    r, v, d = _inputs(0)
    g = 0.97
    adv, ret = gae(r, v, d, g, 0.0)
    td = r + g * (1 - d) * v[1:] - v[:-1]
    np.testing.assert_allclose(adv, td, rtol=0, atol=1e-14)
    np.testing.assert_allclose(ret, adv + v[:-1], rtol=0, atol=1e-14)


def test_lambda_one_no_dones_is_discounted_return_minus_value():
    r, v, _ = _inputs(1)
    L, S = r.shape
    g = 0.998
    adv, _ = gae(r, v, np.zeros((L, S), np.uint8), g, 1.0)
    for t in range(L):
        disc = sum(g ** l * r[t + l] for l in range(L - t)) + g ** (L - t) * v[L]
        np.testing.assert_allclose(adv[t], disc - v[t], rtol=0, atol=1e-12)


def test_gamma_zero_and_all_dones_give_r_minus_v():
    r, v, d = _inputs(2)
    adv0, _ = gae(r, v, d, 0.0, 0.95)
    np.testing.assert_allclose(adv0, r - v[:-1], rtol=0, atol=1e-15)
    adv1, _ = gae(r, v, np.ones_like(d), 0.998, 0.95)
    np.testing.assert_allclose(adv1, r - v[:-1], rtol=0, atol=1e-15)


@pytest.mark.parametrize("seed", [3, 4])
def test_brute_force_sum(seed):
    r, v, d = _inputs(seed, L=29, S=4, p_done=0.2)
    g, lam = 0.99, 0.9
    adv, _ = gae(r, v, d, g, lam)
    L, S = r.shape
    nd = 1.0 - d
    delta = r + g * nd * v[1:] - v[:-1]
    brute = np.zeros((L, S))
    for t in range(L):
        for l in range(L - t):
            alive = np.prod(nd[t:t + l], axis=0) if l > 0 else np.ones(S)
            brute[t] += (g * lam) ** l * alive * delta[t + l]
    np.testing.assert_allclose(adv, brute, rtol=0, atol=1e-12)


def test_segments_to_samples_layout():
    # L = 4 steps, S = 2 segments, T = 2: 2 samples per segment, 4 samples.
    adv = np.array([[0., 10.], [1., 11.], [2., 12.], [3., 13.]])
    ret = adv + 100
    done = np.array([[0, 1], [1, 0], [0, 1], [1, 1]], np.uint8)
    a_s, r_s, reset = segments_to_samples(adv, ret, done, 2)
    # sample b = s*2 + j holds steps 2j, 2j+1 of segment s
    np.testing.assert_array_equal(a_s, [[0., 2., 10., 12.], [1., 3., 11., 13.]])
    np.testing.assert_array_equal(r_s, a_s + 100)
    # reset[1, b] = done at step 2j of segment s; reset[0] = 0
    np.testing.assert_array_equal(reset, [[0, 0, 0, 0], [0, 0, 1, 1]])
