"""Pin for the oracle's composed optimizer step (CPU only): the gradient it
hands to Adam must be the derivative of the total PPO loss with respect to
every parameter through heads and LSTM, checked by central differences."""
import numpy as np

from oracle import gae as ogae
from oracle import lstm as olstm
from oracle import ppo as oppo
from oracle.step import PARAM_ORDER, flatten, ppo_step, unflatten


def _tiny():
    rng = np.random.default_rng(0)
    T, L, S, D, H = 3, 6, 2, 3, 4
    B = S * L // T
    heads = (3, 2)
    A1 = sum(heads) + 1
    params = {
        "Wx": rng.uniform(-0.6, 0.6, (4 * H, D)), "Wh": rng.uniform(-0.6, 0.6, (4 * H, H)),
        "b": rng.uniform(-0.3, 0.3, 4 * H), "Wp": rng.uniform(-0.6, 0.6, (A1, H)),
        "bp": rng.uniform(-0.3, 0.3, A1),
    }
    x = rng.standard_normal((T, B, D))
    h0 = rng.standard_normal((B, H)) * 0.3
    c0 = rng.standard_normal((B, H)) * 0.3
    r = rng.standard_normal((L, S))
    d = np.zeros((L, S), np.uint8)
    d[1, 0] = 1
    d[4, 1] = 1
    v = rng.standard_normal((L + 1, S))
    act = np.stack([rng.integers(0, n, T * B) for n in heads], axis=1)
    logp_old = rng.uniform(-2.5, -1.0, T * B)
    return params, x, h0, c0, r, d, v, act, logp_old, heads, T


def _loss(params, x, h0, c0, r, d, v, act, logp_old, heads, T):
    adv, ret = ogae.gae(r, v, d, 0.998, 0.95)
    adv_s, ret_s, reset = ogae.segments_to_samples(adv, ret, d, T)
    h, c, g = olstm.lstm_forward(x, params["Wx"], params["Wh"], params["b"], h0, c0, reset)
    N = h.shape[0] * h.shape[1]
    st, *_ = oppo.ppo_loss_grad(h.reshape(N, -1), params["Wp"], params["bp"], act, logp_old,
                                adv_s.ravel(), ret_s.ravel(), heads)
    return st["total"]


def test_step_gradient_is_derivative_of_total_loss():
    params, x, h0, c0, r, d, v, act, logp_old, heads, T = _tiny()
    out = ppo_step(params, x, h0, c0, r, d, v, act, logp_old, heads, T)
    # the reset mask derived from dones is exercised
    assert out["reset"].any()
    g = out["grad_flat"]
    flat = flatten(params)
    eps = 1e-6
    num = np.zeros_like(flat)
    for i in range(flat.size):
        fp, fm = flat.copy(), flat.copy()
        fp[i] += eps
        fm[i] -= eps
        num[i] = (_loss(unflatten(fp, params), x, h0, c0, r, d, v, act, logp_old, heads, T) -
                  _loss(unflatten(fm, params), x, h0, c0, r, d, v, act, logp_old, heads, T)) / (2 * eps)
    rel = np.max(np.abs(num - g)) / np.max(np.abs(num))
    assert rel < 1e-7, rel
    assert abs(out["stats"]["total"] - _loss(params, x, h0, c0, r, d, v, act, logp_old, heads, T)) < 1e-15
    # first Adam step moves every parameter by lr * g / (|g| + eps)
    np.testing.assert_allclose(out["p_new"] - flat, -5e-5 * g / (np.abs(g) + 1e-8), rtol=1e-9)
    assert list(out["params_new"].keys()) == list(PARAM_ORDER)
