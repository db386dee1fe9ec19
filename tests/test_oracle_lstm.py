"""Pins for the oracle's LSTM forward pass and truncated BPTT (CPU only).

Each check ties the oracle to something other than itself: PyTorch's float64
LSTMCell and autograd (an independent implementation with the same gate order
i, f, g, o), a closed form, central finite differences, or an invariant.
"""
import numpy as np
import pytest
import torch

from oracle.lstm import lstm_bptt, lstm_forward, sigmoid


def _tiny(seed, T=4, B=2, D=3, H=4, with_reset=False, state=0.5):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, B, D))
    Wx = rng.uniform(-0.7, 0.7, (4 * H, D))
    Wh = rng.uniform(-0.7, 0.7, (4 * H, H))
    b = rng.uniform(-0.5, 0.5, 4 * H)
    h0 = rng.standard_normal((B, H)) * state
    c0 = rng.standard_normal((B, H)) * state
    reset = None
    if with_reset:
        reset = np.zeros((T, B), np.uint8)
        reset[2, 0] = 1
        reset[1, 1] = 1
    return x, Wx, Wh, b, h0, c0, reset


def _torch_cell_forward(x, Wx, Wh, b, h0, c0, reset):
    T, B, D = x.shape
    H = Wh.shape[1]
    cell = torch.nn.LSTMCell(D, H).double()
    with torch.no_grad():
        cell.weight_ih.copy_(torch.from_numpy(Wx))
        cell.weight_hh.copy_(torch.from_numpy(Wh))
        cell.bias_ih.copy_(torch.from_numpy(b))
        cell.bias_hh.zero_()
    h = torch.from_numpy(h0).clone()
    c = torch.from_numpy(c0).clone()
    hs, cs = [], []
    for t in range(T):
        if reset is not None:
            keep = 1.0 - torch.from_numpy(reset[t].astype(np.float64))[:, None]
            h, c = h * keep, c * keep
        h, c = cell(torch.from_numpy(x[t]), (h, c))
        hs.append(h)
        cs.append(c)
    return cell, torch.stack(hs), torch.stack(cs)


@pytest.mark.parametrize("with_reset", [False, True])
def test_forward_matches_torch_lstmcell(with_reset):
    x, Wx, Wh, b, h0, c0, reset = _tiny(1, T=6, B=3, D=5, H=7, with_reset=with_reset)
    h, c, gates = lstm_forward(x, Wx, Wh, b, h0, c0, reset)
    _, th, tc = _torch_cell_forward(x, Wx, Wh, b, h0, c0, reset)
    assert np.max(np.abs(h - th.detach().numpy())) < 1e-12
    assert np.max(np.abs(c - tc.detach().numpy())) < 1e-12


def test_forward_closed_form_zero_weights():
    # W = 0, b = 0: i = f = o = 1/2 and g = 0, so c_t = c0 / 2^(t+1), h_t = tanh(c_t) / 2.
    T, B, D, H = 5, 3, 4, 6
    rng = np.random.default_rng(2)
    x = rng.standard_normal((T, B, D))
    c0 = rng.standard_normal((B, H))
    h0 = rng.standard_normal((B, H))
    h, c, gates = lstm_forward(x, np.zeros((4 * H, D)), np.zeros((4 * H, H)),
                               np.zeros(4 * H), h0, c0)
    for t in range(T):
        np.testing.assert_allclose(c[t], c0 * 0.5 ** (t + 1), rtol=0, atol=1e-15)
        np.testing.assert_allclose(h[t], 0.5 * np.tanh(c0 * 0.5 ** (t + 1)), rtol=0, atol=1e-15)
    assert np.all(gates[:, :, 2 * H:3 * H] == 0.0)


def test_forward_reset_everywhere_ignores_start_state():
    x, Wx, Wh, b, h0, c0, _ = _tiny(3, T=4, B=2, D=3, H=4)
    reset = np.ones((4, 2), np.uint8)
    h1, c1, _ = lstm_forward(x, Wx, Wh, b, h0, c0, reset)
    h2, c2, _ = lstm_forward(x, Wx, Wh, b, 5 * h0 + 1, -c0, reset)
    assert np.array_equal(h1, h2) and np.array_equal(c1, c2)
    # and each step is then a fresh cell started from zeros
    h3, c3, _ = lstm_forward(x[2:3], Wx, Wh, b, np.zeros_like(h0), np.zeros_like(c0))
    assert np.array_equal(h1[2], h3[0])


def test_sigmoid_extremes():
    a = np.array([-800.0, -30.0, 0.0, 30.0, 800.0])
    s = sigmoid(a)
    assert np.all(np.isfinite(s))
    assert s[2] == 0.5 and s[0] == 0.0 and s[4] == 1.0
    np.testing.assert_allclose(s + sigmoid(-a), 1.0, rtol=0, atol=1e-15)


def _objective(x, Wx, Wh, b, h0, c0, reset, dh, dhT, dcT):
    h, c, _ = lstm_forward(x, Wx, Wh, b, h0, c0, reset)
    return float((dh * h).sum() + (dhT * h[-1]).sum() + (dcT * c[-1]).sum())


@pytest.mark.parametrize("with_reset", [False, True])
@pytest.mark.parametrize("T", [3, 5])
def test_bptt_central_finite_differences(T, with_reset):
    x, Wx, Wh, b, h0, c0, reset = _tiny(10 + T, T=T, B=2, D=3, H=4, with_reset=with_reset)
    rng = np.random.default_rng(99)
    dh = rng.standard_normal((T, 2, 4))
    dhT = rng.standard_normal((2, 4))
    dcT = rng.standard_normal((2, 4))
    h, c, gates = lstm_forward(x, Wx, Wh, b, h0, c0, reset)
    dWx, dWh, db, dx = lstm_bptt(x, Wx, Wh, h0, c0, reset, h, c, gates, dh, dhT, dcT,
                                 want_dx=True)
    eps = 1e-6

    def fd(arr_name):
        arrs = {"x": x, "Wx": Wx, "Wh": Wh, "b": b}
        base = arrs[arr_name]
        g = np.zeros_like(base)
        it = np.nditer(base, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            plus = {k: v.copy() for k, v in arrs.items()}
            minus = {k: v.copy() for k, v in arrs.items()}
            plus[arr_name][idx] += eps
            minus[arr_name][idx] -= eps
            fp = _objective(plus["x"], plus["Wx"], plus["Wh"], plus["b"], h0, c0, reset, dh, dhT, dcT)
            fm = _objective(minus["x"], minus["Wx"], minus["Wh"], minus["b"], h0, c0, reset, dh, dhT, dcT)
            g[idx] = (fp - fm) / (2 * eps)
        return g

    for name, analytic in (("Wx", dWx), ("Wh", dWh), ("b", db), ("x", dx)):
        num = fd(name)
        rel = np.max(np.abs(num - analytic)) / np.max(np.abs(num))
        assert rel < 1e-7, (name, rel)


def test_bptt_matches_torch_autograd():
    T, B, D, H = 6, 3, 5, 7
    x, Wx, Wh, b, h0, c0, reset = _tiny(21, T=T, B=B, D=D, H=H, with_reset=True)
    rng = np.random.default_rng(5)
    dh = rng.standard_normal((T, B, H))
    dhT = rng.standard_normal((B, H))
    dcT = rng.standard_normal((B, H))
    cell, th, tc = _torch_cell_forward(x, Wx, Wh, b, h0, c0, reset)
    J = (torch.from_numpy(dh) * th).sum() + (torch.from_numpy(dhT) * th[-1]).sum() + \
        (torch.from_numpy(dcT) * tc[-1]).sum()
    J.backward()
    h, c, gates = lstm_forward(x, Wx, Wh, b, h0, c0, reset)
    dWx, dWh, db, _ = lstm_bptt(x, Wx, Wh, h0, c0, reset, h, c, gates, dh, dhT, dcT)
    assert np.max(np.abs(dWx - cell.weight_ih.grad.numpy())) < 1e-11
    assert np.max(np.abs(dWh - cell.weight_hh.grad.numpy())) < 1e-11
    assert np.max(np.abs(db - cell.bias_ih.grad.numpy())) < 1e-11


def test_bptt_zero_upstream_gives_zero_gradients():
    x, Wx, Wh, b, h0, c0, reset = _tiny(4, T=5, with_reset=True)
    h, c, gates = lstm_forward(x, Wx, Wh, b, h0, c0, reset)
    dWx, dWh, db, dx = lstm_bptt(x, Wx, Wh, h0, c0, reset, h, c, gates,
                                 np.zeros_like(h), want_dx=True)
    assert not dWx.any() and not dWh.any() and not db.any() and not dx.any()


def test_bptt_truncation_no_gradient_into_start_state():
    # Changing h0 only through a reset at t = 0 must not change anything.
    x, Wx, Wh, b, h0, c0, _ = _tiny(6, T=3)
    reset = np.zeros((3, 2), np.uint8)
    reset[0, :] = 1
    rng = np.random.default_rng(1)
    dh = rng.standard_normal((3, 2, 4))
    outs = []
    for hh in (h0, 3 * h0 - 1):
        h, c, gates = lstm_forward(x, Wx, Wh, b, hh, c0, reset)
        outs.append(lstm_bptt(x, Wx, Wh, hh, c0, reset, h, c, gates, dh)[:3])
    for a, bb in zip(*outs):
        assert np.array_equal(a, bb)


def test_store_rounds_at_the_storage_points():
    """With store = bf16 rounding, h and the saved gates are bf16 values, the
    recurrence reads the rounded h, and the cell state is built from the exact
    gates."""
    from oracle.bf16 import round_to_bf16
    rng = np.random.default_rng(11)
    T, B, D, H = 2, 3, 5, 4
    x = rng.standard_normal((T, B, D))
    Wx = rng.standard_normal((4 * H, D)) * 0.5
    Wh = rng.standard_normal((4 * H, H)) * 0.5
    b = rng.standard_normal(4 * H) * 0.1
    h0 = rng.standard_normal((B, H)) * 0.3
    c0 = rng.standard_normal((B, H)) * 0.3
    h, c, gates = lstm_forward(x, Wx, Wh, b, h0, c0, store=round_to_bf16)
    assert np.array_equal(round_to_bf16(h), h)
    assert np.array_equal(round_to_bf16(gates), gates)
    # step 1 by hand from the rounded h_0 and the exact c_0
    a = x[1] @ Wx.T + h[0] @ Wh.T + b
    sig = lambda v: 1.0 / (1.0 + np.exp(-v))
    i, f, g, o = sig(a[:, :H]), sig(a[:, H:2 * H]), np.tanh(a[:, 2 * H:3 * H]), sig(a[:, 3 * H:])
    np.testing.assert_allclose(c[1], f * c[0] + i * g, rtol=1e-14, atol=1e-15)
    np.testing.assert_array_equal(h[1], round_to_bf16(o * np.tanh(c[1])))
    # the first step reads the rounded h0
    a0 = x[0] @ Wx.T + round_to_bf16(h0) @ Wh.T + b
    np.testing.assert_array_equal(gates[0][:, :H], round_to_bf16(sig(a0[:, :H])))
