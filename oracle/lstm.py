"""Single-layer LSTM forward pass and truncated BPTT, in fp64.

Test infrastructure (see the package docstring).

The policy is a single-layer 4096-unit LSTM of the forget-gate kind the paper
cites (Gers et al. 1999), section "Training System", subsection "Playing Dota
using AI".  Gradients are computed by truncated backpropagation through time
over samples of 16 timesteps that start from the LSTM state stored with the
rollout, subsection "Optimizing the Policy".

Readings where the paper is silent:
* no peepholes, one bias vector, gate order (i, f, g, o) along the 4H axis,
  exact logistic sigmoid and tanh;
* ``reset[t, b] = 1`` zeroes the carried state (h, c) before step t of row b
  (an episode boundary inside a sample);
* truncation: no gradient flows into the stored start state h0, c0.

Layouts are time-major: x [T, B, D], h and c [T, B, H], gates [T, B, 4H].
W_x is [4H, D] and W_h is [4H, H]: row g*H + j holds gate g of unit j.

Optional ``store``: a rounding function (e.g. to bf16) applied where a
reduced-precision implementation stores a tensor that a later product reads:
the hidden state (fed back, returned, and used by the weight gradient), the
saved gates, and the gate-gradient dG as an operand of the recurrent and
weight-gradient products.  The cell state, the bias gradient and all
arithmetic stay fp64.  Without it every value is fp64.
"""
import numpy as np

from .precision import F


def sigmoid(a):
    """Logistic function, evaluated without overflow for either sign."""
    a = np.asarray(a, dtype=F())
    out = np.empty_like(a)
    pos = a >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-a[pos]))
    e = np.exp(a[~pos])
    out[~pos] = e / (1.0 + e)
    return out


def _keep(reset, t, B):
    if reset is None:
        return np.ones((B, 1), F())
    return 1.0 - np.asarray(reset[t], dtype=F()).reshape(B, 1)


def _identity(a):
    return a


def lstm_forward(x, Wx, Wh, b, h0, c0, reset=None, store=None):
    """Run T steps of the LSTM.

    Returns (h [T,B,H], c [T,B,H], gates [T,B,4H]) where ``gates`` holds the
    post-activation values (i, f, g, o) that backpropagation needs.  With
    ``store``, h and the saved gates are stored through it (the cell state is
    computed from the exact gates) and the recurrent input is the stored h.
    """
    store = store or _identity
    x = np.asarray(x, F())
    Wx = np.asarray(Wx, F())
    Wh = np.asarray(Wh, F())
    b = np.asarray(b, F())
    T, B, _ = x.shape
    H = Wh.shape[1]
    h = np.empty((T, B, H), F())
    c = np.empty((T, B, H), F())
    gates = np.empty((T, B, 4 * H), F())
    h_prev = store(np.asarray(h0, F()))
    c_prev = np.asarray(c0, F())
    for t in range(T):
        keep = _keep(reset, t, B)
        h_tilde = keep * h_prev
        c_tilde = keep * c_prev
        a = x[t] @ Wx.T + h_tilde @ Wh.T + b
        i = sigmoid(a[:, 0 * H:1 * H])
        f = sigmoid(a[:, 1 * H:2 * H])
        g = np.tanh(a[:, 2 * H:3 * H])
        o = sigmoid(a[:, 3 * H:4 * H])
        c[t] = f * c_tilde + i * g
        h[t] = store(o * np.tanh(c[t]))
        gates[t] = store(np.concatenate([i, f, g, o], axis=1))
        h_prev, c_prev = h[t], c[t]
    return h, c, gates


def lstm_bptt(x, Wx, Wh, h0, c0, reset, h, c, gates, dh, dhT=None, dcT=None,
              want_dx=False, store=None):
    """Truncated BPTT through the T steps of ``lstm_forward``.

    The objective differentiated is
        J = sum_t <dh[t], h[t]> + <dhT, h[T-1]> + <dcT, c[T-1]>,
    i.e. ``dh`` holds the gradient arriving at every step's output from the
    heads and ``dhT``/``dcT`` the gradient arriving at the final state.
    Nothing flows into h0 or c0.

    With ``store``, h0 enters the weight gradient through it and the gate
    gradient enters every product (dW, dx and the recurrent term) through it;
    the bias gradient sums the exact gate gradient.

    Returns (dWx [4H,D], dWh [4H,H], db [4H], dx [T,B,D] or None).
    """
    store = store or _identity
    x = np.asarray(x, F())
    Wx = np.asarray(Wx, F())
    Wh = np.asarray(Wh, F())
    T, B, D = x.shape
    H = Wh.shape[1]
    dWx = np.zeros_like(Wx)
    dWh = np.zeros_like(Wh)
    db = np.zeros(4 * H, F())
    dx = np.zeros((T, B, D), F()) if want_dx else None

    dh_next = np.zeros((B, H), F()) if dhT is None else np.array(dhT, F())
    dc_next = np.zeros((B, H), F()) if dcT is None else np.array(dcT, F())
    for t in reversed(range(T)):
        keep = _keep(reset, t, B)
        h_prev = store(np.asarray(h0, F())) if t == 0 else h[t - 1]
        c_prev = np.asarray(c0, F()) if t == 0 else c[t - 1]
        h_tilde = keep * h_prev
        c_tilde = keep * c_prev
        i = gates[t][:, 0 * H:1 * H]
        f = gates[t][:, 1 * H:2 * H]
        g = gates[t][:, 2 * H:3 * H]
        o = gates[t][:, 3 * H:4 * H]
        tc = np.tanh(c[t])

        dh_t = dh[t] + dh_next
        do = dh_t * tc
        dc = dc_next + dh_t * o * (1.0 - tc * tc)
        di = dc * g
        dg = dc * i
        df = dc * c_tilde
        dc_tilde = dc * f

        da = np.concatenate([di * i * (1.0 - i),
                             df * f * (1.0 - f),
                             dg * (1.0 - g * g),
                             do * o * (1.0 - o)], axis=1)      # [B, 4H]

        dab = store(da)
        dWx += dab.T @ x[t]
        dWh += dab.T @ h_tilde
        db += da.sum(axis=0)
        if want_dx:
            dx[t] = dab @ Wx

        # gradient into the carried state of step t-1; truncated at t = 0
        dh_next = keep * (dab @ Wh)
        dc_next = keep * dc_tilde
    return dWx, dWh, db, dx
