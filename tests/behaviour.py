"""Behaviour-policy data for full-step tests, computed by the oracle.

The rollout that produced a minibatch ran an older policy; its actions,
log-probabilities and values are inputs of the optimizer step.  Recipe:
perturbed weights theta' = theta + N(0, sigma^2); the oracle runs the LSTM
with theta' over every sample from its stored state, samples actions with the
Gumbel-max sampler (seed 1, counter 0), and takes logp_old and the values V
from theta'.  The bootstrap value after each segment is one more theta' step
from the final state of the segment's last sample on the input x_boot.
"""
import numpy as np

from oracle.gae import segments_to_samples
from oracle.lstm import lstm_forward
from oracle.philox import gumbel_max_sample
from oracle.ppo import heads_forward


def oracle_behaviour(inp):
    cfg = inp["cfg"]
    T, B, H, L, S = cfg.T, cfg.B, cfg.H, cfg.L, cfg.S
    J = L // T
    th = {k: inp[k].astype(np.float64) + inp["noise_" + k] for k in ("Wx", "Wh", "b", "Wp", "bp")}
    zeros = np.zeros((L, S))
    _, _, reset = segments_to_samples(zeros, zeros, inp["dones"], T)
    h, c, _ = lstm_forward(inp["x"], th["Wx"], th["Wh"], th["b"], inp["h0"], inp["c0"], reset)
    N = T * B
    z = heads_forward(h.reshape(N, H), th["Wp"], th["bp"])
    act, logp, val, _ = gumbel_max_sample(z, cfg.head_sizes, seed=1, counter=0)
    val = val.reshape(T, B)
    values = np.empty((L + 1, S))
    for s in range(S):
        for j in range(J):
            values[T * j:T * j + T, s] = val[:, s * J + j]
    last = np.arange(S) * J + (J - 1)
    hb, cb, _ = lstm_forward(inp["x_boot"][None], th["Wx"], th["Wh"], th["b"], h[T - 1, last], c[T - 1, last])
    values[L] = heads_forward(hb[0], th["Wp"], th["bp"])[:, -1]
    return {"act": act, "logp_old": logp.astype(np.float32), "values": values.astype(np.float32)}
