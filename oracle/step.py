"""One full PPO optimizer step composed from the oracle parts, in fp64.

Test infrastructure (see the package docstring).

Order of the step (subsection "Optimizing the Policy"): advantages by GAE over
each rollout segment; forward pass of the LSTM over each 16-step sample from
its stored start state; heads, PPO loss and its gradient; truncated BPTT;
Adam with the per-parameter clip.

Parameters are passed as a dict {Wx, Wh, b, Wp, bp}; the caller's flat
parameter vector order is (Wx, Wh, b, Wp, bp), each row-major.
"""
import numpy as np

from .precision import F

from . import adam as _adam
from . import gae as _gae
from . import lstm as _lstm
from . import ppo as _ppo
from .bf16 import round_to_bf16

PARAM_ORDER = ("Wx", "Wh", "b", "Wp", "bp")


def flatten(params):
    return np.concatenate([np.asarray(params[k], F()).ravel() for k in PARAM_ORDER])


def unflatten(flat, like):
    out, o = {}, 0
    for k in PARAM_ORDER:
        n = np.asarray(like[k]).size
        out[k] = np.asarray(flat[o:o + n]).reshape(np.asarray(like[k]).shape)
        o += n
    return out


def gemm_inputs(params, x, bf16):
    """The GEMM operands as the device sees them: bf16-rounded on the bf16 path."""
    if not bf16:
        return (np.asarray(params["Wx"], F()), np.asarray(params["Wh"], F()),
                np.asarray(params["Wp"], F()), np.asarray(x, F()))
    return (round_to_bf16(params["Wx"]), round_to_bf16(params["Wh"]),
            round_to_bf16(params["Wp"]), round_to_bf16(x))


def ppo_step(params, x, h0, c0, rewards, dones, values, act, logp_old,
             head_sizes, T, gamma=0.998, lam=0.95, clip_eps=0.2, vf_coef=1.0,
             ent_coef=0.01, adam_state=None, lr=5e-5, beta1=0.9, beta2=0.999,
             eps=1e-8, clip_k=5.0, step=1, bf16=False, head_mask=None, store=True):
    """rewards, dones [L, S]; values [L+1, S]; x [T, B, D] with B = S*L/T;
    act [T*B, K]; logp_old [T*B].  Returns a dict with the advantages, the
    loss statistics, each row's joint log-probability, every gradient, and
    the updated parameters/moments.

    bf16 path: the GEMM inputs (x, W_x, W_h, W_p) are bf16-rounded; with
    ``store`` (the default) h, the saved gates and dG are also rounded where
    a bf16 implementation stores them as product operands, and with
    ``store=False`` every intermediate stays fp64 (the plain definition)."""
    adv, ret = _gae.gae(rewards, values, dones, gamma, lam)
    adv_s, ret_s, reset = _gae.segments_to_samples(adv, ret, dones, T)
    Wx, Wh, Wp, xx = gemm_inputs(params, x, bf16)
    b = np.asarray(params["b"], F())
    bp = np.asarray(params["bp"], F())
    Tn, B, _ = xx.shape
    H = Wh.shape[1]

    store = round_to_bf16 if (bf16 and store) else None
    h, c, gates = _lstm.lstm_forward(xx, Wx, Wh, b, h0, c0, reset, store=store)
    N = Tn * B
    stats, dh_rows, dWp, dbp, z = _ppo.ppo_loss_grad(
        h.reshape(N, H), Wp, bp, act, logp_old, adv_s.reshape(N), ret_s.reshape(N),
        head_sizes, clip_eps, vf_coef, ent_coef, head_mask)
    logp_k, _, _ = _ppo.head_logprob_entropy(z, np.asarray(act, np.int64), head_sizes)
    on = np.ones_like(logp_k) if head_mask is None else np.asarray(head_mask, F())
    logpi = np.where(on != 0, logp_k, 0.0).sum(axis=1)
    dWx, dWh, db, _ = _lstm.lstm_bptt(xx, Wx, Wh, h0, c0, reset, h, c, gates,
                                      dh_rows.reshape(Tn, B, H), store=store)
    grads = {"Wx": dWx, "Wh": dWh, "b": db, "Wp": dWp, "bp": dbp}

    p = flatten(params)
    g = flatten(grads)
    if adam_state is None:
        m = np.zeros_like(p)
        v = np.zeros_like(p)
    else:
        m, v = adam_state
    p_new, m_new, v_new = _adam.adam_step(p, m, v, g, lr, beta1, beta2, eps, clip_k, step)
    return {
        "adv": adv, "ret": ret, "adv_s": adv_s, "ret_s": ret_s, "reset": reset,
        "h": h, "c": c, "stats": stats, "logpi": logpi, "grads": grads, "grad_flat": g,
        "params_new": unflatten(p_new, params), "p_new": p_new, "m": m_new, "v": v_new,
    }
