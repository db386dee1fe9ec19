"""Python binding of libo5 (ctypes).

Argument marshalling only: every function below has the name of the C entry
point it calls, takes torch tensors (device memory) where the C call takes
device pointers, and raises ``O5Error`` when the call returns a nonzero
status.  No computation happens here; if ``libo5.so`` has not been built the
first call raises instead of falling back to anything else.

Default stream: the current torch stream of the current device.
"""
import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libo5.so")

O5_F32 = 0
O5_BF16 = 1

EXPORTED = (
    "o5_version", "o5_status_str", "o5_last_error",
    "o5_lstm_fwd_workspace_bytes", "o5_lstm_fwd",
    "o5_lstm_bptt_workspace_bytes", "o5_lstm_bptt", "o5_lstm_bptt_factored",
    "o5_gae", "o5_segments_to_samples",
    "o5_reward_process_workspace_bytes", "o5_reward_process",
    "o5_obs_normalize_workspace_bytes", "o5_obs_normalize", "o5_prelstm_fwd",
    "o5_prelstm_bwd_workspace_bytes", "o5_prelstm_bwd",
    "o5_ppo_loss_grad_workspace_bytes", "o5_ppo_loss_grad", "o5_ppo_head_grad_ld", "o5_ppo_loss_grad_factored",
    "o5_adam_step",
    "o5_policy_sample_workspace_bytes", "o5_policy_sample", "o5_policy_sample_static",
    "o5_f32_to_bf16",
    "o5_param_count", "o5_surgery_widen", "o5_surgery_fold_input",
    "o5_ktimer_enable", "o5_ktimer_enable_sites", "o5_ktimer_read", "o5_ktimer_site_name",
)

KTIMER_SITES = ("lstm_fwd_gemm", "lstm_fwd_cell", "lstm_dh_gemm", "lstm_bwd_cell", "lstm_dw_gemm",
                "lstm_dx_gemm", "ppo_loss_grad", "adam_step", "gae", "policy_sample", "reward_process",
                "obs_normalize", "prelstm_fwd", "prelstm_bwd", "lstm_fwd_call")


class O5Error(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn} failed with status {status}: {msg}")
        self.status = status


class PpoHp(ctypes.Structure):
    _fields_ = [("clip_eps", ctypes.c_float), ("vf_coef", ctypes.c_float), ("ent_coef", ctypes.c_float)]


class AdamHp(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("clip_k", ctypes.c_float)]


class UnitHead(ctypes.Structure):
    _fields_ = [("head", ctypes.c_int), ("d", ctypes.c_int), ("Wq", ctypes.c_void_p), ("bq", ctypes.c_void_p),
                ("E", ctypes.c_void_p), ("dWq", ctypes.c_void_p), ("dbq", ctypes.c_void_p)]


def unit_head(head, d, Wq, bq, E, dWq=None, dbq=None):
    """An o5_unit_head over torch tensors (keep the tensors alive for the call)."""
    return UnitHead(int(head), int(d), _p(Wq), _p(bq), _p(E), _p(dWq), _p(dbq))


def _unit(u):
    return None if u is None else ctypes.byref(u)


class RewardHp(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_float), ("decay_base", ctypes.c_float), ("decay_minutes", ctypes.c_float),
                ("eps", ctypes.c_float)]


_vp = ctypes.c_void_p
_i = ctypes.c_int
_sz = ctypes.c_size_t
_f = ctypes.c_float
_u64 = ctypes.c_uint64

_SIGS = {
    "o5_version": (_i, []),
    "o5_status_str": (ctypes.c_char_p, [_i]),
    "o5_last_error": (ctypes.c_char_p, []),
    "o5_lstm_fwd_workspace_bytes": (_sz, [_i, _i, _i, _i, _i]),
    "o5_lstm_fwd": (_i, [_i, _i, _i, _i, _i] + [_vp] * 11 + [_sz, _vp]),
    "o5_lstm_bptt_workspace_bytes": (_sz, [_i, _i, _i, _i, _i]),
    "o5_lstm_bptt": (_i, [_i, _i, _i, _i, _i] + [_vp] * 17 + [_sz, _vp]),
    "o5_lstm_bptt_factored": (_i, [_i, _i, _i, _i, _i] + [_vp] * 11 + [_i] + [_vp] * 7 + [_sz, _vp]),
    "o5_gae": (_i, [_i, _i, _vp, _vp, _vp, _f, _f, _vp, _vp, _vp]),
    "o5_segments_to_samples": (_i, [_i, _i, _i] + [_vp] * 6 + [_vp]),
    "o5_reward_process_workspace_bytes": (_sz, [_i, _i]),
    "o5_reward_process": (_i, [_i, _i, _vp, _vp, _vp, RewardHp, _vp, _vp, _vp, _sz, _vp]),
    "o5_obs_normalize_workspace_bytes": (_sz, [_i, _i]),
    "o5_obs_normalize": (_i, [_i, _i, _i, _vp, _vp, _f, _f, _vp, _vp, _sz, _vp]),
    "o5_prelstm_fwd": (_i, [_i, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp, _vp]),
    "o5_prelstm_bwd_workspace_bytes": (_sz, [_i, _i, _i, _i, _i]),
    "o5_prelstm_bwd": (_i, [_i, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "o5_ppo_loss_grad_workspace_bytes": (_sz, [_i, _i, _i, _i, _vp, _vp]),
    "o5_ppo_loss_grad": (_i, [_i, _i, _i, _i, _vp] + [_vp] * 10 + [PpoHp] + [_vp] * 5 + [_sz, _vp]),
    "o5_ppo_head_grad_ld": (_i, [_i, _i, _vp, _vp]),
    "o5_ppo_loss_grad_factored": (_i, [_i, _i, _i, _i, _vp] + [_vp] * 10 + [PpoHp] + [_vp] * 3 + [_i] + [_vp] * 3
                                  + [_sz, _vp]),
    "o5_adam_step": (_i, [_sz, _vp, _vp, _vp, _vp, _vp, AdamHp, _i, _vp]),
    "o5_policy_sample_workspace_bytes": (_sz, [_i, _i, _i, _i, _vp, _vp]),
    "o5_policy_sample": (_i, [_i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp, _vp, _u64, _u64, _vp, _vp, _vp, _vp, _sz,
                              _vp]),
    "o5_policy_sample_static": (_i, [_i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp, _vp, _u64, _u64, _vp, _vp, _vp,
                                     _vp]),
    "o5_f32_to_bf16": (_i, [_sz, _vp, _vp, _vp]),
    "o5_param_count": (_sz, [_i, _i, _i]),
    "o5_surgery_widen": (_i, [_i, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp, _vp, _f, _u64, _vp]),
    "o5_surgery_fold_input": (_i, [_i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "o5_ktimer_enable": (_i, [_i]),
    "o5_ktimer_enable_sites": (_i, [ctypes.c_uint]),
    "o5_ktimer_read": (_i, [_i, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int)]),
    "o5_ktimer_site_name": (ctypes.c_char_p, [_i]),
}

_lib = None


def lib():
    """The loaded libo5 (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "or `python -m paper_1912_06680_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def _p(t):
    """Device pointer of a tensor (None -> NULL)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(fn, status):
    if status != 0:
        msg = lib().o5_last_error().decode()
        raise O5Error(fn, status, msg)


def _ws(ws):
    if ws is None:
        return None, 0
    return ws.data_ptr(), ws.numel() * ws.element_size()


def _heads(head_sizes):
    arr = (ctypes.c_int * len(head_sizes))(*[int(n) for n in head_sizes])
    return arr


def o5_version():
    return lib().o5_version()


def o5_status_str(status):
    return lib().o5_status_str(status).decode()


def o5_last_error():
    return lib().o5_last_error().decode()


def o5_lstm_fwd_workspace_bytes(dt, T, B, D, H):
    return lib().o5_lstm_fwd_workspace_bytes(dt, T, B, D, H)


def o5_lstm_fwd(dt, T, B, D, H, x, Wx, Wh, b, h0, c0, reset, h, c, gates, ws, stream=None):
    wp, wn = _ws(ws)
    _check("o5_lstm_fwd", lib().o5_lstm_fwd(
        dt, T, B, D, H, _p(x), _p(Wx), _p(Wh), _p(b), _p(h0), _p(c0), _p(reset),
        _p(h), _p(c), _p(gates), wp, wn, _stream(stream)))


def o5_lstm_bptt_workspace_bytes(dt, T, B, D, H):
    return lib().o5_lstm_bptt_workspace_bytes(dt, T, B, D, H)


def o5_lstm_bptt(dt, T, B, D, H, x, Wx, Wh, h0, c0, reset, h, c, gates, dh, dhT, dcT,
                 dWx, dWh, db, dx, ws, stream=None):
    wp, wn = _ws(ws)
    _check("o5_lstm_bptt", lib().o5_lstm_bptt(
        dt, T, B, D, H, _p(x), _p(Wx), _p(Wh), _p(h0), _p(c0), _p(reset), _p(h), _p(c),
        _p(gates), _p(dh), _p(dhT), _p(dcT), _p(dWx), _p(dWh), _p(db), _p(dx), wp, wn,
        _stream(stream)))


def o5_lstm_bptt_factored(dt, T, B, D, H, x, Wx, Wh, h0, c0, reset, h, c, gates, P, W, ld, dhT, dcT,
                          dWx, dWh, db, dx, ws, stream=None):
    wp, wn = _ws(ws)
    _check("o5_lstm_bptt_factored", lib().o5_lstm_bptt_factored(
        dt, T, B, D, H, _p(x), _p(Wx), _p(Wh), _p(h0), _p(c0), _p(reset), _p(h), _p(c),
        _p(gates), _p(P), _p(W), int(ld), _p(dhT), _p(dcT), _p(dWx), _p(dWh), _p(db), _p(dx), wp, wn,
        _stream(stream)))


def o5_gae(L, S, r, v, done, gamma, lam, adv, ret, stream=None):
    _check("o5_gae", lib().o5_gae(L, S, _p(r), _p(v), _p(done), float(gamma), float(lam),
                                  _p(adv), _p(ret), _stream(stream)))


def o5_segments_to_samples(L, S, T, adv, ret, done, adv_s, ret_s, reset, stream=None):
    _check("o5_segments_to_samples", lib().o5_segments_to_samples(
        L, S, T, _p(adv), _p(ret), _p(done), _p(adv_s), _p(ret_s), _p(reset), _stream(stream)))


def o5_reward_process_workspace_bytes(L, G):
    return lib().o5_reward_process_workspace_bytes(L, G)


def o5_reward_process(L, G, shaped, outcome, game_time, tau, decay_base, decay_minutes, eps, stats, r, ws,
                      stream=None):
    wp, wn = _ws(ws)
    hp = RewardHp(tau, decay_base, decay_minutes, eps)
    _check("o5_reward_process", lib().o5_reward_process(L, G, _p(shaped), _p(outcome), _p(game_time), hp,
                                                        _p(stats), _p(r), wp, wn, _stream(stream)))


def o5_obs_normalize_workspace_bytes(N, Do):
    return lib().o5_obs_normalize_workspace_bytes(N, Do)


def o5_obs_normalize(dt, N, Do, obs, stats, clip, eps, o, ws, stream=None):
    wp, wn = _ws(ws)
    _check("o5_obs_normalize", lib().o5_obs_normalize(dt, N, Do, _p(obs), _p(stats), float(clip), float(eps), _p(o),
                                                      wp, wn, _stream(stream)))


def o5_prelstm_fwd(dt, T, B, Do, D, o, W, b, y, x, stream=None):
    _check("o5_prelstm_fwd", lib().o5_prelstm_fwd(dt, T, B, Do, D, _p(o), _p(W), _p(b), _p(y), _p(x),
                                                  _stream(stream)))


def o5_prelstm_bwd_workspace_bytes(dt, T, B, Do, D):
    return lib().o5_prelstm_bwd_workspace_bytes(dt, T, B, Do, D)


def o5_prelstm_bwd(dt, T, B, Do, D, o, y, dx, dW, db, ws, stream=None):
    wp, wn = _ws(ws)
    _check("o5_prelstm_bwd", lib().o5_prelstm_bwd(dt, T, B, Do, D, _p(o), _p(y), _p(dx), _p(dW), _p(db), wp, wn,
                                                  _stream(stream)))


def o5_ppo_loss_grad_workspace_bytes(dt, N, H, head_sizes, unit=None):
    return lib().o5_ppo_loss_grad_workspace_bytes(dt, N, H, len(head_sizes), _heads(head_sizes), _unit(unit))


def o5_ppo_loss_grad(dt, N, H, head_sizes, h, Wp, bp, act, logp_old, adv, ret, head_mask,
                     clip_eps, vf_coef, ent_coef, stats, dh, dWp, dbp, ws, stream=None, avail=None, unit=None):
    wp, wn = _ws(ws)
    hp = PpoHp(clip_eps, vf_coef, ent_coef)
    _check("o5_ppo_loss_grad", lib().o5_ppo_loss_grad(
        dt, N, H, len(head_sizes), _heads(head_sizes), _p(h), _p(Wp), _p(bp), _p(act),
        _p(logp_old), _p(adv), _p(ret), _p(head_mask), _p(avail), _unit(unit), hp, _p(stats), _p(dh), _p(dWp),
        _p(dbp), wp, wn, _stream(stream)))


def o5_ppo_head_grad_ld(H, head_sizes, unit=None):
    return lib().o5_ppo_head_grad_ld(H, len(head_sizes), _heads(head_sizes), _unit(unit))


def o5_ppo_loss_grad_factored(dt, N, H, head_sizes, h, Wp, bp, act, logp_old, adv, ret, head_mask,
                              clip_eps, vf_coef, ent_coef, stats, P, W, ld, dWp, dbp, ws, stream=None,
                              avail=None, unit=None):
    wp, wn = _ws(ws)
    hp = PpoHp(clip_eps, vf_coef, ent_coef)
    _check("o5_ppo_loss_grad_factored", lib().o5_ppo_loss_grad_factored(
        dt, N, H, len(head_sizes), _heads(head_sizes), _p(h), _p(Wp), _p(bp), _p(act),
        _p(logp_old), _p(adv), _p(ret), _p(head_mask), _p(avail), _unit(unit), hp, _p(stats), _p(P), _p(W),
        int(ld), _p(dWp), _p(dbp), wp, wn, _stream(stream)))


def o5_adam_step(n, p, m, v, g, p_bf16, lr, beta1, beta2, eps, clip_k, step, stream=None):
    hp = AdamHp(lr, beta1, beta2, eps, clip_k)
    _check("o5_adam_step", lib().o5_adam_step(n, _p(p), _p(m), _p(v), _p(g), _p(p_bf16), hp,
                                              int(step), _stream(stream)))


def o5_policy_sample_workspace_bytes(dt, B, H, head_sizes, unit=None):
    return lib().o5_policy_sample_workspace_bytes(dt, B, H, len(head_sizes), _heads(head_sizes), _unit(unit))


def o5_policy_sample(dt, B, H, head_sizes, h, Wp, bp, seed, counter, act, logp, value, ws,
                     stream=None, avail=None, unit=None):
    wp, wn = _ws(ws)
    _check("o5_policy_sample", lib().o5_policy_sample(
        dt, B, H, len(head_sizes), _heads(head_sizes), _p(h), _p(Wp), _p(bp), _p(avail), _unit(unit), int(seed),
        int(counter), _p(act), _p(logp), _p(value), wp, wn, _stream(stream)))


def o5_policy_sample_static(dt, B, H, head_sizes, h, Wp, bp, seed, counter, act, logp, value, stream=None,
                            avail=None, unit=None):
    _check("o5_policy_sample_static", lib().o5_policy_sample_static(
        dt, B, H, len(head_sizes), _heads(head_sizes), _p(h), _p(Wp), _p(bp), _p(avail), _unit(unit), int(seed),
        int(counter), _p(act), _p(logp), _p(value), _stream(stream)))


def o5_param_count(D, H, A1):
    return lib().o5_param_count(D, H, A1)


def o5_surgery_widen(D, H, A1, D2, H2, p_old, m_old, v_old, p_new, m_new, v_new, scale, seed, stream=None):
    _check("o5_surgery_widen", lib().o5_surgery_widen(D, H, A1, D2, H2, _p(p_old), _p(m_old), _p(v_old), _p(p_new),
                                                      _p(m_new), _p(v_new), float(scale), int(seed),
                                                      _stream(stream)))


def o5_surgery_fold_input(D, H, A1, Dk, E, p_old, m_old, v_old, p_new, m_new, v_new, stream=None):
    _check("o5_surgery_fold_input", lib().o5_surgery_fold_input(D, H, A1, Dk, _p(E), _p(p_old), _p(m_old),
                                                                _p(v_old), _p(p_new), _p(m_new), _p(v_new),
                                                                _stream(stream)))


def o5_f32_to_bf16(n, src, dst, stream=None):
    _check("o5_f32_to_bf16", lib().o5_f32_to_bf16(n, _p(src), _p(dst), _stream(stream)))


def o5_ktimer_enable(on):
    _check("o5_ktimer_enable", lib().o5_ktimer_enable(1 if on else 0))


def o5_ktimer_enable_sites(names):
    """Record only the named sites (an empty list stops recording)."""
    mask = 0
    for nm in names:
        mask |= 1 << KTIMER_SITES.index(nm)
    _check("o5_ktimer_enable_sites", lib().o5_ktimer_enable_sites(mask))


def o5_ktimer_read(site):
    """(total device milliseconds, launches) recorded for one site."""
    t = ctypes.c_double(0.0)
    n = ctypes.c_int(0)
    _check("o5_ktimer_read", lib().o5_ktimer_read(int(site), ctypes.byref(t), ctypes.byref(n)))
    return t.value, n.value


def o5_ktimer_site_name(site):
    return lib().o5_ktimer_site_name(int(site)).decode()
