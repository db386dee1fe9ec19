"""One PPO optimizer step on one GPU, sequenced through the C ABI.

The optimizer step of the paper's method (subsection "Optimizing the
Policy"): GAE over each 256-step segment, the cut into 16-step samples, the
LSTM forward pass from each sample's stored state, the heads with the PPO
loss and its gradient, truncated BPTT, and Adam with the per-parameter clip.
This module only allocates device buffers (torch) and calls the library in
order on one stream; all arithmetic runs in libo5's kernels.  On the bf16
path the heads hand their gradient to the backward pass in factored form
(dh = P W^T, o5_ppo_loss_grad_factored and o5_lstm_bptt_factored), so the
[T*B, H] fp32 dh is never stored; the fp32 path passes dh itself.

Parameter storage: one flat fp32 master vector in the order
(W_x, W_h, b, W_p, b_p), each row-major, with a flat bf16 mirror for the bf16
path that the Adam kernel rewrites on every step; gradients use the same
flat layout so Adam is a single call.
"""
import numpy as np
import torch

from . import o5
from .synth import Config

PARAM_ORDER = ("Wx", "Wh", "b", "Wp", "bp")


def param_shapes(cfg: Config):
    H, D = cfg.H, cfg.D
    A1 = sum(cfg.head_sizes) + 1
    return {"Wx": (4 * H, D), "Wh": (4 * H, H), "b": (4 * H,), "Wp": (A1, H), "bp": (A1,)}


def _views(flat, shapes):
    out, o = {}, 0
    for k in PARAM_ORDER:
        n = int(np.prod(shapes[k]))
        out[k] = flat[o:o + n].view(shapes[k])
        o += n
    return out


class PPOStep:
    """Device buffers and the call sequence of one optimizer step."""

    def __init__(self, cfg: Config, device="cuda"):
        assert cfg.L % cfg.T == 0 and cfg.S * (cfg.L // cfg.T) == cfg.B, "B must equal S * L / T"
        self.cfg = cfg
        self.bf16 = cfg.dtype == "bf16"
        self.dt = o5.O5_BF16 if self.bf16 else o5.O5_F32
        T, B, D, H, L, S = cfg.T, cfg.B, cfg.D, cfg.H, cfg.L, cfg.S
        self.N = T * B
        self.heads = tuple(cfg.head_sizes)
        K = len(self.heads)
        f32 = dict(dtype=torch.float32, device=device)
        edt = dict(dtype=torch.bfloat16 if self.bf16 else torch.float32, device=device)
        self.shapes = param_shapes(cfg)
        self.n_params = sum(int(np.prod(s)) for s in self.shapes.values())
        n = self.n_params
        self.p32 = torch.empty(n, **f32)
        self.m = torch.zeros(n, **f32)
        self.v = torch.zeros(n, **f32)
        self.g = torch.empty(n, **f32)
        self.p16 = torch.empty(n, dtype=torch.bfloat16, device=device) if self.bf16 else None
        self.P = _views(self.p32, self.shapes)           # fp32 master views
        self.G = _views(self.g, self.shapes)             # gradient views
        self.W = _views(self.p16, self.shapes) if self.bf16 else self.P   # GEMM-operand views
        # inputs
        self.x = torch.empty((T, B, D), **edt)
        self.h0 = torch.empty((B, H), **f32)
        self.c0 = torch.empty((B, H), **f32)
        self.rewards = torch.empty((L, S), **f32)
        self.dones = torch.empty((L, S), dtype=torch.uint8, device=device)
        self.values = torch.empty((L + 1, S), **f32)
        self.act = torch.empty((self.N, K), dtype=torch.int32, device=device)
        self.logp_old = torch.empty(self.N, **f32)
        # intermediates and outputs
        self.adv = torch.empty((L, S), **f32)
        self.ret = torch.empty((L, S), **f32)
        self.adv_s = torch.empty((T, B), **f32)
        self.ret_s = torch.empty((T, B), **f32)
        self.reset = torch.empty((T, B), dtype=torch.uint8, device=device)
        self.h = torch.empty((T, B, H), **edt)
        self.c = torch.empty((T, B, H), **f32)
        self.gates = torch.empty((T, B, 4 * H), **edt)
        if self.bf16:
            self.ld = o5.o5_ppo_head_grad_ld(H, self.heads)
            self.hgP = torch.empty((self.N, self.ld), dtype=torch.bfloat16, device=device)
            self.hgW = torch.empty((H, self.ld), dtype=torch.bfloat16, device=device)
        else:
            self.dh = torch.empty((self.N, H), **f32)
        self.stats = torch.empty(8, **f32)
        ws = max(o5.o5_lstm_fwd_workspace_bytes(self.dt, T, B, D, H),
                 o5.o5_lstm_bptt_workspace_bytes(self.dt, T, B, D, H),
                 o5.o5_ppo_loss_grad_workspace_bytes(self.dt, self.N, H, self.heads))
        self.ws = torch.empty(ws, dtype=torch.uint8, device=device)
        self.step_count = 0

    # ------------------------------------------------------------- inputs
    def load_params(self, params):
        flat = np.concatenate([np.asarray(params[k], np.float32).ravel() for k in PARAM_ORDER])
        self.p32.copy_(torch.from_numpy(flat))
        self.sync_bf16()

    def sync_bf16(self):
        if self.bf16:
            o5.o5_f32_to_bf16(self.n_params, self.p32, self.p16)

    def load_x(self, x):
        x32 = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(self.x.device)
        if self.bf16:
            o5.o5_f32_to_bf16(x32.numel(), x32, self.x)
        else:
            self.x.copy_(x32)

    def load_rollout(self, h0, c0, rewards, dones, values, act, logp_old):
        for dst, src in ((self.h0, h0), (self.c0, c0), (self.rewards, rewards), (self.values, values),
                         (self.logp_old, logp_old)):
            dst.copy_(torch.from_numpy(np.ascontiguousarray(src, dtype=np.float32)))
        self.dones.copy_(torch.from_numpy(np.ascontiguousarray(dones, dtype=np.uint8)))
        self.act.copy_(torch.from_numpy(np.ascontiguousarray(act, dtype=np.int32)))

    # --------------------------------------------------------------- step
    def run(self, stream=None):
        """One optimizer step; returns nothing (stats stay on the device)."""
        c = self.cfg
        T, B, D, H, L, S = c.T, c.B, c.D, c.H, c.L, c.S
        W, G = self.W, self.G
        self.step_count += 1
        o5.o5_gae(L, S, self.rewards, self.values, self.dones, c.gamma, c.lam, self.adv, self.ret, stream)
        o5.o5_segments_to_samples(L, S, T, self.adv, self.ret, self.dones, self.adv_s, self.ret_s,
                                  self.reset, stream)
        o5.o5_lstm_fwd(self.dt, T, B, D, H, self.x, W["Wx"], W["Wh"], self.P["b"], self.h0, self.c0,
                       self.reset, self.h, self.c, self.gates, self.ws, stream)
        if self.bf16:
            o5.o5_ppo_loss_grad_factored(self.dt, self.N, H, self.heads, self.h, W["Wp"], self.P["bp"], self.act,
                                         self.logp_old, self.adv_s, self.ret_s, None, c.clip_eps, c.vf_coef,
                                         c.ent_coef, self.stats, self.hgP, self.hgW, self.ld, G["Wp"], G["bp"],
                                         self.ws, stream)
            o5.o5_lstm_bptt_factored(self.dt, T, B, D, H, self.x, W["Wx"], W["Wh"], self.h0, self.c0, self.reset,
                                     self.h, self.c, self.gates, self.hgP, self.hgW, self.ld, None, None, G["Wx"],
                                     G["Wh"], G["b"], None, self.ws, stream)
        else:
            o5.o5_ppo_loss_grad(self.dt, self.N, H, self.heads, self.h, W["Wp"], self.P["bp"], self.act,
                                self.logp_old, self.adv_s, self.ret_s, None, c.clip_eps, c.vf_coef, c.ent_coef,
                                self.stats, self.dh, G["Wp"], G["bp"], self.ws, stream)
            o5.o5_lstm_bptt(self.dt, T, B, D, H, self.x, W["Wx"], W["Wh"], self.h0, self.c0, self.reset,
                            self.h, self.c, self.gates, self.dh, None, None, G["Wx"], G["Wh"], G["b"], None,
                            self.ws, stream)
        o5.o5_adam_step(self.n_params, self.p32, self.m, self.v, self.g, self.p16, c.lr, c.beta1, c.beta2,
                        c.adam_eps, c.clip_k, self.step_count, stream)
