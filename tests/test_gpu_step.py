"""GPU parity of whole PPO optimizer steps (GAE -> samples -> LSTM forward ->
heads + PPO loss -> BPTT -> Adam) against the oracle's composed step, two
steps in a row, and checkpoint/resume equality."""
import numpy as np
import pytest
import torch

from oracle.adam import adam_step
from oracle.step import flatten, ppo_step, unflatten
from paper_1912_06680_amd import o5, synth
from paper_1912_06680_amd.step import PARAM_ORDER, PPOStep
from tests.behaviour import oracle_behaviour
from tests.gpu_util import TOL_BF16, TOL_F32, assert_close, assert_close_both, banner, host, need_gpu

pytestmark = pytest.mark.gpu


def _setup(cfg, seed=0):
    inp = synth.make_inputs(cfg, seed)
    beh = oracle_behaviour(inp)
    st = PPOStep(cfg)
    st.load_params({k: inp[k] for k in PARAM_ORDER})
    st.load_x(inp["x"])
    st.load_rollout(inp["h0"], inp["c0"], inp["rewards"], inp["dones"], beh["values"], beh["act"], beh["logp_old"])
    return inp, beh, st


def _oracle_step(cfg, inp, beh, adam_state=None, step=1, params=None, plain=False):
    """The oracle's composed step.  bf16 path: the storage-point oracle, or
    with ``plain`` the plain definition (bf16-rounded inputs, fp64 else)."""
    params = params or {k: inp[k] for k in PARAM_ORDER}
    return ppo_step(params, inp["x"], inp["h0"], inp["c0"], inp["rewards"], inp["dones"], beh["values"],
                    beh["act"], beh["logp_old"], cfg.head_sizes, cfg.T, cfg.gamma, cfg.lam, cfg.clip_eps,
                    cfg.vf_coef, cfg.ent_coef, adam_state, cfg.lr, cfg.beta1, cfg.beta2, cfg.adam_eps,
                    cfg.clip_k, step, bf16=cfg.dtype == "bf16", store=not plain)


KINK_MARGIN = 0.005   # in log-ratio (5x the largest log-probability difference of the two oracles)


def _oracles_away_from_kinks(cfg, inp, beh, st, bf16, **kw):
    """The oracle's step (and on the bf16 path its plain-definition step),
    with every row whose log-ratio lies within KINK_MARGIN of a clip kink
    log(1 +- eps) in either oracle moved 0.1 away from it.

    At a kink the clipped surrogate has two valid sub-gradients (the
    gradient is discontinuous there), and a row within the arithmetic's own
    uncertainty of it may take either on the device and in the oracle; one
    such row moves a weight gradient by a few percent.  Its behaviour
    log-probability is raised by 0.1 on both sides (on the device through
    st.logp_old), which lowers its log-ratio by 0.1: away from both kinks.
    Returns (ref, ref_plain or None, number of rows moved)."""
    kinks = (np.log1p(cfg.clip_eps), np.log1p(-cfg.clip_eps))
    ref = _oracle_step(cfg, inp, beh, **kw)
    ref_plain = _oracle_step(cfg, inp, beh, plain=True, **kw) if bf16 else None
    near = np.zeros(ref["logpi"].shape, bool)
    for r in (ref, ref_plain):
        if r is not None:
            d = r["logpi"] - beh["logp_old"]
            for k in kinks:
                near |= np.abs(d - k) < KINK_MARGIN
    moved = int(near.sum())
    if ref_plain is not None:
        print(f"    max |logpi| difference between the two oracles: "
              f"{np.max(np.abs(ref['logpi'] - ref_plain['logpi'])):.3e}", flush=True)
    if moved:
        beh = dict(beh)
        beh["logp_old"] = (beh["logp_old"].astype(np.float64) + np.where(near, 0.1, 0.0)).astype(np.float32)
        st.logp_old.copy_(torch.from_numpy(beh["logp_old"]))
        ref = _oracle_step(cfg, inp, beh, **kw)
        ref_plain = _oracle_step(cfg, inp, beh, plain=True, **kw) if bf16 else None
    return ref, ref_plain, moved, beh


def _adam_update(cfg, g_hist):
    """The oracle's Adam update (parameter change) after the gradients
    g_hist[0], g_hist[1], ... from zero moments, as an array."""
    m = np.zeros_like(g_hist[0])
    v = np.zeros_like(g_hist[0])
    p = np.zeros_like(g_hist[0])
    for t, g in enumerate(g_hist, 1):
        p_new, m, v = adam_step(p, m, v, g, cfg.lr, cfg.beta1, cfg.beta2, cfg.adam_eps, cfg.clip_k, t)
        if t == len(g_hist):
            return p_new - p
        p = p_new


def _update_range(cfg, g_hist, deltas):
    """Per element, an enclosure [lo, hi] of the oracle's Adam update (from
    zero moments) over every gradient history whose step-i gradient lies
    within +-deltas[i] of g_hist[i].

    Over one or two steps the clip cannot bind (5 sqrt(v_hat) >= |g|), so
    the update is -lr m_hat / (sqrt(v_hat) + eps) with m_hat = sum w_i g_i
    and v_hat = sum u_i g_i^2, both weight vectors summing to 1.  At step 1
    the update is monotone in g and the ends of the interval give its exact
    range.  Otherwise m_hat moves by at most sum w_i delta_i, sqrt(v_hat) (a
    weighted 2-norm) by at most sqrt(sum u_i delta_i^2), and the quotient's
    range is that of the corners of the resulting rectangle, capped by the
    Cauchy-Schwarz bound |m_hat| / sqrt(v_hat) <= sqrt(sum w_i^2 / u_i)."""
    t = len(g_hist)
    if t == 1:
        a = _adam_update(cfg, [g_hist[0] - deltas[0]])
        b = _adam_update(cfg, [g_hist[0] + deltas[0]])
        return np.minimum(a, b), np.maximum(a, b)
    b1, b2, eps, lr = cfg.beta1, cfg.beta2, cfg.adam_eps, cfg.lr
    w = np.array([(1 - b1) * b1 ** (t - i) for i in range(1, t + 1)]) / (1 - b1 ** t)
    u = np.array([(1 - b2) * b2 ** (t - i) for i in range(1, t + 1)]) / (1 - b2 ** t)
    m = sum(wi * g for wi, g in zip(w, g_hist))
    sv = np.sqrt(sum(ui * g * g for ui, g in zip(u, g_hist)))
    dm = sum(wi * d for wi, d in zip(w, deltas))
    ds = np.sqrt(sum(ui * d * d for ui, d in zip(u, deltas)))
    q = [mm / (ss + eps) for mm in (m - dm, m + dm) for ss in (np.maximum(sv - ds, 0.0), sv + ds)]
    kappa = float(np.sqrt(np.sum(w * w / u)))
    lo = np.maximum(np.minimum.reduce(q), -kappa)
    hi = np.minimum(np.maximum.reduce(q), kappa)
    return -lr * hi, -lr * lo


def _check_update(cfg, tol, label, p_before, p_after, ref_p_new, ref_p_old, g_hist, deltas):
    """Adam's parameter change against the oracle's.

    Adam divides by the root of the second moment, so its update is
    ill-conditioned in the gradient: at step 1 it is lr g / (|g| + eps),
    nearly lr sign(g), and an element whose gradient lies within the
    gradient's own error of zero may change sign legitimately.  The bound is
    therefore the plain tolerance (tol max|dtheta| plus one fp32 rounding of
    each stored theta) plus, per element, how far the oracle's own update
    can move over gradient histories within +-deltas of the oracle's
    (``_update_range``), the delta of a step being, per parameter tensor,
    the largest measured gradient difference in that tensor (which the
    gradient comparison has already held to its tolerance), or 0 for a
    step whose moments both sides took from the oracle.  The elements for which
    that term exceeds the plain tolerance are counted and printed, as are
    those whose error exceeds the plain tolerance; at most 10 % of the
    vector may do the latter (a slip in a bias correction, a moment or the
    step count changes every element's update by a factor, which would put
    nearly all of them outside it)."""
    dref = ref_p_new - ref_p_old
    err = np.abs((p_after - p_before) - dref)
    ulp = np.spacing(np.abs(ref_p_new).astype(np.float32)).astype(np.float64) + \
        np.spacing(np.abs(ref_p_old).astype(np.float32)).astype(np.float64)
    base = tol * np.max(np.abs(dref))
    lo, hi = _update_range(cfg, g_hist, deltas)
    sens = np.maximum(hi - dref, dref - lo)
    exempt = int(np.sum(sens > base))
    frac = err / (base + ulp + sens)
    plain_fail = int(np.sum(err > base + ulp))
    print(f"    adam {label}: max err/bound = {frac.max():.3f}; {exempt} of {err.size} elements "
          f"({100.0 * exempt / err.size:.3f} %) have a gradient-sensitivity term above the plain tolerance, "
          f"{plain_fail} ({100.0 * plain_fail / err.size:.3f} %) exceed the plain tolerance", flush=True)
    assert frac.max() <= 1.0
    assert plain_fail <= 0.1 * err.size


def _tensor_deltas(g_gpu, g_ref, st):
    """Per element: the largest |g_gpu - g_ref| within its parameter tensor."""
    out = np.empty_like(g_ref)
    o = 0
    for k in PARAM_ORDER:
        n = int(np.prod(st.shapes[k]))
        out[o:o + n] = np.max(np.abs(g_gpu[o:o + n] - g_ref[o:o + n]))
        o += n
    return out


def _compare_state(tol, label, st, ref, ref_plain):
    """Gradients against both oracles (bf16) or the fp64 oracle (fp32), then
    Adam's moments: m (linear in the clipped gradient) and sqrt(v) (the
    scale Adam divides by; 1-Lipschitz in the gradients)."""
    for k in PARAM_ORDER:
        if ref_plain is None:
            assert_close(f"grad {k} {label}", host(st.G[k]), ref["grads"][k], tol)
        else:
            assert_close_both(f"grad {k} {label}", host(st.G[k]), ref["grads"][k], ref_plain["grads"][k], tol)
    assert_close(f"m {label}", host(st.m), ref["m"], tol)
    assert_close(f"sqrt(v) {label}", np.sqrt(host(st.v)), np.sqrt(ref["v"]), tol)


def _compare_stats(cfg, tol, st, ref):
    names = ("total", "pg", "vf", "ent", "clipfrac", "approx_kl", "mean_ratio", "nonfinite")
    s = host(st.stats)
    for i, k in enumerate(names):
        r = ref["stats"][k]
        e = abs(s[i] - r) / max(abs(r), 1e-6)
        print(f"    stat {k}: gpu={s[i]:.6g} ref={r:.6g} rel={e:.2e}", flush=True)
        # clipfrac counts rows past a threshold: allow a few rows to flip in bf16
        lim = tol if (k != "clipfrac" or cfg.dtype != "bf16") else max(tol, 8.0 / st.N)
        assert e <= lim or abs(s[i] - r) <= lim, k


@pytest.mark.parametrize("name", ["tiny", "mid", "mid_bf16", "big_bf16"])
def test_full_step_matches_oracle(name):
    """Two optimizer steps in a row on the device, each against the oracle's
    step from the oracle's own state: advantages, the cut into samples, the
    loss statistics, every gradient, Adam's moments and the parameter
    change.  On the bf16 path every gradient is also compared with the plain
    definition (no storage-point rounding) at the same tolerance."""
    need_gpu()
    cfg = synth.CONFIGS[name]
    bf16 = cfg.dtype == "bf16"
    banner(f"full step {name}: B={cfg.B} T={cfg.T} D={cfg.D} H={cfg.H} dtype={cfg.dtype}")
    inp, beh, st = _setup(cfg)
    tol = TOL_BF16 if bf16 else TOL_F32
    ref, ref_plain, moved, beh = _oracles_away_from_kinks(cfg, inp, beh, st, bf16)
    print(f"    {moved} rows moved away from a clip kink", flush=True)
    p0 = host(st.p32)
    st.run()
    p1 = host(st.p32)
    assert_close("adv", host(st.adv), ref["adv"], tol)
    assert_close("adv_s", host(st.adv_s), ref["adv_s"], tol)
    assert np.array_equal(st.reset.cpu().numpy(), ref["reset"])
    _compare_stats(cfg, tol, st, ref)
    _compare_state(tol, "step 1", st, ref, ref_plain)
    g1 = ref["grad_flat"]
    d1 = _tensor_deltas(host(st.g), g1, st)
    _check_update(cfg, tol, "step 1", p0, p1, ref["p_new"], flatten({k: inp[k] for k in PARAM_ORDER}), [g1], [d1])

    # Step 2 from the oracle's step-1 state, as the device stores it (fp32
    # parameters and moments), on both sides: Adam legitimately flips the
    # update of elements whose gradient is within the gradient's error of
    # zero, and parameters that differ by such flips move a few rows across
    # the clipped surrogate's kinks, where the gradient is discontinuous.
    # (The device's own two steps in a row are compared bitwise with a
    # checkpoint-resume run below.)
    banner(f"full step {name}: second step from the oracle's step-1 state")
    f32 = lambda a: np.asarray(a, np.float32).astype(np.float64)  # noqa: E731
    p1r, m1r, v1r = f32(ref["p_new"]), f32(ref["m"]), f32(ref["v"])
    for dst, src in ((st.p32, p1r), (st.m, m1r), (st.v, v1r)):
        dst.copy_(torch.from_numpy(src.astype(np.float32)))
    st.sync_bf16()
    params1 = unflatten(p1r, {k: inp[k] for k in PARAM_ORDER})
    ref2, ref2_plain, moved, beh = _oracles_away_from_kinks(cfg, inp, beh, st, bf16, adam_state=(m1r, v1r), step=2,
                                                             params=params1)
    print(f"    {moved} rows moved away from a clip kink", flush=True)
    st.run()
    p2 = host(st.p32)
    _compare_stats(cfg, tol, st, ref2)
    _compare_state(tol, "step 2", st, ref2, ref2_plain)
    g2 = ref2["grad_flat"]
    d2 = _tensor_deltas(host(st.g), g2, st)
    _check_update(cfg, tol, "step 2", p1r, p2, ref2["p_new"], p1r, [g1, g2], [np.zeros_like(g1), d2])


def test_two_steps_equal_checkpoint_resume():
    """Two steps in a row == one step, save (p, m, v, step), restore, one step."""
    need_gpu()
    cfg = synth.CONFIGS["tiny"]
    banner("checkpoint/resume equality (tiny)")
    _, _, a = _setup(cfg)
    a.run()
    a.run()
    _, _, b = _setup(cfg)
    b.run()
    ck = {k: getattr(b, k).clone().cpu() for k in ("p32", "m", "v")}
    n = b.step_count
    _, _, c = _setup(cfg)
    for k in ("p32", "m", "v"):
        getattr(c, k).copy_(ck[k].cuda())
    c.sync_bf16()
    c.step_count = n
    c.run()
    for k in ("p32", "m", "v", "g"):
        assert torch.equal(getattr(a, k), getattr(c, k)), k


def test_full_size_step_is_deterministic():
    """The benchmark's step (B = 2048 x T = 16, D = H = 4096, bf16) run twice
    from the same state gives bitwise identical parameters, Adam moments,
    gradients and loss statistics: every reduction has a fixed order."""
    need_gpu()
    cfg = synth.CONFIGS["full4096"]
    banner(f"full-size determinism: B={cfg.B} T={cfg.T} D={cfg.D} H={cfg.H} {cfg.dtype}")
    inp = synth.make_inputs(cfg, 0)
    rng = np.random.Generator(np.random.PCG64(3))
    N = cfg.T * cfg.B
    act = np.stack([rng.integers(0, n, N) for n in cfg.head_sizes], axis=1).astype(np.int32)
    logp_old = (rng.standard_normal(N) - 8.0).astype(np.float32)
    values = rng.standard_normal((cfg.L + 1, cfg.S)).astype(np.float32)
    st = PPOStep(cfg)
    st.load_x(inp["x"])
    st.load_rollout(inp["h0"], inp["c0"], inp["rewards"], inp["dones"], values, act, logp_old)
    outs = []
    for _ in range(2):
        st.load_params({k: inp[k] for k in PARAM_ORDER})
        st.m.zero_()
        st.v.zero_()
        st.step_count = 0
        st.run()
        torch.cuda.synchronize()
        outs.append({k: getattr(st, k).clone() for k in ("p32", "m", "v", "g", "stats")})
    for k in outs[0]:
        assert torch.equal(outs[0][k], outs[1][k]), k
    assert torch.isfinite(outs[0]["stats"]).all()


def test_full_size_backward_is_additive_over_samples():
    """At the benchmark's shape (B = 2048 x T = 16, D = H = 4096, bf16, in the
    launch configuration bench.py times) the weight gradients are a sum over
    samples, a property that holds at any size: the step's backward pass over
    all 2048 samples equals the sum of the same call over samples 0..1023
    and 1024..2047 (each from the step's own forward outputs and factored
    head gradient), up to the order of the fp32 sums.  The halves run in
    another launch configuration (another K split of the recurrent product,
    half the weight-gradient product's K), and the B = 1024 backward pass is
    compared with the oracle in tests/test_gpu_lstm.py."""
    need_gpu()
    cfg = synth.CONFIGS["full4096"]
    T, B, D, H = cfg.T, cfg.B, cfg.D, cfg.H
    banner(f"full-size additivity over samples: B={B} T={T} D={D} H={H} {cfg.dtype}")
    inp = synth.make_inputs(cfg, 0)
    rng = np.random.Generator(np.random.PCG64(4))
    N = T * B
    act = np.stack([rng.integers(0, n, N) for n in cfg.head_sizes], axis=1).astype(np.int32)
    logp_old = (rng.standard_normal(N) - 8.0).astype(np.float32)
    values = rng.standard_normal((cfg.L + 1, cfg.S)).astype(np.float32)
    st = PPOStep(cfg)
    st.load_x(inp["x"])
    st.load_rollout(inp["h0"], inp["c0"], inp["rewards"], inp["dones"], values, act, logp_old)
    st.load_params({k: inp[k] for k in PARAM_ORDER})
    st.run()
    st.load_params({k: inp[k] for k in PARAM_ORDER})   # the weights the step's passes used
    torch.cuda.synchronize()
    full = {k: st.G[k].clone() for k in ("Wx", "Wh", "b")}
    Bh = B // 2
    ws = torch.empty(o5.o5_lstm_bptt_workspace_bytes(st.dt, T, Bh, D, H), dtype=torch.uint8, device="cuda")
    P3 = st.hgP.view(T, B, st.ld)
    total = None
    for half in (slice(0, Bh), slice(Bh, B)):
        part = {"Wx": torch.empty((4 * H, D), device="cuda"), "Wh": torch.empty((4 * H, H), device="cuda"),
                "b": torch.empty(4 * H, device="cuda")}
        o5.o5_lstm_bptt_factored(st.dt, T, Bh, D, H, st.x[:, half].contiguous(), st.W["Wx"], st.W["Wh"],
                                 st.h0[half].contiguous(), st.c0[half].contiguous(), st.reset[:, half].contiguous(),
                                 st.h[:, half].contiguous(), st.c[:, half].contiguous(),
                                 st.gates[:, half].contiguous(), P3[:, half].contiguous().view(T * Bh, st.ld),
                                 st.hgW, st.ld, None, None, part["Wx"], part["Wh"], part["b"], None, ws)
        torch.cuda.synchronize()
        total = part if total is None else {k: total[k] + part[k] for k in total}
    for k in ("Wx", "Wh", "b"):
        err = float((total[k] - full[k]).abs().max() / full[k].abs().max())
        print(f"    d{k}: max|sum of halves - full| / max|full| = {err:.2e}", flush=True)
        assert err <= 1e-3, k

