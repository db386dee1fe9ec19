"""GPU parity: o5_ppo_loss_grad and o5_policy_sample against the fp64 oracle."""
import numpy as np
import pytest
import torch

from oracle.bf16 import round_to_bf16
from oracle.philox import gumbel_max_sample
from oracle.ppo import STAT_NAMES, head_logprob_entropy, heads_forward, ppo_loss_grad
from paper_1912_06680_amd import o5
from tests.gpu_util import (TOL_BF16, TOL_F32, assert_close, banner, dev, dev_dt, dev_f32, host, need_gpu,
                            workspace)

pytestmark = pytest.mark.gpu

HEADS = (30, 8, 32, 4)
KINKS = (np.log(1.2), np.log(0.8))


def _avail(rng, N, heads, mask):
    """Availability [N, A]: each logit available with probability 0.7, at
    least one per head, the taken action among them; where a head's mask is
    0, one row in three has no available logit at all (an empty head)."""
    off = np.concatenate([[0], np.cumsum(heads)])
    av = rng.random((N, off[-1])) < 0.7
    act = np.zeros((N, len(heads)), np.int32)
    for k, n in enumerate(heads):
        blk = av[:, off[k]:off[k + 1]]
        none = ~blk.any(axis=1)
        blk[none, rng.integers(0, n, none.sum())] = True
        for i in range(N):
            act[i, k] = rng.choice(np.flatnonzero(blk[i]))
        if mask is not None:
            empty = (mask[:, k] == 0) & (rng.random(N) < 1 / 3)
            blk[empty] = False
    return av.astype(np.uint8), act


def _inputs(N, H, heads, seed, bf16, with_mask, with_avail=False, wscale=4.0):
    rng = np.random.Generator(np.random.PCG64(seed))
    A1 = sum(heads) + 1
    bound = 1.0 / np.sqrt(H)
    h = np.tanh(rng.standard_normal((N, H), dtype=np.float32)).astype(np.float32)
    Wp = ((rng.random((A1, H), dtype=np.float32) * 2 - 1) * bound * wscale).astype(np.float32)
    bp = ((rng.random(A1, dtype=np.float32) * 2 - 1) * bound).astype(np.float32)
    act = np.stack([rng.integers(0, n, N) for n in heads], axis=1).astype(np.int32)
    adv = rng.standard_normal(N, dtype=np.float32)
    ret = rng.standard_normal(N, dtype=np.float32)
    mask = (rng.random((N, len(heads))) < 0.8).astype(np.uint8) if with_mask else None
    avail = None
    if with_avail:
        avail, act = _avail(rng, N, heads, mask)
    # behaviour log-probabilities: the oracle's current log-probability shifted
    # by U(-0.4, 0.4), kept >= 0.01 away from the clip kinks log(1.2), log(0.8)
    hh = round_to_bf16(h) if bf16 else h.astype(np.float64)
    ww = round_to_bf16(Wp) if bf16 else Wp.astype(np.float64)
    z = heads_forward(hh, ww, bp)
    logp, _, _ = head_logprob_entropy(z, act, heads, avail)
    m = np.ones_like(logp) if mask is None else mask.astype(np.float64)
    logpi = np.where(m != 0, logp, 0.0).sum(axis=1)
    shift = rng.uniform(-0.4, 0.4, N)
    for kk in KINKS:   # r = exp(-shift); keep -shift away from the kinks
        near = np.abs(-shift - kk) < 0.01
        shift[near] += 0.03
    logp_old = (logpi + shift).astype(np.float32)
    return dict(h=h, Wp=Wp, bp=bp, act=act, adv=adv, ret=ret, mask=mask, avail=avail, logp_old=logp_old, hh=hh,
                ww=ww)


PPO_CASES = [
    ("f32-small", 64, 64, HEADS, False, False, False),
    ("f32-mask-ragged", 1001, 128, (5, 3, 7), False, True, False),
    ("bf16-mid", 4096, 1024, HEADS, True, True, False),
    ("bf16-one-head", 333, 192, (8,), True, False, False),
    # 191 logit columns: three per lane, heads crossing the 64-column lane
    # blocks, and the dWp product without the transposed pair
    ("bf16-wide-heads", 500, 128, (100, 60, 30), True, True, False),
    # availability masks, with empty heads under a zero head mask
    ("f32-avail", 777, 128, HEADS, False, True, True),
    ("bf16-avail-wide", 500, 128, (100, 60, 30), True, True, True),
    ("f32-avail-no-head-mask", 300, 64, (5, 3, 7), False, False, True),
    # a single row; single-logit heads (certain actions)
    ("f32-one-row", 1, 64, HEADS, False, False, False),
    ("bf16-single-logit-heads", 100, 64, (1, 4, 1), True, True, False),
    # the benchmark's shape: N = T B = 16 x 2048 rows of the 4096-unit LSTM
    ("bf16-step-shape", 32768, 4096, HEADS, True, True, False),
    # the largest logit count (A + 1 = 1024: 16 columns per lane, dWp without
    # the transposed pair) and the largest head count
    ("bf16-max-logits", 300, 128, (512, 300, 211), True, True, False),
    ("f32-max-logits-avail", 200, 64, (512, 300, 211), False, True, True),
    ("f32-max-heads", 200, 64, (3, 5, 7, 2, 9, 4, 6, 8), False, True, True),
]


@pytest.mark.parametrize("name,N,H,heads,bf16,with_mask,with_avail", PPO_CASES, ids=[c[0] for c in PPO_CASES])
def test_ppo_loss_grad_matches_oracle(name, N, H, heads, bf16, with_mask, with_avail):
    need_gpu()
    banner(f"ppo {name} N={N} H={H} heads={heads} bf16={bf16} avail={with_avail}")
    inp = _inputs(N, H, heads, seed=N + H, bf16=bf16, with_mask=with_mask, with_avail=with_avail)
    stats_ref, dh_ref, dWp_ref, dbp_ref, _ = ppo_loss_grad(
        inp["hh"], inp["ww"], inp["bp"], inp["act"], inp["logp_old"], inp["adv"], inp["ret"], heads,
        0.2, 1.0, 0.01, inp["mask"], inp["avail"])
    dt = o5.O5_BF16 if bf16 else o5.O5_F32
    A1 = sum(heads) + 1
    stats = torch.empty(8, dtype=torch.float32, device="cuda")
    dh = torch.empty((N, H), dtype=torch.float32, device="cuda")
    dWp = torch.empty((A1, H), dtype=torch.float32, device="cuda")
    dbp = torch.empty(A1, dtype=torch.float32, device="cuda")
    ws = workspace(o5.o5_ppo_loss_grad_workspace_bytes(dt, N, H, heads))
    mask = dev(inp["mask"]) if inp["mask"] is not None else None
    avail = dev(inp["avail"]) if inp["avail"] is not None else None
    o5.o5_ppo_loss_grad(dt, N, H, heads, dev_dt(inp["h"], bf16), dev_dt(inp["Wp"], bf16), dev_f32(inp["bp"]),
                        dev(inp["act"]), dev_f32(inp["logp_old"]), dev_f32(inp["adv"]), dev_f32(inp["ret"]),
                        mask, 0.2, 1.0, 0.01, stats, dh, dWp, dbp, ws, avail=avail)
    tol = TOL_BF16 if bf16 else TOL_F32
    st = host(stats)
    for i, name_ in enumerate(STAT_NAMES):
        ref = stats_ref[name_]
        e = abs(st[i] - ref) / max(abs(ref), 1e-6)
        print(f"    stat {name_}: gpu={st[i]:.6g} ref={ref:.6g} rel={e:.2e}", flush=True)
        assert e <= tol, name_
    assert_close("dh", host(dh), dh_ref, tol)
    assert_close("dWp", host(dWp), dWp_ref, tol)
    assert_close("dbp", host(dbp), dbp_ref, tol)


@pytest.mark.parametrize("bf16", [False, True])
def test_ppo_peaked_softmax(bf16):
    """Logits 35 times the usual scale (spreads above 120 within the first
    head): each softmax is one-hot to fp32 precision, the probabilities of
    the far logits underflow (e^-104 is below the smallest fp32 subnormal),
    and log-probabilities away from the argmax reach a hundred and more
    below zero; the statistics and gradients stay finite and match the
    oracle.  (At 100x the usual scale, log-probabilities near -1000, fp32
    rounding alone puts the fp32 path's policy-gradient statistic 1.0e-4
    from the oracle, the edge of a tolerance meant for logits of order 1.)"""
    need_gpu()
    N, H, heads = 500, 128, HEADS
    banner(f"ppo peaked softmax N={N} H={H} bf16={bf16}")
    inp = _inputs(N, H, heads, seed=29, bf16=bf16, with_mask=True, wscale=140.0)
    z = heads_forward(inp["hh"], inp["ww"], inp["bp"])
    assert np.ptp(z[:, :heads[0]], axis=1).min() > 120
    stats_ref, dh_ref, dWp_ref, dbp_ref, _ = ppo_loss_grad(
        inp["hh"], inp["ww"], inp["bp"], inp["act"], inp["logp_old"], inp["adv"], inp["ret"], heads,
        0.2, 1.0, 0.01, inp["mask"])
    dt = o5.O5_BF16 if bf16 else o5.O5_F32
    A1 = sum(heads) + 1
    stats = torch.empty(8, dtype=torch.float32, device="cuda")
    dh = torch.empty((N, H), dtype=torch.float32, device="cuda")
    dWp = torch.empty((A1, H), dtype=torch.float32, device="cuda")
    dbp = torch.empty(A1, dtype=torch.float32, device="cuda")
    ws = workspace(o5.o5_ppo_loss_grad_workspace_bytes(dt, N, H, heads))
    o5.o5_ppo_loss_grad(dt, N, H, heads, dev_dt(inp["h"], bf16), dev_dt(inp["Wp"], bf16), dev_f32(inp["bp"]),
                        dev(inp["act"]), dev_f32(inp["logp_old"]), dev_f32(inp["adv"]), dev_f32(inp["ret"]),
                        dev(inp["mask"]), 0.2, 1.0, 0.01, stats, dh, dWp, dbp, ws)
    tol = TOL_BF16 if bf16 else TOL_F32
    st = host(stats)
    assert np.isfinite(st).all() and st[7] == 0.0
    for i, name_ in enumerate(STAT_NAMES):
        ref = stats_ref[name_]
        e = abs(st[i] - ref) / max(abs(ref), 1e-6)
        print(f"    stat {name_}: gpu={st[i]:.6g} ref={ref:.6g} rel={e:.2e}", flush=True)
        assert e <= tol, name_
    assert_close("dh", host(dh), dh_ref, tol)
    assert_close("dWp", host(dWp), dWp_ref, tol)
    assert_close("dbp", host(dbp), dbp_ref, tol)


@pytest.mark.parametrize("bf16", [False, True])
def test_ppo_nonfinite_rows_are_counted_on_gpu(bf16):
    """NaN advantages on two rows and an infinite return on a third: the
    device's stats[7] counts exactly those three rows, and the gradient dh
    of every other row (which depends on its own row only) stays finite and
    matches the oracle."""
    need_gpu()
    N, H, heads = 300, 128, HEADS
    banner(f"ppo non-finite rows N={N} H={H} bf16={bf16}")
    inp = _inputs(N, H, heads, seed=17, bf16=bf16, with_mask=True)
    bad = np.array([3, 100, 257])
    inp["adv"][bad[:2]] = np.nan
    inp["ret"][bad[2]] = np.inf
    with np.errstate(invalid="ignore"):
        stats_ref, dh_ref, _, _, _ = ppo_loss_grad(
            inp["hh"], inp["ww"], inp["bp"], inp["act"], inp["logp_old"], inp["adv"], inp["ret"], heads,
            0.2, 1.0, 0.01, inp["mask"])
    assert stats_ref["nonfinite"] == 3.0
    dt = o5.O5_BF16 if bf16 else o5.O5_F32
    A1 = sum(heads) + 1
    stats = torch.empty(8, dtype=torch.float32, device="cuda")
    dh = torch.empty((N, H), dtype=torch.float32, device="cuda")
    dWp = torch.empty((A1, H), dtype=torch.float32, device="cuda")
    dbp = torch.empty(A1, dtype=torch.float32, device="cuda")
    ws = workspace(o5.o5_ppo_loss_grad_workspace_bytes(dt, N, H, heads))
    o5.o5_ppo_loss_grad(dt, N, H, heads, dev_dt(inp["h"], bf16), dev_dt(inp["Wp"], bf16), dev_f32(inp["bp"]),
                        dev(inp["act"]), dev_f32(inp["logp_old"]), dev_f32(inp["adv"]), dev_f32(inp["ret"]),
                        dev(inp["mask"]), 0.2, 1.0, 0.01, stats, dh, dWp, dbp, ws)
    st = host(stats)
    print(f"    nonfinite: gpu={st[7]} oracle={stats_ref['nonfinite']}", flush=True)
    assert st[7] == 3.0
    clean = np.setdiff1d(np.arange(N), bad)
    dh_h = host(dh)
    assert not np.all(np.isfinite(dh_h[bad]))
    assert_close("dh[clean rows]", dh_h[clean], dh_ref[clean], TOL_BF16 if bf16 else TOL_F32)


def test_ppo_ratio_one_invariant_on_gpu():
    """logp_old = logpi makes every ratio 1: pg = -mean(A) and clipfrac = 0."""
    need_gpu()
    banner("ppo ratio=1 invariant")
    N, H = 512, 64
    inp = _inputs(N, H, HEADS, seed=1, bf16=False, with_mask=False)
    z = heads_forward(inp["hh"], inp["ww"], inp["bp"])
    logp, _, _ = head_logprob_entropy(z, inp["act"], HEADS)
    logp_old = logp.sum(axis=1).astype(np.float32)
    stats = torch.empty(8, dtype=torch.float32, device="cuda")
    dh = torch.empty((N, H), dtype=torch.float32, device="cuda")
    dWp = torch.empty((sum(HEADS) + 1, H), dtype=torch.float32, device="cuda")
    dbp = torch.empty(sum(HEADS) + 1, dtype=torch.float32, device="cuda")
    ws = workspace(o5.o5_ppo_loss_grad_workspace_bytes(0, N, H, HEADS))
    o5.o5_ppo_loss_grad(0, N, H, HEADS, dev_f32(inp["h"]), dev_f32(inp["Wp"]), dev_f32(inp["bp"]), dev(inp["act"]),
                        dev_f32(logp_old), dev_f32(inp["adv"]), dev_f32(inp["ret"]), None, 0.2, 1.0, 0.01, stats, dh,
                        dWp, dbp, ws)
    st = host(stats)
    assert abs(st[1] - (-inp["adv"].astype(np.float64).mean())) < 1e-5
    assert st[4] == 0.0 and abs(st[6] - 1.0) < 1e-5


# the largest logit count (A + 1 = 1024) and the largest head count (8)
MAX_LOGITS = (512, 300, 211)
MAX_HEADS = (3, 5, 7, 2, 9, 4, 6, 8)
SAMPLE_CASES = [("f32", 512, 256, False, False, HEADS), ("bf16", 1000, 512, True, False, HEADS),
                ("f32-avail", 600, 128, False, True, HEADS), ("bf16-avail", 700, 256, True, True, HEADS),
                ("bf16-max-logits", 300, 128, True, False, MAX_LOGITS),
                ("f32-max-heads-avail", 300, 64, False, True, MAX_HEADS)]


@pytest.mark.parametrize("name,B,H,bf16,with_avail,heads", SAMPLE_CASES, ids=[c[0] for c in SAMPLE_CASES])
def test_policy_sample_matches_oracle(name, B, H, bf16, with_avail, heads):
    need_gpu()
    banner(f"policy_sample {name} B={B} H={H} heads={heads} avail={with_avail}")
    inp = _inputs(B, H, heads, seed=B, bf16=bf16, with_mask=with_avail, with_avail=with_avail)
    seed, counter = 12345, 7
    act_ref, logp_ref, v_ref, scores = gumbel_max_sample(heads_forward(inp["hh"], inp["ww"], inp["bp"]), heads,
                                                          seed, counter, inp["avail"])
    dt = o5.O5_BF16 if bf16 else o5.O5_F32
    act = torch.empty((B, len(heads)), dtype=torch.int32, device="cuda")
    logp = torch.empty(B, dtype=torch.float32, device="cuda")
    value = torch.empty(B, dtype=torch.float32, device="cuda")
    ws = workspace(o5.o5_policy_sample_workspace_bytes(dt, B, H, heads))
    o5.o5_policy_sample(dt, B, H, heads, dev_dt(inp["h"], bf16), dev_dt(inp["Wp"], bf16), dev_f32(inp["bp"]), seed,
                        counter, act, logp, value, ws,
                        avail=dev(inp["avail"]) if inp["avail"] is not None else None)
    a = act.cpu().numpy()
    if inp["avail"] is not None:
        off = np.concatenate([[0], np.cumsum(heads)])
        for k in range(len(heads)):
            blk = inp["avail"][:, off[k]:off[k + 1]]
            empty = ~blk.any(axis=1)
            assert np.all(a[empty, k] == -1) and np.all(act_ref[empty, k] == -1)
            taken = a[~empty, k]
            assert np.all(blk[~empty][np.arange(taken.size), taken] == 1), "an unavailable action was drawn"
    # unique where the oracle's best score leads the runner-up by > 1e-4
    agree = np.ones(B, bool)
    for k in range(len(heads)):
        s = np.sort(scores[k], axis=1)
        with np.errstate(invalid="ignore"):       # empty heads: -inf - -inf
            clear = ~(s[:, -1] - s[:, -2] <= 1e-4)  # (a single available logit leads by +inf)
        mism = (a[:, k] != act_ref[:, k])
        assert not np.any(mism & clear), f"head {k}: {np.sum(mism & clear)} clear-cut mismatches"
        # near ties: the GPU's choice must be one of the near-maximal logits
        for b in np.where(mism)[0]:
            assert scores[k][b, a[b, k]] >= s[b, -1] - 1e-4
        agree &= ~mism
    assert agree.mean() > 0.99
    tol = TOL_BF16 if bf16 else TOL_F32
    assert_close("logp", host(logp)[agree], logp_ref[agree], tol)
    assert_close("value", host(value), v_ref, tol)


def test_policy_sample_frequencies_follow_softmax():
    """Property at any size: with identical rows, the sampled actions follow
    softmax(z) (chi-square), and another counter gives other draws."""
    need_gpu()
    banner("policy_sample frequencies")
    from scipy import stats as sstats
    B, H = 100000, 64
    rng = np.random.Generator(np.random.PCG64(3))
    heads = (6, 3)
    h_row = rng.standard_normal(H, dtype=np.float32) * 0.5
    Wp = rng.standard_normal((10, H), dtype=np.float32) * 0.3
    bp = np.zeros(10, np.float32)
    h = np.broadcast_to(h_row, (B, H)).copy()
    act = torch.empty((B, 2), dtype=torch.int32, device="cuda")
    logp = torch.empty(B, dtype=torch.float32, device="cuda")
    value = torch.empty(B, dtype=torch.float32, device="cuda")
    ws = workspace(o5.o5_policy_sample_workspace_bytes(0, B, H, heads))
    o5.o5_policy_sample(0, B, H, heads, dev_f32(h), dev_f32(Wp), dev_f32(bp), 99, 0, act, logp, value, ws)
    a = act.cpu().numpy()
    z = Wp.astype(np.float64) @ h_row.astype(np.float64)
    off = 0
    for k, n in enumerate(heads):
        p = np.exp(z[off:off + n] - z[off:off + n].max())
        p /= p.sum()
        counts = np.bincount(a[:, k], minlength=n)
        assert sstats.chisquare(counts, B * p).pvalue > 1e-3
        off += n
