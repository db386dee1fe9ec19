"""GPU parity: the unit-selection head (appendix "Neural Network
Architecture": unit embeddings carried beside the LSTM choose the unit to
target) in o5_ppo_loss_grad and o5_policy_sample, against the fp64 oracle on
identical seeded inputs."""
import numpy as np
import pytest
import torch

from oracle.bf16 import round_to_bf16
from oracle.philox import gumbel_max_sample
from oracle.ppo import STAT_NAMES, head_logprob_entropy, head_offsets, heads_forward, ppo_loss_grad, unit_logits
from paper_1912_06680_amd import o5
from tests.gpu_util import TOL_BF16, TOL_F32, assert_close, banner, dev, dev_dt, dev_f32, host, need_gpu, workspace

pytestmark = pytest.mark.gpu


def _inputs(N, H, heads, ku, d, seed, bf16, with_avail):
    rng = np.random.Generator(np.random.PCG64(seed))
    A1 = sum(heads) + 1
    bound = 1.0 / np.sqrt(H)
    f = lambda a: np.asarray(a, np.float32)
    h = f(np.tanh(rng.standard_normal((N, H))))
    Wp = f((rng.random((A1, H)) * 2 - 1) * bound * 4)
    bp = f((rng.random(A1) * 2 - 1) * bound)
    Wq = f((rng.random((d, H)) * 2 - 1) * bound * 2)
    bq = f((rng.random(d) * 2 - 1) * 0.1)
    E = f(rng.standard_normal((N, heads[ku], d)) / np.sqrt(d))
    act = np.stack([rng.integers(0, n, N) for n in heads], axis=1).astype(np.int32)
    mask = (rng.random((N, len(heads))) < 0.8).astype(np.uint8)
    avail = None
    if with_avail:
        off = head_offsets(heads)
        avail = np.ones((N, off[-1]), np.uint8)
        blk = rng.random((N, heads[ku])) < 0.6
        blk[np.arange(N), act[:, ku]] = True       # units present, the chosen one among them
        avail[:, off[ku]:off[ku + 1]] = blk
    rb = round_to_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    ref = dict(h=rb(h), Wp=rb(Wp), Wq=rb(Wq), E=rb(E))
    unit_ref = dict(head=ku, Wq=ref["Wq"], bq=bq.astype(np.float64), E=ref["E"])
    z = heads_forward(ref["h"], ref["Wp"], bp)
    off = head_offsets(heads)
    _, z[:, off[ku]:off[ku + 1]] = unit_logits(ref["h"], ref["Wq"], bq, ref["E"])
    logp, _, _ = head_logprob_entropy(z, act, heads, avail)
    shift = rng.uniform(-0.3, 0.3, N)
    for kk in (np.log(1.2), np.log(0.8)):
        near = np.abs(-shift - kk) < 0.01
        shift[near] += 0.03
    logp_old = f(np.where(mask != 0, logp, 0.0).sum(axis=1) + shift)
    return dict(h=h, Wp=Wp, bp=bp, Wq=Wq, bq=bq, E=E, act=act, mask=mask, avail=avail, logp_old=logp_old,
                adv=f(rng.standard_normal(N)), ret=f(rng.standard_normal(N)), ref=ref, unit_ref=unit_ref, z=z)


CASES = [
    ("f32-small", 300, 128, (5, 24, 3), 1, 64, False, True),
    ("bf16-small", 300, 128, (5, 24, 3), 1, 64, True, False),
    ("bf16-paper-heads", 2048, 512, (30, 189, 32, 4), 1, 128, True, True),
    ("f32-last-head", 257, 64, (7, 4, 13), 2, 8, False, True),
]


@pytest.mark.parametrize("name,N,H,heads,ku,d,bf16,with_avail", CASES, ids=[c[0] for c in CASES])
def test_ppo_with_unit_head_matches_oracle(name, N, H, heads, ku, d, bf16, with_avail):
    need_gpu()
    banner(f"ppo unit head {name} N={N} H={H} heads={heads} head={ku} d={d} bf16={bf16}")
    x = _inputs(N, H, heads, ku, d, seed=N + d, bf16=bf16, with_avail=with_avail)
    r = x["ref"]
    stats_ref, dh_ref, dWp_ref, dbp_ref, _, (dWq_ref, dbq_ref) = ppo_loss_grad(
        r["h"], r["Wp"], x["bp"], x["act"], x["logp_old"], x["adv"], x["ret"], heads, 0.2, 1.0, 0.01, x["mask"],
        x["avail"], x["unit_ref"])
    dt = o5.O5_BF16 if bf16 else o5.O5_F32
    A1 = sum(heads) + 1
    Wq_d, bq_d, E_d = dev_dt(x["Wq"], bf16), dev_f32(x["bq"]), dev_dt(x["E"], bf16)
    dWq = torch.empty((d, H), dtype=torch.float32, device="cuda")
    dbq = torch.empty(d, dtype=torch.float32, device="cuda")
    u = o5.unit_head(ku, d, Wq_d, bq_d, E_d, dWq, dbq)
    stats = torch.empty(8, dtype=torch.float32, device="cuda")
    dh = torch.empty((N, H), dtype=torch.float32, device="cuda")
    dWp = torch.empty((A1, H), dtype=torch.float32, device="cuda")
    dbp = torch.empty(A1, dtype=torch.float32, device="cuda")
    ws = workspace(o5.o5_ppo_loss_grad_workspace_bytes(dt, N, H, heads, unit=u))
    o5.o5_ppo_loss_grad(dt, N, H, heads, dev_dt(x["h"], bf16), dev_dt(x["Wp"], bf16), dev_f32(x["bp"]),
                        dev(x["act"]), dev_f32(x["logp_old"]), dev_f32(x["adv"]), dev_f32(x["ret"]), dev(x["mask"]),
                        0.2, 1.0, 0.01, stats, dh, dWp, dbp, ws,
                        avail=dev(x["avail"]) if x["avail"] is not None else None, unit=u)
    tol = TOL_BF16 if bf16 else TOL_F32
    st = host(stats)
    for i, nm in enumerate(STAT_NAMES):
        e = abs(st[i] - stats_ref[nm]) / max(abs(stats_ref[nm]), 1e-6)
        print(f"    stat {nm}: gpu={st[i]:.6g} ref={stats_ref[nm]:.6g} rel={e:.2e}", flush=True)
        assert e <= tol, nm
    assert_close("dh", host(dh), dh_ref, tol)
    assert_close("dWp", host(dWp), dWp_ref, tol)
    assert_close("dbp", host(dbp), dbp_ref, tol)
    assert_close("dWq", host(dWq), dWq_ref, tol)
    assert_close("dbq", host(dbq), dbq_ref, tol)
    off = head_offsets(heads)
    assert np.all(host(dWp)[off[ku]:off[ku + 1]] == 0.0)


@pytest.mark.parametrize("bf16", [False, True])
def test_policy_sample_with_unit_head_matches_oracle(bf16):
    need_gpu()
    heads, ku, d, B, H = (30, 189, 32, 4), 1, 64, 700, 256
    banner(f"policy_sample unit head bf16={bf16} B={B}")
    x = _inputs(B, H, heads, ku, d, seed=11, bf16=bf16, with_avail=True)
    seed, counter = 77, 3
    act_ref, logp_ref, v_ref, scores = gumbel_max_sample(x["z"], heads, seed, counter, x["avail"])
    dt = o5.O5_BF16 if bf16 else o5.O5_F32
    Wq_d, bq_d, E_d = dev_dt(x["Wq"], bf16), dev_f32(x["bq"]), dev_dt(x["E"], bf16)
    u = o5.unit_head(ku, d, Wq_d, bq_d, E_d)
    act = torch.empty((B, len(heads)), dtype=torch.int32, device="cuda")
    logp = torch.empty(B, dtype=torch.float32, device="cuda")
    value = torch.empty(B, dtype=torch.float32, device="cuda")
    ws = workspace(o5.o5_policy_sample_workspace_bytes(dt, B, H, heads, unit=u))
    o5.o5_policy_sample(dt, B, H, heads, dev_dt(x["h"], bf16), dev_dt(x["Wp"], bf16), dev_f32(x["bp"]), seed, counter,
                        act, logp, value, ws, avail=dev(x["avail"]), unit=u)
    a = act.cpu().numpy()
    agree = np.ones(B, bool)
    for k in range(len(heads)):
        s = np.sort(scores[k], axis=1)
        with np.errstate(invalid="ignore"):
            clear = ~(s[:, -1] - s[:, -2] <= 1e-4)
        mism = a[:, k] != act_ref[:, k]
        assert not np.any(mism & clear), f"head {k}: {np.sum(mism & clear)} clear-cut mismatches"
        agree &= ~mism
    assert agree.mean() > 0.99
    tol = TOL_BF16 if bf16 else TOL_F32
    assert_close("logp", host(logp)[agree], logp_ref[agree], tol)
    assert_close("value", host(value), v_ref, tol)
