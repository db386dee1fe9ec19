"""GPU: the heads' gradient in factored form (bf16).

o5_ppo_loss_grad_factored must give o5_ppo_loss_grad's statistics and head
gradients bit for bit and a pair P, W with P W^T equal to its dh; and
o5_lstm_bptt_factored, fed that pair, must give o5_lstm_bptt's weight and
input gradients for that dh.  The composed bf16 step (tests/test_gpu_step.py)
runs this path against the oracle."""
import numpy as np
import pytest
import torch

from paper_1912_06680_amd import o5
from tests.gpu_util import TOL_BF16, banner, dev, dev_bf16, dev_f32, host, need_gpu, workspace
from tests.test_gpu_ppo_sample import HEADS, _inputs

pytestmark = pytest.mark.gpu


def _unit(rng, N, H, heads, head, d):
    """Random unit-head tensors (query weights, bias, per-row embeddings)."""
    nk = heads[head]
    Wq = dev_bf16((rng.random((d, H), dtype=np.float32) * 2 - 1) / np.sqrt(H))
    bq = dev_f32(rng.standard_normal(d, dtype=np.float32) * 0.1)
    E = dev_bf16(rng.standard_normal((N, nk, d), dtype=np.float32) * 0.1)
    return Wq, bq, E


def _both_loss_calls(N, H, heads, seed, with_mask, with_avail, unit_d):
    rng = np.random.Generator(np.random.PCG64(seed + 100))
    inp = _inputs(N, H, heads, seed, True, with_mask, with_avail)
    A1 = sum(heads) + 1
    h, Wp = dev_bf16(inp["h"]), dev_bf16(inp["Wp"])
    bp, act = dev_f32(inp["bp"]), dev(inp["act"])
    lpo, adv, ret = dev_f32(inp["logp_old"]), dev_f32(inp["adv"]), dev_f32(inp["ret"])
    mask = dev(inp["mask"]) if inp["mask"] is not None else None
    avail = dev(inp["avail"]) if inp["avail"] is not None else None
    uq = _unit(rng, N, H, heads, 1, unit_d) if unit_d else None
    out = []
    for factored in (False, True):
        stats = torch.full((8,), -7.0, device="cuda")
        dWp = torch.empty((A1, H), device="cuda")
        dbp = torch.empty(A1, device="cuda")
        u, ug = None, None
        if uq is not None:
            ug = (torch.empty((unit_d, H), device="cuda"), torch.empty(unit_d, device="cuda"))
            u = o5.unit_head(1, unit_d, uq[0], uq[1], uq[2], ug[0], ug[1])
        ws = workspace(o5.o5_ppo_loss_grad_workspace_bytes(o5.O5_BF16, N, H, heads, u))
        if factored:
            ld = o5.o5_ppo_head_grad_ld(H, heads, u)
            assert ld > 0 and ld % 64 == 0
            P = torch.empty((N, ld), dtype=torch.bfloat16, device="cuda")
            W = torch.empty((H, ld), dtype=torch.bfloat16, device="cuda")
            o5.o5_ppo_loss_grad_factored(o5.O5_BF16, N, H, heads, h, Wp, bp, act, lpo, adv, ret, mask, 0.2, 1.0,
                                         0.01, stats, P, W, ld, dWp, dbp, ws, avail=avail, unit=u)
            dh = (P.float().double() @ W.float().double().t())
        else:
            dh = torch.empty((N, H), device="cuda")
            o5.o5_ppo_loss_grad(o5.O5_BF16, N, H, heads, h, Wp, bp, act, lpo, adv, ret, mask, 0.2, 1.0, 0.01,
                                stats, dh, dWp, dbp, ws, avail=avail, unit=u)
        out.append(dict(stats=host(stats), dWp=host(dWp), dbp=host(dbp), dh=host(dh),
                        dWq=host(ug[0]) if ug else None, dbq=host(ug[1]) if ug else None))
    return out


@pytest.mark.parametrize("name,N,H,heads,with_mask,with_avail,unit_d", [
    ("mid", 4096, 1024, HEADS, True, False, 0),
    ("ragged-avail", 1001, 256, (5, 3, 7), True, True, 0),
    ("unit-head", 2048, 512, (30, 40, 32, 4), False, True, 128),
    ("wide-heads", 500, 128, (100, 60, 30), True, False, 0),
    # 1023 logits + value: the widest heads the call takes, 2048 pair columns
    ("widest", 300, 64, (512, 511), True, False, 0),
    ("unit-d512", 700, 128, (7, 9), True, True, 512),
])
def test_factored_loss_matches_the_plain_call(name, N, H, heads, with_mask, with_avail, unit_d):
    need_gpu()
    banner(f"factored loss {name} N={N} H={H} heads={heads} unit_d={unit_d}")
    plain, fact = _both_loss_calls(N, H, heads, 5, with_mask, with_avail, unit_d)
    for k in ("stats", "dWp", "dbp", "dWq", "dbq"):
        if plain[k] is not None:
            assert np.array_equal(plain[k], fact[k]), k
    err = np.max(np.abs(fact["dh"] - plain["dh"])) / np.max(np.abs(plain["dh"]))
    print(f"    max|P W^T - dh| / max|dh| = {err:.2e}", flush=True)
    # the same bf16 products, summed in fp64 here and in fp32 by the GEMM
    assert err <= 5e-5


def test_factored_call_rejects_fp32_and_a_wrong_ld():
    need_gpu()
    banner("factored loss: rejected calls")
    N, H = 64, 64
    inp = _inputs(N, H, HEADS, 3, True, False)
    A1 = sum(HEADS) + 1
    h, Wp = dev_bf16(inp["h"]), dev_bf16(inp["Wp"])
    bp, act = dev_f32(inp["bp"]), dev(inp["act"])
    lpo, adv, ret = dev_f32(inp["logp_old"]), dev_f32(inp["adv"]), dev_f32(inp["ret"])
    stats = torch.full((8,), -7.0, device="cuda")
    dWp = torch.full((A1, H), -7.0, device="cuda")
    dbp = torch.full((A1,), -7.0, device="cuda")
    ld = o5.o5_ppo_head_grad_ld(H, HEADS)
    P = torch.full((N, ld), -7.0, dtype=torch.bfloat16, device="cuda")
    W = torch.full((H, ld), -7.0, dtype=torch.bfloat16, device="cuda")
    ws = workspace(o5.o5_ppo_loss_grad_workspace_bytes(o5.O5_BF16, N, H, HEADS))
    L = o5.lib()
    for dt, ldx, code in ((o5.O5_F32, ld, 3), (o5.O5_BF16, ld + 64, 2), (o5.O5_BF16, 0, 2)):
        st = L.o5_ppo_loss_grad_factored(dt, N, H, len(HEADS), o5._heads(HEADS), o5._p(h), o5._p(Wp), o5._p(bp),
                                         o5._p(act), o5._p(lpo), o5._p(adv), o5._p(ret), None, None, None,
                                         o5.PpoHp(0.2, 1.0, 0.01), o5._p(stats), o5._p(P), o5._p(W), ldx,
                                         o5._p(dWp), o5._p(dbp), o5._p(ws), ws.numel(), None)
        assert st == code, (dt, ldx, st, o5.o5_last_error())
    torch.cuda.synchronize()
    for t in (stats, dWp, dbp, P.float(), W.float()):
        assert bool((t == -7.0).all())


def _lstm_case(T, B, D, H, seed, p_reset):
    rng = np.random.Generator(np.random.PCG64(seed))
    bound = 1.0 / np.sqrt(H)
    Wx = dev_bf16((rng.random((4 * H, D), dtype=np.float32) * 2 - 1) * bound)
    Wh = dev_bf16((rng.random((4 * H, H), dtype=np.float32) * 2 - 1) * bound)
    b = dev_f32((rng.random(4 * H, dtype=np.float32) * 2 - 1) * bound)
    x = dev_bf16(rng.standard_normal((T, B, D), dtype=np.float32))
    h0 = dev_f32(rng.standard_normal((B, H), dtype=np.float32) * 0.1)
    c0 = dev_f32(rng.standard_normal((B, H), dtype=np.float32) * 0.1)
    reset = dev((rng.random((T, B)) < p_reset).astype(np.uint8))
    h = torch.empty((T, B, H), dtype=torch.bfloat16, device="cuda")
    c = torch.empty((T, B, H), device="cuda")
    gates = torch.empty((T, B, 4 * H), dtype=torch.bfloat16, device="cuda")
    ws = workspace(max(o5.o5_lstm_fwd_workspace_bytes(o5.O5_BF16, T, B, D, H),
                       o5.o5_lstm_bptt_workspace_bytes(o5.O5_BF16, T, B, D, H)))
    o5.o5_lstm_fwd(o5.O5_BF16, T, B, D, H, x, Wx, Wh, b, h0, c0, reset, h, c, gates, ws)
    return dict(x=x, Wx=Wx, Wh=Wh, h0=h0, c0=c0, reset=reset, h=h, c=c, gates=gates, ws=ws)


@pytest.mark.parametrize("T,B,D,H,heads,p_reset,with_dx", [
    (16, 256, 1024, 1024, HEADS, 0.05, True),
    (5, 77, 128, 192, (5, 3, 7), 0.2, False),
    (1, 130, 64, 64, (4,), 0.5, True),
    (16, 1024, 4096, 4096, HEADS, 0.01, False),
])
def test_factored_bptt_matches_the_dh_bptt(T, B, D, H, heads, p_reset, with_dx):
    """The heads' loss on the forward pass's own h, once with dh stored and
    once factored; the two backward passes see the same dh up to the fp32
    rounding of where it is summed."""
    need_gpu()
    banner(f"factored bptt T={T} B={B} D={D} H={H} p_reset={p_reset}")
    s = _lstm_case(T, B, D, H, 11, p_reset)
    N = T * B
    inp = _inputs(N, H, heads, 13, True, True)
    A1 = sum(heads) + 1
    Wp, bp, act = dev_bf16(inp["Wp"]), dev_f32(inp["bp"]), dev(inp["act"])
    lpo, adv, ret = dev_f32(inp["logp_old"]), dev_f32(inp["adv"]), dev_f32(inp["ret"])
    mask = dev(inp["mask"])
    hN = s["h"].view(N, H)
    stats = torch.empty(8, device="cuda")
    dWp, dbp = torch.empty((A1, H), device="cuda"), torch.empty(A1, device="cuda")
    pws = workspace(o5.o5_ppo_loss_grad_workspace_bytes(o5.O5_BF16, N, H, heads))
    dh = torch.empty((N, H), device="cuda")
    o5.o5_ppo_loss_grad(o5.O5_BF16, N, H, heads, hN, Wp, bp, act, lpo, adv, ret, mask, 0.2, 1.0, 0.01, stats, dh,
                        dWp, dbp, pws)
    ld = o5.o5_ppo_head_grad_ld(H, heads)
    P = torch.empty((N, ld), dtype=torch.bfloat16, device="cuda")
    W = torch.empty((H, ld), dtype=torch.bfloat16, device="cuda")
    o5.o5_ppo_loss_grad_factored(o5.O5_BF16, N, H, heads, hN, Wp, bp, act, lpo, adv, ret, mask, 0.2, 1.0, 0.01,
                                 stats, P, W, ld, dWp, dbp, pws)
    outs = []
    for factored in (False, True):
        dWx = torch.empty((4 * H, D), device="cuda")
        dWh = torch.empty((4 * H, H), device="cuda")
        db = torch.empty(4 * H, device="cuda")
        dx = torch.empty((T, B, D), dtype=torch.bfloat16, device="cuda") if with_dx else None
        args = (o5.O5_BF16, T, B, D, H, s["x"], s["Wx"], s["Wh"], s["h0"], s["c0"], s["reset"], s["h"], s["c"],
                s["gates"])
        if factored:
            o5.o5_lstm_bptt_factored(*args, P, W, ld, None, None, dWx, dWh, db, dx, s["ws"])
        else:
            o5.o5_lstm_bptt(*args, dh, None, None, dWx, dWh, db, dx, s["ws"])
        torch.cuda.synchronize()
        outs.append((dWx, dWh, db, dx))
    for name, a, b in zip(("dWx", "dWh", "db", "dx"), outs[0], outs[1]):
        if a is None:
            continue
        a, b = a.float(), b.float()
        err = float((a - b).abs().max() / a.abs().max())
        print(f"    {name}: max|factored - dh path| / max|dh path| = {err:.2e}", flush=True)
        # dG (and dx) are stored in bf16 on both paths: a rounding that lands
        # either side of a tie moves an element by one bf16 ulp (2^-8)
        assert err <= TOL_BF16 / 3, name
