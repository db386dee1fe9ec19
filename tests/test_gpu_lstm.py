"""GPU parity: o5_lstm_fwd and o5_lstm_bptt against the fp64 oracle.

fp32 path: every input fp32, tolerance 1e-4.  bf16 path, tolerance 3e-2,
against two oracles on the same inputs: the plain definition (the oracle
takes the bf16-rounded x, W_x, W_h and keeps every intermediate in fp64),
and the oracle that also rounds h, the saved gates and dG where the GPU
stores them in bf16 (the oracle's ``store``), which measures the kernels'
own error without the propagated rounding of the stored operands.  Shapes
span several tiles with ragged edges in B and in the 4H / D+H dimensions,
resets inside samples, and the paper-scale shapes (B=1024 and 2048, T=16,
D=H=4096) on one sampled row in every 256-row tile.
"""
import numpy as np
import pytest
import torch

from oracle.bf16 import round_to_bf16
from oracle.lstm import lstm_bptt, lstm_forward
from paper_1912_06680_amd import o5
from tests.gpu_util import (TOL_BF16, TOL_F32, assert_close, assert_close_both, banner, dev, dev_dt, dev_f32,
                            empty_dt, host, need_gpu, tile_rows, workspace)

pytestmark = pytest.mark.gpu


def _inputs(T, B, D, H, seed, state_std=0.1, p_reset=0.0):
    rng = np.random.Generator(np.random.PCG64(seed))
    bound = 1.0 / np.sqrt(H)
    Wx = ((rng.random((4 * H, D), dtype=np.float32) * 2 - 1) * bound).astype(np.float32)
    Wh = ((rng.random((4 * H, H), dtype=np.float32) * 2 - 1) * bound).astype(np.float32)
    b = ((rng.random(4 * H, dtype=np.float32) * 2 - 1) * bound).astype(np.float32)
    x = rng.standard_normal((T, B, D), dtype=np.float32)
    h0 = (rng.standard_normal((B, H), dtype=np.float32) * state_std).astype(np.float32)
    c0 = (rng.standard_normal((B, H), dtype=np.float32) * state_std).astype(np.float32)
    reset = (rng.random((T, B)) < p_reset).astype(np.uint8) if p_reset > 0 else None
    dh = rng.standard_normal((T, B, H), dtype=np.float32)
    dhT = rng.standard_normal((B, H), dtype=np.float32)
    dcT = rng.standard_normal((B, H), dtype=np.float32)
    return dict(Wx=Wx, Wh=Wh, b=b, x=x, h0=h0, c0=c0, reset=reset, dh=dh, dhT=dhT, dcT=dcT)


def _run_gpu(inp, T, B, D, H, bf16, with_final=True, want_dx=True):
    dt = o5.O5_BF16 if bf16 else o5.O5_F32
    x, Wx, Wh = dev_dt(inp["x"], bf16), dev_dt(inp["Wx"], bf16), dev_dt(inp["Wh"], bf16)
    b, h0, c0 = dev_f32(inp["b"]), dev_f32(inp["h0"]), dev_f32(inp["c0"])
    reset = dev(inp["reset"]) if inp["reset"] is not None else None
    h = empty_dt((T, B, H), bf16)
    c = torch.empty((T, B, H), dtype=torch.float32, device="cuda")
    gates = empty_dt((T, B, 4 * H), bf16)
    ws = workspace(max(o5.o5_lstm_fwd_workspace_bytes(dt, T, B, D, H),
                       o5.o5_lstm_bptt_workspace_bytes(dt, T, B, D, H)))
    o5.o5_lstm_fwd(dt, T, B, D, H, x, Wx, Wh, b, h0, c0, reset, h, c, gates, ws)
    dWx = torch.empty((4 * H, D), dtype=torch.float32, device="cuda")
    dWh = torch.empty((4 * H, H), dtype=torch.float32, device="cuda")
    db = torch.empty(4 * H, dtype=torch.float32, device="cuda")
    dx = empty_dt((T, B, D), bf16) if want_dx else None
    dhT = dev_f32(inp["dhT"]) if with_final else None
    dcT = dev_f32(inp["dcT"]) if with_final else None
    o5.o5_lstm_bptt(dt, T, B, D, H, x, Wx, Wh, h0, c0, reset, h, c, gates, dev_f32(inp["dh"]), dhT, dcT,
                    dWx, dWh, db, dx, ws)
    return dict(h=h, c=c, gates=gates, dWx=dWx, dWh=dWh, db=db, dx=dx)


def _oracle(inp, bf16, with_final=True, plain=False):
    """fp64 oracle; on the bf16 path the inputs are bf16-rounded and, unless
    ``plain``, h, the saved gates and dG are rounded where the GPU stores them."""
    rnd = round_to_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    store = round_to_bf16 if (bf16 and not plain) else None
    x, Wx, Wh = rnd(inp["x"]), rnd(inp["Wx"]), rnd(inp["Wh"])
    h, c, gates = lstm_forward(x, Wx, Wh, inp["b"], inp["h0"], inp["c0"], inp["reset"], store=store)
    dWx, dWh, db, dx = lstm_bptt(x, Wx, Wh, inp["h0"], inp["c0"], inp["reset"], h, c, gates, inp["dh"],
                                 inp["dhT"] if with_final else None, inp["dcT"] if with_final else None,
                                 want_dx=True, store=store)
    return dict(h=h, c=c, gates=gates, dWx=dWx, dWh=dWh, db=db, dx=dx)


CASES = [
    # name, T, B, D, H, bf16, p_reset
    ("f32-tiny", 16, 8, 64, 128, False, 0.0),
    ("f32-ragged-reset", 5, 7, 64, 64, False, 0.2),
    ("f32-mid", 16, 256, 1024, 1024, False, 0.005),
    ("bf16-ragged-reset", 3, 300, 128, 192, True, 0.2),
    ("bf16-mid", 16, 256, 1024, 1024, True, 0.005),
    ("bf16-tall", 4, 520, 256, 320, True, 0.05),
    # one step (no recurrent-gradient GEMM at all), a single sequence, an
    # input wider than the state
    ("f32-T1-B1", 1, 1, 64, 64, False, 0.0),
    ("bf16-T1", 1, 130, 128, 64, True, 0.0),
    ("bf16-wide-input", 2, 96, 320, 128, True, 0.1),
]


@pytest.mark.parametrize("name,T,B,D,H,bf16,p_reset", CASES, ids=[c[0] for c in CASES])
def test_lstm_fwd_bptt_matches_oracle(name, T, B, D, H, bf16, p_reset):
    need_gpu()
    banner(f"lstm {name} T={T} B={B} D={D} H={H} bf16={bf16}")
    inp = _inputs(T, B, D, H, seed=T * 1000 + B + H, p_reset=p_reset)
    got = _run_gpu(inp, T, B, D, H, bf16)
    ref = _oracle(inp, bf16)
    if not bf16:
        for k in ("h", "c", "gates", "dWx", "dWh", "db", "dx"):
            assert_close(k, host(got[k]), ref[k], TOL_F32)
        return
    plain = _oracle(inp, True, plain=True)
    for k in ("h", "c", "gates", "dWx", "dWh", "db", "dx"):
        assert_close_both(k, host(got[k]), ref[k], plain[k], TOL_BF16)


def test_lstm_without_final_state_gradient_and_dx():
    need_gpu()
    banner("lstm f32 no dhT/dcT, no dx")
    T, B, D, H = 4, 9, 64, 64
    inp = _inputs(T, B, D, H, seed=5, p_reset=0.3)
    got = _run_gpu(inp, T, B, D, H, False, with_final=False, want_dx=False)
    ref = _oracle(inp, False, with_final=False)
    for k in ("dWx", "dWh", "db"):
        assert_close(k, host(got[k]), ref[k], TOL_F32)


def test_lstm_inference_without_gates_and_determinism():
    need_gpu()
    banner("lstm bf16 inference (gates=NULL) and determinism")
    T, B, D, H = 2, 64, 256, 256
    inp = _inputs(T, B, D, H, seed=9)
    dt = o5.O5_BF16
    x, Wx, Wh = dev_dt(inp["x"], True), dev_dt(inp["Wx"], True), dev_dt(inp["Wh"], True)
    b, h0, c0 = dev_f32(inp["b"]), dev_f32(inp["h0"]), dev_f32(inp["c0"])
    ws = workspace(o5.o5_lstm_fwd_workspace_bytes(dt, T, B, D, H))
    outs = []
    for _ in range(2):
        h = empty_dt((T, B, H), True)
        c = torch.empty((T, B, H), dtype=torch.float32, device="cuda")
        o5.o5_lstm_fwd(dt, T, B, D, H, x, Wx, Wh, b, h0, c0, None, h, c, None, ws)
        outs.append((host(h), host(c)))
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
    assert_close_both("h", outs[0][0], _oracle(inp, True)["h"], _oracle(inp, True, plain=True)["h"], TOL_BF16)


def test_rollout_step_paper_scale():
    """One rollout inference step at the paper's scale (B = 4096 environments,
    D = H = 4096, bf16, no saved gates) followed by the heads and the
    Gumbel-max draw, in the launch configuration the benchmark times.  The
    LSTM step is checked on sampled rows (rows are independent); the draw
    takes the device's bf16 h of every row through the oracle's heads and
    Philox sampler."""
    from oracle.philox import gumbel_max_sample
    from oracle.ppo import heads_forward
    need_gpu()
    T, B, D, H = 1, 4096, 4096, 4096
    heads = (30, 8, 32, 4)
    A1 = sum(heads) + 1
    banner(f"rollout step B={B} D={D} H={H} heads={heads}")
    inp = _inputs(T, B, D, H, 41)
    rng = np.random.Generator(np.random.PCG64(42))
    Wp = ((rng.random((A1, H), dtype=np.float32) * 2 - 1) * 4 / np.sqrt(H)).astype(np.float32)
    bp = ((rng.random(A1, dtype=np.float32) * 2 - 1) / np.sqrt(H)).astype(np.float32)
    dt = o5.O5_BF16
    x, Wx, Wh = dev_dt(inp["x"], True), dev_dt(inp["Wx"], True), dev_dt(inp["Wh"], True)
    b, h0, c0 = dev_f32(inp["b"]), dev_f32(inp["h0"]), dev_f32(inp["c0"])
    h = empty_dt((T, B, H), True)
    c = torch.empty((T, B, H), dtype=torch.float32, device="cuda")
    ws = workspace(o5.o5_lstm_fwd_workspace_bytes(dt, T, B, D, H))
    o5.o5_lstm_fwd(dt, T, B, D, H, x, Wx, Wh, b, h0, c0, None, h, c, None, ws)
    act = torch.empty((B, len(heads)), dtype=torch.int32, device="cuda")
    logp = torch.empty(B, dtype=torch.float32, device="cuda")
    value = torch.empty(B, dtype=torch.float32, device="cuda")
    sws = workspace(o5.o5_policy_sample_workspace_bytes(dt, B, H, heads))
    seed, counter = 5, 7
    o5.o5_policy_sample(dt, B, H, heads, h[0], dev_dt(Wp, True), dev_f32(bp), seed, counter, act, logp, value, sws)
    rows = np.array(tile_rows(B))
    refs = [lstm_forward(round_to_bf16(inp["x"][:, rows]), round_to_bf16(inp["Wx"]), round_to_bf16(inp["Wh"]),
                         inp["b"], inp["h0"][rows], inp["c0"][rows], None, store=st)
            for st in (round_to_bf16, None)]
    hg = host(h)
    assert_close_both("h[rows]", hg[:, rows], refs[0][0], refs[1][0], TOL_BF16)
    assert_close_both("c[rows]", host(c)[:, rows], refs[0][1], refs[1][1], TOL_BF16)
    z = heads_forward(hg[0], round_to_bf16(Wp), bp)
    act_ref, logp_ref, v_ref, scores = gumbel_max_sample(z, heads, seed, counter)
    a = act.cpu().numpy()
    agree = np.ones(B, bool)
    for k in range(len(heads)):
        srt = np.sort(scores[k], axis=1)
        clear = srt[:, -1] - srt[:, -2] > 1e-4
        mism = a[:, k] != act_ref[:, k]
        assert not np.any(mism & clear), f"head {k}: {np.sum(mism & clear)} clear-cut mismatches"
        agree &= ~mism
    assert agree.mean() > 0.99
    assert_close("logp", host(logp)[agree], logp_ref[agree], TOL_BF16)
    assert_close("value", host(value), v_ref, TOL_BF16)


@pytest.mark.parametrize("B", [1024, 2048])
def test_lstm_paper_scale_sampled_rows(B):
    """B=1024 and the benchmark's B=2048, T=16, D=H=4096, in the benchmark's
    launch configuration.

    Forward: rows are independent, so the oracle recomputes one row in every
    256-row tile of the GEMMs (plus the first and last row).  BPTT: the
    upstream gradient is nonzero only on those rows, so every weight
    gradient is the sum over those rows alone, which the oracle computes
    exactly.  Compared with both oracles (storage-point and plain)."""
    need_gpu()
    T, D, H = 16, 4096, 4096
    banner(f"lstm paper-scale sampled rows T={T} B={B} D={D} H={H}")
    rng = np.random.Generator(np.random.PCG64(B))
    bound = 1.0 / np.sqrt(H)
    inp = dict(
        Wx=((rng.random((4 * H, D), dtype=np.float32) * 2 - 1) * bound).astype(np.float32),
        Wh=((rng.random((4 * H, H), dtype=np.float32) * 2 - 1) * bound).astype(np.float32),
        b=((rng.random(4 * H, dtype=np.float32) * 2 - 1) * bound).astype(np.float32),
        x=rng.standard_normal((T, B, D), dtype=np.float32),
        h0=(rng.standard_normal((B, H), dtype=np.float32) * 0.1).astype(np.float32),
        c0=(rng.standard_normal((B, H), dtype=np.float32) * 0.1).astype(np.float32),
        reset=None,
    )
    rows = np.array(tile_rows(B))
    dh = np.zeros((T, B, H), np.float32)
    dh[:, rows] = rng.standard_normal((T, len(rows), H), dtype=np.float32)
    inp["dh"] = dh
    inp["dhT"] = None
    inp["dcT"] = None
    got = _run_gpu(inp, T, B, D, H, True, with_final=False, want_dx=False)
    sub = dict(inp)
    sub["x"] = inp["x"][:, rows]
    sub["h0"] = inp["h0"][rows]
    sub["c0"] = inp["c0"][rows]
    sub["dh"] = dh[:, rows]
    ref = _oracle(sub, True, with_final=False)
    plain = _oracle(sub, True, with_final=False, plain=True)
    print(f"    rows {rows.tolist()}", flush=True)
    assert_close_both("h[rows]", host(got["h"][:, rows.tolist()]), ref["h"], plain["h"], TOL_BF16)
    assert_close_both("c[rows]", host(got["c"][:, rows.tolist()]), ref["c"], plain["c"], TOL_BF16)
    assert_close_both("gates[rows]", host(got["gates"][:, rows.tolist()]), ref["gates"], plain["gates"], TOL_BF16)
    for k in ("dWx", "dWh", "db"):
        assert_close_both(k, host(got[k]), ref[k], plain[k], TOL_BF16)


def test_lstm_dma_engine_ragged_sampled_rows():
    """Shapes that select the direct-to-LDS engine with partial tiles in every
    dimension: B = 2000 rows (last M tile partial), H = 1984 (4H and D+H not
    multiples of 256, dh's N = H ragged), D = 1088, T*B = 4000 (K of the
    weight-gradient GEMM not a multiple of 32), with state resets.  Checked
    on sampled rows as in the paper-scale test."""
    need_gpu()
    T, B, D, H = 2, 2000, 1088, 1984
    banner(f"lstm dma ragged T={T} B={B} D={D} H={H}")
    rng = np.random.Generator(np.random.PCG64(7))
    bound = 1.0 / np.sqrt(H)
    inp = dict(
        Wx=((rng.random((4 * H, D), dtype=np.float32) * 2 - 1) * bound).astype(np.float32),
        Wh=((rng.random((4 * H, H), dtype=np.float32) * 2 - 1) * bound).astype(np.float32),
        b=((rng.random(4 * H, dtype=np.float32) * 2 - 1) * bound).astype(np.float32),
        x=rng.standard_normal((T, B, D), dtype=np.float32),
        h0=(rng.standard_normal((B, H), dtype=np.float32) * 0.1).astype(np.float32),
        c0=(rng.standard_normal((B, H), dtype=np.float32) * 0.1).astype(np.float32),
    )
    reset = np.zeros((T, B), np.uint8)
    rows = np.array([3, 1790, 1999])
    reset[1, 1790] = 1          # reset inside a sampled row
    reset[0, 3] = 1
    reset[1, 500] = 1
    inp["reset"] = reset
    dh = np.zeros((T, B, H), np.float32)
    dh[:, rows] = rng.standard_normal((T, len(rows), H), dtype=np.float32)
    inp["dh"] = dh
    inp["dhT"] = None
    inp["dcT"] = None
    got = _run_gpu(inp, T, B, D, H, True, with_final=False, want_dx=False)
    sub = dict(inp)
    sub["x"] = inp["x"][:, rows]
    sub["h0"] = inp["h0"][rows]
    sub["c0"] = inp["c0"][rows]
    sub["reset"] = reset[:, rows]
    sub["dh"] = dh[:, rows]
    ref = _oracle(sub, True, with_final=False)
    plain = _oracle(sub, True, with_final=False, plain=True)
    assert_close_both("h[rows]", host(got["h"][:, rows.tolist()]), ref["h"], plain["h"], TOL_BF16)
    assert_close_both("c[rows]", host(got["c"][:, rows.tolist()]), ref["c"], plain["c"], TOL_BF16)
    assert_close_both("gates[rows]", host(got["gates"][:, rows.tolist()]), ref["gates"], plain["gates"], TOL_BF16)
    for k in ("dWx", "dWh", "db"):
        assert_close_both(k, host(got[k]), ref[k], plain[k], TOL_BF16)


def test_lstm_largest_batch_sampled_rows():
    """The largest batch the calls accept (B = 2,097,088, the cell kernels'
    grid bound) at T = 3, D = H = 64, bf16, with resets: every cell grid at
    its limit, and T * B rows of [x | h~] that the weight gradient's
    transposes walk in more row tiles than one grid dimension holds.
    Checked on sampled rows as in the paper-scale test (the upstream
    gradient is nonzero only there)."""
    need_gpu()
    T, B, D, H = 3, 32767 * 64, 64, 64
    banner(f"lstm largest batch T={T} B={B} D={D} H={H}")
    rng = np.random.Generator(np.random.PCG64(17))
    bound = 1.0 / np.sqrt(H)
    inp = dict(
        Wx=((rng.random((4 * H, D), dtype=np.float32) * 2 - 1) * bound).astype(np.float32),
        Wh=((rng.random((4 * H, H), dtype=np.float32) * 2 - 1) * bound).astype(np.float32),
        b=((rng.random(4 * H, dtype=np.float32) * 2 - 1) * bound).astype(np.float32),
        x=rng.standard_normal((T, B, D), dtype=np.float32),
        h0=(rng.standard_normal((B, H), dtype=np.float32) * 0.1).astype(np.float32),
        c0=(rng.standard_normal((B, H), dtype=np.float32) * 0.1).astype(np.float32),
    )
    rows = np.array([0, 63, 64, 1 << 20, 1_500_001, B - 65, B - 1])
    reset = np.zeros((T, B), np.uint8)
    reset[1, rows[1]] = 1
    reset[2, rows[4]] = 1
    inp["reset"] = reset
    dh = np.zeros((T, B, H), np.float32)
    dh[:, rows] = rng.standard_normal((T, len(rows), H), dtype=np.float32)
    inp["dh"] = dh
    inp["dhT"] = None
    inp["dcT"] = None
    got = _run_gpu(inp, T, B, D, H, True, with_final=False, want_dx=False)
    torch.cuda.synchronize()
    sub = dict(inp)
    sub["x"] = inp["x"][:, rows]
    sub["h0"] = inp["h0"][rows]
    sub["c0"] = inp["c0"][rows]
    sub["reset"] = reset[:, rows]
    sub["dh"] = dh[:, rows]
    ref = _oracle(sub, True, with_final=False)
    plain = _oracle(sub, True, with_final=False, plain=True)
    assert_close_both("h[rows]", host(got["h"][:, rows.tolist()]), ref["h"], plain["h"], TOL_BF16)
    assert_close_both("c[rows]", host(got["c"][:, rows.tolist()]), ref["c"], plain["c"], TOL_BF16)
    for k in ("dWx", "dWh", "db"):
        assert_close_both(k, host(got[k]), ref[k], plain[k], TOL_BF16)


@pytest.mark.parametrize("bf16", [False, True])
def test_lstm_saturated_gates(bf16):
    """Pre-activations far beyond the range where exp over- or underflows in
    fp32: biases of +-100 and +-150 on four gate rows in five (|a| > 89),
    the weights at their usual scale so the GEMM sums stay well conditioned.
    Those gates saturate to 0 or 1 (tanh to -1 or 1) through the
    exponential's infinity or zero, with nothing non-finite, and the forward
    pass and BPTT still match the oracle (whose logistic function is
    evaluated without overflow)."""
    need_gpu()
    T, B, D, H = 3, 130, 128, 128
    banner(f"lstm saturated gates T={T} B={B} D={D} H={H} bf16={bf16}")
    inp = _inputs(T, B, D, H, 23, p_reset=0.1)
    rng = np.random.Generator(np.random.PCG64(24))
    inp["b"] = rng.choice(np.array([-150.0, -100.0, 0.0, 100.0, 150.0], np.float32), 4 * H).astype(np.float32)
    got = _run_gpu(inp, T, B, D, H, bf16)
    torch.cuda.synchronize()
    for k in ("h", "c", "gates", "dWx", "dWh", "db", "dx"):
        assert bool(torch.isfinite(got[k].float()).all()), k
    ref = _oracle(inp, bf16)
    tol = TOL_BF16 if bf16 else TOL_F32
    if bf16:
        plain = _oracle(inp, bf16, plain=True)
        for k in ("h", "c", "gates", "dWx", "dWh", "db", "dx"):
            assert_close_both(k, host(got[k]), ref[k], plain[k], tol)
    else:
        for k in ("h", "c", "gates", "dWx", "dWh", "db", "dx"):
            assert_close(k, host(got[k]), ref[k], tol)
