"""GPU parity: o5_obs_normalize, o5_prelstm_fwd and o5_prelstm_bwd against
the fp64 oracle (appendix "Observation Space"; appendix "Neural Network
Architecture") on identical seeded inputs.  The backward's integer
decisions (ReLU mask, first arg-maximum of the pool) are taken by both
sides on the layer output the device computed in fp32."""
import numpy as np
import pytest
import torch

from oracle.bf16 import round_to_bf16
from oracle.prelstm import obs_normalize, prelstm_backward, prelstm_forward
from paper_1912_06680_amd import o5
from tests.gpu_util import TOL_BF16, TOL_F32, assert_close, banner, dev, dev_dt, dev_f32, empty_dt, host, need_gpu, \
    workspace

pytestmark = pytest.mark.gpu


def _obs(N, Do, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    mu = rng.uniform(-3, 3, Do).astype(np.float32)
    sd = rng.uniform(0.1, 4, Do).astype(np.float32)
    obs = (mu + sd * rng.standard_normal((N, Do), dtype=np.float32)).astype(np.float32)
    obs[:, 3] = 1.0                                   # a constant feature
    obs[rng.integers(0, N, 5), 5] = 1e4              # outliers, clipped
    return obs


@pytest.mark.parametrize("dt,N,Do", [(0, 1000, 64), (1, 777, 128), (0, 4096, 256)])
def test_obs_normalize_running_statistics(dt, N, Do):
    need_gpu()
    banner(f"obs_normalize dt={dt} N={N} Do={Do}")
    stats = torch.zeros((3, Do), dtype=torch.float64, device="cuda")
    ref = (0.0, np.zeros(Do), np.zeros(Do))
    ws = workspace(o5.o5_obs_normalize_workspace_bytes(N, Do))
    for k in range(3):
        obs = _obs(N, Do, seed=10 * N + k)
        o = empty_dt((N, Do), dt == 1)
        o5.o5_obs_normalize(dt, N, Do, dev_f32(obs), stats, 5.0, 1e-8, o, ws)
        o_ref, ref = obs_normalize(obs, ref)
        assert_close(f"o[{k}]", host(o), o_ref, TOL_BF16 if dt == 1 else TOL_F32)
        st = host(stats)
        assert np.all(st[0] == ref[0])
        sd = np.sqrt(ref[2] / ref[0]) + 1e-12
        assert np.max(np.abs(st[1] - ref[1]) / sd) < 1e-9
        assert np.max(np.abs(st[2] - ref[2]) / np.maximum(ref[2], 1e-300)) < 1e-7


def _layer(T, B, Do, D, seed, bf16):
    rng = np.random.Generator(np.random.PCG64(seed))
    o = np.clip(rng.standard_normal((T * B, Do), dtype=np.float32), -5, 5)
    W = (rng.standard_normal((D, Do), dtype=np.float32) / np.float32(np.sqrt(Do))).astype(np.float32)
    b = (0.1 * rng.standard_normal(D, dtype=np.float32)).astype(np.float32)
    dx = rng.standard_normal((T * B, D), dtype=np.float32)
    oo = round_to_bf16(o) if bf16 else o.astype(np.float64)
    ww = round_to_bf16(W) if bf16 else W.astype(np.float64)
    dd = round_to_bf16(dx) if bf16 else dx.astype(np.float64)
    return o, W, b, dx, oo, ww, dd


# (T, B, Do, D): one team, ragged pool widths, the paper's per-GPU batch of
# 120 teams x 5 replicas at reduced widths, and grids of the MFMA engines
@pytest.mark.parametrize("name,T,B,Do,D,bf16", [
    ("f32-tiny", 2, 5, 64, 64, False),
    ("f32-small", 3, 40, 128, 192, False),
    ("bf16-small", 4, 40, 128, 256, True),
    ("bf16-paper-batch", 16, 600, 256, 512, True),
    ("bf16-wide", 2, 1280, 1024, 2048, True),
])
def test_prelstm_matches_oracle(name, T, B, Do, D, bf16):
    need_gpu()
    banner(f"prelstm {name} T={T} B={B} Do={Do} D={D}")
    o, W, b, dx, oo, ww, dd = _layer(T, B, Do, D, seed=T * B + D, bf16=bf16)
    dt = o5.O5_BF16 if bf16 else o5.O5_F32
    N = T * B
    y = torch.empty((N, D), dtype=torch.float32, device="cuda")
    x = empty_dt((N, D), bf16)
    do_, dW_ = dev_dt(o, bf16), dev_dt(W, bf16)
    o5.o5_prelstm_fwd(dt, T, B, Do, D, do_, dW_, dev_f32(b), y, x)
    x_ref, y_ref = prelstm_forward(oo, ww, b, T, B)
    tol = TOL_BF16 if bf16 else TOL_F32
    y_gpu = host(y)
    assert_close("y", y_gpu, y_ref, tol)
    assert_close("x", host(x), x_ref, tol)
    dW = torch.empty((D, Do), dtype=torch.float32, device="cuda")
    db = torch.empty(D, dtype=torch.float32, device="cuda")
    ws = workspace(o5.o5_prelstm_bwd_workspace_bytes(dt, T, B, Do, D))
    o5.o5_prelstm_bwd(dt, T, B, Do, D, do_, y, dev_dt(dx, bf16), dW, db, ws)
    dW_ref, db_ref, _ = prelstm_backward(oo, ww, y_gpu, dd, T, B)
    assert_close("dW", host(dW), dW_ref, tol)
    assert_close("db", host(db), db_ref, tol)


def test_prelstm_tie_goes_to_first_replica_and_is_deterministic():
    need_gpu()
    banner("prelstm ties and determinism")
    T, B, Do, D = 2, 10, 64, 64
    rng = np.random.Generator(np.random.PCG64(5))
    o = rng.standard_normal((T * B, Do), dtype=np.float32)
    W = np.zeros((D, Do), np.float32)
    b = np.full(D, 0.5, np.float32)                   # every replica equal: all pooled features tie
    dx = rng.standard_normal((T * B, D), dtype=np.float32)
    outs = []
    for _ in range(2):
        y = torch.empty((T * B, D), dtype=torch.float32, device="cuda")
        x = torch.empty((T * B, D), dtype=torch.float32, device="cuda")
        o5.o5_prelstm_fwd(0, T, B, Do, D, dev_f32(o), dev_f32(W), dev_f32(b), y, x)
        dW = torch.empty((D, Do), dtype=torch.float32, device="cuda")
        db = torch.empty(D, dtype=torch.float32, device="cuda")
        o5.o5_prelstm_bwd(0, T, B, Do, D, dev_f32(o), y, dev_f32(dx), dW, db,
                          workspace(o5.o5_prelstm_bwd_workspace_bytes(0, T, B, Do, D)))
        outs.append((host(dW), host(db)))
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
    dW_ref, db_ref, _ = prelstm_backward(o.astype(np.float64), W, np.full((T * B, D), 0.5), dx.astype(np.float64),
                                         T, B)
    assert_close("dW", outs[0][0], dW_ref, TOL_F32)
    assert_close("db", outs[0][1], db_ref, TOL_F32)
