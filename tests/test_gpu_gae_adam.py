"""GPU parity: o5_gae, o5_segments_to_samples, o5_adam_step, o5_f32_to_bf16
against the fp64 oracle on identical seeded inputs."""
import numpy as np
import pytest
import torch

from oracle.adam import adam_step
from oracle.bf16 import bf16_bits
from oracle.gae import gae, segments_to_samples
from paper_1912_06680_amd import o5
from tests.gpu_util import TOL_F32, assert_close, banner, dev, dev_f32, host, need_gpu

pytestmark = pytest.mark.gpu


def _gae_inputs(L, S, p_done, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    r = rng.standard_normal((L, S), dtype=np.float32)
    v = rng.standard_normal((L + 1, S), dtype=np.float32)
    d = (rng.random((L, S)) < p_done).astype(np.uint8)
    return r, v, d


# (L, S): the four kernels (wave scan for S <= 256, and for L > 256 up to S
# = 4096; chunked lanes for L <= 256 and 256 < S < 32768; otherwise a lane
# per 4 segments when S % 4 == 0, else a lane per segment), ragged L (not a
# multiple of 64, of the 16 chunks or of the unroll; empty trailing chunks),
# ragged S (not a multiple of 64), a single segment/step.
@pytest.mark.parametrize("L,S,gamma,lam", [
    (1, 1, 0.998, 0.95), (16, 8, 0.998, 0.95), (256, 128, 0.998, 0.95), (37, 3, 0.9, 0.8),
    (300, 7, 0.998, 0.95), (256, 4097, 0.998, 0.95), (45, 5000, 0.99, 0.9), (256, 128, 0.998, 0.0),
    (256, 4100, 0.998, 1.0), (250, 4500, 0.998, 0.95), (9, 5000, 0.998, 0.95), (1, 4200, 0.998, 0.95),
    (256, 20000, 0.998, 0.95), (257, 4201, 0.998, 0.95), (600, 4160, 0.99, 0.9), (256, 32772, 0.998, 0.95),
    (37, 40000, 0.99, 0.9), (3, 32769, 0.998, 0.95),
    (256, 1000, 0.998, 0.95), (255, 257, 0.99, 0.9), (17, 300, 0.998, 0.95), (300, 1000, 0.998, 0.95),
])
def test_gae_matches_oracle(L, S, gamma, lam):
    need_gpu()
    banner(f"gae L={L} S={S} gamma={gamma} lambda={lam}")
    r, v, d = _gae_inputs(L, S, 0.05, seed=L * 7 + S)
    adv_ref, ret_ref = gae(r, v, d, gamma, lam)
    adv = torch.empty((L, S), dtype=torch.float32, device="cuda")
    ret = torch.empty_like(adv)
    o5.o5_gae(L, S, dev(r), dev(v), dev(d), gamma, lam, adv, ret)
    assert_close("adv", host(adv), adv_ref, TOL_F32)
    assert_close("ret", host(ret), ret_ref, TOL_F32)


def test_gae_is_deterministic():
    need_gpu()
    banner("gae determinism")
    r, v, d = _gae_inputs(256, 9000, 0.01, 3)
    outs = []
    for _ in range(2):
        adv = torch.empty((256, 9000), dtype=torch.float32, device="cuda")
        ret = torch.empty_like(adv)
        o5.o5_gae(256, 9000, dev(r), dev(v), dev(d), 0.998, 0.95, adv, ret)
        outs.append(host(adv))
    assert np.array_equal(outs[0], outs[1])


@pytest.mark.parametrize("L,S,T", [(256, 128, 16), (16, 8, 16), (12, 5, 3)])
def test_segments_to_samples_bit_exact(L, S, T):
    need_gpu()
    banner(f"segments_to_samples L={L} S={S} T={T}")
    r, v, d = _gae_inputs(L, S, 0.1, 11)
    B = S * L // T
    a_s = torch.empty((T, B), dtype=torch.float32, device="cuda")
    r_s = torch.empty_like(a_s)
    reset = torch.empty((T, B), dtype=torch.uint8, device="cuda")
    o5.o5_segments_to_samples(L, S, T, dev(r), dev(v[:L]), dev(d), a_s, r_s, reset)
    ea, er, erst = segments_to_samples(r.astype(np.float64), v[:L].astype(np.float64), d, T)
    assert np.array_equal(host(a_s), ea) and np.array_equal(host(r_s), er)
    assert np.array_equal(reset.cpu().numpy(), erst)


def test_segments_to_samples_beyond_2_pow_31_elements():
    """L * S = 16 * (2^27 + 8) > 2^31 elements (about 38 GB of buffers): the
    cut indexes in 64 bits.  Values are distinct integers (exact in fp32)
    so a misplaced element cannot pass; sampled segments are cut by the
    oracle from their own columns and compared bit for bit."""
    need_gpu()
    L, T = 16, 4
    S = (1 << 27) + 8
    J = L // T
    banner(f"segments_to_samples L={L} S={S} T={T} (L*S = {L * S} > 2^31)")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)
    adv = torch.randint(0, 1 << 24, (L, S), generator=gen, device="cuda").to(torch.float32)
    ret = torch.randint(0, 1 << 24, (L, S), generator=gen, device="cuda").to(torch.float32)
    done = (torch.rand((L, S), generator=gen, device="cuda") < 0.3).to(torch.uint8)
    B = S * J
    a_s = torch.empty((T, B), dtype=torch.float32, device="cuda")
    r_s = torch.empty_like(a_s)
    reset = torch.empty((T, B), dtype=torch.uint8, device="cuda")
    o5.o5_segments_to_samples(L, S, T, adv, ret, done, a_s, r_s, reset)
    torch.cuda.synchronize()
    segs = torch.tensor([0, 1, 12345, (1 << 27) - 1, 1 << 27, S - 1], device="cuda")
    cols = (segs[:, None] * J + torch.arange(J, device="cuda")[None]).reshape(-1)
    ea, er, erst = segments_to_samples(host(adv[:, segs]), host(ret[:, segs]), done[:, segs].cpu().numpy(), T)
    assert np.array_equal(host(a_s[:, cols]), ea)
    assert np.array_equal(host(r_s[:, cols]), er)
    assert np.array_equal(reset[:, cols].cpu().numpy(), erst)
    del adv, ret, done, a_s, r_s, reset
    torch.cuda.empty_cache()


def _adam_inputs(n, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    p = rng.standard_normal(n, dtype=np.float32) * 0.05
    m = rng.standard_normal(n, dtype=np.float32) * 1e-3
    v = (rng.random(n, dtype=np.float32) * 1e-5).astype(np.float32)
    g = (rng.standard_normal(n, dtype=np.float32) * (10.0 ** rng.uniform(-5, -1, n))).astype(np.float32)
    g[::97] *= 300.0  # spikes beyond 5 sqrt(v_hat)
    return p, m, v, g


@pytest.mark.parametrize("n,step,clip_k,bf16_out", [
    (1, 1, 5.0, False), (7, 3, 5.0, True), (1000003, 10, 5.0, True), (4096, 2, 0.0, False),
])
def test_adam_matches_oracle(n, step, clip_k, bf16_out):
    need_gpu()
    banner(f"adam n={n} step={step} clip_k={clip_k} bf16_out={bf16_out}")
    p, m, v, g = _adam_inputs(n, n + step)
    lr = 5e-5
    p_ref, m_ref, v_ref = adam_step(p, m, v, g, lr, 0.9, 0.999, 1e-8, clip_k, step)
    tp, tm, tv, tg = dev_f32(p), dev_f32(m), dev_f32(v), dev_f32(g)
    pb = torch.empty(n, dtype=torch.bfloat16, device="cuda") if bf16_out else None
    o5.o5_adam_step(n, tp, tm, tv, tg, pb, lr, 0.9, 0.999, 1e-8, clip_k, step)
    pg = host(tp)
    # the stored parameter is fp32: allow one fp32 rounding of it on top of the tolerance
    dref = p_ref - p.astype(np.float64)
    ulp = np.spacing(np.abs(p_ref).astype(np.float32)).astype(np.float64)
    err = np.abs(pg - p_ref)
    bound = TOL_F32 * np.max(np.abs(dref)) + ulp
    print(f"    p: max(err/bound)={np.max(err / bound):.3f}", flush=True)
    assert np.all(err <= bound)
    assert_close("m", host(tm), m_ref, TOL_F32)
    assert_close("v", host(tv), v_ref, TOL_F32)
    if bf16_out:
        # property: the bf16 copy is the round-to-nearest-even of the new fp32
        # parameter (torch's conversion, itself pinned against the oracle's rounding)
        assert torch.equal(pb.view(torch.int16), tp.to(torch.bfloat16).view(torch.int16))


def test_adam_full_size_sampled_elements():
    """The full step's parameter count (the 4096-unit LSTM with 4096 inputs
    and the heads, 134.5M; and 158.5M): the update is elementwise, so the
    oracle checks a sample of elements, the first and last ones included."""
    need_gpu()
    for n in (134_541_387, 158_502_815):
        banner(f"adam full size n={n}")
        p, m, v, g = _adam_inputs(n, 7)
        tp, tm, tv, tg = dev_f32(p), dev_f32(m), dev_f32(v), dev_f32(g)
        pb = torch.empty(n, dtype=torch.bfloat16, device="cuda")
        o5.o5_adam_step(n, tp, tm, tv, tg, pb, 5e-5, 0.9, 0.999, 1e-8, 5.0, 3)
        rng = np.random.Generator(np.random.PCG64(n))
        idx = np.unique(np.concatenate([np.arange(64), n - 64 + np.arange(64), rng.integers(0, n, 1 << 20)]))
        p_ref, m_ref, v_ref = adam_step(p[idx], m[idx], v[idx], g[idx], 5e-5, 0.9, 0.999, 1e-8, 5.0, 3)
        ti = torch.from_numpy(idx).to("cuda")
        pg = tp[ti].cpu().numpy().astype(np.float64)
        dref = p_ref - p[idx].astype(np.float64)
        ulp = np.spacing(np.abs(p_ref).astype(np.float32)).astype(np.float64)
        bound = TOL_F32 * np.max(np.abs(dref)) + ulp
        assert np.all(np.abs(pg - p_ref) <= bound)
        assert_close("m", tm[ti].cpu().numpy(), m_ref, TOL_F32)
        assert_close("v", tv[ti].cpu().numpy(), v_ref, TOL_F32)
        assert torch.equal(pb[ti].view(torch.int16), tp[ti].to(torch.bfloat16).view(torch.int16))
        del tp, tm, tv, tg, pb
        torch.cuda.empty_cache()


def test_adam_lr_zero_leaves_parameters_bitwise_and_is_deterministic():
    need_gpu()
    banner("adam lr=0 and determinism")
    n = 100003
    p, m, v, g = _adam_inputs(n, 5)
    tp, tm, tv, tg = dev_f32(p), dev_f32(m), dev_f32(v), dev_f32(g)
    o5.o5_adam_step(n, tp, tm, tv, tg, None, 0.0, 0.9, 0.999, 1e-8, 5.0, 4)
    assert np.array_equal(tp.cpu().numpy(), p)
    assert not np.array_equal(tm.cpu().numpy(), m)
    runs = []
    for _ in range(2):
        tp, tm, tv = dev_f32(p), dev_f32(m), dev_f32(v)
        o5.o5_adam_step(n, tp, tm, tv, tg, None, 5e-5, 0.9, 0.999, 1e-8, 5.0, 4)
        runs.append(tp.cpu().numpy())
    assert np.array_equal(runs[0], runs[1])


@pytest.mark.parametrize("n", [1, 9, 1 << 20])
def test_f32_to_bf16_matches_oracle_rounding(n):
    need_gpu()
    banner(f"f32_to_bf16 n={n}")
    rng = np.random.Generator(np.random.PCG64(n))
    a = (rng.standard_normal(n, dtype=np.float32) * np.float32(10.0) ** rng.integers(-20, 20, n)).astype(np.float32)
    a[:: max(1, n // 5)] = np.float32(1.00390625)  # exact ties
    dst = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    o5.o5_f32_to_bf16(n, dev_f32(a), dst)
    got = dst.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got, bf16_bits(a))


def test_f32_to_bf16_every_bit_pattern():
    """All 2^32 float32 bit patterns through the conversion kernel, in chunks
    of 2^28, against round-to-nearest-even written out on the bits (torch
    integer arithmetic): (u + 0x7fff + ((u >> 16) & 1)) >> 16, and for NaN
    the top half with the quiet bit set."""
    need_gpu()
    banner("f32_to_bf16 all 2^32 patterns")
    chunk = 1 << 28
    dst = torch.empty(chunk, dtype=torch.bfloat16, device="cuda")
    for c0 in range(0, 1 << 32, chunk):
        u = torch.arange(c0, c0 + chunk, dtype=torch.int64, device="cuda")
        src = torch.where(u >= (1 << 31), u - (1 << 32), u).to(torch.int32).view(torch.float32)
        o5.o5_f32_to_bf16(chunk, src, dst)
        got = dst.view(torch.int16).to(torch.int64) & 0xFFFF
        nan = (u & 0x7FFFFFFF) > 0x7F800000
        exp = torch.where(nan, (u >> 16) | 0x40, (u + 0x7FFF + ((u >> 16) & 1)) >> 16) & 0xFFFF
        bad = int((got != exp).sum())
        assert bad == 0, f"chunk {c0:#x}: {bad} patterns differ"
        del u, src, got, nan, exp
    torch.cuda.synchronize()


def test_f32_to_bf16_every_top_pattern():
    """Every sign, exponent and top-7-mantissa pattern (all 2^16 upper
    halves) with lower halves 0, 1, 0x7fff, 0x8000 (the tie), 0x8001 and
    0xffff: ties to even both ways, carries into the exponent, overflow to
    infinity, subnormals, infinities and NaN.  Non-NaN inputs give the
    oracle's bits; NaN gives the input's top half with the quiet bit set."""
    need_gpu()
    banner("f32_to_bf16 every top pattern")
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lo = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF], dtype=np.uint32)
    u = (hi[:, None] | lo[None, :]).ravel()
    a = u.view(np.float32)
    dst = torch.empty(a.size, dtype=torch.bfloat16, device="cuda")
    o5.o5_f32_to_bf16(a.size, dev_f32(a), dst)
    got = dst.view(torch.int16).cpu().numpy().view(np.uint16)
    nan = np.isnan(a)
    assert np.array_equal(got[~nan], bf16_bits(a[~nan]))
    assert np.array_equal(got[nan], ((u[nan] >> 16) | 0x40).astype(np.uint16))
