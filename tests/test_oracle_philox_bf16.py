"""Pins for the oracle's Philox4x64-10, Gumbel-max sampler and bf16 rounding
(CPU only).  Philox is compared with NumPy's independent Philox bit generator
(which increments its 256-bit counter before each block); the sampler with a
chi-square test against softmax(z); the rounding with PyTorch's float32 ->
bfloat16 conversion."""
import numpy as np
import pytest
import torch
from scipy import stats as sstats

from oracle.bf16 import bf16_bits, round_to_bf16
from oracle.philox import gumbel_max_sample, philox4x64, philox4x64_scalar, uniform_for_logits


def _numpy_block(ctr, key):
    # NumPy adds 1 to the counter (with carry) before producing a block.
    c = (ctr[0] | (ctr[1] << 64) | (ctr[2] << 128) | (ctr[3] << 192)) - 1
    c %= 1 << 256
    words = [(c >> (64 * i)) & ((1 << 64) - 1) for i in range(4)]
    bg = np.random.Philox(counter=np.array(words, dtype=np.uint64),
                          key=np.array(key, dtype=np.uint64))
    return [int(w) for w in bg.random_raw(4)]


@pytest.mark.parametrize("ctr,key", [
    ((1, 0, 0, 0), (0, 0)),
    ((7, 3, 4095, 0), (0, 0)),
    ((2, 1, 17, 12345), (2024, 0)),
    ((2 ** 64 - 1, 2 ** 63, 5, 2 ** 40 + 3), (2 ** 64 - 1, 2 ** 64 - 1)),
])
def test_philox_matches_numpy(ctr, key):
    ref = _numpy_block(list(ctr), key)
    assert philox4x64_scalar(ctr, key) == ref
    vec = philox4x64(*[np.uint64(w) for w in ctr], np.uint64(key[0]), np.uint64(key[1]))
    assert [int(w) for w in vec] == ref


def test_uniform_words_chi_square():
    us = uniform_for_logits(4096, (30, 8, 32, 4), seed=0, counter=0)
    u = np.concatenate([x.ravel() for x in us])
    assert u.min() > 0.0 and u.max() < 1.0
    counts, _ = np.histogram(u, bins=64, range=(0, 1))
    assert sstats.chisquare(counts).pvalue > 1e-3


def test_gumbel_max_frequencies_match_softmax():
    rng = np.random.default_rng(3)
    heads = (6, 3)
    z_row = np.concatenate([rng.normal(0, 1.5, 6), rng.normal(0, 0.5, 3), [0.0]])
    B = 200_000
    z = np.broadcast_to(z_row, (B, 10))
    act, logp, value, _ = gumbel_max_sample(z, heads, seed=11, counter=5)
    off = 0
    for k, n in enumerate(heads):
        p = np.exp(z_row[off:off + n] - z_row[off:off + n].max())
        p /= p.sum()
        counts = np.bincount(act[:, k], minlength=n)
        assert sstats.chisquare(counts, B * p).pvalue > 1e-3
        off += n
    assert np.all(value == 0.0)


def test_gumbel_max_logp_and_determinism():
    rng = np.random.default_rng(4)
    heads = (5, 4)
    z = rng.standard_normal((64, 10))
    a1, lp1, v1, _ = gumbel_max_sample(z, heads, 1, 0)
    a2, lp2, v2, _ = gumbel_max_sample(z, heads, 1, 0)
    a3, *_ = gumbel_max_sample(z, heads, 1, 1)
    assert np.array_equal(a1, a2) and np.array_equal(lp1, lp2)
    assert not np.array_equal(a1, a3)
    t = torch.from_numpy(z)
    ref = torch.distributions.Categorical(logits=t[:, :5]).log_prob(torch.from_numpy(a1[:, 0]).long()) + \
        torch.distributions.Categorical(logits=t[:, 5:9]).log_prob(torch.from_numpy(a1[:, 1]).long())
    np.testing.assert_allclose(lp1, ref.numpy(), rtol=0, atol=1e-13)
    np.testing.assert_array_equal(v1, z[:, 9])


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(5)
    a = np.concatenate([
        rng.standard_normal(10000).astype(np.float32) * 10.0 ** rng.uniform(-30, 30, 10000).astype(np.float32),
        np.array([0.0, -0.0, 1.0, 1.00390625, 1.005859375, 1.0078125, 3.3895314e38, -3.4e38,
                  1e-40, -1e-41, np.inf, -np.inf], np.float32),
    ]).astype(np.float32)
    ours = round_to_bf16(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(ours, ref)
    # exact ties round to even: 1 + 2^-8 -> 1, 1 + 3*2^-8 -> 1 + 2^-6
    assert round_to_bf16(np.float32(1.00390625)) == 1.0
    assert round_to_bf16(np.float32(1.01171875)) == 1.015625
    assert bf16_bits(np.float32(1.0)) == 0x3F80
    assert np.isnan(round_to_bf16(np.float32(np.nan)))
