"""Pins for the surgery oracle (appendix "Surgery"): with zero-scale new
weights the widened LSTM computes exactly the old function on the old units
and keeps its new units at zero; with a small scale the old units move by an
amount second order in that scale; an Adam step on the widened vector
updates the old parameters exactly as on the old vector; widening to the
same shape is the identity; the new values are uniform in (-scale, scale)."""
import numpy as np
import pytest
import scipy.stats as sstats

from oracle.adam import adam_step
from oracle.lstm import lstm_forward
from oracle.ppo import heads_forward
from oracle.surgery import n_params, noise, split, widen

D, H, A1, D2, H2 = 6, 5, 4, 9, 8


def _old(seed):
    rng = np.random.default_rng(seed)
    n = n_params(D, H, A1)
    p = (rng.uniform(-0.5, 0.5, n)).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    v = (rng.random(n) * 1e-6).astype(np.float32)
    return p, m, v


def _run(flat, d, h, x, h0, c0, reset):
    P = split(flat, d, h, A1)
    hs, cs, _ = lstm_forward(x, P["Wx"], P["Wh"], P["b"], h0, c0, reset)
    z = heads_forward(hs.reshape(-1, h), P["Wp"], P["bp"])
    return hs, cs, z


def _inputs(seed, T=4, B=3):
    rng = np.random.default_rng(seed)
    x2 = rng.standard_normal((T, B, D2))
    h0 = rng.standard_normal((B, H)) * 0.3
    c0 = rng.standard_normal((B, H)) * 0.3
    reset = (rng.random((T, B)) < 0.2).astype(np.uint8)
    h02 = np.concatenate([h0, np.zeros((B, H2 - H))], axis=1)
    c02 = np.concatenate([c0, np.zeros((B, H2 - H))], axis=1)
    return x2, h0, c0, h02, c02, reset


def test_zero_scale_widening_preserves_the_function():
    p, m, v = _old(0)
    p2, _, _ = widen(p, m, v, D, H, A1, D2, H2, 0.0, seed=7)
    x2, h0, c0, h02, c02, reset = _inputs(1)
    hs, cs, z = _run(p, D, H, x2[..., :D], h0, c0, reset)
    hs2, cs2, z2 = _run(p2, D2, H2, x2, h02, c02, reset)   # the new inputs carry arbitrary values
    np.testing.assert_allclose(hs2[..., :H], hs, rtol=0, atol=1e-14)
    np.testing.assert_allclose(cs2[..., :H], cs, rtol=0, atol=1e-14)
    assert np.all(hs2[..., H:] == 0.0) and np.all(cs2[..., H:] == 0.0)
    np.testing.assert_allclose(z2, z, rtol=0, atol=1e-14)


def test_small_scale_moves_old_units_at_second_order():
    p, m, v = _old(2)
    x2, h0, c0, h02, c02, reset = _inputs(3)
    hs, _, _ = _run(p, D, H, x2[..., :D], h0, c0, reset)
    devs = []
    for scale in (1e-3, 1e-2):
        p2, _, _ = widen(p, m, v, D, H, A1, D2, H2, scale, seed=11)
        hs2, _, _ = _run(p2, D2, H2, x2, h02, c02, reset)
        devs.append(np.max(np.abs(hs2[..., :H] - hs)))
        assert np.max(np.abs(hs2[..., H:])) > 0.0
    # the old units read the new ones through weights of order scale, and the
    # new units' states are themselves of order scale: the change is second
    # order in the scale
    assert 0 < devs[0] < 1e-3 ** 2 * 10 and 50.0 < devs[1] / devs[0] < 200.0


def test_adam_on_widened_vector_updates_old_parameters_as_before():
    p, m, v = _old(4)
    p2, m2, v2 = widen(p, m, v, D, H, A1, D2, H2, 0.01, seed=5)
    rng = np.random.default_rng(6)
    g = rng.standard_normal(p.size) * 1e-2
    # the same gradient on the old positions of the widened vector
    marker = widen(np.arange(p.size, dtype=np.float32) + 1, m, v, D, H, A1, D2, H2, 0.0, seed=5)[0]
    old_pos = np.flatnonzero(marker)
    src = marker[old_pos].astype(np.int64) - 1
    g2 = rng.standard_normal(p2.size) * 1e-2
    g2[old_pos] = g[src]
    po, mo, vo = adam_step(p, m, v, g, 5e-5, 0.9, 0.999, 1e-8, 5.0, 7)
    pn, mn, vn = adam_step(p2, m2, v2, g2, 5e-5, 0.9, 0.999, 1e-8, 5.0, 7)
    assert np.array_equal(pn[old_pos], po[src]) and np.array_equal(mn[old_pos], mo[src])
    assert np.array_equal(vn[old_pos], vo[src])
    new_pos = np.setdiff1d(np.arange(p2.size), old_pos)
    assert np.all(m2[new_pos] == 0.0) and np.all(v2[new_pos] == 0.0)


def test_same_shape_is_identity():
    p, m, v = _old(8)
    out = widen(p, m, v, D, H, A1, D, H, 0.3, seed=1)
    for a, b in zip(out, (p, m, v)):
        assert np.array_equal(a, b)


def test_noise_is_uniform_and_seeded():
    u = noise(200_000, seed=3, scale=0.25)
    assert u.dtype == np.float32 and np.all(np.abs(u) < 0.25)
    counts, _ = np.histogram(u, bins=50, range=(-0.25, 0.25))
    assert sstats.chisquare(counts).pvalue > 1e-3
    assert np.array_equal(u, noise(200_000, 3, 0.25)) and not np.array_equal(u, noise(200_000, 4, 0.25))
    # the value is fp32(scale * (2U - 1)) with both factors fp32: sign symmetry of the construction
    assert abs(float(np.mean(u))) < 2e-3


def test_folding_a_constant_input_into_the_bias_preserves_the_function():
    from oracle.surgery import fold_input
    p, m, v = _old(9)
    Dk = 4
    E = np.random.default_rng(10).standard_normal(D - Dk)
    p2, m2, v2 = fold_input(p, m, v, D, H, A1, Dk, E)
    assert p2.size == n_params(Dk, H, A1)
    x2, h0, c0, _, _, reset = _inputs(11)
    xk = x2[..., :Dk]
    xfull = np.concatenate([xk, np.broadcast_to(E, xk.shape[:2] + (D - Dk,))], axis=-1)
    hs, cs, z = _run(p, D, H, xfull, h0, c0, reset)
    hs2, cs2, z2 = _run(p2, Dk, H, xk, h0, c0, reset)
    np.testing.assert_allclose(hs2, hs, rtol=0, atol=1e-13)
    np.testing.assert_allclose(cs2, cs, rtol=0, atol=1e-13)
    np.testing.assert_allclose(z2, z, rtol=0, atol=1e-13)
    # moments: the kept parameters keep theirs, the dropped columns' are gone
    Po, Pn = split(m, D, H, A1), split(m2, Dk, H, A1)
    assert np.array_equal(Pn["Wx"], Po["Wx"][:, :Dk]) and np.array_equal(Pn["b"], Po["b"])
    assert np.array_equal(Pn["Wh"], Po["Wh"]) and np.array_equal(Pn["Wp"], Po["Wp"])
