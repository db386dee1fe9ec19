"""Pins for the unit-selection head (appendix "Neural Network Architecture":
unit embeddings carried beside the LSTM choose the unit to target): it
reduces to the pinned linear head when every row sees the same embeddings
and the query is the identity; central finite differences of the total loss
with respect to Wq, bq and h (with availability and head masks); the rows of
Wp and bp of that head receive no gradient."""
import numpy as np
import pytest

from oracle.ppo import head_logprob_entropy, head_offsets, ppo_loss_grad, unit_logits

HEADS = (5, 6, 3)   # head 1 selects one of 6 units
KU = 1


def _setup(seed, N=10, H=6, d=4, with_avail=False):
    rng = np.random.default_rng(seed)
    A1 = sum(HEADS) + 1
    h = rng.uniform(-1, 1, (N, H))
    Wp = rng.uniform(-0.6, 0.6, (A1, H))
    bp = rng.uniform(-0.3, 0.3, A1)
    Wq = rng.uniform(-0.6, 0.6, (d, H))
    bq = rng.uniform(-0.3, 0.3, d)
    E = rng.standard_normal((N, HEADS[KU], d))
    act = np.stack([rng.integers(0, n, N) for n in HEADS], axis=1)
    avail = None
    if with_avail:
        off = head_offsets(HEADS)
        avail = np.ones((N, off[-1]), np.uint8)
        blk = rng.random((N, HEADS[KU])) < 0.7
        blk[np.arange(N), act[:, KU]] = True
        avail[:, off[KU]:off[KU + 1]] = blk
    return h, Wp, bp, Wq, bq, E, act, avail, rng.standard_normal(N), rng.standard_normal(N)


def test_shared_embeddings_with_identity_query_reduce_to_the_linear_head():
    h, Wp, bp, _, _, _, act, _, adv, ret = _setup(0)
    N, H = h.shape
    off = head_offsets(HEADS)
    bp[off[KU]:off[KU + 1]] = 0.0
    E = np.broadcast_to(Wp[off[KU]:off[KU + 1]], (N, HEADS[KU], H))
    unit = dict(head=KU, Wq=np.eye(H), bq=np.zeros(H), E=E)
    lo = np.zeros(N)
    a = ppo_loss_grad(h, Wp, bp, act, lo, adv, ret, HEADS)
    b = ppo_loss_grad(h, Wp, bp, act, lo, adv, ret, HEADS, unit=unit)
    assert b[0]["total"] == pytest.approx(a[0]["total"], abs=1e-13)
    np.testing.assert_allclose(b[1], a[1], rtol=0, atol=1e-13)       # dh
    np.testing.assert_allclose(b[4], a[4], rtol=0, atol=1e-13)       # logits
    # the linear head's own rows of Wp, bp get nothing in the unit form
    assert np.all(b[2][off[KU]:off[KU + 1]] == 0.0) and np.all(b[3][off[KU]:off[KU + 1]] == 0.0)


@pytest.mark.parametrize("with_avail,with_mask", [(False, False), (True, True)])
def test_unit_head_central_finite_differences(with_avail, with_mask):
    h, Wp, bp, Wq, bq, E, act, avail, adv, ret = _setup(1, with_avail=with_avail)
    N = h.shape[0]
    mask = (np.random.default_rng(2).random((N, len(HEADS))) < 0.75).astype(np.float64) if with_mask else None
    unit = dict(head=KU, Wq=Wq, bq=bq, E=E)
    z = ppo_loss_grad(h, Wp, bp, act, np.zeros(N), adv, ret, HEADS, unit=unit, avail=avail)[4]
    logp, _, _ = head_logprob_entropy(z, act, HEADS, avail)
    m = np.ones_like(logp) if mask is None else mask
    shift = np.linspace(-0.5, 0.5, N) + 0.013
    logp_old = np.where(m != 0, logp, 0.0).sum(axis=1) + shift

    def total(h_, Wq_, bq_):
        u = dict(head=KU, Wq=Wq_, bq=bq_, E=E)
        return ppo_loss_grad(h_, Wp, bp, act, logp_old, adv, ret, HEADS, 0.2, 0.7, 0.05, mask, avail, u)[0]["total"]

    out = ppo_loss_grad(h, Wp, bp, act, logp_old, adv, ret, HEADS, 0.2, 0.7, 0.05, mask, avail, unit)
    dh, (dWq, dbq) = out[1], out[5]
    eps = 1e-6
    for name, arr, analytic in (("h", h, dh), ("Wq", Wq, dWq), ("bq", bq, dbq)):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            p_, m_ = arr.copy(), arr.copy()
            p_[idx] += eps
            m_[idx] -= eps
            args_p = {"h_": h, "Wq_": Wq, "bq_": bq}
            args_m = dict(args_p)
            args_p[name + "_"], args_m[name + "_"] = p_, m_
            num[idx] = (total(**args_p) - total(**args_m)) / (2 * eps)
        assert np.max(np.abs(num - analytic)) / np.max(np.abs(num)) < 1e-7, name


def test_unit_logits_are_dot_products():
    rng = np.random.default_rng(3)
    h, Wq, bq = rng.standard_normal((2, 3)), rng.standard_normal((4, 3)), rng.standard_normal(4)
    E = rng.standard_normal((2, 5, 4))
    q, z = unit_logits(h, Wq, bq, E)
    for n in range(2):
        for u in range(5):
            assert z[n, u] == pytest.approx(sum((h[n] @ Wq[j] + bq[j]) * E[n, u, j] for j in range(4)), abs=1e-12)
