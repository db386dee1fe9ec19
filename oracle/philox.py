"""Philox4x64-10 and Gumbel-max action sampling.

Test infrastructure (see the package docstring).

The rollout policy samples an action from its output distribution at every
timestep (section "Training System", subsection "Playing Dota using AI").  The
paper does not say how; here each categorical head is drawn with the
Gumbel-max rule, argmax_a (z_a + G_a) with G = -ln(-ln U), U uniform on
(0, 1), using the counter-based generator Philox4x64 with 10 rounds
(Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3",
SC'11).  A counter-based generator lets every logit draw its own noise with
no state carried between threads.

Philox4x64 round (two 64x64 -> 128-bit products per round):
    (hi0, lo0) = M0 * c0          (hi1, lo1) = M1 * c2
    c' = (hi1 ^ c1 ^ k0,  lo1,  hi0 ^ c3 ^ k1,  lo0)
    k' = (k0 + W0, k1 + W1)        (mod 2^64)
with M0 = 0xD2E7470EE14C6C93, M1 = 0xCA5A826395121157 and the Weyl
increments W0 = 0x9E3779B97F4A7C15 (golden ratio), W1 = 0xBB67AE8584CAA73B
(sqrt(3) - 1).  The key update happens between rounds.

Counter assignment (the convention used here): the noise for logit ``a`` of
head ``k`` in row ``b`` is output word ``a mod 4`` of the block with counter
(a div 4, k, b, counter) and key (seed, 0).  U = ((word >> 40) + 1/2) / 2^24.
"""
import numpy as np

M0 = 0xD2E7470EE14C6C93
M1 = 0xCA5A826395121157
W0 = 0x9E3779B97F4A7C15
W1 = 0xBB67AE8584CAA73B
_MASK64 = (1 << 64) - 1
_U64 = np.uint64


def philox4x64_scalar(ctr, key, rounds=10):
    """Reference generator on Python integers (one block)."""
    c = [int(w) & _MASK64 for w in ctr]
    k = [int(w) & _MASK64 for w in key]
    for r in range(rounds):
        if r > 0:
            k = [(k[0] + W0) & _MASK64, (k[1] + W1) & _MASK64]
        p0 = M0 * c[0]
        p1 = M1 * c[2]
        c = [(p1 >> 64) ^ c[1] ^ k[0], p1 & _MASK64,
             (p0 >> 64) ^ c[3] ^ k[1], p0 & _MASK64]
    return c


def _mulhilo(a, b):
    """128-bit product of uint64 arrays a and b, as (hi, lo), via 32-bit limbs."""
    m32 = _U64(0xFFFFFFFF)
    s32 = _U64(32)
    a0, a1 = a & m32, a >> s32
    b0, b1 = b & m32, b >> s32
    p00, p01, p10, p11 = a0 * b0, a0 * b1, a1 * b0, a1 * b1
    mid = (p00 >> s32) + (p01 & m32) + (p10 & m32)
    lo = (p00 & m32) | ((mid & m32) << s32)
    hi = p11 + (p01 >> s32) + (p10 >> s32) + (mid >> s32)
    return hi, lo


def philox4x64(c0, c1, c2, c3, k0, k1, rounds=10):
    """Vectorised generator: counter words and key words are uint64 arrays
    (broadcastable).  Returns the four output words."""
    with np.errstate(over="ignore"):
        c0, c1, c2, c3 = (np.asarray(w, dtype=np.uint64) for w in (c0, c1, c2, c3))
        k0 = np.asarray(k0, dtype=np.uint64)
        k1 = np.asarray(k1, dtype=np.uint64)
        for r in range(rounds):
            if r > 0:
                k0 = k0 + _U64(W0)
                k1 = k1 + _U64(W1)
            hi0, lo0 = _mulhilo(_U64(M0), c0)
            hi1, lo1 = _mulhilo(_U64(M1), c2)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


def uniform_for_logits(B, head_sizes, seed, counter):
    """U in (0,1) for every (row b, head k, logit a): list over k of [B, n_k]."""
    out = []
    b = np.arange(B, dtype=np.uint64)[:, None]
    for k, n in enumerate(head_sizes):
        a = np.arange(n, dtype=np.uint64)[None, :]
        words = philox4x64(a >> _U64(2), _U64(k), b, _U64(counter),
                           _U64(seed), _U64(0))
        sel = (a & _U64(3)).astype(np.int64)
        w = np.choose(np.broadcast_to(sel, (B, n)), [np.broadcast_to(x, (B, n)) for x in words])
        u = ((w >> _U64(40)).astype(np.float64) + 0.5) * 2.0 ** -24
        out.append(u)
    return out


def gumbel_max_sample(z, head_sizes, seed, counter, avail=None):
    """Sample one action per head by argmax(z + Gumbel noise) over the
    head's available logits (avail [B, A], 1 = available, or None).

    z is [B, A+1] (last column = value).  Returns (act [B,K] int32,
    logp [B] = sum_k log softmax(z_k)[a_k] over the available logits,
    value [B], scores list of [B, n_k] = z_k + G for near-tie inspection,
    -inf where unavailable).  A head with no available logit gets action -1
    and adds nothing to logp.
    """
    z = np.asarray(z, np.float64)
    B = z.shape[0]
    us = uniform_for_logits(B, head_sizes, seed, counter)
    A = int(sum(head_sizes))
    av_all = np.ones((B, A), bool) if avail is None else np.asarray(avail) != 0
    act = np.empty((B, len(head_sizes)), dtype=np.int32)
    logp = np.zeros(B)
    scores = []
    off = 0
    rows = np.arange(B)
    for k, n in enumerate(head_sizes):
        zk = z[:, off:off + n]
        av = av_all[:, off:off + n]
        some = av.any(axis=1)
        s = np.where(av, zk - np.log(-np.log(us[k])), -np.inf)
        a = np.argmax(s, axis=1)          # first maximum wins ties
        act[:, k] = np.where(some, a, -1)
        zmax = np.where(av, zk, -np.inf).max(axis=1, keepdims=True)
        zmax = np.where(some[:, None], zmax, 0.0)
        se = np.where(av, np.exp(zk - zmax), 0.0).sum(axis=1)
        lse = zmax[:, 0] + np.log(np.where(some, se, 1.0))
        logp += np.where(some, zk[rows, a] - lse, 0.0)
        scores.append(s)
        off += n
    return act, logp, z[:, off], scores
