"""Surgery on the flat parameter vector: widening the LSTM and extending its
input, in fp64 / exact copies.

Test infrastructure (see the package docstring).

Appendix "Surgery" (paragraphs "Changing the architecture", "Changing the
Observation Space", "Smooth Training Restart"; subsection "Continual
Transfer via Surgery"):
* widening a layer keeps the old weights in place, gives the new rows random
  values and zeroes the next layer's weights that read the new units, so the
  next layer's output is unchanged;
* for the LSTM (2048 -> 4096 units) the recurrence makes that separation
  impossible; the new weights get random values much smaller than the
  existing ones;
* new observations consumed by a weight matrix get zero weights, so the
  output is unchanged;
* training restarts with learning rate 0 for a while so that Adam's moments
  adapt to the new shapes.

Parameter layout (one flat fp32 vector, as the optimizer step uses it):
Wx [4H, D], Wh [4H, H], b [4H], Wp [A1, H], bp [A1]; gate blocks (i, f, g, o)
along 4H.  Widening maps (D, H) -> (D2, H2) with D2 >= D, H2 >= H.

Readings where the paper is silent: every new LSTM parameter (rows of new
units, columns of Wh reading new units, new biases) is uniform in
(-scale, scale); LSTM columns reading new inputs are 0; head columns reading
new units are 0; Adam's moments are copied for old parameters and 0 for new
ones.  The uniform values come from Philox4x64-10: new-vector element e uses
word (e mod 4) of the block with counter (e div 4, 0, 0, 0) and key
(seed, 1), U = ((word >> 40) + 1/2) / 2^24 and value
fp32(scale * (2U - 1)) (both factors fp32, so the product is one rounding).
With scale = 0 the widened network computes exactly the old function on
the old units, and its new units stay at zero.
"""
import numpy as np

from oracle.philox import philox4x64

_U64 = np.uint64


def sizes(D, H, A1):
    return {"Wx": (4 * H, D), "Wh": (4 * H, H), "b": (4 * H,), "Wp": (A1, H), "bp": (A1,)}


def n_params(D, H, A1):
    return sum(int(np.prod(s)) for s in sizes(D, H, A1).values())


def split(flat, D, H, A1):
    out, o = {}, 0
    for k, s in sizes(D, H, A1).items():
        n = int(np.prod(s))
        out[k] = np.asarray(flat[o:o + n]).reshape(s)
        o += n
    return out


def noise(n, seed, scale):
    """fp32 uniform values in (-scale, scale) for new-vector elements 0..n-1."""
    e = np.arange(n, dtype=np.uint64)
    words = philox4x64(e >> _U64(2), _U64(0), _U64(0), _U64(0), _U64(seed), _U64(1))
    sel = (e & _U64(3)).astype(np.int64)
    w = np.choose(sel, words)
    u = ((w >> _U64(40)).astype(np.float64) + 0.5) * 2.0 ** -24
    return (np.float64(np.float32(scale)) * (2.0 * u - 1.0)).astype(np.float32)


def widen(p, m, v, D, H, A1, D2, H2, scale, seed):
    """Widened (p, m, v) flat fp32 vectors for (D2, H2)."""
    assert D2 >= D and H2 >= H
    old_p, old_m, old_v = (split(a, D, H, A1) for a in (p, m, v))
    n2 = n_params(D2, H2, A1)
    rnd = split(noise(n2, seed, scale), D2, H2, A1)
    new_p = {k: np.array(a, np.float32) for k, a in rnd.items()}
    new_m = {k: np.zeros(s, np.float32) for k, s in sizes(D2, H2, A1).items()}
    new_v = {k: np.zeros(s, np.float32) for k, s in sizes(D2, H2, A1).items()}
    for g in range(4):
        rows_old = slice(g * H, (g + 1) * H)
        rows_new = slice(g * H2, g * H2 + H)
        for tgt, src in ((new_p, old_p), (new_m, old_m), (new_v, old_v)):
            tgt["Wx"][rows_new, :D] = src["Wx"][rows_old]
            tgt["Wh"][rows_new, :H] = src["Wh"][rows_old]
            tgt["b"][rows_new] = src["b"][rows_old]
        # old units do not read the new inputs
        new_p["Wx"][rows_new, D:] = 0.0
    for tgt, src in ((new_p, old_p), (new_m, old_m), (new_v, old_v)):
        tgt["Wp"][:, :H] = src["Wp"]
        tgt["bp"][:] = src["bp"]
    # the heads do not read the new units
    new_p["Wp"][:, H:] = 0.0
    cat = lambda d: np.concatenate([d[k].ravel() for k in ("Wx", "Wh", "b", "Wp", "bp")])
    return cat(new_p), cat(new_m), cat(new_v)


def fold_input(p, m, v, D, H, A1, Dk, E):
    """Fold the last D - Dk LSTM inputs, a constant vector E, into the bias
    (appendix "Bloopers", subsection "Zero Team Spirit Embedding": a constant
    part of the input of a fully-connected layer is the same as a modified
    bias, B' = W [0, E] + B):
    b' = b + Wx[:, Dk:] E and Wx' = Wx[:, :Dk].  The moments of the dropped
    columns are discarded; every other parameter keeps its moments."""
    parts = [split(a, D, H, A1) for a in (p, m, v)]
    outs = []
    for i, P in enumerate(parts):
        Q = {k: np.array(a, copy=True) for k, a in P.items()}
        Q["Wx"] = np.ascontiguousarray(P["Wx"][:, :Dk])
        if i == 0:
            Q["b"] = (P["b"].astype(np.float64) + P["Wx"][:, Dk:].astype(np.float64) @ np.asarray(E, np.float64))
        outs.append(np.concatenate([np.asarray(Q[k], np.float64).ravel() for k in ("Wx", "Wh", "b", "Wp", "bp")]))
    return tuple(outs)
