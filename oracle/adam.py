"""Adam with the paper's per-parameter gradient clip, in fp64.

Test infrastructure (see the package docstring).

Subsection "Optimizing the Policy": the optimizer is Adam, and each gradient
element is first clipped to within +-5 sqrt(v), v being the running estimate
of the second moment of the unclipped gradient.  Table "Hyperparameters":
beta1 = 0.9, beta2 = 0.999, learning rate 5e-5 (baseline).

Readings where the paper is silent: bias correction on; epsilon = 1e-8 added
outside the square root; no weight decay; 1-based step counter.  The clip uses
the bias-corrected second moment that already includes the current
(unclipped) gradient; the clipped gradient feeds only the first moment.
``clip_k <= 0`` turns the clip off (plain Adam).
"""
import numpy as np

from .precision import F


def adam_step(p, m, v, g, lr, beta1, beta2, eps, clip_k, step):
    """One update.  Returns new (p, m, v) as fp64 arrays; inputs untouched."""
    p = np.asarray(p, F())
    m = np.asarray(m, F())
    v = np.asarray(v, F())
    g = np.asarray(g, F())
    v_new = beta2 * v + (1.0 - beta2) * g * g
    v_hat = v_new / (1.0 - beta2 ** step)
    if clip_k > 0:
        bound = clip_k * np.sqrt(v_hat)
        g_used = np.minimum(np.maximum(g, -bound), bound)
    else:
        g_used = g
    m_new = beta1 * m + (1.0 - beta1) * g_used
    m_hat = m_new / (1.0 - beta1 ** step)
    p_new = p - lr * m_hat / (np.sqrt(v_hat) + eps)
    return p_new, m_new, v_new
