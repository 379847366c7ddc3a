"""Oracle: the AdamW update used to train the LWC and LET parameters
(Sec. 4.1 training settings: AdamW, zero weight decay, learning rate 5e-3 for
the clipping logits and 1e-2 for the equivalent-transformation parameters).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

The paper fixes neither the moment decay rates nor epsilon; the oracle uses
beta1 = 0.9, beta2 = 0.999, eps = 1e-8 with bias correction (decoupled weight
decay applied as p *= 1 - lr*wd before the moment step).
"""
import numpy as np

LR_LWC = 5e-3
LR_LET = 1e-2


def adamw(p, g, m, v, step, lr, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0):
    """One AdamW step in fp64.  ``step`` counts from 1.  Returns (p, m, v)."""
    p = np.asarray(p, np.float64) * (1.0 - lr * wd)
    g = np.asarray(g, np.float64)
    m = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** step)
    v_hat = v / (1.0 - beta2 ** step)
    p = p - lr * m_hat / (np.sqrt(v_hat) + eps)
    return p, m, v
