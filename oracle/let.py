"""Oracle: learnable equivalent transformation for a linear layer (Eq.3) and
its initialisation (Sec. 4.1 training settings).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Layouts: X is [T, C_in] (tokens x channels); W is [C_out, C_in] (one row per
output channel, the transpose of the paper's C_in x C_out matrix); s, delta
are [C_in]; B is [C_out].

Readings of points the paper leaves open:
  * X~ = (X - delta) / s is evaluated as fl(fl(x - delta) * fl(1/s));
  * W~ = s (.) W is one fp32 product per element;
  * B~ = B + delta W uses the original W, summed in fp64, rounded once;
  * initialisation: s_c = sqrt(max_t |X[t,c]|) / sqrt(max_o |W[o,c]|) over
    all linears fed by the site (SmoothQuant with migration strength 0.5),
    each max floored at 1e-5; delta_c = mean_t X[t,c] (the channel mean).
"""
import numpy as np

LET_MAX_FLOOR = 1e-5


def let_x(X, s, delta, ft=np.float32):
    """X~ = (X - delta) (/) s  (Eq.3)."""
    X = np.asarray(X, dtype=ft)
    if ft == np.float32:
        rs = np.float32(1.0) / np.asarray(s, dtype=np.float32)
        return (X - np.asarray(delta, np.float32)[None, :]) * rs[None, :]
    return (X - np.asarray(delta, ft)[None, :]) / np.asarray(s, ft)[None, :]


def let_w(W, s, ft=np.float32):
    """W~ = s (.) W, s scaling input channel c of every output row (Eq.3)."""
    return np.asarray(W, dtype=ft) * np.asarray(s, dtype=ft)[None, :]


def let_bias(W, B, delta, ft=np.float32):
    """B~ = B + delta W  (Eq.3), fp64 sum over input channels, one rounding."""
    acc = np.asarray(W, np.float64) @ np.asarray(delta, np.float64)
    if B is not None:
        acc = acc + np.asarray(B, np.float64)
    return acc.astype(ft)


def let_fold(W, B, s, delta, ft=np.float32):
    """The folded operands of Eq.3: (W~, B~)."""
    return let_w(W, s, ft), let_bias(W, B, delta, ft)


def let_init(X, Ws):
    """SmoothQuant scale and Outlier-Suppression+ shift (Sec. 4.1).

    ``X`` [T, C] is the site's calibration input; ``Ws`` the weights
    ([C_out_l, C]) of every linear the site feeds.  Returns fp32 (s, delta).
    """
    X = np.asarray(X, np.float32)
    ax = np.max(np.abs(X), axis=0)
    aw = np.max(np.stack([np.max(np.abs(np.asarray(W, np.float32)), axis=0) for W in Ws]), axis=0)
    ax = np.maximum(ax, np.float32(LET_MAX_FLOOR))
    aw = np.maximum(aw, np.float32(LET_MAX_FLOOR))
    s = np.sqrt(ax) / np.sqrt(aw)
    delta = (np.sum(X.astype(np.float64), axis=0) / X.shape[0]).astype(np.float32)
    return s.astype(np.float32), delta
