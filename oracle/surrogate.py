"""Oracle: fp64 frozen-selection surrogate of one calibration step, for
finite-difference checks of the straight-through gradients.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

At a parameter point theta0 the step's forward is evaluated once in fp64 and
every discrete choice it makes is frozen: the rounding residual of each
round() in Eq.2 (for the codes and for the zero point), the clamp branch of
each element, the max/min positions of each group or token row, and whether
the h >= 1e-5 guard was active.  With those frozen, the forward is a smooth
function of (gamma logits, beta logits, s, delta) whose exact gradient at
theta0 is, by construction, the straight-through gradient (round has
derivative 1; clamp, max/min and the guard are differentiated exactly).  The
forward below is written independently of ``block.py``: it rebuilds Eq.2-4
from the frozen choices alone, so a central difference of it checks the
chain-rule bookkeeping of ``block.block_step``.
"""
import numpy as np

from .block import block_forward


def _frozen_choices(st):
    """The discrete choices of one quantiser call (rows = groups/tokens)."""
    u = st["u"].astype(np.float64)
    qmax = float(st["qmax"])
    c = st["c"].astype(np.float64)
    b = st["b"].astype(np.float64)
    r = st["r"].astype(np.float64)
    return dict(rho=np.rint(u) - u,
                rho_z=np.rint(b * r) - b * r,
                below=c < 0, above=c > qmax,
                i_mx=st["i_mx"], i_mn=st["i_mn"], hclamp=st["hclamp"], qmax=qmax)


def freeze(desc, X_q, Y_fp, params):
    """Run the fp64 forward at ``params`` and record its discrete choices."""
    _, S, L = block_forward(desc, X_q, Y_fp, params, ft=np.float64)
    return dict(act=[_frozen_choices(rec["act"]) if "act" in rec else None for rec in S],
                lwc=[_frozen_choices(rec["st"]) for rec in L])


def _quant_frozen(vals, gamma, beta, f):
    """Eq.2 on rows of ``vals`` with the choices ``f`` held fixed."""
    rows = np.arange(vals.shape[0])
    mx = vals[rows, f["i_mx"]]
    mn = vals[rows, f["i_mn"]]
    hi_clip = gamma * mx
    lo_clip = beta * mn
    h = np.where(f["hclamp"], 1e-5, (hi_clip - lo_clip) / f["qmax"])
    z = -(lo_clip / h + f["rho_z"])
    c = vals / h[:, None] + f["rho"] + z[:, None]
    q = np.where(f["below"], 0.0, np.where(f["above"], f["qmax"], c))
    return (q - z[:, None]) * h[:, None]


def surrogate_loss(desc, X_q, Y_fp, params, frozen):
    """fp64 loss of the step with every discrete choice frozen."""
    T = desc["T"]
    xhat = []
    for k, site in enumerate(desc["sites"]):
        x = np.asarray(X_q[k], np.float64)
        if site["let"]:
            x = (x - np.asarray(params["delta"][k], np.float64)) / np.asarray(params["s"][k], np.float64)
        if site["act_bits"] < 16:
            ones = np.ones(x.shape[0])
            x = _quant_frozen(x, ones, ones, frozen["act"][k])
        xhat.append(x)
    loss = 0.0
    for l, lin in enumerate(desc["linears"]):
        k = lin["site"]
        W = np.asarray(params["W"][l], np.float64)
        c_out, c_in = W.shape
        g = lin["group"]
        Wt = W * np.asarray(params["s"][k], np.float64)[None, :] if desc["sites"][k]["let"] else W
        gam = 1.0 / (1.0 + np.exp(-np.asarray(params["gamma_logit"][l], np.float64).reshape(-1)))
        bet = 1.0 / (1.0 + np.exp(-np.asarray(params["beta_logit"][l], np.float64).reshape(-1)))
        What = _quant_frozen(Wt.reshape(-1, g), gam, bet, frozen["lwc"][l]).reshape(c_out, c_in)
        B = params["B"][l] if params.get("B") is not None else None
        bias = np.zeros(c_out) if B is None else np.asarray(B, np.float64)
        if desc["sites"][k]["let"]:
            bias = bias + W @ np.asarray(params["delta"][k], np.float64)
        Y = xhat[k] @ What.T + bias[None, :]
        R = Y - np.asarray(Y_fp[l], np.float64)
        loss += float(np.sum(R * R)) / (T * c_out)
    return loss
