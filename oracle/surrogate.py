"""Oracle: fp64 frozen-selection surrogate of one calibration step, for
finite-difference checks of the straight-through gradients.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

At a parameter point theta0 the step's forward is evaluated once in fp64 and
every discrete choice it makes is frozen: the rounding residual of each
round() in Eq.2 (for the codes and for the zero point), the clamp branch of
each element, the max/min positions of each group or token row, and whether
the h >= 1e-5 guard was active.  (For PACT, whose own rule treats the
quantiser as the identity on the clipped weight, the frozen forward is that
identity plus the frozen offset to the quantised value.)  With those frozen,
the forward is a smooth
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


def _frozen_variant(st, params_l):
    """Frozen choices of a PACT / LSQ weight quantiser or a symmetric
    activation quantiser (``params_l`` = the variant's two parameters)."""
    u = st["u"].astype(np.float64)
    c = st["c"].astype(np.float64)
    qmax = float(st["qmax"])
    f = dict(rho=np.rint(u) - u, below=c < 0, above=c > qmax, hclamp=st["hclamp"], qmax=qmax,
             quant=st.get("quant"))
    if st.get("quant") == "pact":
        f.update(w0=st["wdq"].astype(np.float64), wt0=st["wt"].reshape(st["wdq"].shape).astype(np.float64),
                 p0=[np.asarray(p, np.float64).reshape(-1) for p in params_l])
    elif st.get("quant") == "lsq":
        zp = np.asarray(params_l[1], np.float64).reshape(-1)
        f.update(rho_z=np.rint(zp) - zp)
    elif st.get("sym"):
        f.update(i_ab=st["i_ab"], sgn=st["sgn"], qs=float(st["qs"]), z=st["z"].astype(np.float64))
    return f


def freeze(desc, X_q, Y_fp, params):
    """Run the fp64 forward at ``params`` and record its discrete choices."""
    _, S, L = block_forward(desc, X_q, Y_fp, params, ft=np.float64)
    act = []
    for k, rec in enumerate(S):
        if "act" not in rec:
            act.append(None)
        elif desc["sites"][k].get("act_sym"):
            act.append(_frozen_variant(rec["act"], None))
        else:
            act.append(_frozen_choices(rec["act"]))
    lwc = []
    for l, rec in enumerate(L):
        if desc["linears"][l].get("quant", "lwc") == "lwc":
            lwc.append(_frozen_choices(rec["st"]))
        else:
            lwc.append(_frozen_variant(rec["st"], (params["gamma_logit"][l], params["beta_logit"][l])))
    return dict(act=act, lwc=lwc)


def _pact_frozen(vals, hi, lo, f):
    """PACT's straight-through surrogate: the quantiser is the identity on the
    clipped weight, w^ = w^0 + m (w - w0) + [above](hi - hi0) + [below](lo - lo0)."""
    m = ~(f["below"] | f["above"])
    return (f["w0"] + m * (vals - f["wt0"]) + f["above"] * (hi - f["p0"][0])[:, None]
            + f["below"] * (lo - f["p0"][1])[:, None])


def _lsq_frozen(vals, step, zero, f):
    """LSQ with the rounding residuals (codes and zero point) and clamp
    branches frozen: w^ = (q - z')h, z' = z + rho_z, q = w/h + rho + z'."""
    h = np.where(f["hclamp"], 1e-5, step)
    z = zero + f["rho_z"]
    c = vals / h[:, None] + f["rho"] + z[:, None]
    q = np.where(f["below"], 0.0, np.where(f["above"], f["qmax"], c))
    return (q - z[:, None]) * h[:, None]


def _sym_frozen(vals, f):
    """Symmetric absmax quantiser with its choices frozen (absmax element and
    sign, residuals, clamp branches, floor)."""
    rows = np.arange(vals.shape[0])
    h = np.where(f["hclamp"], 1e-5, f["sgn"] * vals[rows, f["i_ab"]] / f["qs"])
    c = vals / h[:, None] + f["rho"] + f["z"][:, None]
    q = np.where(f["below"], 0.0, np.where(f["above"], f["qmax"], c))
    return (q - f["z"][:, None]) * h[:, None]


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
        if site["act_bits"] < 16 and site.get("act_sym"):
            x = _sym_frozen(x, frozen["act"][k])
        elif site["act_bits"] < 16:
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
        p1 = np.asarray(params["gamma_logit"][l], np.float64).reshape(-1)
        p2 = np.asarray(params["beta_logit"][l], np.float64).reshape(-1)
        quant = lin.get("quant", "lwc")
        if quant == "pact":
            What = _pact_frozen(Wt.reshape(-1, g), p1, p2, frozen["lwc"][l])
        elif quant == "lsq":
            What = _lsq_frozen(Wt.reshape(-1, g), p1, p2, frozen["lwc"][l])
        else:
            gam = 1.0 / (1.0 + np.exp(-p1))
            bet = 1.0 / (1.0 + np.exp(-p2))
            What = _quant_frozen(Wt.reshape(-1, g), gam, bet, frozen["lwc"][l])
        What = What.reshape(c_out, c_in)
        B = params["B"][l] if params.get("B") is not None else None
        bias = np.zeros(c_out) if B is None else np.asarray(B, np.float64)
        if desc["sites"][k]["let"]:
            bias = bias + W @ np.asarray(params["delta"][k], np.float64)
        Y = xhat[k] @ What.T + bias[None, :]
        R = Y - np.asarray(Y_fp[l], np.float64)
        loss += float(np.sum(R * R)) / (T * c_out)
    return loss
