"""Oracle: one calibration step over a transformer block's linear sub-graph.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Follows Algorithm 1's inner-loop body (apply LET, quantise with LWC, run the
quantised block on x_q, squared error to x_fp, backward) with the block
objective of Eq.1 and the quantised linear of Eq.4: Y = Q_a(X~) Q_w(W~) + B~.

``mean_rows`` (default ``c_out``) is the output-channel count of the whole
linear in the mean-squared-error normaliser.  Without LET each output row's
loss and clipping gradients depend on that row alone, so a check may pass a
subset of a linear's rows together with the whole linear's normaliser.

"The block" here is its linear sub-graph: every linear l reads the input of
its site k and is compared with its own full-precision target Y_fp,l.  The
loss is the sum over linears of the mean squared error (Eq.1 and Algorithm 1
write a squared norm; a mean per linear fixes its scale, which sets the size
of every gradient).

Description (plain dicts):
  desc  = {"T": tokens, "bf16": bool,
           "sites":   [{"width": C, "let": bool, "act_bits": 16 | N,
                        "act_sym": bool (optional: symmetric absmax Q_a)}, ...],
           "linears": [{"site": k, "c_out": C_out, "bits": N, "group": g,
                        "quant": "lwc" | "pact" | "lsq" (optional, default LWC),
                        "mean_rows": C_out_whole (optional)}, ...]}
  X_q   = [ [T, C_k] per site ]            (the quantised model's input x_q)
  Y_fp  = [ [T, C_out_l] per linear ]      (the full-precision target x_fp)
  params= {"W": [[C_out, C_in]], "B": [[C_out] | None],
           "gamma_logit": [[C_out, C_in/g]], "beta_logit": [...],
                (for PACT these hold the thresholds hi, lo; for LSQ the step h
                 and zero point z of each group)
           "s": [[C_k] | None per site], "delta": [...]}

With ``bf16`` the matrix-product operands (X^, W^, dY) are rounded to bf16,
as the kernels feed them to the matrix cores; sums are fp64 throughout.
"""
import numpy as np

from .quant import (act_bwd, act_fwd, act_sym_bwd, act_sym_fwd, bf16_round, lsq_bwd, lsq_fwd,
                    lwc_bwd, lwc_fwd, pact_bwd, pact_fwd)
from .let import let_bias, let_x


def _op(x, bf16):
    """A matrix-product operand: bf16-rounded in bf16 mode, else unchanged."""
    return bf16_round(x).astype(np.float64) if bf16 else np.asarray(x, np.float64)


def block_forward(desc, X_q, Y_fp, params, ft=np.float32):
    """Forward half of the step: per-site X^, per-linear W^, Y, residual, loss."""
    T = desc["T"]
    bf16 = desc.get("bf16", False) and ft == np.float32
    sites, lins = desc["sites"], desc["linears"]
    S = []
    for k, site in enumerate(sites):
        x = np.asarray(X_q[k], dtype=ft)
        rec = {"x": x}
        if site["let"]:
            rec["xt"] = let_x(x, params["s"][k], params["delta"][k], ft)
        else:
            rec["xt"] = x
        if site["act_bits"] < 16:
            fwd = act_sym_fwd if site.get("act_sym") else act_fwd
            rec["act"] = fwd(rec["xt"], site["act_bits"], ft)
            rec["xhat"] = rec["act"]["X_dq"]
        else:
            rec["xhat"] = rec["xt"]
        rec["xop"] = _op(rec["xhat"], bf16)
        S.append(rec)

    L = []
    loss = 0.0
    for l, lin in enumerate(lins):
        k = lin["site"]
        site = sites[k]
        W = np.asarray(params["W"][l], dtype=ft)
        s = params["s"][k] if site["let"] else None
        fwd = {"lwc": lwc_fwd, "pact": pact_fwd, "lsq": lsq_fwd}[lin.get("quant", "lwc")]
        st = fwd(W, params["gamma_logit"][l], params["beta_logit"][l],
                 lin["bits"], lin["group"], s=s, ft=ft)
        B = params["B"][l] if params.get("B") is not None else None
        if site["let"]:
            Bt = let_bias(W, B, params["delta"][k], ft)
        elif B is not None:
            Bt = np.asarray(B, ft)
        else:
            Bt = np.zeros(lin["c_out"], ft)
        wop = _op(st["W_dq"], bf16)
        acc = S[k]["xop"] @ wop.T                       # [T, C_out], fp64 sum
        Y = (acc + np.asarray(Bt, np.float64)[None, :]).astype(ft)
        R = Y - np.asarray(Y_fp[l], dtype=ft)           # residual, one rounding
        n = T * lin.get("mean_rows", lin["c_out"])
        R64 = R.astype(np.float64)
        row_loss = np.sum(R64 * R64, axis=0)            # per output channel
        loss += float(np.sum(row_loss)) / n
        scale = ft(2.0) / ft(n)
        dY = _op(R * scale, bf16)                       # dL/dY (mean-squared error)
        L.append(dict(st=st, Bt=Bt, wop=wop, Y=Y, R=R, dY=dY, row_loss=row_loss,
                      W=W, n=n))
    return loss, S, L


def block_step(desc, X_q, Y_fp, params, ft=np.float32):
    """Loss and straight-through gradients of one calibration step.

    Returns (loss, out) with out = {"d_gamma_logit": [...], "d_beta_logit":
    [...], "d_s": [...], "d_delta": [...], "row_loss": [...], "fwd": (S, L)}.
    """
    sites, lins = desc["sites"], desc["linears"]
    loss, S, L = block_forward(desc, X_q, Y_fp, params, ft)
    d_gl, d_bl, row_loss = [], [], []
    ds_w = [np.zeros(s_["width"]) for s_ in sites]
    dd_b = [np.zeros(s_["width"]) for s_ in sites]
    dXhat = [np.zeros((desc["T"], s_["width"])) if s_["let"] else None for s_ in sites]
    for l, lin in enumerate(lins):
        k = lin["site"]
        rec = L[l]
        dWdq = rec["dY"].T @ S[k]["xop"]                # [C_out, C_in], fp64 sum over tokens
        quant = lin.get("quant", "lwc")
        if quant == "lwc":
            g = lwc_bwd(rec["st"], dWdq, W=rec["W"], with_s=sites[k]["let"])
            d_gl.append(g["d_gamma_logit"])
            d_bl.append(g["d_beta_logit"])
        else:
            bwd = pact_bwd if quant == "pact" else lsq_bwd
            g = bwd(rec["st"], dWdq, W=rec["W"], with_s=sites[k]["let"])
            d_gl.append(g["d_p1"])
            d_bl.append(g["d_p2"])
        row_loss.append(rec["row_loss"])
        if sites[k]["let"]:
            ds_w[k] += g["d_s"]                          # W~ = s (.) W
            dBt = np.sum(rec["dY"], axis=0)              # B~ = B + delta W
            dd_b[k] += dBt @ rec["W"].astype(np.float64)
            dXhat[k] += rec["dY"] @ rec["wop"]           # dL/dX^, summed over the site
    d_s, d_delta = [], []
    for k, site in enumerate(sites):
        if not site["let"]:
            d_s.append(None)
            d_delta.append(None)
            continue
        if site["act_bits"] < 16:
            bwd = act_sym_bwd if site.get("act_sym") else act_bwd
            dxt = bwd(S[k]["act"], dXhat[k])            # through Q_a (straight-through)
        else:
            dxt = dXhat[k]                              # X^ = X~
        s = np.asarray(params["s"][k], np.float64)
        xt = S[k]["xt"].astype(np.float64)
        # X~ = (X - delta) / s:  dX~/ds = -X~/s,  dX~/ddelta = -1/s
        d_s.append(ds_w[k] - np.sum(dxt * xt, axis=0) / s)
        d_delta.append(dd_b[k] - np.sum(dxt, axis=0) / s)
        S[k]["dxt"] = dxt
    return loss, dict(d_gamma_logit=d_gl, d_beta_logit=d_bl, d_s=d_s, d_delta=d_delta,
                      row_loss=row_loss, fwd=(S, L))


def fp_target(X, W, B=None, bf16=True):
    """Full-precision output of one linear (Algorithm 1: the fp block output
    the quantised block is trained to match): X W^T + B, fp64 sum, rounded
    once to the storage type (bf16 or fp32).  Layout [T, C_out]."""
    acc = np.asarray(X, np.float64) @ np.asarray(W, np.float64).T
    if B is not None:
        acc = acc + np.asarray(B, np.float64)[None, :]
    y = acc.astype(np.float32)
    return bf16_round(y) if bf16 else y
