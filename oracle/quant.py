"""Oracle: the LWC weight quantiser (Eq.2) and the per-token MinMax activation
quantiser (Eq.4's Q_a), forward and straight-through backward.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Readings of points the paper leaves open:
  * the round operation of Eq.2 rounds half to even (``np.rint``);
  * dequantisation, which Eq.2 does not write, is ``(W_q - z) * h``;
  * fp32 operation order: a = gamma*max, b = beta*min, h = (a - b)/qmax,
    h = max(h, 1e-5), r = 1/h, z = -rint(b*r), u = w*r, c = rint(u) + z;
    every named quantity is one IEEE fp32 rounding, no fused multiply-add;
  * a group is a contiguous run of ``group`` weights along the input
    dimension of one output row (W stored [C_out, C_in]);
  * max/min ties go to the lowest index inside the group, and the gradient
    of max/min flows to that element only;
  * straight-through estimation replaces only the derivative of rint by 1;
    clamp, max/min and the h >= 1e-5 guard are differentiated exactly
    (the guard passes no gradient to gamma, beta, max or min when active);
  * Q_a is Eq.2 with gamma = beta = 1 applied to each token row.
"""
import numpy as np

H_MIN = 1e-5


def clip_strength(logit, ft=np.float32):
    """gamma = Sigmoid(logit) (Sec. 3.2 footnote: 1 / (1 + e^-t)).

    Evaluated in fp64 and rounded once to ``ft``.
    """
    t = np.asarray(logit, dtype=np.float64)
    return (1.0 / (1.0 + np.exp(-t))).astype(ft)


def bf16_round(x):
    """Round fp32 values to the nearest bfloat16 (ties to even); fp32 result."""
    # add 0x7FFF plus the lowest kept bit, then clear the 16 dropped bits: a
    # tie rounds to the even neighbour.  Finite inputs never carry past bit
    # 31 (the largest finite magnitude is 0x7F7FFFFF), so uint32 suffices.
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u >> np.uint32(16)) & np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r &= np.uint32(0xFFFF0000)
    return r.view(np.float32).reshape(np.shape(x))


def minmax_quant_rows(wt, gamma, beta, bits, ft=np.float32):
    """Eq.2 applied independently to every row of ``wt`` ([n, g]).

    ``wt`` holds the (already transformed) values to quantise; ``gamma`` and
    ``beta`` ([n]) are the clip strengths in [0, 1].  Returns a dict with the
    per-row statistics and the per-element codes and dequantised values.
    """
    wt = np.asarray(wt, dtype=ft)
    gamma = np.asarray(gamma, dtype=ft)
    beta = np.asarray(beta, dtype=ft)
    qmax = ft(2 ** bits - 1)
    # max / min with the lowest index on ties (numpy's argmax/argmin rule)
    i_mx = np.argmax(wt, axis=1)
    i_mn = np.argmin(wt, axis=1)
    rows = np.arange(wt.shape[0])
    mx = wt[rows, i_mx]
    mn = wt[rows, i_mn]
    a = gamma * mx                       # upper clip bound   gamma * max(W)
    b = beta * mn                        # lower clip bound   beta * min(W)
    h_raw = (a - b) / qmax               # normalisation factor h
    hclamp = h_raw < ft(H_MIN)
    h = np.where(hclamp, ft(H_MIN), h_raw).astype(ft)
    r = ft(1.0) / h
    z = -np.rint(b * r)                  # zero point  z = -round(beta*min / h)
    u = wt * r[:, None]                  # W / h
    c = np.rint(u) + z[:, None]          # round(W/h) + z, before the clamp
    m = (c >= 0) & (c <= qmax)           # clamp passes the gradient here
    q = np.clip(c, ft(0), qmax).astype(ft)
    wdq = (q - z[:, None]) * h[:, None]  # dequantised weight (W_q - z) * h
    return dict(mx=mx, mn=mn, i_mx=i_mx, i_mn=i_mn, a=a, b=b, h=h, hclamp=hclamp,
                r=r, z=z, u=u, c=c, m=m, q=q, wdq=wdq, gamma=gamma, beta=beta,
                qmax=qmax, bits=bits)


def minmax_quant_rows_bwd(st, g, need_ratio_grads=True):
    """Straight-through backward of :func:`minmax_quant_rows` (fp64).

    ``g`` ([n, gsize]) is dL/d(dequantised value).  Returns dL/d(input value)
    per element and, when asked, dL/dgamma and dL/dbeta per row.
    """
    g = np.asarray(g, dtype=np.float64)
    q = st["q"].astype(np.float64)
    u = st["u"].astype(np.float64)
    m = st["m"].astype(np.float64)
    z = st["z"].astype(np.float64)[:, None]
    h = st["h"].astype(np.float64)
    b = st["b"].astype(np.float64)
    mx = st["mx"].astype(np.float64)
    mn = st["mn"].astype(np.float64)
    gamma = st["gamma"].astype(np.float64)
    beta = st["beta"].astype(np.float64)
    qmax = float(st["qmax"])
    live = ~st["hclamp"]

    # dwhat_i/dh = (q_i - z) - m_i*u_i + (m_i - 1)*b/h ;  dwhat_i/db (through z) = 1 - m_i
    s_h = np.sum(g * ((q - z) - m * u), axis=1)
    s_z = np.sum(g * (1.0 - m), axis=1)
    dh = s_h - s_z * b / h
    dh_live = np.where(live, dh, 0.0)
    da = dh_live / qmax                  # h = (a - b) / qmax
    db = s_z - dh_live / qmax
    dmx = da * gamma                     # a = gamma * max
    dmn = db * beta                      # b = beta * min
    dx = g * m
    rows = np.arange(g.shape[0])
    np.add.at(dx, (rows, st["i_mx"]), dmx)
    np.add.at(dx, (rows, st["i_mn"]), dmn)
    out = dict(dx=dx, dh=dh, s_h=s_h, s_z=s_z)
    if need_ratio_grads:
        out["dgamma"] = da * mx
        out["dbeta"] = db * mn
    return out


def lwc_fwd(W, gamma_logit, beta_logit, bits, group, s=None, ft=np.float32):
    """LWC forward (Eq.2) on a weight [C_out, C_in], optionally LET-scaled.

    With ``s`` given, the quantised tensor is W~ = s (.) W (Eq.3), computed as
    one fp32 product per element.  ``gamma_logit``/``beta_logit`` are
    [C_out, C_in // group].  Returns the row-level dict of
    :func:`minmax_quant_rows` plus ``codes``/``wdq`` in [C_out, C_in] layout.
    """
    W = np.asarray(W, dtype=ft)
    c_out, c_in = W.shape
    if c_in % group:
        raise ValueError("group must divide C_in")
    wt = W * np.asarray(s, dtype=ft)[None, :] if s is not None else W
    ng = c_in // group
    gamma = clip_strength(gamma_logit, ft).reshape(c_out * ng)
    beta = clip_strength(beta_logit, ft).reshape(c_out * ng)
    st = minmax_quant_rows(wt.reshape(c_out * ng, group), gamma, beta, bits, ft)
    st["wt"] = wt
    st["shape"] = (c_out, c_in, group)
    st["codes"] = st["q"].reshape(c_out, c_in).astype(np.uint8)
    st["W_dq"] = st["wdq"].reshape(c_out, c_in)
    st["h_g"] = st["h"].reshape(c_out, ng)
    st["z_g"] = st["z"].reshape(c_out, ng)
    return st


def lwc_bwd(st, dW_dq, W=None, with_s=False):
    """LWC straight-through backward.

    ``dW_dq`` = dL/d(dequantised weight) [C_out, C_in].  Returns
    d_gamma_logit, d_beta_logit ([C_out, C_in/g]), dW_tilde ([C_out, C_in])
    and, when ``with_s``, the weight-path part of dL/ds:
    sum_o dW~[o, c] * W[o, c]  (since W~ = s (.) W).
    """
    c_out, c_in, group = st["shape"]
    ng = c_in // group
    r = minmax_quant_rows_bwd(st, np.asarray(dW_dq, np.float64).reshape(c_out * ng, group))
    gam = st["gamma"].astype(np.float64)
    bet = st["beta"].astype(np.float64)
    out = dict(
        d_gamma_logit=(r["dgamma"] * gam * (1.0 - gam)).reshape(c_out, ng),
        d_beta_logit=(r["dbeta"] * bet * (1.0 - bet)).reshape(c_out, ng),
        dW_tilde=r["dx"].reshape(c_out, c_in),
    )
    if with_s:
        out["d_s"] = np.sum(out["dW_tilde"] * np.asarray(W, np.float64), axis=0)
    return out


def act_fwd(Xt, bits, ft=np.float32):
    """Per-token asymmetric MinMax fake-quant (Q_a of Eq.4; Sec. 4.1
    per-token activations): Eq.2 with gamma = beta = 1 on each row of Xt."""
    Xt = np.asarray(Xt, dtype=ft)
    n = Xt.shape[0]
    ones = np.ones(n, dtype=ft)
    st = minmax_quant_rows(Xt, ones, ones, bits, ft)
    st["codes"] = st["q"].astype(np.uint8)
    st["X_dq"] = st["wdq"]
    return st


def act_bwd(st, dX_dq):
    """Straight-through backward of :func:`act_fwd`: dL/dX~ (no learnable
    parameters inside Q_a; its scale still carries gradient)."""
    return minmax_quant_rows_bwd(st, dX_dq, need_ratio_grads=False)["dx"]
