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


# ---------------------------------------------------------------- quantiser variants
# The paper's appendix compares LWC with PACT and LSQ "by replacing LWC in our
# pipeline" (weight clipping only), and names symmetric uniform quantisation
# as the other format of the field.  Their readings here:
#   * PACT learns the clipping thresholds themselves, one upper (hi) and one
#     lower (lo) per group, initialised to the group's max and min; the grid
#     spans [lo, hi] exactly as Eq. 2 spans [beta*min, gamma*max]; PACT's own
#     straight-through rule treats the quantiser as the identity on the
#     clipped weight, so dL/dhi sums the gradient of the elements whose code
#     saturates at qmax, dL/dlo of those at 0, and dL/dw = g*m.
#   * LSQ learns the step size h and the zero point z directly (initialised
#     to MinMax's), with z rounded in the forward; its straight-through rule
#     gives rint derivative 1 (codes and zero point), and its gradient scale
#     1/sqrt(n * qmax) (n = group size) multiplies dL/dh and dL/dz.
#   * Symmetric per-token activation quantisation: h = max|x| / (2^(N-1) - 1)
#     (floored at 1e-5), zero point fixed at 2^(N-1), so codes span
#     [1, 2^N - 1] around it; the gradient of the row's absolute maximum goes
#     to the lowest index holding it, with that element's sign.


def _grid_rows(wt, a, b, h_direct, z_direct, bits, ft):
    """Eq. 2's grid with given bounds (a, b) or a given step / zero point."""
    qmax = ft(2 ** bits - 1)
    if h_direct is None:
        h_raw = (a - b) / qmax
    else:
        h_raw = np.asarray(h_direct, ft)
    hclamp = h_raw < ft(H_MIN)
    h = np.where(hclamp, ft(H_MIN), h_raw).astype(ft)
    r = ft(1.0) / h
    if z_direct is None:
        z = -np.rint(b * r)
    else:
        z = np.rint(np.asarray(z_direct, ft))
    u = wt * r[:, None]
    c = np.rint(u) + z[:, None]
    m = (c >= 0) & (c <= qmax)
    q = np.clip(c, ft(0), qmax).astype(ft)
    wdq = (q - z[:, None]) * h[:, None]
    return dict(h=h, hclamp=hclamp, r=r, z=z, u=u, c=c, m=m, q=q, wdq=wdq, qmax=qmax, bits=bits)


def _as_layer(st, wt, c_out, c_in, group):
    ng = c_in // group
    st["wt"] = wt
    st["shape"] = (c_out, c_in, group)
    st["codes"] = st["q"].reshape(c_out, c_in).astype(np.uint8)
    st["W_dq"] = st["wdq"].reshape(c_out, c_in)
    st["h_g"] = st["h"].reshape(c_out, ng)
    st["z_g"] = st["z"].reshape(c_out, ng)
    return st


def pact_fwd(W, hi, lo, bits, group, s=None, ft=np.float32):
    """PACT weight clipping in LWC's place: learned thresholds hi, lo
    [C_out, C_in/g] bound the grid directly (a = hi, b = lo)."""
    W = np.asarray(W, dtype=ft)
    c_out, c_in = W.shape
    wt = W * np.asarray(s, dtype=ft)[None, :] if s is not None else W
    a = np.asarray(hi, ft).reshape(-1)
    b = np.asarray(lo, ft).reshape(-1)
    st = _grid_rows(wt.reshape(-1, group), a, b, None, None, bits, ft)
    st.update(a=a, b=b, quant="pact")
    return _as_layer(st, wt, c_out, c_in, group)


def pact_bwd(st, dW_dq, W=None, with_s=False):
    """PACT's straight-through rule: dhi = sum g [code above qmax],
    dlo = sum g [code below 0], dW~ = g*m."""
    c_out, c_in, group = st["shape"]
    ng = c_in // group
    g = np.asarray(dW_dq, np.float64).reshape(-1, group)
    c = st["c"].astype(np.float64)
    m = st["m"].astype(np.float64)
    out = dict(d_p1=np.sum(g * (c > float(st["qmax"])), axis=1).reshape(c_out, ng),
               d_p2=np.sum(g * (c < 0), axis=1).reshape(c_out, ng),
               dW_tilde=(g * m).reshape(c_out, c_in))
    if with_s:
        out["d_s"] = np.sum(out["dW_tilde"] * np.asarray(W, np.float64), axis=0)
    return out


def lsq_fwd(W, step, zero, bits, group, s=None, ft=np.float32):
    """LSQ in LWC's place: learned step h and zero point z [C_out, C_in/g]
    (the zero point is rounded in the forward; the step floored at 1e-5)."""
    W = np.asarray(W, dtype=ft)
    c_out, c_in = W.shape
    wt = W * np.asarray(s, dtype=ft)[None, :] if s is not None else W
    st = _grid_rows(wt.reshape(-1, group), None, None, np.asarray(step, ft).reshape(-1),
                    np.asarray(zero, ft).reshape(-1), bits, ft)
    st.update(quant="lsq", group=group)
    return _as_layer(st, wt, c_out, c_in, group)


def lsq_grad_scale(group, bits):
    """LSQ's gradient scale 1/sqrt(n * Q_P), n = weights per step size."""
    return 1.0 / np.sqrt(float(group) * float(2 ** bits - 1))


def lsq_bwd(st, dW_dq, W=None, with_s=False):
    """LSQ's straight-through rule (rint derivative 1 on the codes and the
    zero point), times the gradient scale:
      dh = gs * sum g ((q - z) - m u)   (0 where the 1e-5 floor is active)
      dz = -gs * h * sum g (1 - m),     dW~ = g*m."""
    c_out, c_in, group = st["shape"]
    ng = c_in // group
    g = np.asarray(dW_dq, np.float64).reshape(-1, group)
    q, u, m = (st[k].astype(np.float64) for k in ("q", "u", "m"))
    z = st["z"].astype(np.float64)[:, None]
    h = st["h"].astype(np.float64)
    gs = lsq_grad_scale(group, st["bits"])
    s_h = np.sum(g * ((q - z) - m * u), axis=1)
    s_z = np.sum(g * (1.0 - m), axis=1)
    out = dict(d_p1=(gs * np.where(st["hclamp"], 0.0, s_h)).reshape(c_out, ng),
               d_p2=(-gs * h * s_z).reshape(c_out, ng),
               dW_tilde=(g * m).reshape(c_out, c_in))
    if with_s:
        out["d_s"] = np.sum(out["dW_tilde"] * np.asarray(W, np.float64), axis=0)
    return out


def wquant_init(W, bits, group, quant, s=None, ft=np.float32):
    """MinMax initial parameters of a quantiser variant, per group:
    PACT (hi, lo) = (max, min); LSQ (h, z) = MinMax's h and z (Eq. 2 at
    gamma = beta = 1); LWC (gamma_logit, beta_logit) = (4, 4)."""
    W = np.asarray(W, dtype=ft)
    c_out, c_in = W.shape
    ng = c_in // group
    wt = W * np.asarray(s, dtype=ft)[None, :] if s is not None else W
    rows = wt.reshape(-1, group)
    if quant == "lwc":
        return np.full((c_out, ng), 4.0, ft), np.full((c_out, ng), 4.0, ft)
    if quant == "pact":
        return rows.max(axis=1).reshape(c_out, ng), rows.min(axis=1).reshape(c_out, ng)
    ones = np.ones(rows.shape[0], ft)
    st = minmax_quant_rows(rows, ones, ones, bits, ft)
    return st["h"].reshape(c_out, ng), st["z"].reshape(c_out, ng).astype(ft)


def act_sym_fwd(Xt, bits, ft=np.float32):
    """Symmetric per-token absmax fake-quant: h = max(absmax/(2^(N-1)-1), 1e-5),
    z = 2^(N-1), codes clamp(rint(x/h) + z, 0, 2^N - 1)."""
    Xt = np.asarray(Xt, dtype=ft)
    qs = ft(2 ** (bits - 1) - 1)
    ax = np.abs(Xt)
    i_ab = np.argmax(ax, axis=1)                     # lowest index of the largest |x|
    rows = np.arange(Xt.shape[0])
    amax = ax[rows, i_ab]
    sgn = np.where(Xt[rows, i_ab] < 0, -1.0, 1.0)
    st = _grid_rows(Xt, None, None, amax / qs, np.full(Xt.shape[0], ft(2 ** (bits - 1))), bits, ft)
    st.update(i_ab=i_ab, amax=amax, sgn=sgn, qs=qs, sym=True)
    st["codes"] = st["q"].astype(np.uint8)
    st["X_dq"] = st["wdq"]
    return st


def act_sym_bwd(st, dX_dq):
    """Straight-through backward of :func:`act_sym_fwd`: dx = g*m plus, at
    the row's absmax element, sign * dh / (2^(N-1) - 1) with
    dh = sum g ((q - z) - m u) (0 under the floor)."""
    g = np.asarray(dX_dq, np.float64)
    q, u, m = (st[k].astype(np.float64) for k in ("q", "u", "m"))
    z = st["z"].astype(np.float64)[:, None]
    s_h = np.sum(g * ((q - z) - m * u), axis=1)
    dh = np.where(st["hclamp"], 0.0, s_h)
    dx = g * m
    rows = np.arange(g.shape[0])
    np.add.at(dx, (rows, st["i_ab"]), st["sgn"] * dh / float(st["qs"]))
    return dx
