"""Oracle: one calibration step over a whole LLaMA transformer block.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Eq. 1 trains each block against its full-precision output F(W, X); here F is
the block itself (Sec. 2 and Sec. 3.1 calibrate transformer blocks):

    x1 = RMSNorm(h0) g1                    (LET site 1: q, k, v input)
    q, k, v = Q_w(W~) Q_a(X1~) + B~        (Eq. 3-4 on each linear)
    q, k <- RoPE(q), RoPE(k)               (rotate-half pairs (i, i + d/2))
    Q~ = q / s_a, K~ = k * s_a             (Eq. 5: LET on the attention affinity)
    Q^, K^, V^ = Q_a(Q~), Q_a(K~), Q_a(v)  (per-token activation quantisation)
    o_att = softmax(Q^ K^T / sqrt(d) + causal mask) V^   per sample and head
    h1 = h0 + Q_w(W_o~) Q_a(X2~) + B~_o    (LET site 2: the o input, paired with v)
    x3 = RMSNorm(h1) g2                    (LET site 3: gate, up input)
    x4 = SiLU(gate) * up                   (site 4: down input, no LET)
    h2 = h1 + Q_w(W_d) Q_a(x4)
    loss = mean((h2 - h2_fp)^2)

Readings (the paper writes the equations, not the block's code):
  * the [Q, K] scale s_a acts after RoPE, per channel of a key head and
    shared by the query heads of its group (grouped-query attention), so
    softmax((Q/s_a)(s_a K)^T) = softmax(Q K^T) exactly without quantisation;
  * Q_a applies per token to Q~, K~ and V (all heads of a token together) as
    it does to the linears' inputs; the softmax output stays unquantised
    unless ``desc["softmax_bits"]`` < 16 (the ablation on softmax
    quantisation: Q_a on every query row of probabilities, see
    :func:`attention`);
  * the residual stream, norms, RoPE, softmax and SiLU are evaluated in fp64;
    the quantisers in fp32 in Eq. 2's fixed order (the functions of
    ``oracle.quant``); the operands the kernels feed to matrix cores
    (quantised activations, quantised weights, gradients entering a product)
    are rounded to bf16 when ``bf16`` is set;
  * no weight is trained but the clipping logits, s, delta and s_a; the
    norm gains are frozen block weights;
  * straight-through estimation as in ``oracle.quant`` (only rint has
    derivative 1).

Shapes: h0, h2_fp [T, D] with T = n_seq * seq_len (the samples follow each
other); W in PyTorch layout [C_out, C_in]: q [H d, D], k and v [Hkv d, D],
o [D, H d], gate and up [F, D], down [D, F]; s_a [Hkv d].

``frozen`` (optional, from :func:`freeze`): every discrete choice of every
quantiser held fixed, the quantisers then evaluated in fp64 as smooth
functions of their inputs and parameters (the frozen-selection surrogate of
``oracle.surrogate``), for finite-difference checks of :func:`block_step`.
"""
import numpy as np

from .quant import (act_bwd, act_fwd, act_sym_bwd, act_sym_fwd, bf16_round, clip_strength, lwc_bwd,
                    lwc_fwd)
from .surrogate import _frozen_choices, _frozen_variant, _quant_frozen, _sym_frozen

LINEARS = ("q", "k", "v", "o", "gate", "up", "down")
SITE_OF = (0, 0, 0, 1, 2, 2, 3)          # input site of each linear


def _op(x, bf16):
    return bf16_round(np.asarray(x, np.float32)).astype(np.float64) if bf16 else np.asarray(x, np.float64)


# ---------------------------------------------------------------- smooth pieces
def rmsnorm(h, g, eps):
    """h / sqrt(mean(h^2) + eps) * g per token row (fp64)."""
    h = np.asarray(h, np.float64)
    rstd = 1.0 / np.sqrt(np.mean(h * h, axis=1) + eps)
    return h * rstd[:, None] * np.asarray(g, np.float64)[None, :], rstd


def rmsnorm_bwd(h, g, rstd, dy):
    """Gradient of :func:`rmsnorm` with respect to h."""
    h = np.asarray(h, np.float64)
    g = np.asarray(g, np.float64)
    gd = dy * g[None, :]
    D = h.shape[1]
    dot = np.sum(gd * h, axis=1)
    return rstd[:, None] * gd - h * (rstd ** 3 * dot / D)[:, None]


def rope_angles(T, seq_len, d, base):
    """cos, sin [T, d/2]: position p = t mod seq_len, frequency base^(-2i/d)."""
    pos = np.arange(T) % seq_len
    inv = base ** (-np.arange(0, d // 2) * 2.0 / d)
    ang = pos[:, None].astype(np.float64) * inv[None, :]
    return np.cos(ang), np.sin(ang)


def rope(x, n_heads, d, cos, sin, inverse=False):
    """Rotate the pairs (i, i + d/2) of every head by the token's angles
    (the inverse rotation for the backward)."""
    T = x.shape[0]
    x = np.asarray(x, np.float64).reshape(T, n_heads, d)
    a, b = x[:, :, : d // 2], x[:, :, d // 2:]
    c, s = cos[:, None, :], sin[:, None, :]
    if inverse:
        s = -s
    out = np.concatenate([a * c - b * s, b * c + a * s], axis=2)
    return out.reshape(T, n_heads * d)


def attention(q, k, v, H, Hkv, d, seq_len, bf16=False, p_bits=16, rec=None, frozen=None,
              ft=np.float32):
    """Causal softmax(q k^T / sqrt(d)) v per sample and query head; query
    head h reads key/value head h // (H / Hkv).  Returns (out, probs, phat):
    probs the exact softmax, phat the probabilities that multiply v (None
    without softmax quantisation).

    ``bf16``: the weights enter the product with v as bf16 matrix-core
    operands.  Reading: a row's weights are 2^(t - M) with t the logit in
    base 2 (s log2(e)) and M = ceil(max t) (an integral reference, so that
    the rounded weights do not depend on how the maximum was found), each
    rounded to bf16, and the output is divided by the sum of those rounded
    weights (a weighted mean of v rows).

    ``p_bits`` < 16 (the softmax-quantisation ablation): each query row of
    probabilities (its S entries, the causally masked zeros included) goes
    through Q_a -- per-row asymmetric MinMax, in ``ft`` (the quantiser's fp32
    order), its state kept in ``rec`` under "pq<b>_<h>" -- or, with
    ``frozen``, the frozen surrogate; the quantised row multiplies v as it
    is (bf16 operands with ``bf16``, no renormalisation)."""
    T = q.shape[0]
    ns = T // seq_len
    grp = H // Hkv
    q = q.reshape(ns, seq_len, H, d)
    k = k.reshape(ns, seq_len, Hkv, d)
    v = v.reshape(ns, seq_len, Hkv, d)
    out = np.zeros((ns, seq_len, H, d))
    P = np.zeros((ns, H, seq_len, seq_len))
    PH = np.zeros_like(P) if p_bits < 16 else None
    mask = np.triu(np.ones((seq_len, seq_len), bool), 1)
    for b in range(ns):
        for h in range(H):
            kv = h // grp
            s = q[b, :, h, :] @ k[b, :, kv, :].T / np.sqrt(d)
            s[mask] = -np.inf
            if bf16 and p_bits >= 16:
                t = s * np.log2(np.e)
                w = _op(np.exp2(t - np.ceil(np.max(t, axis=1, keepdims=True))), True)
                out[b, :, h, :] = (w @ v[b, :, kv, :]) / np.sum(w, axis=1, keepdims=True)
            s = s - np.max(s, axis=1, keepdims=True)
            p = np.exp(s)
            p /= np.sum(p, axis=1, keepdims=True)
            P[b, h] = p
            if p_bits < 16:
                key = f"pq{b}_{h}"
                if frozen is not None:
                    ones = np.ones(seq_len)
                    ph = _quant_frozen(p, ones, ones, frozen[key])
                else:
                    st = act_fwd(np.asarray(p, ft), p_bits, ft=ft)
                    if rec is not None:
                        rec[key] = st
                    ph = st["X_dq"].astype(np.float64)
                PH[b, h] = ph
                out[b, :, h, :] = _op(ph, bf16) @ v[b, :, kv, :]
            elif not bf16:
                out[b, :, h, :] = p @ v[b, :, kv, :]
    return out.reshape(T, H * d), P, PH


def attention_bwd(q, k, v, P, dout, H, Hkv, d, seq_len, bf16=False, PH=None, rec=None):
    """Gradients of :func:`attention` with respect to q, k, v (from the exact
    softmax ``P``).  ``bf16``: P enters the dV product as a bf16 operand.
    With softmax quantisation (``PH`` the quantised probabilities, ``rec``
    the quantiser states): dV from PH, and dP through Q_a's straight-through
    backward before the softmax backward."""
    T = q.shape[0]
    ns = T // seq_len
    grp = H // Hkv
    q = q.reshape(ns, seq_len, H, d)
    k = k.reshape(ns, seq_len, Hkv, d)
    v = v.reshape(ns, seq_len, Hkv, d)
    do = dout.reshape(ns, seq_len, H, d)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for b in range(ns):
        for h in range(H):
            kv = h // grp
            p = P[b, h]
            pv = p if PH is None else PH[b, h]
            dv[b, :, kv, :] += _op(pv, bf16).T @ do[b, :, h, :]
            dp = do[b, :, h, :] @ v[b, :, kv, :].T
            if PH is not None:
                dp = act_bwd(rec[f"pq{b}_{h}"], dp)
            ds = p * (dp - np.sum(dp * p, axis=1, keepdims=True)) / np.sqrt(d)
            dq[b, :, h, :] = ds @ k[b, :, kv, :]
            dk[b, :, kv, :] += ds.T @ q[b, :, h, :]
    return dq.reshape(T, H * d), dk.reshape(T, Hkv * d), dv.reshape(T, Hkv * d)


def silu(x):
    return x / (1.0 + np.exp(-x))


def silu_grad(x):
    sg = 1.0 / (1.0 + np.exp(-x))
    return sg * (1.0 + x * (1.0 - sg))


# ---------------------------------------------------------------- quantiser wrappers
def _act(x, bits, frozen, key, rec, ft, sym=False):
    """Q_a on token rows (in ``ft``: fp32 spec or fp64; or the frozen fp64
    surrogate): per-token MinMax, or symmetric absmax when ``sym``."""
    if bits >= 16:
        return np.asarray(x, np.float64)
    if frozen is not None:
        if sym:
            return _sym_frozen(np.asarray(x, np.float64), frozen[key])
        ones = np.ones(x.shape[0])
        return _quant_frozen(np.asarray(x, np.float64), ones, ones, frozen[key])
    st = (act_sym_fwd if sym else act_fwd)(np.asarray(x, ft), bits, ft=ft)
    rec[key] = st
    return st["X_dq"].astype(np.float64)


def _act_bwd(g, bits, key, rec):
    if bits >= 16:
        return g
    st = rec[key]
    return act_sym_bwd(st, g) if st.get("sym") else act_bwd(st, g)


def _lwc(W, gl, bl, bits, group, s, frozen, key, rec, ft, quantise=True):
    if not quantise:                         # weights used unquantised (pins only)
        Wt = np.asarray(W, np.float64)
        return Wt * np.asarray(s, np.float64)[None, :] if s is not None else Wt
    if frozen is not None:
        Wt = np.asarray(W, np.float64)
        if s is not None:
            Wt = Wt * np.asarray(s, np.float64)[None, :]
        gam = clip_strength(np.asarray(gl).reshape(-1), np.float64)
        bet = clip_strength(np.asarray(bl).reshape(-1), np.float64)
        return _quant_frozen(Wt.reshape(-1, group), gam, bet, frozen[key]).reshape(W.shape)
    st = lwc_fwd(np.asarray(W, ft), gl, bl, bits, group, s=s, ft=ft)
    rec[key] = st
    return st["W_dq"].astype(np.float64)


def _let_x(x, s, dl, frozen, ft):
    """X~ = (X - delta) / s (fp32 order of Eq. 3's reading; fp64 otherwise)."""
    if s is None:
        return np.asarray(x, np.float64)
    if frozen is not None or ft == np.float64:
        return (np.asarray(x, np.float64) - np.asarray(dl, np.float64)) / np.asarray(s, np.float64)
    x32 = np.asarray(x, np.float32)
    rs = np.float32(1.0) / np.asarray(s, np.float32)
    return ((x32 - np.asarray(dl, np.float32)) * rs).astype(np.float64)


# ---------------------------------------------------------------- the block
def block_forward(desc, h0, target, params, frozen=None, ft=np.float32):
    """Forward of the quantised block.  Returns (loss, cache).  ``ft``: the
    quantisers' precision (fp32 per the spec; fp64 for the finite-difference
    checks, with no bf16 rounding).  ``desc["w_quant"] = False`` uses the
    weights unquantised (for the equivalence pins)."""
    D, H, Hkv, F = desc["hidden"], desc["heads"], desc["kv_heads"], desc["ffn"]
    d = D // H
    S = desc["seq_len"]
    T = h0.shape[0]
    ab = desc["act_bits"]
    sym = bool(desc.get("act_sym", False))
    let = desc["let"]
    bf16 = desc.get("bf16", True) and frozen is None and ft == np.float32
    wq = desc.get("w_quant", True)
    P = params
    rec = {}
    c = dict(rec=rec)
    h0 = np.asarray(h0, np.float64)
    cos, sin = rope_angles(T, S, d, desc["rope_base"])
    c.update(cos=cos, sin=sin)

    def site_input(x, k):
        s = P["s"][k] if let and k < 3 else None
        dl = P["delta"][k] if let and k < 3 else None
        xt = _let_x(x, s, dl, frozen, ft)
        xh = _act(xt, ab, frozen, f"act{k}", rec, ft, sym)
        c[f"xt{k}"] = xt
        return _op(xh, bf16)

    def linear(l, xop):
        k = SITE_OF[l]
        s = P["s"][k] if let and k < 3 else None
        W = np.asarray(P["W"][l], np.float64)
        wdq = _lwc(P["W"][l], P["gamma_logit"][l], P["beta_logit"][l], desc["w_bits"][l],
                   desc["w_group"][l], s, frozen, f"w{l}", rec, ft, wq)
        wop = _op(wdq, bf16)
        c[f"wop{l}"] = wop
        y = xop @ wop.T
        if let and k < 3:
            bt = W @ np.asarray(P["delta"][k], np.float64)          # B~ = delta W (Eq. 3)
            y = y + bt[None, :]
        return y

    # attention half
    x1, rstd1 = rmsnorm(h0, P["g1"], desc["norm_eps"])
    c.update(x1=x1, rstd1=rstd1)
    x1op = site_input(x1, 0)
    c["xop0"] = x1op
    q = rope(linear(0, x1op), H, d, cos, sin)
    kk = rope(linear(1, x1op), Hkv, d, cos, sin)
    v = linear(2, x1op)
    sa = np.asarray(P["s_a"], np.float64) if let else np.ones(Hkv * d)
    sa_q = np.tile(sa.reshape(Hkv, 1, d), (1, H // Hkv, 1)).reshape(H * d)
    qt = q / sa_q[None, :]
    kt = kk * sa[None, :]
    qh = _op(_act(qt, ab, frozen, "actq", rec, ft, sym), bf16)
    kh = _op(_act(kt, ab, frozen, "actk", rec, ft, sym), bf16)
    vh = _op(_act(v, ab, frozen, "actv", rec, ft, sym), bf16)
    pb = desc.get("softmax_bits", 16)
    att, probs, ph = attention(qh, kh, vh, H, Hkv, d, S, bf16, p_bits=pb, rec=rec, frozen=frozen,
                               ft=ft)
    c.update(qt=qt, kt=kt, v=v, qh=qh, kh=kh, vh=vh, probs=probs, ph=ph, sa=sa, sa_q=sa_q)
    x2op = site_input(att, 1)
    c.update(x2=att, xop1=x2op)
    h1 = h0 + linear(3, x2op)
    # feed-forward half
    x3, rstd2 = rmsnorm(h1, P["g2"], desc["norm_eps"])
    c.update(h1=h1, x3=x3, rstd2=rstd2)
    x3op = site_input(x3, 2)
    c["xop2"] = x3op
    gate = linear(4, x3op)
    up = linear(5, x3op)
    x4 = silu(gate) * up
    c.update(gate=gate, up=up, x4=x4)
    x4op = site_input(x4, 3)
    c["xop3"] = x4op
    h2 = h1 + linear(6, x4op)
    R = h2 - np.asarray(target, np.float64)
    n = T * D
    loss = float(np.sum(R * R)) / n
    c.update(h2=h2, R=R, n=n)
    return loss, c


def block_step(desc, h0, target, params, ft=np.float32):
    """Loss and straight-through gradients of one calibration step over the
    whole block (Algorithm 1's inner loop body).  Returns (loss, grads) with
    grads = {"d_gamma_logit": [7], "d_beta_logit": [7], "d_s": [3],
    "d_delta": [3], "d_s_a": [Hkv d] | None}."""
    D, H, Hkv = desc["hidden"], desc["heads"], desc["kv_heads"]
    d = D // H
    S = desc["seq_len"]
    ab = desc["act_bits"]
    let = desc["let"]
    bf16 = desc.get("bf16", True) and ft == np.float32
    P = params
    loss, c = block_forward(desc, h0, target, params, ft=ft)
    rec = c["rec"]
    dgl, dbl = [None] * 7, [None] * 7
    ds = [np.zeros(D), np.zeros(H * d), np.zeros(D)]
    dd = [np.zeros(D), np.zeros(H * d), np.zeros(D)]

    def linear_bwd(l, dy):
        """dy [T, C_out] (bf16 operand when bf16): returns dL/dX^ and fills
        the clipping and weight/bias-path LET gradients."""
        k = SITE_OF[l]
        dyop = _op(dy, bf16)
        xop = c[f"xop{k}"]
        dW = dyop.T @ xop
        g = lwc_bwd(rec[f"w{l}"], dW, W=P["W"][l], with_s=let and k < 3)
        dgl[l], dbl[l] = g["d_gamma_logit"], g["d_beta_logit"]
        if let and k < 3:
            ds[k] += g["d_s"]
            dd[k] += np.sum(dyop, axis=0) @ np.asarray(P["W"][l], np.float64)
        return dyop @ c[f"wop{l}"]

    def site_bwd(k, dxh):
        """From dL/dX^ of a site to dL/dX (through Q_a and the LET transform)."""
        dxt = _act_bwd(dxh, ab, f"act{k}", rec)
        if let and k < 3:
            s = np.asarray(P["s"][k], np.float64)
            ds[k] -= np.sum(dxt * c[f"xt{k}"], axis=0) / s
            dd[k] -= np.sum(dxt, axis=0) / s
            return dxt / s[None, :]
        return dxt

    dh2 = 2.0 * c["R"] / c["n"]
    # feed-forward half
    dx4 = site_bwd(3, linear_bwd(6, dh2))
    gate, up = c["gate"], c["up"]
    dgate = dx4 * up * silu_grad(gate)
    dup = dx4 * silu(gate)
    dx3h = linear_bwd(4, dgate) + linear_bwd(5, dup)
    dx3 = site_bwd(2, dx3h)
    dh1 = dh2 + rmsnorm_bwd(c["h1"], P["g2"], c["rstd2"], dx3)
    # attention half
    datt = site_bwd(1, linear_bwd(3, dh1))
    # dO enters the attention backward's products (dP = dO V^T, dV = P^T dO)
    dqh, dkh, dvh = attention_bwd(c["qh"], c["kh"], c["vh"], c["probs"], _op(datt, bf16), H, Hkv,
                                  d, S, bf16, PH=c["ph"], rec=rec)
    dqt = _act_bwd(dqh, ab, "actq", rec)
    dkt = _act_bwd(dkh, ab, "actk", rec)
    dv = _act_bwd(dvh, ab, "actv", rec)
    sa, sa_q = c["sa"], c["sa_q"]
    c.update(dqt=dqt, dkt=dkt)
    dsa = None
    if let:
        # Q~ = q / s_a: dQ~/ds_a = -Q~ / s_a;  K~ = k s_a: dK~/ds_a = K~ / s_a
        dq_sa = -np.sum(dqt * c["qt"], axis=0) / sa_q
        dsa = np.sum(dkt * c["kt"], axis=0) / sa + dq_sa.reshape(Hkv, H // Hkv, d).sum(axis=1).reshape(-1)
    dq = rope(dqt / sa_q[None, :], H, d, c["cos"], c["sin"], inverse=True)
    dk = rope(dkt * sa[None, :], Hkv, d, c["cos"], c["sin"], inverse=True)
    dx1h = linear_bwd(0, dq) + linear_bwd(1, dk) + linear_bwd(2, dv)
    site_bwd(0, dx1h)
    out = dict(d_gamma_logit=dgl, d_beta_logit=dbl,
               d_s=ds if let else [None] * 3, d_delta=dd if let else [None] * 3, d_s_a=dsa,
               cache=c)
    return loss, out


def freeze(desc, h0, target, params):
    """Every discrete choice of the block's quantisers at ``params``, from the
    fp64 forward (the frozen-selection surrogate of the straight-through
    gradients)."""
    _, c = block_forward(desc, h0, target, params, ft=np.float64)
    return {k: _frozen_variant(st, None) if st.get("sym") else _frozen_choices(st)
            for k, st in c["rec"].items()}


def surrogate_loss(desc, h0, target, params, frozen):
    """fp64 loss with every quantiser choice frozen."""
    loss, _ = block_forward(desc, h0, target, params, frozen=frozen)
    return loss


def fp_block(desc, h0, params):
    """The full-precision block (Algorithm 1's target x_fp = B(x_fp)): no
    quantiser, no LET (fp64)."""
    d2 = dict(desc, act_bits=16, let=False, bf16=False)
    D, H, Hkv = d2["hidden"], d2["heads"], d2["kv_heads"]
    d = D // H
    S = d2["seq_len"]
    T = h0.shape[0]
    W = [np.asarray(w, np.float64) for w in params["W"]]
    cos, sin = rope_angles(T, S, d, d2["rope_base"])
    h0 = np.asarray(h0, np.float64)
    x1, _ = rmsnorm(h0, params["g1"], d2["norm_eps"])
    q = rope(x1 @ W[0].T, H, d, cos, sin)
    k = rope(x1 @ W[1].T, Hkv, d, cos, sin)
    v = x1 @ W[2].T
    att, _, _ = attention(q, k, v, H, Hkv, d, S)
    h1 = h0 + att @ W[3].T
    x3, _ = rmsnorm(h1, params["g2"], d2["norm_eps"])
    x4 = silu(x3 @ W[4].T) * (x3 @ W[5].T)
    return h1 + x4 @ W[6].T


# ---------------------------------------------------------------- Algorithm 1 over a stack
def _adam_update(params, grads, mom, step, lr_lwc, lr_let):
    """One AdamW step (oracle.adamw, fp64, stored back as fp32) on every
    trained tensor: the clipping logits at lr_lwc, s, delta and s_a at
    lr_let."""
    from .adamw import adamw
    pairs = [("gamma_logit", "d_gamma_logit", lr_lwc), ("beta_logit", "d_beta_logit", lr_lwc),
             ("s", "d_s", lr_let), ("delta", "d_delta", lr_let)]
    for pk, gk, lr in pairs:
        for i, g in enumerate(grads[gk]):
            if g is None:
                continue
            key = (pk, i)
            m, v = mom.get(key, (0.0, 0.0))
            p, m, v = adamw(params[pk][i], g, m, v, step, lr)
            params[pk][i] = p.astype(np.float32)
            mom[key] = (m, v)
    if grads["d_s_a"] is not None:
        m, v = mom.get("s_a", (0.0, 0.0))
        p, m, v = adamw(params["s_a"], grads["d_s_a"], m, v, step, lr_let)
        params["s_a"] = p.astype(np.float32)
        mom["s_a"] = (m, v)


def algorithm1(desc, blocks, samples, epochs, lr_lwc=5e-3, lr_let=1e-2):
    """Algorithm 1 over a stack of blocks, calibrated one after another.

    ``blocks``: per block a params dict as block_step takes (W, g1, g2 and the
    initial clipping logits, s, delta, s_a); ``samples``: the calibration
    inputs, one [seq_len, D] array per sample (batch size 1).  Block i is
    trained against its full-precision output on the full-precision stream
    (the targets, rounded to bf16 as the kernels store them), from the
    quantised stream as input, for ``epochs`` passes over the samples in
    order with one AdamW step per sample (a fresh AdamW state per block);
    then both streams move on: the full-precision stream through the block
    unquantised (the targets), the quantised one through the block with its
    learned parameters (bf16).
    Returns (losses [blocks][epochs * samples], trained params per block,
    final quantised stream)."""
    x_fp = [np.asarray(x, np.float64) for x in samples]
    x_q = [np.asarray(x, np.float64) for x in samples]
    losses, trained = [], []
    for params in blocks:
        P = {k: (list(v) if isinstance(v, list) else v) for k, v in params.items()}
        targets = [bf16_round(fp_block(desc, x, P)) for x in x_fp]
        mom, step = {}, 0              # a fresh optimizer for every block
        block_losses = []
        for _ in range(epochs):
            for j in range(len(samples)):
                step += 1
                loss, g = block_step(desc, x_q[j], targets[j], P)
                block_losses.append(loss)
                _adam_update(P, g, mom, step, lr_lwc, lr_let)
        x_q = [bf16_round(block_forward(desc, x, t, P)[1]["h2"]) for x, t in zip(x_q, targets)]
        x_fp = targets
        losses.append(block_losses)
        trained.append(P)
    return losses, trained, x_q
