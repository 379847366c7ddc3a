"""GPU parity where max/min ties decide the gradient (reading: the lowest index
in the group or token row takes the whole max/min gradient).

Weights and activations are drawn on coarse grids, so every group and token
row holds its largest and its smallest value several times, and the extreme
values are also copied to the far end and the middle of each group or row,
so tied copies sit in different lanes, chunks and waves.  LET scales are
powers of two and shifts are grid values, so the transformed values W~ = s W
and X~ = (X - delta)/s tie exactly as well.  Every element of dW~ and dX~
is compared with the oracle, next to the clipping-logit and LET gradients."""
import numpy as np
import pytest
import torch

from oracle.block import block_step, fp_target
from oracle.let import let_x
from oracle.quant import act_bwd, act_fwd, lwc_bwd, lwc_fwd
from paper_2308_13137_amd import oq
from tests.cases import bf16_exact, dev, elemwise, normwise, quant_grad_bounds, within

pytestmark = pytest.mark.gpu

TOL_FP32 = 1e-5


def host(t):
    return t.detach().float().cpu().numpy()


def grid_ties(rng, rows, cols, group, step, span, s=None, delta=None, bf16=True):
    """[rows, cols] values k*step (|k| <= span), with each group's transformed
    max copied to its last element and to the one a quarter in, and its min
    to its middle element and to the one three quarters in.  With s
    (powers of two) and delta (grid values) the copies are planted in the
    transformed values t = (v - delta)/s resp. v*s, so those tie too."""
    v = rng.integers(-span, span + 1, (rows, cols)).astype(np.float32) * np.float32(step)
    if bf16:
        v = bf16_exact(v)
    ng = cols // group
    q1, mid, q3, last = group // 4, group // 2, 3 * group // 4, group - 1
    for g in range(ng):
        c0 = g * group
        blk = v[:, c0:c0 + group]
        if delta is not None:                        # activation: t = (v - delta) / s
            t = (blk - delta[c0:c0 + group]) / s[c0:c0 + group]
        elif s is not None:                          # weight: t = v * s
            t = blk * s[c0:c0 + group]
        else:
            t = blk
        tmx, tmn = t.max(axis=1), t.min(axis=1)
        for j, tv in ((last, tmx), (q1, tmx), (mid, tmn), (q3, tmn)):
            c = c0 + j
            if delta is not None:
                blk[:, j] = tv * s[c] + delta[c]
            elif s is not None:
                blk[:, j] = tv / s[c]
            else:
                blk[:, j] = tv
    return v


def pow2_scales(rng, n):
    return np.float32(2.0) ** rng.integers(-1, 2, n).astype(np.float32)


LWC_TIE_CASES = [
    dict(c_out=64, c_in=4096, group=128, bits=3, let=False),      # run kernel, dW~ output
    dict(c_out=48, c_in=4096, group=128, bits=4, let=True),       # grouped with LET, ds partials
    dict(c_out=40, c_in=4096, group=4096, bits=4, let=True),      # whole row with LET
    dict(c_out=24, c_in=11008, group=11008, bits=4, let=False),   # whole row, many chunks per lane
    dict(c_out=32, c_in=1024, group=64, bits=2, let=False, bf16=False),
    dict(c_out=16, c_in=512, group=32, bits=8, let=True),
    dict(c_out=20, c_in=2048, group=512, bits=5, let=True),
]


@pytest.mark.parametrize("case", LWC_TIE_CASES, ids=[str(c) for c in LWC_TIE_CASES])
def test_lwc_ties(case):
    print(f"lwc ties {case}", flush=True)
    rng = np.random.default_rng(case["c_in"] * 3 + case["group"] + case["bits"])
    bf16 = case.get("bf16", True)
    s = pow2_scales(rng, case["c_in"]) if case["let"] else None
    W = grid_ties(rng, case["c_out"], case["c_in"], case["group"], 0.01, 6, s=s, bf16=bf16)
    ng = case["c_in"] // case["group"]
    gl = rng.uniform(1.0, 6.0, (case["c_out"], ng)).astype(np.float32)
    bl = rng.uniform(1.0, 6.0, (case["c_out"], ng)).astype(np.float32)
    G = rng.standard_normal(W.shape).astype(np.float32)
    st = lwc_fwd(W, gl, bl, case["bits"], case["group"], s=s)
    # the construction really ties: every group's max and min occur twice or more
    wt = st["wt"].reshape(-1, case["group"])
    assert np.all(np.sum(wt == wt.max(axis=1, keepdims=True), axis=1) >= 2)
    assert np.all(np.sum(wt == wt.min(axis=1, keepdims=True), axis=1) >= 2)
    ref = lwc_bwd(st, G, W=W, with_s=True)
    dt = torch.bfloat16 if bf16 else torch.float32
    sd = None if s is None else dev(s)
    _, codes, h, z = oq.lwc_fakequant_fwd(dev(W, dt), dev(gl), dev(bl), case["bits"], case["group"],
                                          s=sd, dq_dtype=torch.float32)
    assert np.array_equal(codes.cpu().numpy(), st["codes"])
    assert np.array_equal(host(h), st["h_g"]) and np.array_equal(host(z), st["z_g"])
    dg, db, ds, dwt = oq.lwc_fakequant_bwd(dev(W, dt), dev(gl), dev(bl), case["bits"], case["group"],
                                           dev(G), s=sd, want_d_s=True, want_dW_tilde=True)
    bx, bg, bb = quant_grad_bounds(st, G)
    # every element not holding a max/min gradient is exactly g*m
    routed = np.zeros(st["q"].shape, bool)
    routed[np.arange(routed.shape[0]), st["i_mx"]] = True
    routed[np.arange(routed.shape[0]), st["i_mn"]] = True
    routed = routed.reshape(W.shape)
    plain = (G.astype(np.float64) * st["m"].reshape(W.shape))
    assert np.array_equal(host(dwt)[~routed], plain[~routed].astype(np.float32))
    r_w = within(host(dwt), ref["dW_tilde"], bx.reshape(W.shape), "dW~")
    r_g = within(host(dg), ref["d_gamma_logit"], bg.reshape(dg.shape), "d_gamma_logit")
    r_b = within(host(db), ref["d_beta_logit"], bb.reshape(db.shape), "d_beta_logit")
    e_s = normwise(host(ds), ref["d_s"])
    print(f"  error/bound: dW~ {r_w:.2e}  dgl {r_g:.2e}  dbl {r_b:.2e};  ds {e_s:.2e}", flush=True)
    assert e_s < TOL_FP32


ACT_TIE_CASES = [
    dict(T=300, C=4096, bits=4, let=True),
    dict(T=64, C=11008, bits=4, let=True),
    dict(T=2500, C=2048, bits=3, let=False),       # several rows per workgroup (row pipeline)
    dict(T=50, C=256, bits=6, let=True, bf16=False),
    dict(T=40, C=1000, bits=8, let=False),
]


@pytest.mark.parametrize("case", ACT_TIE_CASES, ids=[str(c) for c in ACT_TIE_CASES])
def test_act_ties(case):
    print(f"act ties {case}", flush=True)
    rng = np.random.default_rng(case["T"] + case["C"] + case["bits"])
    bf16 = case.get("bf16", True)
    s = d = None
    if case["let"]:
        s = pow2_scales(rng, case["C"])
        d = (rng.integers(-2, 3, case["C"]) * 0.25).astype(np.float32)
    X = grid_ties(rng, case["T"], case["C"], case["C"], 0.25, 12, s=s, delta=d, bf16=bf16)
    xt = let_x(X, s, d) if case["let"] else X
    assert np.all(np.sum(xt == xt.max(axis=1, keepdims=True), axis=1) >= 2)
    assert np.all(np.sum(xt == xt.min(axis=1, keepdims=True), axis=1) >= 2)
    G = rng.standard_normal(X.shape).astype(np.float32)
    st = act_fwd(xt, case["bits"])
    dxt = act_bwd(st, G)
    sv = np.ones(case["C"]) if s is None else s.astype(np.float64)
    ref_ds = -np.sum(dxt * xt, axis=0) / sv
    ref_dd = -np.sum(dxt, axis=0) / sv
    dt = torch.bfloat16 if bf16 else torch.float32
    sd = None if s is None else dev(s)
    dd_ = None if d is None else dev(d)
    _, codes, h, z = oq.act_fakequant_fwd(dev(X, dt), case["bits"], s=sd, delta=dd_,
                                          dq_dtype=torch.float32)
    assert np.array_equal(codes.cpu().numpy(), st["codes"])
    gx, ds, dd = oq.act_fakequant_bwd(dev(X, dt), case["bits"], dev(G), s=sd, delta=dd_)
    bx, _, _ = quant_grad_bounds(st, G)
    routed = np.zeros(X.shape, bool)
    routed[np.arange(X.shape[0]), st["i_mx"]] = True
    routed[np.arange(X.shape[0]), st["i_mn"]] = True
    plain = G.astype(np.float64) * st["m"]
    assert np.array_equal(host(gx)[~routed], plain[~routed].astype(np.float32))
    r_x = within(host(gx), dxt, bx, "dX~")
    e_s = normwise(host(ds), ref_ds)
    e_d = normwise(host(dd), ref_dd)
    print(f"  error/bound: dX~ {r_x:.2e};  ds {e_s:.2e}  ddelta {e_d:.2e}", flush=True)
    assert e_s < TOL_FP32 and e_d < TOL_FP32


@pytest.mark.parametrize("act_bits", [4, 16])
def test_block_step_with_ties(act_bits):
    """A whole LET block step on tie-heavy weights and activations: the LET
    gradients collect the weight-path (dW~) and input-path (dX~) tie routing."""
    print(f"block ties act_bits={act_bits}", flush=True)
    rng = np.random.default_rng(900 + act_bits)
    T, hid, ffn = 256, 512, 1024
    sites = [dict(width=hid, let=True, act_bits=act_bits), dict(width=ffn, let=False, act_bits=16)]
    lins = [dict(site=0, c_out=hid, bits=4, group=128), dict(site=0, c_out=256, bits=4, group=hid),
            dict(site=1, c_out=hid, bits=3, group=128)]
    s0 = pow2_scales(rng, hid)
    d0 = (rng.integers(-2, 3, hid) * 0.25).astype(np.float32)
    X = [grid_ties(rng, T, hid, hid, 0.25, 12, s=s0, delta=d0),
         grid_ties(rng, T, ffn, ffn, 0.25, 12)]
    W = [grid_ties(rng, l["c_out"], sites[l["site"]]["width"], l["group"], 0.01, 6,
                   s=s0 if l["site"] == 0 else None) for l in lins]
    gl = [rng.uniform(1.0, 6.0, (l["c_out"], sites[l["site"]]["width"] // l["group"])).astype(np.float32)
          for l in lins]
    bl = [rng.uniform(1.0, 6.0, g.shape).astype(np.float32) for g in gl]
    Y = [fp_target(X[l["site"]] + 0.03, W[i], None, bf16=True) for i, l in enumerate(lins)]
    desc = dict(T=T, bf16=True, sites=sites, linears=lins)
    params = dict(W=W, B=[None] * 3, gamma_logit=gl, beta_logit=bl, s=[s0, None], delta=[d0, None])
    ref_loss, ref = block_step(desc, X, Y, params)
    blk = oq.Block(T, [(s_["width"], s_["let"], s_["act_bits"]) for s_ in sites],
                   [(l["site"], l["c_out"], l["bits"], l["group"]) for l in lins])
    b16 = torch.bfloat16
    loss = float(blk.step([dev(x, b16) for x in X], [dev(np.ascontiguousarray(y.T), b16) for y in Y],
                          [dev(w, b16) for w in W], [dev(g) for g in gl], [dev(b) for b in bl],
                          s=[dev(s0), None], delta=[dev(d0), None]).cpu())
    errs = {"loss": abs(loss - ref_loss) / abs(ref_loss),
            "ds": elemwise(host(blk.d_s[0]), ref["d_s"][0], floor=1e-2),
            "dd": elemwise(host(blk.d_delta[0]), ref["d_delta"][0], floor=1e-2)}
    for i in range(len(lins)):
        errs[f"dgl{i}"] = elemwise(host(blk.d_gamma[i]), ref["d_gamma_logit"][i], floor=1e-2)
        errs[f"dbl{i}"] = elemwise(host(blk.d_beta[i]), ref["d_beta_logit"][i], floor=1e-2)
    print("  " + "  ".join(f"{k} {v:.2e}" for k, v in errs.items()), flush=True)
    assert max(errs.values()) < 2e-2, errs
